"""Seeded synthetic workloads for the compression hot path.

This module holds tensor-shape recipes and seeded input generators only: no
part of the compression method's arithmetic lives here.  Sizes that depend
on the method (the number of sparse entries per tensor, the number of sign
words per tensor) are passed in by the caller.

The paper trains VGG16, ResNet101, UGATIT, BERT-base, GPT2 and LSTM on real
datasets (paper Sec. 5.1, benchmark-model table); no dataset or trained
weight is used here.  Instead every gradient tensor is drawn from a normal
distribution whose scale is itself random per tensor, with the tensor shapes
of the model families named by each workload.  Randomness comes from numpy's
PCG64 seeded by SeedSequence([2205, workload, tensor_id, role]) with
role 0 = gradient, 1 = residual, 2 = per-tensor scale, 3 + w = worker w.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

ROLE_G, ROLE_E, ROLE_SIGMA, ROLE_WORKER = 0, 1, 2, 3
SEED = 14465  # API seed used for random-k and the threshold sample


def rng_for(workload: int, tid: int, role: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([2205, workload, tid, role])))


# ------------------------------------------------------------------ shapes

def resnet50_shapes():
    """ResNet-50: 7x7 stem conv + BN, bottleneck stages [3, 4, 6, 3] of
    widths 64/128/256/512 (expansion 4, 1x1 downsample + BN on each stage's
    first block), then the 1000-way classifier.  161 tensors."""
    shapes = [(64, 3, 7, 7), (64,), (64,)]
    cin = 64
    for width, blocks in zip((64, 128, 256, 512), (3, 4, 6, 3)):
        for b in range(blocks):
            shapes += [(width, cin, 1, 1), (width,), (width,),
                       (width, width, 3, 3), (width,), (width,),
                       (4 * width, width, 1, 1), (4 * width,), (4 * width,)]
            if b == 0:
                shapes += [(4 * width, cin, 1, 1), (4 * width,), (4 * width,)]
            cin = 4 * width
    shapes += [(1000, 2048), (1000,)]
    return shapes


def bert_base_shapes():
    """BERT-base: word/position/token-type embeddings + LayerNorm, 12 layers
    of Q/K/V/O projections with biases, attention-output LayerNorm, FFN
    768->3072->768 with biases and output LayerNorm, then the pooler.
    199 tensors."""
    d, f = 768, 3072
    shapes = [(30522, d), (512, d), (2, d), (d,), (d,)]
    for _ in range(12):
        for _q in range(4):
            shapes += [(d, d), (d,)]
        shapes += [(d,), (d,)]
        shapes += [(f, d), (f,), (d, f), (d,)]
        shapes += [(d,), (d,)]
    shapes += [(d, d), (d,)]
    return shapes


def gpt2_xl_shapes():
    """GPT-2-XL: 50257x1600 token embedding, 1024x1600 position table,
    48 blocks of (LN, fused QKV 1600x4800, projection, LN, MLP 1600->6400
    ->1600 with biases), final LN.  580 tensors."""
    d, f = 1600, 6400
    shapes = [(50257, d), (1024, d)]
    for _ in range(48):
        shapes += [(d,), (d,), (d, 3 * d), (3 * d,), (d, d), (d,),
                   (d,), (d,), (d, f), (f,), (f, d), (d,)]
    shapes += [(d,), (d,)]
    return shapes


def many_small_sizes(count=4096, lo=768, hi=65536, workload=5):
    """Sizes floor(exp(U(ln lo, ln hi))), one draw per tensor."""
    out = []
    for t in range(count):
        u = rng_for(workload, t, ROLE_SIGMA).uniform(math.log(lo), math.log(hi))
        out.append(int(math.floor(math.exp(u))))
    return out


def numel(shape):
    n = 1
    for s in shape:
        n *= int(s)
    return n


# --------------------------------------------------------------- workloads

@dataclass
class Workload:
    """One tensor set plus the aggregation fan-in it is measured with."""
    wid: int
    name: str
    kind: str              # "topk" | "topk_sampled" | "randk" | "sign" | "terngrad" | "qsgd4" | "qsgd8"
    ratio: float
    W: int
    sizes: list = field(default_factory=list)
    grad_dtype: str = "float32"
    sigma_mode: str = "loguniform"   # or "fixed:<sigma>"
    resid_mode: str = "tenth"        # "zero" | "tenth" | "fixed:<sigma>"
    momentum: float = 0.0            # > 0: DGC momentum correction and masking

    @property
    def T(self):
        return len(self.sizes)

    @property
    def n_total(self):
        return int(sum(self.sizes))

    @property
    def slug(self):
        """Short file-name form of the workload."""
        return {1: "single2p20_topk_w8", 2: "resnet50_sign_w64", 3: "bertbase_topksampled_w64",
                4: "gpt2xl_randk_w16", 5: "small4096_fp16sign_w32", 6: "resnet50_terngrad_w64",
                7: "bertbase_qsgd8_w16", 8: "bertbase_qsgd4_w32", 9: "bertbase_dgc_w64"}[self.wid]


def workload(wid: int, shrink: int = 1) -> Workload:
    """The measured workloads (1-5: the hot path's five operator configs;
    6-8: the stochastic quantizers on the same model shapes; 9: DGC's
    momentum correction around the sampled top-k); `shrink` > 1
    divides every tensor size (at least 1 element) for fast parity runs of
    the same structure."""
    def s(ns):
        return [max(1, n // shrink) for n in ns]
    if wid == 1:
        return Workload(1, "single 2^20 fp32 tensor, exact top-k 1%, W=8", "topk", 0.01, 8,
                        s([1 << 20]), "float32", "fixed:0.01", "zero")
    if wid == 2:
        return Workload(2, "ResNet-50 gradients (161 fp32 tensors, 25.6M), sign+EF, W=64", "sign",
                        0.01, 64, s([numel(x) for x in resnet50_shapes()]))
    if wid == 3:
        return Workload(3, "BERT-base gradients (199 fp32 tensors, 109.5M), sampled top-k 1%, W=64",
                        "topk_sampled", 0.01, 64, s([numel(x) for x in bert_base_shapes()]))
    if wid == 4:
        return Workload(4, "GPT-2-XL gradients (580 fp32 tensors, 1.56B), random-k 1%, W=16",
                        "randk", 0.01, 16, s([numel(x) for x in gpt2_xl_shapes()]))
    if wid == 5:
        return Workload(5, "4096 small fp16 tensors (768..65536, ~60M), sign+fp32 EF, W=32", "sign",
                        0.01, 32, s(many_small_sizes()), "float16", "fixed:1e-3", "fixed:1e-4")
    if wid == 6:
        return Workload(6, "ResNet-50 gradients (161 fp32 tensors, 25.6M), TernGrad 2-bit+EF, W=64",
                        "terngrad", 0.01, 64, s([numel(x) for x in resnet50_shapes()]))
    if wid == 7:
        return Workload(7, "BERT-base gradients (199 fp32 tensors, 109.5M), QSGD 8-bit+EF, W=16",
                        "qsgd8", 0.01, 16, s([numel(x) for x in bert_base_shapes()]))
    if wid == 8:
        return Workload(8, "BERT-base gradients (199 fp32 tensors, 109.5M), QSGD 4-bit+EF, W=32",
                        "qsgd4", 0.01, 32, s([numel(x) for x in bert_base_shapes()]))
    if wid == 9:
        return Workload(9, "BERT-base gradients (199 fp32 tensors, 109.5M), DGC: momentum 0.9 correction and "
                           "masking around sampled top-k 1%, W=64", "topk_sampled", 0.01, 64,
                        s([numel(x) for x in bert_base_shapes()]), momentum=0.9)
    raise ValueError(wid)


QUANT_BITS = {"terngrad": 2, "qsgd4": 4, "qsgd8": 8}
WORD_KINDS = ("sign", "terngrad", "qsgd4", "qsgd8")  # payload: packed words + one scale per tensor


def sigma_of(wl: Workload, tid: int) -> float:
    if wl.sigma_mode.startswith("fixed:"):
        return float(wl.sigma_mode.split(":")[1])
    return float(10.0 ** rng_for(wl.wid, tid, ROLE_SIGMA).uniform(-4.0, -1.0))


def gradient(wl: Workload, tid: int, tie_heavy: bool = False) -> np.ndarray:
    n = wl.sizes[tid]
    sig = sigma_of(wl, tid)
    rng = rng_for(wl.wid, tid, ROLE_G)
    if tie_heavy:
        levels = (np.arange(-8, 8, dtype=np.float64) + 0.5) * (sig / 4.0)
        x = levels[rng.integers(0, 16, size=n)]
    else:
        x = rng.standard_normal(n) * sig
    return x.astype(np.float16 if wl.grad_dtype == "float16" else np.float32)


def residual(wl: Workload, tid: int) -> np.ndarray:
    n = wl.sizes[tid]
    if wl.resid_mode == "zero":
        return np.zeros(n, np.float32)
    if wl.resid_mode.startswith("fixed:"):
        sig = float(wl.resid_mode.split(":")[1])
    else:
        sig = sigma_of(wl, tid) / 10.0
    return (rng_for(wl.wid, tid, ROLE_E).standard_normal(n) * sig).astype(np.float32)


def sparse_payload(wl: Workload, w: int, counts, offs):
    """Worker w's sparse payload: for tensor t, counts[t] distinct indices in
    [0, n_t), ascending, at offs[t], and values ~ N(0, sigma_t^2)."""
    total = int(offs[-1])
    idx = np.empty(total, np.uint32)
    val = np.empty(total, np.float32)
    for t, n in enumerate(wl.sizes):
        k = int(counts[t])
        rng = rng_for(wl.wid, t, ROLE_WORKER + w)
        sel = np.sort(rng.choice(n, size=k, replace=False)).astype(np.uint32)
        idx[offs[t]:offs[t] + k] = sel
        val[offs[t]:offs[t] + k] = (rng.standard_normal(k) * sigma_of(wl, t)).astype(np.float32)
    return idx, val


def sign_payload(wl: Workload, w: int, word_counts, offs):
    """Worker w's sign payload: uniformly random words (bits past the end of
    each tensor cleared) and scales sigma_t*sqrt(2/pi)*(1 + 0.05 N(0,1))."""
    total = int(offs[-1])
    bits = np.empty(total, np.uint32)
    scale = np.empty(wl.T, np.float32)
    for t, n in enumerate(wl.sizes):
        nw = int(word_counts[t])
        rng = rng_for(wl.wid, t, ROLE_WORKER + w)
        words = rng.integers(0, 1 << 32, size=nw, dtype=np.uint64).astype(np.uint32)
        tail = n - 32 * (nw - 1) if nw else 0
        if nw and tail < 32:
            words[-1] &= np.uint32((1 << tail) - 1)
        bits[offs[t]:offs[t] + nw] = words
        scale[t] = np.float32(sigma_of(wl, t) * math.sqrt(2.0 / math.pi)
                              * (1.0 + 0.05 * rng.standard_normal()))
    return bits, scale


def quant_payload(wl: Workload, w: int, word_counts, offs):
    """Worker w's quantizer payload: uniformly random b-bit codes (codes past
    the end of each tensor cleared) and scales 4 sigma_t (1 + 0.05 N(0,1)),
    about the largest magnitude of the tensor's normal draws."""
    b = QUANT_BITS[wl.kind]
    total = int(offs[-1])
    bits = np.empty(total, np.uint32)
    scale = np.empty(wl.T, np.float32)
    for t, n in enumerate(wl.sizes):
        rng = rng_for(wl.wid, t, ROLE_WORKER + w)
        bits[offs[t]:offs[t] + int(word_counts[t])] = random_code_words(rng, [n], [word_counts[t]], b)[0]
        scale[t] = np.float32(4.0 * sigma_of(wl, t) * (1.0 + 0.05 * rng.standard_normal()))
    return bits, scale


# ------------------------------------------------- generic test inputs

def random_sparse_lists(rng: np.random.Generator, ns, counts, sigma=1.0):
    """One worker's payload for arbitrary tensor sizes: counts[t] distinct
    ascending indices in [0, ns[t]) and N(0, sigma^2) values, concatenated."""
    idx = [np.sort(rng.choice(int(n), size=int(k), replace=False)).astype(np.uint32) if k else
           np.zeros(0, np.uint32) for n, k in zip(ns, counts)]
    val = [(rng.standard_normal(int(k)) * sigma).astype(np.float32) for k in counts]
    return idx, val


def random_sign_words(rng: np.random.Generator, ns, word_counts):
    """One worker's sign words for arbitrary tensor sizes (bits past each
    tensor's end cleared), one list entry per tensor."""
    out = []
    for n, nw in zip(ns, word_counts):
        w = rng.integers(0, 1 << 32, size=int(nw), dtype=np.uint64).astype(np.uint32)
        tail = int(n) - 32 * (int(nw) - 1) if nw else 0
        if nw and tail < 32:
            w[-1] &= np.uint32((1 << tail) - 1)
        out.append(w)
    return out


def random_code_words(rng: np.random.Generator, ns, word_counts, bits):
    """One worker's packed b-bit code words for arbitrary tensor sizes (codes
    past each tensor's end cleared), one list entry per tensor."""
    out = []
    for n, nw in zip(ns, word_counts):
        w = rng.integers(0, 1 << 32, size=int(nw), dtype=np.uint64).astype(np.uint32)
        used = int(n) * bits % 32
        if nw and used:
            w[-1] &= np.uint32((1 << used) - 1)
        out.append(w)
    return out


# --------------------------------------------- on-device generation (large)
# For the 1.56B-element workload, drawing every input with numpy on the host
# takes minutes; these generators draw the same distributions on the device
# with torch's seeded generator.  A sparse worker payload of tensor t is a
# uniformly random k-subset of [0, n_t): k + k/32 + 64 indices drawn with
# replacement, their distinct values, and a uniformly random k of those
# (redrawn in the rare case of fewer than k distinct values); every k-subset
# is equally likely, since each step treats all indices alike.

def _torch_gen(device, *key):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(np.random.SeedSequence([2205, *key]).generate_state(1, np.uint64)[0] >> 1))
    return g


def device_gradient(wl: Workload, tid: int, out, gen):
    import torch
    n = wl.sizes[tid]
    x = torch.randn(n, generator=gen, device=out.device, dtype=torch.float32) * sigma_of(wl, tid)
    out.copy_(x.to(out.dtype))


def device_residual(wl: Workload, tid: int, out, gen):
    import torch
    n = wl.sizes[tid]
    if wl.resid_mode == "zero":
        out.zero_()
        return
    sig = float(wl.resid_mode.split(":")[1]) if wl.resid_mode.startswith("fixed:") else sigma_of(wl, tid) / 10.0
    out.copy_(torch.randn(n, generator=gen, device=out.device, dtype=torch.float32) * sig)


def device_sparse_payload(wl: Workload, w: int, counts, offs, device):
    import torch
    gen = _torch_gen(device, wl.wid, w, ROLE_WORKER)
    total = int(offs[-1])
    idx = torch.empty(total, dtype=torch.int64, device=device)
    val = torch.empty(total, dtype=torch.float32, device=device)
    for t, n in enumerate(wl.sizes):
        k = int(counts[t])
        if k == 0:
            continue
        if k == n:
            sel = torch.arange(n, device=device, dtype=torch.int64)
        else:
            while True:
                x = torch.randint(0, n, (k + k // 32 + 64,), generator=gen, device=device, dtype=torch.int64)
                u = torch.unique(x)
                if u.numel() >= k:
                    break
            pick = torch.randperm(u.numel(), generator=gen, device=device)[:k]
            sel = torch.sort(u[pick]).values
        idx[offs[t]:offs[t] + k] = sel
        val[offs[t]:offs[t] + k] = torch.randn(k, generator=gen, device=device) * sigma_of(wl, t)
    return idx.to(torch.int32), val


HOST_GEN_LIMIT = 200_000_000  # elements; larger workloads draw their inputs on the device


def device_inputs(wl, off, device):
    """Device-resident inputs of a workload: gradients and residuals as views
    of one flat buffer each (256-byte aligned tensors, as a framework's
    gradient buckets would be), the W worker payloads and the aggregate
    outputs.  Workloads above HOST_GEN_LIMIT elements draw on the device."""
    import torch
    kind = wl.kind
    on_device = wl.n_total > HOST_GEN_LIMIT
    tdt = torch.float16 if wl.grad_dtype == "float16" else torch.float32
    # gradients and residuals live in one flat buffer each, tensors as views
    # at 256-byte aligned offsets (as a framework's gradient buckets would)
    starts, pos = [], 0
    for n in wl.sizes:
        starts.append(pos)
        pos += (n + 63) // 64 * 64
    g_flat = torch.empty(pos, dtype=tdt, device=device)
    e_flat = torch.empty(pos, dtype=torch.float32, device=device)
    gen = _torch_gen(device, wl.wid, 0, ROLE_G) if on_device else None
    for t, n in enumerate(wl.sizes):
        if on_device:
            device_gradient(wl, t, g_flat[starts[t]:starts[t] + n], gen)
            device_residual(wl, t, e_flat[starts[t]:starts[t] + n], gen)
        else:
            g_flat[starts[t]:starts[t] + n].copy_(torch.from_numpy(gradient(wl, t)))
            e_flat[starts[t]:starts[t] + n].copy_(torch.from_numpy(residual(wl, t)))
    grads = [g_flat[s:s + n] for s, n in zip(starts, wl.sizes)]
    resids = [e_flat[s:s + n] for s, n in zip(starts, wl.sizes)]
    counts = [int(off[t + 1] - off[t]) for t in range(wl.T)]
    payloads = []
    for w in range(wl.W):
        if kind in WORD_KINDS:
            b, s = (sign_payload if kind == "sign" else quant_payload)(wl, w, counts, off)
            payloads.append({"bits": torch.from_numpy(b.view(np.int32)).to(device),
                             "scale": torch.from_numpy(s).to(device)})
        elif on_device:
            i, v = device_sparse_payload(wl, w, counts, off, device)
            payloads.append({"idx": i, "val": v})
        else:
            i, v = sparse_payload(wl, w, counts, off)
            payloads.append({"idx": torch.from_numpy(i.view(np.int32)).to(device),
                             "val": torch.from_numpy(v).to(device)})
    out_flat = torch.empty(pos, dtype=torch.float32, device=device)
    outs = [out_flat[s:s + n] for s, n in zip(starts, wl.sizes)]
    return grads, resids, payloads, outs
