"""Parity at the five workloads' full sizes, in the launch configuration
bench.py times: one compress call over the whole tensor list and one
aggregate call over all W generated payloads, on the same device-resident
inputs.  The oracle then recomputes a sample of tensors one by one (their
payloads, residuals and aggregates; sign aggregates on element windows,
since each output element depends only on its own bits and the scales),
and every tensor's payload is checked against the properties that hold at
any size."""
import numpy as np
import pytest

import oracle as O
from paper_2205_14465_amd import workloads as WL
from tests.helpers import bits, sign_tolerances

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _sample(wl, rng, extra=4):
    """Tensors the oracle recomputes: the first two, the last two, the
    largest, the smallest, and a few seeded picks."""
    T = wl.T
    sizes = np.array(wl.sizes)
    pick = {0, min(1, T - 1), T - 1, max(T - 2, 0), int(sizes.argmax()), int(sizes.argmin())}
    pick |= set(int(x) for x in rng.choice(T, size=min(extra, T), replace=False))
    return sorted(pick)


def _run(wid):
    import torch
    from paper_2205_14465_amd import binding as B
    wl = WL.workload(wid)
    dev = torch.device("cuda:0")
    off = B.bytecomp_layout(wl.kind, wl.ratio, wl.sizes)
    grads, resids, payloads, outs = WL.device_inputs(wl, off, dev)
    rng = np.random.default_rng(1000 + wid)
    sample = _sample(wl, rng)
    g_host = {t: grads[t].cpu().numpy() for t in sample}
    e_host = {t: resids[t].cpu().numpy().copy() for t in sample}
    own = B.alloc_payload(wl.kind, wl.ratio, wl.sizes, device=dev)
    ws = B.alloc_workspace(wl.kind, wl.ratio, wl.sizes, wl.W, device=dev)
    stream = torch.cuda.current_stream()
    alpha = 1.0 / wl.W
    B.CompressCall(wl.kind, wl.ratio, grads, resids, own, ws, stream=stream)(WL.SEED)
    B.AggregateCall(wl.kind, wl.ratio, payloads, wl.sizes, outs, alpha, ws, stream=stream)()
    torch.cuda.synchronize()
    assert B.bytecomp_device_status(ws) == 0
    return wl, off, grads, resids, payloads, outs, own, sample, g_host, e_host, alpha


def _check_sparse_payload_properties(wl, off, own):
    """Every tensor: exactly k_t indices, strictly ascending, in range."""
    idx = own["idx"].cpu().numpy().view(np.uint32)
    for t, n in enumerate(wl.sizes):
        seg = idx[off[t]:off[t + 1]].astype(np.int64)
        assert seg.size == O.k_for(n, wl.ratio), t
        if seg.size:
            assert seg[0] >= 0 and seg[-1] < n, t
            assert np.all(np.diff(seg) > 0), t


@pytest.mark.parametrize("wid", [1, 3, 4])
def test_full_size_sparse_workload(wid):
    wl, off, grads, resids, payloads, outs, own, sample, g_host, e_host, alpha = _run(wid)
    _check_sparse_payload_properties(wl, off, own)
    idx = own["idx"].cpu().numpy().view(np.uint32)
    val = own["val"].cpu().numpy()
    p_idx = [p["idx"].cpu().numpy().view(np.uint32) for p in payloads]
    p_val = [p["val"].cpu().numpy() for p in payloads]
    for t in sample:
        n = wl.sizes[t]
        g, e0 = g_host[t], e_host[t]
        if wl.kind == "topk":
            wi, wv, we = O.compress_topk(g, e0, wl.ratio)
        elif wl.kind == "topk_sampled":
            wi, wv, we = O.compress_topk_sampled(g, e0, wl.ratio, WL.SEED, t)
        else:
            wi, wv, we = O.compress_randk(g, e0, wl.ratio, WL.SEED, t)
        assert np.array_equal(idx[off[t]:off[t + 1]], wi), (t, n)
        assert np.array_equal(bits(val[off[t]:off[t + 1]]), bits(wv)), (t, n)
        assert np.array_equal(bits(resids[t].cpu().numpy()), bits(we)), (t, n)
        want = O.aggregate_sparse(n, [a[off[t]:off[t + 1]] for a in p_idx],
                                  [a[off[t]:off[t + 1]] for a in p_val], alpha)
        assert np.array_equal(bits(outs[t].cpu().numpy()), bits(want)), (t, n)


def _windows(n, rng):
    """Element windows [a, b) starting on a word boundary: the head, the
    tail and two seeded windows of 2048 elements (whole tensor if small)."""
    if n <= 8192:
        return [(0, n)]
    w = 2048
    mids = [32 * int(x) for x in rng.integers(0, (n - w) // 32, size=2)]
    tail = (n - w) // 32 * 32
    return [(0, w), (tail, n)] + [(a, a + w) for a in mids]


@pytest.mark.parametrize("wid", [2, 5])
def test_full_size_sign_workload(wid):
    wl, off, grads, resids, payloads, outs, own, sample, g_host, e_host, alpha = _run(wid)
    words = own["bits"].cpu().numpy().view(np.uint32)
    scale = own["scale"].cpu().numpy()
    # every tensor: padding bits clear
    for t, n in enumerate(wl.sizes):
        if n % 32:
            assert words[off[t + 1] - 1] >> np.uint32(n % 32) == 0, t
    # the compress sample against the oracle
    for t in sample:
        g, e0 = g_host[t], e_host[t]
        ww, ws_, we = O.compress_sign(g, e0)
        assert np.array_equal(words[off[t]:off[t + 1]], ww), t
        tol = sign_tolerances([g])[0]
        assert abs(float(scale[t]) - float(ws_)) <= tol * abs(float(ws_)), (t, scale[t], ws_)
        got_e = resids[t].cpu().numpy()
        if scale[t] == ws_:
            assert np.array_equal(bits(got_e), bits(we)), t
        else:
            v = g.astype(np.float32) + e0
            lim = tol * (np.abs(v).astype(np.float64) + float(ws_))
            assert np.all(np.abs(got_e.astype(np.float64) - we.astype(np.float64)) <= lim), t
    # aggregate: windows of the sampled tensors, and of every tensor's head
    p_bits = [p["bits"].cpu().numpy().view(np.uint32) for p in payloads]
    p_scale = np.stack([p["scale"].cpu().numpy() for p in payloads])  # [W, T]
    rng = np.random.default_rng(77 + wid)
    heads = range(0, wl.T, max(1, wl.T // 64))
    for t in sorted(set(sample) | set(heads)):
        n = wl.sizes[t]
        got = outs[t].cpu().numpy()
        wins = _windows(n, rng) if t in sample else [(0, min(n, 1024))]
        for a, b in wins:
            w0, w1 = off[t] + a // 32, off[t] + (b + 31) // 32
            want = O.aggregate_sign(b - a, [x[w0:w1] for x in p_bits], p_scale[:, t], alpha)
            assert np.array_equal(bits(got[a:b]), bits(want)), (t, a, b)


@pytest.mark.parametrize("wid", [6, 7, 8])
def test_full_size_quant_workload(wid):
    wl, off, grads, resids, payloads, outs, own, sample, g_host, e_host, alpha = _run(wid)
    b = O.QUANT_BITS[wl.kind]
    words = own["bits"].cpu().numpy().view(np.uint32)
    scale = own["scale"].cpu().numpy()
    for t in sample:
        ww, ss, we = O.compress_quant(g_host[t], e_host[t], b, WL.SEED, t)
        assert np.array_equal(words[off[t]:off[t + 1]], ww), t
        assert bits(scale[t]) == bits(np.float32(ss)), t
        assert np.array_equal(bits(resids[t].cpu().numpy()), bits(we)), t
    p_bits = [p["bits"].cpu().numpy().view(np.uint32) for p in payloads]
    p_scale = np.stack([p["scale"].cpu().numpy() for p in payloads])
    for t in sample:
        n = wl.sizes[t]
        want = O.aggregate_quant(n, b, [x[off[t]:off[t + 1]] for x in p_bits], p_scale[:, t], alpha)
        assert np.array_equal(bits(outs[t].cpu().numpy()), bits(want)), t


def test_full_size_dgc_workload():
    """The DGC workload's tensor list (BERT-base, momentum 0.9 around the
    sampled top-k at 1 %, W = 64) in the launch configuration the benchmark
    times, with non-zero velocities: the sampled tensors' payloads,
    residuals and velocities bit for bit against the oracle's DGC step;
    every tensor's payload by its properties and its velocity +0.0 at its
    payload's indices."""
    import torch
    from paper_2205_14465_amd import binding as B
    wl = WL.workload(9)
    dev = torch.device("cuda:0")
    off = B.bytecomp_layout(wl.kind, wl.ratio, wl.sizes)
    grads, resids, payloads, outs = WL.device_inputs(wl, off, dev)
    del payloads, outs
    gen = torch.Generator(device=dev)
    gen.manual_seed(909)
    vels = [torch.randn(n, generator=gen, device=dev, dtype=torch.float32) * 0.01 for n in wl.sizes]
    rng = np.random.default_rng(1009)
    sample = _sample(wl, rng)
    g_host = {t: grads[t].cpu().numpy() for t in sample}
    e_host = {t: resids[t].cpu().numpy().copy() for t in sample}
    u_host = {t: vels[t].cpu().numpy().copy() for t in sample}
    own = B.alloc_payload(wl.kind, wl.ratio, wl.sizes, device=dev)
    ws = B.alloc_workspace(wl.kind, wl.ratio, wl.sizes, wl.W, device=dev)
    B.DgcCall(wl.kind, wl.ratio, wl.momentum, grads, resids, vels, own, ws,
              stream=torch.cuda.current_stream())(WL.SEED)
    torch.cuda.synchronize()
    assert B.bytecomp_device_status(ws) == 0
    _check_sparse_payload_properties(wl, off, own)
    idx = own["idx"].cpu().numpy().view(np.uint32)
    val = own["val"].cpu().numpy()
    for t in sample:
        wi, wv, we, wu = O.compress_dgc(wl.kind, g_host[t], e_host[t], u_host[t], wl.momentum, wl.ratio,
                                        WL.SEED, t)
        assert np.array_equal(idx[off[t]:off[t + 1]], wi), t
        assert np.array_equal(bits(val[off[t]:off[t + 1]]), bits(wv)), t
        assert np.array_equal(bits(resids[t].cpu().numpy()), bits(we)), t
        assert np.array_equal(bits(vels[t].cpu().numpy()), bits(wu)), t
    for t in range(wl.T):
        sel = idx[off[t]:off[t + 1]].astype(np.int64)
        assert np.all(bits(vels[t].cpu().numpy()[sel]) == 0), t
