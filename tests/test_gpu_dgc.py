"""GPU parity of bytecomp_compress_dgc (DGC momentum correction, sparse
compression with error feedback, momentum-factor masking; DGC is the
paper's sparsification operator, Sec. 5.1) against the oracle, over two
consecutive steps so that the velocity and residual states carry over.
Payloads, residuals and velocities must match bit for bit.  The top-k kinds
fold the velocity step and the masking into their own passes; both of their
launch sequences (the few-chunk path and the general pipeline) are run."""
import contextlib

import numpy as np
import pytest

import oracle as O
from tests.helpers import bits, torch_dev

pytestmark = pytest.mark.gpu

RAGGED = [0, 1, 3, 64, 1000, 4095, 4097, 3 * 4096 + 17, 65537, 140001]

KIND_PATHS = [("topk", "few"), ("topk", "general"), ("topk_sampled", "few"), ("topk_sampled", "general"),
              ("randk", "few")]


@contextlib.contextmanager
def topk_path(path):
    from paper_2205_14465_amd import binding as B
    B.bytecomp_set_topk_few_chunks(2048 if path == "few" else 0)
    try:
        yield
    finally:
        B.bytecomp_set_topk_few_chunks(2048)


@pytest.mark.parametrize("kind,path", KIND_PATHS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_dgc_two_steps(kind, path, dtype):
    with topk_path(path):
        _two_steps(kind, dtype)


def _two_steps(kind, dtype):
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(3 + (dtype == np.float16))
    ns = RAGGED
    ratio, m = 0.02, 0.9
    grads1 = [(rng.standard_normal(n) * 0.01).astype(dtype) for n in ns]
    grads2 = [(rng.standard_normal(n) * 0.01).astype(dtype) for n in ns]
    e = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in ns]
    u = [np.zeros(n, np.float32) for n in ns]
    de = [torch_dev(x) for x in e]
    du = [torch_dev(x) for x in u]
    out = B.alloc_payload(kind, ratio, ns)
    ws = B.alloc_workspace(kind, ratio, ns, 1)
    for step, (grads, seed) in enumerate([(grads1, 11), (grads2, 12)]):
        dg = [torch_dev(g) for g in grads]
        B.bytecomp_compress_dgc(kind, ratio, seed, m, dg, de, du, out, ws)
        torch.cuda.synchronize()
        assert B.bytecomp_device_status(ws) == 0
        want, e, u = O.compress_dgc_set(kind, ratio, seed, m, grads, e, u)
        total = int(want["off"][-1])
        got_idx = out["idx"].cpu().numpy().view(np.uint32)[:total]
        got_val = out["val"].cpu().numpy()[:total]
        assert np.array_equal(got_idx, want["idx"]), step
        assert np.array_equal(bits(got_val), bits(want["val"])), step
        for t in range(len(ns)):
            assert np.array_equal(bits(de[t].cpu().numpy()), bits(e[t])), (step, t)
            assert np.array_equal(bits(du[t].cpu().numpy()), bits(u[t])), (step, t)


@pytest.mark.parametrize("kind,path", KIND_PATHS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_dgc_clip_two_steps(kind, path, dtype):
    """Local gradient clipping: the factor within one fp32 place of the
    oracle's (the two add the fp64 squares in different orders); where the
    factors agree (the usual case), payloads, residuals and velocities bit
    for bit.  The first step clips (threshold below the norm), the second
    does not (threshold above it: factor exactly 1)."""
    with topk_path(path):
        _clip_two_steps(kind, dtype)


def _clip_two_steps(kind, dtype):
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(23 + (dtype == np.float16))
    ns = RAGGED
    ratio, m = 0.02, 0.9
    grads1 = [(rng.standard_normal(n) * 0.01).astype(dtype) for n in ns]
    grads2 = [(rng.standard_normal(n) * 0.01).astype(dtype) for n in ns]
    e = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in ns]
    u = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in ns]
    de = [torch_dev(x) for x in e]
    du = [torch_dev(x) for x in u]
    out = B.alloc_payload(kind, ratio, ns)
    ws = B.alloc_workspace(kind, ratio, ns, 1)
    fac = torch.zeros(1, dtype=torch.float32, device="cuda")
    norm1 = float(np.sqrt(sum(float(np.sum(g.astype(np.float64) ** 2)) for g in grads1)))
    for step, (grads, seed, clip) in enumerate([(grads1, 11, norm1 / 3.0), (grads2, 12, 1e9)]):
        dg = [torch_dev(g) for g in grads]
        B.bytecomp_compress_dgc_clip(kind, ratio, seed, m, clip, dg, de, du, out, ws, clip_factor=fac)
        torch.cuda.synchronize()
        assert B.bytecomp_device_status(ws) == 0
        c_gpu = np.float32(fac.item())
        c_ref = O.dgc_clip_factor(grads, clip)
        assert abs(float(c_gpu) - float(c_ref)) <= float(np.spacing(c_ref)), (step, c_gpu, c_ref)
        if step == 1:
            assert c_gpu == np.float32(1.0)
        else:
            assert c_gpu < np.float32(0.34)
        want, e, u = O.compress_dgc_set(kind, ratio, seed, m, grads, e, u, clip=clip)
        if c_gpu != c_ref:  # the last place of the factor differs: the states diverge
            pytest.skip(f"factor differs in the last place at step {step}")
        total = int(want["off"][-1])
        assert np.array_equal(out["idx"].cpu().numpy().view(np.uint32)[:total], want["idx"]), step
        assert np.array_equal(bits(out["val"].cpu().numpy()[:total]), bits(want["val"])), step
        for t in range(len(ns)):
            assert np.array_equal(bits(de[t].cpu().numpy()), bits(e[t])), (step, t)
            assert np.array_equal(bits(du[t].cpu().numpy()), bits(u[t])), (step, t)


def test_dgc_clip_rejects_bad_threshold():
    from paper_2205_14465_amd import binding as B
    ns = [100]
    out = B.alloc_payload("topk", 0.1, ns)
    ws = B.alloc_workspace("topk", 0.1, ns, 1)
    g = [torch_dev(np.ones(100, np.float32))]
    e = [torch_dev(np.zeros(100, np.float32))]
    u = [torch_dev(np.zeros(100, np.float32))]
    for bad in (-1.0, float("nan")):
        with pytest.raises(B.BytecompError, match="BC_E_RATIO"):
            B.bytecomp_compress_dgc_clip("topk", 0.1, 1, 0.9, bad, g, e, u, out, ws)


@pytest.mark.parametrize("ratio", [1.0, 0.5])
def test_dgc_sampled_fallback_mixed(ratio):
    """General pipeline, sampled kind: a tensor whose sample misses the k-th
    key falls back to the exact path, which re-reads the v that the fused
    stream pass stored (after the velocity step); beside it a tensor whose
    values are mostly zero (threshold 0) and tensors below the sampling
    size.  Two steps, so the masked velocities feed the second."""
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(41)
    ns = [70000, 140001, 100, 5000]
    m = 0.9
    e = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in ns]
    u = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in ns]
    u[1][rng.random(ns[1]) < 0.3] = 0.0
    e[1][u[1] == 0.0] = 0.0
    de = [torch_dev(x) for x in e]
    du = [torch_dev(x) for x in u]
    out = B.alloc_payload("topk_sampled", ratio, ns)
    ws = B.alloc_workspace("topk_sampled", ratio, ns, 1)
    with topk_path("general"):
        for step, seed in enumerate((5, 6)):
            grads = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in ns]
            grads[1][u[1] == 0.0] = 0.0
            dg = [torch_dev(g) for g in grads]
            B.bytecomp_compress_dgc("topk_sampled", ratio, seed, m, dg, de, du, out, ws)
            torch.cuda.synchronize()
            assert B.bytecomp_device_status(ws) == 0
            want, e, u = O.compress_dgc_set("topk_sampled", ratio, seed, m, grads, e, u)
            total = int(want["off"][-1])
            assert np.array_equal(out["idx"].cpu().numpy().view(np.uint32)[:total], want["idx"]), step
            assert np.array_equal(bits(out["val"].cpu().numpy()[:total]), bits(want["val"])), step
            for t in range(len(ns)):
                assert np.array_equal(bits(de[t].cpu().numpy()), bits(e[t])), (step, t)
                assert np.array_equal(bits(du[t].cpu().numpy()), bits(u[t])), (step, t)


@pytest.mark.timeout(600)
def test_dgc_randk_many_chunks():
    """Random-k DGC on a call of more than 32768 chunks (40000 one-chunk
    tensors): buckets of 8 chunks streamed in runs of 4 by two workgroups
    each, the velocity step and the masking inside that pass.  Two steps,
    payloads, residuals and velocities bit for bit."""
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(43)
    ns = [int(x) for x in rng.integers(1, 4097, size=40000)]
    ns[7] = 0
    ratio, m = 0.01, 0.9
    e = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in ns]
    u = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in ns]
    de = [torch_dev(x) for x in e]
    du = [torch_dev(x) for x in u]
    out = B.alloc_payload("randk", ratio, ns)
    ws = B.alloc_workspace("randk", ratio, ns, 1)
    for step, seed in enumerate((21, 22)):
        grads = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in ns]
        B.bytecomp_compress_dgc("randk", ratio, seed, m, [torch_dev(g) for g in grads], de, du, out, ws)
        torch.cuda.synchronize()
        assert B.bytecomp_device_status(ws) == 0
        want, e, u = O.compress_dgc_set("randk", ratio, seed, m, grads, e, u)
        total = int(want["off"][-1])
        assert np.array_equal(out["idx"].cpu().numpy().view(np.uint32)[:total], want["idx"]), step
        assert np.array_equal(bits(out["val"].cpu().numpy()[:total]), bits(want["val"])), step
        got_e = torch.cat([x for x in de if x.numel()]).cpu().numpy()
        got_u = torch.cat([x for x in du if x.numel()]).cpu().numpy()
        assert np.array_equal(bits(got_e), bits(np.concatenate(e))), step
        assert np.array_equal(bits(got_u), bits(np.concatenate(u))), step
