"""GPU parity: the HIP library (through its C ABI) against the CPU oracle,
element by element, on seeded inputs that span several chunks and ragged
tails, plus the edge cases (single elements, empty tensors, ties, signed
zeros, fp16 subnormals, error feedback off, the sampled path's fallback).

Bars: indices, packed sign bits, selected values, sparse residuals and both
aggregates bit-exact; sign scales within 1e-6 relative (fp32 gradients) or
1e-3 (fp16 gradients); sign residuals bit-exact where the scales agree,
else within the same relative bound of |v| + s.
"""
import numpy as np
import pytest

import oracle as O
from tests.exact_ref import same_f32_arrays
from tests.helpers import (_first_diff, assert_resid_equal, assert_sign_close, assert_sparse_equal, bits,
                           gpu_aggregate, gpu_compress, torch_dev)
from paper_2205_14465_amd import workloads as WL

pytestmark = pytest.mark.gpu

RAGGED = [1, 2, 31, 32, 33, 63, 64, 65, 1000, 4095, 4096, 4097, 8191, 3 * 4096 + 17, 65536, 65537,
          100003, 300001]
SEED = 14465


def make_set(ns, rng, dtype=np.float32, sigma=0.01, mode="normal"):
    grads, resids = [], []
    for n in ns:
        if mode == "ties":
            levels = np.array([-4, -3, -2, -1, -0.5, -0.25, 0, -0.0, 0.25, 0.5, 1, 2, 3, 4, 5, -5])
            g = (levels[rng.integers(0, 16, n)] * sigma).astype(dtype)
            e = np.zeros(n, np.float32)
        else:
            g = (rng.standard_normal(n) * sigma).astype(dtype)
            e = (rng.standard_normal(n) * sigma * 0.1).astype(np.float32)
        if n >= 4:
            g[:2] = np.array([0.0, -0.0], dtype)
            e[:2] = np.array([-0.0, -0.0], np.float32)
        grads.append(g)
        resids.append(e)
    return grads, resids


# ------------------------------------------------------------- compression

@pytest.fixture(params=["few", "general"])
def topk_path(request):
    """Top-k calls through the few-chunk path (the default at these sizes)
    and through the general pipeline."""
    from paper_2205_14465_amd import binding as B
    B.bytecomp_set_topk_few_chunks(2048 if request.param == "few" else 0)
    yield request.param
    B.bytecomp_set_topk_few_chunks(2048)


@pytest.fixture
def general_path():
    from paper_2205_14465_amd import binding as B
    B.bytecomp_set_topk_few_chunks(0)
    yield
    B.bytecomp_set_topk_few_chunks(2048)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk"])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_sparse_compress_ragged(kind, dtype, topk_path):
    rng = np.random.default_rng(100 + len(kind))
    grads, resids = make_set(RAGGED, rng, dtype)
    got, got_e = gpu_compress(kind, 0.01, SEED, grads, resids)
    want, want_e = O.compress_set(kind, 0.01, SEED, grads, resids)
    assert_sparse_equal(got, want, RAGGED)
    assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk"])
@pytest.mark.parametrize("ratio", [0.001, 0.05, 0.3, 1.0])
def test_sparse_compress_ratios(kind, ratio, topk_path):
    rng = np.random.default_rng(7)
    ns = [5, 4097, 70001, 131072]
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress(kind, ratio, SEED + 1, grads, resids)
    want, want_e = O.compress_set(kind, ratio, SEED + 1, grads, resids)
    assert_sparse_equal(got, want, ns)
    assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled"])
def test_topk_tie_heavy(kind, topk_path):
    rng = np.random.default_rng(9)
    ns = [100, 4096 * 5 + 3, 200000]
    grads, resids = make_set(ns, rng, mode="ties")
    for ratio in (0.01, 0.2, 0.5):
        got, got_e = gpu_compress(kind, ratio, SEED, grads, resids)
        want, want_e = O.compress_set(kind, ratio, SEED, grads, resids)
        assert_sparse_equal(got, want, ns)
        assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk", "sign"])
def test_error_feedback_off(kind, topk_path):
    rng = np.random.default_rng(11)
    ns = [3, 4096, 70000]
    grads, _ = make_set(ns, rng)
    got, got_e = gpu_compress(kind, 0.01, SEED, grads, None)
    want, want_e = O.compress_set(kind, 0.01, SEED, grads, None)
    assert got_e is None
    if kind == "sign":
        assert_sign_close(got, want, grads, None, None, None)
    else:
        assert_sparse_equal(got, want, ns)


def test_sampled_fallback_path_matches_exact(general_path):
    # ratio 1 (and 0.95) on tensors above the all-candidates size forces the
    # candidate set from the sample to fall short of k: exact fallback
    rng = np.random.default_rng(13)
    ns = [70000, 140001]
    grads, resids = make_set(ns, rng)
    for ratio in (1.0, 0.95):
        got, got_e = gpu_compress("topk_sampled", ratio, SEED, grads, resids)
        want, want_e = O.compress_set("topk", ratio, SEED, grads, resids)
        assert_sparse_equal(got, want, ns)
        assert_resid_equal(got_e, want_e)


def test_sampled_fallback_mixed_with_kept_candidates(general_path):
    # one call where a tensor falls back (its stream pass had zeroed its
    # candidates in e_new, which the fallback writes back), a large tensor
    # whose sample holds zeros (threshold 0: every element a candidate, no
    # zeroing) and small tensors below the sampling size
    rng = np.random.default_rng(29)
    ns = [70000, 140001, 100, 5000]
    grads, resids = make_set(ns, rng)
    grads[1][rng.random(ns[1]) < 0.3] = 0.0
    resids[1][grads[1] == 0.0] = 0.0
    for ratio in (1.0, 0.5):
        got, got_e = gpu_compress("topk_sampled", ratio, SEED, grads, resids)
        want, want_e = O.compress_set("topk", ratio, SEED, grads, resids)
        assert_sparse_equal(got, want, ns)
        assert_resid_equal(got_e, want_e)


def _stats_after(kind, ratio, grads, resids):
    import torch
    from paper_2205_14465_amd import binding as B
    ns = [g.size for g in grads]
    out = B.alloc_payload(kind, ratio, ns)
    ws = B.alloc_workspace(kind, ratio, ns, 1)
    B.bytecomp_compress(kind, ratio, SEED, [torch_dev(g) for g in grads],
                        [torch_dev(np.asarray(e, np.float32)) for e in resids], out, ws)
    torch.cuda.synchronize()
    return B.bytecomp_topk_stats(kind, ratio, ns, ws)


@pytest.mark.parametrize("path", ["few", "general"])
def test_topk_stats_exact_kind(path):
    """bytecomp_topk_stats after an exact top-k call: no fallbacks, and the
    candidates are the entries whose key (|v| bits) lies in the bin of the
    k-th key (bits 30..20) or above, counted here from v = g + e."""
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(37)
    ns = [5000, 70000, 140001, 3]
    grads, resids = make_set(ns, rng)
    B.bytecomp_set_topk_few_chunks(2048 if path == "few" else 0)
    try:
        cand, fb = _stats_after("topk", 0.01, grads, resids)
    finally:
        B.bytecomp_set_topk_few_chunks(2048)
    want = 0
    for g, e in zip(grads, resids):
        v = g.astype(np.float32) + e
        key = v.view(np.uint32) & np.uint32(0x7FFFFFFF)
        k = O.k_for(v.size, 0.01)
        b0 = np.sort(key)[::-1][k - 1] >> np.uint32(20)
        want += int(np.count_nonzero((key >> np.uint32(20)) >= b0))
    assert fb == 0
    assert cand == want


def test_topk_stats_sampled_kind(general_path):
    """Sampled top-k: at ratio 1 the sample leaves fewer than k candidates in
    both tensors, which fall back and examine every element; at 1 % none
    falls back and the candidates lie between the k_t and the n_t."""
    rng = np.random.default_rng(13)
    ns = [70000, 140001]
    grads, resids = make_set(ns, rng)
    cand, fb = _stats_after("topk_sampled", 1.0, grads, resids)
    assert (cand, fb) == (sum(ns), 2)
    cand, fb = _stats_after("topk_sampled", 0.01, grads, resids)
    assert fb == 0
    assert sum(O.k_for(n, 0.01) for n in ns) <= cand <= sum(ns)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled"])
def test_topk_two_paths_bitwise(kind):
    """The same call through the few-chunk path and the general pipeline
    (different kernels and launch geometries): payloads and residuals
    identical bit for bit, and equal to the oracle's; includes a call of
    exactly 2048 chunks (the few-chunk limit), tensors whose k-th key is
    shared by many entries, and an all-zero tensor."""
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(31)
    cases = [[2048 * 4096], [1, 4095, 4096 * 700 + 5, 3, 4096 * 300]]
    for ns in cases:
        grads, resids = make_set(ns, rng)
        if len(ns) > 1:
            grads[2][::3] = np.float32(0.02)  # a key shared by a third of the tensor
            resids[2][::3] = 0.0
            grads[4][:] = 0.0
            resids[4][:] = 0.0
        outs = []
        for limit in (2048, 0):
            B.bytecomp_set_topk_few_chunks(limit)
            try:
                outs.append(gpu_compress(kind, 0.01, SEED, grads, resids))
            finally:
                B.bytecomp_set_topk_few_chunks(2048)
        (p0, e0), (p1, e1) = outs
        assert np.array_equal(p0["idx"], p1["idx"]) and np.array_equal(bits(p0["val"]), bits(p1["val"]))
        for a, b in zip(e0, e1):
            assert np.array_equal(bits(a), bits(b))
        want, want_e = O.compress_set("topk", 0.01, SEED, grads, resids)
        assert_sparse_equal(p0, want, ns)
        assert_resid_equal(e0, want_e)


def test_topk_path_knob_limits():
    from paper_2205_14465_amd import binding as B
    with pytest.raises(B.BytecompError, match="BC_E_SIZE"):
        B.bytecomp_set_topk_few_chunks(2049)
    B.bytecomp_set_topk_few_chunks(2048)


@pytest.mark.parametrize("T, ratio", [(9000, 0.05), (17000, 0.02), (17000, 1.0)])
def test_randk_many_chunks(T, ratio):
    """More than 8192 chunks: indices are bucketed by runs of 2 and 4 chunks
    (each run here spans several tensors), and buckets of ratio 1 hold every
    element."""
    rng = np.random.default_rng(T)
    ns = [int(x) for x in rng.integers(1, 4097, size=T)]
    for z in (0, 1, T // 2, T - 1):
        ns[z] = 0 if z != T // 2 else 4096
    ns += [3 * 4096 + 5, 20000]
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress("randk", ratio, SEED + T, grads, resids)
    want, want_e = O.compress_set("randk", ratio, SEED + T, grads, resids)
    assert_sparse_equal(got, want, ns)
    assert_resid_equal(got_e, want_e)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", ["small_tensors", "large_tensors"])
def test_randk_bucket_split_into_runs(case):
    """Calls of more than 32768 chunks at a 1 % rate: each bucket of 2^S
    chunks is streamed by several workgroups, each taking a run of 2 chunks
    of it, half a chunk per wave (40000 one-chunk tensors: buckets of 8
    chunks in 4 runs; about 296 M elements in five tensors: buckets of 16
    chunks in 8 runs)."""
    rng = np.random.default_rng(61 if case == "small_tensors" else 62)
    if case == "small_tensors":
        ns = [int(x) for x in rng.integers(1, 4097, size=40000)]
        ns[123] = 0
    else:
        ns = [40_000_000, 33_554_432 + 5, 77, 4096 * 30000 + 1, 100_000_000]
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress("randk", 0.01, SEED + 5, grads, resids)
    want, want_e = O.compress_set("randk", 0.01, SEED + 5, grads, resids)
    assert_sparse_equal(got, want, ns)
    assert_resid_equal(got_e, want_e)


def test_randk_tensor_id_keys_the_stream():
    rng = np.random.default_rng(15)
    ns = [50000, 50000]
    grads, resids = make_set(ns, rng)
    ids = [7, 123456]
    got, _ = gpu_compress("randk", 0.01, 99, grads, resids, tensor_ids=ids)
    for t in range(2):
        i, v, _ = O.compress_randk(grads[t], resids[t], 0.01, 99, ids[t])
        assert np.array_equal(got["idx"][got["off"][t]:got["off"][t + 1]], i)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_sign_compress_ragged(dtype):
    rng = np.random.default_rng(17)
    grads, resids = make_set(RAGGED + [0, 5], rng, dtype, sigma=1e-3)
    got, got_e = gpu_compress("sign", 0.01, 0, grads, resids)
    want, want_e = O.compress_set("sign", 0.01, 0, grads, resids)
    assert_sign_close(got, want, grads, resids, got_e, want_e)


def test_sign_fp16_subnormals_exact():
    # every fp16 subnormal and a spread of normals: widening must be exact
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    g = h.view(np.float16)
    g = g[np.isfinite(g)].copy()
    e = np.zeros(g.size, np.float32)
    got, got_e = gpu_compress("sign", 0.01, 0, [g], [e])
    want, want_e = O.compress_set("sign", 0.01, 0, [g], [e])
    assert_sign_close(got, want, [g], [e], got_e, want_e)
    got, got_e = gpu_compress("topk", 0.3, 0, [g], [e])
    want, want_e = O.compress_set("topk", 0.3, 0, [g], [e])
    assert_sparse_equal(got, want, [g.size])
    assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["sign", "terngrad", "qsgd8"])
@pytest.mark.parametrize("fill", [0xA5, 0xFF])
def test_one_pass_compress_ignores_stale_workspace(kind, fill):
    # the one-pass kernels publish chunk partials through workspace slots;
    # a workspace body left dirty by an earlier call (here every byte
    # `fill`, the header initialised) must not read as published
    rng = np.random.default_rng(29)
    ns = [4096 * 40 + 3, 5000, 1, 0, 4096]
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress(kind, 0.01, SEED, grads, resids, ws_fill=fill)
    want, want_e = O.compress_set(kind, 0.01, SEED, grads, resids)
    if kind == "sign":
        assert_sign_close(got, want, grads, resids, got_e, want_e)
    else:
        assert np.array_equal(got["off"], want["off"])
        assert np.array_equal(got["bits"], want["bits"])
        assert np.array_equal(bits(got["scale"]), bits(want["scale"]))
        assert_resid_equal(got_e, want_e)


def _check_word_kind(kind, got, want, grads, resids, got_e, want_e):
    if kind == "sign":
        assert_sign_close(got, want, grads, resids, got_e, want_e)
    else:
        assert np.array_equal(got["off"], want["off"])
        assert np.array_equal(got["bits"], want["bits"])
        assert np.array_equal(bits(got["scale"]), bits(want["scale"]))
        if got_e is not None:
            assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["sign", "terngrad", "qsgd4", "qsgd8"])
@pytest.mark.parametrize("ef", [True, False])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_one_pass_waits_given_up_from_the_host_stay_exact(kind, ef, dtype):
    # a wait limit of 0 makes every wait of the one-pass kernels stop
    # waiting at once (the condition of a grid that is not wholly resident,
    # forced from the host): a workgroup that finds a chunk partial missing
    # computes it itself; results equal the oracle's, and no failure is
    # reported
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(71)
    ns = [4096 * 40 + 3, 5000, 1, 0, 4096, 4096 * 9, 12345]
    grads, resids = make_set(ns, rng, dtype)
    r_in = resids if ef else None
    B.bytecomp_set_wait_limit(0)
    try:
        got, got_e = gpu_compress(kind, 0.01, SEED, grads, r_in)
    finally:
        B.bytecomp_set_wait_limit(200)
    want, want_e = O.compress_set(kind, 0.01, SEED, grads, r_in)
    _check_word_kind(kind, got, want, grads, r_in, got_e, want_e)


@pytest.mark.parametrize("kind", ["sign", "qsgd8"])
def test_one_pass_compress_beside_a_long_kernel_on_another_stream(kind):
    # the one-pass kernel starts while matrix products queued on another
    # stream (default priority) hold compute units, so its grid may not be
    # wholly resident: waits may run out and workgroups compute missing
    # partials themselves; results still equal the oracle's and no failure
    # is reported
    import torch
    from paper_2205_14465_amd import binding as B
    from tests.helpers import torch_dev, to_np_u32
    rng = np.random.default_rng(72)
    ns = [4096 * 200 + 9, 4096 * 150, 70001, 4096 * 300 + 1, 5000]
    grads, resids = make_set(ns, rng)
    dg = [torch_dev(g) for g in grads]
    de = [torch_dev(e) for e in resids]
    out = B.alloc_payload(kind, 0.01, ns)
    ws = B.alloc_workspace(kind, 0.01, ns, 1)
    a = torch.randn(4096, 4096, device="cuda")
    b = torch.randn(4096, 4096, device="cuda")
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        for _ in range(8):
            c = torch.mm(a, b)
    B.bytecomp_compress(kind, 0.01, SEED, dg, de, out, ws)
    torch.cuda.synchronize()
    del c
    assert B.bytecomp_device_status(ws) == 0
    total = out["off"][-1]
    got = {"off": np.array(out["off"], dtype=np.int64), "bits": to_np_u32(out["bits"])[:total],
           "scale": out["scale"].cpu().numpy()[:len(ns)]}
    got_e = [e.cpu().numpy() for e in de]
    want, want_e = O.compress_set(kind, 0.01, SEED, grads, resids)
    _check_word_kind(kind, got, want, grads, resids, got_e, want_e)


@pytest.mark.parametrize("kind", ["sign", "terngrad"])
def test_one_pass_compress_calls_in_a_row_share_a_workspace(kind):
    # successive calls on one workspace, with new inputs each time and a
    # call of another shape between them: slots left by an earlier call of
    # the same shape must not read as published in a later one
    import torch
    from paper_2205_14465_amd import binding as B
    from tests.helpers import torch_dev, to_np_u32
    ns_a = [4096 * 40 + 3, 5000, 4096 * 7]
    ns_b = [4096 * 12 + 1, 77]
    ws = B.alloc_workspace(kind, 0.01, ns_a, 1)
    ws_b_bytes = B.bytecomp_workspace_size(kind, 0.01, ns_b, 1)
    assert ws.numel() >= ws_b_bytes
    for call, ns in enumerate([ns_a, ns_a, ns_b, ns_a, ns_a]):
        rng = np.random.default_rng(300 + call)
        grads, resids = make_set(ns, rng)
        dg = [torch_dev(g) for g in grads]
        de = [torch_dev(e) for e in resids]
        out = B.alloc_payload(kind, 0.01, ns)
        B.bytecomp_compress(kind, 0.01, SEED + call, dg, de, out, ws)
        torch.cuda.synchronize()
        assert B.bytecomp_device_status(ws) == 0
        total = out["off"][-1]
        got = {"off": np.array(out["off"], dtype=np.int64), "bits": to_np_u32(out["bits"])[:total],
               "scale": out["scale"].cpu().numpy()[:len(ns)]}
        got_e = [e.cpu().numpy() for e in de]
        want, want_e = O.compress_set(kind, 0.01, SEED + call, grads, resids)
        if kind == "sign":
            assert_sign_close(got, want, grads, resids, got_e, want_e)
        else:
            assert np.array_equal(got["bits"], want["bits"]), call
            assert np.array_equal(bits(got["scale"]), bits(want["scale"])), call
            assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk", "sign", "terngrad", "qsgd4", "qsgd8"])
def test_every_kind_ignores_a_dirty_workspace(kind):
    # compress and aggregate with a workspace whose body is all 0xA5 bytes
    # (header initialised): every region a call reads must be set by the
    # call itself
    rng = np.random.default_rng(31)
    ns = [4096 * 40 + 3, 5000, 1, 0, 4096]
    ratio = 0.01
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress(kind, ratio, SEED, grads, resids, ws_fill=0xA5)
    want, want_e = O.compress_set(kind, ratio, SEED, grads, resids)
    if kind == "sign":
        assert_sign_close(got, want, grads, resids, got_e, want_e)
    elif kind in ("terngrad", "qsgd4", "qsgd8"):
        assert np.array_equal(got["bits"], want["bits"])
        assert np.array_equal(bits(got["scale"]), bits(want["scale"]))
        assert_resid_equal(got_e, want_e)
    else:
        assert_sparse_equal(got, want, ns)
        assert_resid_equal(got_e, want_e)
    W = 5
    payloads = [dict(want, off=want["off"])]
    for w in range(1, W):
        g2, e2 = make_set(ns, np.random.default_rng(100 + w))
        p, _ = O.compress_set(kind, ratio, SEED + w, g2, e2)
        payloads.append(p)
    out = gpu_aggregate(kind, ratio, ns, payloads, 1.0 / W, ws_fill=0xA5)
    ref = O.aggregate_set(kind, ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(out[t]), bits(ref[t])), t


def test_compress_is_deterministic():
    rng = np.random.default_rng(19)
    ns = [4096 * 300 + 5, 77]
    grads, resids = make_set(ns, rng)
    for kind in ("sign", "topk_sampled", "randk"):
        a, ae = gpu_compress(kind, 0.01, SEED, grads, resids)
        b, be = gpu_compress(kind, 0.01, SEED, grads, resids)
        for key in a:
            assert np.array_equal(np.asarray(a[key]).view(np.uint8), np.asarray(b[key]).view(np.uint8)), (kind, key)
        assert_resid_equal(ae, be)


# ------------------------------------------------------------- aggregation

@pytest.mark.parametrize("W", [1, 2, 8, 64])
def test_sparse_aggregate_ragged(W):
    rng = np.random.default_rng(21 + W)
    ns = [1, 31, 2048, 2049, 4096 * 3 + 5, 100000, 0, 7]
    counts = [O.k_for(n, 0.05) for n in ns]
    payloads = []
    for w in range(W):
        idx, val = WL.random_sparse_lists(rng, ns, counts)
        payloads.append({"idx": np.concatenate(idx), "val": np.concatenate(val),
                         "off": O.sparse_offsets(ns, 0.05)})
    alpha = 1.0 / W
    got = gpu_aggregate("topk", 0.05, ns, payloads, alpha)
    want = O.aggregate_set("topk", ns, payloads, alpha)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


@pytest.mark.parametrize("W", [16, 32, 48])
def test_sparse_aggregate_several_tiles_per_wave(W):
    # a tensor of more than 8192 x 2 tiles, so that waves walk several
    # consecutive tiles of it and carry their next-tile loads across tiles
    # (W a multiple of 16)
    rng = np.random.default_rng(23 + W)
    ns = [2048 * 16384 * 2 + 777, 5000]
    ratio = 0.002
    counts = [O.k_for(n, ratio) for n in ns]
    payloads = []
    for w in range(W):
        idx, val = WL.random_sparse_lists(rng, ns, counts)
        payloads.append({"idx": np.concatenate(idx), "val": np.concatenate(val),
                         "off": O.sparse_offsets(ns, ratio)})
    got = gpu_aggregate("topk", ratio, ns, payloads, 1.0)
    want = O.aggregate_set("topk", ns, payloads, 1.0)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


def _clustered_lists(rng, ns, counts, spread):
    """One worker's payload whose indices crowd into the first `spread`
    fraction of each tensor (dense windows: more than 128 entries per
    8192-element tile)."""
    idx, val = [], []
    for n, k in zip(ns, counts):
        span = max(int(k), int(n * spread))
        idx.append(np.sort(rng.choice(span, size=int(k), replace=False)).astype(np.uint32))
        val.append((rng.standard_normal(int(k))).astype(np.float32))
    return idx, val


@pytest.mark.parametrize("W", [24, 72])
def test_sparse_aggregate_large_tiles(W):
    # at least 2^24 elements at low density: 8192-element tiles, 128-entry
    # windows; W = 24 takes 8-slot steps, W = 72 the LDS-held worker state;
    # every fourth worker crowds its entries (dense windows, the slow path)
    rng = np.random.default_rng(90 + W)
    ns = [(1 << 24) + 12345, 7000, 1]
    ratio = 0.01
    counts = [O.k_for(n, ratio) for n in ns]
    payloads = []
    for w in range(W):
        if w % 4 == 1:
            idx, val = _clustered_lists(rng, ns, counts, 0.02)
        else:
            idx, val = WL.random_sparse_lists(rng, ns, counts)
        payloads.append({"idx": np.concatenate(idx), "val": np.concatenate(val),
                         "off": O.sparse_offsets(ns, ratio)})
    got = gpu_aggregate("topk", ratio, ns, payloads, 1.0 / W)
    want = O.aggregate_set("topk", ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


@pytest.mark.parametrize("W,ratio", [(5, 0.01), (33, 0.03), (64, 0.01), (64, 0.004)])
def test_sparse_aggregate_windows_across_tensors(W, ratio):
    # many small tensors at low density (the register-window path): waves
    # cross tensor boundaries inside their runs and start runs inside
    # tensors; empty tensors and tensors without entries are mixed in, and
    # every seventh worker crowds its entries (windows that run dry inside
    # a tile)
    rng = np.random.default_rng(400 + W)
    ns = [int(x) for x in rng.integers(1, 60000, size=150)] + [0, 1, 3, 250000, 4096, 4097, 1 << 20]
    counts = [O.k_for(n, ratio) for n in ns]
    payloads = []
    for w in range(W):
        if w % 7 == 3:
            idx, val = _clustered_lists(rng, ns, counts, 0.03)
        else:
            idx, val = WL.random_sparse_lists(rng, ns, counts)
        payloads.append({"idx": np.concatenate(idx), "val": np.concatenate(val),
                         "off": O.sparse_offsets(ns, ratio)})
    got = gpu_aggregate("topk", ratio, ns, payloads, 1.0 / W)
    want = O.aggregate_set("topk", ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


def test_sparse_aggregate_dense_overlap():
    # every worker sends every index (ratio 1): maximal overlap, long runs
    rng = np.random.default_rng(23)
    ns = [5000, 70001]
    W = 5
    payloads = []
    for w in range(W):
        idx = [np.arange(n, dtype=np.uint32) for n in ns]
        val = [(rng.standard_normal(n) * 10.0 ** rng.integers(-3, 3)).astype(np.float32) for n in ns]
        payloads.append({"idx": np.concatenate(idx), "val": np.concatenate(val),
                         "off": O.sparse_offsets(ns, 1.0)})
    got = gpu_aggregate("randk", 1.0, ns, payloads, 1.0)
    want = O.aggregate_set("randk", ns, payloads, 1.0)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


@pytest.mark.parametrize("W", [1, 3, 8, 17, 24, 32, 64, 71, 130])
def test_sign_aggregate_ragged(W):
    rng = np.random.default_rng(31 + W)
    ns = [1, 31, 32, 33, 511, 512, 513, 2047, 2048, 2049, 8191, 8192, 8193, 8192 * 2 + 7, 100001, 0]
    wc = [O.words_for(n) for n in ns]
    payloads = []
    for w in range(W):
        words = WL.random_sign_words(rng, ns, wc)
        payloads.append({"bits": np.concatenate(words),
                         "scale": (np.abs(rng.standard_normal(len(ns))) * 1e-3).astype(np.float32),
                         "off": O.word_offsets(ns)})
    got = gpu_aggregate("sign", 0.01, ns, payloads, 1.0 / W)
    want = O.aggregate_set("sign", ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


def _sign_payloads(rng, ns, per_t):
    """W sign payloads over tensors ns; per_t[t][w] is worker w's scale of
    tensor t."""
    wc = [O.words_for(n) for n in ns]
    W = len(per_t[0])
    payloads = []
    for w in range(W):
        words = WL.random_sign_words(rng, ns, wc)
        payloads.append({"bits": np.concatenate(words),
                         "scale": np.array([per_t[t][w] for t in range(len(ns))], np.float32),
                         "off": O.word_offsets(ns)})
    return payloads


def _scales_with_span(rng, W, span, base_exp=-10):
    """W fp32 scales whose binary exponents span exactly `span` binades
    (worker 0 at the low end, worker 1 at the high end), random signs for
    the wide spans."""
    base = np.float32(2.0 ** base_exp)
    s = (base * (1 + rng.random(W))).astype(np.float32)
    if W >= 2:
        s[0] = base * np.float32(1.25)
        s[1] = np.float32(np.ldexp(1.5, base_exp + span))
        if W > 2:
            s[2:] = np.ldexp(1.0 + rng.random(W - 2), rng.integers(base_exp, base_exp + span + 1, W - 2))
    return s


def _gpu_tiers(W):
    """Binade spans the kernel's int32 and fp64 table forms take (the test
    aims tensors at both sides of each; the result must not depend on it)."""
    int_limit = 7 - int(np.ceil(np.log2(8 * ((W + 7) // 8))))
    f64_limit = 29 - int(np.ceil(np.log2(W))) if W > 1 else 29
    return int_limit, f64_limit


@pytest.mark.parametrize("W", [4, 64, 130])
def test_sign_aggregate_wide_scale_spans_are_exact(W):
    # tensors whose worker scales spread over 30 to 253 binades, beside a
    # narrow one: every output is the exact sum rounded once
    rng = np.random.default_rng(33 + W)
    spans = [30, 45, 60, 120, 253]
    ns = [8192 + 100, 5000, 4096 * 2, 77, 4097, 3000]
    per_t = [_scales_with_span(rng, W, sp, base_exp=-126) for sp in spans]
    per_t.append((1e-3 * (1 + 0.05 * rng.standard_normal(W))).astype(np.float32))
    payloads = _sign_payloads(rng, ns, per_t)
    got = gpu_aggregate("sign", 0.01, ns, payloads, 1.0 / W)
    want = O.aggregate_set("sign", ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert same_f32_arrays(got[t], want[t]), (t, _first_diff(bits(got[t]), bits(want[t])))


@pytest.mark.parametrize("W", [3, 64])
def test_sign_aggregate_subnormal_negative_and_non_finite_scales(W):
    # subnormal scales, negative scales, sums past the fp32 range, and NaN
    # or infinite scales (the order-free rule), each in its own tensor
    rng = np.random.default_rng(90 + W)
    fmax = np.float32(np.finfo(np.float32).max)
    ns = [4096 + 5, 300, 2000, 129, 4096 * 2, 64]
    per_t = []
    per_t.append(np.ldexp(1.0 + rng.random(W), rng.integers(-149, -126, W)).astype(np.float32))  # subnormal
    per_t.append((-np.abs(rng.standard_normal(W)) * 1e-3).astype(np.float32))                    # negative
    per_t.append(np.full(W, fmax, np.float32))                                                   # overflow
    t3 = (1e-3 * (1 + rng.random(W))).astype(np.float32)
    t3[W // 2] = np.inf
    per_t.append(t3)                                                                             # one +Inf
    t4 = (1e-3 * (1 + rng.random(W))).astype(np.float32)
    t4[0], t4[-1] = np.inf, -np.inf
    per_t.append(t4)                                                                             # both
    t5 = (1e-3 * (1 + rng.random(W))).astype(np.float32)
    t5[1 % W] = np.nan
    per_t.append(t5)                                                                             # NaN
    payloads = _sign_payloads(rng, ns, per_t)
    got = gpu_aggregate("sign", 0.01, ns, payloads, 0.5)
    want = O.aggregate_set("sign", ns, payloads, 0.5)
    for t in range(len(ns)):
        assert same_f32_arrays(got[t], want[t]), (t, _first_diff(bits(got[t]), bits(want[t])))


@pytest.mark.parametrize("W", [8, 32, 64, 71, 128, 130])
def test_sign_aggregate_exact_forms_by_scale_span(W):
    # one call whose tensors fall on both sides of each of the kernel's
    # table forms (int32, fp64) and far beyond them: results match the
    # oracle's exact sum bit for bit whatever path computes them
    rng = np.random.default_rng(51 + W)
    int_limit, limit = _gpu_tiers(W)
    spans = sorted({0, 1, max(int_limit, 0), int_limit + 1, limit - 1, limit, limit + 1, limit + 5, 40, 60})
    spans = [sp for sp in spans if sp >= 0]
    ns = [4096 * 3 + 77 if i % 2 == 0 else 5000 + 31 * i for i in range(len(spans))]
    per_t = [_scales_with_span(rng, W, sp) for sp in spans]
    payloads = _sign_payloads(rng, ns, per_t)
    got = gpu_aggregate("sign", 0.01, ns, payloads, 1.0 / W)
    want = O.aggregate_set("sign", ns, payloads, 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), (t, spans[t])


@pytest.mark.parametrize("W", [32, 64, 128])
def test_sign_aggregate_integer_form_extremes(W):
    # largest sums the int32 form admits: every scale at the top of the
    # widest span it takes, all signs equal (both polarities) and mixed
    int_limit, _ = _gpu_tiers(W)
    top = np.float32(np.nextafter(np.float32(2.0 ** (-9 + int_limit)), np.float32(0)))
    scales = np.full(W, top, np.float32)
    scales[0] = np.float32(2.0 ** -10)  # sets emin, so the span is int_limit
    ns = [4096 + 64, 4096 + 64, 777]
    wc = [O.words_for(n) for n in ns]
    rng = np.random.default_rng(61)
    payloads = []
    for w in range(W):
        words = [np.zeros(wc[0], np.uint32), np.full(wc[1], 0xFFFFFFFF, np.uint32),
                 WL.random_sign_words(rng, [ns[2]], [wc[2]])[0]]
        words[1][-1] &= np.uint32((1 << (ns[1] % 32)) - 1) if ns[1] % 32 else np.uint32(0xFFFFFFFF)
        payloads.append({"bits": np.concatenate(words), "scale": scales.copy(), "off": O.word_offsets(ns)})
    got = gpu_aggregate("sign", 0.01, ns, payloads, 1.0)
    want = O.aggregate_set("sign", ns, payloads, 1.0)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t
    assert np.all(got[0] > 0) and np.all(got[1] < 0)


# ---------------------------------------------------- residual update (API)

@pytest.mark.parametrize("kind", ["topk", "randk", "sign"])
def test_residual_update_matches_fused(kind):
    import torch
    from paper_2205_14465_amd import binding as B
    from tests.helpers import torch_dev
    rng = np.random.default_rng(41)
    ns = [33, 4096 * 2 + 9, 70000]
    grads, resids = make_set(ns, rng)
    fused, fused_e = gpu_compress(kind, 0.01, SEED, grads, resids)
    v = [g + e for g, e in zip(grads, resids)]
    own, _ = gpu_compress(kind, 0.01, SEED, v, None)
    dg = [torch_dev(g) for g in grads]
    de = [torch_dev(e) for e in resids]
    if kind == "sign":
        dp = {"bits": torch_dev(own["bits"].view(np.int32)), "scale": torch_dev(own["scale"])}
    else:
        dp = {"idx": torch_dev(own["idx"].view(np.int32)), "val": torch_dev(own["val"])}
    B.bytecomp_residual_update(kind, 0.01, dg, de, dp)
    torch.cuda.synchronize()
    split_e = [e.cpu().numpy() for e in de]
    assert_resid_equal(split_e, fused_e)
    # and against the oracle's residual update
    for t in range(len(ns)):
        sl = slice(own["off"][t], own["off"][t + 1])
        if kind == "sign":
            want = O.residual_update_sign(grads[t], resids[t], own["bits"][sl], own["scale"][t])
        else:
            want = O.residual_update_sparse(grads[t], resids[t], own["idx"][sl], own["val"][sl])
        assert np.array_equal(bits(split_e[t]), bits(want)), t


@pytest.mark.parametrize("kind, kernel", [("sign", "aggregate_sign"), ("topk", "aggregate_sparse")])
def test_time_next_launch_brackets_the_kernel(kind, kernel):
    """The timed launch records both events once, inside the call's span;
    the following call is not timed again."""
    import torch
    from paper_2205_14465_amd import binding as B
    from tests.helpers import torch_dev
    rng = np.random.default_rng(5)
    ns = [70001, 4096, 300000]
    grads, resids = make_set(ns, rng)
    pay, _ = gpu_compress(kind, 0.01, SEED, grads, resids)
    payloads = [pay] * 3
    outs_dev = [torch.empty(n, dtype=torch.float32, device="cuda") for n in ns]
    ws = B.alloc_workspace(kind, 0.01, ns, 3)
    dev_pay = []
    for p in payloads:
        if kind == "sign":
            dev_pay.append({"bits": torch_dev(p["bits"].view(np.int32)), "scale": torch_dev(p["scale"])})
        else:
            dev_pay.append({"idx": torch_dev(p["idx"].view(np.int32)), "val": torch_dev(p["val"])})
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record()
    torch.cuda.synchronize()
    B.bytecomp_time_next_launch(kernel, ev[1], ev[2])
    ev[0].record()
    B.bytecomp_decompress_aggregate(kind, 0.01, dev_pay, ns, outs_dev, 1.0, ws)
    ev[3].record()
    torch.cuda.synchronize()
    k_ms = ev[1].elapsed_time(ev[2])
    call_ms = ev[0].elapsed_time(ev[3])
    assert 0.0 < k_ms <= call_ms
    # the request was consumed: a second call leaves the events where they were
    assert not B.bytecomp_time_next_launch(None, None, None)
    B.bytecomp_decompress_aggregate(kind, 0.01, dev_pay, ns, outs_dev, 1.0, ws)
    torch.cuda.synchronize()
    assert ev[1].elapsed_time(ev[2]) == k_ms
    assert B.bytecomp_device_status(ws) == 0
    # a request for a kernel the call does not launch stays pending
    B.bytecomp_time_next_launch("randk_stream", ev[1], ev[2])
    B.bytecomp_decompress_aggregate(kind, 0.01, dev_pay, ns, outs_dev, 1.0, ws)
    torch.cuda.synchronize()
    assert B.bytecomp_time_next_launch(None, None, None)
