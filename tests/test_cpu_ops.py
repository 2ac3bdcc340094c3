"""The library's host (CPU-offloading) operators against the oracle.

bytecomp_cpu_compress / bytecomp_cpu_decompress_aggregate run on the CPU in
libbytecomp.so (no GPU call), so these tests run without a GPU.  Bar:
sparse payloads, residuals and every aggregate bit-exact; the sign scale
within the fp64-summation-order tolerance (one fp32 rounding of an fp64
sum taken in another order), with sign bits exact and the residual exactly
v - (+-s) for the scale the operator produced.
"""
import numpy as np
import pytest

import oracle as O

from .exact_ref import same_f32_arrays

B = pytest.importorskip("paper_2205_14465_amd.binding")

SPARSE = ("topk", "randk")
NS = [0, 1, 31, 32, 33, 4097, 65535, 65536, 65537, 300001, 5000]


def _set(rng, ns, f16=False):
    grads = [(rng.standard_normal(n) * 10.0 ** rng.uniform(-3, -1)).astype(np.float16 if f16 else np.float32)
             for n in ns]
    resids = [(rng.standard_normal(n) * 1e-4).astype(np.float32) for n in ns]
    return grads, resids


def _cpu_compress(kind, ratio, seed, grads, resids, threads):
    out = B.cpu_alloc_payload(kind, ratio, [g.size for g in grads])
    e = None if resids is None else [r.copy() for r in resids]
    B.bytecomp_cpu_compress(kind, ratio, seed, grads, e, out, threads)
    return out, e


@pytest.mark.parametrize("kind", SPARSE)
@pytest.mark.parametrize("threads", [1, 4])
@pytest.mark.parametrize("f16", [False, True])
def test_cpu_sparse_compress_bit_exact(kind, threads, f16):
    rng = np.random.default_rng(700 + 3 * SPARSE.index(kind) + threads + (50 if f16 else 0))
    grads, resids = _set(rng, NS, f16)
    want, want_e = O.compress_set(kind, 0.01, 77, grads, resids)
    got, got_e = _cpu_compress(kind, 0.01, 77, grads, resids, threads)
    assert got["off"] == [int(x) for x in want["off"]]
    total = int(want["off"][-1])
    assert np.array_equal(got["idx"][:total], want["idx"])
    assert np.array_equal(got["val"][:total].view(np.uint32), want["val"].view(np.uint32))
    for a, b in zip(got_e, want_e):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_cpu_sampled_kind_is_exact_topk():
    """The host form of the sampled kind selects the exact top-k (the CPU
    has no use for the sampling shortcut); its result is the oracle's
    exact top-k."""
    rng = np.random.default_rng(711)
    grads, resids = _set(rng, [70001, 4097, 3])
    want, want_e = O.compress_set("topk", 0.02, 5, grads, resids)
    got, got_e = _cpu_compress("topk_sampled", 0.02, 5, grads, resids, 3)
    total = int(want["off"][-1])
    assert np.array_equal(got["idx"][:total], want["idx"])
    assert np.array_equal(got["val"][:total].view(np.uint32), want["val"].view(np.uint32))
    for a, b in zip(got_e, want_e):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_cpu_topk_ties_take_lower_index():
    g = np.zeros(200000, np.float32)
    g[::7] = 1.0
    g[5] = -1.0
    got, _ = _cpu_compress("topk", 0.001, 0, [g], None, 4)
    want, _ = O.compress_set("topk", 0.001, 0, [g], None)
    assert np.array_equal(got["idx"][:want["idx"].size], want["idx"])


@pytest.mark.parametrize("threads", [1, 4])
@pytest.mark.parametrize("f16", [False, True])
def test_cpu_sign_compress(threads, f16):
    rng = np.random.default_rng(720 + threads + (9 if f16 else 0))
    grads, resids = _set(rng, NS, f16)
    want, _ = O.compress_set("sign", 0.0, 0, grads, resids)
    got, got_e = _cpu_compress("sign", 0.0, 0, grads, resids, threads)
    total = int(want["off"][-1])
    assert np.array_equal(got["bits"][:total], want["bits"])
    for t, g in enumerate(grads):
        s_want, s_got = float(want["scale"][t]), float(got["scale"][t])
        assert abs(s_got - s_want) <= 1e-6 * abs(s_want), (t, s_got, s_want)
        # residual: exactly the oracle's residual rule at the operator's scale
        ref_e = O.residual_update_sign(g, resids[t], got["bits"][got["off"][t]:got["off"][t + 1]],
                                       np.float32(s_got))
        assert np.array_equal(got_e[t].view(np.uint32), ref_e.view(np.uint32))


@pytest.mark.parametrize("kind", ("topk", "randk", "sign"))
@pytest.mark.parametrize("threads", [1, 4])
def test_cpu_aggregate_bit_exact(kind, threads):
    rng = np.random.default_rng(740 + threads + 7 * ("topk", "randk", "sign").index(kind))
    ns = NS
    pays = []
    for w in range(5):
        grads, _ = _set(rng, ns, f16=False)
        p, _ = O.compress_set(kind, 0.01, 11 + w, grads, None)
        pays.append(p)
    ref = O.aggregate_set(kind, ns, pays, 0.2)
    outs = [np.full(n, np.nan, np.float32) for n in ns]
    B.bytecomp_cpu_decompress_aggregate(kind, 0.01, pays, ns, outs, 0.2, threads)
    for t, (a, b) in enumerate(zip(outs, ref)):
        assert same_f32_arrays(a, b), t


def _sign_payloads(rng, n, scales):
    pays = []
    for s in scales:
        w = rng.integers(0, 2**32, (n + 31) // 32, dtype=np.uint64).astype(np.uint32)
        pays.append({"bits": w, "scale": np.array([s], np.float32), "off": [0, w.size]})
    return pays


@pytest.mark.parametrize("scales", [
    # spans the fp64 form covers, and spans that need the wide limbs
    [1.0, 0.5, 3.0, 1e-3],
    [1.0, 2.0 ** -40, 3.0, 2.0 ** 60],
    [2.0 ** 127 * 1.5, 2.0 ** -126, 2.0 ** -149, 1e-45, 7.0],
    [3.4e38, 3.4e38, 3.4e38, 1.0],
    [0.0, 0.0, 1e-40, 0.0],
    [np.inf, 1.0, 2.0, 3.0],
    [np.inf, -np.inf, 1.0, 1.0],
    [np.nan, 1.0, 1.0, 1.0],
    [-1.0, 1.0, 2.0 ** -100, -2.0 ** 100],
])
def test_cpu_sign_aggregate_exact_sum(scales):
    rng = np.random.default_rng(760)
    n = 70001
    pays = _sign_payloads(rng, n, scales)
    ref = O.aggregate_set("sign", [n], pays, 0.5)[0]
    out = [np.empty(n, np.float32)]
    B.bytecomp_cpu_decompress_aggregate("sign", 0.0, pays, [n], out, 0.5, 3)
    assert same_f32_arrays(out[0], ref)


def test_cpu_payload_crosses_to_oracle_aggregate():
    """A payload made by the host compressor aggregates like the oracle's."""
    rng = np.random.default_rng(780)
    ns = [4097, 65537, 3]
    pays = []
    for w in range(3):
        grads, _ = _set(rng, ns)
        pays.append(_cpu_compress("randk", 0.05, 40 + w, grads, None, 2)[0])
    ref = O.aggregate_set("randk", ns, pays, 1.0)
    outs = [np.empty(n, np.float32) for n in ns]
    B.bytecomp_cpu_decompress_aggregate("randk", 0.05, pays, ns, outs, 1.0, 2)
    for a, b in zip(outs, ref):
        assert same_f32_arrays(a, b)


def test_cpu_errors():
    g = np.ones(100, np.float32)
    out = B.cpu_alloc_payload("topk", 0.1, [100])
    with pytest.raises(B.BytecompError, match="BC_E_KIND"):
        B.bytecomp_cpu_compress("terngrad", 0.1, 0, [g], None, B.cpu_alloc_payload("terngrad", 0.1, [100]))
    with pytest.raises(B.BytecompError, match="BC_E_RATIO"):
        B.bytecomp_cpu_compress("topk", 0.0, 0, [g], None, out)
    with pytest.raises(B.BytecompError, match="BC_E_DTYPE"):
        B.bytecomp_cpu_compress("topk", 0.1, 0, [g.astype(np.float64)], None, out)
    with pytest.raises(B.BytecompError, match="BC_E_COUNT"):
        B.bytecomp_cpu_decompress_aggregate("topk", 0.1, [], [100], [np.empty(100, np.float32)], 1.0)
    with pytest.raises(B.BytecompError, match="BC_E_KIND"):
        B.bytecomp_cpu_decompress_aggregate("qsgd8", 0.1, [out], [100], [np.empty(100, np.float32)], 1.0)
