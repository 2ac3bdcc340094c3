"""GPU parity of the stochastic quantizers (TernGrad 2-bit, QSGD 4- and
8-bit; paper Sec. 2.3) against the CPU oracle, through the C ABI.

Every result is deterministic for a given seed, so codes, scales,
residuals and aggregates must all match the oracle bit for bit: the scale
is a maximum (no summation order), the rounding decisions use the same
fp32 operations and the same Philox4x64-10 uniforms on both sides, and
the aggregate adds the workers in the same order (4- and 8-bit, and 2-bit
outside the exact form) or forms the exact sum (2-bit exact form).
"""
import numpy as np
import pytest

import oracle as O
from tests.exact_ref import same_f32_arrays
from tests.helpers import assert_resid_equal, bits, gpu_aggregate, gpu_compress

pytestmark = pytest.mark.gpu

KINDS = ["terngrad", "qsgd4", "qsgd8"]
RAGGED = [0, 1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 33, 1000, 4095, 4096, 4097, 8191, 3 * 4096 + 17, 65537,
          100003]
SEED = 2205


def make_set(ns, rng, dtype=np.float32, ef=True):
    grads = [(rng.standard_normal(n) * 10.0 ** rng.uniform(-3, -1)).astype(dtype) for n in ns]
    for g in grads:
        if g.size >= 4:
            g[:2] = np.array([0.0, -0.0], dtype)
    resids = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in ns] if ef else None
    return grads, resids


def check(kind, got, got_e, want, want_e):
    assert np.array_equal(got["off"], want["off"])
    assert np.array_equal(got["bits"], want["bits"]), np.flatnonzero(got["bits"] != want["bits"])[:5]
    assert np.array_equal(bits(got["scale"]), bits(want["scale"]))
    if want_e is not None:
        assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_quant_compress_ragged(kind, dtype):
    rng = np.random.default_rng(1 + KINDS.index(kind))
    grads, resids = make_set(RAGGED, rng, dtype)
    got, got_e = gpu_compress(kind, 1.0, SEED, grads, resids)
    want, want_e = O.compress_set(kind, 1.0, SEED, grads, resids)
    check(kind, got, got_e, want, want_e)


@pytest.mark.parametrize("kind", KINDS)
def test_quant_error_feedback_off_and_zero_tensors(kind):
    rng = np.random.default_rng(9)
    ns = [0, 5, 4096, 5000]
    grads, _ = make_set(ns, rng)
    grads[2][:] = 0.0  # all-zero tensor: scale 0, codes 0
    got, _ = gpu_compress(kind, 1.0, SEED, grads, None)
    want, _ = O.compress_set(kind, 1.0, SEED, grads, None)
    check(kind, got, None, want, None)


@pytest.mark.parametrize("kind", KINDS)
def test_quant_large_tensor_takes_the_finalize_path(kind):
    # more than 1024 chunks of 4096 elements: the scale comes from a
    # separate reduction over the tensor's chunk maxima
    rng = np.random.default_rng(13)
    ns = [1024 * 4096 + 4097, 300]
    grads, resids = make_set(ns, rng)
    got, got_e = gpu_compress(kind, 1.0, SEED + 1, grads, resids, tensor_ids=[7, 3])
    # the oracle keys each tensor's stream by its id
    want_e = []
    for t, tid in enumerate([7, 3]):
        w, s, e = O.compress_quant(grads[t], resids[t], O.QUANT_BITS[kind], SEED + 1, tid)
        seg = slice(got["off"][t], got["off"][t + 1])
        assert np.array_equal(got["bits"][seg], w), t
        assert bits(got["scale"][t]) == bits(np.float32(s))
        want_e.append(e)
    assert_resid_equal(got_e, want_e)


@pytest.mark.parametrize("kind", KINDS)
def test_quant_seed_changes_the_codes(kind):
    rng = np.random.default_rng(21)
    grads, resids = make_set([50000], rng)
    a, _ = gpu_compress(kind, 1.0, 1, grads, resids)
    b, _ = gpu_compress(kind, 1.0, 2, grads, resids)
    assert not np.array_equal(a["bits"], b["bits"])
    assert bits(a["scale"][0]) == bits(b["scale"][0])


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("W", [1, 3, 16, 64])
def test_quant_aggregate_ragged(kind, W):
    rng = np.random.default_rng(100 + W)
    ns = RAGGED
    pays = []
    for w in range(W):
        grads, _ = make_set(ns, rng)
        pays.append(O.compress_set(kind, 1.0, 1000 + w, grads, None)[0])
    alpha = 1.0 / W
    got = gpu_aggregate(kind, 1.0, ns, pays, alpha)
    want = O.aggregate_set(kind, ns, pays, alpha)
    for t, n in enumerate(ns):
        assert np.array_equal(bits(got[t]), bits(want[t])), (t, n)


@pytest.mark.parametrize("kind", KINDS)
def test_quant_aggregate_any_code_pattern(kind):
    # arbitrary words (codes with the sign bit and level 0 included) and
    # scales spread over many binades, zero among them
    rng = np.random.default_rng(77)
    ns = [1, 33, 4096, 9000]
    W = 5
    b = O.QUANT_BITS[kind]
    off = O.quant_word_offsets(ns, b)
    pays = []
    for w in range(W):
        words = rng.integers(0, 2**32, size=int(off[-1]), dtype=np.uint64).astype(np.uint32)
        for t, n in enumerate(ns):  # codes past each tensor's end are zero
            used = n * b % 32
            if used:
                words[off[t + 1] - 1] &= np.uint32((1 << used) - 1)
        scale = (10.0 ** rng.uniform(-8, 3, size=len(ns))).astype(np.float32)
        if w == 1:
            scale[0] = 0.0
        pays.append({"bits": words, "scale": scale, "off": off})
    got = gpu_aggregate(kind, 1.0, ns, pays, 0.5)
    want = O.aggregate_set(kind, ns, pays, 0.5)
    for t in range(len(ns)):
        assert np.array_equal(bits(got[t]), bits(want[t])), t


@pytest.mark.parametrize("kind", KINDS)
def test_quant_residual_update_matches_fused(kind):
    import torch
    from paper_2205_14465_amd import binding as B
    from tests.helpers import torch_dev
    rng = np.random.default_rng(31)
    ns = [100, 4097, 70000]
    grads, resids = make_set(ns, rng)
    fused, fused_e = gpu_compress(kind, 1.0, SEED, grads, resids)
    dg = [torch_dev(g) for g in grads]
    de = [torch_dev(e) for e in resids]
    own = {"bits": torch_dev(fused["bits"].view(np.int32)), "scale": torch_dev(fused["scale"])}
    B.bytecomp_residual_update(kind, 1.0, dg, de, own)
    torch.cuda.synchronize()
    assert_resid_equal([e.cpu().numpy() for e in de], fused_e)
    want = [O.residual_update_quant(grads[t], resids[t], O.QUANT_BITS[kind],
                                    fused["bits"][fused["off"][t]:fused["off"][t + 1]], fused["scale"][t])
            for t in range(len(ns))]
    assert_resid_equal([e.cpu().numpy() for e in de], want)


def _tern_payloads(rng, ns, W, spread):
    """Arbitrary 2-bit code words (every code, the sign bit with level 0
    included) and per-tensor scales 2^e (1 + 0.05 N(0,1)) with e drawn per
    worker from `spread` binades (0: one band, so the exact form applies)."""
    off = O.quant_word_offsets(ns, 2)
    pays = []
    for w in range(W):
        words = rng.integers(0, 2**32, size=max(int(off[-1]), 1), dtype=np.uint64).astype(np.uint32)[:int(off[-1])]
        for t, n in enumerate(ns):  # codes past each tensor's end are zero
            used = n * 2 % 32
            if used:
                words[off[t + 1] - 1] &= np.uint32((1 << used) - 1)
        e = rng.integers(0, spread + 1, size=len(ns)) if spread else np.zeros(len(ns), int)
        scale = (1e-3 * 2.0 ** e * (1 + 0.05 * rng.standard_normal(len(ns)))).astype(np.float32)
        pays.append({"bits": words, "scale": scale, "off": off})
    return pays


@pytest.mark.parametrize("W", [1, 2, 4, 5, 13, 16, 17, 33, 48, 64])
def test_terngrad_aggregate_exact_form(W):
    # every tensor in the exact form: the table path, exact sums rounded once
    rng = np.random.default_rng(700 + W)
    ns = [1, 15, 16, 17, 4095, 4096, 4097, 3 * 4096 + 33, 0, 50000]
    pays = _tern_payloads(rng, ns, W, 0)
    got = gpu_aggregate("terngrad", 1.0, ns, pays, 1.0 / W)
    want = O.aggregate_set("terngrad", ns, pays, 1.0 / W)
    for t, n in enumerate(ns):
        assert np.array_equal(bits(got[t]), bits(want[t])), (t, n)


@pytest.mark.parametrize("W", [8, 64, 65, 72])
def test_terngrad_aggregate_mixed_forms(W):
    # tensors of one call on both sides of the kernel's table form: spreads
    # of a few binades and of 40 to 200, zero, subnormal and non-finite
    # scales among narrow ones, and more than 64 workers (no tables); every
    # output is the exact sum rounded once (NaN where the rule says so)
    rng = np.random.default_rng(800 + W)
    ns = [5000, 4096 * 5 + 7, 300, 12000, 4100, 999, 64]
    pays = _tern_payloads(rng, ns, W, 0)
    for w, p in enumerate(pays):
        p["scale"][1] = np.float32(p["scale"][1] * 2.0 ** (3 * (w % 4)))       # a few binades
        if w == 2:
            p["scale"][2] = np.float32(0.0)                                 # a zero scale
        p["scale"][3] = np.float32(np.ldexp(1.0 + rng.random(), int(rng.integers(-100, 100))))  # ~200
        p["scale"][4] = np.float32(np.ldexp(1.0 + rng.random(), int(rng.integers(-149, -127))))  # subnormal
        if w == 1:
            p["scale"][5] = np.float32(np.inf)
        if w == W - 1:
            p["scale"][6] = np.float32(np.nan)
    got = gpu_aggregate("terngrad", 1.0, ns, pays, 0.25)
    want = O.aggregate_set("terngrad", ns, pays, 0.25)
    for t, n in enumerate(ns):
        assert same_f32_arrays(got[t], want[t]), (t, n)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_quant_compress_long_and_short_tensors(kind, dtype):
    # calls with tensors longer than the resident grid of the one-pass
    # kernel (more than 1280 chunks on any current part) among short ones
    # take the two passes; empty tensors included
    rng = np.random.default_rng(41 + KINDS.index(kind))
    ns = [5000, 1400 * 4096 + 123, 0, 77, 4096 * 3, 1300 * 4096, 1]
    grads, resids = make_set(ns, rng, dtype)
    got, got_e = gpu_compress(kind, 1.0, SEED + 7, grads, resids)
    want, want_e = O.compress_set(kind, 1.0, SEED + 7, grads, resids)
    check(kind, got, got_e, want, want_e)
