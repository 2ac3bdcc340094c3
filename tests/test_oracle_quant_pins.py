"""Pins of the oracle's stochastic quantizers (TernGrad 2-bit, QSGD 4-bit
and 8-bit with the largest magnitude as the scale; paper Sec. 2.3 names
8-, 2- and 1-bit quantization with error feedback).

Against things other than the oracle itself: numpy.random.Philox for the
uniforms, numpy's little-endian byte view for the code packing, the
hand-worked examples in tests/golden/hand_examples.json, closed forms on
inputs whose levels are whole numbers, the unbiasedness and variance bound
of stochastic rounding measured over many seeds, brute-force ordered sums
for the 4- and 8-bit aggregate, and exact rational sums rounded once (with
the order-free rule for non-finite scales) for the 2-bit aggregate.
"""
import json
import os

import numpy as np
import pytest

import oracle as O

from .exact_ref import exact_round_f32, same_f32, xsum_f32

f32 = np.float32
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
BITS = (2, 4, 8)


def numpy_philox_block(ctr, key):
    """The Philox4x64-10 block at counter ctr from numpy (which advances its
    counter once before producing a block)."""
    prev = np.array(ctr, dtype=np.uint64)
    m = np.uint64(2**64 - 1)
    for i in range(4):
        if prev[i] == 0:
            prev[i] = m
        else:
            prev[i] -= np.uint64(1)
            break
    bg = np.random.Philox(counter=prev, key=np.array(key, dtype=np.uint64))
    return bg.random_raw(4).astype(np.uint64)


def numpy_uniform(seed, tid, i):
    w = numpy_philox_block([tid, i // 8, 0, 0], [seed, 2])
    x = int(w[(i % 8) // 2])
    u = (x >> 32) if i % 2 else (x & 0xFFFFFFFF)
    return f32((u >> 8) * 2.0**-24)


def unpack_codes(words, n, bits):
    """Codes from packed words through numpy's little-endian byte view."""
    b = np.ascontiguousarray(words, np.uint32).view(np.uint8)
    if bits == 8:
        return b[:n].astype(np.uint32)
    per = 8 // bits
    out = np.zeros(b.size * per, np.uint32)
    for j in range(per):
        out[j::per] = (b >> (bits * j)) & ((1 << bits) - 1)
    return out[:n]


def decode_np(codes, bits, m):
    s = (1 << (bits - 1)) - 1
    level = (codes & ((1 << (bits - 1)) - 1)).astype(f32)
    unit = f32(np.float64(m) / np.float64(s))
    mag = (level * unit).astype(f32)
    neg = ((codes >> (bits - 1)) & 1).astype(bool) & (level > 0)
    d = np.where(neg, -mag, mag).astype(f32)
    return np.where(level > 0, d, f32(0.0)).astype(f32)


def test_levels_and_word_counts():
    assert [O.quant_levels(b) for b in BITS] == [1, 7, 127]
    assert O.quant_levels(3) == 0
    for b in BITS:
        for n in (0, 1, 15, 16, 17, 33, 1000):
            assert O.quant_words(n, b) == -(-n * b // 32)


def test_uniform_matches_numpy_philox():
    rng = np.random.default_rng(3)
    for _ in range(60):
        seed = int(rng.integers(0, 2**63))
        tid = int(rng.integers(0, 5000))
        i = int(rng.integers(0, 2**33))
        assert O.quant_uniform(seed, tid, i) == numpy_uniform(seed, tid, i)


@pytest.mark.parametrize("case", [0, 1])
def test_hand_examples(case):
    ex = json.load(open(GOLDEN))["quant"][case]
    g = np.array([float(x) for x in ex["g"]], dtype=np.float64).astype(f32)
    e = np.array([float(x) for x in ex["e"]], dtype=np.float64).astype(f32)
    words, scale, e_new = O.compress_quant(g, e, ex["bits"], ex["seed"], ex["tensor_id"])
    assert scale == f32(float(ex["scale"]))
    assert [int(w) for w in words] == [int(h, 16) for h in ex["words"]]
    assert [int(x) for x in e_new.view(np.uint32)] == [int(h, 16) for h in ex["e_new_bits"]]


@pytest.mark.parametrize("bits", BITS)
def test_whole_number_levels_are_deterministic(bits):
    # max |v| = s makes inv = unit = 1: every |v| that is a whole number is
    # its own level, for any seed; decoding returns v exactly
    s = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(bits)
    n = 301
    v = rng.integers(-s, s + 1, size=n).astype(f32)
    v[7] = f32(s)
    for seed in (0, 1, 12345):
        words, scale, e_new = O.compress_quant(v, np.zeros(n, f32), bits, seed, 11)
        assert scale == f32(s)
        codes = unpack_codes(words, n, bits)
        level = np.abs(v).astype(np.uint32)
        want = np.where(level > 0, level | ((v < 0).astype(np.uint32) << (bits - 1)), 0)
        assert np.array_equal(codes, want)
        assert np.all(e_new == 0.0)


@pytest.mark.parametrize("bits", BITS)
def test_half_levels_follow_the_uniform(bits):
    # |v| = l + 1/2 in units of 1 (max = s): level l + 1 exactly when U < 1/2
    s = (1 << (bits - 1)) - 1
    n = 200
    rng = np.random.default_rng(40 + bits)
    lv = rng.integers(0, s, size=n)
    v = (lv + 0.5).astype(f32) * np.where(rng.random(n) < 0.5, -1, 1).astype(f32)
    v[0] = f32(s)
    seed, tid = 777, 2
    words, scale, _ = O.compress_quant(v, None, bits, seed, tid)
    codes = unpack_codes(words, n, bits)
    for i in range(1, n):
        up = numpy_uniform(seed, tid, i) < f32(0.5)
        want_level = int(lv[i]) + (1 if up else 0)
        assert int(codes[i]) & s == want_level, i
        if want_level:
            assert int(codes[i]) >> (bits - 1) == int(v[i] < 0), i


@pytest.mark.parametrize("bits", BITS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_scale_and_level_bracket(bits, dtype):
    s = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(5 + bits)
    n = 3000
    g = (rng.standard_normal(n) * 0.02).astype(dtype)
    e = (rng.standard_normal(n) * 0.002).astype(f32)
    words, m, e_new = O.compress_quant(g, e, bits, 99, 4)
    v = (g.astype(f32) + e).astype(f32)
    assert m == np.max(np.abs(v))
    codes = unpack_codes(words, n, bits)
    level = codes & s
    inv = f32(np.float64(s) / np.float64(m))
    x = (np.abs(v) * inv).astype(f32)
    lo = np.minimum(np.floor(x), s)
    assert np.all((level == lo) | (level == lo + 1))
    assert np.all(level <= s)
    nz = level > 0
    assert np.array_equal((codes[nz] >> (bits - 1)).astype(bool), np.signbit(v[nz]))
    assert np.all(codes[~nz] == 0)
    # padding bits of the last word are clear
    used = n * bits % 32
    if used:
        assert int(words[-1]) >> used == 0


@pytest.mark.parametrize("bits", BITS)
def test_residual_is_correctly_rounded(bits):
    rng = np.random.default_rng(60 + bits)
    n = 4000
    g = (rng.standard_normal(n) * 0.01).astype(f32)
    e = (rng.standard_normal(n) * 0.001).astype(f32)
    words, m, e_new = O.compress_quant(g, e, bits, 3, 8)
    v = (g + e).astype(f32)
    d = decode_np(unpack_codes(words, n, bits), bits, m)
    exact = v.astype(np.float64) - d.astype(np.float64)
    assert np.array_equal(e_new, exact.astype(f32))
    ulp = np.spacing(np.abs(e_new)).astype(np.float64)
    assert np.all(np.abs(e_new.astype(np.float64) - exact) <= 0.5 * ulp)
    # the residual update entry point from the same payload agrees
    assert np.array_equal(O.residual_update_quant(g, e, bits, words, m), e_new)


@pytest.mark.parametrize("bits", BITS)
def test_stochastic_rounding_is_unbiased(bits):
    # E[decode] = v and Var <= unit^2 / 4 per element: over N seeds the mean
    # decode lies within 6 standard errors of v (levels rounded to fp32 add
    # at most a few ulp of the level value)
    s = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(80 + bits)
    n, N = 257, 2000
    v = (rng.standard_normal(n) * 0.05).astype(f32)
    v[:3] = [0.0, -0.0, np.max(np.abs(v)) * 0.5]
    acc = np.zeros(n, np.float64)
    for seed in range(N):
        words, m, _ = O.compress_quant(v, None, bits, seed, 1)
        acc += decode_np(unpack_codes(words, n, bits), bits, m).astype(np.float64)
    mean = acc / N
    unit = float(np.max(np.abs(v))) / s
    tol = 6 * (unit / 2) / np.sqrt(N) + 4 * np.spacing(f32(float(np.max(np.abs(v))))).astype(np.float64)
    assert np.all(np.abs(mean - v.astype(np.float64)) <= tol)
    assert mean[0] == 0.0 and mean[1] == 0.0


def test_terngrad_nonzero_frequency():
    # TernGrad: element i is nonzero with probability |v_i| / max|v|
    n, N = 64, 3000
    v = np.linspace(-1.0, 1.0, n).astype(f32)
    hits = np.zeros(n)
    for seed in range(N):
        words, m, _ = O.compress_quant(v, None, 2, seed, 0)
        hits += unpack_codes(words, n, 2) != 0
    p = np.abs(v).astype(np.float64) / float(np.max(np.abs(v)))
    se = np.sqrt(np.maximum(p * (1 - p), 1e-12) / N)
    assert np.all(np.abs(hits / N - p) <= 6 * se + 1e-9)


@pytest.mark.parametrize("bits", BITS)
def test_zero_and_empty_tensors(bits):
    words, m, e_new = O.compress_quant(np.zeros(0, f32), np.zeros(0, f32), bits, 1, 0)
    assert words.size == 0 and m == 0.0 and e_new.size == 0
    v = np.array([0.0, -0.0, 0.0], f32)
    e = np.array([-0.0, -0.0, 0.0], f32)
    words, m, e_new = O.compress_quant(v, e, bits, 1, 0)
    assert m == 0.0 and np.all(words == 0)
    assert np.array_equal(e_new.view(np.uint32), ((v + e).astype(f32)).view(np.uint32))


@pytest.mark.parametrize("bits", (4, 8))
def test_aggregate_ordered_bruteforce(bits):
    # 4- and 8-bit codes: worker-ordered fp32 sums; worker w's gradient is
    # scaled by 2^(3w) so that the additions round
    rng = np.random.default_rng(90 + bits)
    n, W = 37, 5
    pays = [O.compress_quant((rng.standard_normal(n) * 10.0 ** rng.uniform(-3, 0) * 2.0 ** (3 * w)).astype(f32),
                             None, bits, 100 + w, 0)[:2] for w in range(W)]
    alpha = f32(0.25)
    got = O.aggregate_quant(n, bits, [p[0] for p in pays], [p[1] for p in pays], float(alpha))
    for i in range(n):
        acc = f32(0.0)
        for wds, m in pays:
            acc = f32(acc + decode_np(unpack_codes(wds, n, bits), bits, m)[i])
        assert got[i].view(np.uint32) == f32(alpha * acc).view(np.uint32), i
    # W = 1 and alpha = 1: the decode itself
    one = O.aggregate_quant(n, bits, [pays[0][0]], [pays[0][1]], 1.0)
    assert np.array_equal(one.view(np.uint32),
                          (f32(0.0) + decode_np(unpack_codes(pays[0][0], n, bits), bits, pays[0][1])).view(np.uint32))


@pytest.mark.parametrize("W", [1, 3, 16, 64])
def test_terngrad_aggregate_exact_form_per_element(W):
    # the exact rational sum of the decoded values, rounded once, times alpha
    rng = np.random.default_rng(400 + W)
    n = 53
    pays = []
    for w in range(W):
        g = (rng.standard_normal(n) * 1e-3 * (1 + 0.05 * rng.standard_normal())).astype(f32)
        pays.append(O.compress_quant(g, None, 2, 500 + w, 0)[:2])
    scales = [p[1] for p in pays]
    alpha = f32(1.0 / W)
    got = O.aggregate_quant(n, 2, [p[0] for p in pays], scales, float(alpha))
    dec = [decode_np(unpack_codes(wds, n, 2), 2, m) for wds, m in pays]
    for i in range(n):
        want = f32(alpha * exact_round_f32([d[i] for d in dec]))
        assert got[i].view(np.uint32) == want.view(np.uint32), i


def test_terngrad_aggregate_exact_differs_from_ordered_somewhere():
    # the two readings are distinguishable: with scales that are not exact
    # multiples of each other some ordered fp32 sums round differently
    rng = np.random.default_rng(411)
    n, W = 4000, 64
    pays = []
    for w in range(W):
        g = (rng.standard_normal(n) * 1e-3 * (1 + 0.05 * rng.standard_normal())).astype(f32)
        pays.append(O.compress_quant(g, None, 2, 600 + w, 0)[:2])
    got = O.aggregate_quant(n, 2, [p[0] for p in pays], [p[1] for p in pays], 1.0)
    dec = np.array([decode_np(unpack_codes(wds, n, 2), 2, m) for wds, m in pays])
    ordered = np.zeros(n, f32)
    for w in range(W):
        ordered = (ordered + dec[w]).astype(f32)
    assert np.any(got.view(np.uint32) != ordered.view(np.uint32))
    exact64 = dec.astype(np.float64).sum(axis=0)  # exact: 24 + 1 + 6 bits
    assert np.array_equal(got, exact64.astype(f32))


@pytest.mark.parametrize("W", [2, 7, 64, 100])
def test_terngrad_aggregate_exact_at_wide_spans(W):
    # worker scales spread over up to 200 binades (subnormal ones included):
    # still the exact sum of the decoded values, rounded once
    rng = np.random.default_rng(700 + W)
    n = 45
    pays = []
    for w in range(W):
        g = (rng.standard_normal(n) * 2.0 ** int(rng.integers(-140, 60))).astype(f32)
        pays.append(O.compress_quant(g, None, 2, 800 + w, 0)[:2])
    scales = [p[1] for p in pays]
    got = O.aggregate_quant(n, 2, [p[0] for p in pays], scales, 0.5)
    dec = [decode_np(unpack_codes(wds, n, 2), 2, m) for wds, m in pays]
    for i in range(n):
        want = f32(f32(0.5) * exact_round_f32([d[i] for d in dec]))
        assert same_f32(got[i], want), i


def test_terngrad_aggregate_non_finite_scales():
    # a level-0 code decodes to 0 whatever the scale; a nonzero code of an
    # infinite or NaN scale follows the order-free rule
    def word(codes):
        return np.array([sum(int(c) << (2 * q) for q, c in enumerate(codes))], np.uint32)
    inf, nan = f32(np.inf), f32(np.nan)
    cases = [
        ([[0, 1], [1, 1]], [nan, f32(2.0)], [2.0, np.nan]),      # NaN scale, level 0 then 1
        ([[1, 3], [1, 1]], [inf, f32(2.0)], [np.inf, -np.inf]),  # code 3: -scale
        ([[1, 1], [3, 0]], [inf, inf], [np.nan, np.inf]),        # +Inf and -Inf
    ]
    for codes, scales, want in cases:
        words = [word(c) for c in codes]
        got = O.aggregate_quant(2, 2, words, scales, 1.0)
        for i in range(2):
            dec = [O.quant_decode((int(wd[0]) >> (2 * i)) & 3, 2, sc) for wd, sc in zip(words, scales)]
            assert same_f32(got[i], want[i]), (codes, scales, i, got[i])
            assert same_f32(got[i], xsum_f32(dec))


@pytest.mark.parametrize("kind", ["terngrad", "qsgd4", "qsgd8"])
def test_tensor_list_layout(kind):
    bits = O.QUANT_BITS[kind]
    rng = np.random.default_rng(7)
    ns = [0, 1, 15, 16, 17, 1000]
    grads = [(rng.standard_normal(n) * 0.01).astype(f32) for n in ns]
    resids = [np.zeros(n, f32) for n in ns]
    pay, new_e = O.compress_set(kind, 1.0, 55, grads, resids)
    for t, n in enumerate(ns):
        w, m, e_out = O.compress_quant(grads[t], resids[t], bits, 55, t)
        assert np.array_equal(pay["bits"][pay["off"][t]:pay["off"][t + 1]], w)
        assert pay["scale"][t] == m
        assert np.array_equal(new_e[t], e_out)
    outs = O.aggregate_set(kind, ns, [pay, pay], 0.5)
    for t, n in enumerate(ns):
        d = decode_np(unpack_codes(pay["bits"][pay["off"][t]:pay["off"][t + 1]], n, bits), bits, pay["scale"][t])
        assert np.array_equal(outs[t], (f32(0.5) * ((f32(0.0) + d).astype(f32) + d).astype(f32)).astype(f32))
