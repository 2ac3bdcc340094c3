"""Pins of the CPU oracle against things other than itself.

Each test checks an oracle function against brute force, a closed form, a
hand-worked example (tests/golden/hand_examples.json), an invariant that the
definition implies, or an independent library routine (numpy.lexsort,
numpy.packbits, numpy float16 conversion, numpy.random.Philox).
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

from .exact_ref import exact_round_f32, same_f32, same_f32_arrays, xsum_f32

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
f32 = np.float32


def F(xs):
    return np.array([float(x) for x in xs], dtype=np.float64).astype(f32) if xs is not None else None


def bits(x):
    return np.asarray(x, f32).view(np.uint32)


def hexbits(xs):
    return np.array([int(h, 16) for h in xs], dtype=np.uint32)


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as fh:
        return json.load(fh)


# ------------------------------------------------------------------ sizes

def test_k_rule_stated_value():
    # the single-tensor workload states k = 1% of 2^20 = 10486
    assert O.k_for(1 << 20, 0.01) == 10486


@pytest.mark.parametrize("ratio", [0.01, 0.001, 0.25, 0.5, 0.999, 1.0, 0.123457])
def test_k_rule_is_exact_ceiling(ratio):
    ppm = round(ratio * 1e6)
    for n in list(range(0, 300)) + [767, 768, 1000, 4095, 4096, 65536, 1048577, 80411200, (1 << 32) - 1]:
        want = 0 if n == 0 else min(n, max(1, math.ceil(Fraction(n * ppm, 10**6))))
        assert O.k_for(n, ratio) == want, (n, ratio)


def test_word_count():
    for n in range(0, 200):
        assert O.words_for(n) == -(-n // 32)


# ------------------------------------------------------------- fp16 input

def test_f16_widening_matches_numpy_for_every_pattern():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    want = h.view(np.float16).astype(np.float32)
    got = np.array([O.f16_to_f32(int(x)) for x in h], dtype=np.float32)
    finite = np.isfinite(want)
    assert np.array_equal(bits(got[finite]), bits(want[finite]))
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(got[np.isinf(want)], want[np.isinf(want)])


# ------------------------------------------------------------------ top-k

def brute_topk(v, k):
    key = bits(v) & np.uint32(0x7FFFFFFF)
    order = np.lexsort((np.arange(v.size), -key.astype(np.int64)))
    return np.sort(order[:k]).astype(np.uint32)


def _inputs(rng, n, mode):
    if mode == "normal":
        g = (rng.standard_normal(n) * 0.01).astype(f32)
        e = (rng.standard_normal(n) * 0.001).astype(f32)
    elif mode == "ties":
        levels = np.array([-4, -3, -2, -1, -0.5, -0.25, 0, -0.0, 0.25, 0.5, 1, 2, 3, 4, 5, -5], f32)
        g = levels[rng.integers(0, 16, n)]
        e = np.zeros(n, f32)
    elif mode == "equal":
        g = np.full(n, 0.75, f32)
        e = np.zeros(n, f32)
    elif mode == "zeros":
        g = np.where(rng.random(n) < 0.5, f32(0.0), f32(-0.0)).astype(f32)
        e = np.where(rng.random(n) < 0.5, f32(0.0), f32(-0.0)).astype(f32)
    elif mode == "huge":
        g = (rng.standard_normal(n) * 1e-3).astype(f32)
        g[rng.integers(0, n)] = f32(3e38)
        e = np.zeros(n, f32)
    else:
        raise ValueError(mode)
    return g, e


@pytest.mark.parametrize("mode", ["normal", "ties", "equal", "zeros", "huge"])
@pytest.mark.parametrize("n", [1, 2, 7, 31, 32, 33, 64, 65, 257, 1000, 4096])
def test_topk_matches_lexsort_brute_force(mode, n):
    rng = np.random.default_rng(n * 7 + len(mode))
    g, e = _inputs(rng, n, mode)
    v = g + e
    for ratio in (0.01, 0.1, 0.37, 1.0):
        idx, val, e_out = O.compress_topk(g, e, ratio)
        k = O.k_for(n, ratio)
        want = brute_topk(v, k)
        assert np.array_equal(idx, want)
        assert np.array_equal(bits(val), bits(v[idx]))
        # reconstruction: decompress + residual == v, bit for bit
        rec = e_out.copy()
        rec[idx] = val
        assert np.array_equal(bits(rec), bits(v))
        assert np.all(bits(e_out[idx]) == 0)


def test_topk_tie_invariant_on_tie_heavy_input():
    rng = np.random.default_rng(5)
    g, e = _inputs(rng, 3000, "ties")
    v = g + e
    key = bits(v) & np.uint32(0x7FFFFFFF)
    for ratio in (0.05, 0.2, 0.5):
        idx, _, _ = O.compress_topk(g, e, ratio)
        sel = np.zeros(v.size, bool)
        sel[idx] = True
        tau = key[sel].min()
        assert key[~sel].max(initial=0) <= tau
        # among entries equal to the k-th key, the selected ones have the lowest indices
        eq = np.nonzero(key == tau)[0]
        chosen = eq[sel[eq]]
        rest = eq[~sel[eq]]
        if rest.size and chosen.size:
            assert chosen.max() < rest.min()
        assert np.all(np.diff(idx.astype(np.int64)) > 0)


def test_topk_hand_examples(golden):
    a, b, z = golden["topk"]
    idx, val, e_out = O.compress_topk(F(a["g"]), F(a["e"]), a["ratio"])
    assert idx.tolist() == a["idx"]
    assert np.array_equal(val, F(a["val"]))
    assert np.array_equal(e_out, F(a["e_new"]))
    g, e = F(b["g"]), F(b["e"])
    assert np.array_equal(bits(g + e), hexbits(b["v_bits"]))
    for case in b["cases"]:
        idx, val, _ = O.compress_topk(g, e, case["ratio"])
        assert idx.tolist() == case["idx"]
        if "val_bits" in case:
            assert np.array_equal(bits(val), hexbits(case["val_bits"]))
    idx, val, e_out = O.compress_topk(F(z["g"]), F(z["e"]), z["ratio"])
    assert idx.tolist() == z["idx"]
    assert np.array_equal(val, F(z["val"]))
    assert np.array_equal(bits(e_out), hexbits(z["e_new_bits"]))


def test_topk_without_residual_uses_gradient():
    rng = np.random.default_rng(3)
    g = (rng.standard_normal(500)).astype(f32)
    idx, val, e_out = O.compress_topk(g, None, 0.1)
    assert e_out is None
    assert np.array_equal(idx, brute_topk(g, 50))


def test_topk_fp16_gradient():
    rng = np.random.default_rng(4)
    g = (rng.standard_normal(999) * 1e-3).astype(np.float16)
    e = (rng.standard_normal(999) * 1e-4).astype(f32)
    v = g.astype(f32) + e
    idx, val, _ = O.compress_topk(g, e, 0.05)
    assert np.array_equal(idx, brute_topk(v, O.k_for(999, 0.05)))


# -------------------------------------------------------- sampled top-k

def test_sampled_topk_equals_exact_topk_and_exercises_both_paths():
    rng = np.random.default_rng(11)
    saw_trim = saw_topup = False
    for trial in range(60):
        n = int(rng.integers(1, 3000))
        mode = ["normal", "ties", "equal", "zeros"][trial % 4]
        g, e = _inputs(rng, n, mode)
        for ratio in (0.01, 0.3, 0.6):
            k = O.k_for(n, ratio)
            idx, val, e_out, nc = O.compress_topk_sampled(g, e, ratio, 14465 + trial, trial,
                                                          want_candidates=True)
            i2, v2, e2 = O.compress_topk(g, e, ratio)
            assert np.array_equal(idx, i2)
            assert np.array_equal(bits(val), bits(v2))
            assert np.array_equal(bits(e_out), bits(e2))
            saw_trim |= nc >= k
            saw_topup |= nc < k
    assert saw_trim and saw_topup


# ------------------------------------------------------------- Philox

def test_philox_matches_numpy_philox4x64():
    rng = np.random.default_rng(21)
    m = np.uint64(2**64 - 1)
    for _ in range(40):
        ctr = rng.integers(0, 2**63, size=4, dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, size=4, dtype=np.uint64)
        key = rng.integers(0, 2**63, size=2, dtype=np.uint64)
        # numpy increments the 256-bit counter before producing a block
        prev = ctr.copy()
        i = 0
        while True:
            if prev[i] == 0:
                prev[i] = m
                i += 1
                if i == 4:
                    break
            else:
                prev[i] -= np.uint64(1)
                break
        # pass uint64 arrays: numpy converts Python-int lists through float
        bg = np.random.Philox(counter=prev.astype(np.uint64), key=key.astype(np.uint64))
        want = bg.random_raw(4).astype(np.uint64)
        got = O.philox4x64_10(ctr, key)
        assert np.array_equal(got, want)


def test_philox_published_zero_vector_via_numpy():
    m = 2**64 - 1
    bg = np.random.Philox(counter=[m, m, m, m], key=[0, 0])
    assert np.array_equal(O.philox4x64_10([0, 0, 0, 0], [0, 0]), bg.random_raw(4).astype(np.uint64))


# ------------------------------------------------------------- random-k

@pytest.mark.parametrize("h", [1, 2, 3, 5, 8])
def test_feistel_is_a_bijection(h):
    rk = O.randk_round_keys(987654321, 17)
    dom = 1 << (2 * h)
    img = [O.feistel_encrypt(x, h, rk) for x in range(dom)]
    assert sorted(img) == list(range(dom))


def test_feistel_domain_bits():
    for n, h in [(1, 1), (2, 1), (4, 1), (5, 2), (16, 2), (17, 3), (64, 3), (65, 4),
                 (1 << 20, 10), ((1 << 20) + 1, 11), (80411200, 14)]:
        assert O.feistel_half_bits(n) == h, n


@pytest.mark.parametrize("n", [1, 2, 3, 5, 17, 100, 777, 1024])
def test_cycle_walk_is_a_permutation_of_the_tensor(n):
    img = [O.randk_index(n, 42, 3, j) for j in range(n)]
    assert sorted(img) == list(range(n))


def test_randk_payload_properties():
    rng = np.random.default_rng(8)
    for n in (1, 10, 99, 1000, 12345):
        g = rng.standard_normal(n).astype(f32)
        e = rng.standard_normal(n).astype(f32) * f32(0.1)
        v = g + e
        for ratio in (0.01, 0.2, 1.0):
            k = O.k_for(n, ratio)
            idx, val, e_out = O.compress_randk(g, e, ratio, 14465, 7)
            assert idx.size == k and np.all(np.diff(idx.astype(np.int64)) > 0)
            assert idx.max(initial=0) < n
            assert np.array_equal(bits(val), bits(v[idx]))
            rec = e_out.copy()
            rec[idx] = val
            assert np.array_equal(bits(rec), bits(v))
            want = np.sort([O.randk_index(n, 14465, 7, j) for j in range(k)]).astype(np.uint32)
            assert np.array_equal(idx, want)
            if ratio == 1.0:
                assert np.array_equal(idx, np.arange(n, dtype=np.uint32))


def test_randk_depends_on_seed_and_tensor_id():
    g = np.ones(5000, f32)
    a, _, _ = O.compress_randk(g, None, 0.01, 1, 0)
    b, _, _ = O.compress_randk(g, None, 0.01, 2, 0)
    c, _, _ = O.compress_randk(g, None, 0.01, 1, 1)
    d, _, _ = O.compress_randk(g, None, 0.01, 1, 0)
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
    assert np.array_equal(a, d)


def test_randk_inclusion_frequency_is_uniform():
    # chi-square over 2000 seeds: every coordinate of a 1000-element tensor is
    # included with probability k/n = 1/100
    n, k, seeds = 1000, 10, 2000
    counts = np.zeros(n)
    g = np.ones(n, f32)
    for s in range(seeds):
        idx, _, _ = O.compress_randk(g, None, 0.01, 1_000_003 * s + 17, 5)
        counts[idx] += 1
    expected = seeds * k / n
    chi2 = float(((counts - expected) ** 2 / expected).sum())
    # 999 degrees of freedom: mean 999, sd ~ 44.7; 5-sigma band
    assert 999 - 5 * 44.7 < chi2 < 999 + 5 * 44.7, chi2
    # pairs: the permutation is not a fixed stride (consecutive picks differ)
    idx, _, _ = O.compress_randk(np.ones(10**6, f32), None, 0.01, 99, 0)
    gaps = np.diff(idx.astype(np.int64))
    assert gaps.std() > 0.5 * gaps.mean()


# ------------------------------------------------------------------- sign

def test_sign_hand_examples(golden):
    c, c1, c2, c3 = golden["sign"]
    w, s, e_out = O.compress_sign(F(c["g"]), F(c["e"]))
    assert np.array_equal(w, hexbits(c["words"]))
    assert s == f32(c["scale"])
    assert np.array_equal(e_out, F(c["e_new"]))
    w, s, e_out = O.compress_sign(F(c1["g"]), F(c1["e"]))
    assert np.array_equal(w, hexbits(c1["words"]))
    assert bits(s) == int(c1["scale_bits"], 16)
    assert bits(e_out[0]) == int(c1["e_new0_bits"], 16)
    w, s, e_out = O.compress_sign(F(c2["g"]), F(c2["e"]))
    assert np.array_equal(w, hexbits(c2["words"]))
    assert s == f32(c2["scale"])
    assert bits(e_out[0]) == int(c2["e_new0_bits"], 16)
    x = np.array([(-1) ** i * (i + 1) / 64 for i in range(40)], f32)
    w, s, _ = O.compress_sign(x, None)
    assert np.array_equal(w, hexbits(c3["words"]))
    assert s == f32(c3["scale"])


@pytest.mark.parametrize("n", [0, 1, 31, 32, 33, 63, 64, 65, 1000, 4097])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_sign_against_packbits_and_closed_forms(n, dtype):
    rng = np.random.default_rng(n + 3)
    g = (rng.standard_normal(n) * 1e-3).astype(dtype)
    if n > 4:
        g[:4] = np.array([0.0, -0.0, 0.0, -0.0], dtype)
    e = (rng.standard_normal(n) * 1e-4).astype(f32)
    if n > 4:
        e[:4] = np.array([0.0, -0.0, -0.0, 0.0], f32)
    v = g.astype(f32) + e
    w, s, e_out = O.compress_sign(g, e)
    sb = (bits(v) >> 31).astype(np.uint8)
    packed = np.packbits(np.concatenate([sb, np.zeros((-n) % 32, np.uint8)]), bitorder="little")
    assert np.array_equal(w, packed.view("<u4"))
    assert sum(bin(int(x)).count("1") for x in w) == int(sb.sum())
    if n == 0:
        assert bits(s) == 0
        return
    # the scale is the fp64 mean of |v|: compare with the exact mean
    exact = Fraction(0)
    for x in np.abs(v.astype(np.float64)):
        exact += Fraction(float(x))
    mean = exact / n
    assert abs(Fraction(float(s)) - mean) <= Fraction(float(np.spacing(f32(s))))
    # decoded magnitudes sum to n*s exactly
    dec = np.where(sb == 1, -s, s).astype(f32)
    assert math.fsum(np.abs(dec.astype(np.float64))) == n * float(s)
    # residual is the correctly rounded difference v - decoded
    for i in range(min(n, 300)):
        exact_r = Fraction(float(v[i])) - Fraction(float(dec[i]))
        r = Fraction(float(e_out[i]))
        half_ulp = Fraction(float(np.spacing(np.abs(e_out[i])))) / 2
        assert abs(r - exact_r) <= half_ulp


# -------------------------------------------------------- residual update

@pytest.mark.parametrize("kind", ["topk", "randk", "sign"])
def test_fused_equals_split_residual_update(kind):
    rng = np.random.default_rng(12)
    n = 3001
    g = (rng.standard_normal(n) * 0.02).astype(f32)
    e = (rng.standard_normal(n) * 0.002).astype(f32)
    v = g + e
    if kind == "sign":
        w, s, e_fused = O.compress_sign(g, e)
        w2, s2, _ = O.compress_sign(v, None)
        assert np.array_equal(w, w2) and s == s2
        e_split = O.residual_update_sign(g, e, w2, s2)
    else:
        comp = O.compress_topk if kind == "topk" else (lambda a, b, r: O.compress_randk(a, b, r, 5, 1))
        idx, val, e_fused = comp(g, e, 0.01)
        idx2, val2, _ = comp(v, None, 0.01)
        assert np.array_equal(idx, idx2) and np.array_equal(val, val2)
        e_split = O.residual_update_sparse(g, e, idx2, val2)
    assert np.array_equal(bits(e_fused), bits(e_split))


# -------------------------------------------------------------- aggregates

def test_sparse_aggregate_hand_example(golden):
    d = golden["aggregate_sparse"][0]
    out = O.aggregate_sparse(d["n"], [np.array(w["idx"]) for w in d["workers"]],
                             [F(w["val"]) for w in d["workers"]], float(d["alpha"]))
    assert np.array_equal(out, F(d["out"]))


def test_sign_aggregate_hand_example(golden):
    # the two workers' values are exact binary fractions: both forms agree
    d = golden["aggregate_sign"][0]
    for ordered in (False, True):
        out = O.aggregate_sign(d["n"], [hexbits(w["words"]) for w in d["workers"]],
                               [f32(w["scale"]) for w in d["workers"]], float(d["alpha"]), ordered=ordered)
        assert np.array_equal(out, F(d["out"]))


def test_sparse_aggregate_single_worker_is_decompress():
    rng = np.random.default_rng(2)
    n = 1000
    idx = np.sort(rng.choice(n, 77, replace=False)).astype(np.uint32)
    val = rng.standard_normal(77).astype(f32)
    out = O.aggregate_sparse(n, [idx], [val], 1.0)
    dense = np.zeros(n, f32)
    dense[idx] = val
    assert np.array_equal(bits(out), bits(dense))


def test_sparse_aggregate_disjoint_supports_is_exact_sum():
    rng = np.random.default_rng(3)
    n, W = 4096, 8
    perm = rng.permutation(n)
    parts = np.array_split(perm[:W * 100], W)
    idx = [np.sort(p).astype(np.uint32) for p in parts]
    val = [rng.standard_normal(p.size).astype(f32) for p in parts]
    out = O.aggregate_sparse(n, idx, val, 0.125)
    dense = np.zeros(n, np.float64)
    for i, v in zip(idx, val):
        dense[i] += v
    assert np.array_equal(out, (dense * 0.125).astype(f32))


def test_sparse_aggregate_brute_force_order():
    # worker-ascending fp32 accumulation, checked element by element with
    # Python floats rounded through numpy float32 at every step
    rng = np.random.default_rng(4)
    n, W = 64, 6
    idx = [np.sort(rng.choice(n, 20, replace=False)).astype(np.uint32) for _ in range(W)]
    val = [(rng.standard_normal(20) * 10.0 ** rng.integers(-3, 3)).astype(f32) for _ in range(W)]
    out = O.aggregate_sparse(n, idx, val, 0.5)
    for i in range(n):
        acc = f32(0.0)
        for w in range(W):
            hit = np.nonzero(idx[w] == i)[0]
            if hit.size:
                acc = f32(acc + val[w][hit[0]])
        assert bits(out[i]) == bits(f32(f32(0.5) * acc))


def exact_round(values):
    """Exact rational sum of float32 values rounded once to float32."""
    return exact_round_f32(values)


@pytest.mark.parametrize("seed", range(6))
def test_exact_sum_matches_rational_arithmetic(seed):
    rng = np.random.default_rng(seed)
    for trial in range(300):
        m = int(rng.integers(1, 70))
        kind = trial % 5
        if kind == 0:      # wide exponent range, subnormals included
            x = (rng.standard_normal(m) * 10.0 ** rng.integers(-44, 38, m)).astype(f32)
        elif kind == 1:    # cancellation: pairs x, -x plus a tiny remainder
            h = (rng.standard_normal(m) * 1e3).astype(f32)
            x = np.concatenate([h, -h, (rng.standard_normal(2) * 1e-30).astype(f32)])
        elif kind == 2:    # ties at the rounding point: 1 + 2^-24 patterns
            x = np.array([1.0, 2.0 ** -24] + [2.0 ** -60] * int(rng.integers(0, 3)), f32)
        elif kind == 3:    # similar magnitudes (the sign aggregate's case)
            x = (np.where(rng.random(m) < 0.5, -1, 1) * 1e-3 * (1 + 0.05 * rng.standard_normal(m))).astype(f32)
        else:              # subnormal-only
            x = (rng.integers(-(1 << 23), 1 << 23, m) * 2.0 ** -149).astype(f32)
        got = O.exact_sum_f32(x)
        want = exact_round(x)
        assert bits(got) == bits(want), (trial, x.tolist())


def test_sign_aggregate_exact_form_per_element():
    rng = np.random.default_rng(77)
    n, W = 90, 7
    words = [rng.integers(0, 1 << 32, 3, dtype=np.uint64).astype(np.uint32) for _ in range(W)]
    scales = (np.abs(rng.standard_normal(W)) * 1e-3).astype(f32)
    out = O.aggregate_sign(n, words, scales, 0.25)
    for i in range(n):
        d = [(-scales[w] if (words[w][i // 32] >> (i % 32)) & 1 else scales[w]) for w in range(W)]
        assert bits(out[i]) == bits(f32(f32(0.25) * exact_round(d))), i


def test_sign_aggregate_exact_is_within_recursive_sum_bound_of_ordered():
    # |exact_rounded - ordered| <= (W-1) u sum|d| + u |sum|  (Higham, recursive summation)
    rng = np.random.default_rng(78)
    n, W = 4000, 64
    words = [rng.integers(0, 1 << 32, 125, dtype=np.uint64).astype(np.uint32) for _ in range(W)]
    scales = (1e-3 * (1 + 0.05 * rng.standard_normal(W))).astype(f32)
    a = O.aggregate_sign(n, words, scales, 1.0)
    b = O.aggregate_sign(n, words, scales, 1.0, ordered=True)
    u = 2.0 ** -24
    bound = (W - 1) * u * float(np.sum(scales, dtype=np.float64)) + u * np.abs(a.astype(np.float64))
    assert np.all(np.abs(a.astype(np.float64) - b.astype(np.float64)) <= bound + 1e-45)
    assert np.any(a != b)  # the two forms are genuinely different readings


def _decoded_sign(words, scales, i):
    return [(-scales[w] if (words[w][i // 32] >> (i % 32)) & 1 else scales[w]) for w in range(len(scales))]


@pytest.mark.parametrize("W", [2, 5, 16, 64])
@pytest.mark.parametrize("span", [30, 45, 60, 120, 253])
def test_sign_aggregate_is_exact_at_any_scale_span(W, span):
    # scales whose binary exponents spread over `span` binades: the output
    # is still the exact rational sum rounded once (no span-dependent form)
    rng = np.random.default_rng(1000 * W + span)
    n = 96
    words = [rng.integers(0, 1 << 32, 3, dtype=np.uint64).astype(np.uint32) for _ in range(W)]
    ex = rng.integers(-126, -126 + span + 1, W)
    ex[0], ex[-1] = -126, -126 + span
    scales = (np.ldexp(1.0 + rng.random(W), ex)).astype(f32)
    scales[rng.random(W) < 0.3] *= f32(-1.0)     # negative scales are summed as given
    out = O.aggregate_sign(n, words, scales, 0.5)
    for i in range(n):
        want = f32(f32(0.5) * exact_round(_decoded_sign(words, scales, i)))
        assert same_f32(out[i], want), (i, out[i], want)


def test_sign_aggregate_small_terms_decide_the_rounding():
    # two large scales cancel or tie at a rounding point; a scale 40 and 60
    # binades below breaks the tie, which any truncated sum would lose
    big, half_ulp = f32(1.0), f32(2.0 ** -24)
    for tiny, wbits, want in [
        (f32(2.0 ** -64), [0, 0, 0], f32(1.0 + 2.0 ** -23)),   # 1 + half ulp + tiny: up
        (f32(2.0 ** -64), [0, 0, 1], f32(1.0)),                # 1 + half ulp - tiny: down
        (f32(2.0 ** -84), [1, 0, 0], f32(-1.0 + 2.0 ** -24)),  # tiny term below the last place
    ]:
        words = [np.array([b], np.uint32) for b in wbits]
        out = O.aggregate_sign(1, words, [big, half_ulp, tiny], 1.0)
        assert same_f32(out[0], want), (tiny, wbits, out[0], want)
        assert same_f32(out[0], exact_round(_decoded_sign(words, [big, half_ulp, tiny], 0)))


def test_sign_aggregate_subnormal_scales_and_results():
    # subnormal scales are summed exactly; a subnormal result is exact
    s = np.array([2.0 ** -149, 3 * 2.0 ** -149, 2.0 ** -130, 2.0 ** -127], f32)
    rng = np.random.default_rng(5)
    words = [rng.integers(0, 1 << 32, 2, dtype=np.uint64).astype(np.uint32) for _ in range(4)]
    out = O.aggregate_sign(64, words, s, 1.0)
    for i in range(64):
        assert same_f32(out[i], exact_round(_decoded_sign(words, s, i))), i


def test_sign_aggregate_overflow_rounds_to_infinity():
    fmax = np.finfo(np.float32).max
    ones, zeros = np.array([0xFFFFFFFF], np.uint32), np.zeros(1, np.uint32)
    # FLT_MAX + half an ulp is a tie with an odd last bit: rounds up to +Inf
    out = O.aggregate_sign(1, [zeros, zeros], [fmax, f32(2.0 ** 103)], 1.0)
    assert out[0] == np.inf
    out = O.aggregate_sign(1, [zeros, zeros], [fmax, f32(2.0 ** 102)], 1.0)
    assert out[0] == fmax
    out = O.aggregate_sign(1, [ones, ones], [fmax, f32(2.0 ** 103)], 1.0)
    assert out[0] == -np.inf
    # large terms cancel exactly and leave a finite sum
    out = O.aggregate_sign(1, [zeros, zeros, ones], [fmax, fmax, fmax], 1.0)
    assert out[0] == fmax


def test_sign_aggregate_non_finite_rule():
    z, o = np.zeros(1, np.uint32), np.ones(1, np.uint32)
    inf, nan = f32(np.inf), f32(np.nan)
    cases = [
        ([z, z], [inf, f32(1.0)], np.inf),          # +Inf with a finite value
        ([o, z], [inf, f32(1.0)], -np.inf),         # the bit flips the infinity
        ([z, o], [inf, inf], np.nan),               # +Inf and -Inf
        ([z, z], [f32(-np.inf), f32(-1.0)], -np.inf),
        ([z, z], [nan, f32(1.0)], np.nan),          # NaN wins over everything
        ([z, z, o], [nan, inf, inf], np.nan),
    ]
    for words, scales, want in cases:
        out = O.aggregate_sign(1, words, scales, 1.0)
        assert same_f32(out[0], want), (scales, out[0])
        assert same_f32(out[0], xsum_f32(_decoded_sign(words, scales, 0)))


def test_sign_aggregate_is_independent_of_worker_order():
    # a definition with no addition order: permuting the workers changes
    # nothing, at any span, with cancellations and non-finite scales
    rng = np.random.default_rng(9)
    n, W = 200, 24
    words = [rng.integers(0, 1 << 32, 7, dtype=np.uint64).astype(np.uint32) for _ in range(W)]
    scales = np.ldexp(1.0 + rng.random(W), rng.integers(-120, 120, W)).astype(f32)
    scales[3] = scales[7]
    for variant in range(3):
        sc = scales.copy()
        if variant == 1:
            sc[5] = np.inf
        if variant == 2:
            sc[5], sc[6] = np.inf, np.nan
        ref = O.aggregate_sign(n, words, sc, 1.0)
        for _ in range(4):
            perm = rng.permutation(W)
            got = O.aggregate_sign(n, [words[p] for p in perm], sc[perm], 1.0)
            assert same_f32_arrays(got, ref)
        for i in range(0, n, 17):
            assert same_f32(ref[i], xsum_f32(_decoded_sign(words, sc, i)))


def test_sign_aggregate_zero_bits_and_single_worker():
    n, W = 100, 5
    words = [np.zeros(4, np.uint32) for _ in range(W)]
    scales = [f32(0.1 * (w + 1)) for w in range(W)]
    out = O.aggregate_sign(n, words, scales, 1.0)
    assert np.all(out == exact_round(scales))
    rng = np.random.default_rng(6)
    g = rng.standard_normal(n).astype(f32)
    w, s, _ = O.compress_sign(g, None)
    out = O.aggregate_sign(n, [w], [s], 1.0)
    assert np.array_equal(out, np.where(g < 0, -s, s).astype(f32))


# ------------------------------------------------------ divisible scheme

def _div_bounds(rng, ns, P):
    out = []
    for n in ns:
        inner = sorted(int(x) * 32 for x in rng.integers(0, n // 32 + 1, size=P - 1))
        out.append([0] + inner + [n])
    return out


WORD_KINDS = ("sign", "terngrad", "qsgd4", "qsgd8")


@pytest.mark.parametrize("kind", ["topk", "randk", "sign", "terngrad", "qsgd4", "qsgd8"])
def test_parts_reassemble_the_payload(kind):
    """Packing every part and undoing the rebase gives back the payload
    exactly: the parts are disjoint and cover every entry (word)."""
    rng = np.random.default_rng(31)
    ns = [1, 31, 32, 100, 4097, 70000]
    grads = [rng.standard_normal(n).astype(np.float32) for n in ns]
    pay, _ = O.compress_set(kind, 0.05, 3, grads, None)
    P = 4
    bounds = _div_bounds(rng, ns, P)
    parts = [O.pack_part_set(kind, ns, pay, bounds, j) for j in range(P)]
    for t, n in enumerate(ns):
        seg = slice(pay["off"][t], pay["off"][t + 1])
        if kind in WORD_KINDS:
            got = np.concatenate([p["bits"][p["off"][t]:p["off"][t + 1]] for p in parts])
            assert np.array_equal(got, pay["bits"][seg])
            for p in parts:
                assert np.array_equal(p["scale"], pay["scale"])
        else:
            ii = np.concatenate([p["idx"][p["off"][t]:p["off"][t + 1]] + np.uint32(bounds[t][j])
                                 for j, p in enumerate(parts)])
            vv = np.concatenate([p["val"][p["off"][t]:p["off"][t + 1]] for p in parts])
            assert np.array_equal(ii, pay["idx"][seg])
            assert np.array_equal(vv.view(np.uint32), pay["val"][seg].view(np.uint32))


@pytest.mark.parametrize("kind", ["topk", "sign", "terngrad", "qsgd4", "qsgd8"])
def test_part_aggregates_assemble_the_whole_aggregate(kind):
    """The node-j aggregates of all parts, placed at their ranges, equal the
    indivisible aggregate bit for bit (each element's sum sees the same
    workers in the same order)."""
    rng = np.random.default_rng(32)
    ns = [33, 4096, 20001]
    W, P = 5, 3
    pays = []
    for w in range(W):
        grads = [rng.standard_normal(n).astype(np.float32) for n in ns]
        pays.append(O.compress_set(kind, 0.1, 7 + w, grads, None)[0])
    bounds = _div_bounds(rng, ns, P)
    whole = O.aggregate_set(kind, ns, pays, 0.5)
    for j in range(P):
        lens = [bounds[t][j + 1] - bounds[t][j] for t in range(len(ns))]
        parts = [O.pack_part_set(kind, ns, p, bounds, j) for p in pays]
        got = O.aggregate_part_set(kind, lens, parts, 0.5)
        for t in range(len(ns)):
            lo, hi = bounds[t][j], bounds[t][j + 1]
            assert np.array_equal(got[t].view(np.uint32), whole[t][lo:hi].view(np.uint32)), (j, t)


def test_part_bounds_rules():
    with pytest.raises(AssertionError):
        O.check_part_bounds(100, [0, 50, 100])   # inner bound not word aligned
    with pytest.raises(AssertionError):
        O.check_part_bounds(100, [0, 64, 32, 100])
    with pytest.raises(AssertionError):
        O.check_part_bounds(100, [0, 96])
    assert O.check_part_bounds(100, [0, 0, 96, 100]) == [0, 0, 96, 100]
