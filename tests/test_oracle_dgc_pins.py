"""Pins of the oracle's DGC momentum correction and masking (DGC is the
paper's sparsification operator, Sec. 5.1): the hand-worked example in
tests/golden/hand_examples.json, the reduction to the plain compressor at
zero momentum, the masking invariants, and the partition identity
decompress(payload) + e_new == u_new + e_old."""
import json
import os

import numpy as np
import pytest

import oracle as O

f32 = np.float32
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def F(xs):
    return np.array([float(x) for x in xs], dtype=np.float64).astype(f32)


def test_hand_example():
    ex = json.load(open(GOLDEN))["dgc"][0]
    idx, val, e_new, u_new = O.compress_dgc(ex["kind"], F(ex["g"]), F(ex["e"]), F(ex["u"]), ex["momentum"],
                                            ex["ratio"], 1, 0)
    assert list(idx) == ex["idx"]
    assert np.array_equal(val, F(ex["val"]))
    assert np.array_equal(e_new, F(ex["e_new"]))
    assert np.array_equal(u_new, F(ex["u_new"]))


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk"])
def test_zero_momentum_is_the_plain_compressor(kind):
    rng = np.random.default_rng(4)
    n = 5000
    g = (rng.standard_normal(n) * 0.01).astype(f32)
    g[g == 0] = f32(1e-3)  # no signed zeros: 0 * u + g keeps g's bits then
    e = (rng.standard_normal(n) * 0.001).astype(f32)
    u = (rng.standard_normal(n) * 0.01).astype(f32)
    idx, val, e_new, u_new = O.compress_dgc(kind, g, e, u, 0.0, 0.02, 9, 3)
    want = {"topk": lambda: O.compress_topk(g, e, 0.02),
            "topk_sampled": lambda: O.compress_topk_sampled(g, e, 0.02, 9, 3),
            "randk": lambda: O.compress_randk(g, e, 0.02, 9, 3)}[kind]()
    assert np.array_equal(idx, want[0])
    assert np.array_equal(val.view(np.uint32), want[1].view(np.uint32))
    assert np.array_equal(e_new.view(np.uint32), want[2].view(np.uint32))


@pytest.mark.parametrize("kind", ["topk", "topk_sampled", "randk"])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_masking_and_partition(kind, dtype):
    rng = np.random.default_rng(8)
    n = 7001
    g = (rng.standard_normal(n) * 0.01).astype(dtype)
    e = (rng.standard_normal(n) * 0.001).astype(f32)
    u = (rng.standard_normal(n) * 0.01).astype(f32)
    m = 0.9
    idx, val, e_new, u_new = O.compress_dgc(kind, g, e, u, m, 0.01, 5, 1)
    assert idx.size == O.k_for(n, 0.01)
    sel = idx.astype(np.int64)
    rest = np.setdiff1d(np.arange(n), sel)
    # the velocity step alone, then the residual accumulation
    un = O.dgc_momentum(g, u, m)
    assert np.all(u_new[sel] == 0.0) and np.all(~np.signbit(u_new[sel]))
    assert np.array_equal(u_new[rest].view(np.uint32), un[rest].view(np.uint32))
    v = (un + e).astype(f32)
    assert np.array_equal(val.view(np.uint32), v[sel].view(np.uint32))
    dec = np.zeros(n, f32)
    dec[sel] = val
    assert np.array_equal((dec + e_new).astype(f32).view(np.uint32)[rest], v.view(np.uint32)[rest])
    assert np.all(e_new[sel] == 0.0)
    # m u + g against exact rational arithmetic: fl32 of fl32(m u) + g
    from fractions import Fraction
    for i in range(0, n, 701):
        mu = f32(Fraction(float(f32(m))) * Fraction(float(u[i])))  # one rounding
        want = f32(float(Fraction(float(mu)) + Fraction(float(np.float32(g[i])))))
        assert un[i] == want


def test_tensor_list_keys_streams_by_position():
    rng = np.random.default_rng(12)
    ns = [300, 5000, 0, 9000]
    grads = [(rng.standard_normal(n) * 0.01).astype(f32) for n in ns]
    resids = [np.zeros(n, f32) for n in ns]
    vels = [(rng.standard_normal(n) * 0.01).astype(f32) for n in ns]
    pay, new_e, new_u = O.compress_dgc_set("randk", 0.05, 77, 0.9, grads, resids, vels)
    for t, n in enumerate(ns):
        i, v, e_out, u_out = O.compress_dgc("randk", grads[t], resids[t], vels[t], 0.9, 0.05, 77, t)
        assert np.array_equal(pay["idx"][pay["off"][t]:pay["off"][t + 1]], i)
        assert np.array_equal(new_u[t], u_out)


# ---------------------------------------------------- local gradient clipping

def test_clip_factor_closed_form():
    # 4096 entries of 0.5 (split over two tensors): ||g|| = sqrt(4096 / 4) = 32
    g = [np.full(1000, 0.5, f32), np.full(3096, 0.5, np.float16)]
    assert O.dgc_clip_factor(g, 8.0) == f32(0.25)
    assert O.dgc_clip_factor(g, 32.0) == f32(1.0)   # at the threshold: no clipping
    assert O.dgc_clip_factor(g, 100.0) == f32(1.0)
    assert O.dgc_clip_factor([np.zeros(10, f32)], 1.0) == f32(1.0)
    assert O.dgc_clip_factor([], 1.0) == f32(1.0)


def test_clip_factor_against_correctly_rounded_norm():
    import math
    rng = np.random.default_rng(41)
    g = [(rng.standard_normal(n) * 10.0 ** rng.uniform(-3, 1)).astype(dt)
         for n, dt in [(7, f32), (4097, np.float16), (100003, f32), (1, f32)]]
    exact = math.sqrt(math.fsum(float(x) * float(x) for a in g for x in a.astype(np.float64)))
    clip = exact / 3.0
    c = O.dgc_clip_factor(g, clip)
    want = f32(clip / exact)
    assert abs(float(c) - float(want)) <= float(np.spacing(want))  # one fp32 place at most
    # the norm covers the whole list, not each tensor
    assert O.dgc_clip_factor(g[:1], clip) == f32(1.0)


def test_clipped_momentum_step():
    rng = np.random.default_rng(42)
    n = 3000
    g = (rng.standard_normal(n) * 0.01).astype(f32)
    u = (rng.standard_normal(n) * 0.01).astype(f32)
    m = f32(0.9)
    # c = 1/2: the clipped gradient is exact, u = fl32(fl32(m u) + g/2)
    got = O.dgc_momentum_clipped(g, u, m, 0.5)
    want = (m * u) + (g * f32(0.5))
    assert np.array_equal(got.view(np.uint32), want.astype(f32).view(np.uint32))
    # c = 1 is the unclipped step, bit for bit
    assert np.array_equal(O.dgc_momentum_clipped(g, u, m, 1.0).view(np.uint32), O.dgc_momentum(g, u, m).view(np.uint32))
    # a general factor: each product and sum rounded once in fp32
    c = f32(0.3712)
    got = O.dgc_momentum_clipped(g, u, m, c)
    want = ((m * u).astype(f32) + (c * g).astype(f32)).astype(f32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_clipping_above_the_norm_changes_nothing(kind):
    rng = np.random.default_rng(43)
    grads = [(rng.standard_normal(n) * 0.01).astype(f32) for n in (5000, 300)]
    resids = [(rng.standard_normal(g.size) * 0.001).astype(f32) for g in grads]
    vels = [(rng.standard_normal(g.size) * 0.01).astype(f32) for g in grads]
    a = O.compress_dgc_set(kind, 0.05, 7, 0.9, grads, resids, vels)
    b = O.compress_dgc_set(kind, 0.05, 7, 0.9, grads, resids, vels, clip=1e6)
    for x, y in zip(a[0].values(), b[0].values()):
        assert np.array_equal(np.asarray(x), np.asarray(y))
    for x, y in zip(a[2], b[2]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
