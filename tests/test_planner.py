"""The decision algorithm (paper Sec. 4.4: Algorithm 1, GPU compression;
Algorithm 2, CPU offloading) on synthetic timelines: hand-worked timelines
with fixed step times, the bubble rule, and the searches against brute
force on small instances."""
import itertools
import math
import os
import random

import pytest

from paper_2205_14465_amd import planner as P

TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles",
                     "compression_time_model.txt")


class FixedModel(P.CostModel):
    """Step times given by hand: allreduce `ar`, and for a compressed
    tensor compress `cp`, allgather `ag`, aggregate `agg` on its device."""

    def __init__(self, ar, cp=5.0, ag=8.0, agg=4.0):
        self.ar, self.cp, self.ag, self.agg = ar, cp, ag, agg

    def stages(self, t, opt):
        if opt is None:
            return [("net", self.ar, "allreduce")]
        dev, _ = opt
        return [(dev, self.cp, "compress"), ("net", self.ag, "allgather"), (dev, self.agg, "aggregate")]


def test_timeline_without_compression():
    # compute 10 + 10 on the GPU; allreduces of 30 one after the other
    tl = P.simulate([P.Tensor(100, 10.0), P.Tensor(100, 10.0)], [None, None], FixedModel(30.0))
    assert tl.net == [(10.0, 40.0, 0), (40.0, 70.0, 1)]
    assert tl.iteration_us == 70.0
    assert P.bubble_cut(tl) == -math.inf


def test_gpu_compression_delays_the_next_computation():
    # tensor 0 compressed on the GPU: compress [10, 15] runs before tensor
    # 1's computation [15, 25] (same release time, lower index first);
    # allgather [15, 23]; aggregate waits for the GPU: [25, 29]; tensor 1's
    # allreduce [25, 55]
    tl = P.simulate([P.Tensor(100, 10.0), P.Tensor(100, 10.0)], [("gpu", "indivisible"), None], FixedModel(30.0))
    assert tl.net == [(15.0, 23.0, 0), (25.0, 55.0, 1)]
    assert tl.done_us == [29.0, 55.0]
    assert tl.iteration_us == 55.0


def test_cpu_compression_leaves_the_gpu_free():
    # offloaded: tensor 1 computes [10, 20] while tensor 0 compresses on the CPU
    tl = P.simulate([P.Tensor(100, 10.0), P.Tensor(100, 10.0)], [("cpu", "indivisible"), None], FixedModel(30.0))
    assert tl.net == [(15.0, 23.0, 0), (23.0, 53.0, 1)]
    assert tl.done_us == [27.0, 53.0]


def test_bubble_rule_keeps_earlier_tensors_uncompressed():
    # tensor 1 computes until 60: a bubble [40, 60] follows tensor 0's
    # allreduce, so compressing tensor 0 cannot help and it is dropped
    tensors = [P.Tensor(100, 10.0), P.Tensor(100, 50.0)]
    m = FixedModel(30.0, cp=1.0, ag=2.0, agg=1.0)
    tl = P.simulate(tensors, [None, None], m)
    assert P.bubble_cut(tl) == 40.0
    S = P.plan_gpu(tensors, m)
    assert S[0] is None
    assert S[1] is not None  # 1 + 2 + 1 beats a 30 us allreduce after the computation
    assert P.simulate(tensors, S, m).iteration_us == 64.0


def _instances(count, seed=0):
    rows = P.load_profile_rows(TABLE)
    pcie = P.load_profile_pcie(TABLE)
    for trial in range(count):
        rnd = random.Random(seed + trial)
        T = rnd.randint(3, 6)
        tensors = [P.Tensor(rnd.choice([1 << 16, 1 << 20, 1 << 22]), rnd.uniform(50, 2000)) for _ in range(T)]
        cl = P.Cluster(N=rnd.choice([4, 8, 16]), link_gbs=rnd.choice([3.0, 12.5]))
        # the measured CPU times, and hosts 4x faster or slower than the one profiled
        f = rnd.choice([0.25, 1.0, 4.0])
        scaled = [dict(r, compress_us=r["compress_us"] * f, aggregate_us=r["aggregate_us"] * f)
                  if r["device"] == "cpu" else r for r in rows]
        yield tensors, P.CostModel(rnd.choice(["sign", "topk", "randk"]), 0.01, scaled, cl, pcie=pcie)


def test_profile_table_loads():
    rows = P.load_profile_rows(TABLE)
    for dev in ("gpu", "cpu"):
        kinds = {r["kind"] for r in rows if r["device"] == dev}
        assert {"topk", "topk_sampled", "randk", "sign"} <= kinds, dev
    assert all(r["compress_us"] > 0 and r["aggregate_us"] > 0 and r["runs"] >= 3 for r in rows)
    pcie = P.load_profile_pcie(TABLE)
    assert pcie and pcie["h2d"] > 1.0 and pcie["d2h"] > 1.0
    m = P.CostModel("topk", 0.01, rows, P.Cluster(), pcie=pcie)
    assert m.has_cpu
    # the CPU curve is the measured one: at a profiled size it returns the row
    r = next(r for r in rows if r["device"] == "cpu" and r["kind"] == "topk" and r["n"] == 1 << 20)
    assert m.compress("cpu", 1 << 20) == pytest.approx(r["compress_us"])
    assert m.aggregate("cpu", 1 << 20, 8) == pytest.approx(r["aggregate_us"])


def test_no_cpu_option_without_measured_cpu_times():
    rows = [r for r in P.load_profile_rows(TABLE) if r["device"] == "gpu"]
    m = P.CostModel("sign", 0.01, rows, P.Cluster(), pcie=P.load_profile_pcie(TABLE))
    assert not m.has_cpu
    tensors = [P.Tensor(1 << 20, 500.0) for _ in range(4)]
    S1 = P.plan_gpu(tensors, m)
    S2, evals = P.plan_cpu(tensors, S1, m)
    assert S2 == S1 and evals == 0


def test_algorithm1_never_worse_than_no_compression():
    for tensors, m in _instances(40):
        S = P.plan_gpu(tensors, m)
        assert P.simulate(tensors, S, m).iteration_us <= P.simulate(tensors, [None] * len(tensors), m).iteration_us
        assert all(o is None or o[0] == "gpu" for o in S)


def _group_offload(S1, groups, U, farthest):
    S = list(S1)
    for g, u in zip(groups.values(), U):
        for i in sorted(g, reverse=farthest)[:u]:
            S[i] = ("cpu", S[i][1])
    return S


@pytest.mark.parametrize("order", ["earliest", "farthest"])
def test_algorithm2_is_the_best_lemma_restricted_offloading(order):
    # Algorithm 2 against brute force over its own search space: in each
    # (size, option) group, offload the first u tensors in the lemma's order
    for tensors, m in _instances(25, seed=100):
        S1 = P.plan_gpu(tensors, m)
        S2, evals = P.plan_cpu(tensors, S1, m, lemma_order=order)
        groups = {}
        for i, o in enumerate(S1):
            if o:
                groups.setdefault((tensors[i].n, o), []).append(i)
        best = math.inf
        for U in itertools.product(*[range(len(g) + 1) for g in groups.values()]):
            best = min(best, P.simulate(tensors, _group_offload(S1, groups, U, order == "farthest"), m).iteration_us)
        f2 = P.simulate(tensors, S2, m).iteration_us
        assert f2 == pytest.approx(best, abs=1e-9)
        assert f2 <= P.simulate(tensors, S1, m).iteration_us


def _best_subset(tensors, S1, m):
    comp = [i for i, o in enumerate(S1) if o]
    best = math.inf
    for mask in range(1 << len(comp)):
        S = list(S1)
        for b, i in enumerate(comp):
            if mask >> b & 1:
                S[i] = ("cpu", S[i][1])
        best = min(best, P.simulate(tensors, S, m).iteration_us)
    return best


def test_algorithm2_against_every_offloading_subset():
    # the lemma restricts each group to offloading its first u tensors; in
    # this timeline model, with the measured GPU and CPU times, the
    # earliest-ready-first order reaches the best of all 2^|T_gpu| subsets
    # on every random instance
    for tensors, m in _instances(60, seed=200):
        S1 = P.plan_gpu(tensors, m)
        S2, _ = P.plan_cpu(tensors, S1, m)
        assert P.simulate(tensors, S2, m).iteration_us <= _best_subset(tensors, S1, m) + 1e-9


def test_lemma_statement_order_is_not_always_best_here():
    # the statement's order (farthest from the output layer first) misses
    # the best subset on some instances of this model (the reading the
    # default order takes); it is never worse than GPU-only compression
    miss = 0
    for tensors, m in _instances(60, seed=200):
        S1 = P.plan_gpu(tensors, m)
        S2, _ = P.plan_cpu(tensors, S1, m, lemma_order="farthest")
        f2 = P.simulate(tensors, S2, m).iteration_us
        assert f2 <= P.simulate(tensors, S1, m).iteration_us
        miss += f2 > _best_subset(tensors, S1, m) + 1e-9
    assert miss > 0


def test_cli_runs_on_the_committed_table(capsys):
    P.main(["--model", "resnet50", "--kind", "sign", "--N", "8", "--json"])
    import json
    res = json.loads(capsys.readouterr().out)
    assert res["algorithm1_2_us"] <= res["algorithm1_us"] <= res["fp32_us"]
    assert res["tensors"] == 161


def test_native_timeline_model_matches_simulate():
    """The library's timeline model (bytecomp_plan_simulate) and simulate()
    give the same iteration time, bit for bit, on random instances and
    strategies of every option."""
    opts = [None, ("gpu", "indivisible"), ("gpu", "divisible"), ("cpu", "indivisible"), ("cpu", "divisible")]
    for k, (tensors, m) in enumerate(_instances(40, seed=300)):
        table = P.NativeTable(tensors, m)
        rnd = random.Random(k)
        for _ in range(10):
            S = [rnd.choice(opts) for _ in tensors]
            assert table.simulate(S) == P.simulate(tensors, S, m).iteration_us, (k, S)


def test_native_enumeration_matches_the_python_loop():
    for tensors, m in _instances(25, seed=400):
        S1 = P.plan_gpu(tensors, m)
        assert S1 == P.plan_gpu(tensors, m, native=False)
        a, ea = P.plan_cpu(tensors, S1, m, native=True)
        b, eb = P.plan_cpu(tensors, S1, m, native=False)
        assert a == b and ea == eb


def test_native_enumeration_limits():
    tensors = [P.Tensor(1 << 20, 100.0) for _ in range(12)]
    m = P.CostModel("topk", 0.01, P.load_profile_rows(TABLE), P.Cluster(N=16, link_gbs=3.0),
                    pcie=P.load_profile_pcie(TABLE))
    S = [("gpu", "indivisible")] * 12
    table = P.NativeTable(tensors, m)
    assert table.enumerate(S, [list(range(12))], max_evals=12) is None   # 13 vectors
    U, f, ev = table.enumerate(S, [list(range(12))], max_evals=13)
    assert ev == 13 and 0 <= U[0] <= 12
    assert f == table.simulate([("cpu", "indivisible") if i < U[0] else S[i] for i in range(12)])
