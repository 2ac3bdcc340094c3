"""The compression-time profiler: the communication model's closed forms
(CPU) and one small profiling run (GPU)."""
import math

import pytest

from paper_2205_14465_amd import profiler as P


def test_ring_collectives_closed_forms():
    # one GPU communicates nothing
    assert P.allreduce_us(1e6, 1, 100.0, 5.0) == 0.0
    assert P.allgather_us(1e6, 1, 100.0, 5.0) == 0.0
    # N = 2: allreduce = 2 latency steps + the whole buffer once over a link
    assert math.isclose(P.allreduce_us(1e6, 2, 100.0, 5.0), 2 * 5.0 + 1e6 / 1e5)
    # N = 8: 14 steps, 2*7/8 of the bytes
    assert math.isclose(P.allreduce_us(8e6, 8, 100.0, 0.0), 2 * 7 / 8 * 8e6 / 1e5)
    # allgather moves the other N-1 GPUs' payloads
    assert math.isclose(P.allgather_us(1e6, 8, 100.0, 1.0), 7 * 1.0 + 7 * 1e6 / 1e5)


def test_benefit_ratio_grows_with_size_for_fixed_overhead():
    """A fixed per-call cost plus a per-byte cost gives a ratio that rises
    with the tensor size (the paper's Property #2)."""
    rows = [P.Row("topk", n, 8 * max(1, n // 100), 10.0 + n * 1e-5, 5.0 + n * 1e-6, 8, 1)
            for n in (1 << 10, 1 << 16, 1 << 22)]
    r = [P.benefit_ratio(x, 8, 153.0, 5.0) for x in rows]
    assert r[0] < r[1] < r[2]


def test_cpu_profile_runs_every_kind():
    """The CPU side times the library's host operators (no GPU needed)."""
    rows = P.profile_cpu(sizes=[1 << 10, 1 << 16], runs=3, W=4, warmup=1, threads=2)
    assert len(rows) == 2 * len(P.KINDS)
    for r in rows:
        assert r.device == "cpu" and r.runs == 3
        assert r.compress_us > 0 and r.aggregate_us > 0 and r.payload_bytes > 0
    assert " cpu " in P.table(rows)


def test_cpu_profile_cuts_runs_to_the_budget():
    rows = P.profile_cpu(kinds=["topk"], sizes=[1 << 20], runs=1000, W=2, warmup=1, threads=2, budget_s=0.01)
    assert 3 <= rows[0].runs < 1000


@pytest.mark.gpu
def test_profile_runs_every_kind():
    rows = P.profile(sizes=[1 << 10, 1 << 16], runs=3, W=4, warmup=1)
    assert len(rows) == 2 * len(P.KINDS)
    for r in rows:
        assert r.compress_us > 0 and r.aggregate_us > 0
        assert r.payload_bytes > 0
    assert "benefit" in P.table(rows)
