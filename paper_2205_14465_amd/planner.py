"""Compression-strategy planner: the paper's decision algorithm on
synthetic timelines (paper Sec. 4.2-4.4).

Given a training job's tensors in backward order (index 0 is the tensor
closest to the output layer, whose gradient is computed first), one
compression algorithm, and empirical time models, the planner picks a
compression option for every tensor so as to shorten the iteration:

  * the timeline model (Sec. 4.3, "Expressing interactions"): F(S), the
    iteration time of strategy S, from a simulation of the GPU (backward
    computation, GPU compression and decompression, served in order of
    release), the network (collectives one at a time) and the CPU
    (offloaded compression); compression on the GPU therefore delays the
    tensor computations behind it, as the paper's contention argument has
    it;
  * Algorithm 1, GPU compression (Sec. 4.4.2): tensors are visited in
    descending size, ties in ascending distance to the output layer
    (Property #2); uncompressed tensors communicated before a bubble of the
    communication timeline are dropped (Property #1), again after every
    decision; each visited tensor takes the GPU option (or none) that
    minimises F with the others fixed (Property #3);
  * Algorithm 2, CPU offloading (Sec. 4.4.3): the compressed tensors are
    grouped by size and option; in each group the tensors are offloaded in
    the order the paper's lemma fixes; every vector of per-group counts is
    evaluated and the best kept.  The lemma's statement names the tensors
    farthest from the output layer, while its stated intuition is that
    tensors offloaded earlier overlap more CPU work with communication and
    computation; in backward order the gradients that are ready earliest
    are those closest to the output layer, so the two point in opposite
    directions.  The default order follows the intuition (earliest-ready
    first, lemma_order="earliest"), which in this timeline model always
    matched the best of all offloading subsets on random instances; the
    statement's order is lemma_order="farthest".

The options are the decision tree's leaves reduced to what this library
computes: no compression (ring allreduce of the fp32 tensor), or the
compression algorithm on the GPU or the CPU with the indivisible scheme
(compress, ring allgather of the payloads, decompress-and-aggregate of the N
payloads) or the divisible scheme (compress, all-to-all of the N parts,
aggregate one part, compress it again, allgather, decompress).  Times come
from a CostModel: the GPU and CPU compress / aggregate times of the
compression-time profiler (paper_2205_14465_amd.profiler: the library's
device kernels and its host operators, interpolated in log-log over tensor
size), the profiler's ring-collective formulas, and its measured host <->
device copy rates.  Without CPU rows in the profile there is no CPU option.  The per-tensor computation times are an
input (the paper takes them from execution traces of 100 iterations; here
they are synthetic, since no training trace is available).
"""
from __future__ import annotations

import argparse
import heapq
import itertools
import json
import math
import os
import re
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

from .profiler import allgather_us, allreduce_us

Option = Optional[Tuple[str, str]]  # None, or (device "gpu"|"cpu", scheme "indivisible"|"divisible")
GPU_OPTIONS: Tuple[Tuple[str, str], ...] = (("gpu", "indivisible"), ("gpu", "divisible"))
EPS_US = 1e-3  # a change of strategy must shorten the iteration by more than this


@dataclass
class Tensor:
    n: int             # elements
    compute_us: float  # backward computation time of its gradient


@dataclass
class Cluster:
    N: int = 8               # GPUs in the ring
    link_gbs: float = 12.5   # per-link bandwidth, GB/s (100 Gb/s)
    alpha_us: float = 5.0    # per-step latency of a collective
    pcie_gbs: Optional[float] = None  # host <-> device copy rate; None: the profile's measured rates


def alltoall_us(nbytes_per_gpu: float, N: int, link_gbs: float, alpha_us: float) -> float:
    """Pairwise all-to-all: every GPU sends 1/N of its nbytes to each peer,
    N - 1 steps."""
    if N <= 1:
        return 0.0
    return (N - 1) * alpha_us + (N - 1) / N * nbytes_per_gpu / (link_gbs * 1e3)


class CostModel:
    """Time models of one compression algorithm on one cluster."""

    def __init__(self, kind: str, ratio: float, rows: Sequence[dict], cluster: Cluster, table_W: int = 8,
                 pcie: Optional[Dict[str, float]] = None):
        self.kind, self.ratio, self.c, self.table_W = kind, ratio, cluster, table_W
        self.curves: Dict[str, Tuple[List[float], List[float], List[float]]] = {}
        for dev in ("gpu", "cpu"):
            pts = sorted((int(r["n"]), float(r["compress_us"]), float(r["aggregate_us"])) for r in rows
                         if r["kind"] == kind and r.get("device", "gpu") == dev)
            if pts:
                self.curves[dev] = ([math.log(p[0]) for p in pts], [p[1] for p in pts], [p[2] for p in pts])
        if "gpu" not in self.curves:
            raise ValueError(f"no GPU compression-time rows for {kind}")
        rate = {"h2d": cluster.pcie_gbs, "d2h": cluster.pcie_gbs} if cluster.pcie_gbs else pcie
        self.pcie_rate = rate if rate and rate.get("h2d") and rate.get("d2h") else None
        # the CPU option needs measured CPU times and a copy rate
        self.has_cpu = "cpu" in self.curves and self.pcie_rate is not None

    @staticmethod
    def _interp(ln: List[float], ys: List[float], n: float) -> float:
        """Log-log interpolation in the size; past the largest size the time
        grows in proportion to n, below the smallest it stays constant."""
        x = math.log(max(n, 1.0))
        if x <= ln[0]:
            return ys[0]
        if x >= ln[-1]:
            return ys[-1] * math.exp(x - ln[-1])
        i = max(j for j in range(len(ln)) if ln[j] <= x)
        t = (x - ln[i]) / (ln[i + 1] - ln[i])
        return math.exp(math.log(ys[i]) * (1 - t) + math.log(ys[i + 1]) * t)

    def payload_bytes(self, n: int) -> float:
        if self.kind == "sign":
            return 4 * math.ceil(n / 32) + 4
        bits = {"terngrad": 2, "qsgd4": 4, "qsgd8": 8}.get(self.kind)
        if bits:
            return 4 * math.ceil(n * bits / 32) + 4
        ppm = round(self.ratio * 1e6)
        k = min(n, max(1, -(-n * ppm // 1000000))) if n else 0
        return 8 * k

    # compute-resource times
    def compress(self, device: str, n: float) -> float:
        ln, comp, _ = self.curves[device]
        return self._interp(ln, comp, n)

    def aggregate(self, device: str, n: float, parts: int) -> float:
        """Decompress and aggregate `parts` payloads of a tensor of n elements
        (the profile aggregates table_W payloads; the time is taken in
        proportion to the payload count)."""
        ln, _, agg = self.curves[device]
        return self._interp(ln, agg, n) * parts / self.table_W

    def pcie(self, nbytes: float, direction: str) -> float:
        """Copy of nbytes between host and device; direction 'h2d' or 'd2h'."""
        return nbytes / (self.pcie_rate[direction] * 1e3)

    # network times
    def allreduce(self, n: int) -> float:
        return allreduce_us(4.0 * n, self.c.N, self.c.link_gbs, self.c.alpha_us)

    def allgather(self, nbytes: float) -> float:
        return allgather_us(nbytes, self.c.N, self.c.link_gbs, self.c.alpha_us)

    def alltoall(self, nbytes: float) -> float:
        return alltoall_us(nbytes, self.c.N, self.c.link_gbs, self.c.alpha_us)

    def stages(self, t: Tensor, opt: Option) -> List[Tuple[str, float, str]]:
        """(resource, microseconds, label) of a tensor's steps after its
        computation, in order; resources are 'gpu', 'cpu', 'pcie', 'net'."""
        n = t.n
        if opt is None:
            return [("net", self.allreduce(n), "allreduce")]
        dev, scheme = opt
        N = self.c.N
        p = self.payload_bytes(n)
        st: List[Tuple[str, float, str]] = []
        if dev == "cpu":
            st.append(("pcie", self.pcie(4.0 * n, "d2h"), "to host"))
        st.append((dev, self.compress(dev, n), "compress"))
        if scheme == "indivisible":
            st.append(("net", self.allgather(p), "allgather"))
            st.append((dev, self.aggregate(dev, n, N), "aggregate"))
        else:
            st.append(("net", self.alltoall(p), "alltoall"))
            st.append((dev, self.aggregate(dev, n / N, N), "aggregate part"))
            st.append((dev, self.compress(dev, n / N), "compress part"))
            st.append(("net", self.allgather(self.payload_bytes(max(1, n // N))), "allgather"))
            st.append((dev, self.aggregate(dev, n, 1), "decompress"))
        if dev == "cpu":
            st.append(("pcie", self.pcie(4.0 * n, "h2d"), "to device"))
        return st


@dataclass
class Timeline:
    iteration_us: float
    net: List[Tuple[float, float, int]] = field(default_factory=list)  # (start, end, tensor) in service order
    net_first: List[bool] = field(default_factory=list)  # the tensor's first collective
    done_us: List[float] = field(default_factory=list)


def simulate(tensors: Sequence[Tensor], S: Sequence[Option], model: CostModel) -> Timeline:
    """Iteration time of strategy S.  Every resource serves one job at a
    time, in order of release (ties: lower tensor index, then earlier step).
    Tensor i's computation is released when tensor i-1's computation ends;
    its later steps follow one another as each ends."""
    T = len(tensors)
    stages = [[("gpu", tensors[i].compute_us, "compute")] + model.stages(tensors[i], S[i]) for i in range(T)]
    free = {"gpu": 0.0, "cpu": 0.0, "pcie": 0.0, "net": 0.0}
    waiting: Dict[str, list] = {r: [] for r in free}
    running: Dict[str, Optional[tuple]] = {r: None for r in free}
    events: list = []  # (time, seq, resource) completions
    seq = itertools.count()
    done = [0.0] * T
    net: List[Tuple[float, float, int]] = []
    net_first: List[bool] = []
    seen = set()

    def release(t: float, i: int, s: int) -> None:
        r = stages[i][s][0]
        heapq.heappush(waiting[r], (t, i, s))

    def start(r: str, now: float) -> None:
        if running[r] is None and waiting[r]:
            t_rel, i, s = heapq.heappop(waiting[r])
            begin = max(now, t_rel, free[r])
            end = begin + stages[i][s][1]
            running[r] = (i, s, begin, end)
            free[r] = end
            heapq.heappush(events, (end, next(seq), r))

    if T:
        release(0.0, 0, 0)
        start("gpu", 0.0)
    while events:
        now, _, r = heapq.heappop(events)
        i, s, begin, end = running[r]
        running[r] = None
        if r == "net":
            net.append((begin, end, i))
            net_first.append(i not in seen)
            seen.add(i)
        if s + 1 < len(stages[i]):
            release(now, i, s + 1)
        else:
            done[i] = now
        if s == 0 and i + 1 < T:
            release(now, i + 1, 0)
        for res in free:
            start(res, now)
    return Timeline(max(done) if T else 0.0, net=net, net_first=net_first, done_us=done)


def bubble_cut(tl: Timeline, eps_us: float = 1.0) -> float:
    """Start time of the last bubble of the communication timeline: a gap
    longer than eps before a tensor's first collective, i.e. the tensor was
    not ready when the previous communication ended (Property #1).  A gap
    between the two collectives of one divisible-scheme tensor is that
    tensor's own processing, not a bubble.  -inf without a bubble."""
    last = -math.inf
    for k in range(1, len(tl.net)):
        if tl.net_first[k] and tl.net[k][0] - tl.net[k - 1][1] > eps_us:
            last = tl.net[k - 1][1]
    return last


def _remove(tensors, S, model, live: set) -> None:
    """Property #1: drop uncompressed tensors whose communication ends at or
    before the last bubble."""
    tl = simulate(tensors, S, model)
    cut = bubble_cut(tl)
    if cut == -math.inf:
        return
    for s0, e0, i in tl.net:
        if S[i] is None and e0 <= cut:
            live.discard(i)


def plan_gpu(tensors: Sequence[Tensor], model: CostModel, options=GPU_OPTIONS, native: bool = True) -> List[Option]:
    """Algorithm 1: GPU compression decisions.  The candidates' iteration
    times come from the library's timeline model (native=False: from
    simulate(), for tests); the bubbles of Property #1 from simulate()."""
    T = len(tensors)
    S: List[Option] = [None] * T
    order = sorted(range(T), key=lambda i: (-tensors[i].n, i))  # Property #2
    live = set(range(T))
    table = NativeTable(tensors, model) if native else None

    def F(strategy):
        return table.simulate(strategy) if table is not None else simulate(tensors, strategy, model).iteration_us

    _remove(tensors, S, model, live)
    for i in order:
        if i not in live:
            continue
        best, best_f = S, F(S)
        for c in options:  # Property #3
            cand = list(S)
            cand[i] = c
            f = F(cand)
            if f < best_f - EPS_US:
                best, best_f = cand, f
        S = best
        _remove(tensors, S, model, live)
    return S


# ------------------------------------------- the native timeline model
# The library's host functions bytecomp_plan_simulate / _enumerate evaluate
# the same timeline model as simulate() (a CPU test compares them bit for
# bit); Algorithm 2 uses them so that its exhaustive search reaches far
# more count vectors.

OPTION_CODE = {None: 0, ("gpu", "indivisible"): 1, ("gpu", "divisible"): 2, ("cpu", "indivisible"): 3,
               ("cpu", "divisible"): 4}
RESOURCE_CODE = {"gpu": 0, "cpu": 1, "pcie": 2, "net": 3}


class NativeTable:
    """Every tensor's steps under every option, flattened for the library."""

    def __init__(self, tensors: Sequence[Tensor], model: CostModel):
        import ctypes

        import numpy as np
        self.T = len(tensors)
        opts = [None, ("gpu", "indivisible"), ("gpu", "divisible"), ("cpu", "indivisible"), ("cpu", "divisible")]
        cpu_ok = getattr(model, "has_cpu", True)
        off, res, dur = [0], [], []
        for t in tensors:
            for o in opts:
                st = model.stages(t, o) if (o is None or o[0] == "gpu" or cpu_ok) else []
                for r, us, _ in st:
                    res.append(RESOURCE_CODE[r])
                    dur.append(float(us))
                off.append(len(res))
        self.compute = np.array([float(t.compute_us) for t in tensors] or [0.0], dtype=np.float64)
        self.off = np.array(off, dtype=np.uint64)
        self.res = np.array(res or [0], dtype=np.int32)
        self.dur = np.array(dur or [0.0], dtype=np.float64)
        self._c = ctypes

    def _args(self):
        return (self.T, self.compute.ctypes.data, self.off.ctypes.data, self.res.ctypes.data, self.dur.ctypes.data)

    def simulate(self, S: Sequence[Option]) -> float:
        import numpy as np

        from . import binding as B
        opt = np.array([OPTION_CODE[o] for o in S] or [0], dtype=np.int32)
        out = self._c.c_double(0.0)
        B._check("bytecomp_plan_simulate",
                 B.lib().bytecomp_plan_simulate(*self._args(), opt.ctypes.data, self._c.byref(out)))
        return out.value

    def enumerate(self, S: Sequence[Option], groups: Sequence[Sequence[int]], max_evals: int,
                  threads: int = 0) -> Optional[Tuple[List[int], float, int]]:
        """Algorithm 2's exhaustive search; None when the count vectors
        exceed max_evals."""
        import numpy as np

        from . import binding as B
        opt = np.array([OPTION_CODE[o] for o in S] or [0], dtype=np.int32)
        goff = np.array([0] + list(itertools.accumulate(len(g) for g in groups)), dtype=np.uint64)
        mem = np.array([i for g in groups for i in g] or [0], dtype=np.int32)
        G = len(groups)
        best = np.zeros(max(G, 1), dtype=np.int32)
        bus = self._c.c_double(0.0)
        ev = self._c.c_uint64(0)
        rc = B.lib().bytecomp_plan_enumerate(*self._args(), opt.ctypes.data, G, goff.ctypes.data, mem.ctypes.data,
                                             int(max_evals), float(EPS_US), int(threads), best.ctypes.data,
                                             self._c.byref(bus), self._c.byref(ev))
        if rc == -5:  # BC_E_SIZE: beyond max_evals
            return None
        B._check("bytecomp_plan_enumerate", rc)
        return [int(x) for x in best[:G]], bus.value, int(ev.value)


def plan_cpu(tensors: Sequence[Tensor], S: Sequence[Option], model: CostModel, max_evals: int = 2_000_000,
             lemma_order: str = "earliest", native: bool = True) -> Tuple[List[Option], int]:
    """Algorithm 2: CPU offloading of the GPU-compressed tensors.  Returns
    the strategy and the number of strategies evaluated.  Every count
    vector is evaluated when their number (the Theorem's bound) is at most
    max_evals (by the library's native timeline model; native=False: by
    simulate(), for tests); beyond that the counts are chosen one group at
    a time instead (each group's count minimising F with the others fixed,
    repeated until no count changes)."""
    if not getattr(model, "has_cpu", True):
        return list(S), 0
    groups: Dict[tuple, List[int]] = {}
    for i, o in enumerate(S):
        if o is not None and o[0] == "gpu":
            groups.setdefault((tensors[i].n, o), []).append(i)
    keys = sorted(groups)
    if lemma_order not in ("earliest", "farthest"):
        raise ValueError(lemma_order)
    for k in keys:  # tensor index = backward order: 0 is ready first, closest to the output layer
        groups[k].sort(reverse=(lemma_order == "farthest"))

    def apply(U):
        out = list(S)
        for k, u in zip(keys, U):
            for i in groups[k][:u]:
                out[i] = ("cpu", out[i][1])
        return out

    sizes = [len(groups[k]) + 1 for k in keys]
    total = math.prod(sizes) if sizes else 1
    evals = 0
    table = NativeTable(tensors, model) if native else None

    def F(strategy):
        return table.simulate(strategy) if table is not None else simulate(tensors, strategy, model).iteration_us

    if total <= max_evals:
        if table is not None:
            res = table.enumerate(S, [groups[k] for k in keys], max_evals)
            if res is not None:
                U, _, evals = res
                return apply(U), evals
        best, best_f = list(S), math.inf
        for U in itertools.product(*[range(m) for m in sizes]):
            f = F(apply(U))
            evals += 1
            if f < best_f - EPS_US:
                best, best_f = apply(U), f
        return best, evals
    U = [0] * len(keys)
    best_f = F(apply(U))
    changed = True
    while changed:
        changed = False
        for g in range(len(keys)):
            for u in range(sizes[g]):
                if u == U[g]:
                    continue
                V = list(U)
                V[g] = u
                f = F(apply(V))
                evals += 1
                if f < best_f - EPS_US:
                    U, best_f, changed = V, f, True
    return apply(U), evals


# ------------------------------------------------------------ CLI, inputs

def load_profile_rows(path: str) -> List[dict]:
    """Rows of the compression-time table the profiler writes (its text form)."""
    rows = []
    pat = re.compile(r"^(\w+)\s+(gpu|cpu)\s+(\d+)\s+(\d+)\s+([\d.]+)\s+([\d.]+)\s+([\d.]+)\s+(\d+)\s*$")
    with open(path) as fh:
        for line in fh:
            m = pat.match(line)
            if m:
                rows.append({"kind": m.group(1), "device": m.group(2), "n": int(m.group(3)),
                             "compress_us": float(m.group(5)), "aggregate_us": float(m.group(6)),
                             "runs": int(m.group(8))})
    return rows


def load_profile_pcie(path: str) -> Optional[Dict[str, float]]:
    """The host <-> device copy rates (GB/s) the profiler measured, if any."""
    pat = re.compile(r"^# pcie_gbs h2d ([\d.]+) d2h ([\d.]+)")
    with open(path) as fh:
        for line in fh:
            m = pat.match(line)
            if m:
                return {"h2d": float(m.group(1)), "d2h": float(m.group(2))}
    return None


def synthetic_job(model_name: str, us_per_mparam: float) -> List[Tensor]:
    """Tensors of a model family in backward order with computation time
    proportional to the tensor's size plus a fixed 20 us per layer."""
    from . import workloads as WL
    shapes = {"resnet50": WL.resnet50_shapes, "bertbase": WL.bert_base_shapes,
              "gpt2xl": WL.gpt2_xl_shapes}[model_name]()
    sizes = [WL.numel(s) for s in shapes][::-1]  # the output side first
    return [Tensor(n, 20.0 + us_per_mparam * n / 1e6) for n in sizes]


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--model", default="resnet50", choices=["resnet50", "bertbase", "gpt2xl"])
    ap.add_argument("--kind", default="sign")
    ap.add_argument("--ratio", type=float, default=0.01)
    ap.add_argument("--N", type=int, default=64)
    ap.add_argument("--link-gbs", type=float, default=12.5)
    ap.add_argument("--alpha-us", type=float, default=5.0)
    ap.add_argument("--us-per-mparam", type=float, default=40.0,
                    help="synthetic backward time per million parameters")
    ap.add_argument("--table", default=os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                                                    "profiles", "compression_time_model.txt"))
    ap.add_argument("--json", action="store_true")
    a = ap.parse_args(argv)
    tensors = synthetic_job(a.model, a.us_per_mparam)
    model = CostModel(a.kind, a.ratio, load_profile_rows(a.table),
                      Cluster(N=a.N, link_gbs=a.link_gbs, alpha_us=a.alpha_us), pcie=load_profile_pcie(a.table))
    from . import binding as B
    B.lib()  # load the library (and torch) before the clock starts
    t0 = time.perf_counter()
    S1 = plan_gpu(tensors, model)
    t1 = time.perf_counter()
    S2, evals = plan_cpu(tensors, S1, model)
    t2 = time.perf_counter()
    T = len(tensors)
    res = {
        "model": a.model, "kind": a.kind, "N": a.N, "link_gbs": a.link_gbs, "tensors": T,
        "fp32_us": simulate(tensors, [None] * T, model).iteration_us,
        "all_gpu_indivisible_us": simulate(tensors, [("gpu", "indivisible")] * T, model).iteration_us,
        "all_gpu_divisible_us": simulate(tensors, [("gpu", "divisible")] * T, model).iteration_us,
        "algorithm1_us": simulate(tensors, S1, model).iteration_us,
        "algorithm1_2_us": simulate(tensors, S2, model).iteration_us,
        "compressed_gpu": sum(1 for o in S2 if o and o[0] == "gpu"),
        "compressed_cpu": sum(1 for o in S2 if o and o[0] == "cpu"),
        "plan_gpu_s": round(t1 - t0, 3), "plan_cpu_s": round(t2 - t1, 3), "cpu_evals": evals,
    }
    if a.json:
        print(json.dumps(res))
    else:
        for k, v in res.items():
            print(f"{k:24s} {v:.1f}" if isinstance(v, float) else f"{k:24s} {v}")


if __name__ == "__main__":
    main()
