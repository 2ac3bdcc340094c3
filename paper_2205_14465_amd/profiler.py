"""Compression-time profiler and the benefit ratio of GPU compression.

The paper's system predicts the compression time of every tensor size it
will meet: it runs the compression and decompression operations of each
gradient-compression algorithm on each kind of compute resource, 100 times
per tensor size, and averages the runs (paper Sec. 4.3, "Compression
time").  Combined with communication cost models it gives the ratio of the
communication time that compression saves to the compression time it costs,
which grows with the tensor size because every compression launch has a
fixed cost (Sec. 4.4.2, Property #2, and the benefit-ratio figure).

This module measures both kinds of resource with the library's C ABI: for
each kind and tensor size, the mean time of one compress call (with error
feedback) and of one decompress-aggregate of W payloads.  The GPU side uses
the device entry points, timed by HIP events on the launch stream around
`runs` back-to-back calls; the CPU side uses the library's host operators
(bytecomp_cpu_compress, bytecomp_cpu_decompress_aggregate, multi-threaded),
timed by the host clock, with the run count cut down for sizes whose runs
would exceed a time budget (the row records the runs taken).  The host <->
device copy rate an offloaded tensor pays is measured too (pinned host
memory, one large copy each way).  The communication model is
the usual latency-bandwidth one for ring collectives among N GPUs
(Patarasuk and Yuan, JPDC 2009; Thakur et al., IJHPCA 2005):

    allreduce of B bytes:              2 (N-1) alpha + 2 (N-1)/N * B / beta
    allgather of B bytes per GPU:        (N-1) alpha +   (N-1)  * B / beta

with alpha the per-step latency and beta the per-link bandwidth.  The
benefit ratio of a tensor is (allreduce of its 4n dense bytes - allgather
of its payload) / (compress time + decompress-aggregate time of N payloads).
"""
from __future__ import annotations

import json
import math
import sys
from dataclasses import asdict, dataclass
from typing import Iterable, List, Sequence

KINDS = ("topk", "topk_sampled", "randk", "sign")
DEFAULT_SIZES = tuple(1 << p for p in range(6, 28))


@dataclass
class Row:
    kind: str
    n: int
    payload_bytes: int
    compress_us: float
    aggregate_us: float
    W: int
    runs: int
    device: str = "gpu"


def allreduce_us(nbytes: float, N: int, link_gbs: float, alpha_us: float) -> float:
    """Ring allreduce of nbytes among N GPUs, in microseconds."""
    if N <= 1:
        return 0.0
    return 2 * (N - 1) * alpha_us + 2 * (N - 1) / N * nbytes / (link_gbs * 1e3)


def allgather_us(nbytes_per_gpu: float, N: int, link_gbs: float, alpha_us: float) -> float:
    """Ring allgather of nbytes_per_gpu from each of N GPUs, in microseconds."""
    if N <= 1:
        return 0.0
    return (N - 1) * alpha_us + (N - 1) * nbytes_per_gpu / (link_gbs * 1e3)


def benefit_ratio(row: Row, N: int, link_gbs: float, alpha_us: float) -> float:
    """Communication time saved by compressing the tensor / time compression
    costs (compress + decompress-aggregate of N payloads)."""
    saved = allreduce_us(4.0 * row.n, N, link_gbs, alpha_us) - allgather_us(row.payload_bytes, N, link_gbs,
                                                                             alpha_us)
    cost = row.compress_us + row.aggregate_us
    return saved / cost if cost > 0 else math.inf


def profile(kinds: Iterable[str] = KINDS, sizes: Sequence[int] = DEFAULT_SIZES, runs: int = 100, W: int = 8,
            ratio: float = 0.01, warmup: int = 5, seed: int = 14465, on_row=None) -> List[Row]:
    """Mean GPU time of compress and of decompress-aggregate of W payloads,
    per kind and tensor size (one tensor per call), on cuda:0."""
    import torch

    from . import binding as B
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    gen = torch.Generator(device=dev)
    rows: List[Row] = []
    for kind in kinds:
        for n in sizes:
            gen.manual_seed(int(n))
            g = torch.randn(n, device=dev, generator=gen) * 0.01
            e = torch.zeros(n, device=dev)
            ns = [int(n)]
            out = B.alloc_payload(kind, ratio, ns, device=dev)
            ws = B.alloc_workspace(kind, ratio, ns, W, device=dev)
            agg_out = torch.empty(n, device=dev)
            comp = B.CompressCall(kind, ratio, [g], [e], out, ws, stream=stream)
            comp(seed)
            agg = B.AggregateCall(kind, ratio, [out] * W, ns, [agg_out], 1.0 / W, ws, stream=stream)
            for _ in range(warmup):
                comp(seed)
                agg()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            ev[0].record(stream)
            for _ in range(runs):
                comp(seed)
            ev[1].record(stream)
            ev[2].record(stream)
            for _ in range(runs):
                agg()
            ev[3].record(stream)
            torch.cuda.synchronize()
            assert B.bytecomp_device_status(ws) == 0
            rows.append(Row(kind, int(n), _payload_bytes(kind, out["off"]), 1e3 * ev[0].elapsed_time(ev[1]) / runs,
                            1e3 * ev[2].elapsed_time(ev[3]) / runs, W, runs))
            if on_row:
                on_row(rows[-1])
            del g, e, out, ws, agg_out, comp, agg
    return rows


def _payload_bytes(kind: str, off: Sequence[int]) -> int:
    units = int(off[-1])
    return 4 * units + 4 if kind == "sign" else 8 * units


def profile_cpu(kinds: Iterable[str] = KINDS, sizes: Sequence[int] = DEFAULT_SIZES, runs: int = 100, W: int = 8,
                ratio: float = 0.01, warmup: int = 2, seed: int = 14465, threads: int = 0,
                budget_s: float = 2.0, on_row=None) -> List[Row]:
    """Mean host time of the library's CPU operators: compress (error
    feedback on) and decompress-aggregate of W payloads, per kind and size,
    on `threads` host threads (0: every hardware thread).  A size whose
    `runs` runs would take longer than budget_s takes fewer runs (at least
    3) and says so in its row."""
    import time

    import numpy as np

    from . import binding as B
    rows: List[Row] = []
    for kind in kinds:
        for n in sizes:
            rng = np.random.default_rng(int(n))
            g = (rng.standard_normal(int(n), dtype=np.float32) * np.float32(0.01))
            e = np.zeros(int(n), np.float32)
            ns = [int(n)]
            out = B.cpu_alloc_payload(kind, ratio, ns)
            agg_out = [np.empty(int(n), np.float32)]

            call = B.CpuCompressCall(kind, ratio, [g], [e], out, threads)

            def comp():
                call(seed)

            agg = B.CpuAggregateCall(kind, ratio, [out] * W, ns, agg_out, 1.0 / W, threads)

            times = []
            for fn in (comp, agg):
                t0 = time.perf_counter()
                for _ in range(warmup):
                    fn()
                once = (time.perf_counter() - t0) / max(warmup, 1)
                r = runs if once * runs <= budget_s else max(3, int(budget_s / max(once, 1e-9)))
                t0 = time.perf_counter()
                for _ in range(r):
                    fn()
                times.append(((time.perf_counter() - t0) / r * 1e6, r))
            rows.append(Row(kind, int(n), _payload_bytes(kind, out["off"]), times[0][0], times[1][0], W,
                            min(times[0][1], times[1][1]), "cpu"))
            if on_row:
                on_row(rows[-1])
    return rows


def pcie_gbs(nbytes: int = 256 << 20, runs: int = 10) -> dict:
    """Host -> device and device -> host copy rates (GB/s) between pinned
    host memory and cuda:0, one nbytes copy at a time."""
    import torch
    dev = torch.device("cuda:0")
    h = torch.empty(nbytes // 4, dtype=torch.float32, pin_memory=True)
    d = torch.empty(nbytes // 4, dtype=torch.float32, device=dev)
    res = {}
    for name, dst, src in (("h2d", d, h), ("d2h", h, d)):
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(runs):
            dst.copy_(src, non_blocking=True)
        ev[1].record()
        torch.cuda.synchronize()
        res[name] = nbytes * runs / (ev[0].elapsed_time(ev[1]) * 1e6)
    return res


def table(rows: Sequence[Row], N: int = 8, link_gbs: float = 153.0, alpha_us: float = 5.0) -> str:
    """Text table of the profile with the benefit ratio at N GPUs."""
    lines = [f"{'kind':14s} {'device':>6s} {'n':>11s} {'payload B':>11s} {'compress us':>12s} "
             f"{'aggregate us':>13s} {'benefit':>8s} {'runs':>5s}"]
    for r in rows:
        lines.append(f"{r.kind:14s} {r.device:>6s} {r.n:11d} {r.payload_bytes:11d} {r.compress_us:12.2f} "
                     f"{r.aggregate_us:13.2f} {benefit_ratio(r, N, link_gbs, alpha_us):8.3f} {r.runs:5d}")
    return "\n".join(lines)


def main(argv=None) -> None:
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--runs", type=int, default=100)
    ap.add_argument("--W", type=int, default=8)
    ap.add_argument("--min-log2", type=int, default=6)
    ap.add_argument("--max-log2", type=int, default=27)
    ap.add_argument("--N", type=int, default=8, help="GPUs in the communication model")
    ap.add_argument("--link-gbs", type=float, default=153.0, help="per-link bandwidth (GB/s)")
    ap.add_argument("--alpha-us", type=float, default=5.0, help="per-step latency (us)")
    ap.add_argument("--devices", default="gpu,cpu", help="resources to profile: gpu, cpu or both")
    ap.add_argument("--cpu-threads", type=int, default=0, help="host threads of the CPU operators (0: all)")
    ap.add_argument("--cpu-budget-s", type=float, default=2.0, help="host time per size and operation")
    ap.add_argument("--json", action="store_true")
    args = ap.parse_args(argv)
    sizes = [1 << p for p in range(args.min_log2, args.max_log2 + 1)]
    devices = args.devices.split(",")
    rows: List[Row] = []
    copy = None

    def progress(r):
        print(f"# {r.device} {r.kind} n={r.n} done", file=sys.stderr, flush=True)

    if "gpu" in devices:
        rows += profile(sizes=sizes, runs=args.runs, W=args.W, on_row=progress)
        copy = pcie_gbs()
    if "cpu" in devices:
        rows += profile_cpu(sizes=sizes, runs=args.runs, W=args.W, threads=args.cpu_threads,
                            budget_s=args.cpu_budget_s, on_row=progress)
    if args.json:
        print(json.dumps({"pcie_gbs": copy,
                          "rows": [dict(asdict(r), benefit=benefit_ratio(r, args.N, args.link_gbs, args.alpha_us))
                                   for r in rows]}))
    else:
        if copy:
            print(f"# pcie_gbs h2d {copy['h2d']:.2f} d2h {copy['d2h']:.2f}")
        print(table(rows, args.N, args.link_gbs, args.alpha_us))


if __name__ == "__main__":
    main()
