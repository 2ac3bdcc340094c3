"""Benchmark of the compression hot path on one MI355X.

One step = compress (with error feedback) every tensor of the workload, then
decompress-and-aggregate W workers' payloads of the same tensor list: the
whole hot path for that workload's operator.  Inputs (gradients, residuals,
the W generated worker payloads) are resident in HBM before timing starts.
The default workload is the largest single-GPU one: GPT-2-XL gradients
(1.56B fp32 elements), random-k 1%, W = 16.

value = algorithmic bytes per step / time per step, in GB/s, where the
algorithmic bytes are what the method must move:
  compress:  read g (4 B/elem fp32, 2 B fp16) + read e (4 B) + write e (4 B)
             + write the payload (8 B per sparse entry; 4 B per sign or
             quantizer code word + 4 B per tensor scale)
  aggregate: read W payloads + write the dense fp32 output (4 B/elem).
Timing: K steps between two synchronisations; before each step, untimed,
one kernel writes 1 GiB (more than the 256 MB last-level cache) and another
reads a second 1 GiB buffer (which writes back the dirty lines of the
first), so that no step starts with its inputs in the cache or pays for
another kernel's write-backs, and HIP events on the launch stream bracket
each step (the flush stays outside).  Per-operation times are the
median, 10th and 90th percentile of --reps flushed repetitions.  The
roofline entry is the dominant kernel -- the longest of the step's
timeable kernels, measured -- with its algorithmic bytes per launch over
its average launch duration (events the library records at that kernel's
start and end) against the 8 TB/s HBM peak.  The CPU baseline times the
oracle on a bounded sample of the same workload, on one core and on every
core the process may use (OpenMP over tensors and element ranges).
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORD_KINDS = ("sign", "terngrad", "qsgd4", "qsgd8")  # payload: packed words + one scale per tensor
METRIC = "gradient GB/s through compress+EF and decompress-aggregate; % of HBM peak"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(wl, off, kind):
    n = wl.n_total
    gbytes = 2 if wl.grad_dtype == "float16" else 4
    if wl.momentum:  # DGC: the velocity is read and written as well
        gbytes += 8
    if kind in WORD_KINDS:
        payload = 4 * int(off[-1]) + 4 * wl.T
    else:
        payload = 8 * int(off[-1])
    comp = (gbytes + 8) * n + payload
    agg = wl.W * payload + 4 * n
    return comp, agg, payload


def host_description():
    """Host facts for the CPU baseline: logical CPUs, the ones this process
    may run on, the CPU model and the RAM."""
    model, ram_gb = None, None
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
        with open("/proc/meminfo") as fh:
            for ln in fh:
                if ln.startswith("MemTotal"):
                    ram_gb = round(int(ln.split()[1]) / 2**20, 1)
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"nproc": os.cpu_count(), "usable_cpus": usable, "model": model, "ram_gib": ram_gb}


def cpu_baseline(wl, off, budget_s=10.0):
    """Time the oracle on a bounded sample of the workload: whole tensors in
    workload order until about budget_s of single-thread compress plus
    aggregate work, each tensor aggregated over all W generated payloads;
    then the same sample through the oracle's all-core list calls (OpenMP
    over tensors and element ranges, bit-identical results)."""
    import oracle as O
    from paper_2205_14465_amd import workloads as WL
    kind = wl.kind
    word = kind in WORD_KINDS
    counts = [int(off[t + 1] - off[t]) for t in range(wl.T)]
    comp_bytes = agg_bytes = 0
    comp_s = agg_s = 0.0
    used, gs, es, pays_t = [], [], [], []
    gbytes = (2 if wl.grad_dtype == "float16" else 4) + (8 if wl.momentum else 0)
    serial_payload = []
    for t in range(wl.T):
        if comp_s + agg_s > budget_s:
            break
        g = WL.gradient(wl, t)
        e = WL.residual(wl, t)
        t0 = time.perf_counter()
        if wl.momentum:
            res = O.compress_dgc(kind, g, e, np.zeros(g.size, np.float32), wl.momentum, wl.ratio, WL.SEED, t)
        elif kind == "sign":
            res = O.compress_sign(g, e)
        elif kind in O.QUANT_BITS:
            res = O.compress_quant(g, e, O.QUANT_BITS[kind], WL.SEED, t)
        elif kind == "topk":
            res = O.compress_topk(g, e, wl.ratio)
        elif kind == "topk_sampled":
            res = O.compress_topk_sampled(g, e, wl.ratio, WL.SEED, t)
        else:
            res = O.compress_randk(g, e, wl.ratio, WL.SEED, t)
        comp_s += time.perf_counter() - t0
        serial_payload.append(res[:2])
        n = wl.sizes[t]
        pay = (4 * counts[t] + 4) if word else 8 * counts[t]
        comp_bytes += (gbytes + 8) * n + pay
        # aggregate this tensor over W generated payloads
        lists = []
        for w in range(wl.W):
            rng = WL.rng_for(wl.wid, t, WL.ROLE_WORKER + w)
            if kind == "sign":
                lists.append(WL.random_sign_words(rng, [n], [counts[t]])[0])
            elif kind in O.QUANT_BITS:
                lists.append(WL.random_code_words(rng, [n], [counts[t]], O.QUANT_BITS[kind])[0])
            else:
                i, v = WL.random_sparse_lists(rng, [n], [counts[t]])
                lists.append((i[0], v[0]))
        scale = np.float32(1e-3 if kind == "sign" else 4e-3)
        t0 = time.perf_counter()
        if kind == "sign":
            O.aggregate_sign(n, lists, [scale] * wl.W, 1.0 / wl.W)
        elif kind in O.QUANT_BITS:
            O.aggregate_quant(n, O.QUANT_BITS[kind], lists, [scale] * wl.W, 1.0 / wl.W)
        else:
            O.aggregate_sparse(n, [a for a, _ in lists], [b for _, b in lists], 1.0 / wl.W)
        agg_s += time.perf_counter() - t0
        agg_bytes += wl.W * pay + 4 * n
        used.append(t)
        gs.append(g)
        es.append(e)
        pays_t.append(lists)
    total = comp_bytes + agg_bytes
    secs = comp_s + agg_s
    one = {"value": round(total / secs / 1e9, 4), "cores": 1, "seconds": round(secs, 2),
           "compress_gbs": round(comp_bytes / comp_s / 1e9, 4) if comp_s else None,
           "aggregate_gbs": round(agg_bytes / agg_s / 1e9, 4) if agg_s else None}
    sample = (f"{len(used)} of {wl.T} tensors ({sum(wl.sizes[t] for t in used)} elements) in workload order, "
              f"compress+EF and aggregate over W={wl.W}")
    out = {"value": one["value"], "unit": "GB/s", "cores": 1, "kind": "oracle", "sample": sample,
           "one_core": one, "host": host_description()}
    if wl.momentum:
        out["all_cores"] = None  # the list calls cover the plain kinds only
        return out
    threads = O.omp_max_threads()
    ns = [wl.sizes[t] for t in used]
    t0 = time.perf_counter()
    pay_omp, _ = O.compress_list_omp(kind, wl.ratio, WL.SEED, gs, es, threads, tensor_ids=used)
    c_s = time.perf_counter() - t0
    # the all-core payload equals the serial one
    for q, (a, b) in enumerate(serial_payload):
        seg = slice(pay_omp["off"][q], pay_omp["off"][q + 1])
        got = pay_omp["bits"][seg] if word else pay_omp["idx"][seg]
        assert np.array_equal(got, a), ("all-core oracle differs from the serial one", used[q])
    off_s = np.asarray(pay_omp["off"])
    pay_dicts = []
    for w in range(wl.W):
        if word:
            pay_dicts.append({"bits": np.concatenate([pays_t[q][w] for q in range(len(used))]),
                              "scale": np.full(len(used), scale, np.float32), "off": off_s})
        else:
            pay_dicts.append({"idx": np.concatenate([pays_t[q][w][0] for q in range(len(used))]),
                              "val": np.concatenate([pays_t[q][w][1] for q in range(len(used))]), "off": off_s})
    t0 = time.perf_counter()
    O.aggregate_list_omp(kind, ns, pay_dicts, 1.0 / wl.W, threads)
    a_s = time.perf_counter() - t0
    allc = {"value": round(total / (c_s + a_s) / 1e9, 4), "cores": threads, "seconds": round(c_s + a_s, 2),
            "compress_gbs": round(comp_bytes / c_s / 1e9, 4), "aggregate_gbs": round(agg_bytes / a_s / 1e9, 4)}
    out.update({"value": allc["value"], "cores": threads, "all_cores": allc,
                "compress_gbs": allc["compress_gbs"], "aggregate_gbs": allc["aggregate_gbs"]})
    return out


def source_digest(files):
    """sha256 over the named source files (paths relative to the repo root)."""
    h = hashlib.sha256()
    for f in sorted(files):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def counted_traffic(kernel, slug):
    """HBM bytes per launch of `kernel` counted by rocprofv3 (FETCH_SIZE and
    WRITE_SIZE, each in its own run), scaled by what the same counters read
    for the 1 GiB read + 1 GiB write calibration pass.  The figures live in
    profiles/traffic_<kernel>_<workload slug>.txt on a line starting 'TRAFFIC ';
    they are dropped (None) once the kernel's sources differ from the ones
    the counters were taken on."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{slug}.txt")
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as fh:
        for ln in fh:
            if ln.startswith("TRAFFIC "):
                rec = json.loads(ln[len("TRAFFIC "):])
    if rec is None or rec.get("kernel") != kernel:
        return None
    try:
        if source_digest(rec["sources"]) != rec["source_sha256"]:
            return None
    except OSError:
        return None
    cal = float(1 << 30) / 1024.0  # KiB the calibration pass moves each way
    fetch = rec["fetch_kib"] * 1024.0 * cal / rec["copy_fetch_kib"]
    write = rec["write_kib"] * 1024.0 * cal / rec["copy_write_kib"]
    return round(fetch + write)


def kernel_candidates(wl, kind, comp_b, agg_b, pay_b):
    """Kernels of the step that the library can time, with the algorithmic
    bytes one launch moves (what the method must move, attributed to the
    kernel that moves it)."""
    n = wl.n_total
    # DGC: the top-k stream pass also takes the velocity step (reads g and u, writes u)
    g_in = (2 if wl.grad_dtype == "float16" else 4) + (8 if wl.momentum else 0)
    if kind == "randk":
        return [("randk_stream", comp_b), ("aggregate_sparse", agg_b)]
    if kind in ("topk", "topk_sampled"):
        # the streaming EF pass (topk_compact in the general pipeline,
        # topk_hist in the few-chunk path) reads g and e and writes e; the
        # payload is written by the emit kernel
        return [("topk_compact", (g_in + 8) * n), ("topk_hist", (g_in + 8) * n), ("aggregate_sparse", agg_b)]
    if kind == "sign":
        # one pass: everything; two passes: the first reads g and e and
        # writes the bits and scales
        return [("sign_onepass", comp_b), ("sign_pass1", (g_in + 4) * n + pay_b), ("aggregate_sign", agg_b)]
    return [("quant_onepass", comp_b), ("quant_pass1", (g_in + 4) * n), ("aggregate_quant", agg_b)]


def pct(sorted_ms, q):
    return sorted_ms[min(len(sorted_ms) - 1, int(q * len(sorted_ms)))]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--reps", type=int, default=100, help="flushed repetitions of each operation")
    ap.add_argument("--workload", type=int, default=4, choices=[1, 2, 3, 4, 5, 6, 7, 8, 9])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-flush", action="store_true", help="no cache flush between steps (warm-cache numbers)")
    ap.add_argument("--scheme", choices=["indivisible", "divisible"], default="indivisible",
                    help="divisible: time node 0's step of the divisible scheme instead")
    ap.add_argument("--parts", type=int, default=8)
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the compression hot path has no inter-GPU step "
              "here (worker payloads are generated inputs); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2205_14465_amd import binding as B
    from paper_2205_14465_amd import workloads as WL

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B.lib()
    wl = WL.workload(args.workload)
    kind = wl.kind
    off = B.bytecomp_layout(kind, wl.ratio, wl.sizes)
    log(f"workload {wl.wid}: {wl.name}; generating inputs")
    grads, resids, payloads, outs = WL.device_inputs(wl, off, dev)
    own = B.alloc_payload(kind, wl.ratio, wl.sizes, device=dev)
    ws = B.alloc_workspace(kind, wl.ratio, wl.sizes, wl.W, device=dev)
    comp_b, agg_b, pay_b = algorithmic_bytes(wl, off, kind)
    alpha = 1.0 / wl.W
    stream = torch.cuda.current_stream()

    if args.scheme == "divisible" and wl.momentum:
        sys.exit("bench.py: the divisible-scheme step is not timed for the DGC workload")
    if args.scheme == "divisible":
        return divisible(args, wl, off, payloads, ws, dev, stream)

    # argument arrays are marshalled once; each call is one C-ABI call
    if wl.momentum:
        vels = [torch.zeros(n, dtype=torch.float32, device=dev) for n in wl.sizes]
        compress_call = B.DgcCall(kind, wl.ratio, wl.momentum, grads, resids, vels, own, ws, stream=stream)
    else:
        compress_call = B.CompressCall(kind, wl.ratio, grads, resids, own, ws, stream=stream)
    aggregate_call = B.AggregateCall(kind, wl.ratio, payloads, wl.sizes, outs, alpha, ws, stream=stream)

    # the caller varies the seed per iteration (random-k indices, the
    # sampled threshold's sample)
    seeds = iter(range(WL.SEED, WL.SEED + (1 << 62)))

    def compress():
        compress_call(next(seeds))

    def aggregate():
        aggregate_call()

    # before each timed step or operation, untimed: a write of 1 GiB (a
    # torch fill kernel) evicts the 256 MB last-level cache, then a read of
    # another 1 GiB (a torch sum) writes back the dirty lines the fill left,
    # so that the timed kernels start from a cold, clean cache and do not
    # pay for writing back the flush's data
    flush_buf = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    flush_rd = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    flush_sum = torch.empty((), dtype=torch.float32, device=dev)

    def flush():
        if not args.no_flush:
            flush_buf.fill_(1.0)
            torch.sum(flush_rd, dim=0, out=flush_sum)

    def events(k):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(k)]
        for e in ev:
            e.record(stream)  # creates the HIP events (the library records on some of them)
        return ev

    log("warmup")
    for _ in range(args.warmup):
        compress()
        aggregate()
    torch.cuda.synchronize()
    assert B.bytecomp_device_status(ws) == 0

    # the timed region: exactly K steps between two synchronisations, each
    # bracketed by events on the launch stream, a flush before each
    K = args.steps
    log(f"timing {K} steps")
    sev = [events(2) for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for r in range(K):
        flush()
        sev[r][0].record(stream)
        compress()
        aggregate()
        sev[r][1].record(stream)
    torch.cuda.synchronize()
    wall_s = (time.perf_counter() - t0) / K
    step_ms = sorted(sev[r][0].elapsed_time(sev[r][1]) for r in range(K))
    step_avg = sum(step_ms) / K
    assert B.bytecomp_device_status(ws) == 0

    # per-operation device time: --reps flushed repetitions of each call
    R = args.reps
    log(f"timing {R} repetitions of each operation")
    oev = [events(4) for _ in range(R)]
    torch.cuda.synchronize()
    for r in range(R):
        flush()
        oev[r][0].record(stream)
        compress()
        oev[r][1].record(stream)
        flush()
        oev[r][2].record(stream)
        aggregate()
        oev[r][3].record(stream)
    torch.cuda.synchronize()
    comp_ms = sorted(oev[r][0].elapsed_time(oev[r][1]) for r in range(R))
    agg_ms = sorted(oev[r][2].elapsed_time(oev[r][3]) for r in range(R))
    assert B.bytecomp_device_status(ws) == 0

    # the dominant kernel: each timeable kernel of the step, timed by the
    # library's events around its own launch; the longest one
    RK = max(5, R // 5)
    kstats = {}
    for name, kbytes in kernel_candidates(wl, kind, comp_b, agg_b, pay_b):
        kev = [events(2) for _ in range(RK)]
        torch.cuda.synchronize()
        ran = True
        for r in range(RK):
            flush()
            B.bytecomp_time_next_launch(name, kev[r][0], kev[r][1])
            compress()
            aggregate()
            if B.bytecomp_time_next_launch(None, None, None):
                ran = False  # the step does not launch this kernel
                break
        torch.cuda.synchronize()
        if not ran:
            continue
        ms = sorted(kev[r][0].elapsed_time(kev[r][1]) for r in range(RK))
        kstats[name] = {"bytes": kbytes, "ms_avg": sum(ms) / RK, "ms_p50": pct(ms, 0.5)}
    dom_kernel = max(kstats, key=lambda k: kstats[k]["ms_avg"])
    dom = kstats[dom_kernel]

    # achievable-bandwidth reference and the counter calibration kernel: a
    # plain elementwise pass reading 1 GiB and writing 1 GiB
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)
    ce = events(2)
    torch.cuda.synchronize()
    ce[0].record(stream)
    for _ in range(5):
        torch.neg(src, out=dst)
    ce[1].record(stream)
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * src.numel() * 4 / (ce[0].elapsed_time(ce[1]) * 1e-3) / 1e9
    del src, dst
    # the access pattern of the compress stream passes (read g and e, write
    # e): a plain elementwise e += g over the workload's element count (at
    # least 2^28 fp32, so that it streams from HBM)
    n_add = max(1 << 28, wl.n_total)
    src = torch.zeros(n_add, dtype=torch.float32, device=dev)
    dst = torch.zeros_like(src)
    dst.add_(src)
    torch.cuda.synchronize()
    ce[0].record(stream)
    for _ in range(5):
        dst.add_(src)
    ce[1].record(stream)
    torch.cuda.synchronize()
    add_gbs = 5 * 12 * n_add / (ce[0].elapsed_time(ce[1]) * 1e-3) / 1e9
    del src, dst, flush_buf, flush_rd

    value = (comp_b + agg_b) / (step_avg * 1e-3) / 1e9
    comp_med, agg_med = pct(comp_ms, 0.5), pct(agg_ms, 0.5)
    achieved = dom["bytes"] / (dom["ms_avg"] * 1e-3) / 1e9
    traffic = counted_traffic(dom_kernel, wl.slug)
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(step_avg, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16+f32" if wl.grad_dtype == "float16" else "f32",
        "data": "synthetic",
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "config": {"workload": wl.name, "kind": kind, "tensors": wl.T, "elements": wl.n_total,
                   "ratio": wl.ratio if kind not in WORD_KINDS else None, "W": wl.W,
                   "payload_bytes_per_worker": pay_b, "bytes_per_step": comp_b + agg_b},
        "timing": {"cache_flush_gib": 0 if args.no_flush else 1,
                   "step_ms_p10_p50_p90": [round(pct(step_ms, q), 4) for q in (0.1, 0.5, 0.9)],
                   "wall_ms_per_step_incl_flush": round(wall_s * 1e3, 4)},
        "ops": {"reps": R,
                "compress_ms_p10_p50_p90": [round(pct(comp_ms, q), 4) for q in (0.1, 0.5, 0.9)],
                "compress_gbs": round(comp_b / (comp_med * 1e-3) / 1e9, 1),
                "compress_pct_peak": round(100 * comp_b / (comp_med * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
                "aggregate_ms_p10_p50_p90": [round(pct(agg_ms, q), 4) for q in (0.1, 0.5, 0.9)],
                "aggregate_gbs": round(agg_b / (agg_med * 1e-3) / 1e9, 1),
                "aggregate_pct_peak": round(100 * agg_b / (agg_med * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
                "kernels_ms_avg": {k: round(v["ms_avg"], 4) for k, v in kstats.items()}},
        "copy_gbs_reference": round(copy_gbs, 1),
        "add_gbs_reference": round(add_gbs, 1),
        "add_reference_elements": n_add,
        "roofline": {"bound": "hbm", "kernel": dom_kernel, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": dom["bytes"], "kernel_ms": round(dom["ms_avg"], 4)},
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one core and all cores)")
        line["cpu_baseline"] = cpu_baseline(wl, off, args.cpu_budget)
    print(json.dumps(line), flush=True)


def divisible(args, wl, off, payloads, ws_unused, dev, stream):
    """Node 0's step of the divisible scheme (paper Sec. 3.1, Reason #2):
    the W senders each pack their part 0 (bytecomp_pack_part), node 0
    aggregates the W parts (bytecomp_aggregate_part) and compresses the
    aggregate again without error feedback (bytecomp_compress).  Parts are
    P near-equal word-aligned element ranges of every tensor.

    Algorithmic bytes: each pack reads and writes its part's entries (or
    words); the aggregate reads the W parts and writes the dense fp32
    slices; the second compression reads the slices and writes their
    payload."""
    import torch
    from paper_2205_14465_amd import binding as B
    from paper_2205_14465_amd import workloads as WL
    kind, W, P = wl.kind, wl.W, args.parts
    bounds = []
    for n in wl.sizes:
        b = [0] + [min(n, (q * n // P) // 32 * 32) for q in range(1, P)] + [n]
        bounds.append(b)
    lens = [b[1] - b[0] for b in bounds]
    parts = [B.alloc_payload(kind, wl.ratio, wl.sizes, device=dev) for _ in range(W)]
    offs = [torch.zeros(wl.T + 1, dtype=torch.int64, device=dev) for _ in range(W)]
    slice_flat = torch.empty(sum((n + 63) // 64 * 64 for n in lens) + 64, dtype=torch.float32, device=dev)
    slices, pos = [], 0
    for n in lens:
        slices.append(slice_flat[pos:pos + n])
        pos += (n + 63) // 64 * 64
    sec = B.alloc_payload(kind, wl.ratio, lens, device=dev)
    ws_agg = B.alloc_workspace(kind, wl.ratio, lens, W, device=dev)
    ws_cmp = B.alloc_workspace(kind, wl.ratio, lens, 1, device=dev)
    alpha = 1.0 / W

    packs = [B.PackPartCall(kind, wl.ratio, wl.sizes, payloads[w], bounds, 0, parts[w], offs[w], stream=stream)
             for w in range(W)]
    agg_call = B.AggregatePartCall(kind, wl.ratio, parts, None if kind in WORD_KINDS else offs, lens, slices, alpha,
                                   ws_agg, stream=stream)
    cmp_call = B.CompressCall(kind, wl.ratio, slices, None, sec, ws_cmp, stream=stream)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        for pk in packs:
            pk()
        if ev is not None:
            ev[1].record(stream)
        agg_call()
        if ev is not None:
            ev[2].record(stream)
        cmp_call(WL.SEED)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # bytes actually present in each part
    if kind in WORD_KINDS:
        part_units = [int(o[-1].item()) for o in offs]
        part_bytes = [4 * u + 4 * wl.T for u in part_units]
        sec_off = B.bytecomp_layout(kind, wl.ratio, lens)
        sec_bytes = 4 * int(sec_off[-1]) + 4 * wl.T
    else:
        part_units = [int(o[-1].item()) for o in offs]
        part_bytes = [8 * u for u in part_units]
        sec_off = B.bytecomp_layout(kind, wl.ratio, lens)
        sec_bytes = 8 * int(sec_off[-1])
    n_slice = sum(lens)
    pack_b = 2 * sum(part_bytes)
    agg_b = sum(part_bytes) + 4 * n_slice
    cmp_b = 4 * n_slice + sec_bytes
    reps = args.steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        step()
    torch.cuda.synchronize()
    step_s = (time.perf_counter() - t0) / reps
    dom_kernel = {"sign": "aggregate_sign", "terngrad": "aggregate_quant", "qsgd4": "aggregate_quant",
                  "qsgd8": "aggregate_quant"}.get(kind, "aggregate_sparse")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(reps)]
    for r in range(reps):
        for e in ev[r][4:]:
            e.record(stream)
    torch.cuda.synchronize()
    for r in range(reps):
        B.bytecomp_time_next_launch(dom_kernel, ev[r][4], ev[r][5])
        step(ev[r])
    torch.cuda.synchronize()
    B.bytecomp_time_next_launch(None, None, None)
    pack_ms = sum(ev[r][0].elapsed_time(ev[r][1]) for r in range(reps)) / reps
    agg_ms = sum(ev[r][1].elapsed_time(ev[r][2]) for r in range(reps)) / reps
    cmp_ms = sum(ev[r][2].elapsed_time(ev[r][3]) for r in range(reps)) / reps
    dom_ms = sum(ev[r][4].elapsed_time(ev[r][5]) for r in range(reps)) / reps
    assert B.bytecomp_device_status(ws_agg) == 0
    value = (pack_b + agg_b + cmp_b) / step_s / 1e9
    achieved = agg_b / (dom_ms * 1e-3) / 1e9
    line = {
        "metric": METRIC + " (divisible scheme, node 0's step)",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": reps, "warmup": args.warmup,
        "ms_per_step": round(step_s * 1e3, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic", "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "config": {"workload": wl.name, "kind": kind, "tensors": wl.T, "elements": wl.n_total, "W": W,
                   "parts": P, "part_elements": n_slice},
        "ops": {"pack_ms": round(pack_ms, 4), "pack_calls": W, "pack_gbs": round(pack_b / (pack_ms * 1e-3) / 1e9, 1),
                "aggregate_part_ms": round(agg_ms, 4),
                "aggregate_part_gbs": round(agg_b / (agg_ms * 1e-3) / 1e9, 1),
                "recompress_ms": round(cmp_ms, 4), "recompress_gbs": round(cmp_b / (cmp_ms * 1e-3) / 1e9, 1)},
        "roofline": {"bound": "hbm", "kernel": dom_kernel, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel_ms": round(dom_ms, 4)},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
