"""Shared helpers of the GPU tests: move numpy inputs to the device, run the
library through its C ABI (via the ctypes binding), bring results back, and
compare them with the oracle under the stated tolerances."""
import numpy as np

f32 = np.float32


def bits(x):
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def torch_dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def to_np_u32(t):
    return t.cpu().numpy().view(np.uint32)


WORD_KINDS = ("sign", "terngrad", "qsgd4", "qsgd8")  # packed words + scales


def gpu_compress(kind, ratio, seed, grads, resids, tensor_ids=None, ws_fill=None):
    """Returns (payload dict of numpy arrays, list of new residuals or None).
    ws_fill: byte that fills the workspace past its (initialised) header,
    as an earlier call of another kind sharing it might have left it."""
    import torch
    from paper_2205_14465_amd import binding as B
    ns = [g.size for g in grads]
    dg = [torch_dev(g) for g in grads]
    de = None if resids is None else [torch_dev(np.asarray(e, np.float32)) for e in resids]
    out = B.alloc_payload(kind, ratio, ns)
    ws = B.alloc_workspace(kind, ratio, ns, 1)
    if ws_fill is not None:
        B.bytecomp_workspace_init(ws)
        ws[256:].fill_(ws_fill)
    B.bytecomp_compress(kind, ratio, seed, dg, de, out, ws, tensor_ids=tensor_ids)
    torch.cuda.synchronize()
    assert B.bytecomp_device_status(ws) == 0
    res = {"off": np.array(out["off"], dtype=np.int64)}
    total = out["off"][-1]
    if kind in WORD_KINDS:
        res["bits"] = to_np_u32(out["bits"])[:total]
        res["scale"] = out["scale"].cpu().numpy()[:len(ns)]
    else:
        res["idx"] = to_np_u32(out["idx"])[:total]
        res["val"] = out["val"].cpu().numpy()[:total]
    new_e = None if de is None else [e.cpu().numpy() for e in de]
    return res, new_e


def gpu_aggregate(kind, ratio, ns, payloads, alpha, ws_fill=None):
    """payloads: list of dicts with numpy 'idx','val' or 'bits','scale'.
    ws_fill: as for gpu_compress."""
    import torch
    from paper_2205_14465_amd import binding as B
    dev = []
    for p in payloads:
        if kind in WORD_KINDS:
            dev.append({"bits": torch_dev(p["bits"].view(np.int32)), "scale": torch_dev(p["scale"])})
        else:
            dev.append({"idx": torch_dev(p["idx"].view(np.int32)), "val": torch_dev(p["val"])})
    outs = [torch.full((max(n, 1),), float("nan"), dtype=torch.float32, device="cuda") for n in ns]
    outs = [o[:n] if n else o[:0] for o, n in zip(outs, ns)]
    ws = B.alloc_workspace(kind, ratio, ns, len(payloads))
    if ws_fill is not None:
        B.bytecomp_workspace_init(ws)
        ws[256:].fill_(ws_fill)
    B.bytecomp_decompress_aggregate(kind, ratio, dev, ns, outs, alpha, ws)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs]


def assert_sparse_equal(got, want, ns):
    assert np.array_equal(got["off"], want["off"])
    assert np.array_equal(got["idx"], want["idx"]), _first_diff(got["idx"], want["idx"])
    assert np.array_equal(bits(got["val"]), bits(want["val"])), _first_diff(bits(got["val"]), bits(want["val"]))


def assert_resid_equal(got, want):
    for t, (a, b) in enumerate(zip(got, want)):
        assert np.array_equal(bits(a), bits(b)), (t, _first_diff(bits(a), bits(b)))


def sign_tolerances(grads):
    return [1e-3 if g.dtype == np.float16 else 1e-6 for g in grads]


def assert_sign_close(got, want, grads, resids_in, got_e, want_e):
    """Bits exact; scales within the relative tolerance (1e-6 fp32 input,
    1e-3 fp16 input); residuals bit-exact where the scales agree exactly,
    else |delta| <= tol * (|v| + s)."""
    assert np.array_equal(got["off"], want["off"])
    assert np.array_equal(got["bits"], want["bits"]), _first_diff(got["bits"], want["bits"])
    tols = sign_tolerances(grads)
    gs, ws_ = got["scale"], want["scale"]
    for t in range(len(grads)):
        tol = tols[t]
        assert abs(float(gs[t]) - float(ws_[t])) <= tol * abs(float(ws_[t])), (t, gs[t], ws_[t])
    if got_e is None:
        return
    for t in range(len(grads)):
        a, b = got_e[t], want_e[t]
        if gs[t] == ws_[t]:
            assert np.array_equal(bits(a), bits(b)), (t, _first_diff(bits(a), bits(b)))
        else:
            v = grads[t].astype(np.float32) + (0 if resids_in is None else resids_in[t])
            lim = tols[t] * (np.abs(v).astype(np.float64) + float(ws_[t]))
            assert np.all(np.abs(a.astype(np.float64) - b.astype(np.float64)) <= lim), t


def _first_diff(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    if a.shape != b.shape:
        return f"shape {a.shape} vs {b.shape}"
    d = np.nonzero(a != b)[0]
    if d.size == 0:
        return "equal"
    i = int(d[0])
    return f"{d.size} differ; first at {i}: {a[i]!r} vs {b[i]!r}"
