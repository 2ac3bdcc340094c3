"""Thin ctypes binding of libbytecomp.so (the C ABI in include/bytecomp.h).

Argument marshalling only: every step of the compression path runs in the
gfx950 kernels of the library.  PyTorch supplies device memory and streams.
The library must have been built in-tree (paper_2205_14465_amd/build.py);
importing this module without it raises, so a missing extension fails
loudly instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbytecomp.so")

BC_TOPK, BC_TOPK_SAMPLED, BC_RANDK, BC_SIGN1 = 0, 1, 2, 3
BC_TERNGRAD, BC_QSGD4, BC_QSGD8 = 4, 5, 6
BC_F32, BC_F16 = 0, 1
KIND = {"topk": BC_TOPK, "topk_sampled": BC_TOPK_SAMPLED, "randk": BC_RANDK, "sign": BC_SIGN1,
        "terngrad": BC_TERNGRAD, "qsgd4": BC_QSGD4, "qsgd8": BC_QSGD8}
# kinds whose payload is packed words plus one scale per tensor
WORD_KINDS = (BC_SIGN1, BC_TERNGRAD, BC_QSGD4, BC_QSGD8)
STATUS = {0: "BC_OK", -1: "BC_E_NULL", -2: "BC_E_KIND", -3: "BC_E_DTYPE", -4: "BC_E_RATIO",
          -5: "BC_E_SIZE", -6: "BC_E_COUNT", -7: "BC_E_WORKSPACE", -8: "BC_E_HIP",
          -9: "BC_E_ALIGN", -10: "BC_E_DEVICE"}


class bc_tensor(ctypes.Structure):
    _fields_ = [("grad", ctypes.c_void_p), ("residual", ctypes.c_void_p), ("n", ctypes.c_uint64),
                ("dtype", ctypes.c_uint32), ("tensor_id", ctypes.c_uint32)]


class bc_payload(ctypes.Structure):
    _fields_ = [("idx", ctypes.c_void_p), ("val", ctypes.c_void_p), ("bits", ctypes.c_void_p),
                ("scale", ctypes.c_void_p)]


class BytecompError(RuntimeError):
    def __init__(self, fn, code):
        self.code = code
        super().__init__(f"{fn} failed: {STATUS.get(code, code)} ({_strerror(code)})")


_lib = None


def lib():
    global _lib
    if _lib is None:
        # PyTorch ships its own copy of the HIP runtime (same soname).  Load
        # it first so that this library binds to the copy torch uses; loading
        # ours first would put two HIP runtimes in the process.
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2205_14465_amd/build.py "
                              "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, u64, i32, dbl, flt, sz = (ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int, ctypes.c_double,
                                      ctypes.c_float, ctypes.c_size_t)
        L.bytecomp_strerror.restype = ctypes.c_char_p
        L.bytecomp_strerror.argtypes = [i32]
        L.bytecomp_layout.restype = i32
        L.bytecomp_layout.argtypes = [i32, dbl, vp, i32, vp]
        L.bytecomp_workspace_size.restype = i32
        L.bytecomp_workspace_size.argtypes = [i32, dbl, vp, i32, i32, ctypes.POINTER(sz)]
        L.bytecomp_workspace_init.restype = i32
        L.bytecomp_workspace_init.argtypes = [vp, sz, vp]
        L.bytecomp_compress.restype = i32
        L.bytecomp_compress.argtypes = [i32, dbl, u64, ctypes.POINTER(bc_tensor), i32, bc_payload, vp,
                                        sz, vp]
        L.bytecomp_compress_noalloc.restype = i32
        L.bytecomp_compress_noalloc.argtypes = [i32, dbl, u64, ctypes.POINTER(bc_tensor), i32, bc_payload, vp]
        L.bytecomp_plan_simulate.restype = i32
        L.bytecomp_plan_simulate.argtypes = [i32, vp, vp, vp, vp, vp, vp]
        L.bytecomp_plan_enumerate.restype = i32
        L.bytecomp_plan_enumerate.argtypes = [i32, vp, vp, vp, vp, vp, i32, vp, vp, u64, dbl, i32, vp, vp, vp]
        L.bytecomp_cpu_compress.restype = i32
        L.bytecomp_cpu_compress.argtypes = [i32, dbl, u64, ctypes.POINTER(bc_tensor), i32, bc_payload, i32]
        L.bytecomp_cpu_decompress_aggregate.restype = i32
        L.bytecomp_cpu_decompress_aggregate.argtypes = [i32, dbl, ctypes.POINTER(bc_payload), i32,
                                                        ctypes.POINTER(ctypes.c_uint64), i32,
                                                        ctypes.POINTER(ctypes.c_void_p), flt, i32]
        L.bytecomp_compress_dgc.restype = i32
        L.bytecomp_compress_dgc.argtypes = [i32, dbl, u64, ctypes.c_float, ctypes.POINTER(bc_tensor), vp, i32,
                                            bc_payload, vp, sz, vp]
        L.bytecomp_compress_dgc_clip.restype = i32
        L.bytecomp_compress_dgc_clip.argtypes = [i32, dbl, u64, ctypes.c_float, dbl, ctypes.POINTER(bc_tensor), vp,
                                                 i32, bc_payload, vp, vp, sz, vp]
        L.bytecomp_decompress_aggregate.restype = i32
        L.bytecomp_decompress_aggregate.argtypes = [i32, dbl, ctypes.POINTER(bc_payload), i32, vp, i32,
                                                    vp, flt, vp, sz, vp]
        L.bytecomp_residual_update.restype = i32
        L.bytecomp_residual_update.argtypes = [i32, dbl, ctypes.POINTER(bc_tensor), i32, bc_payload, vp]
        L.bytecomp_device_status.restype = i32
        L.bytecomp_device_status.argtypes = [vp, sz, vp, ctypes.POINTER(ctypes.c_uint32)]
        L.bytecomp_topk_stats.restype = i32
        L.bytecomp_topk_stats.argtypes = [i32, dbl, vp, i32, vp, sz, vp, ctypes.POINTER(ctypes.c_uint64),
                                          ctypes.POINTER(ctypes.c_uint32)]
        L.bytecomp_pack_part.restype = i32
        L.bytecomp_pack_part.argtypes = [i32, dbl, vp, i32, bc_payload, i32, vp, i32, bc_payload, vp, vp]
        L.bytecomp_aggregate_part.restype = i32
        L.bytecomp_aggregate_part.argtypes = [i32, dbl, ctypes.POINTER(bc_payload), vp, i32, vp, i32, vp,
                                              ctypes.c_float, vp, sz, vp]
        L.bytecomp_time_next_launch.restype = i32
        L.bytecomp_time_next_launch.argtypes = [ctypes.c_char_p, vp, vp]
        L.bytecomp_set_wait_limit.restype = i32
        L.bytecomp_set_wait_limit.argtypes = [ctypes.c_uint32]
        L.bytecomp_set_topk_few_chunks.restype = i32
        L.bytecomp_set_topk_few_chunks.argtypes = [ctypes.c_uint32]
        _lib = L
    return _lib


def _strerror(code):
    try:
        return lib().bytecomp_strerror(code).decode()
    except Exception:
        return "?"


def _check(fn, code):
    if code != 0:
        raise BytecompError(fn, code)


def _kind(kind):
    return KIND[kind] if isinstance(kind, str) else int(kind)


def _u64_array(values):
    arr = (ctypes.c_uint64 * max(len(values), 1))(*[int(v) for v in values])
    return arr


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ------------------------------------------------------------ host-only

def bytecomp_layout(kind, ratio, ns: Sequence[int]):
    off = (ctypes.c_uint64 * (len(ns) + 1))()
    _check("bytecomp_layout", lib().bytecomp_layout(_kind(kind), float(ratio), _u64_array(ns), len(ns), off))
    return [int(x) for x in off]


def bytecomp_workspace_size(kind, ratio, ns: Sequence[int], W: int = 1):
    out = ctypes.c_size_t(0)
    _check("bytecomp_workspace_size",
           lib().bytecomp_workspace_size(_kind(kind), float(ratio), _u64_array(ns), len(ns), int(W),
                                         ctypes.byref(out)))
    return int(out.value)


# --------------------------------------------------------------- device

def _tensor_list(grads, resids, tensor_ids):
    import torch
    T = len(grads)
    arr = (bc_tensor * max(T, 1))()
    for t, g in enumerate(grads):
        e = None if resids is None else resids[t]
        if g.dtype == torch.float32:
            dt = BC_F32
        elif g.dtype == torch.float16:
            dt = BC_F16
        else:
            dt = 99  # rejected by the library with BC_E_DTYPE
        arr[t].grad = g.data_ptr() if g.numel() else None
        arr[t].residual = None if e is None else e.data_ptr()
        arr[t].n = g.numel()
        arr[t].dtype = dt
        arr[t].tensor_id = t if tensor_ids is None else int(tensor_ids[t])
    return arr


def _payload(p):
    if p is None:
        return bc_payload()
    return bc_payload(idx=p.get("idx") is not None and p["idx"].data_ptr() or None,
                      val=p.get("val") is not None and p["val"].data_ptr() or None,
                      bits=p.get("bits") is not None and p["bits"].data_ptr() or None,
                      scale=p.get("scale") is not None and p["scale"].data_ptr() or None)


def bytecomp_workspace_init(ws, stream=None):
    _check("bytecomp_workspace_init",
           lib().bytecomp_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream_handle(stream)))


def bytecomp_compress(kind, ratio, seed, grads, resids, out, ws, stream=None, tensor_ids=None):
    """grads/resids: lists of device tensors (resids None = error feedback off);
    out: payload dict of device tensors ('idx','val' or 'bits','scale');
    ws: device uint8 tensor of at least bytecomp_workspace_size bytes."""
    arr = _tensor_list(grads, resids, tensor_ids)
    _check("bytecomp_compress",
           lib().bytecomp_compress(_kind(kind), float(ratio), int(seed) & (2**64 - 1), arr, len(grads),
                                   _payload(out), _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream_handle(stream)))


def bytecomp_compress_noalloc(kind, ratio, seed, grads, resids, out, stream=None, tensor_ids=None):
    """bytecomp_compress without a workspace: the library's own per-GPU
    device array serves as workspace and descriptor table (no allocation)."""
    arr = _tensor_list(grads, resids, tensor_ids)
    _check("bytecomp_compress_noalloc",
           lib().bytecomp_compress_noalloc(_kind(kind), float(ratio), int(seed) & (2**64 - 1), arr, len(grads),
                                           _payload(out), _stream_handle(stream)))


# ------------------------------------------------------------- CPU side
# The host operators (CPU offloading): numpy arrays in host memory.

def _np_tensor_list(grads, resids, tensor_ids):
    import numpy as np
    T = len(grads)
    arr = (bc_tensor * max(T, 1))()
    for t, g in enumerate(grads):
        e = None if resids is None else resids[t]
        assert g.flags.c_contiguous and (e is None or (e.flags.c_contiguous and e.dtype == np.float32))
        arr[t].grad = g.ctypes.data if g.size else None
        arr[t].residual = None if e is None else e.ctypes.data
        arr[t].n = g.size
        arr[t].dtype = BC_F32 if g.dtype == np.float32 else BC_F16 if g.dtype == np.float16 else 99
        arr[t].tensor_id = t if tensor_ids is None else int(tensor_ids[t])
    return arr


def _np_payload(p):
    def ptr(key):
        a = p.get(key)
        return a.ctypes.data if a is not None and a.size else None
    return bc_payload(idx=ptr("idx"), val=ptr("val"), bits=ptr("bits"), scale=ptr("scale"))


def cpu_alloc_payload(kind, ratio, ns):
    """Host payload arrays (numpy) laid out as bytecomp_layout describes."""
    import numpy as np
    off = bytecomp_layout(kind, ratio, ns)
    total = off[-1]
    if _kind(kind) in (KIND["sign"], KIND["terngrad"], KIND["qsgd4"], KIND["qsgd8"]):
        return {"bits": np.zeros(max(total, 1), np.uint32), "scale": np.zeros(max(len(ns), 1), np.float32),
                "off": off}
    return {"idx": np.zeros(max(total, 1), np.uint32), "val": np.zeros(max(total, 1), np.float32), "off": off}


class CpuCompressCall:
    """bytecomp_cpu_compress with its arguments marshalled once."""

    def __init__(self, kind, ratio, grads, resids, out, threads=0, tensor_ids=None):
        self.kind, self.ratio, self.T, self.threads = _kind(kind), float(ratio), len(grads), int(threads)
        self.arr = _np_tensor_list(grads, resids, tensor_ids)
        self.out = _np_payload(out)
        self._keep = (grads, resids, out)

    def __call__(self, seed):
        _check("bytecomp_cpu_compress",
               lib().bytecomp_cpu_compress(self.kind, self.ratio, int(seed) & (2**64 - 1), self.arr, self.T,
                                           self.out, self.threads))


class CpuAggregateCall:
    """bytecomp_cpu_decompress_aggregate with its arguments marshalled once."""

    def __init__(self, kind, ratio, payloads, ns, outs, alpha, threads=0):
        self.kind, self.ratio, self.alpha, self.threads = _kind(kind), float(ratio), float(alpha), int(threads)
        self.W, self.T = len(payloads), len(ns)
        self.pa = (bc_payload * max(self.W, 1))(*[_np_payload(p) for p in payloads])
        self.ns = _u64_array(ns)
        self.op = (ctypes.c_void_p * max(self.T, 1))(*[o.ctypes.data if o.size else None for o in outs])
        self._keep = (payloads, outs)

    def __call__(self):
        _check("bytecomp_cpu_decompress_aggregate",
               lib().bytecomp_cpu_decompress_aggregate(self.kind, self.ratio, self.pa, self.W, self.ns, self.T,
                                                       self.op, self.alpha, self.threads))


def bytecomp_cpu_compress(kind, ratio, seed, grads, resids, out, threads=0, tensor_ids=None):
    """Host compression: grads/resids numpy arrays (resids updated in place,
    None = error feedback off); out from cpu_alloc_payload."""
    CpuCompressCall(kind, ratio, grads, resids, out, threads, tensor_ids)(seed)


def bytecomp_cpu_decompress_aggregate(kind, ratio, payloads, ns, outs, alpha, threads=0):
    """Host decompress-and-aggregate of W numpy payloads into numpy outputs."""
    CpuAggregateCall(kind, ratio, payloads, ns, outs, alpha, threads)()


def bytecomp_decompress_aggregate(kind, ratio, payloads, ns, outs, alpha, ws, stream=None):
    W = len(payloads)
    pa = (bc_payload * max(W, 1))(*[_payload(p) for p in payloads])
    T = len(ns)
    op = (ctypes.c_void_p * max(T, 1))(*[o.data_ptr() if o.numel() else None for o in outs])
    _check("bytecomp_decompress_aggregate",
           lib().bytecomp_decompress_aggregate(_kind(kind), float(ratio), pa, W, _u64_array(ns), T, op,
                                               float(alpha), _ptr(ws), ws.numel() * ws.element_size(),
                                               _stream_handle(stream)))


def bytecomp_residual_update(kind, ratio, grads, resids, own, stream=None, tensor_ids=None):
    arr = _tensor_list(grads, resids, tensor_ids)
    _check("bytecomp_residual_update",
           lib().bytecomp_residual_update(_kind(kind), float(ratio), arr, len(grads), _payload(own),
                                          _stream_handle(stream)))


def bytecomp_pack_part(kind, ratio, ns, payload, bounds, j, out, part_off, stream=None):
    """Pack part j of `payload` into `out` (a payload dict sized like the
    input); bounds is a list of per-tensor boundary lists (parts + 1 each);
    part_off a device uint64 (int64) tensor of T + 1 entries."""
    T = len(ns)
    parts = len(bounds[0]) - 1 if T else 1
    flat = _u64_array([int(x) for b in bounds for x in b])
    _check("bytecomp_pack_part",
           lib().bytecomp_pack_part(_kind(kind), float(ratio), _u64_array(ns), T, _payload(payload), parts,
                                    flat, int(j), _payload(out), _ptr(part_off), _stream_handle(stream)))


def bytecomp_aggregate_part(kind, ratio, parts, part_offs, lens, outs, alpha, ws, stream=None):
    """Aggregate W packed parts (payload dicts from bytecomp_pack_part, with
    their part_off tensors) into dense slices `outs` of lengths `lens`."""
    W = len(parts)
    T = len(lens)
    pa = (bc_payload * W)(*[_payload(p) for p in parts])
    po = (ctypes.c_void_p * W)(*[_ptr(x) for x in part_offs]) if part_offs is not None else None
    op = (ctypes.c_void_p * max(T, 1))(*[_ptr(o) for o in outs])
    _check("bytecomp_aggregate_part",
           lib().bytecomp_aggregate_part(_kind(kind), float(ratio), pa, po, W, _u64_array(lens), T, op,
                                         float(alpha), _ptr(ws), ws.numel() * ws.element_size(),
                                         _stream_handle(stream)))


def bytecomp_time_next_launch(kernel, start_event, stop_event):
    """Have the next launch of `kernel` bracketed by two torch.cuda.Event
    objects (recorded once before, so that their HIP events exist); None
    for both clears a pending request and returns True if one was pending
    (the kernel did not run since the request)."""
    if start_event is None and stop_event is None:
        rc = lib().bytecomp_time_next_launch(None, None, None)
        if rc < 0:
            _check("bytecomp_time_next_launch", rc)
        return rc == 1
    _check("bytecomp_time_next_launch",
           lib().bytecomp_time_next_launch(kernel.encode(), ctypes.c_void_p(start_event.cuda_event),
                                           ctypes.c_void_p(stop_event.cuda_event)))


def bytecomp_set_wait_limit(microseconds):
    """How long a one-pass compress workgroup waits for the rest of its
    tensor's chunk partials before it computes the missing ones itself
    (process-wide; default 200)."""
    _check("bytecomp_set_wait_limit", lib().bytecomp_set_wait_limit(int(microseconds)))


def bytecomp_set_topk_few_chunks(chunks):
    """Top-k calls of at most `chunks` chunks take the few-chunk path
    (default and maximum 2048; 0: always the general pipeline)."""
    _check("bytecomp_set_topk_few_chunks", lib().bytecomp_set_topk_few_chunks(int(chunks)))


def bytecomp_device_status(ws, stream=None):
    f = ctypes.c_uint32(0)
    _check("bytecomp_device_status",
           lib().bytecomp_device_status(_ptr(ws), ws.numel() * ws.element_size(), _stream_handle(stream),
                                        ctypes.byref(f)))
    return int(f.value)


def bytecomp_topk_stats(kind, ratio, sizes, ws, stream=None):
    """(candidates, fallbacks) of the last top-k compress call of this shape
    on the workspace ws (a device tensor, or None for calls of empty
    tensors only)."""
    n = (ctypes.c_uint64 * max(len(sizes), 1))(*[int(x) for x in sizes])
    cand = ctypes.c_uint64(0)
    fb = ctypes.c_uint32(0)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("bytecomp_topk_stats",
           lib().bytecomp_topk_stats(_kind(kind), float(ratio), n, len(sizes), _ptr(ws), ws_bytes,
                                     _stream_handle(stream), ctypes.byref(cand), ctypes.byref(fb)))
    return int(cand.value), int(fb.value)


# ---------------------------------------------------------- prepared calls
# For tensor lists that stay the same across iterations (a model's
# gradients), the ctypes argument arrays are built once; a call then costs
# one foreign-function call.

class CompressCall:
    def __init__(self, kind, ratio, grads, resids, out, ws, stream=None, tensor_ids=None):
        self.kind = _kind(kind)
        self.ratio = float(ratio)
        self.T = len(grads)
        self.arr = _tensor_list(grads, resids, tensor_ids)
        self.out = _payload(out)
        self.ws = _ptr(ws)
        self.ws_bytes = ws.numel() * ws.element_size()
        self.stream = _stream_handle(stream)
        self._keep = (grads, resids, out, ws)

    def __call__(self, seed):
        _check("bytecomp_compress",
               lib().bytecomp_compress(self.kind, self.ratio, int(seed) & (2**64 - 1), self.arr, self.T,
                                       self.out, self.ws, self.ws_bytes, self.stream))


class DgcCall:
    """bytecomp_compress_dgc with its argument arrays marshalled once:
    velocities is a list of fp32 device tensors, one per gradient.  With
    clip_norm (not None) the call is bytecomp_compress_dgc_clip, and
    clip_factor (a one-element fp32 device tensor, or None) receives the
    clipping factor."""

    def __init__(self, kind, ratio, momentum, grads, resids, velocities, out, ws, stream=None, tensor_ids=None,
                 clip_norm=None, clip_factor=None):
        self.kind = _kind(kind)
        self.ratio = float(ratio)
        self.momentum = float(momentum)
        self.clip_norm = None if clip_norm is None else float(clip_norm)
        self.clip_factor = _ptr(clip_factor)
        self.T = len(grads)
        self.arr = _tensor_list(grads, resids, tensor_ids)
        self.vel = (ctypes.c_void_p * max(self.T, 1))(*[v.data_ptr() if v.numel() else None for v in velocities])
        self.out = _payload(out)
        self.ws = _ptr(ws)
        self.ws_bytes = ws.numel() * ws.element_size()
        self.stream = _stream_handle(stream)
        self._keep = (grads, resids, velocities, out, ws, clip_factor)

    def __call__(self, seed):
        if self.clip_norm is None:
            _check("bytecomp_compress_dgc",
                   lib().bytecomp_compress_dgc(self.kind, self.ratio, int(seed) & (2**64 - 1), self.momentum,
                                               self.arr, self.vel, self.T, self.out, self.ws, self.ws_bytes,
                                               self.stream))
        else:
            _check("bytecomp_compress_dgc_clip",
                   lib().bytecomp_compress_dgc_clip(self.kind, self.ratio, int(seed) & (2**64 - 1), self.momentum,
                                                    self.clip_norm, self.arr, self.vel, self.T, self.out,
                                                    self.clip_factor, self.ws, self.ws_bytes, self.stream))


def bytecomp_compress_dgc(kind, ratio, seed, momentum, grads, resids, velocities, out, ws, stream=None,
                          tensor_ids=None):
    """One DGC step: velocities (fp32 device tensors) and resids are updated in place."""
    DgcCall(kind, ratio, momentum, grads, resids, velocities, out, ws, stream, tensor_ids)(seed)


def bytecomp_compress_dgc_clip(kind, ratio, seed, momentum, clip_norm, grads, resids, velocities, out, ws,
                               clip_factor=None, stream=None, tensor_ids=None):
    """One DGC step with local gradient clipping at clip_norm; clip_factor:
    a one-element fp32 device tensor that receives the factor, or None."""
    DgcCall(kind, ratio, momentum, grads, resids, velocities, out, ws, stream, tensor_ids, clip_norm=clip_norm,
            clip_factor=clip_factor)(seed)


class AggregateCall:
    def __init__(self, kind, ratio, payloads, ns, outs, alpha, ws, stream=None):
        self.kind = _kind(kind)
        self.ratio = float(ratio)
        self.W = len(payloads)
        self.pa = (bc_payload * max(self.W, 1))(*[_payload(p) for p in payloads])
        self.T = len(ns)
        self.ns = _u64_array(ns)
        self.op = (ctypes.c_void_p * max(self.T, 1))(*[o.data_ptr() if o.numel() else None for o in outs])
        self.alpha = float(alpha)
        self.ws = _ptr(ws)
        self.ws_bytes = ws.numel() * ws.element_size()
        self.stream = _stream_handle(stream)
        self._keep = (payloads, outs, ws)

    def __call__(self):
        _check("bytecomp_decompress_aggregate",
               lib().bytecomp_decompress_aggregate(self.kind, self.ratio, self.pa, self.W, self.ns, self.T,
                                                   self.op, self.alpha, self.ws, self.ws_bytes, self.stream))


class PackPartCall:
    """bytecomp_pack_part with its argument arrays marshalled once."""

    def __init__(self, kind, ratio, ns, payload, bounds, j, out, part_off, stream=None):
        self.kind = _kind(kind)
        self.ratio = float(ratio)
        self.T = len(ns)
        self.ns = _u64_array(ns)
        self.parts = len(bounds[0]) - 1 if self.T else 1
        self.flat = _u64_array([int(x) for b in bounds for x in b])
        self.j = int(j)
        self.inp = _payload(payload)
        self.out = _payload(out)
        self.po = _ptr(part_off)
        self.stream = _stream_handle(stream)
        self._keep = (payload, out, part_off)

    def __call__(self):
        _check("bytecomp_pack_part",
               lib().bytecomp_pack_part(self.kind, self.ratio, self.ns, self.T, self.inp, self.parts, self.flat,
                                        self.j, self.out, self.po, self.stream))


class AggregatePartCall:
    """bytecomp_aggregate_part with its argument arrays marshalled once."""

    def __init__(self, kind, ratio, parts, part_offs, lens, outs, alpha, ws, stream=None):
        self.kind = _kind(kind)
        self.ratio = float(ratio)
        self.W = len(parts)
        self.pa = (bc_payload * max(self.W, 1))(*[_payload(p) for p in parts])
        self.po = (ctypes.c_void_p * self.W)(*[x.data_ptr() for x in part_offs]) if part_offs is not None else None
        self.T = len(lens)
        self.lens = _u64_array(lens)
        self.op = (ctypes.c_void_p * max(self.T, 1))(*[o.data_ptr() if o.numel() else None for o in outs])
        self.alpha = float(alpha)
        self.ws = _ptr(ws)
        self.ws_bytes = ws.numel() * ws.element_size()
        self.stream = _stream_handle(stream)
        self._keep = (parts, part_offs, outs, ws)

    def __call__(self):
        _check("bytecomp_aggregate_part",
               lib().bytecomp_aggregate_part(self.kind, self.ratio, self.pa, self.po, self.W, self.lens, self.T,
                                             self.op, self.alpha, self.ws, self.ws_bytes, self.stream))


# ------------------------------------------------------------ allocation

def alloc_payload(kind, ratio, ns, device="cuda"):
    """Device buffers for one worker's payload of the given tensor list."""
    import torch
    off = bytecomp_layout(kind, ratio, ns)
    total = off[-1]
    if _kind(kind) in WORD_KINDS:
        return {"bits": torch.zeros(max(total, 1), dtype=torch.int32, device=device),
                "scale": torch.zeros(max(len(ns), 1), dtype=torch.float32, device=device), "off": off}
    return {"idx": torch.zeros(max(total, 1), dtype=torch.int32, device=device),
            "val": torch.zeros(max(total, 1), dtype=torch.float32, device=device), "off": off}


def alloc_workspace(kind, ratio, ns, W=1, device="cuda"):
    import torch
    return torch.zeros(bytecomp_workspace_size(kind, ratio, ns, W), dtype=torch.uint8, device=device)
