"""ctypes front end of the CPU oracle (test infrastructure only).

Only tests/, the smoke check and the benchmark's CPU-baseline leg import
this package.  It wraps the plain C oracle in bytecomp_oracle.c one tensor
at a time and, for tensor lists, loops over tensors in Python and lays the
payloads out back to back: sparse payloads at offsets that are prefix sums
of the per-tensor k, sign payloads at prefix sums of the per-tensor word
counts, one scale per tensor.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

F32, F16 = 0, 1
_DT = {np.dtype(np.float32): F32, np.dtype(np.float16): F16}

_u64 = ctypes.c_uint64
_u32 = ctypes.c_uint32
_vp = ctypes.c_void_p
_dbl = ctypes.c_double
_int = ctypes.c_int
_flt = ctypes.c_float


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        L.bco_k.restype = _u64
        L.bco_k.argtypes = [_u64, _dbl]
        L.bco_words.restype = _u64
        L.bco_words.argtypes = [_u64]
        L.bco_f16_to_f32.restype = _flt
        L.bco_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.bco_compress_topk.restype = _int
        L.bco_compress_topk.argtypes = [_vp, _int, _vp, _u64, _u64, _vp, _vp, _vp]
        L.bco_compress_topk_sampled.restype = _int
        L.bco_compress_topk_sampled.argtypes = [_vp, _int, _vp, _u64, _u64, _dbl, _u64, _u32,
                                                _vp, _vp, _vp, _vp]
        L.bco_compress_randk.restype = _int
        L.bco_compress_randk.argtypes = [_vp, _int, _vp, _u64, _u64, _u64, _u32, _vp, _vp, _vp]
        L.bco_compress_sign.restype = _int
        L.bco_compress_sign.argtypes = [_vp, _int, _vp, _u64, _vp, _vp, _vp]
        L.bco_residual_update_sparse.restype = _int
        L.bco_residual_update_sparse.argtypes = [_vp, _int, _vp, _u64, _u64, _vp, _vp]
        L.bco_residual_update_sign.restype = _int
        L.bco_residual_update_sign.argtypes = [_vp, _int, _vp, _u64, _vp, _flt]
        L.bco_aggregate_sparse.restype = _int
        L.bco_aggregate_sparse.argtypes = [_int, _u64, _vp, _vp, _vp, _flt, _vp]
        L.bco_aggregate_sign.restype = _int
        L.bco_aggregate_sign.argtypes = [_int, _u64, _vp, _vp, _flt, _vp]
        L.bco_aggregate_sign_ordered.restype = _int
        L.bco_aggregate_sign_ordered.argtypes = [_int, _u64, _vp, _vp, _flt, _vp]
        L.bco_exact_sum_f32.restype = _flt
        L.bco_exact_sum_f32.argtypes = [_vp, _u64]
        L.bco_philox4x64_10.restype = None
        L.bco_philox4x64_10.argtypes = [_vp, _vp, _vp]
        L.bco_feistel_half_bits.restype = _u32
        L.bco_feistel_half_bits.argtypes = [_u64]
        L.bco_randk_round_keys.restype = None
        L.bco_randk_round_keys.argtypes = [_u64, _u32, _vp]
        L.bco_feistel_encrypt.restype = _u64
        L.bco_feistel_encrypt.argtypes = [_u64, _u32, _vp]
        L.bco_randk_index.restype = _u64
        L.bco_randk_index.argtypes = [_u64, _u64, _u32, _u64]
        L.bco_sample_size.restype = _u64
        L.bco_sample_size.argtypes = [_u64]
        L.bco_quant_levels.restype = _int
        L.bco_quant_levels.argtypes = [_int]
        L.bco_quant_words.restype = _u64
        L.bco_quant_words.argtypes = [_u64, _int]
        L.bco_quant_uniform.restype = _flt
        L.bco_quant_uniform.argtypes = [_u64, _u32, _u64]
        L.bco_quant_decode.restype = _flt
        L.bco_quant_decode.argtypes = [_u32, _int, _flt]
        L.bco_compress_quant.restype = _int
        L.bco_compress_quant.argtypes = [_vp, _int, _vp, _u64, _int, _u64, _u32, _vp, _vp, _vp]
        L.bco_residual_update_quant.restype = _int
        L.bco_residual_update_quant.argtypes = [_vp, _int, _vp, _u64, _int, _vp, _flt]
        L.bco_dgc_momentum.restype = _int
        L.bco_dgc_momentum.argtypes = [_vp, _int, _vp, _u64, _flt]
        L.bco_dgc_clip_factor.restype = ctypes.c_float
        L.bco_dgc_clip_factor.argtypes = [_int, _vp, _vp, _vp, _dbl]
        L.bco_dgc_momentum_clipped.restype = _int
        L.bco_dgc_momentum_clipped.argtypes = [_vp, _int, _vp, _u64, _flt, _flt]
        L.bco_aggregate_quant.restype = _int
        L.bco_aggregate_quant.argtypes = [_int, _u64, _int, _vp, _vp, _flt, _vp]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


# ---------------------------------------------------------------- sizes

def k_for(n, ratio):
    return int(lib().bco_k(int(n), float(ratio)))


def words_for(n):
    return int(lib().bco_words(int(n)))


def sparse_offsets(ns, ratio):
    off = np.zeros(len(ns) + 1, dtype=np.int64)
    for t, n in enumerate(ns):
        off[t + 1] = off[t] + k_for(n, ratio)
    return off


def word_offsets(ns):
    off = np.zeros(len(ns) + 1, dtype=np.int64)
    for t, n in enumerate(ns):
        off[t + 1] = off[t] + words_for(n)
    return off


# ------------------------------------------------------- per-tensor calls

def f16_to_f32(h):
    return lib().bco_f16_to_f32(int(h))


def _grad(g):
    g = np.ascontiguousarray(g)
    if g.dtype not in _DT:
        raise TypeError("gradient dtype must be float32 or float16")
    return g, _DT[g.dtype]


def _resid(e, n):
    if e is None:
        return None
    e = np.ascontiguousarray(e, dtype=np.float32)
    assert e.size == n
    return e


def compress_topk(g, e, ratio):
    g, dt = _grad(g)
    n = g.size
    e = _resid(e, n)
    k = k_for(n, ratio)
    idx = np.empty(k, np.uint32)
    val = np.empty(k, np.float32)
    e_out = np.empty(n, np.float32) if e is not None else None
    rc = lib().bco_compress_topk(_p(g), dt, _p(e), n, k, _p(idx), _p(val), _p(e_out))
    assert rc == 0, rc
    return idx, val, e_out


def compress_topk_sampled(g, e, ratio, seed, tensor_id, want_candidates=False):
    g, dt = _grad(g)
    n = g.size
    e = _resid(e, n)
    k = k_for(n, ratio)
    idx = np.empty(k, np.uint32)
    val = np.empty(k, np.float32)
    e_out = np.empty(n, np.float32) if e is not None else None
    nc = np.zeros(1, np.uint64)
    rc = lib().bco_compress_topk_sampled(_p(g), dt, _p(e), n, k, float(ratio), int(seed),
                                         int(tensor_id), _p(idx), _p(val), _p(e_out), _p(nc))
    assert rc == 0, rc
    if want_candidates:
        return idx, val, e_out, int(nc[0])
    return idx, val, e_out


def compress_randk(g, e, ratio, seed, tensor_id):
    g, dt = _grad(g)
    n = g.size
    e = _resid(e, n)
    k = k_for(n, ratio)
    idx = np.empty(k, np.uint32)
    val = np.empty(k, np.float32)
    e_out = np.empty(n, np.float32) if e is not None else None
    rc = lib().bco_compress_randk(_p(g), dt, _p(e), n, k, int(seed), int(tensor_id),
                                  _p(idx), _p(val), _p(e_out))
    assert rc == 0, rc
    return idx, val, e_out


def compress_sign(g, e):
    g, dt = _grad(g)
    n = g.size
    e = _resid(e, n)
    words = np.empty(words_for(n), np.uint32)
    scale = np.zeros(1, np.float32)
    e_out = np.empty(n, np.float32) if e is not None else None
    rc = lib().bco_compress_sign(_p(g), dt, _p(e), n, _p(words), _p(scale), _p(e_out))
    assert rc == 0, rc
    return words, scale[0], e_out


def residual_update_sparse(g, e, idx, val):
    g, dt = _grad(g)
    n = g.size
    e = np.array(e, dtype=np.float32, copy=True)
    idx = np.ascontiguousarray(idx, np.uint32)
    val = np.ascontiguousarray(val, np.float32)
    rc = lib().bco_residual_update_sparse(_p(g), dt, _p(e), n, idx.size, _p(idx), _p(val))
    assert rc == 0, rc
    return e


def residual_update_sign(g, e, words, scale):
    g, dt = _grad(g)
    n = g.size
    e = np.array(e, dtype=np.float32, copy=True)
    words = np.ascontiguousarray(words, np.uint32)
    rc = lib().bco_residual_update_sign(_p(g), dt, _p(e), n, _p(words), float(scale))
    assert rc == 0, rc
    return e


def aggregate_sparse(n, idx_list, val_list, alpha=1.0):
    W = len(idx_list)
    idx_list = [np.ascontiguousarray(a, np.uint32) for a in idx_list]
    val_list = [np.ascontiguousarray(a, np.float32) for a in val_list]
    ip = (ctypes.c_void_p * max(W, 1))(*[a.ctypes.data for a in idx_list])
    vp = (ctypes.c_void_p * max(W, 1))(*[a.ctypes.data for a in val_list])
    kw = np.array([a.size for a in idx_list] or [0], dtype=np.uint64)
    out = np.empty(n, np.float32)
    rc = lib().bco_aggregate_sparse(W, n, ctypes.cast(ip, _vp), ctypes.cast(vp, _vp),
                                    _p(kw), float(alpha), _p(out))
    assert rc == 0, rc
    return out


def aggregate_sign(n, words_list, scales, alpha=1.0, ordered=False):
    W = len(words_list)
    words_list = [np.ascontiguousarray(a, np.uint32) for a in words_list]
    wp = (ctypes.c_void_p * max(W, 1))(*[a.ctypes.data for a in words_list])
    sc = np.ascontiguousarray(np.asarray(scales, dtype=np.float32).reshape(-1))
    out = np.empty(n, np.float32)
    fn = lib().bco_aggregate_sign_ordered if ordered else lib().bco_aggregate_sign
    rc = fn(W, n, ctypes.cast(wp, _vp), _p(sc), float(alpha), _p(out))
    assert rc == 0, rc
    return out


def exact_sum_f32(x):
    x = np.ascontiguousarray(x, np.float32)
    return np.float32(lib().bco_exact_sum_f32(_p(x), x.size))


def philox4x64_10(ctr, key):
    c = np.ascontiguousarray(ctr, np.uint64)
    k = np.ascontiguousarray(key, np.uint64)
    out = np.empty(4, np.uint64)
    lib().bco_philox4x64_10(_p(c), _p(k), _p(out))
    return out


def feistel_half_bits(n):
    return int(lib().bco_feistel_half_bits(int(n)))


def randk_round_keys(seed, tensor_id):
    rk = np.empty(4, np.uint32)
    lib().bco_randk_round_keys(int(seed), int(tensor_id), _p(rk))
    return rk


def feistel_encrypt(x, h, rk):
    rk = np.ascontiguousarray(rk, np.uint32)
    return int(lib().bco_feistel_encrypt(int(x), int(h), _p(rk)))


def randk_index(n, seed, tensor_id, j):
    return int(lib().bco_randk_index(int(n), int(seed), int(tensor_id), int(j)))


def sample_size(n):
    return int(lib().bco_sample_size(int(n)))


# ------------------------------------------------ stochastic quantizers
# Paper Sec. 2.3: quantization to 8 bits, 2 bits (TernGrad) or 1 bit, with
# error feedback.  Kinds here: "terngrad" (2-bit codes, 1 level),
# "qsgd4" (4-bit, 7 levels), "qsgd8" (8-bit, 127 levels); the definitions
# are in the C source.

QUANT_BITS = {"terngrad": 2, "qsgd4": 4, "qsgd8": 8}


def quant_levels(bits):
    return int(lib().bco_quant_levels(int(bits)))


def quant_words(n, bits):
    return int(lib().bco_quant_words(int(n), int(bits)))


def quant_uniform(seed, tensor_id, i):
    return np.float32(lib().bco_quant_uniform(int(seed), int(tensor_id), int(i)))


def quant_decode(code, bits, scale):
    return np.float32(lib().bco_quant_decode(int(code), int(bits), float(scale)))


def compress_quant(g, e, bits, seed, tensor_id):
    g, dt = _grad(g)
    n = g.size
    e = _resid(e, n)
    words = np.empty(quant_words(n, bits), np.uint32)
    scale = np.zeros(1, np.float32)
    e_out = np.empty(n, np.float32) if e is not None else None
    rc = lib().bco_compress_quant(_p(g), dt, _p(e), n, int(bits), int(seed), int(tensor_id),
                                  _p(words), _p(scale), _p(e_out))
    assert rc == 0, rc
    return words, scale[0], e_out


def residual_update_quant(g, e, bits, words, scale):
    g, dt = _grad(g)
    n = g.size
    e = np.array(e, dtype=np.float32, copy=True)
    words = np.ascontiguousarray(words, np.uint32)
    rc = lib().bco_residual_update_quant(_p(g), dt, _p(e), n, int(bits), _p(words), float(scale))
    assert rc == 0, rc
    return e


def aggregate_quant(n, bits, words_list, scales, alpha=1.0):
    W = len(words_list)
    words_list = [np.ascontiguousarray(a, np.uint32) for a in words_list]
    wp = (ctypes.c_void_p * max(W, 1))(*[a.ctypes.data for a in words_list])
    sc = np.ascontiguousarray(np.asarray(scales, dtype=np.float32).reshape(-1))
    out = np.empty(n, np.float32)
    rc = lib().bco_aggregate_quant(W, n, int(bits), ctypes.cast(wp, _vp), _p(sc), float(alpha), _p(out))
    assert rc == 0, rc
    return out


def quant_word_offsets(ns, bits):
    off = np.zeros(len(ns) + 1, dtype=np.int64)
    for t, n in enumerate(ns):
        off[t + 1] = off[t] + quant_words(n, bits)
    return off


# ----------------------------------------------- DGC momentum correction
# DGC (the paper's sparsification operator, Sec. 5.1) keeps a velocity u
# per tensor: u_new = fl32(fl32(m u) + g); the sparse kind compresses
# u_new with the error-feedback residual e; momentum-factor masking then
# zeroes u_new at the chosen entries (e_new is already zero there).

def dgc_momentum(g, u, m):
    g, dt = _grad(g)
    u = np.array(u, dtype=np.float32, copy=True)
    assert u.size == g.size
    rc = lib().bco_dgc_momentum(_p(g), dt, _p(u), g.size, float(m))
    assert rc == 0, rc
    return u


def dgc_clip_factor(grads, clip):
    """Local gradient clipping factor over a tensor list (bco_dgc_clip_factor)."""
    gs = [_grad(g) for g in grads]
    T = len(gs)
    gp_ = (ctypes.c_void_p * max(T, 1))(*[a.ctypes.data if a.size else None for a, _ in gs])
    dts = np.array([dt for _, dt in gs] or [0], dtype=np.int32)
    ns = np.array([a.size for a, _ in gs] or [0], dtype=np.uint64)
    return np.float32(lib().bco_dgc_clip_factor(T, ctypes.cast(gp_, _vp), _p(dts), _p(ns), float(clip)))


def dgc_momentum_clipped(g, u, m, c):
    g, dt = _grad(g)
    u = np.array(u, dtype=np.float32, copy=True)
    assert u.size == g.size
    rc = lib().bco_dgc_momentum_clipped(_p(g), dt, _p(u), g.size, float(m), float(c))
    assert rc == 0, rc
    return u


def compress_dgc(kind, g, e, u, m, ratio, seed, tensor_id, clip_c=None):
    """One DGC step of one tensor: (idx, val, e_new, u_new); clip_c: the
    local clipping factor of the step (None: no clipping)."""
    u_new = dgc_momentum(g, u, m) if clip_c is None else dgc_momentum_clipped(g, u, m, clip_c)
    if kind == "topk":
        idx, val, e_new = compress_topk(u_new, e, ratio)
    elif kind == "topk_sampled":
        idx, val, e_new = compress_topk_sampled(u_new, e, ratio, seed, tensor_id)
    elif kind == "randk":
        idx, val, e_new = compress_randk(u_new, e, ratio, seed, tensor_id)
    else:
        raise ValueError(kind)
    u_new[idx.astype(np.int64)] = np.float32(0.0)
    return idx, val, e_new, u_new


def compress_dgc_set(kind, ratio, seed, m, grads, resids, vels, clip=None):
    """DGC step of a tensor list: (payload dict, new residuals, new velocities);
    clip: the local clipping threshold on the list's L2 norm (None: none)."""
    ns = [g.size for g in grads]
    off = sparse_offsets(ns, ratio)
    idx = np.empty(int(off[-1]), np.uint32)
    val = np.empty(int(off[-1]), np.float32)
    new_e, new_u = [], []
    c = None if clip is None else dgc_clip_factor(grads, clip)
    for t in range(len(grads)):
        i, v, e_out, u_out = compress_dgc(kind, grads[t], resids[t], vels[t], m, ratio, seed, t, c)
        idx[off[t]:off[t + 1]] = i
        val[off[t]:off[t + 1]] = v
        new_e.append(e_out)
        new_u.append(u_out)
    return {"idx": idx, "val": val, "off": off}, new_e, new_u


# ------------------------------------------------------ tensor-list calls

KINDS = ("topk", "topk_sampled", "randk", "sign", "terngrad", "qsgd4", "qsgd8")


def compress_set(kind, ratio, seed, grads, resids):
    """Compress a list of tensors; returns (payload dict, list of new residuals).

    Sparse kinds: payload {"idx", "val", "off"}; sign and the quantizers:
    {"bits", "scale", "off"} (packed code words, one scale per tensor).
    """
    T = len(grads)
    ns = [g.size for g in grads]
    new_e = []
    if kind in QUANT_BITS:
        bits_per = QUANT_BITS[kind]
        off = quant_word_offsets(ns, bits_per)
        bits = np.empty(int(off[-1]), np.uint32)
        scale = np.empty(T, np.float32)
        for t in range(T):
            w, s, e_out = compress_quant(grads[t], None if resids is None else resids[t], bits_per, seed, t)
            bits[off[t]:off[t + 1]] = w
            scale[t] = s
            new_e.append(e_out)
        return {"bits": bits, "scale": scale, "off": off}, new_e
    if kind == "sign":
        off = word_offsets(ns)
        bits = np.empty(int(off[-1]), np.uint32)
        scale = np.empty(T, np.float32)
        for t in range(T):
            w, s, e_out = compress_sign(grads[t], None if resids is None else resids[t])
            bits[off[t]:off[t + 1]] = w
            scale[t] = s
            new_e.append(e_out)
        return {"bits": bits, "scale": scale, "off": off}, new_e
    off = sparse_offsets(ns, ratio)
    idx = np.empty(int(off[-1]), np.uint32)
    val = np.empty(int(off[-1]), np.float32)
    for t in range(T):
        e = None if resids is None else resids[t]
        if kind == "topk":
            i, v, e_out = compress_topk(grads[t], e, ratio)
        elif kind == "topk_sampled":
            i, v, e_out = compress_topk_sampled(grads[t], e, ratio, seed, t)
        elif kind == "randk":
            i, v, e_out = compress_randk(grads[t], e, ratio, seed, t)
        else:
            raise ValueError(kind)
        idx[off[t]:off[t + 1]] = i
        val[off[t]:off[t + 1]] = v
        new_e.append(e_out)
    return {"idx": idx, "val": val, "off": off}, new_e


def aggregate_set(kind, ns, payloads, alpha=1.0):
    """Aggregate W payload dicts (laid out as compress_set returns) per tensor."""
    outs = []
    for t, n in enumerate(ns):
        if kind in QUANT_BITS:
            ws = [p["bits"][p["off"][t]:p["off"][t + 1]] for p in payloads]
            ss = [p["scale"][t] for p in payloads]
            outs.append(aggregate_quant(n, QUANT_BITS[kind], ws, ss, alpha))
        elif kind == "sign":
            ws = [p["bits"][p["off"][t]:p["off"][t + 1]] for p in payloads]
            ss = [p["scale"][t] for p in payloads]
            outs.append(aggregate_sign(n, ws, ss, alpha))
        else:
            ii = [p["idx"][p["off"][t]:p["off"][t + 1]] for p in payloads]
            vv = [p["val"][p["off"][t]:p["off"][t + 1]] for p in payloads]
            outs.append(aggregate_sparse(n, ii, vv, alpha))
    return outs


# ------------------------------------------------------ divisible scheme
# Paper Sec. 3.1, Reason #2 (and the alltoall figure): in a divisible
# scheme a compressed tensor is partitioned into parts; node j receives
# part j from every node, decompresses and aggregates those parts, and
# compresses the aggregate again (the second compression) before it is
# broadcast.  Parts are element ranges [lo, hi) of each tensor.

def check_part_bounds(n, b):
    """Part boundaries of one tensor: 0 = b[0] <= ... <= b[-1] = n, every
    inner boundary a multiple of 32 (word aligned for sign payloads)."""
    b = [int(x) for x in b]
    assert b[0] == 0 and b[-1] == n, (b, n)
    assert all(x <= y for x, y in zip(b, b[1:])), b
    assert all(x % 32 == 0 for x in b[1:-1]), b
    return b


def pack_part_sparse(idx, val, lo, hi):
    """Entries of one tensor's sparse payload whose index lies in [lo, hi),
    in payload order, with indices rebased to the range (index - lo)."""
    idx = np.asarray(idx, np.uint32)
    val = np.asarray(val, np.float32)
    keep = (idx >= lo) & (idx < hi)
    return (idx[keep] - np.uint32(lo)).astype(np.uint32), val[keep].copy()


def pack_part_sign(words, lo, hi, bits=1):
    """Words of one tensor's sign (bits = 1) or b-bit quantizer payload that
    cover [lo, hi), lo a multiple of 32: words lo*b/32 .. ceil(hi*b/32) - 1
    (the scale travels unchanged)."""
    assert lo % 32 == 0
    return np.asarray(words, np.uint32)[lo * bits // 32:(hi * bits + 31) // 32].copy()


def pack_part_set(kind, ns, payload, bounds, j):
    """Part j of every tensor of one payload dict (as compress_set returns),
    laid out tensor by tensor: {'idx', 'val', 'off'} for sparse kinds (off
    = prefix sums of the per-tensor counts), {'bits', 'scale', 'off'} for
    sign and the quantizers (off = prefix sums of the range word counts)."""
    words_kind = kind == "sign" or kind in QUANT_BITS
    out_a, out_b, off = [], [], [0]
    for t, n in enumerate(ns):
        b = check_part_bounds(n, bounds[t])
        lo, hi = b[j], b[j + 1]
        seg = slice(payload["off"][t], payload["off"][t + 1])
        if words_kind:
            w = pack_part_sign(payload["bits"][seg], lo, hi, QUANT_BITS.get(kind, 1))
            out_a.append(w)
        else:
            i, v = pack_part_sparse(payload["idx"][seg], payload["val"][seg], lo, hi)
            out_a.append(i)
            out_b.append(v)
        off.append(off[-1] + out_a[-1].size)
    res = {"off": np.array(off, dtype=np.int64)}
    if words_kind:
        res["bits"] = np.concatenate(out_a) if out_a else np.zeros(0, np.uint32)
        res["scale"] = np.asarray(payload["scale"], np.float32).copy()
    else:
        res["idx"] = np.concatenate(out_a) if out_a else np.zeros(0, np.uint32)
        res["val"] = np.concatenate(out_b) if out_b else np.zeros(0, np.float32)
    return res


def aggregate_part_set(kind, lens, parts, alpha=1.0):
    """Node j's aggregate of the part-j payloads of W senders (each laid out
    as pack_part_set returns): per tensor, the dense slice of length
    lens[t] -- the same decompress-and-aggregate as the whole tensors."""
    return aggregate_set(kind, lens, parts, alpha)


# ------------------------------------------------ all-core list calls
# The same per-tensor functions run over a tensor list with OpenMP (the
# benchmark's all-core CPU baseline); results are bit-identical to
# compress_set / aggregate_set at any thread count.

_lib_omp = None
_KIND_CODE = {"topk": 0, "topk_sampled": 1, "randk": 2, "sign": 3, "terngrad": 4, "qsgd4": 5, "qsgd8": 6}


def omp_lib():
    global _lib_omp
    if _lib_omp is None:
        if not os.path.exists(_build.LIB_OMP):
            _build.build()
        L = ctypes.CDLL(_build.LIB_OMP)
        L.bco_omp_max_threads.restype = _int
        L.bco_omp_max_threads.argtypes = []
        L.bco_compress_list.restype = _int
        L.bco_compress_list.argtypes = [_int, _int, _vp, _vp, _vp, _vp, _vp, _dbl, _u64, _vp, _vp, _vp, _vp,
                                        _vp, _vp, _int]
        L.bco_aggregate_list.restype = _int
        L.bco_aggregate_list.argtypes = [_int, _int, _int, _vp, _vp, _vp, _vp, _flt, _vp, _int]
        _lib_omp = L
    return _lib_omp


def omp_max_threads():
    return int(omp_lib().bco_omp_max_threads())


def _ptrs(arrs):
    return (ctypes.c_void_p * max(len(arrs), 1))(*[None if a is None else a.ctypes.data for a in arrs])


def _payload_offsets(kind, ns, ratio):
    if kind in QUANT_BITS:
        return quant_word_offsets(ns, QUANT_BITS[kind])
    if kind == "sign":
        return word_offsets(ns)
    return sparse_offsets(ns, ratio)


def compress_list_omp(kind, ratio, seed, grads, resids, threads, tensor_ids=None):
    """compress_set on `threads` threads (tensors in parallel)."""
    T = len(grads)
    gs = [_grad(g)[0] for g in grads]
    dts = np.array([_DT[g.dtype] for g in gs], np.int32)
    ns = np.array([g.size for g in gs], np.uint64)
    es = [None] * T if resids is None else [_resid(e, g.size) for e, g in zip(resids, gs)]
    eo = [None if e is None else np.empty(g.size, np.float32) for e, g in zip(es, gs)]
    tids = np.array(range(T) if tensor_ids is None else tensor_ids, np.uint32)
    off = _payload_offsets(kind, [int(x) for x in ns], ratio)
    offu = off.astype(np.uint64)
    word = kind in QUANT_BITS or kind == "sign"
    a = np.empty(max(int(off[-1]), 1), np.uint32)
    b = np.empty(max(int(off[-1]), 1) if not word else max(T, 1), np.float32)
    rc = omp_lib().bco_compress_list(_KIND_CODE[kind], T, _ptrs(gs), _p(dts), _ptrs(es), _p(ns), _p(tids),
                                     float(ratio), int(seed), _p(offu), None if word else _p(a),
                                     None if word else _p(b), _p(a) if word else None, _p(b) if word else None,
                                     _ptrs(eo), int(threads))
    assert rc == 0, rc
    if word:
        return {"bits": a[:int(off[-1])], "scale": b[:T], "off": off}, eo
    return {"idx": a[:int(off[-1])], "val": b[:int(off[-1])], "off": off}, eo


def aggregate_list_omp(kind, ns, payloads, alpha, threads, ratio=None):
    """aggregate_set on `threads` threads (tensors and 4096-element ranges
    in parallel).  payloads: dicts as compress_set returns (their 'off')."""
    T, W = len(ns), len(payloads)
    word = kind in QUANT_BITS or kind == "sign"
    off = np.asarray(payloads[0]["off"]).astype(np.uint64)
    na = np.array(ns, np.uint64)
    if word:
        aa = [np.ascontiguousarray(p["bits"], np.uint32) for p in payloads]
        bb = [np.ascontiguousarray(p["scale"], np.float32) for p in payloads]
    else:
        aa = [np.ascontiguousarray(p["idx"], np.uint32) for p in payloads]
        bb = [np.ascontiguousarray(p["val"], np.float32) for p in payloads]
    outs = [np.empty(int(n), np.float32) for n in ns]
    rc = omp_lib().bco_aggregate_list(_KIND_CODE[kind], W, T, _p(na), _p(off), _ptrs(aa), _ptrs(bb),
                                      float(alpha), _ptrs(outs), int(threads))
    assert rc == 0, rc
    return outs
