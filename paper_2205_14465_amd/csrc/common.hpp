// common.hpp -- device-side descriptors and helpers shared by the gfx950
// kernels of the compression library.  Everything here is product code;
// nothing is shared with the CPU oracle.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

// ---------------------------------------------------------------- geometry
// Streaming passes: one 256-thread workgroup (four wave64s) owns a chunk of
// 4096 consecutive elements of one tensor; thread j holds elements
// 1024*r + 4*j + q (r, q = 0..3) so every load instruction of a wave reads
// 1 KiB of fp32 contiguously.
constexpr int kBlock = 256;
constexpr int kChunk = 4096;
constexpr int kEpt = kChunk / kBlock;     // 16 elements per thread
constexpr int kRounds = 4;                // 4 rounds of 1024 elements
constexpr int kChunkWords = kChunk / 32;  // 128 sign words per chunk
constexpr int kBins0 = 2048;              // radix digit 0: key bits 30..20
constexpr int kBins12 = 1024;             // radix digits 1, 2: bits 19..10, 9..0

// ------------------------------------------------------------ descriptors
// One tensor of a compress or residual-update call (48 bytes).
struct TDesc {
    const void* grad;
    float* resid;       // nullptr: error feedback off
    uint32_t n;
    uint32_t dtype;     // 0 fp32, 1 fp16
    uint32_t tid;
    uint32_t k;         // sparse: k_t; sign: word count
    uint64_t off;       // payload offset of this tensor (entries or words)
    uint32_t chunk0;    // first global chunk index
    uint32_t nchunks;
};
static_assert(sizeof(TDesc) == 48, "TDesc layout");

// One tensor of a pack-part call (32 bytes): its payload offset and count
// (entries, or words for sign), the part's element range, and (sign) the
// part's word offset in the packed layout.
struct PDesc {
    uint64_t in_off;
    uint64_t out_off;
    uint32_t k;
    uint32_t lo, hi;
    uint32_t pad;
};
static_assert(sizeof(PDesc) == 32, "PDesc layout");

// Device pointers of one payload (the C-ABI bc_payload, without torch).
struct bc_payload_dev {
    uint32_t* idx;
    float* val;
    uint32_t* bits;
    float* scale;
};

// One tensor of an aggregate call (32 bytes).
struct ADesc {
    float* out;
    uint32_t n;
    uint32_t k;         // sparse: k_t; sign: word count
    uint64_t off;       // payload offset (same for every worker)
    uint32_t unit0;     // first global work unit (tile / wave chunk)
    uint32_t nunits;
};
static_assert(sizeof(ADesc) == 32, "ADesc layout");

// One worker's payload in an aggregate call.
// Worker table of the aggregate descriptor (pointers stored as uint64):
// a[Wp] (sparse: idx, sign: bits), then b[Wp] (sparse: val, sign: scale),
// then the unit -> tensor map; Wp = padded_workers(W) (below) and the
// slots past W repeat worker W-1.

// Largest t with d[t].chunk0 <= c (tensors without chunks share chunk0 with
// their successor, so the search lands on the tensor that owns chunk c).
template <typename D, uint32_t D::*Field>
__device__ __forceinline__ int find_owner(const D* __restrict__ d, int T, uint32_t c) {
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (d[mid].*Field <= c) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// The device descriptor table of a call is followed by a chunk -> tensor
// map (one uint32 per chunk), built on the host when the table is cached.
__device__ __forceinline__ int tensor_of_chunk(const TDesc* __restrict__ d, int T, uint32_t c) {
    return (int)reinterpret_cast<const uint32_t*>(d + T)[c];
}

// Pointers read from descriptor tables are generic; viewing them in the
// global address space lets the compiler use global (not flat) memory
// instructions with scalar base addresses.
#define BC_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ BC_GLOBAL T* gp(T* p) { return (BC_GLOBAL T*)p; }
template <typename T>
__device__ __forceinline__ const BC_GLOBAL T* gp(const T* p) { return (const BC_GLOBAL T*)p; }

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
// 16- and 8-byte global loads/stores (addresses aligned accordingly)
__device__ __forceinline__ f32x4 ldg4f(const float* p) { return *(const BC_GLOBAL f32x4*)p; }
__device__ __forceinline__ u32x4 ldg4u(const void* p) { return *(const BC_GLOBAL u32x4*)p; }
__device__ __forceinline__ u32x2 ldg2u(const void* p) { return *(const BC_GLOBAL u32x2*)p; }
__device__ __forceinline__ void stg4f(float* p, f32x4 v) { *(BC_GLOBAL f32x4*)p = v; }
// The same with the non-temporal hint when kNT: streaming passes over
// tensor sets larger than the last-level cache skip allocating their lines
// (measured: a two-read-one-write stream over 1.5 G elements moves 6.2 TB/s
// this way against 5.5 TB/s with cached accesses).
template <bool kNT>
__device__ __forceinline__ f32x4 ldg4f_s(const float* p) {
    if constexpr (kNT) return __builtin_nontemporal_load((const BC_GLOBAL f32x4*)p);
    else return *(const BC_GLOBAL f32x4*)p;
}
template <bool kNT>
__device__ __forceinline__ u32x2 ldg2u_s(const void* p) {
    if constexpr (kNT) return __builtin_nontemporal_load((const BC_GLOBAL u32x2*)p);
    else return *(const BC_GLOBAL u32x2*)p;
}
template <bool kNT>
__device__ __forceinline__ void stg4f_s(float* p, f32x4 v) {
    if constexpr (kNT) __builtin_nontemporal_store(v, (BC_GLOBAL f32x4*)p);
    else *(BC_GLOBAL f32x4*)p = v;
}

// ------------------------------------------------------------- bit helpers
__device__ __forceinline__ uint32_t f2u(float x) { return __float_as_uint(x); }
__device__ __forceinline__ float u2f(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t key_of(float x) { return f2u(x) & 0x7FFFFFFFu; }

// IEEE binary16 bits -> fp32 (exact, subnormals included: v_cvt_f32_f16
// with fp16 denormals enabled, the HIP default).
__device__ __forceinline__ float h2f(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// ----------------------------------------------------------- chunk loading
// A chunk that lies wholly inside its tensor (every chunk but a tensor's
// last, in general) is read by straight-line code that issues all of a
// thread's vector loads before it uses any of them, so that they are in
// flight together; the per-element path serves the tensor's last chunk.
// The test is uniform over the workgroup (one chunk, one tensor).
__device__ __forceinline__ bool whole_chunk(const TDesc& td, uint32_t j) {
    return (uint64_t)j * kChunk + kChunk <= td.n;
}

// Widened gradient element q (0..3) of a thread's round: fp32 bits, or the
// fp16 halves of two packed words.
template <int DT>
__device__ __forceinline__ float g_elem(const f32x4& gf, const u32x2& gh, int q) {
    if constexpr (DT == 0) return gf[q];
    else return h2f(((q < 2 ? gh.x : gh.y) >> (16 * (q & 1))) & 0xFFFFu);
}

// Load the 16 elements a thread owns of chunk `j` of tensor `td`, forming
// v = widen(g) + e (e = 0 when there is no residual or `use_resid` is
// false).  Elements past the tensor's end read as +0.0 and are reported
// invalid through `valid` (bit 4*r + q).
template <int DT, bool kNT = false>
__device__ __forceinline__ void load_chunk(const TDesc& td, uint32_t j, bool use_resid,
                                           float v[kEpt], uint32_t& valid) {
    const uint32_t base = j * (uint32_t)kChunk;
    const uint32_t n = td.n;
    if (whole_chunk(td, j)) {
        f32x4 gf[kRounds];
        u32x2 gh[kRounds];
        const uint32_t e0 = base + 4u * threadIdx.x;
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
            if constexpr (DT == 0) gf[r] = ldg4f_s<kNT>((const float*)td.grad + e0 + 1024u * r);
            else gh[r] = ldg2u_s<kNT>((const uint16_t*)td.grad + e0 + 1024u * r);
        }
        if (use_resid) {
            f32x4 ev[kRounds];
#pragma unroll
            for (int r = 0; r < kRounds; ++r) ev[r] = ldg4f_s<kNT>(td.resid + e0 + 1024u * r);
#pragma unroll
            for (int r = 0; r < kRounds; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) v[4 * r + q] = g_elem<DT>(gf[r], gh[r], q) + ev[r][q];
        } else {
#pragma unroll
            for (int r = 0; r < kRounds; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) v[4 * r + q] = g_elem<DT>(gf[r], gh[r], q);
        }
        valid = 0xFFFFu;
        return;
    }
    valid = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = base + 1024u * r + 4u * threadIdx.x;
        float g4[4] = {0.f, 0.f, 0.f, 0.f};
        float e4[4] = {0.f, 0.f, 0.f, 0.f};
        if (e0 + 3 < n) {
            if (DT == 0) {
                const f32x4 x = ldg4f_s<kNT>((const float*)td.grad + e0);
                g4[0] = x.x; g4[1] = x.y; g4[2] = x.z; g4[3] = x.w;
            } else {
                const u32x2 h = ldg2u_s<kNT>((const uint16_t*)td.grad + e0);
                g4[0] = h2f(h.x & 0xFFFFu);
                g4[1] = h2f(h.x >> 16);
                g4[2] = h2f(h.y & 0xFFFFu);
                g4[3] = h2f(h.y >> 16);
            }
            if (use_resid) {
                const f32x4 y = ldg4f_s<kNT>(td.resid + e0);
                e4[0] = y.x; e4[1] = y.y; e4[2] = y.z; e4[3] = y.w;
            }
            valid |= 0xFu << (4 * r);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (e0 + q < n) {
                    if (DT == 0) g4[q] = gp((const float*)td.grad)[e0 + q];
                    else g4[q] = h2f(gp((const uint16_t*)td.grad)[e0 + q]);
                    if (use_resid) e4[q] = gp(td.resid)[e0 + q];
                    valid |= 1u << (4 * r + q);
                }
            }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * r + q] = use_resid ? g4[q] + e4[q] : g4[q];
    }
}

// Runtime dtype dispatch (uniform per workgroup: a chunk has one tensor).
template <bool kNT = false>
__device__ __forceinline__ void load_v(const TDesc& td, uint32_t j, bool use_resid, float v[kEpt],
                                       uint32_t& valid) {
    if (td.dtype == 0) load_chunk<0, kNT>(td, j, use_resid, v, valid);
    else load_chunk<1, kNT>(td, j, use_resid, v, valid);
}

// Raw chunk data held in registers between issuing the loads and using
// them (lets a kernel prefetch its next chunk before a wait).  g[4r + q]
// holds element 4r + q's fp32 bits or, for fp16 gradients, g[4r] and
// g[4r + 1] hold round r's four elements as packed halves (low half
// first); e is written only when the residual is read.
struct RawChunk {
    uint32_t g[kEpt];
    float e[kEpt];
    uint32_t valid;
};

// kDT: 0 every tensor of the call is fp32, 1 every tensor is fp16, 2 both
// occur (td.dtype decides).  A kernel that keeps loads in flight across
// iterations is instantiated per kDT so that the common single-dtype calls
// have one load sequence (no merge of two register sets that would make
// the compiler wait for the loads).
template <int kDT>
__device__ __forceinline__ void load_raw(const TDesc& td, uint32_t j, bool use_resid, RawChunk& r) {
    if constexpr (kDT == 2) {
        if (td.dtype == 0) load_raw<0>(td, j, use_resid, r);
        else load_raw<1>(td, j, use_resid, r);
    } else {
        const uint32_t base = j * (uint32_t)kChunk;
        const uint32_t n = td.n;
        if (whole_chunk(td, j)) {
            const uint32_t e0 = base + 4u * threadIdx.x;
#pragma unroll
            for (int rr = 0; rr < kRounds; ++rr) {
                if constexpr (kDT == 0) {
                    const u32x4 x = ldg4u((const float*)td.grad + e0 + 1024u * rr);
                    r.g[4 * rr] = x.x; r.g[4 * rr + 1] = x.y; r.g[4 * rr + 2] = x.z; r.g[4 * rr + 3] = x.w;
                } else {
                    const u32x2 h = ldg2u((const uint16_t*)td.grad + e0 + 1024u * rr);
                    r.g[4 * rr] = h.x;
                    r.g[4 * rr + 1] = h.y;
                }
            }
            if (use_resid) {
#pragma unroll
                for (int rr = 0; rr < kRounds; ++rr) {
                    const f32x4 y = ldg4f(td.resid + e0 + 1024u * rr);
                    r.e[4 * rr] = y.x; r.e[4 * rr + 1] = y.y; r.e[4 * rr + 2] = y.z; r.e[4 * rr + 3] = y.w;
                }
            }
            r.valid = 0xFFFFu;
            return;
        }
        r.valid = 0;
#pragma unroll
        for (int rr = 0; rr < kRounds; ++rr) {
            const uint32_t e0 = base + 1024u * rr + 4u * threadIdx.x;
            if constexpr (kDT == 1) {
                r.g[4 * rr] = 0u;
                r.g[4 * rr + 1] = 0u;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bool ok = e0 + q < n;
                if constexpr (kDT == 0) {
                    r.g[4 * rr + q] = ok ? gp((const uint32_t*)td.grad)[e0 + q] : 0u;
                } else {
                    const uint32_t hb = ok ? (uint32_t)gp((const uint16_t*)td.grad)[e0 + q] : 0u;
                    r.g[4 * rr + (q >> 1)] |= hb << (16 * (q & 1));
                }
                if (use_resid) r.e[4 * rr + q] = ok ? gp(td.resid)[e0 + q] : 0.f;
                r.valid |= (ok ? 1u : 0u) << (4 * rr + q);
            }
        }
    }
}

// v = widen(g) + e from a RawChunk (e = 0 without residual), exactly as
// load_v forms it; elements past the tensor's end read as +0.0.
template <int kDT>
__device__ __forceinline__ void raw_to_v(const TDesc& td, bool use_resid, const RawChunk& r, float v[kEpt]) {
    const bool f16 = kDT == 1 || (kDT == 2 && td.dtype != 0);
#pragma unroll
    for (int i = 0; i < kEpt; ++i) {
        float g = f16 ? h2f((r.g[(i & ~3) + ((i >> 1) & 1)] >> (16 * (i & 1))) & 0xFFFFu) : u2f(r.g[i]);
        g = ((r.valid >> i) & 1u) ? g : 0.f;
        v[i] = use_resid ? g + r.e[i] : g;
    }
}

// Load v that an earlier pass already stored (the residual buffer holds v),
// or recompute it from the gradient when error feedback is off.
__device__ __forceinline__ void load_stored_v(const TDesc& td, uint32_t j, float v[kEpt],
                                              uint32_t& valid) {
    if (td.resid) {
        const uint32_t base = j * (uint32_t)kChunk;
        if (whole_chunk(td, j)) {
            f32x4 y[kRounds];
#pragma unroll
            for (int r = 0; r < kRounds; ++r) y[r] = ldg4f(td.resid + base + 1024u * r + 4u * threadIdx.x);
#pragma unroll
            for (int r = 0; r < kRounds; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) v[4 * r + q] = y[r][q];
            valid = 0xFFFFu;
            return;
        }
        valid = 0;
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
            const uint32_t e0 = base + 1024u * r + 4u * threadIdx.x;
            if (e0 + 3 < td.n) {
                const f32x4 y = ldg4f(td.resid + e0);
                v[4 * r] = y.x; v[4 * r + 1] = y.y; v[4 * r + 2] = y.z; v[4 * r + 3] = y.w;
                valid |= 0xFu << (4 * r);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    bool ok = e0 + q < td.n;
                    v[4 * r + q] = ok ? gp(td.resid)[e0 + q] : 0.f;
                    valid |= (ok ? 1u : 0u) << (4 * r + q);
                }
            }
        }
    } else if (td.dtype == 0) {
        load_chunk<0>(td, j, false, v, valid);
    } else {
        load_chunk<1>(td, j, false, v, valid);
    }
}

// Store 16 per-thread values back to a dense fp32 tensor (same pattern).
template <bool kNT = false>
__device__ __forceinline__ void store_chunk(float* dst, uint32_t n, uint32_t j, const float v[kEpt]) {
    const uint32_t base = j * (uint32_t)kChunk;
    if ((uint64_t)base + kChunk <= n) {
#pragma unroll
        for (int r = 0; r < kRounds; ++r)
            stg4f_s<kNT>(dst + base + 1024u * r + 4u * threadIdx.x,
                         f32x4{v[4 * r], v[4 * r + 1], v[4 * r + 2], v[4 * r + 3]});
        return;
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = base + 1024u * r + 4u * threadIdx.x;
        if (e0 + 3 < n) {
            stg4f_s<kNT>(dst + e0, f32x4{v[4 * r], v[4 * r + 1], v[4 * r + 2], v[4 * r + 3]});
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (e0 + q < n) gp(dst)[e0 + q] = v[4 * r + q];
        }
    }
}

// --------------------------------------------------------- block reductions
// Sum of a double over the 256 threads in a fixed tree (deterministic for a
// given block shape); every thread receives the total.
__device__ __forceinline__ double block_sum_f64(double x, double* sh /* >= 4 */) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
    if (lane_id() == 0) sh[threadIdx.x >> 6] = x;
    __syncthreads();
    double t = (sh[0] + sh[1]) + (sh[2] + sh[3]);
    __syncthreads();
    return t;
}

// Exclusive prefix of a 64-bit value over the block (thread order), plus
// the block total.  `sh` needs 4 entries.
__device__ __forceinline__ uint64_t block_excl_scan_u64(uint64_t x, uint64_t* sh, uint64_t& total) {
    const int lane = lane_id();
    uint64_t inc = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        uint64_t y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
    }
    if (lane == 63) sh[threadIdx.x >> 6] = inc;
    __syncthreads();
    const int w = threadIdx.x >> 6;
    uint64_t before = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) before += (q < w) ? sh[q] : 0;
    total = sh[0] + sh[1] + sh[2] + sh[3];
    __syncthreads();
    return before + inc - x;
}

// ------------------------------------------------------- device atomics
__device__ __forceinline__ uint32_t atomic_add_agent(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t atomic_load_acquire(uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void atomic_store_release(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void atomic_store_relaxed(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------- Philox
// Philox4x64-10 counter-based generator (Salmon et al., SC'11): ten rounds
// of two 64x64->128-bit multiplies on counter words 0 and 2, a fixed word
// permutation and xor with the remaining words and the key; the key is
// advanced by the two Weyl constants before every round but the first.
struct U64x4 { uint64_t v[4]; };

__host__ __device__ inline void mul_hilo64(uint64_t a, uint64_t b, uint64_t& hi, uint64_t& lo) {
#if defined(__HIP_DEVICE_COMPILE__)
    // the 128-bit product from four 32x32+64-bit multiply-adds (v_mad_u64_u32),
    // sharing the partial products between the two halves; no sum overflows:
    // (2^32 - 1)^2 + (2^32 - 1) < 2^64
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p00 = (uint64_t)a0 * b0;
    const uint64_t p10 = (uint64_t)a1 * b0 + (p00 >> 32);
    const uint64_t p01 = (uint64_t)a0 * b1 + (uint32_t)p10;
    hi = (uint64_t)a1 * b1 + (p10 >> 32) + (p01 >> 32);
    lo = (p01 << 32) | (uint32_t)p00;
#else
    unsigned __int128 p = (unsigned __int128)a * b;
    hi = (uint64_t)(p >> 64);
    lo = (uint64_t)p;
#endif
}

__host__ __device__ inline U64x4 philox4x64_10(U64x4 c, uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) { k0 += W0; k1 += W1; }
        uint64_t h0, l0, h1, l1;
        mul_hilo64(M0, c.v[0], h0, l0);
        mul_hilo64(M1, c.v[2], h1, l1);
        U64x4 o;
        o.v[0] = h1 ^ c.v[1] ^ k0;
        o.v[1] = l1;
        o.v[2] = h0 ^ c.v[3] ^ k1;
        o.v[3] = l0;
        c = o;
    }
    return c;
}

// Random-stream ids (second key word).
constexpr uint64_t kStreamRandk = 0;
constexpr uint64_t kStreamSample = 1;
constexpr uint64_t kStreamQuant = 2;

// Workspace header: failure flags reported by bytecomp_device_status.  No
// current kernel sets one: the one-pass compress kernels wait for other
// workgroups, but only for a bounded time, and a wait that runs out takes
// a path whose results are exact (the workgroup computes the missing
// partials itself), so it is no failure.

// --------------------------------------------- one-pass compress protocol
// A one-pass compress kernel defers each chunk's residual (and, for the
// quantizers, its codes) until its tensor's scale is known, which needs a
// published partial (a sum of |v|, or a largest |v|) of every chunk of the
// tensor.  A workgroup waits for missing partials only for a bounded time;
// then it computes each still-missing partial itself, from the chunk's
// gradient and residual, with exactly the owner's arithmetic (so the value
// is bit-identical), and publishes it by compare-and-swap from empty: if the
// owner published first, the owner's value stays.  The owner writes the
// chunk's residual only once its tensor's partials are all published, and a
// helper reads the chunk's residual only while its partial is still
// missing, so a helper's publication never rests on a residual the owner
// has already overwritten (had the owner begun, its partial would be
// published and the helper's swap would fail).  Every wait therefore ends
// after at most the limit plus the workgroup's own work, whatever the
// residency of the grid.

// ------------------------------------------------- aggregate worker table
// Worker descriptors in the aggregate table are padded to a multiple of 16.
__host__ __device__ constexpr int padded_workers(int W) { return (W + 15) & ~15; }

// The aggregate table is [ADesc x T][a x Wp][b x Wp][unit -> tensor map]
// with Wp = padded_workers(W); slots past W repeat worker W-1.
__device__ __forceinline__ const uint32_t* w_a(const uint64_t* __restrict__ wp, int w) {
    return (const uint32_t*)wp[w];
}
__device__ __forceinline__ const float* w_b(const uint64_t* __restrict__ wp, int W, int w) {
    return (const float*)wp[padded_workers(W) + w];
}
__device__ __forceinline__ int unit_owner(const uint64_t* __restrict__ wp, int W, uint32_t u) {
    return (int)reinterpret_cast<const uint32_t*>(wp + 2 * padded_workers(W))[u];
}

// Tensor whose payload entries hold flattened entry j: the last tensor
// with off <= j (tensors without entries share the next one's offset).
__device__ __forceinline__ int tensor_of_entry(const TDesc* __restrict__ d, int T, uint64_t j) {
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (d[mid].off <= j) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// First position p in [0, k) with idx[p] >= x (k if none).
__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* idx, uint32_t k, uint32_t x) {
    uint32_t lo = 0, hi = k;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (gp(idx)[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}


}  // namespace bc
