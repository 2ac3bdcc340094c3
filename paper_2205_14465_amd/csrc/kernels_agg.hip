// kernels_agg.hip -- decompress-and-aggregate of W workers' payloads on
// gfx950 (paper Sec. 3.1, Reason #2: after the gather each node decompresses
// the N payloads and aggregates them; Sec. 4.2.1, Dimension 3: the
// aggregation of compressed tensors is not associative, so it is not an
// Allreduce), plus the sparse residual update.
//
// Both aggregates add the workers' decoded values in ascending worker order,
// one fp32 addition each, starting from +0.0, then multiply by alpha; no
// floating-point atomics are used, so results are deterministic and match
// that order bit for bit.
//
// Sparse: each wave owns a run of 2048-element output tiles held in LDS.
// For every tile it walks the workers in order; worker w's entries for the
// tile are the next ones after its cursor (indices ascending), read 64 at a
// time and added into the tile (indices are unique within a worker, so a
// worker's adds never collide and need no atomics).  Cursors are found by a
// binary search only where a wave's run starts inside a tensor.
//
// Sign: the exact sum of the workers' decoded values, rounded once to fp32,
// computed with fp64 lookup tables of eight-worker partial sums (exact while
// the scales' exponents stay within a span fp64 can hold); outside that
// range the worker-ordered fp32 sum.
#include "launch.hpp"

namespace bc {

namespace {

typedef const float __attribute__((address_space(4)))* cf32p;

// The aggregate table is [ADesc x T][WDesc x W][unit -> tensor map].
__device__ __forceinline__ int unit_owner(const WDesc* __restrict__ wd, int W, uint32_t u) {
    return (int)reinterpret_cast<const uint32_t*>(wd + W)[u];
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


}  // namespace

// ----------------------------------------------------------------- sparse
// Dynamic LDS: 4 waves x (2048 floats tile + W cursors).
//
// The next entries of kSparseSlots workers are kept in flight in registers
// (slot w % kSparseSlots holds worker w): as soon as a worker's entries for
// the tile have been added, its slot is refilled with the worker that comes
// kSparseSlots later, or, when W is a multiple of kSparseSlots and the
// next tile continues the tensor, with the same worker's entries for the
// next tile (its cursor is then final).
constexpr int kSparseSlots = 16;

__global__ __launch_bounds__(kBlock) void aggregate_sparse(const ADesc* __restrict__ a, int T,
                                                           uint32_t U, const WDesc* __restrict__ wd,
                                                           int W, float alpha) {
    extern __shared__ uint32_t lds[];
    const int wave = wave_id();
    const int lane = lane_id();
    float* tile = reinterpret_cast<float*>(lds) + wave * (int)kSparseTile;
    uint32_t* cur = lds + 4 * kSparseTile + wave * W;
    const uint64_t nw = (uint64_t)gridDim.x * 4;
    const uint64_t gw = (uint64_t)blockIdx.x * 4 + wave;
    const uint32_t u_beg = (uint32_t)((gw * U) / nw);
    const uint32_t u_end = (uint32_t)(((gw + 1) * U) / nw);
    const bool cross = (W % kSparseSlots) == 0;
    // Every slot load is issued unconditionally (index clamped into the
    // tensor's entries, validity kept apart) so that the compiler can count
    // the loads in flight exactly and wait only for the one it needs.
    uint32_t x[kSparseSlots];
    float y[kSparseSlots];
    bool ok[kSparseSlots];
    int t = -1;
    ADesc ad{};
    bool primed = false;  // slots already hold this tile's first entries
    for (uint32_t u = u_beg; u < u_end; ++u) {
        if (t < 0 || u >= ad.unit0 + ad.nunits) {
            t = unit_owner(wd, W, u);
            ad = a[t];
            const uint32_t lo0 = (u - ad.unit0) * kSparseTile;
            for (int w = lane; w < W; w += 64)
                cur[w] = lo0 == 0 ? 0u : lower_bound_u32(wd[w].a + ad.off, ad.k, lo0);
            __builtin_amdgcn_wave_barrier();
            primed = false;
        }
        const uint32_t klast = ad.k - 1;  // a tile exists, so k >= 1
        if (!primed) {
#pragma unroll
            for (int q = 0; q < kSparseSlots; ++q) {
                const int w = q < W ? q : W - 1;
                const uint32_t i = cur[w] + lane;
                const uint32_t ic = i < ad.k ? i : klast;
                x[q] = gp(wd[w].a)[ad.off + ic];
                y[q] = gp(wd[w].b)[ad.off + ic];
                ok[q] = q < W && i < ad.k;
            }
        }
        const uint32_t lo = (u - ad.unit0) * kSparseTile;
        const uint32_t hi = (lo + kSparseTile < ad.n) ? lo + kSparseTile : ad.n;
        const bool next_same = cross && u + 1 < u_end && u + 1 < ad.unit0 + ad.nunits;
        for (int i = lane; i < (int)kSparseTile; i += 64) tile[i] = 0.f;
        __builtin_amdgcn_wave_barrier();
        for (int w0 = 0; w0 < W; w0 += kSparseSlots) {
#pragma unroll
            for (int q = 0; q < kSparseSlots; ++q) {
                const int w = w0 + q;
                if (w >= W) break;
                uint32_t cc = cur[w];
                uint32_t cnt;
                {
                    const bool in = ok[q] && x[q] < hi;
                    const uint64_t m = __ballot(in);
                    // entries below the tile can only come from an unsorted
                    // payload; they are skipped rather than written out of range
                    if (in && x[q] >= lo) tile[x[q] - lo] += y[q];
                    cnt = (uint32_t)__popcll(m);
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                }
                // more than 64 entries of this worker in the tile (dense
                // payloads): keep reading in a loop of its own
                while (cnt == 64) {
                    const uint32_t i = cc + lane;
                    const bool oki = i < ad.k;
                    const uint32_t ic = oki ? i : klast;
                    const uint32_t xi = gp(wd[w].a)[ad.off + ic];
                    const float yi = gp(wd[w].b)[ad.off + ic];
                    const bool in = oki && xi < hi;
                    const uint64_t m = __ballot(in);
                    if (in && xi >= lo) tile[xi - lo] += yi;
                    cnt = (uint32_t)__popcll(m);
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                }
                if (lane == 0) cur[w] = cc;
                // refill the slot: the worker kSparseSlots later in this
                // tile, or this worker's entries for the next tile
                const int wn = w + kSparseSlots;
                const bool later = wn < W;
                const int wr = later ? wn : w;
                const uint32_t i = (later ? cur[wn] : cc) + lane;
                const uint32_t ic = i < ad.k ? i : klast;
                x[q] = gp(wd[wr].a)[ad.off + ic];
                y[q] = gp(wd[wr].b)[ad.off + ic];
                ok[q] = (later || next_same) && i < ad.k;
            }
        }
        primed = next_same;
        float* out = ad.out + lo;
        const uint32_t len = hi - lo;
        for (uint32_t i = 4u * lane; i < len; i += 256u) {
            if (i + 3 < len) {
                stg4f(out + i, f32x4{alpha * tile[i], alpha * tile[i + 1], alpha * tile[i + 2],
                                     alpha * tile[i + 3]});
            } else {
                for (uint32_t q = i; q < len; ++q) gp(out)[q] = alpha * tile[q];
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ------------------------------------------------------------------- sign
namespace {

constexpr int kSignGroup = 4;  // workers whose words are in flight together (ordered form)

// Ordered form: acc[q] += (bit q of word) ? -s : +s for the lane's 32
// elements, one fp32 addition per element and worker in worker order: the
// bit is moved to the sign position (v_lshlrev) and spliced into s (v_bfi).
__device__ __forceinline__ void sign_word_accumulate(float (&acc)[32], uint32_t word, float s) {
    const uint32_t su = f2u(s);
    const uint32_t sign = 0x80000000u;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        const uint32_t t = word << (31 - q);
        uint32_t d;
        asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(d) : "v"(sign), "v"(t), "v"(su));
        acc[q] += u2f(d);
    }
}

}  // namespace

// Each workgroup owns 8192 output elements of one tensor: lane l the 32
// elements of word l of the workgroup's 256-word block (one coalesced
// 1 KiB load per worker).
//
// Exact form (scale exponents within span_limit binades, all finite and
// normal or zero): every partial sum of the decoded values is exact in
// fp64.  Workers are taken eight at a time; the 256 possible sums of a
// group's eight +-s_w are tabulated in LDS (fp64), the eight sign bits of an
// element form the table index, and the fp64 sum of the group entries is
// the exact sum, rounded once to fp32 at the end.  The eight words of a
// group are transposed into per-element bytes with rotate/and-or steps that
// each serve four elements.
//
// Ordered form (otherwise): worker-ordered fp32 additions.
__global__ __launch_bounds__(kBlock) void aggregate_sign(const ADesc* __restrict__ a, int T,
                                                         uint32_t U, const WDesc* __restrict__ wd,
                                                         int W, float alpha, int span_limit) {
    __shared__ double tab[8 * 256];
    __shared__ float sc[1024];
    __shared__ int emin_sh, emax_sh, bad_sh;
    const uint32_t u = blockIdx.x;
    const int t = unit_owner(wd, W, u);
    const ADesc ad = a[t];
    const uint32_t j = u - ad.unit0;
    const uint32_t wi = j * 256u + threadIdx.x;  // word of the tensor this lane owns
    const bool has = wi < ad.k;
    const uint64_t woff = ad.off + wi;
    if (threadIdx.x == 0) {
        emin_sh = 1000;
        emax_sh = -1000;
        bad_sh = 0;
    }
    __syncthreads();
    for (int w = threadIdx.x; w < W; w += kBlock) {
        const float sv = ((cf32p)wd[w].b)[t];
        sc[w] = sv;
        const uint32_t e = (f2u(sv) >> 23) & 255u;
        if (e == 255u || (e == 0u && (f2u(sv) & 0x7FFFFFu))) atomicOr(&bad_sh, 1);
        else if (e) {
            atomicMin(&emin_sh, (int)e);
            atomicMax(&emax_sh, (int)e);
        }
    }
    __syncthreads();
    const bool exact = !bad_sh && (emax_sh < emin_sh || emax_sh - emin_sh <= span_limit);
    const uint32_t e0 = wi * 32u;
    float* out = ad.out + e0;
    float res[32];
    if (exact) {
        double S[32];
#pragma unroll
        for (int q = 0; q < 32; ++q) S[q] = 0.0;
        const int G = (W + 7) / 8;
        for (int g0 = 0; g0 < G; g0 += 8) {
            __syncthreads();
            for (int x = threadIdx.x; x < 8 * 256; x += kBlock) {
                const int gi = g0 + (x >> 8), pat = x & 255;
                double acc = 0.0;
                if (gi < G) {
#pragma unroll
                    for (int jj = 0; jj < 8; ++jj) {
                        const int w = 8 * gi + jj;
                        const double sv = w < W ? (double)sc[w] : 0.0;
                        acc += ((pat >> jj) & 1) ? -sv : sv;
                    }
                }
                tab[x] = acc;
            }
            __syncthreads();
            const int gend = (G - g0) < 8 ? (G - g0) : 8;
            for (int gg = 0; gg < gend; ++gg) {
                const int wbase = 8 * (g0 + gg);
                uint32_t idx4[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) idx4[q] = 0u;
#pragma unroll
                for (int jj = 0; jj < 8; ++jj) {
                    const int w = wbase + jj;
                    const uint32_t word = (has && w < W) ? gp(wd[w].a)[woff] : 0u;
                    const uint32_t m = 0x01010101u << jj;
                    // rotate bits q, q+8, q+16, q+24 of the word to jj, jj+8,
                    // jj+16, jj+24 (v_alignbit), then mask them in (v_and_or)
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        idx4[q] |= __builtin_amdgcn_alignbit(word, word, (uint32_t)((q - jj) & 31)) & m;
                }
                const double* tb = tab + gg * 256;
#pragma unroll
                for (int q = 0; q < 32; ++q) S[q] += tb[(idx4[q & 7] >> (8 * (q >> 3))) & 255u];
            }
        }
#pragma unroll
        for (int q = 0; q < 32; ++q) res[q] = alpha * (float)S[q];
    } else {
        float acc[32];
#pragma unroll
        for (int q = 0; q < 32; ++q) acc[q] = 0.f;
        for (int w0 = 0; w0 < W; w0 += kSignGroup) {
            uint32_t word[kSignGroup];
            float sv[kSignGroup];
#pragma unroll
            for (int g = 0; g < kSignGroup; ++g) {
                const int w = w0 + g < W ? w0 + g : W - 1;
                sv[g] = sc[w];
                word[g] = has ? gp(wd[w].a)[woff] : 0u;
            }
#pragma unroll
            for (int g = 0; g < kSignGroup; ++g)
                if (w0 + g < W) sign_word_accumulate(acc, word[g], sv[g]);
        }
#pragma unroll
        for (int q = 0; q < 32; ++q) res[q] = alpha * acc[q];
    }
    if (!has) return;
    if (e0 + 32u <= ad.n) {
#pragma unroll
        for (int q = 0; q < 32; q += 4)
            stg4f(out + q, f32x4{res[q], res[q + 1], res[q + 2], res[q + 3]});
    } else {
#pragma unroll
        for (int q = 0; q < 32; ++q)
            if (e0 + q < ad.n) gp(out)[q] = res[q];
    }
}

// --------------------------------------------------- sparse residual update
// residual <- (g + residual) - decompress(own): a chunk gathers its entries
// of the payload into an LDS copy of the decoded chunk (zeros elsewhere).
__global__ __launch_bounds__(kBlock) void sparse_residual_update(const TDesc* __restrict__ d, int T,
                                                                 const uint32_t* __restrict__ idx,
                                                                 const float* __restrict__ val) {
    __shared__ float dec[kChunk];
    __shared__ uint32_t start_sh;
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    const uint32_t lo = j * (uint32_t)kChunk;
    const uint32_t hi = lo + kChunk;
    for (int i = threadIdx.x; i < kChunk; i += kBlock) dec[i] = 0.f;
    const uint32_t* ix = idx + td.off;
    const float* vx = val + td.off;
    if (threadIdx.x == 0) start_sh = lower_bound_u32(ix, td.k, lo);
    __syncthreads();
    for (uint32_t base = start_sh;; base += kBlock) {
        const uint32_t i = base + threadIdx.x;
        const uint32_t x = i < td.k ? gp(ix)[i] : 0xFFFFFFFFu;
        const bool in = x < hi;
        if (in && x >= lo) dec[x - lo] = gp(vx)[i];
        if (__syncthreads_count(in) < kBlock) break;
    }
    __syncthreads();
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, true, v, valid);
#pragma unroll
    for (int r = 0; r < kRounds; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * r + q] = v[4 * r + q] - dec[1024 * r + 4 * threadIdx.x + q];
    store_chunk(td.resid, td.n, j, v);
}

// -------------------------------------------------------------- launchers
hipError_t launch_aggregate_sparse(const ADesc* a, int T, uint32_t U, const WDesc* w, int W,
                                   float alpha, hipStream_t s) {
    if (U == 0) return hipSuccess;
    // enough waves to fill the chip several times over; each owns ~U/waves tiles
    uint32_t blocks = (U + 3) / 4;
    if (blocks > 2048) blocks = 2048;
    const size_t lds = (size_t)4 * (kSparseTile * 4 + (size_t)W * 4);
    hipLaunchKernelGGL(aggregate_sparse, dim3(blocks), dim3(kBlock), lds, s, a, T, U, w, W, alpha);
    return hipGetLastError();
}

hipError_t launch_aggregate_sign(const ADesc* a, int T, uint32_t U, const WDesc* w, int W,
                                 float alpha, hipStream_t s) {
    if (U == 0) return hipSuccess;
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    const int span_limit = 29 - lg;  // 24 + span + ceil(log2 W) <= 53
    hipLaunchKernelGGL(aggregate_sign, dim3(U), dim3(kBlock), 0, s, a, T, U, w, W, alpha, span_limit);
    return hipGetLastError();
}

hipError_t launch_sign_residual_update(const TDesc* d, int T, uint32_t C, const uint32_t* bits,
                                       const float* scale, hipStream_t s);

hipError_t launch_residual_update(int kind, const TDesc* d, int T, uint32_t C, bool, bool,
                                  const uint32_t* idx, const float* val, const uint32_t* bits,
                                  const float* scale, hipStream_t s) {
    if (C == 0) return hipSuccess;
    if (kind == 3) return launch_sign_residual_update(d, T, C, bits, scale, s);
    hipLaunchKernelGGL(sparse_residual_update, dim3(C), dim3(kBlock), 0, s, d, T, idx, val);
    return hipGetLastError();
}

}  // namespace bc

namespace bc {

__global__ void zero_header(uint32_t* flags) {
    flags[threadIdx.x] = 0u;
}

hipError_t launch_zero_header(uint32_t* flags, hipStream_t s) {
    hipLaunchKernelGGL(zero_header, dim3(1), dim3(64), 0, s, flags);
    return hipGetLastError();
}

}  // namespace bc
