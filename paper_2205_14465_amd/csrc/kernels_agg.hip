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
// Sparse: each wave owns a run of 2048- or 4096-element output tiles held
// in LDS.
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
// Each wave owns a run of consecutive kTS-element tiles held in its own LDS
// slice.  The next 64 entries of kS workers are kept in flight in registers
// (slot w % kS holds worker w): as soon as a worker's entries for the tile
// have been added, its slot is refilled with the worker that comes kS
// later, or, when W is a multiple of kS and the next tile continues the
// tensor, with the entries of the slot's first worker (w % kS) for the next
// tile (its cursor is final by then).
//
// kLanes (W <= 64): lane w of a VGPR holds worker w's cursor and its two
// payload pointers (already offset to the tensor), read with readlane, so
// a step touches neither LDS nor the scalar cache for bookkeeping.
// Otherwise the cursors live in LDS after the tiles and the pointers are
// read from the worker table.
template <uint32_t kTS, int kS, bool kLanes>
__global__ __launch_bounds__(kBlock) void aggregate_sparse(const ADesc* __restrict__ a, int T,
                                                           uint32_t U, const uint64_t* __restrict__ wp,
                                                           int W, float alpha) {
    extern __shared__ uint32_t lds[];
    const int wave = wave_id();
    const int lane = lane_id();
    float* tile = reinterpret_cast<float*>(lds) + wave * (int)kTS;
    uint32_t* cur = lds + 4 * kTS + wave * W;  // !kLanes only
    const uint64_t nw = (uint64_t)gridDim.x * 4;
    const uint64_t gw = (uint64_t)blockIdx.x * 4 + wave;
    const uint32_t u_beg = (uint32_t)((gw * U) / nw);
    const uint32_t u_end = (uint32_t)(((gw + 1) * U) / nw);
    const bool cross = (W % kS) == 0;
    // per-lane worker state (kLanes): cursor, payload pointers of the tensor
    uint32_t curv = 0;
    uint64_t pav = 0, pbv = 0;
    auto get_cur = [&](int w) -> uint32_t {
        if constexpr (kLanes) return (uint32_t)__builtin_amdgcn_readlane((int)curv, w);
        else return cur[w];
    };
    auto set_cur = [&](int w, uint32_t c) {
        if constexpr (kLanes) curv = lane == w ? c : curv;
        else if (lane == 0) cur[w] = c;
    };
    // Every slot load is issued unconditionally (index clamped into the
    // tensor's entries) so that the compiler can count the loads in flight
    // exactly and wait only for the one it needs; a dead slot's entries are
    // masked by setting every bit of its index (never below a tile end).
    uint32_t x[kS];
    float y[kS];
    uint32_t inv[kS];
    int t = -1;
    ADesc ad{};
    bool primed = false;  // slots already hold this tile's first entries
    for (uint32_t u = u_beg; u < u_end; ++u) {
        if (t < 0 || u >= ad.unit0 + ad.nunits) {
            t = unit_owner(wp, W, u);
            ad = a[t];
            const uint32_t lo0 = (u - ad.unit0) * kTS;
            if constexpr (kLanes) {
                const int wl = lane < W ? lane : W - 1;
                pav = wp[wl] + ad.off * 4u;
                pbv = wp[padded_workers(W) + wl] + ad.off * 4u;
                curv = lo0 == 0 ? 0u : lower_bound_u32((const uint32_t*)pav, ad.k, lo0);
            } else {
                for (int w = lane; w < W; w += 64)
                    cur[w] = lo0 == 0 ? 0u : lower_bound_u32(w_a(wp, w) + ad.off, ad.k, lo0);
                __builtin_amdgcn_wave_barrier();
            }
            primed = false;
        }
        const uint32_t klast = ad.k - 1;  // a tile exists, so k >= 1
        auto load_slot = [&](int q, int w, uint32_t c, bool live) {
            const uint32_t i = c + lane;
            const uint32_t ic = i < ad.k ? i : klast;
            const uint32_t* pa;
            const float* pb;
            if constexpr (kLanes) {
                pa = (const uint32_t*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pav >> 32), w) << 32) |
                                       (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pav, w));
                pb = (const float*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pbv >> 32), w) << 32) |
                                    (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pbv, w));
            } else {
                pa = w_a(wp, w) + ad.off;
                pb = w_b(wp, W, w) + ad.off;
            }
            x[q] = gp(pa)[ic];
            y[q] = gp(pb)[ic];
            inv[q] = (live && i < ad.k) ? 0u : 0xFFFFFFFFu;
            asm volatile("" : "+v"(inv[q]));  // computed here, not sunk to its use
        };
        if (!primed) {
            // W through an opaque copy: keeps the sixteen per-slot worker
            // numbers and flags from being hoisted into live SGPRs
            int Wq = W;
            asm volatile("" : "+s"(Wq));
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                const int w = q < Wq ? q : Wq - 1;
                load_slot(q, w, get_cur(w), q < Wq);
            }
        }
        const uint32_t lo = (u - ad.unit0) * kTS;
        const uint32_t hi = (lo + kTS < ad.n) ? lo + kTS : ad.n;
        const uint32_t len = hi - lo;
        const bool next_same = cross && u + 1 < u_end && u + 1 < ad.unit0 + ad.nunits;
#pragma unroll
        for (uint32_t r = 0; r < kTS / 256u; ++r)
            *reinterpret_cast<f32x4*>(tile + 256u * r + 4u * lane) = f32x4{0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_wave_barrier();
        // a worker with 64 or more entries in the tile (dense payloads)
        // ends the pipelined walk: the rest of the tile, from that worker
        // on, is finished one 64-entry window at a time below.  Keeping that
        // loop out of the pipelined steps keeps their load waits exact.
        int dw = -1;
        uint32_t dcc = 0;
        for (int w0 = 0; w0 < W; w0 += kS) {
            // all kS steps issue their two loads on every path (the ones
            // past W or after a dense worker are dead), so that the compiler
            // counts the loads in flight the same way on every path
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                const int w = w0 + q;
                // W through an opaque copy per step, so that the per-step
                // flags are computed here rather than hoisted into SGPRs
                int Wq = W;
                asm volatile("" : "+s"(Wq));
                uint32_t cc = 0;
                if (w < Wq && dw < 0) {  // no load in here
                    cc = get_cur(w);
                    const uint32_t xv = x[q] | inv[q];
                    const uint64_t m = __ballot(xv < hi);
                    // entries below the tile can only come from an unsorted
                    // payload; they are skipped rather than written out of range
                    const uint32_t dd = xv - lo;
                    if (dd < len) tile[dd] += y[q];
                    const uint32_t cnt = (uint32_t)__popcll(m);
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                    if (cnt == 64) {
                        dw = w;
                        dcc = cc;
                    } else {
                        set_cur(w, cc);
                    }
                }
                // refill the slot: the worker kS later in this tile, or else
                // (W a multiple of kS) worker q's entries for the next tile,
                // its cursor being final here
                const int wn = w + kS;
                const bool later = wn < Wq;
                int wr = later ? wn : wn - Wq;
                wr = wr < Wq ? wr : Wq - 1;
                const bool live = w < Wq && dw < 0 && (later || next_same);
                load_slot(q, wr, later ? get_cur(wn) : (wr == w ? cc : get_cur(wr)), live);
            }
            if (dw >= 0) break;
        }
        if (dw >= 0) {
            for (int w = dw; w < W; ++w) {
                uint32_t cc = w == dw ? dcc : get_cur(w);
                const uint32_t* pa;
                const float* pb;
                if constexpr (kLanes) {
                    pa = (const uint32_t*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pav >> 32), w) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pav, w));
                    pb = (const float*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pbv >> 32), w) << 32) |
                                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pbv, w));
                } else {
                    pa = w_a(wp, w) + ad.off;
                    pb = w_b(wp, W, w) + ad.off;
                }
                uint32_t cnt = 64;
                while (cnt == 64) {
                    const uint32_t i = cc + lane;
                    const bool oki = i < ad.k;
                    const uint32_t ic = oki ? i : klast;
                    const uint32_t xi = oki ? gp(pa)[ic] : 0xFFFFFFFFu;
                    const float yi = gp(pb)[ic];
                    const uint64_t m = __ballot(xi < hi);
                    const uint32_t dd = xi - lo;
                    if (dd < len) tile[dd] += yi;
                    cnt = (uint32_t)__popcll(m);
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                }
                set_cur(w, cc);
            }
            primed = false;
        } else {
            primed = next_same;
        }
        float* out = ad.out + lo;
        if (len == kTS) {
#pragma unroll
            for (uint32_t r = 0; r < kTS / 256u; ++r) {
                const uint32_t i = 256u * r + 4u * lane;
                const f32x4 v = *reinterpret_cast<const f32x4*>(tile + i);
                stg4f(out + i, f32x4{alpha * v[0], alpha * v[1], alpha * v[2], alpha * v[3]});
            }
        } else {
            for (uint32_t i = 4u * lane; i < len; i += 256u) {
                if (i + 3 < len) {
                    stg4f(out + i, f32x4{alpha * tile[i], alpha * tile[i + 1], alpha * tile[i + 2],
                                         alpha * tile[i + 3]});
                } else {
                    for (uint32_t q = i; q < len; ++q) gp(out)[q] = alpha * tile[q];
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ------------------------------------------------------------------- sign
namespace {

constexpr int kSignGroup = 4;  // workers whose words are in flight together (ordered form)

// Word at a 32-bit byte offset from a wave-uniform base: the form the
// backend emits as a global load with an SGPR base and a VGPR offset.
__device__ __forceinline__ uint32_t ld_word(const uint32_t* base, uint32_t byte_off) {
    return *(const BC_GLOBAL uint32_t*)((const BC_GLOBAL char*)gp(base) + byte_off);
}

// Transposes the four 8x8 bit matrices held byte-wise in x[0..7]: on
// return bit c of byte r of x[i] is what bit i of byte r of x[c] was.
// Three rounds of block swaps (4x4, 2x2, 1x1 blocks), each exchanging bits
// between two words with a shift, an xor-and and two xors.
__host__ __device__ __forceinline__ void transpose_bytes8(uint32_t (&x)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t t = ((x[i] >> 4) ^ x[i + 4]) & 0x0F0F0F0Fu;
        x[i + 4] ^= t;
        x[i] ^= t << 4;
    }
#pragma unroll
    for (int i = 0; i < 8; i += 4) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const uint32_t t = ((x[i + k] >> 2) ^ x[i + k + 2]) & 0x33333333u;
            x[i + k + 2] ^= t;
            x[i + k] ^= t << 2;
        }
    }
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
        const uint32_t t = ((x[i] >> 1) ^ x[i + 1]) & 0x55555555u;
        x[i + 1] ^= t;
        x[i] ^= t << 1;
    }
}

// Ordered form: acc[q] += (bit q of half) ? -s : +s for the lane's 16
// elements, one fp32 addition per element and worker in worker order: the
// bit is moved to the sign position (v_lshlrev) and spliced into s (v_bfi).
__device__ __forceinline__ void sign_half_accumulate(float (&acc)[16], uint32_t half, float s) {
    const uint32_t su = f2u(s);
    const uint32_t sign = 0x80000000u;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        const uint32_t t = half << (31 - q);
        uint32_t d;
        asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(d) : "v"(sign), "v"(t), "v"(su));
        acc[q] += u2f(d);
    }
}

// Integer image of a scale for the 32-bit exact form: the scale as a
// multiple of 2^(emin - 150), the unit in the last place of the smallest
// normal scale of the tensor (zero stays zero).
__device__ __forceinline__ int32_t scale_units(float s, int emin) {
    const uint32_t b = f2u(s);
    const int e = (int)((b >> 23) & 255u);
    if (e == 0) return 0;
    const int32_t m = (int32_t)(((b & 0x7FFFFFu) | 0x800000u) << (e - emin));
    return (b >> 31) ? -m : m;
}

// Tables of groups g .. g+7 (g a multiple of 8): tab[256 gi + p] = sum over
// the eight workers 8(g+gi)+c of (bit c of p ? -s : +s), each entry the sum
// of two four-worker entries sub[32 gi + 16 hh + p'].  Workers past W count
// as zero.  Called by the whole workgroup.
template <typename Acc>
__device__ __forceinline__ void build_tables(int g, int W, const float* sc, int emin, Acc* tab, Acc* sub) {
    __syncthreads();  // earlier lookups are done with the tables
    {
        const int x = threadIdx.x;  // kBlock == 8 * 32 entries
        const int w0 = 8 * (g + (x >> 5)) + 4 * ((x >> 4) & 1), pat = x & 15;
        Acc acc = (Acc)0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            Acc sv = (Acc)0;
            if (w0 + c < W) {
                if constexpr (sizeof(Acc) == 4) sv = scale_units(sc[w0 + c], emin);
                else sv = (double)sc[w0 + c];
            }
            acc += ((pat >> c) & 1) ? -sv : sv;
        }
        sub[x] = acc;
    }
    __syncthreads();
    for (int x = threadIdx.x; x < 8 * 256; x += kBlock) {
        const int gi = x >> 8, pat = x & 255;
        tab[x] = sub[32 * gi + (pat & 15)] + sub[32 * gi + 16 + (pat >> 4)];
    }
    __syncthreads();
}

// One step: add the table entries of groups g and g+1 for the lane's 16
// elements.  w[jj] is worker 8g+jj's word, w[8+jj] worker 8(g+1)+jj's.
// v_perm packs the lane's half-word of each pair (selectors 0-3 pick bytes
// of the second operand, 4-7 of the first): low half <- group g, high half
// <- group g+1; after the bit-matrix transpose byte r of idx4[q] holds, at
// bit jj, worker 8(g + (r>>1)) + jj's bit for element q + 8 (r & 1) of the
// half.
template <typename Acc>
__device__ __forceinline__ void lookup_step(Acc (&S)[16], const uint32_t* w, uint32_t sel,
                                            const Acc* tab, int g) {
    uint32_t idx4[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) idx4[jj] = __builtin_amdgcn_perm(w[8 + jj], w[jj], sel);
    // pin the packing here (empty asm on its results): the caller reloads
    // w[] right after this step, and the words must be dead by then
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) asm volatile("" : "+v"(idx4[jj]));
    transpose_bytes8(idx4);
    const Acc* ta = tab + (g & 7) * 256;
    const Acc* tb = ta + 256;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        S[q] += ta[idx4[q] & 255u];
        S[q + 8] += ta[(idx4[q] >> 8) & 255u];
        S[q] += tb[(idx4[q] >> 16) & 255u];
        S[q + 8] += tb[idx4[q] >> 24];
    }
}

// Half of a step for the register-lean fp64 path: only elements
// q + 8 half (q < 8) of the lane's sixteen.
__device__ __forceinline__ void lookup_step_half(double (&S)[8], const uint32_t* w, uint32_t sel,
                                                 const double* tab, int g, int half) {
    uint32_t idx4[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) idx4[jj] = __builtin_amdgcn_perm(w[8 + jj], w[jj], sel);
    transpose_bytes8(idx4);
    const double* ta = tab + (g & 7) * 256;
    const double* tb = ta + 256;
    const int sh = 8 * half;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        S[q] += ta[(idx4[q] >> sh) & 255u];
        S[q] += tb[(idx4[q] >> (16 + sh)) & 255u];
    }
}

// Scales of tensor t into sc[] and its form: 0 ordered, 1 int32 exact,
// 2 fp64 exact; emin = smallest biased exponent of its normal scales.
__device__ __forceinline__ void tensor_form(const uint64_t* __restrict__ wp, int W, int t, float* sc,
                                            int* emin_sh, int* emax_sh, int* bad_sh, int span_limit,
                                            int int_span_limit, int& form, int& emin) {
    __syncthreads();  // the previous tensor's scales and tables are done with
    if (threadIdx.x == 0) {
        *emin_sh = 1000;
        *emax_sh = -1000;
        *bad_sh = 0;
    }
    __syncthreads();
    for (int w = threadIdx.x; w < W; w += kBlock) {
        const float sv = ((cf32p)w_b(wp, W, w))[t];
        sc[w] = sv;
        const uint32_t e = (f2u(sv) >> 23) & 255u;
        if (e == 255u || (e == 0u && (f2u(sv) & 0x7FFFFFu))) atomicOr(bad_sh, 1);
        else if (e) {
            atomicMin(emin_sh, (int)e);
            atomicMax(emax_sh, (int)e);
        }
    }
    __syncthreads();
    const int span = *emax_sh < *emin_sh ? 0 : *emax_sh - *emin_sh;
    form = *bad_sh ? 0 : span <= int_span_limit ? 1 : span <= span_limit ? 2 : 0;
    emin = *emax_sh < *emin_sh ? 1 : *emin_sh;
}

__device__ __forceinline__ void store16(const ADesc& ad, uint32_t e0, const float (&res)[16]) {
    float* out = ad.out + e0;
    if (e0 + 16u <= ad.n) {
#pragma unroll
        for (int q = 0; q < 16; q += 4) stg4f(out + q, f32x4{res[q], res[q + 1], res[q + 2], res[q + 3]});
    } else {
#pragma unroll
        for (int q = 0; q < 16; ++q)
            if (e0 + q < ad.n) gp(out)[q] = res[q];
    }
}

}  // namespace

// Sign aggregate.  A unit is 4096 output elements (128 words) of one
// tensor; lanes 2i and 2i+1 share word i of the unit, each taking 16 of its
// elements (half h = lane parity covers elements 16h .. 16h+15 of the word).
//
// Exact forms: workers are taken in groups of eight; the 256 possible sums
// of a group's eight +-s_w are tabulated, the eight sign bits of an element
// form the table index, and the sum of the group entries is the exact sum,
// rounded once to fp32 at the end.  When a tensor's scales span at most
// int_span_limit binades every scale is an integer multiple of 2^(emin-150)
// below 2^(24+span), and the whole sum stays below 2^31 in those units:
// tables and sums are int32.  Up to span_limit binades they are fp64 (every
// partial sum exact).  Ordered form (non-finite or subnormal scales, or a
// wider span): worker-ordered fp32 additions.
//
// Two launches: sign_agg_prep (one wave per tensor) classifies each tensor
// and, for up to 64 workers, writes its int32 tables to the workspace;
// aggregate_sign (one workgroup per unit, in unit order, so that the
// workgroups resident at a time read neighbouring words of every payload)
// copies its tensor's int32 tables into LDS and sums the unit.  Units of the
// other forms (rare) take a slower path in the same kernel that is kept lean
// in registers, so that the common form keeps its occupancy.
__global__ __launch_bounds__(64) void sign_agg_prep(const ADesc* __restrict__ a, int T,
                                                    const uint64_t* __restrict__ wp, int W,
                                                    int span_limit, int int_span_limit,
                                                    uint32_t* __restrict__ info,
                                                    int32_t* __restrict__ tabs, int build) {
    // one wave per tensor
    __shared__ float sc[1024];
    __shared__ int32_t sub[8 * 32];
    const int t = blockIdx.x;
    if (a[t].nunits == 0) return;
    const int lane = (int)threadIdx.x;
    int lo = 1000, hi = -1000, bad = 0;
    for (int w = lane; w < W; w += 64) {
        const float sv = ((cf32p)w_b(wp, W, w))[t];
        sc[w] = sv;
        const int e = (int)((f2u(sv) >> 23) & 255u);
        if (e == 255 || (e == 0 && (f2u(sv) & 0x7FFFFFu))) bad = 1;
        else if (e) {
            lo = e < lo ? e : lo;
            hi = e > hi ? e : hi;
        }
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
        const int lo2 = __shfl_xor(lo, m, 64), hi2 = __shfl_xor(hi, m, 64);
        lo = lo2 < lo ? lo2 : lo;
        hi = hi2 > hi ? hi2 : hi;
        bad |= __shfl_xor(bad, m, 64);
    }
    const int span = hi < lo ? 0 : hi - lo;
    const int form = bad ? 0 : span <= int_span_limit ? 1 : span <= span_limit ? 2 : 0;
    const int emin = hi < lo ? 1 : lo;
    if (lane == 0) info[t] = (uint32_t)form | ((uint32_t)emin << 8);
    if (!build || form != 1) return;
    __builtin_amdgcn_wave_barrier();
    // sub[32 gi + 16 hh + p]: sum over workers 8 gi + 4 hh + c, c < 4, of
    // (bit c of p ? -s : +s) in units of 2^(emin-150); zero past W
    for (int x = lane; x < 8 * 32; x += 64) {
        const int w0 = 8 * (x >> 5) + 4 * ((x >> 4) & 1), pat = x & 15;
        int32_t acc = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int32_t sv = w0 + c < W ? scale_units(sc[w0 + c], emin) : 0;
            acc += ((pat >> c) & 1) ? -sv : sv;
        }
        sub[x] = acc;
    }
    __builtin_amdgcn_wave_barrier();
    // tab[256 gi + p] = sub[32 gi + (p & 15)] + sub[32 gi + 16 + (p >> 4)],
    // four entries per lane and store
    int32_t* tt = tabs + (size_t)t * 2048;
    for (int x = 4 * lane; x < 8 * 256; x += 256) {
        const int gi = x >> 8, p0 = x & 255;
        const int32_t hi16 = sub[32 * gi + 16 + (p0 >> 4)];
        u32x4 v;
        v.x = (uint32_t)(sub[32 * gi + ((p0 + 0) & 15)] + hi16);
        v.y = (uint32_t)(sub[32 * gi + ((p0 + 1) & 15)] + hi16);
        v.z = (uint32_t)(sub[32 * gi + ((p0 + 2) & 15)] + hi16);
        v.w = (uint32_t)(sub[32 * gi + ((p0 + 3) & 15)] + hi16);
        *(BC_GLOBAL u32x4*)(gp(tt) + x) = v;
    }
}

template <int kS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(6))) void aggregate_sign(const ADesc* __restrict__ a, int T, uint32_t U,
                                                         const uint64_t* __restrict__ wp, int W,
                                                         float alpha, const uint32_t* __restrict__ info,
                                                         const int32_t* __restrict__ tabs, int fast_ok) {
    // the tables (int32: 8 KiB, fp64: 16 KiB), then, after the last lookup,
    // the unit's 4096 results (16 KiB) on their way to coalesced stores
    __shared__ __attribute__((aligned(16))) float lds[4096];
    __shared__ float sc[1024];
    __shared__ double sub[8 * 32];
    const uint32_t u = blockIdx.x;
    const int t = unit_owner(wp, W, u);
    const uint32_t inf = ((const uint32_t __attribute__((address_space(4)))*)info)[t];
    const int form = (int)(inf & 255u);
    const int emin = (int)((inf >> 8) & 255u);
    const ADesc ad = a[t];
    const uint32_t h = threadIdx.x & 1u;
    const uint32_t sel = h ? 0x07060302u : 0x05040100u;
    const int G = (W + 7) / 8;
    const uint32_t wi = (u - ad.unit0) * (kSignAggUnit / 32u) + (threadIdx.x >> 1);  // word of the tensor
    const bool has = wi < ad.k;
    // lanes past the tensor read its first word (their sums are dropped)
    const uint32_t wload = (uint32_t)(ad.off + (has ? wi : 0u)) * 4u;
    float res[16];
    if (fast_ok && form == 1) {
        // int32 form, up to 64 workers: the tables of the 2 kS groups the
        // steps read (groups past G are zero in the workspace), 16 bytes per
        // lane and load, are requested first, then the words of the 16 kS
        // workers (16 kS = 16 ceil(G/2) = Wp, so every slot exists)
        int32_t* tab = reinterpret_cast<int32_t*>(lds);
        const int32_t* tt = tabs + (size_t)t * 2048;
        u32x4 tv[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int x = 4 * threadIdx.x + 1024 * r;
            tv[r] = x < 512 * kS ? ldg4u(reinterpret_cast<const uint32_t*>(tt) + x) : u32x4{0u, 0u, 0u, 0u};
        }
        uint32_t wv[16 * kS];
#pragma unroll
        for (int jj = 0; jj < 16 * kS; ++jj) wv[jj] = ld_word(w_a(wp, jj), wload);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int x = 4 * threadIdx.x + 1024 * r;
            if (x < 512 * kS) *reinterpret_cast<u32x4*>(tab + x) = tv[r];
        }
        __syncthreads();
        int32_t S[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) S[q] = 0;
#pragma unroll
        for (int st = 0; st < kS; ++st)
            if (2 * st < G) lookup_step<int32_t>(S, wv + 16 * st, sel, tab, 2 * st);
        // exact: |S| < 2^31 and the unit is a power of two
        const double unit = __builtin_ldexp(1.0, emin - 150);
#pragma unroll
        for (int q = 0; q < 16; ++q) res[q] = alpha * (float)((double)S[q] * unit);
    } else {
        // the other forms (rare: scales spread over many binades, or more
        // than 64 workers), kept lean in registers so that they do not cost
        // the int32 form its occupancy
        for (int w = threadIdx.x; w < W; w += kBlock) sc[w] = ((cf32p)w_b(wp, W, w))[t];
        __syncthreads();
        if (form == 0) {
            float acc[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[q] = 0.f;
            for (int w0 = 0; w0 < W; w0 += kSignGroup) {
                uint32_t word[kSignGroup];
                float sv[kSignGroup];
#pragma unroll
                for (int g = 0; g < kSignGroup; ++g) {
                    const int w = w0 + g < W ? w0 + g : W - 1;
                    sv[g] = sc[w];
                    word[g] = ld_word(w_a(wp, w), wload);
                }
#pragma unroll
                for (int g = 0; g < kSignGroup; ++g)
                    if (w0 + g < W) sign_half_accumulate(acc, word[g] >> (16u * h), sv[g]);
            }
#pragma unroll
            for (int q = 0; q < 16; ++q) res[q] = alpha * acc[q];
        } else {
            // fp64 tables (exact for the int32 form's tensors too), the
            // lane's sixteen elements in two halves of eight
            double* tab = reinterpret_cast<double*>(lds);
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                double S[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) S[q] = 0.0;
                for (int g = 0; g < G; g += 2) {
                    if ((g & 7) == 0 && (half == 0 || G > 8)) build_tables<double>(g, W, sc, emin, tab, sub);
                    uint32_t w16[16];
#pragma unroll
                    for (int jj = 0; jj < 16; ++jj) w16[jj] = ld_word(w_a(wp, 8 * g + jj), wload);
                    lookup_step_half(S, w16, sel, tab, g, half);
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) res[8 * half + q] = alpha * (float)S[q];
            }
        }
    }
    // Lane l holds unit elements 16 l .. 16 l + 15.  Through LDS (element e
    // of the unit at lds[e]), store k of the workgroup writes elements
    // 1024 k + 4 l' .. +3 for lane l': every store instruction covers 1 KiB
    // of the output.
    __syncthreads();  // every wave is past its lookups
#pragma unroll
    for (int c = 0; c < 4; ++c)
        *reinterpret_cast<f32x4*>(lds + 16 * threadIdx.x + 4 * c) =
            f32x4{res[4 * c], res[4 * c + 1], res[4 * c + 2], res[4 * c + 3]};
    __syncthreads();
    const uint32_t ebase = (u - ad.unit0) * kSignAggUnit;  // first element of the unit
    const uint32_t nleft = ad.n - ebase;                     // > 0
    float* out = ad.out + ebase;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t e = 1024u * k + 4u * threadIdx.x;  // element of the unit
        const f32x4 v = *reinterpret_cast<const f32x4*>(lds + e);
        if (e + 4u <= nleft) {
            stg4f(out + e, v);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (e + q < nleft) gp(out)[e + q] = v[q];
        }
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
uint32_t sparse_agg_tile(uint64_t n_total, uint64_t k_total) {
    // 4096-element tiles while a worker holds about 48 entries per tile or
    // fewer (one 64-entry window covers its entries), 2048 otherwise
    return k_total * 4096u <= n_total * 48u ? 4096u : 2048u;
}

namespace {
template <uint32_t kTS, int kS, bool kLanes>
void launch_sparse_t(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                     hipStream_t s) {
    const size_t lds = (size_t)4 * (kTS * 4 + (kLanes ? 0 : (size_t)W * 4));
    // one round of resident workgroups at this LDS size (more waves with
    // shorter runs measured slower)
    size_t per_cu = (160u * 1024u) / lds;
    if (per_cu < 1) per_cu = 1;
    if (per_cu > 8) per_cu = 8;
    uint64_t blocks = (U + 3) / 4;
    const uint64_t cap = per_cu * (uint64_t)(cus > 0 ? cus : 256);
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL((aggregate_sparse<kTS, kS, kLanes>), dim3((uint32_t)blocks), dim3(kBlock), lds, s, a, T, U,
                       w, W, alpha);
}
template <uint32_t kTS>
void launch_sparse_ts(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                      hipStream_t s) {
    if (W > 64) {
        launch_sparse_t<kTS, 16, false>(a, T, U, w, W, alpha, cus, s);
    } else if (W % 16 == 0 || W % 8 != 0) {
        launch_sparse_t<kTS, 16, true>(a, T, U, w, W, alpha, cus, s);
    } else {
        launch_sparse_t<kTS, 8, true>(a, T, U, w, W, alpha, cus, s);
    }
}
}  // namespace

hipError_t launch_aggregate_sparse(const ADesc* a, int T, uint32_t U, uint32_t tile, const uint64_t* w, int W,
                                   float alpha, int cus, hipStream_t s) {
    if (U == 0) return hipSuccess;
    if (tile == 4096u) launch_sparse_ts<4096u>(a, T, U, w, W, alpha, cus, s);
    else if (tile == 2048u) launch_sparse_ts<2048u>(a, T, U, w, W, alpha, cus, s);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_aggregate_sign(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W,
                                 float alpha, uint32_t* info, int32_t* tabs, hipStream_t s) {
    if (U == 0) return hipSuccess;
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    const int span_limit = 29 - lg;  // 24 + span + ceil(log2 W) <= 53
    const int G = (W + 7) / 8;
    int lg8 = 0;
    while ((1 << lg8) < 8 * G) ++lg8;
    const int int_span_limit = 7 - lg8;  // 24 + span + ceil(log2 8G) <= 31
    // the int32 tables (and the fast path) serve up to 64 workers
    const int small = G <= 8;
    hipLaunchKernelGGL(sign_agg_prep, dim3(T), dim3(64), 0, s, a, T, w, W, span_limit, int_span_limit, info,
                       tabs, small);
    const int steps = small ? (G + 1) / 2 : 1;
    const dim3 grid(U), block(kBlock);
    const uint32_t* ci = info;
    const int32_t* ct = tabs;
    if (steps <= 1)
        hipLaunchKernelGGL(aggregate_sign<1>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    else if (steps == 2)
        hipLaunchKernelGGL(aggregate_sign<2>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    else if (steps == 3)
        hipLaunchKernelGGL(aggregate_sign<3>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    else
        hipLaunchKernelGGL(aggregate_sign<4>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
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
