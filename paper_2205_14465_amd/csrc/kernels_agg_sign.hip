// kernels_agg_sign.hip -- 1-bit sign decompress-and-aggregate of W workers'
// payloads on gfx950 (paper Sec. 3.1, Reason #2: each node decompresses the
// gathered payloads and aggregates them; Sec. 4.2.1, Dimension 3: not an
// Allreduce).
//
// out_t[i] = alpha * fl32(exact sum over w of d_w,i), d_w,i = -s_w,t when
// worker w's bit i is set, else +s_w,t: the exact real sum rounded once.
// One kernel: each workgroup takes one unit of 128 payload words (4096
// elements) of one tensor, classifies the tensor by the binary exponents of
// its W scales and builds its lookup tables in LDS: int32 tables of
// eight-worker partial sums (in units of the smallest scale's last place)
// when the exponents span few enough binades for 32-bit sums, fp64 tables
// while the span fits fp64 exactly; other scale sets (wider spans,
// subnormal or non-finite scales) take the multi-word exact path of
// exact_wide.hpp, so every tensor gets the same definition whatever path
// computes it.  It gathers each element's eight-worker bytes with a byte
// permute and an 8x8 bit transpose, sums the table entries, and stores
// through LDS for coalesced writes.  Units start on 128-byte boundaries of
// the payloads (a tensor's first unit is shortened to reach one), so that
// no cache line of a payload is read by two units of a tensor.
#include "exact_wide.hpp"
#include "launch.hpp"

namespace bc {

namespace {

typedef const float __attribute__((address_space(4)))* cf32p;

}  // namespace

namespace {

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

// Workgroup barrier for LDS data: waits for this wave's LDS operations
// only, leaving its global loads in flight (__syncthreads would wait for
// those too, and the payload words requested before the tables are built
// would stop overlapping the build).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

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
__device__ __forceinline__ void build_tables(int g, int W, const float* sc, int emin, Acc* tab, Acc* sub,
                                             int ngroups = 8) {
    lds_barrier();  // earlier lookups are done with the tables
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
    lds_barrier();
    for (int x = threadIdx.x; x < ngroups * 256; x += kBlock) {
        const int gi = x >> 8, pat = x & 255;
        tab[x] = sub[32 * gi + (pat & 15)] + sub[32 * gi + 16 + (pat >> 4)];
    }
    lds_barrier();
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

// Sign aggregate.  A unit is 128 consecutive payload words (4096 output
// elements) of one tensor; lanes 2i and 2i+1 share word i of the unit,
// each taking 16 of its elements (half h = lane parity covers elements
// 16h .. 16h+15 of the word).  Tensor t's unit j covers its words
// 128 j - s .. 128 j - s + 127, s = (payload word offset of the tensor) mod
// 32 (from worker 0's payload address), so that unit boundaries fall on
// 128-byte lines; words outside the tensor are read as its first word and
// their sums dropped.
//
// Exact forms: workers are taken in groups of eight; the 256 possible sums
// of a group's eight +-s_w are tabulated, the eight sign bits of an element
// form the table index, and the sum of the group entries is the exact sum,
// rounded once to fp32 at the end.  When a tensor's scales span at most
// int_span_limit binades every scale is an integer multiple of 2^(emin-150)
// below 2^(24+span), and the whole sum stays below 2^31 in those units:
// tables and sums are int32.  Up to span_limit binades they are fp64 (every
// partial sum exact).  Other scale sets (non-finite or subnormal scales, or
// a wider span): the exact sum in 288-bit integer limbs (exact_wide.hpp).
// Every workgroup classifies its tensor from the W scales and builds the
// tables it needs in LDS; the int32 form for up to 64 workers (fast_ok) is
// the common one, the others take a slower path kept lean in registers, so
// that the common form keeps its occupancy.  Workgroups run in unit order,
// so that the workgroups resident at a time read neighbouring words of
// every payload.
__device__ __forceinline__ uint32_t unit_shift(const uint64_t* __restrict__ wp, const ADesc& ad) {
    return (uint32_t)(((uint64_t)(uintptr_t)w_a(wp, 0) >> 2) + ad.off) & 31u;
}

template <int kS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(5))) void aggregate_sign(const ADesc* __restrict__ a, int T, uint32_t U,
                                                         const uint64_t* __restrict__ wp, int W,
                                                         float alpha, int span_limit, int int_span_limit,
                                                         int fast_ok) {
    // the tables (int32: up to 8 KiB, fp64: 16 KiB), then, after the last
    // lookup, the unit's 4096 results (16 KiB) on their way to coalesced
    // stores
    __shared__ __attribute__((aligned(16))) float lds[4096];
    __shared__ float sc[1024];
    __shared__ double sub[8 * 32];
    __shared__ int red[12];
    const uint32_t u = blockIdx.x;
    const int t = unit_owner(wp, W, u);
    const ADesc ad = a[t];
    const uint32_t h = threadIdx.x & 1u;
    const uint32_t sel = h ? 0x07060302u : 0x05040100u;
    const int G = (W + 7) / 8;
    const uint32_t shift = unit_shift(wp, ad);
    // word of the tensor (wraps past 2^32 below its first word)
    const uint32_t wi = (u - ad.unit0) * (kSignAggUnit / 32u) + (threadIdx.x >> 1) - shift;
    const bool has = wi < ad.k;
    const uint32_t wload = (uint32_t)(ad.off + (has ? wi : 0u)) * 4u;
    const int64_t ebase = ((int64_t)(u - ad.unit0) * (kSignAggUnit / 32u) - shift) * 32;  // unit element 0
    // the tensor's scales (the first kBlock requested before the words, so
    // that waiting for them does not wait for the words)
    const float sv0 = (int)threadIdx.x < W ? ((cf32p)w_b(wp, W, threadIdx.x))[t] : 0.f;
    // the words of the first 16 kS workers (16 kS = 16 ceil(G/2) = Wp for
    // W <= 64, so every slot exists), in flight while the tables are built
    uint32_t wv[16 * kS];
    if (fast_ok) {
#pragma unroll
        for (int jj = 0; jj < 16 * kS; ++jj) wv[jj] = ld_word(w_a(wp, jj), wload);
    }
    // the binades the scales span
    int lo = 1000, hi = -1000, bad = 0;
    for (int w = threadIdx.x; w < W; w += kBlock) {
        const float sv = w == (int)threadIdx.x ? sv0 : ((cf32p)w_b(wp, W, w))[t];
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
    if (lane_id() == 0) {
        red[3 * wave_id()] = lo;
        red[3 * wave_id() + 1] = hi;
        red[3 * wave_id() + 2] = bad;
    }
    lds_barrier();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        lo = red[3 * q] < lo ? red[3 * q] : lo;
        hi = red[3 * q + 1] > hi ? red[3 * q + 1] : hi;
        bad |= red[3 * q + 2];
    }
    const int span = hi < lo ? 0 : hi - lo;
    const int form = bad ? 0 : span <= int_span_limit ? 1 : span <= span_limit ? 2 : 0;
    const int emin = hi < lo ? 1 : lo;
    float res[16];
    if (fast_ok && form == 1) {
        // int32 form, up to 64 workers: the tables of the 2 kS groups the
        // steps read (groups past G are zero: their workers count as zero)
        int32_t* tab = reinterpret_cast<int32_t*>(lds);
        build_tables<int32_t>(0, W, sc, emin, tab, reinterpret_cast<int32_t*>(sub), 2 * kS);
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
    } else if (form == 0) {
        // scales the tables cannot hold exactly: the wide exact path
        // writes the unit's outputs itself
        aggregate_unit_exact_wide<0>(ad, ebase, wp, W, alpha, sc, reinterpret_cast<unsigned char*>(lds));
        return;
    } else {
        // fp64 tables (exact for the int32 form's tensors too), the lane's
        // sixteen elements in two halves of eight
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
    // Lane l holds unit elements 16 l .. 16 l + 15.  Through LDS (element e
    // of the unit at lds[e]), store k of the workgroup writes elements
    // 1024 k + 4 l' .. +3 for lane l': every store instruction covers 1 KiB
    // of the output.  ebase is a multiple of 32, so whole groups of four
    // are inside or outside [0, n) at the tensor's start.
    __syncthreads();  // every wave is past its lookups
#pragma unroll
    for (int c = 0; c < 4; ++c)
        *reinterpret_cast<f32x4*>(lds + 16 * threadIdx.x + 4 * c) =
            f32x4{res[4 * c], res[4 * c + 1], res[4 * c + 2], res[4 * c + 3]};
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t e = 1024u * k + 4u * threadIdx.x;  // element of the unit
        const int64_t g = ebase + e;                       // element of the tensor
        if (g < 0) continue;
        const f32x4 v = *reinterpret_cast<const f32x4*>(lds + e);
        if (g + 4 <= (int64_t)ad.n) {
            stg4f(ad.out + g, v);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (g + q < (int64_t)ad.n) gp(ad.out)[g + q] = v[q];
        }
    }
}


// -------------------------------------------------------------- launcher
hipError_t launch_aggregate_sign(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W,
                                 float alpha, hipStream_t s) {
    if (U == 0) return hipSuccess;
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    const int span_limit = 29 - lg;  // 24 + span + ceil(log2 W) <= 53
    const int G = (W + 7) / 8;
    int lg8 = 0;
    while ((1 << lg8) < 8 * G) ++lg8;
    const int int_span_limit = 7 - lg8;  // 24 + span + ceil(log2 8G) <= 31
    // the int32 form's fast path serves up to 64 workers
    const int small = G <= 8;
    const int steps = small ? (G + 1) / 2 : 1;
    const dim3 grid(U), block(kBlock);
    if (steps <= 1)
        return launch_timed(kTimedAggSign, aggregate_sign<1>, grid, block, 0, s, a, T, U, w, W, alpha, span_limit,
                            int_span_limit, small);
    if (steps == 2)
        return launch_timed(kTimedAggSign, aggregate_sign<2>, grid, block, 0, s, a, T, U, w, W, alpha, span_limit,
                            int_span_limit, small);
    if (steps == 3)
        return launch_timed(kTimedAggSign, aggregate_sign<3>, grid, block, 0, s, a, T, U, w, W, alpha, span_limit,
                            int_span_limit, small);
    return launch_timed(kTimedAggSign, aggregate_sign<4>, grid, block, 0, s, a, T, U, w, W, alpha, span_limit,
                        int_span_limit, small);
}

}  // namespace bc
