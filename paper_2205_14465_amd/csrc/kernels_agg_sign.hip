// kernels_agg_sign.hip -- 1-bit sign decompress-and-aggregate of W workers'
// payloads on gfx950 (paper Sec. 3.1, Reason #2: each node decompresses the
// gathered payloads and aggregates them; Sec. 4.2.1, Dimension 3: not an
// Allreduce).
//
// out_t[i] = alpha * fl32(exact sum over w of d_w,i), d_w,i = -s_w,t when
// worker w's bit i is set, else +s_w,t: the exact real sum rounded once.
// A one-wave prep kernel classifies each tensor by the binary exponents of
// its W scales and builds its lookup tables: int32 tables of eight-worker
// partial sums (in units of the smallest scale's last place) when the
// exponents span few enough binades for 32-bit sums, fp64 tables while the
// span fits fp64 exactly; other scale sets (wider spans, subnormal or
// non-finite scales) take the multi-word exact path of exact_wide.hpp, so
// every tensor gets the same definition whatever path computes it.
// The aggregate kernel takes one 4096-element unit per workgroup, gathers
// each element's eight-worker bytes with a byte permute and an 8x8 bit
// transpose, sums the table entries, and stores through LDS for coalesced
// writes.
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
// partial sum exact).  Other scale sets (non-finite or subnormal scales, or
// a wider span): the exact sum in 288-bit integer limbs (exact_wide.hpp).
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
            // scales the tables cannot hold exactly: the wide exact path
            // writes the unit's outputs itself
            aggregate_unit_exact_wide<0>(ad, u, wp, W, alpha, sc, reinterpret_cast<unsigned char*>(lds));
            return;
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


// -------------------------------------------------------------- launcher
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
        return launch_timed(kTimedAggSign, aggregate_sign<1>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    if (steps == 2)
        return launch_timed(kTimedAggSign, aggregate_sign<2>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    if (steps == 3)
        return launch_timed(kTimedAggSign, aggregate_sign<3>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
    return launch_timed(kTimedAggSign, aggregate_sign<4>, grid, block, 0, s, a, T, U, w, W, alpha, ci, ct, small);
}

}  // namespace bc
