// exact_wide.hpp -- the order-free exact sum of the decoded values of W
// workers for the aggregate kinds whose decoded values are 0 or +-scale
// (1-bit sign, 2-bit TernGrad), for scale sets that the table paths of
// those kernels cannot hold exactly: scales whose binary exponents spread
// over many binades, subnormal scales, infinities and NaNs.
//
// The aggregate is the sum that every order of exact arithmetic reaches
// (each node sums the decompressed payloads, paper Sec. 3.1, Reason #2; the
// paper fixes no addition order): NaN when a decoded value is NaN or when
// both infinities occur, an infinity when one occurs, otherwise the exact
// real sum of the finite values rounded once to fp32 (nearest, ties to
// even; an exact zero gives +0.0; past the fp32 range, an infinity).
//
// Arithmetic.  A finite nonzero scale is m * 2^(E - 150) with m < 2^24 and
// E = max(biased exponent, 1).  With Emin the smallest E of the unit's
// tensor, a decoded value is +-m * 2^sh in units of 2^(Emin - 150),
// sh = E - Emin <= 253.  The sum is held per element in nine int64 limbs of
// 32-bit weight 2^(32 j): m << (sh mod 32) (< 2^56) adds its low word to
// limb sh / 32 and its high word to the next, so no limb ever carries (each
// takes at most 2 W terms below 2^32 in magnitude: |limb| < 2^43 for
// W <= 1024).  Workers are bucketed by their limb so that every limb index
// is a compile-time constant.  At the end the carries are propagated, the
// 288-bit two's-complement total (|total| < 2^287) is turned into sign and
// magnitude, and the magnitude is rounded to 24 significant bits.  Totals
// below 2^24 are exact in fp32 at any Emin >= 1; larger ones round to a
// normal number or overflow, so subnormal results never round.
//
// This path is register-lean (two elements per lane at a time) and serves
// rare scale sets; it is not tuned for speed.
#pragma once

#include "launch.hpp"

namespace bc {

constexpr int kWideLimbs = 9;                 // 288-bit sums
constexpr int kWideScratchBytes = 2048 + 96;  // LDS: worker order + bucket bounds

namespace wide {

// Bucket of a scale: 0..7 the limb of a finite nonzero scale, 8 a NaN or an
// infinity, 9 zero (contributes nothing).
__host__ __device__ __forceinline__ int bucket_of(uint32_t b, int emin) {
    const uint32_t e = (b >> 23) & 255u;
    if (e == 255u) return 8;
    if ((b & 0x7FFFFFFFu) == 0u) return 9;
    const int E = e ? (int)e : 1;
    return (E - emin) >> 5;
}

// Decoded value of worker bits for one element: `act` whether it is
// nonzero (TernGrad level 1, always for sign), `neg` its sign relative to
// the scale's magnitude.
template <int kKind>
__device__ __forceinline__ void decode_bits(uint32_t word, uint32_t pos, uint32_t sbits, bool& act, bool& neg) {
    if constexpr (kKind == 0) {  // sign: bit set -> -s
        act = true;
        neg = (((word >> pos) ^ (sbits >> 31)) & 1u) != 0u;
    } else {                     // TernGrad: level bit, then sign bit
        const uint32_t code = (word >> pos) & 3u;
        act = (code & 1u) != 0u;
        neg = (((code >> 1) ^ (sbits >> 31)) & 1u) != 0u;
    }
}

// Round a 288-bit two's-complement total in units of 2^(emin - 150).
__host__ __device__ __forceinline__ float round_total(int64_t (&acc)[kWideLimbs], int emin) {
    uint32_t d[kWideLimbs];
#pragma unroll
    for (int j = 0; j + 1 < kWideLimbs; ++j) {
        acc[j + 1] += acc[j] >> 32;  // arithmetic shift: the signed carry
        d[j] = (uint32_t)acc[j];
    }
    d[kWideLimbs - 1] = (uint32_t)acc[kWideLimbs - 1];
    const bool neg = acc[kWideLimbs - 1] < 0;
    if (neg) {  // magnitude = ~total + 1
        uint32_t c = 1u;
#pragma unroll
        for (int j = 0; j < kWideLimbs; ++j) {
            const uint32_t x = ~d[j] + c;
            c = (c && x == 0u) ? 1u : 0u;
            d[j] = x;
        }
    }
    int top = -1;
#pragma unroll
    for (int j = kWideLimbs - 1; j >= 0; --j) top = (top < 0 && d[j] != 0u) ? j : top;
    if (top < 0) return 0.0f;  // an exact zero rounds to +0.0
    uint32_t dt = 0u, dn = 0u, below = 0u;
#pragma unroll
    for (int j = 0; j < kWideLimbs; ++j) {
        dt = j == top ? d[j] : dt;
        dn = j == top - 1 ? d[j] : dn;
        below |= j < top - 1 ? d[j] : 0u;
    }
    const int hb = 31 - __builtin_clz(dt);
    const int h = 32 * top + hb;  // highest set bit of the magnitude
    float mag;
    if (h < 24) {
        mag = __builtin_ldexpf((float)d[0], emin - 150);  // fewer than 25 bits: exact
    } else {
        const uint64_t win = ((uint64_t)dt << 32) | dn;  // bit h at 32 + hb
        uint32_t mant = (uint32_t)(win >> (9 + hb)) & 0xFFFFFFu;
        const uint32_t rb = (uint32_t)(win >> (8 + hb)) & 1u;
        const bool sticky = (win & ((1ull << (8 + hb)) - 1ull)) != 0ull || below != 0u;
        mant += rb & ((sticky ? 1u : 0u) | (mant & 1u));
        mag = __builtin_ldexpf((float)mant, h - 23 + emin - 150);  // overflow gives +inf
    }
    return neg ? -mag : mag;
}

}  // namespace wide

// One work unit (kSignAggUnit elements of one tensor) through the exact
// wide path; called by the whole workgroup, which then has nothing else to
// do for the unit.  kKind 0: 1-bit sign payloads (element i at bit i mod 32
// of word i / 32); 1: 2-bit TernGrad payloads (element i at bits 2 (i mod
// 16) of word i / 16).  sc: the tensor's W scales in LDS (read only);
// scratch: kWideScratchBytes of LDS.  Results go straight to the output.
// The unit's output elements are ebase .. ebase + kSignAggUnit - 1 of the
// tensor (ebase may be negative: elements outside [0, n) are skipped).
template <int kKind>
__device__ void aggregate_unit_exact_wide(const ADesc& ad, int64_t ebase, const uint64_t* __restrict__ wp, int W,
                                          float alpha, const float* sc, unsigned char* scratch) {
    uint16_t* order = reinterpret_cast<uint16_t*>(scratch);          // [1024]
    int* cursor = reinterpret_cast<int*>(scratch + 2048);             // [10]
    int* start = cursor + 10;                                         // [11]
    int* emin_sh = start + 11;
    __syncthreads();  // callers may have used the scratch
    if (threadIdx.x < 10) cursor[threadIdx.x] = 0;
    if (threadIdx.x == 0) *emin_sh = 1000;
    __syncthreads();
    for (int w = threadIdx.x; w < W; w += kBlock) {
        const uint32_t b = f2u(sc[w]);
        const uint32_t e = (b >> 23) & 255u;
        if (e != 255u && (b & 0x7FFFFFFFu) != 0u) atomicMin(emin_sh, e ? (int)e : 1);
    }
    __syncthreads();
    const int emin = *emin_sh == 1000 ? 1 : *emin_sh;
    for (int w = threadIdx.x; w < W; w += kBlock) atomicAdd(&cursor[wide::bucket_of(f2u(sc[w]), emin)], 1);
    __syncthreads();
    if (threadIdx.x == 0) {
        int at = 0;
        for (int bk = 0; bk < 10; ++bk) {
            start[bk] = at;
            at += cursor[bk];
            cursor[bk] = start[bk];
        }
        start[10] = at;
    }
    __syncthreads();
    for (int w = threadIdx.x; w < W; w += kBlock) {
        const int bk = wide::bucket_of(f2u(sc[w]), emin);
        order[atomicAdd(&cursor[bk], 1)] = (uint16_t)w;  // order within a bucket is immaterial
    }
    __syncthreads();

    constexpr int kE = 2;  // elements per lane and pass
    for (int q0 = 0; q0 < (int)(kSignAggUnit / kBlock); q0 += kE) {
        uint32_t el[kE], wofs[kE], pos[kE];
        bool ok[kE];
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            const int64_t ge = ebase + (int64_t)threadIdx.x + (int64_t)kBlock * (q0 + i);
            ok[i] = ge >= 0 && ge < (int64_t)ad.n;
            el[i] = ok[i] ? (uint32_t)ge : 0u;
            const uint32_t e = el[i];  // lanes outside the tensor read its first word
            wofs[i] = (uint32_t)ad.off + (kKind == 0 ? e >> 5 : e >> 4);
            pos[i] = kKind == 0 ? (e & 31u) : 2u * (e & 15u);
        }
        int64_t acc[kE][kWideLimbs];
#pragma unroll
        for (int i = 0; i < kE; ++i)
#pragma unroll
            for (int j = 0; j < kWideLimbs; ++j) acc[i][j] = 0;
#pragma unroll
        for (int L = 0; L < 8; ++L) {
            const int p1 = __builtin_amdgcn_readfirstlane(start[L + 1]);
            for (int p = __builtin_amdgcn_readfirstlane(start[L]); p < p1; ++p) {
                const int w = __builtin_amdgcn_readfirstlane((int)order[p]);
                const uint32_t sb = f2u(sc[w]);
                const uint32_t* base = w_a(wp, w);
                uint32_t word[kE];
#pragma unroll
                for (int i = 0; i < kE; ++i) word[i] = gp(base)[wofs[i]];
                const uint32_t e = (sb >> 23) & 255u;
                const int r = ((e ? (int)e : 1) - emin) & 31;
                const uint64_t c = (uint64_t)((sb & 0x7FFFFFu) | (e ? 0x800000u : 0u)) << r;
                const int64_t lo = (int64_t)(uint32_t)c, hi = (int64_t)(uint32_t)(c >> 32);
#pragma unroll
                for (int i = 0; i < kE; ++i) {
                    bool act, neg;
                    wide::decode_bits<kKind>(word[i], pos[i], sb, act, neg);
                    const int64_t a = act ? (neg ? -lo : lo) : 0, b = act ? (neg ? -hi : hi) : 0;
                    acc[i][L] += a;
                    acc[i][L + 1] += b;
                }
            }
        }
        // NaN and infinite scales
        uint32_t nan_m = 0u, pinf_m = 0u, ninf_m = 0u;
        {
            const int p1 = __builtin_amdgcn_readfirstlane(start[9]);
            for (int p = __builtin_amdgcn_readfirstlane(start[8]); p < p1; ++p) {
                const int w = __builtin_amdgcn_readfirstlane((int)order[p]);
                const uint32_t sb = f2u(sc[w]);
                const bool is_nan = (sb & 0x7FFFFFu) != 0u;
#pragma unroll
                for (int i = 0; i < kE; ++i) {
                    bool act, neg;
                    wide::decode_bits<kKind>(gp(w_a(wp, w))[wofs[i]], pos[i], sb, act, neg);
                    if (act) {
                        if (is_nan) nan_m |= 1u << i;
                        else if (neg) ninf_m |= 1u << i;
                        else pinf_m |= 1u << i;
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            float r = wide::round_total(acc[i], emin);
            const bool pinf = (pinf_m >> i) & 1u, ninf = (ninf_m >> i) & 1u;
            if (((nan_m >> i) & 1u) || (pinf && ninf)) r = __builtin_nanf("");
            else if (pinf) r = __builtin_inff();
            else if (ninf) r = -__builtin_inff();
            if (ok[i]) gp(ad.out)[el[i]] = alpha * r;
        }
    }
}

}  // namespace bc
