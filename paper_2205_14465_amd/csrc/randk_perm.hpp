// randk_perm.hpp -- the keyed permutation behind seeded random-k (Randomk,
// paper Sec. 5.1), shared by the GPU kernels and the host compressor: a
// balanced four-round Feistel network on b-bit integers (b = bit length of
// n - 1, at least 2, rounded up to even; half width h = b / 2), restricted
// to [0, n) by cycle-walking (Black & Rogaway, CT-RSA 2002).  The round
// function is the "lowbias32" integer hash (C. Wellons, hash-prospector) of
// the right half xor the round key; the four round keys are the words of one
// Philox4x64-10 block keyed by (seed, stream 0) at counter (tensor_id, 0, 0,
// 0), each folded to 32 bits (high xor low).
#pragma once

#include "common.hpp"

namespace bc {

__host__ __device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// Half width h of the Feistel domain of a tensor of n elements.
__host__ __device__ __forceinline__ uint32_t half_bits(uint32_t n) {
    const uint32_t m = n > 1 ? n - 1 : 0;
    uint32_t b = m ? 32u - (uint32_t)__builtin_clz(m) : 0u;
    if (b < 2) b = 2;
    b += b & 1u;
    return b >> 1;
}

__host__ __device__ __forceinline__ uint32_t feistel(uint32_t x, uint32_t h, uint32_t mask, const uint4 rk) {
    uint32_t L = (x >> h) & mask, R = x & mask;
    uint32_t F;
    F = lowbias32(R ^ rk.x) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.y) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.z) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.w) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    return (h >= 16) ? ((L << 16) | R) : ((L << h) | R);
}

// Round keys of tensor `tid` under `seed`.
__host__ __device__ __forceinline__ uint4 randk_round_keys(uint64_t seed, uint32_t tid) {
    U64x4 ctr = {{(uint64_t)tid, 0, 0, 0}};
    const U64x4 w = philox4x64_10(ctr, seed, kStreamRandk);
    uint4 rk;
    rk.x = (uint32_t)w.v[0] ^ (uint32_t)(w.v[0] >> 32);
    rk.y = (uint32_t)w.v[1] ^ (uint32_t)(w.v[1] >> 32);
    rk.z = (uint32_t)w.v[2] ^ (uint32_t)(w.v[2] >> 32);
    rk.w = (uint32_t)w.v[3] ^ (uint32_t)(w.v[3] >> 32);
    return rk;
}

}  // namespace bc
