// kernels_randk.hip -- seeded random-k sparsification with error feedback
// on gfx950 (Randomk at a 1% rate, paper Sec. 5.1; sparsification with
// error feedback, Sec. 2.3).
//
// The k_t indices of tensor t are the images of 0..k_t-1 under a keyed
// pseudorandom permutation of [0, n_t): a balanced four-round Feistel
// network on b-bit integers (b = bit length of n_t - 1, at least 2, rounded
// up to even), restricted to [0, n_t) by cycle-walking (Black & Rogaway,
// CT-RSA 2002).  Round keys: one Philox4x64-10 block keyed by
// (seed, stream 0) at counter (tensor_id, 0, 0, 0), word r folded to 32
// bits; round function: the "lowbias32" integer hash (C. Wellons,
// hash-prospector) of the right half xor the round key.
//
// Instead of sorting the k indices, they are bucketed by the 4096-element
// chunk they fall in (counts, scan, scatter); the streaming pass over each
// chunk then marks its indices in an LDS bitmap, zeroes them in e_new and
// emits (index, v) in index order, which is the sorted payload.
#include "launch.hpp"

namespace bc {

namespace {

constexpr int kScanBlock = kBlock * 16;  // chunk counters per scan block

__device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

__device__ __forceinline__ uint32_t half_bits(uint32_t n) {
    const uint32_t m = n > 1 ? n - 1 : 0;
    uint32_t b = m ? 32u - __clz(m) : 0u;
    if (b < 2) b = 2;
    b += b & 1u;
    return b >> 1;
}

__device__ __forceinline__ uint32_t feistel(uint32_t x, uint32_t h, uint32_t mask, const uint4 rk) {
    uint32_t L = (x >> h) & mask, R = x & mask;
    uint32_t F;
    F = lowbias32(R ^ rk.x) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.y) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.z) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    F = lowbias32(R ^ rk.w) & mask; { uint32_t t = L ^ F; L = R; R = t; }
    return (h >= 16) ? ((L << 16) | R) : ((L << h) | R);
}

// Tensor owning flat payload entry j: largest t with off[t] <= j.
__device__ __forceinline__ int tensor_of_entry(const TDesc* __restrict__ d, int T, uint64_t j) {
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (d[mid].off <= j) lo = mid; else hi = mid - 1;
    }
    return lo;
}

}  // namespace

// Per-call preparation: clear the chunk counters, derive the round keys.
__global__ void randk_prep(const TDesc* __restrict__ d, int T, uint32_t C, uint64_t seed, Ws ws) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < C) ws.r_ccount[i] = 0u;
    const int t = (int)i;
    if (t >= T) return;
    U64x4 ctr = {{(uint64_t)d[t].tid, 0, 0, 0}};
    const U64x4 w = philox4x64_10(ctr, seed, kStreamRandk);
#pragma unroll
    for (int r = 0; r < 4; ++r) ws.r_keys[4 * t + r] = (uint32_t)w.v[r] ^ (uint32_t)(w.v[r] >> 32);
}

// One thread per payload entry: generate the index, count it in its chunk.
__global__ __launch_bounds__(kBlock) void randk_gen(const TDesc* __restrict__ d, int T,
                                                    uint64_t sum_k, Ws ws) {
    const uint64_t j = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= sum_k) return;
    const int t = tensor_of_entry(d, T, j);
    const TDesc td = d[t];
    const uint4 rk = *reinterpret_cast<const uint4*>(ws.r_keys + 4 * t);
    const uint32_t h = half_bits(td.n);
    const uint32_t mask = h >= 32 ? 0xFFFFFFFFu : ((1u << h) - 1u);
    uint32_t x = feistel((uint32_t)(j - td.off), h, mask, rk);
    while (x >= td.n) x = feistel(x, h, mask, rk);
    ws.r_tmp[j] = x;
    atomicAdd(ws.r_ccount + td.chunk0 + x / (uint32_t)kChunk, 1u);
}

// Scan, step 1: sum of each block of 4096 chunk counters.
__global__ __launch_bounds__(kBlock) void randk_scan_sums(uint32_t C, Ws ws, uint64_t* bsum) {
    __shared__ uint64_t sh[4];
    const uint32_t b0 = blockIdx.x * (uint32_t)kScanBlock;
    uint64_t x = 0;
    for (int q = 0; q < 16; ++q) {
        const uint32_t c = b0 + q * kBlock + threadIdx.x;
        if (c < C) x += ws.r_ccount[c];
    }
    uint64_t tot;
    block_excl_scan_u64(x, sh, tot);
    if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// Scan, step 2: chunk payload offsets and scatter cursors.
__global__ __launch_bounds__(kBlock) void randk_scan_apply(uint32_t C, Ws ws, const uint64_t* bsum) {
    __shared__ uint64_t sh[4];
    uint64_t pre = 0;
    for (uint32_t b = threadIdx.x; b < blockIdx.x; b += kBlock) pre += bsum[b];
    uint64_t base;
    block_excl_scan_u64(pre, sh, base);
    // thread i owns 16 consecutive counters
    const uint32_t c0 = blockIdx.x * (uint32_t)kScanBlock + threadIdx.x * 16u;
    uint32_t cnt[16];
    uint64_t mine = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        cnt[q] = (c0 + q < C) ? ws.r_ccount[c0 + q] : 0u;
        mine += cnt[q];
    }
    uint64_t tot;
    uint64_t run = base + block_excl_scan_u64(mine, sh, tot);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        if (c0 + q < C) {
            ws.r_coff[c0 + q] = run;
            ws.r_cursor[c0 + q] = run;
        }
        run += cnt[q];
    }
    if (c0 < C && c0 + 16 >= C) ws.r_coff[C] = run;  // the thread holding the last counter
}

// Scatter each generated index into its chunk's bucket of the payload.
__global__ __launch_bounds__(kBlock) void randk_scatter(const TDesc* __restrict__ d, int T,
                                                        uint64_t sum_k, uint32_t* __restrict__ idx,
                                                        Ws ws) {
    const uint64_t j = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= sum_k) return;
    const int t = tensor_of_entry(d, T, j);
    const uint32_t x = ws.r_tmp[j];
    const uint32_t c = d[t].chunk0 + x / (uint32_t)kChunk;
    const unsigned long long pos = atomicAdd(ws.r_cursor + c, 1ull);
    if (pos < sum_k) idx[pos] = x;
}

// Stream pass: mark the chunk's indices, write e_new, emit sorted entries.
__global__ __launch_bounds__(kBlock) void randk_stream(const TDesc* __restrict__ d, int T,
                                                       uint32_t* __restrict__ idx,
                                                       float* __restrict__ val, Ws ws) {
    __shared__ uint32_t bm[kChunkWords];
    __shared__ uint64_t sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    const uint32_t lo = j * (uint32_t)kChunk;
    const uint64_t beg = ws.r_coff[c], end = ws.r_coff[c + 1];
    if (threadIdx.x < kChunkWords) bm[threadIdx.x] = 0u;
    __syncthreads();
    for (uint64_t i = beg + threadIdx.x; i < end; i += kBlock) {
        const uint32_t e = idx[i] - lo;
        if (e < (uint32_t)kChunk) atomicOr(&bm[e >> 5], 1u << (e & 31));
    }
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, td.resid != nullptr, v, valid);
    __syncthreads();
    uint32_t pm = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t word = bm[32 * r + (threadIdx.x >> 3)];
        pm |= ((word >> (4 * (threadIdx.x & 7))) & 0xFu) << (4 * r);
    }
    pm &= valid;
    if (td.resid) {
        float e_new[kEpt];
#pragma unroll
        for (int i = 0; i < kEpt; ++i) e_new[i] = ((pm >> i) & 1u) ? 0.f : v[i];
        store_chunk(td.resid, td.n, j, e_new);
    }
    uint64_t packed = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) packed |= (uint64_t)__popc((pm >> (4 * r)) & 0xFu) << (16 * r);
    uint64_t tot;
    const uint64_t pre = block_excl_scan_u64(packed, sh, tot);
    uint64_t base = beg;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        uint64_t at = base + ((pre >> (16 * r)) & 0xFFFFu);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = 4 * r + q;
            if ((pm >> i) & 1u) {
                idx[at] = lo + 1024u * r + 4u * threadIdx.x + q;
                val[at] = v[i];
                ++at;
            }
        }
        base += (tot >> (16 * r)) & 0xFFFFu;
    }
}

hipError_t launch_randk(uint64_t seed, const TDesc* d, int T, uint32_t C, uint64_t sum_k, bool,
                        bool, uint32_t* idx, float* val, const Ws& ws, hipStream_t s) {
    if (C == 0 || T == 0) return hipSuccess;
    const dim3 blk(kBlock);
    const uint32_t nb = (C + kScanBlock - 1) / kScanBlock;
    uint64_t* bsum = ws.r_coff + (size_t)C + 1;  // scratch after the offsets
    const uint32_t prep = ((uint32_t)T > C ? (uint32_t)T : C);
    hipLaunchKernelGGL(randk_prep, dim3((prep + 255) / 256), dim3(256), 0, s, d, T, C, seed, ws);
    if (sum_k) {
        const uint64_t g = (sum_k + kBlock - 1) / kBlock;
        hipLaunchKernelGGL(randk_gen, dim3((uint32_t)g), blk, 0, s, d, T, sum_k, ws);
    }
    hipLaunchKernelGGL(randk_scan_sums, dim3(nb), blk, 0, s, C, ws, bsum);
    hipLaunchKernelGGL(randk_scan_apply, dim3(nb), blk, 0, s, C, ws, bsum);
    if (sum_k) {
        const uint64_t g = (sum_k + kBlock - 1) / kBlock;
        hipLaunchKernelGGL(randk_scatter, dim3((uint32_t)g), blk, 0, s, d, T, sum_k, idx, ws);
    }
    hipLaunchKernelGGL(randk_stream, dim3(C), blk, 0, s, d, T, idx, val, ws);
    return hipGetLastError();
}

}  // namespace bc
