// kernels_part.hip -- the divisible scheme's packing step on gfx950 (paper
// Sec. 3.1, Reason #2, and the alltoall figure: a compressed tensor is
// partitioned into parts and node j receives part j from every node, then
// decompresses, aggregates and compresses it again).
//
// Parts are element ranges [lo, hi) of every tensor.  Packing part j of a
// sparse payload keeps, tensor by tensor, the entries whose index lies in
// the range, in payload order, with the index rebased to the range; a sign
// or quantizer payload (b bits per element) keeps the words that cover the
// range (lo is a multiple of 32, so the range starts on a word) and every
// tensor's scale.  part_off receives the packed offsets of the tensors:
// entries (sparse) or words (sign, quantizers), T + 1 values.
#include "launch.hpp"

namespace bc {

namespace {

// First position p in [0, k) with idx[p] >= x (k if none), found by a
// whole wave: each round probes 64 evenly spaced positions
// of the interval that holds the answer and keeps the one gap between a
// probe below x and the next, so a round divides the interval by 65.
__device__ __forceinline__ uint32_t wave_lower_bound(const uint32_t* idx, uint32_t k, uint32_t x) {
    if (k == 0) return 0;
    const uint32_t lane = (uint32_t)lane_id();
    uint32_t lo = 0, hi = k;  // the answer lies in [lo, hi]
    while (hi - lo > 64u) {
        const uint64_t len = hi - lo;
        const uint32_t pos = lo + (uint32_t)((len * (lane + 1u)) / 65u);
        const uint32_t c = (uint32_t)__popcll(__ballot(gp(idx)[pos] < x));
        const uint32_t nlo = c ? lo + (uint32_t)((len * c) / 65u) + 1u : lo;
        const uint32_t nhi = c < 64u ? lo + (uint32_t)((len * (c + 1u)) / 65u) : hi;
        lo = nlo;
        hi = nhi;
    }
    const bool below = lo + lane < hi && gp(idx)[lo + lane < hi ? lo + lane : lo] < x;
    return lo + (uint32_t)__popcll(__ballot(below));
}

}  // namespace

// Sparse: entries of tensor t in [lo, hi): one wave per tensor.
__global__ __launch_bounds__(kBlock) void part_count(const PDesc* __restrict__ p, int T,
                                                     const uint32_t* __restrict__ idx,
                                                     uint64_t* __restrict__ part_off) {
    const int t = (int)(blockIdx.x * (kBlock / 64) + wave_id());
    if (t >= T) return;
    const PDesc pd = p[t];
    const uint32_t* ix = idx + pd.in_off;
    const uint32_t a = wave_lower_bound(ix, pd.k, pd.lo);
    const uint32_t b = wave_lower_bound(ix, pd.k, pd.hi);
    if (lane_id() == 0) part_off[t] = b - a;
}

// In-place exclusive prefix of T counts into T + 1 offsets: one workgroup,
// each thread a run of consecutive counts.
__global__ __launch_bounds__(1024) void part_scan(int T, uint64_t* __restrict__ part_off) {
    __shared__ uint64_t wsum[16];
    const uint32_t per = ((uint32_t)T + 1023u) / 1024u;
    const uint32_t b = threadIdx.x * per;
    const uint32_t e = b + per < (uint32_t)T ? b + per : (uint32_t)T;
    uint64_t mine = 0;
    for (uint32_t i = b; i < e; ++i) mine += part_off[i];
    // block-wide exclusive scan of `mine`
    const int lane = lane_id(), w = threadIdx.x >> 6;
    uint64_t inc = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    uint64_t before = 0, total = 0;
    for (int q = 0; q < 16; ++q) {
        before += q < w ? wsum[q] : 0u;
        total += wsum[q];
    }
    uint64_t run = before + inc - mine;
    for (uint32_t i = b; i < e; ++i) {
        const uint64_t c = part_off[i];
        part_off[i] = run;
        run += c;
    }
    if (threadIdx.x == 0) part_off[T] = total;
}

// Sparse: copy the packed positions [4096 b, 4096 (b+1)) of the part: the
// tensors covering them in order, each tensor's range entries rebased.
constexpr uint32_t kPackSpan = 4096;

__global__ __launch_bounds__(kBlock) void part_copy_sparse(const PDesc* __restrict__ p, int T,
                                                           const uint32_t* __restrict__ in_idx,
                                                           const float* __restrict__ in_val,
                                                           uint32_t* __restrict__ out_idx,
                                                           float* __restrict__ out_val,
                                                           const uint64_t* __restrict__ part_off) {
    __shared__ int t0_sh;
    __shared__ uint32_t first_sh;
    const uint64_t total = part_off[T];
    const uint64_t b0 = (uint64_t)blockIdx.x * kPackSpan;
    if (b0 >= total) return;
    const uint64_t b1 = b0 + kPackSpan < total ? b0 + kPackSpan : total;
    if (threadIdx.x == 0) {
        // last tensor whose part starts at or before b0
        int lo = 0, hi = T - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (part_off[mid] <= b0) lo = mid; else hi = mid - 1;
        }
        t0_sh = lo;
    }
    __syncthreads();
    for (int t = t0_sh; t < T && part_off[t] < b1; ++t) {
        const uint64_t o0 = part_off[t], o1 = part_off[t + 1];
        const uint64_t s0 = o0 > b0 ? o0 : b0, s1 = o1 < b1 ? o1 : b1;
        if (s0 >= s1) continue;  // uniform: every thread reads the same offsets
        const PDesc pd = p[t];
        __syncthreads();  // the previous tensor is done with first_sh
        if (threadIdx.x < 64) {
            const uint32_t f = wave_lower_bound(in_idx + pd.in_off, pd.k, pd.lo);
            if (threadIdx.x == 0) first_sh = f;
        }
        __syncthreads();
        const uint64_t src0 = pd.in_off + first_sh + (s0 - o0);
        const uint32_t cnt = (uint32_t)(s1 - s0);
        for (uint32_t i = threadIdx.x; i < cnt; i += kBlock) {
            out_idx[s0 + i] = gp(in_idx)[src0 + i] - pd.lo;
            out_val[s0 + i] = gp(in_val)[src0 + i];
        }
    }
}

// Sign and quantizers (`bits` per element): copy tensor t's range words
// and its scale; part_off gets the (host-computed) word offsets.
__global__ __launch_bounds__(kBlock) void part_copy_words(const PDesc* __restrict__ p, int T, uint32_t bits,
                                                          const uint32_t* __restrict__ in_bits,
                                                          const float* __restrict__ in_scale,
                                                          uint32_t* __restrict__ out_bits,
                                                          float* __restrict__ out_scale,
                                                          uint64_t* __restrict__ part_off, uint64_t total) {
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        const PDesc pd = p[t];
        // bits per element: the range starts on a word (lo is a multiple of 32)
        const uint32_t nw = (uint32_t)(((uint64_t)(pd.hi - pd.lo) * bits + 31u) / 32u);
        const uint64_t src = pd.in_off + (uint64_t)pd.lo / 32u * bits;
        for (uint32_t i = threadIdx.x; i < nw; i += kBlock) out_bits[pd.out_off + i] = gp(in_bits)[src + i];
        if (threadIdx.x == 0) {
            out_scale[t] = gp(in_scale)[t];
            part_off[t] = pd.out_off;
            if (t == 0) part_off[T] = total;
        }
    }
}

hipError_t launch_pack_part(int word_bits, const PDesc* p, int T, bc_payload_dev in, bc_payload_dev out,
                            uint64_t* part_off, uint64_t words, uint64_t max_entries, int cus, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const uint32_t grid = (uint32_t)(T < 4 * cus ? T : 4 * cus);
    if (word_bits) {
        hipLaunchKernelGGL(part_copy_words, dim3(grid), dim3(kBlock), 0, s, p, T, (uint32_t)word_bits, in.bits,
                           in.scale, out.bits, out.scale, part_off, words);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(part_count, dim3((T + 3) / 4), dim3(kBlock), 0, s, p, T, in.idx, part_off);
    hipLaunchKernelGGL(part_scan, dim3(1), dim3(1024), 0, s, T, part_off);
    const uint64_t blocks = (max_entries + kPackSpan - 1) / kPackSpan;
    if (blocks)
        hipLaunchKernelGGL(part_copy_sparse, dim3((uint32_t)blocks), dim3(kBlock), 0, s, p, T, in.idx, in.val,
                           out.idx, out.val, part_off);
    return hipGetLastError();
}

}  // namespace bc
