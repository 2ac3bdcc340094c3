// kernels_part.hip -- the divisible scheme's packing step on gfx950 (paper
// Sec. 3.1, Reason #2, and the alltoall figure: a compressed tensor is
// partitioned into parts and node j receives part j from every node, then
// decompresses, aggregates and compresses it again).
//
// Parts are element ranges [lo, hi) of every tensor.  Packing part j of a
// sparse payload keeps, tensor by tensor, the entries whose index lies in
// the range, in payload order, with the index rebased to the range; a sign
// payload keeps the words that cover the range (lo is a multiple of 32) and
// every tensor's scale.  part_off receives the packed offsets of the
// tensors: entries (sparse) or words (sign), T + 1 values.
#include "launch.hpp"

namespace bc {

namespace {

// First position p in [0, k) with idx[p] >= x (k if none).
__device__ __forceinline__ uint32_t lower_bound_idx(const uint32_t* idx, uint32_t k, uint32_t x) {
    uint32_t lo = 0, hi = k;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (gp(idx)[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

}  // namespace

// Sparse: entries of tensor t in [lo, hi): one thread per tensor.
__global__ void part_count(const PDesc* __restrict__ p, int T, const uint32_t* __restrict__ idx,
                           uint64_t* __restrict__ part_off) {
    const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (t >= T) return;
    const PDesc pd = p[t];
    const uint32_t* ix = idx + pd.in_off;
    part_off[t] = lower_bound_idx(ix, pd.k, pd.hi) - lower_bound_idx(ix, pd.k, pd.lo);
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

// Sparse: copy tensor t's range entries, rebased; a workgroup per tensor
// (grid-stride over tensors).
__global__ __launch_bounds__(kBlock) void part_copy_sparse(const PDesc* __restrict__ p, int T,
                                                           const uint32_t* __restrict__ in_idx,
                                                           const float* __restrict__ in_val,
                                                           uint32_t* __restrict__ out_idx,
                                                           float* __restrict__ out_val,
                                                           const uint64_t* __restrict__ part_off) {
    __shared__ uint32_t first;
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        const PDesc pd = p[t];
        const uint64_t o = part_off[t];
        const uint32_t cnt = (uint32_t)(part_off[t + 1] - o);
        __syncthreads();  // the previous tensor is done with `first`
        if (threadIdx.x == 0) first = lower_bound_idx(in_idx + pd.in_off, pd.k, pd.lo);
        __syncthreads();
        const uint64_t src = pd.in_off + first;
        for (uint32_t i = threadIdx.x; i < cnt; i += kBlock) {
            out_idx[o + i] = gp(in_idx)[src + i] - pd.lo;
            out_val[o + i] = gp(in_val)[src + i];
        }
    }
}

// Sign: copy tensor t's range words and its scale; part_off gets the
// (host-computed) word offsets.
__global__ __launch_bounds__(kBlock) void part_copy_sign(const PDesc* __restrict__ p, int T,
                                                         const uint32_t* __restrict__ in_bits,
                                                         const float* __restrict__ in_scale,
                                                         uint32_t* __restrict__ out_bits,
                                                         float* __restrict__ out_scale,
                                                         uint64_t* __restrict__ part_off, uint64_t total) {
    for (int t = blockIdx.x; t < T; t += gridDim.x) {
        const PDesc pd = p[t];
        const uint32_t nw = (pd.hi - pd.lo + 31u) / 32u;
        const uint64_t src = pd.in_off + pd.lo / 32u;
        for (uint32_t i = threadIdx.x; i < nw; i += kBlock) out_bits[pd.out_off + i] = gp(in_bits)[src + i];
        if (threadIdx.x == 0) {
            out_scale[t] = gp(in_scale)[t];
            part_off[t] = pd.out_off;
            if (t == 0) part_off[T] = total;
        }
    }
}

hipError_t launch_pack_part(int kind, const PDesc* p, int T, bc_payload_dev in, bc_payload_dev out,
                            uint64_t* part_off, uint64_t sign_words, int cus, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const uint32_t grid = (uint32_t)(T < 4 * cus ? T : 4 * cus);
    if (kind == 3) {
        hipLaunchKernelGGL(part_copy_sign, dim3(grid), dim3(kBlock), 0, s, p, T, in.bits, in.scale, out.bits,
                           out.scale, part_off, sign_words);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(part_count, dim3((T + 255) / 256), dim3(256), 0, s, p, T, in.idx, part_off);
    hipLaunchKernelGGL(part_scan, dim3(1), dim3(1024), 0, s, T, part_off);
    hipLaunchKernelGGL(part_copy_sparse, dim3(grid), dim3(kBlock), 0, s, p, T, in.idx, in.val, out.idx, out.val,
                       part_off);
    return hipGetLastError();
}

}  // namespace bc
