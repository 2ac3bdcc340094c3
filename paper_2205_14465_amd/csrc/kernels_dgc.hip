// kernels_dgc.hip -- DGC's local gradient clipping for the DGC step of the
// sparse kinds (DGC is the paper's sparsification operator at a 1% rate,
// Sec. 5.1; Sec. 2.3: sparsification with error feedback).
//
// A DGC step of one tensor keeps a velocity u next to the error-feedback
// residual e (DGC's accumulated gradient):
//   c = local clipping factor of the step's gradient list (optional):
//       fl32(clip / ||g||) when the list's L2 norm is above the threshold,
//       else 1 (dgc_sumsq: fp64 sum of squares per chunk; dgc_clip_factor:
//       one workgroup adds the chunk sums, takes the root and the factor)
//   u <- fl32(fl32(m * u) + fl32(c * g))            (c = 1: the unclipped g)
//   compress u with residual e: v = fl32(u + e), select, payload v[idx],
//   e <- v with +0.0 at idx                         (the sparse kind)
//   u[idx] <- +0.0
// The velocity step runs inside the compress pass that forms v and the
// masking where the selection is known: the top-k emit pass
// (kernels_topk.hip), the random-k stream pass (kernels_randk.hip).  This
// file holds the clipping factor.
#include "launch.hpp"

namespace bc {

// Sum of squares of a chunk's widened gradient, each square exact in fp64,
// added per thread then in the fixed tree of block_sum_f64.
__global__ __launch_bounds__(kBlock) void dgc_sumsq(const TDesc* __restrict__ d, int T, double* __restrict__ part) {
    __shared__ double sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float g[kEpt];
    uint32_t valid;
    load_v<false>(td, j, false, g, valid);
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kEpt; ++i) {
        const double x = ((valid >> i) & 1u) ? (double)g[i] : 0.0;
        acc += x * x;
    }
    const double tot = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) part[c] = tot;
}

// One workgroup: thread i adds the chunk sums of its contiguous run in
// order, the block adds the runs in a fixed tree; the norm is the fp64
// square root and the factor fl32(clip / norm) above the threshold, else
// 1.  Written to factor[0] and, when given, to out[0].
__global__ __launch_bounds__(kBlock) void dgc_clip_factor(const double* __restrict__ part, uint32_t C, double clip,
                                                          float* __restrict__ factor, float* __restrict__ out) {
    __shared__ double sh[4];
    const uint32_t per = (C + kBlock - 1) / kBlock;
    const uint32_t lo = threadIdx.x * per, hi = lo + per < C ? lo + per : C;
    double acc = 0.0;
    for (uint32_t q = lo; q < hi; ++q) acc += part[q];
    const double norm = sqrt(block_sum_f64(acc, sh));
    if (threadIdx.x == 0) {
        const float f = norm > clip ? (float)(clip / norm) : 1.0f;
        factor[0] = f;
        if (out) out[0] = f;
    }
}

hipError_t launch_dgc_clip(const TDesc* d, int T, uint32_t C, double clip, double* part, float* factor,
                           float* factor_out, hipStream_t s) {
    if (C > 0) hipLaunchKernelGGL(dgc_sumsq, dim3(C), dim3(kBlock), 0, s, d, T, part);
    hipLaunchKernelGGL(dgc_clip_factor, dim3(1), dim3(kBlock), 0, s, part, C, clip, factor, factor_out);
    return hipGetLastError();
}

}  // namespace bc
