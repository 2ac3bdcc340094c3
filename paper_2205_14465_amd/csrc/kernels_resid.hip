// kernels_resid.hip -- standalone error-feedback residual update for sparse
// payloads (paper Sec. 2.3: the residual keeps what compression dropped),
// the dispatcher of the residual-update entry point, and the workspace
// header reset.
//
// residual <- (g + residual) - decompress(own): a chunk gathers its entries
// of the payload into an LDS copy of the decoded chunk (zeros elsewhere).
#include "launch.hpp"

namespace bc {

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

__global__ void zero_header(uint32_t* flags) {
    flags[threadIdx.x] = 0u;
}

hipError_t launch_zero_header(uint32_t* flags, hipStream_t s) {
    hipLaunchKernelGGL(zero_header, dim3(1), dim3(64), 0, s, flags);
    return hipGetLastError();
}

}  // namespace bc
