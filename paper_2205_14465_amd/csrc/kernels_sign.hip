// kernels_sign.hip -- 1-bit sign compression with error feedback on gfx950
// (EFSignSGD, paper Sec. 5.1; 1-bit quantization with error feedback,
// Sec. 2.3).
//
// For every tensor: v = g + e_old; bit_i = sign bit of v_i (32 per word,
// element i at bit i mod 32, LSB first); s = mean |v| accumulated in fp64
// and rounded once to fp32; e_new = v - (bit ? -s : +s).
//
// The scale needs the whole tensor before any residual can be written, so
// the work takes two passes: pass 1 writes the bits, the chunk partial sums
// and v (into e); pass 2 sums the partials of its tensor in a fixed order,
// re-reads v and writes the residual.  The re-read of v mostly hits the
// 256 MB last-level cache for tensor sets of ResNet-50 size.  (A one-pass
// kernel that keeps v in registers while the tensor's workgroups exchange
// partial sums was slower on every workload measured: the workgroups of a
// tensor wait for each other with nothing to overlap.)
#include "launch.hpp"

namespace bc {

namespace {

// Pack the sign bits of the thread's 16 values and store the chunk's words.
// Word 32r + j/8 of the chunk gathers the nibbles of lanes 8m .. 8m+7.
__device__ __forceinline__ void store_sign_words(const float v[kEpt], uint32_t* words,
                                                 uint32_t words_in_chunk) {
    const int lane = lane_id();
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        uint32_t nib = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) nib |= (f2u(v[4 * r + q]) >> 31) << q;
        uint32_t x = nib << (4 * (lane & 7));
        x |= __shfl_xor(x, 1, 64);
        x |= __shfl_xor(x, 2, 64);
        x |= __shfl_xor(x, 4, 64);
        const uint32_t w = 32u * r + (threadIdx.x >> 3);
        if ((lane & 7) == 0 && w < words_in_chunk) words[w] = x;
    }
}

__device__ __forceinline__ double thread_abs_sum(const float v[kEpt]) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kEpt; ++i) acc += fabs((double)v[i]);
    return acc;
}

// Deterministic sum of m per-chunk partials: thread i adds partials
// i, i+256, ... in order, then a fixed tree over the block.
__device__ __forceinline__ double reduce_partials(const double* p, uint32_t m, double* sh) {
    double acc = 0.0;
    for (uint32_t q = threadIdx.x; q < m; q += kBlock) acc += p[q];
    return block_sum_f64(acc, sh);
}

template <bool kNT>
__device__ __forceinline__ void store_sign_residual(const TDesc& td, uint32_t j, float s,
                                                    float v[kEpt]) {
#pragma unroll
    for (int i = 0; i < kEpt; ++i) v[i] = v[i] - copysignf(s, v[i]);
    store_chunk<kNT>(td.resid, td.n, j, v);
}

__device__ __forceinline__ uint32_t chunk_words(const TDesc& td, uint32_t j) {
    uint32_t first = j * (uint32_t)kChunkWords;
    uint32_t left = td.k - first;
    return left < (uint32_t)kChunkWords ? left : (uint32_t)kChunkWords;
}

}  // namespace

// --------------------------------------------------------------- two pass
constexpr uint32_t kInlineScaleChunks = 1024;

template <bool kNT>
__global__ __launch_bounds__(kBlock) void sign_pass1(const TDesc* __restrict__ d, int T,
                                                     uint32_t* __restrict__ bits, Ws ws) {
    __shared__ double sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v<kNT>(td, j, td.resid != nullptr, v, valid);
    store_sign_words(v, bits + td.off + (uint64_t)j * kChunkWords, chunk_words(td, j));
    if (td.resid) store_chunk(td.resid, td.n, j, v);  // v parked in e for the second pass
    const double p = block_sum_f64(thread_abs_sum(v), sh);
    if (threadIdx.x == 0) ws.s_partial[c] = p;
}

__global__ __launch_bounds__(kBlock) void sign_finalize(const TDesc* __restrict__ d,
                                                        float* __restrict__ scale_out, Ws ws) {
    __shared__ double sh[4];
    const int t = blockIdx.x;
    const TDesc td = d[t];
    if (td.nchunks > 0 && td.nchunks <= kInlineScaleChunks) return;  // pass 2 does it
    float s = 0.f;
    if (td.nchunks > 0) {
        const double tot = reduce_partials(ws.s_partial + td.chunk0, td.nchunks, sh);
        s = (float)(tot / (double)td.n);
    }
    if (threadIdx.x == 0) {
        scale_out[t] = s;
        ws.s_val[t] = s;
    }
}

// Pass 2.  A tensor with at most kInlineScaleChunks chunks has its scale
// summed from the chunk partials by every workgroup of the tensor (the same
// fixed-order sum as sign_finalize; the first workgroup also stores it);
// larger tensors read the scale sign_finalize stored.

template <bool kNT>
__global__ __launch_bounds__(kBlock) void sign_pass2(const TDesc* __restrict__ d, int T,
                                                     float* __restrict__ scale_out, Ws ws) {
    __shared__ double sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float s;
    if (td.nchunks <= kInlineScaleChunks) {
        const double tot = reduce_partials(ws.s_partial + td.chunk0, td.nchunks, sh);
        s = (float)(tot / (double)td.n);
        if (j == 0 && threadIdx.x == 0) scale_out[t] = s;
    } else {
        s = ws.s_val[t];
    }
    if (!td.resid) return;
    float v[kEpt];
    uint32_t valid;
    load_stored_v(td, j, v, valid);  // e holds v after the first pass
    store_sign_residual<kNT>(td, j, s, v);
}

// -------------------------------------------------- residual update (sign)
__global__ __launch_bounds__(kBlock) void sign_residual_update(const TDesc* __restrict__ d, int T,
                                                               const uint32_t* __restrict__ bits,
                                                               const float* __restrict__ scale) {
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, true, v, valid);
    const float s = scale[t];
    const uint32_t* w = bits + td.off + (uint64_t)j * kChunkWords;
    const uint32_t nw = chunk_words(td, j);
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t wi = 32u * r + (threadIdx.x >> 3);
        const uint32_t word = wi < nw ? w[wi] : 0u;
        const uint32_t nib = (word >> (4 * (threadIdx.x & 7))) & 0xFu;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float dec = ((nib >> q) & 1u) ? -s : s;
            v[4 * r + q] = v[4 * r + q] - dec;
        }
    }
    store_chunk(td.resid, td.n, j, v);
}

// ------------------------------------------------------------- launchers
hipError_t launch_sign_compress(const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty,
                                uint32_t* bits, float* scale, const Ws& ws, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    // past the cache size: stream g and e_old past the cache, keep v (re-read
    // by pass 2) in it, and stream e_new out
    const bool nt = C > kNtChunks;
    if (C > 0) {
        if (nt) (void)launch_timed(kTimedSignPass1, sign_pass1<true>, dim3(C), dim3(kBlock), 0, s, d, T, bits, ws);
        else (void)launch_timed(kTimedSignPass1, sign_pass1<false>, dim3(C), dim3(kBlock), 0, s, d, T, bits, ws);
    }
    // tensors without elements, or with more chunks than pass 2 sums inline
    if (max_chunks > kInlineScaleChunks || C == 0 || any_empty)
        hipLaunchKernelGGL(sign_finalize, dim3(T), dim3(kBlock), 0, s, d, scale, ws);
    if (C > 0) {
        if (nt) hipLaunchKernelGGL(sign_pass2<true>, dim3(C), dim3(kBlock), 0, s, d, T, scale, ws);
        else hipLaunchKernelGGL(sign_pass2<false>, dim3(C), dim3(kBlock), 0, s, d, T, scale, ws);
    }
    return hipGetLastError();
}

hipError_t launch_sign_residual_update(const TDesc* d, int T, uint32_t C, const uint32_t* bits,
                                       const float* scale, hipStream_t s) {
    if (C == 0) return hipSuccess;
    hipLaunchKernelGGL(sign_residual_update, dim3(C), dim3(kBlock), 0, s, d, T, bits, scale);
    return hipGetLastError();
}

}  // namespace bc
