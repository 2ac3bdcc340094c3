// kernels_sign.hip -- 1-bit sign compression with error feedback on gfx950
// (EFSignSGD, paper Sec. 5.1; 1-bit quantization with error feedback,
// Sec. 2.3).
//
// For every tensor: v = g + e_old; bit_i = sign bit of v_i (32 per word,
// element i at bit i mod 32, LSB first); s = mean |v| accumulated in fp64
// and rounded once to fp32; e_new = v - (bit ? -s : +s).
//
// The scale needs the whole tensor before any residual can be written.
// The main kernel does this in ONE read of g and e: a persistent,
// cooperatively launched grid keeps each chunk's v in registers, publishes
// the chunk's fp64 partial sum, and waits until the last chunk of the
// tensor has arrived and published the scale.  Chunks are visited in the
// fixed order c = blockIdx.x + r * gridDim.x; because every workgroup of the
// grid is resident and no tensor has more chunks than the grid has
// workgroups, every chunk a waiter depends on is either already held by a
// running workgroup or is the next chunk of a workgroup whose own wait
// ends first, so every wait ends.  The wait is bounded anyway: after
// ~2^22 polls it records kFlagWaitTimeout in the workspace and goes on.
// When a tensor is larger than the grid (or cooperative launch is not
// available) a two-pass variant reads g and e twice.
#include "launch.hpp"

namespace bc {

namespace {

constexpr uint32_t kSpinLimit = 1u << 22;

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

__device__ __forceinline__ void store_sign_residual(const TDesc& td, uint32_t j, float s,
                                                    float v[kEpt]) {
#pragma unroll
    for (int i = 0; i < kEpt; ++i) v[i] = v[i] - copysignf(s, v[i]);
    store_chunk(td.resid, td.n, j, v);
}

__device__ __forceinline__ uint32_t chunk_words(const TDesc& td, uint32_t j) {
    uint32_t first = j * (uint32_t)kChunkWords;
    uint32_t left = td.k - first;
    return left < (uint32_t)kChunkWords ? left : (uint32_t)kChunkWords;
}

}  // namespace

// --------------------------------------------------------------- one pass
__global__ __launch_bounds__(kBlock) void sign_compress_coop(const TDesc* __restrict__ d, int T,
                                                             uint32_t C, uint32_t* __restrict__ bits,
                                                             float* __restrict__ scale_out, Ws ws) {
    __shared__ double sh[4];
    __shared__ float s_sh;
    __shared__ int last_sh;
    for (uint32_t c = blockIdx.x; c < C; c += gridDim.x) {
        const int t = tensor_of_chunk(d, T, c);
        const TDesc td = d[t];
        const uint32_t j = c - td.chunk0;
        float v[kEpt];
        uint32_t valid;
        load_v(td, j, td.resid != nullptr, v, valid);
        store_sign_words(v, bits + td.off + (uint64_t)j * kChunkWords, chunk_words(td, j));
        const double p = block_sum_f64(thread_abs_sum(v), sh);
        float s;
        if (td.nchunks == 1) {
            s = (float)(p / (double)td.n);
            if (threadIdx.x == 0) scale_out[t] = s;
        } else {
            if (threadIdx.x == 0) {
                ws.s_partial[c] = p;
                const uint32_t old = atomic_add_agent(ws.s_cnt + t, 1u);
                last_sh = (old == td.nchunks - 1);
            }
            __syncthreads();
            if (last_sh) {
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                const double tot = reduce_partials(ws.s_partial + td.chunk0, td.nchunks, sh);
                s = (float)(tot / (double)td.n);
                if (threadIdx.x == 0) {
                    scale_out[t] = s;
                    ws.s_val[t] = s;
                    atomic_store_release(ws.s_ready + t, 1u);
                }
            } else {
                if (threadIdx.x == 0) {
                    uint32_t spins = 0;
                    while (atomic_load_acquire(ws.s_ready + t) == 0u) {
                        __builtin_amdgcn_s_sleep(2);
                        if (++spins > kSpinLimit) {
                            __hip_atomic_fetch_or(ws.flags, kFlagWaitTimeout, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                            break;
                        }
                    }
                    s_sh = ws.s_val[t];
                }
                __syncthreads();
                s = s_sh;
            }
        }
        if (td.resid) store_sign_residual(td, j, s, v);
        __syncthreads();
    }
}

// --------------------------------------------------------------- two pass
__global__ __launch_bounds__(kBlock) void sign_pass1(const TDesc* __restrict__ d, int T,
                                                     uint32_t* __restrict__ bits, Ws ws) {
    __shared__ double sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, td.resid != nullptr, v, valid);
    store_sign_words(v, bits + td.off + (uint64_t)j * kChunkWords, chunk_words(td, j));
    const double p = block_sum_f64(thread_abs_sum(v), sh);
    if (threadIdx.x == 0) ws.s_partial[c] = p;
}

__global__ __launch_bounds__(kBlock) void sign_finalize(const TDesc* __restrict__ d,
                                                        float* __restrict__ scale_out, Ws ws) {
    __shared__ double sh[4];
    const int t = blockIdx.x;
    const TDesc td = d[t];
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

__global__ __launch_bounds__(kBlock) void sign_pass2(const TDesc* __restrict__ d, int T, Ws ws) {
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    if (!td.resid) return;
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, true, v, valid);
    store_sign_residual(td, j, ws.s_val[t], v);
}

// Per-call preparation: clear the arrival counters and flags of the
// one-pass kernel and write the scale of tensors without elements.
__global__ void sign_prep(const TDesc* __restrict__ d, int T, float* __restrict__ scale_out, Ws ws) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    ws.s_cnt[t] = 0u;
    ws.s_ready[t] = 0u;
    if (d[t].nchunks == 0) scale_out[t] = 0.f;
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
hipError_t launch_sign_compress(const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool,
                                bool, uint32_t* bits, float* scale, const Ws& ws,
                                const DevInfo& di, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL(sign_prep, dim3((T + 255) / 256), dim3(256), 0, s, d, T, scale, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || C == 0) return e;
    const uint32_t cap = (uint32_t)di.cus * (uint32_t)di.sign_coop_blocks_per_cu;
    const uint32_t G = C < cap ? C : cap;
    if (di.coop_ok && max_chunks <= G) {
        void* args[] = {(void*)&d, (void*)&T, (void*)&C, (void*)&bits, (void*)&scale, (void*)&ws};
        return hipLaunchCooperativeKernel((const void*)sign_compress_coop, dim3(G), dim3(kBlock), args,
                                          0, s);
    }
    hipLaunchKernelGGL(sign_pass1, dim3(C), dim3(kBlock), 0, s, d, T, bits, ws);
    hipLaunchKernelGGL(sign_finalize, dim3(T), dim3(kBlock), 0, s, d, scale, ws);
    hipLaunchKernelGGL(sign_pass2, dim3(C), dim3(kBlock), 0, s, d, T, ws);
    return hipGetLastError();
}

hipError_t sign_coop_occupancy(int* blocks_per_cu) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, sign_compress_coop, kBlock, 0);
}

hipError_t launch_sign_residual_update(const TDesc* d, int T, uint32_t C, const uint32_t* bits,
                                       const float* scale, hipStream_t s) {
    if (C == 0) return hipSuccess;
    hipLaunchKernelGGL(sign_residual_update, dim3(C), dim3(kBlock), 0, s, d, T, bits, scale);
    return hipGetLastError();
}

}  // namespace bc
