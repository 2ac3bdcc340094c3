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
// By default a two-pass variant runs instead (BYTECOMP_SIGN_PATH=onepass
// selects the one-pass kernel where every tensor fits the grid): pass 1
// writes the bits, the chunk partial sums and v (into e); pass 2 sums the
// partials of its tensor, re-reads v and writes the residual.  The re-read
// of v mostly hits the 256 MB last-level cache for tensor sets of
// ResNet-50 size, so its HBM traffic stays close to the one-pass kernel's.
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

// Same sum, reading partials that other workgroups published with
// agent-scope atomic stores.
__device__ __forceinline__ double reduce_partials_atomic(double* p, uint32_t m, double* sh) {
    double acc = 0.0;
    for (uint32_t q = threadIdx.x; q < m; q += kBlock)
        acc += __longlong_as_double((long long)__hip_atomic_load((unsigned long long*)p + q, __ATOMIC_RELAXED,
                                                                 __HIP_MEMORY_SCOPE_AGENT));
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
    // The next chunk's g and e are loaded into registers before this chunk's
    // wait for its tensor's scale, so the wait overlaps the next loads.
    RawChunk raw;
    uint32_t c = blockIdx.x;
    if (c < C) {
        const TDesc td0 = d[tensor_of_chunk(d, T, c)];
        load_raw(td0, c - td0.chunk0, td0.resid != nullptr, raw);
    }
    for (; c < C; c += gridDim.x) {
        const int t = tensor_of_chunk(d, T, c);
        const TDesc td = d[t];
        const uint32_t j = c - td.chunk0;
        float v[kEpt];
        raw_to_v(td, td.resid != nullptr, raw, v);
        const uint32_t cn = c + gridDim.x;
        if (cn < C) {
            const TDesc tdn = d[tensor_of_chunk(d, T, cn)];
            load_raw(tdn, cn - tdn.chunk0, tdn.resid != nullptr, raw);
        }
        store_sign_words(v, bits + td.off + (uint64_t)j * kChunkWords, chunk_words(td, j));
        const double p = block_sum_f64(thread_abs_sum(v), sh);
        float s;
        if (td.nchunks == 1) {
            s = (float)(p / (double)td.n);
            if (threadIdx.x == 0) scale_out[t] = s;
        } else {
            // Cross-workgroup exchange uses agent-scope atomics only (coherent
            // across the chip's L2 caches) and no acquire/release fences, which
            // on this GPU would write back or invalidate a whole L2.
            if (threadIdx.x == 0) {
                __hip_atomic_store((unsigned long long*)ws.s_partial + c, (unsigned long long)__double_as_longlong(p),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                // the partial store completes before the arrival is counted
                __builtin_amdgcn_s_waitcnt(0);
                const uint32_t old = __hip_atomic_fetch_add(ws.s_cnt + t, 1u, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                last_sh = (old == td.nchunks - 1);
            }
            __syncthreads();
            if (last_sh) {
                const double tot = reduce_partials_atomic(ws.s_partial + td.chunk0, td.nchunks, sh);
                s = (float)(tot / (double)td.n);
                if (threadIdx.x == 0) {
                    scale_out[t] = s;
                    // scale and "published" flag travel in one 64-bit word
                    __hip_atomic_store((unsigned long long*)ws.s_ready + t,
                                       (1ull << 32) | (unsigned long long)f2u(s), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            } else {
                if (threadIdx.x == 0) {
                    uint32_t spins = 0;
                    unsigned long long x;
                    for (;;) {
                        x = __hip_atomic_load((unsigned long long*)ws.s_ready + t, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
                        if (x >> 32) break;
                        __builtin_amdgcn_s_sleep(2);
                        if (++spins > kSpinLimit) {
                            __hip_atomic_fetch_or(ws.flags, kFlagWaitTimeout, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                            break;
                        }
                    }
                    s_sh = u2f((uint32_t)x);
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
constexpr uint32_t kInlineScaleChunks = 1024;

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
    store_sign_residual(td, j, s, v);
}

// Per-call preparation: clear the arrival counters and flags of the
// one-pass kernel and write the scale of tensors without elements.
__global__ void sign_prep(const TDesc* __restrict__ d, int T, float* __restrict__ scale_out, Ws ws) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    ws.s_cnt[t] = 0u;
    ((unsigned long long*)ws.s_ready)[t] = 0ull;
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
    const uint32_t cap = (uint32_t)di.cus * (uint32_t)di.sign_coop_blocks_per_cu;
    const uint32_t G = C < cap ? C : cap;
    if (di.sign_one_pass && di.coop_ok && C > 0 && max_chunks <= G) {
        hipLaunchKernelGGL(sign_prep, dim3((T + 255) / 256), dim3(256), 0, s, d, T, scale, ws);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        void* args[] = {(void*)&d, (void*)&T, (void*)&C, (void*)&bits, (void*)&scale, (void*)&ws};
        return hipLaunchCooperativeKernel((const void*)sign_compress_coop, dim3(G), dim3(kBlock), args,
                                          0, s);
    }
    if (C > 0) hipLaunchKernelGGL(sign_pass1, dim3(C), dim3(kBlock), 0, s, d, T, bits, ws);
    // tensors without elements, or with more chunks than pass 2 sums inline
    if (max_chunks > kInlineScaleChunks || C == 0 || di.any_empty)
        hipLaunchKernelGGL(sign_finalize, dim3(T), dim3(kBlock), 0, s, d, scale, ws);
    if (C > 0) hipLaunchKernelGGL(sign_pass2, dim3(C), dim3(kBlock), 0, s, d, T, scale, ws);
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
