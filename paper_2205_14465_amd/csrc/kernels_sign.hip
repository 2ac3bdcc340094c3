// kernels_sign.hip -- 1-bit sign compression with error feedback on gfx950
// (EFSignSGD, paper Sec. 5.1; 1-bit quantization with error feedback,
// Sec. 2.3).
//
// For every tensor: v = g + e_old; bit_i = sign bit of v_i (32 per word,
// element i at bit i mod 32, LSB first); s = mean |v| accumulated in fp64
// and rounded once to fp32; e_new = v - (bit ? -s : +s).
//
// The scale needs the whole tensor before any residual can be written.
// When every tensor has at most as many chunks as the GPU holds resident
// workgroups, ONE pass does it (sign_onepass): a grid of resident
// workgroups visits chunks c = blockIdx + k * grid; for each it loads g and
// e, writes the bits, publishes the chunk's fp64 partial sum, and only then
// writes the residual of its PREVIOUS chunk, kept in registers, whose
// tensor's scale is by then almost always known (every workgroup of the
// tensor sums its partials in the same fixed order).  Otherwise two passes
// run: pass 1 writes the
// bits, the chunk partial sums and v (into e); pass 2 sums the partials of
// its tensor in the same fixed order, re-reads v and writes the residual.
// (An earlier one-pass form that waited for each chunk's own tensor before
// moving on was slower than two passes: the workgroups of a tensor waited
// for each other with nothing to overlap.)
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

// --------------------------------------------------------------- one pass
// Chunk partial sums travel through slots that hold the bitwise complement
// of the fp64 partial once published and 0 before (a sum of magnitudes is
// never all ones), so a slot needs no separate ready flag.  A fill kernel
// empties the slots just before the one-pass kernel runs, so whatever an
// earlier call (of any kind sharing the workspace) left there does not
// matter.  A workgroup writes chunk c's residual only after publishing
// chunk c + grid (and prefetching its next chunk): it then reads all its
// tensor's slots, waiting while any is empty, and sums them in the fixed
// order of the two-pass path.
//
// When every workgroup of the grid is resident (the launcher sizes the
// grid so) every wait ends quickly: the chunks of tensor(c) are published
// by workgroups whose earlier waits concern chunks at least two grids
// before them, which (no tensor being longer than a grid) belong to earlier
// tensors, so by induction over the tensors every slot gets published.
// When the grid is not wholly resident (other kernels holding compute
// units), a wait may find a slot whose owner has not started: after the
// host's wait limit the waiting workgroup computes such partials itself
// and publishes them by compare-and-swap (common.hpp), so every wait ends
// and the results are the same either way.
namespace {

constexpr int kHelpBatch = 256;  // missing partials a waiting workgroup computes per pass

// Partial sum of |v| over chunk j of tensor td, bit-identical to the
// owner's (each thread's sixteen values in element order, then the fixed
// block tree), read one round of four elements at a time (lean in
// registers: it runs inside the one-pass kernel).
__device__ __forceinline__ double chunk_abs_partial(const TDesc& td, uint32_t j, double* sh) {
    double acc = 0.0;
#pragma unroll 1
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float v = 0.f;
            if (e0 + q < td.n) {
                const float g = td.dtype == 0 ? gp((const float*)td.grad)[e0 + q]
                                              : h2f(gp((const uint16_t*)td.grad)[e0 + q]);
                v = td.resid ? g + gp(td.resid)[e0 + q] : g;
            }
            acc += fabs((double)v);
        }
    }
    return block_sum_f64(acc, sh);
}

// Scale of tensor td from its chunk slots (every thread returns it),
// waiting while a slot is empty; once `ticks` of the constant-rate counter
// have passed (thread 0 decides, through LDS), each pass computes up to
// kHelpBatch missing partials and publishes them by compare-and-swap.
// ctl_sh: LDS, 2 + kHelpBatch ints.
__device__ __forceinline__ float onepass_scale(const TDesc& td, uint64_t* slot, double* sh, uint32_t ticks,
                                               int* ctl_sh) {
    int& pending_sh = ctl_sh[0];
    int& help_sh = ctl_sh[1];
    int* miss_sh = ctl_sh + 2;
    const uint64_t t0 = wall_clock64();
    unsigned long long* sl = (unsigned long long*)slot + td.chunk0;
    double acc;
    for (;;) {
        acc = 0.0;
        int missing = 0;
        for (uint32_t q = threadIdx.x; q < td.nchunks; q += kBlock) {
            const unsigned long long x = __hip_atomic_load(sl + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            missing |= x == 0ull;
            acc += __longlong_as_double((long long)~x);
        }
        if (threadIdx.x == 0) pending_sh = 0;
        __syncthreads();
        if (missing) pending_sh = 1;
        __syncthreads();
        const int pending = pending_sh;
        if (threadIdx.x == 0) help_sh = pending && wall_clock64() - t0 >= (uint64_t)ticks ? 1 : 0;
        __syncthreads();
        if (!pending) break;
        if (!help_sh) {
            __builtin_amdgcn_s_sleep(4);
            continue;
        }
        // list up to kHelpBatch empty slots (pending_sh counts them), then
        // compute and publish each
        if (threadIdx.x == 0) pending_sh = 0;
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < td.nchunks; q += kBlock) {
            if (__hip_atomic_load(sl + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0ull) {
                const int k = atomicAdd(&pending_sh, 1);
                if (k < kHelpBatch) miss_sh[k] = (int)q;
            }
        }
        __syncthreads();
        const int m = pending_sh < kHelpBatch ? pending_sh : kHelpBatch;
        for (int i = 0; i < m; ++i) {
            const uint32_t q = (uint32_t)miss_sh[i];
            const double p = chunk_abs_partial(td, q, sh);
            if (threadIdx.x == 0) {
                unsigned long long expected = 0ull;
                __hip_atomic_compare_exchange_strong(sl + q, &expected, ~(unsigned long long)__double_as_longlong(p),
                                                     __ATOMIC_RELAXED, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __syncthreads();  // the list is reused by the next pass
    }
    return (float)(block_sum_f64(acc, sh) / (double)td.n);
}
}  // namespace

template <int kDT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(5))) void sign_onepass(const TDesc* __restrict__ d, int T, uint32_t C,
                                                       uint32_t* __restrict__ bits, float* __restrict__ scale_out,
                                                       Ws ws, uint32_t wait_ticks) {
    __shared__ double sh[4];
    __shared__ int ctl_sh[2 + kHelpBatch];
    float vp[kEpt];  // the previous chunk's v, its residual not yet written
    TDesc tdp{};
    bool prev = false;
    uint32_t jp = 0;
    float sp = 0.f;  // its scale when already known (a single-chunk tensor)
    RawChunk raw;
    uint32_t c = blockIdx.x;
    TDesc td{};
    if (c < C) {
        td = d[tensor_of_chunk(d, T, c)];
        load_raw<kDT>(td, c - td.chunk0, td.resid != nullptr, raw);
    }
    for (;; c += gridDim.x) {
        const bool have = c < C;
        float v[kEpt];
        uint32_t j = 0;
        float s_now = 0.f;
        if (have) {
            const int t = tensor_of_chunk(d, T, c);
            j = c - td.chunk0;
            raw_to_v<kDT>(td, td.resid != nullptr, raw, v);
            store_sign_words(v, bits + td.off + (uint64_t)j * kChunkWords, chunk_words(td, j));
            const double p = block_sum_f64(thread_abs_sum(v), sh);
            if (td.nchunks == 1) {
                s_now = (float)(p / (double)td.n);
                if (threadIdx.x == 0) scale_out[t] = s_now;
            } else if (threadIdx.x == 0) {
                __hip_atomic_store((unsigned long long*)ws.s_slot + c, ~(unsigned long long)__double_as_longlong(p),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        // the next chunk's loads go out before this round's wait
        const uint32_t cn = c + gridDim.x;
        TDesc tdn{};
        if (cn < C) {
            tdn = d[tensor_of_chunk(d, T, cn)];
            load_raw<kDT>(tdn, cn - tdn.chunk0, tdn.resid != nullptr, raw);
        }
        if (prev) {
            float s = sp;
            if (tdp.nchunks > 1) {
                s = onepass_scale(tdp, ws.s_slot, sh, wait_ticks, ctl_sh);
                if (jp == 0 && threadIdx.x == 0) scale_out[tensor_of_chunk(d, T, tdp.chunk0)] = s;
            }
            if (tdp.resid) store_sign_residual<false>(tdp, jp, s, vp);
        }
        if (!have) break;
#pragma unroll
        for (int i = 0; i < kEpt; ++i) vp[i] = v[i];
        tdp = td;
        prev = true;
        jp = j;
        sp = s_now;
        td = tdn;
    }
}

// Scales of empty tensors (+0.0) for the one-pass path.
__global__ void sign_empty_scales(const TDesc* __restrict__ d, int T, float* __restrict__ scale_out) {
    const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (t < T && d[t].nchunks == 0) scale_out[t] = 0.f;
}

// Slots of the one-pass kernel, emptied before it runs (a fill kernel, not
// a memset, so that the sequence stays capturable).
__global__ void sign_onepass_reset(uint32_t C, Ws ws) {
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x)
        ws.s_slot[c] = 0ull;
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
namespace {
// Workgroups of sign_onepass<kDT> resident at once on the whole GPU.
template <int kDT>
uint32_t onepass_capacity(int cus) {
    static int per_cu = -1;
    if (per_cu < 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, sign_onepass<kDT>, kBlock, 0) != hipSuccess) nb = 0;
        per_cu = nb;
    }
    return (uint32_t)per_cu * (uint32_t)(cus > 0 ? cus : 0);
}

// One pass when every tensor fits the resident grid; false otherwise.
template <int kDT>
bool sign_onepass_launch(const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty, uint32_t* bits,
                         float* scale, const Ws& ws, int cus, hipStream_t s) {
    const uint32_t cap = onepass_capacity<kDT>(cus);
    if (C == 0 || cap == 0 || max_chunks > cap) return false;
    const uint32_t grid = C < cap ? C : cap;
    hipLaunchKernelGGL(sign_onepass_reset, dim3((C + 255) / 256 < 1024 ? (C + 255) / 256 : 1024), dim3(256), 0, s,
                       C, ws);
    (void)launch_timed(kTimedSignOnepass, sign_onepass<kDT>, dim3(grid), dim3(kBlock), 0, s, d, T, C, bits, scale, ws,
                       onepass_wait_ticks());
    if (any_empty) hipLaunchKernelGGL(sign_empty_scales, dim3((T + 255) / 256), dim3(256), 0, s, d, T, scale);
    return true;
}
}  // namespace

hipError_t launch_sign_compress(const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty,
                                bool any_f16, bool any_f32, uint32_t* bits, float* scale, const Ws& ws, int cus,
                                hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const bool one = any_f16 && any_f32 ? sign_onepass_launch<2>(d, T, C, max_chunks, any_empty, bits, scale, ws, cus, s)
                     : any_f16          ? sign_onepass_launch<1>(d, T, C, max_chunks, any_empty, bits, scale, ws, cus, s)
                                        : sign_onepass_launch<0>(d, T, C, max_chunks, any_empty, bits, scale, ws, cus, s);
    if (one) return hipGetLastError();
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
