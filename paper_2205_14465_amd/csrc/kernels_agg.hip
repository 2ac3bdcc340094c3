// kernels_agg.hip -- decompress-and-aggregate of W workers' payloads on
// gfx950 (paper Sec. 3.1, Reason #2: after the gather each node decompresses
// the N payloads and aggregates them; Sec. 4.2.1, Dimension 3: the
// aggregation of compressed tensors is not associative, so it is not an
// Allreduce), plus the sparse residual update.
//
// Both aggregates add the workers' decoded values in ascending worker order,
// one fp32 addition each, starting from +0.0, then multiply by alpha; no
// floating-point atomics are used, so results are deterministic and match
// that order bit for bit.
//
// Sparse: each wave owns a run of 2048-element output tiles held in LDS.
// For every tile it walks the workers in order; worker w's entries for the
// tile are the next ones after its cursor (indices ascending), read 64 at a
// time and added into the tile (indices are unique within a worker, so a
// worker's adds never collide and need no atomics).  Cursors are found by a
// binary search only where a wave's run starts inside a tensor.
//
// Sign: each wave owns 512 output elements, 8 per lane.  For worker w the 16
// words covering them are fetched with scalar loads; each 64-bit word pair
// is a lane mask that selects -s_w or +s_w with one v_cndmask, then one
// v_add per element and worker.
#include "launch.hpp"

namespace bc {

namespace {

typedef const uint32_t __attribute__((address_space(4)))* cu32p;
typedef const float __attribute__((address_space(4)))* cf32p;

__device__ __forceinline__ int unit_owner(const ADesc* __restrict__ a, int T, uint32_t u) {
    return find_owner<ADesc, &ADesc::unit0>(a, T, u);
}

// First position p in [0, k) with idx[p] >= x (k if none).
__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* idx, uint32_t k, uint32_t x) {
    uint32_t lo = 0, hi = k;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (idx[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

constexpr int kPrefetch = 8;  // workers whose first 64 entries are loaded together

}  // namespace

// ----------------------------------------------------------------- sparse
// Dynamic LDS: 4 waves x (2048 floats tile + W cursors).
__global__ __launch_bounds__(kBlock) void aggregate_sparse(const ADesc* __restrict__ a, int T,
                                                           uint32_t U, const WDesc* __restrict__ wd,
                                                           int W, float alpha) {
    extern __shared__ uint32_t lds[];
    const int wave = wave_id();
    const int lane = lane_id();
    float* tile = reinterpret_cast<float*>(lds) + wave * (int)kSparseTile;
    uint32_t* cur = lds + 4 * kSparseTile + wave * W;
    const uint64_t nw = (uint64_t)gridDim.x * 4;
    const uint64_t gw = (uint64_t)blockIdx.x * 4 + wave;
    const uint32_t u_beg = (uint32_t)((gw * U) / nw);
    const uint32_t u_end = (uint32_t)(((gw + 1) * U) / nw);
    int t = -1;
    ADesc ad{};
    for (uint32_t u = u_beg; u < u_end; ++u) {
        if (t < 0 || u >= ad.unit0 + ad.nunits) {
            t = unit_owner(a, T, u);
            ad = a[t];
            const uint32_t lo0 = (u - ad.unit0) * kSparseTile;
            for (int w = lane; w < W; w += 64)
                cur[w] = lo0 == 0 ? 0u : lower_bound_u32(wd[w].a + ad.off, ad.k, lo0);
            __builtin_amdgcn_wave_barrier();
        }
        const uint32_t lo = (u - ad.unit0) * kSparseTile;
        const uint32_t hi = (lo + kSparseTile < ad.n) ? lo + kSparseTile : ad.n;
        for (int i = lane; i < (int)kSparseTile; i += 64) tile[i] = 0.f;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        for (int w0 = 0; w0 < W; w0 += kPrefetch) {
            uint32_t x[kPrefetch];
            float y[kPrefetch];
            uint32_t c[kPrefetch];
#pragma unroll
            for (int q = 0; q < kPrefetch; ++q) {
                x[q] = 0xFFFFFFFFu;
                y[q] = 0.f;
                c[q] = 0;
                if (w0 + q < W) {
                    c[q] = cur[w0 + q];
                    const uint32_t i = c[q] + lane;
                    if (i < ad.k) {
                        x[q] = wd[w0 + q].a[ad.off + i];
                        y[q] = wd[w0 + q].b[ad.off + i];
                    }
                }
            }
#pragma unroll
            for (int q = 0; q < kPrefetch; ++q) {
                const int w = w0 + q;
                if (w >= W) break;
                uint32_t cc = c[q];
                uint32_t xi = x[q];
                float yi = y[q];
                for (;;) {
                    const bool in = xi < hi;
                    const uint64_t m = __ballot(in);
                    // entries below the tile can only come from an unsorted
                    // payload; they are skipped rather than written out of range
                    if (in && xi >= lo) tile[xi - lo] += yi;
                    const uint32_t cnt = (uint32_t)__popcll(m);
                    cc += cnt;
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                    if (cnt < 64) break;
                    const uint32_t i = cc + lane;
                    xi = 0xFFFFFFFFu;
                    yi = 0.f;
                    if (i < ad.k) {
                        xi = wd[w].a[ad.off + i];
                        yi = wd[w].b[ad.off + i];
                    }
                }
                if (lane == 0) cur[w] = cc;
            }
            __builtin_amdgcn_wave_barrier();
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        float* out = ad.out + lo;
        const uint32_t len = hi - lo;
        for (uint32_t i = 4u * lane; i < len; i += 256u) {
            if (i + 3 < len) {
                float4 r = make_float4(alpha * tile[i], alpha * tile[i + 1], alpha * tile[i + 2],
                                       alpha * tile[i + 3]);
                *reinterpret_cast<float4*>(out + i) = r;
            } else {
                for (uint32_t q = i; q < len; ++q) out[q] = alpha * tile[q];
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ------------------------------------------------------------------- sign
__global__ __launch_bounds__(kBlock) void aggregate_sign(const ADesc* __restrict__ a, int T,
                                                         uint32_t U, const WDesc* __restrict__ wd,
                                                         int W, float alpha) {
    const uint32_t u = blockIdx.x * 4u + (uint32_t)wave_id();
    if (u >= U) return;
    const int lane = lane_id();
    const int t = unit_owner(a, T, u);
    const ADesc ad = a[t];
    const uint32_t j = u - ad.unit0;
    const uint32_t lo = j * kSignAggUnit;
    const uint64_t woff = ad.off + (uint64_t)j * 16u;
    const uint32_t nwords = (ad.k - j * 16u) < 16u ? (ad.k - j * 16u) : 16u;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int w = 0; w < W; ++w) {
        const WDesc p = wd[w];
        const float s = ((cf32p)p.b)[t];
        uint32_t word[16];
        const cu32p bp = (cu32p)(p.a + woff);
        if (nwords == 16u) {
#pragma unroll
            for (int i = 0; i < 16; ++i) word[i] = bp[i];
        } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) word[i] = (uint32_t)i < nwords ? bp[i] : 0u;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint64_t m = (uint64_t)word[2 * e] | ((uint64_t)word[2 * e + 1] << 32);
            float dv;
            asm("v_cndmask_b32_e64 %0, %1, -%1, %2" : "=v"(dv) : "v"(s), "s"(m));
            acc[e] += dv;
        }
    }
    float* out = ad.out + lo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t i = 64u * e + lane;
        if (lo + i < ad.n) out[i] = alpha * acc[e];
    }
}

// --------------------------------------------------- sparse residual update
// residual <- (g + residual) - decompress(own): a chunk gathers its entries
// of the payload into an LDS copy of the decoded chunk (zeros elsewhere).
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
        const uint32_t x = i < td.k ? ix[i] : 0xFFFFFFFFu;
        const bool in = x < hi;
        if (in && x >= lo) dec[x - lo] = vx[i];
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

// -------------------------------------------------------------- launchers
hipError_t launch_aggregate_sparse(const ADesc* a, int T, uint32_t U, const WDesc* w, int W,
                                   float alpha, hipStream_t s) {
    if (U == 0) return hipSuccess;
    // enough waves to fill the chip several times over; each owns ~U/waves tiles
    uint32_t blocks = (U + 3) / 4;
    if (blocks > 2048) blocks = 2048;
    const size_t lds = (size_t)4 * (kSparseTile * 4 + (size_t)W * 4);
    hipLaunchKernelGGL(aggregate_sparse, dim3(blocks), dim3(kBlock), lds, s, a, T, U, w, W, alpha);
    return hipGetLastError();
}

hipError_t launch_aggregate_sign(const ADesc* a, int T, uint32_t U, const WDesc* w, int W,
                                 float alpha, hipStream_t s) {
    if (U == 0) return hipSuccess;
    hipLaunchKernelGGL(aggregate_sign, dim3((U + 3) / 4), dim3(kBlock), 0, s, a, T, U, w, W, alpha);
    return hipGetLastError();
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

}  // namespace bc

namespace bc {

__global__ void zero_header(uint32_t* flags) {
    flags[threadIdx.x] = 0u;
}

hipError_t launch_zero_header(uint32_t* flags, hipStream_t s) {
    hipLaunchKernelGGL(zero_header, dim3(1), dim3(64), 0, s, flags);
    return hipGetLastError();
}

}  // namespace bc
