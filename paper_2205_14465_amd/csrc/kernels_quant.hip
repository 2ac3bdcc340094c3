// kernels_quant.hip -- stochastic b-bit quantization with error feedback on
// gfx950: TernGrad (2-bit codes, one level), QSGD with 7 levels (4-bit) and
// with 127 levels (8-bit) (paper Sec. 2.3: gradients quantized to 8 bits,
// 2 bits or 1 bit, combined with error feedback).
//
// For every tensor: v = g + e_old; m = max |v| (the payload's scale, exact
// and independent of any summation order); inv = fl32(s / m), unit =
// fl32(m / s); x = fl32(|v| * inv); the level is s when x >= s, else
// floor(x) plus one with probability x - floor(x), decided against a
// uniform U = (u >> 8) * 2^-24 drawn from Philox4x64-10 at counter
// (tensor_id, i / 8), key (seed, stream 2) -- element i takes 32-bit word
// i mod 8 of the block; code = level | sign << (b - 1) (0 for level 0),
// b bits per element, LSB first, each tensor word aligned; decode d =
// +-fl32(level * unit); e_new = fl32(v - d).
//
// Compress in two passes, as for the 1-bit kind: pass 1 forms v, parks it
// in e and writes each chunk's largest |v| bits; pass 2 takes the tensor's
// maximum over its chunks, re-reads v, quantizes, packs the codes with lane
// shuffles and writes the residual.  The aggregate gives each workgroup
// 4096 output elements (16 per lane) and adds the W workers' decoded values
// in worker order, one fp32 addition each.
#include "exact_wide.hpp"
#include "launch.hpp"

namespace bc {

namespace {

template <int kBits>
struct Quant {
    static constexpr int kLevels = (1 << (kBits - 1)) - 1;
    static constexpr uint32_t kMask = (1u << kBits) - 1u;
    static constexpr uint32_t kLevelMask = (1u << (kBits - 1)) - 1u;
    static constexpr uint32_t kWordsPerChunk = (uint32_t)kChunk * kBits / 32u;
};

constexpr uint32_t kQuantInlineChunks = 1024;  // pass 2 reduces the chunk maxima itself

__device__ __forceinline__ uint32_t block_max_u32(uint32_t x, uint32_t* sh /* >= 4 */) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t y = (uint32_t)__shfl_xor((int)x, o, 64);
        x = y > x ? y : x;
    }
    if (lane_id() == 0) sh[threadIdx.x >> 6] = x;
    __syncthreads();
    uint32_t m = sh[0];
#pragma unroll
    for (int w = 1; w < kBlock / 64; ++w) m = sh[w] > m ? sh[w] : m;
    __syncthreads();
    return m;
}

// Largest |v| bits of tensor t from its chunk maxima.
__device__ __forceinline__ uint32_t tensor_max(const uint32_t* __restrict__ q, const TDesc& td, uint32_t* sh) {
    uint32_t m = 0;
    for (uint32_t c = threadIdx.x; c < td.nchunks; c += kBlock) {
        const uint32_t x = q[td.chunk0 + c];
        m = x > m ? x : m;
    }
    return block_max_u32(m, sh);
}

__device__ __forceinline__ void words_to_uniforms(uint64_t w0, uint64_t w1, float (&u)[4]) {
    u[0] = (float)((uint32_t)w0 >> 8) * 0x1p-24f;
    u[1] = (float)((uint32_t)(w0 >> 32) >> 8) * 0x1p-24f;
    u[2] = (float)((uint32_t)w1 >> 8) * 0x1p-24f;
    u[3] = (float)((uint32_t)(w1 >> 32) >> 8) * 0x1p-24f;
}

// The value of lane l ^ 1 (l ^ 2), by a DPP quad permutation: one VALU
// move instead of an LDS permute.
__device__ __forceinline__ uint32_t lane_xor1(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
}
__device__ __forceinline__ uint32_t lane_xor2(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
}
__device__ __forceinline__ uint64_t lane_xor1_64(uint64_t x) {
    return ((uint64_t)lane_xor1((uint32_t)(x >> 32)) << 32) | lane_xor1((uint32_t)x);
}

// The uniforms of the thread's kRounds rounds of chunk j (round r: the
// elements i = 4096 j + 1024 r + 4 tid .. + 3; element i takes 32-bit word
// i mod 8 of the Philox block at counter (tensor id, i / 8)).  The two
// threads of a lane pair share every round's block, each using one half of
// it, so the even thread computes the blocks of the even rounds and the odd
// thread those of the odd rounds, and each hands the other the half it
// needs: every uniform as defined, for half the Philox work.  Called by
// every thread of the workgroup.
__device__ __forceinline__ void chunk_uniforms(uint64_t seed, uint32_t tid, uint32_t j,
                                               float (&u)[kRounds][4]) {
    static_assert(kRounds % 2 == 0, "rounds pair up");
    const bool odd = (threadIdx.x & 1u) != 0u;
#pragma unroll
    for (int rr = 0; rr < kRounds / 2; ++rr) {
        const uint32_t r = 2u * (uint32_t)rr + (odd ? 1u : 0u);  // the round whose block this thread computes
        const uint32_t g = (j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x) >> 3;
        const U64x4 ctr = {{(uint64_t)tid, (uint64_t)g, 0, 0}};
        const U64x4 R = philox4x64_10(ctr, seed, kStreamQuant);
        // own half (words 0, 1 for the even thread, 2, 3 for the odd one),
        // and the partner's half, sent across the pair
        const uint64_t k0 = odd ? R.v[2] : R.v[0], k1 = odd ? R.v[3] : R.v[1];
        const uint64_t q0 = lane_xor1_64(odd ? R.v[0] : R.v[2]), q1 = lane_xor1_64(odd ? R.v[1] : R.v[3]);
        // round 2rr is the even thread's block, round 2rr + 1 the odd one's
        words_to_uniforms(odd ? q0 : k0, odd ? q1 : k1, u[2 * rr]);
        words_to_uniforms(odd ? k0 : q0, odd ? k1 : q1, u[2 * rr + 1]);
    }
}

// Decoded value of a code for a tensor whose decoding unit is `unit`.
template <int kBits>
__device__ __forceinline__ float quant_decode(uint32_t code, float unit) {
    const uint32_t level = code & Quant<kBits>::kLevelMask;
    float d;
    if constexpr (kBits == 2) {
        d = unit;  // the one level
    } else {
        d = (float)level * unit;
    }
    d = u2f(f2u(d) ^ ((code >> (kBits - 1)) << 31));
    return level ? d : 0.f;
}

// Codes of four consecutive elements (kBits each, element q at bit kBits q)
// into the payload: word `wi` of the tensor gathers 32 / kBits codes, so
// 8-bit codes fill a word per lane, 4-bit codes a word per lane pair and
// 2-bit codes a word per four lanes.  Words at or past the tensor's word
// count are not written.
template <int kBits>
__device__ __forceinline__ void store_codes(uint32_t packed, uint32_t e0, uint32_t* __restrict__ words,
                                            uint32_t nwords) {
    const int lane = lane_id();
    if constexpr (kBits == 8) {
        const uint32_t wi = e0 / 4u;
        if (wi < nwords) gp(words)[wi] = packed;
    } else if constexpr (kBits == 4) {
        uint32_t x = packed << (16 * (lane & 1));
        x |= lane_xor1(x);
        const uint32_t wi = e0 / 8u;
        if ((lane & 1) == 0 && wi < nwords) gp(words)[wi] = x;
    } else {
        uint32_t x = packed << (8 * (lane & 3));
        x |= lane_xor1(x);
        x |= lane_xor2(x);
        const uint32_t wi = e0 / 16u;
        if ((lane & 3) == 0 && wi < nwords) gp(words)[wi] = x;
    }
}

// Quantize the four elements e0 .. e0+3 of tensor td held in v4 (valid4:
// which of them exist), with inv = fl32(s / m) and unit = fl32(m / s):
// stores their codes and leaves their residuals v - decode in v4.
template <int kBits>
__device__ __forceinline__ void quantize_round(const TDesc& td, uint32_t e0, bool any, float inv, float unit,
                                               float (&v4)[4], uint32_t valid4, const float (&u)[4],
                                               uint32_t* __restrict__ tw) {
    using Q = Quant<kBits>;
    uint32_t packed = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t level = 0;
        if (any && ((valid4 >> q) & 1u)) {
            const float x = fabsf(v4[q]) * inv;
            if (x >= (float)Q::kLevels) {
                level = (uint32_t)Q::kLevels;
            } else {
                const float fl = floorf(x);
                level = (uint32_t)fl + (u[q] < x - fl ? 1u : 0u);
            }
        }
        const uint32_t code = level ? (level | ((f2u(v4[q]) >> 31) << (kBits - 1))) : 0u;
        packed |= code << (kBits * q);
        v4[q] = v4[q] - quant_decode<kBits>(code, unit);
    }
    store_codes<kBits>(packed, e0, tw, td.k);
}

// Quantize chunk j of tensor td (v in registers, scale m): codes into the
// payload words, residual into e.
template <int kBits, bool kNT>
__device__ __forceinline__ void quantize_chunk(const TDesc& td, uint32_t j, float m, float (&v)[kEpt], uint32_t valid,
                                               uint64_t seed, uint32_t* __restrict__ words) {
    using Q = Quant<kBits>;
    const bool any = m > 0.f;
    const float inv = any ? (float)((double)Q::kLevels / (double)m) : 0.f;
    const float unit = (float)((double)m / (double)Q::kLevels);
    uint32_t* tw = words + td.off;
    float u[kRounds][4];
    chunk_uniforms(seed, td.tid, j, u);
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x;  // element of the tensor
        float v4[4] = {v[4 * r], v[4 * r + 1], v[4 * r + 2], v[4 * r + 3]};
        quantize_round<kBits>(td, e0, any, inv, unit, v4, (valid >> (4 * r)) & 0xFu, u[r], tw);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * r + q] = v4[q];
    }
    if (td.resid) store_chunk<kNT>(td.resid, td.n, j, v);
}

}  // namespace

// Pass 1: v = g + e (parked in e for pass 2) and the chunk's largest |v|
// bits.  Streams g and e_old past the cache for large calls; v is stored
// normally so that pass 2 finds it there.
template <bool kNT>
__global__ __launch_bounds__(kBlock) void quant_pass1(const TDesc* __restrict__ d, int T, Ws ws) {
    __shared__ uint32_t sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v<kNT>(td, j, td.resid != nullptr, v, valid);
    if (td.resid) store_chunk(td.resid, td.n, j, v);
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < kEpt; ++i) {
        const uint32_t k = ((valid >> i) & 1u) ? key_of(v[i]) : 0u;
        m = k > m ? k : m;
    }
    m = block_max_u32(m, sh);
    if (threadIdx.x == 0) ws.q_max[c] = m;
}

// Scales of tensors too large for pass 2 to reduce inline (and of empty
// tensors).
__global__ __launch_bounds__(kBlock) void quant_finalize(const TDesc* __restrict__ d, float* __restrict__ scale_out,
                                                         Ws ws) {
    __shared__ uint32_t sh[4];
    const int t = blockIdx.x;
    const TDesc td = d[t];
    if (td.nchunks > 0 && td.nchunks <= kQuantInlineChunks) return;
    const float m = td.nchunks ? u2f(tensor_max(ws.q_max, td, sh)) : 0.f;
    if (threadIdx.x == 0) {
        scale_out[t] = m;
        ws.s_val[t] = m;
    }
}

// Pass 2: quantize, pack, and write the residual.
template <int kBits, bool kNT>
__global__ __launch_bounds__(kBlock) void quant_pass2(const TDesc* __restrict__ d, int T, uint64_t seed,
                                                      uint32_t* __restrict__ words, float* __restrict__ scale_out,
                                                      Ws ws) {
    __shared__ uint32_t sh[4];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float m;
    if (td.nchunks <= kQuantInlineChunks) {
        m = u2f(tensor_max(ws.q_max, td, sh));
        if (j == 0 && threadIdx.x == 0) scale_out[t] = m;
    } else {
        m = ws.s_val[t];
    }
    float v[kEpt];
    uint32_t valid;
    load_stored_v(td, j, v, valid);  // e holds v after pass 1 (or v = g without error feedback)
    quantize_chunk<kBits, kNT>(td, j, m, v, valid, seed, words);
}

// One pass (tensors no longer than the resident grid), as the one-pass
// sign compress: chunk c publishes its largest |v| bits in a slot (with bit
// 31 set, 0 meaning not yet), the next chunk's loads go out, and chunk
// c - grid, kept in registers, is quantized once every slot of its tensor
// is published (the maximum of the slots is the scale, exact in any
// order).  Waits end by the same induction over the tensors when every
// workgroup is resident; past the host's wait limit a waiting workgroup
// computes the missing chunk maxima itself and publishes them by
// compare-and-swap (common.hpp), so waits end whatever the residency.
namespace {

constexpr int kHelpBatch = 256;  // missing maxima a waiting workgroup computes per pass

// Largest |v| bits over chunk j of tensor td, the owner's value (a maximum,
// so any order gives it), read one round of four elements at a time.
__device__ __forceinline__ uint32_t chunk_max_key(const TDesc& td, uint32_t j, uint32_t* sh) {
    uint32_t mk = 0;
#pragma unroll 1
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (e0 + q < td.n) {
                const float g = td.dtype == 0 ? gp((const float*)td.grad)[e0 + q]
                                              : h2f(gp((const uint16_t*)td.grad)[e0 + q]);
                const uint32_t k = key_of(td.resid ? g + gp(td.resid)[e0 + q] : g);
                mk = k > mk ? k : mk;
            }
        }
    }
    return block_max_u32(mk, sh);
}

// Largest |v| of tensor td from its slots (every thread returns it),
// waiting while a slot is empty; once `ticks` of the constant-rate counter
// have passed, each pass computes up to kHelpBatch missing maxima and
// publishes them by compare-and-swap.  ctl_sh: LDS, 2 + kHelpBatch ints.
__device__ __forceinline__ float quant_onepass_scale(const TDesc& td, uint32_t* slot, uint32_t* sh, uint32_t ticks,
                                                     int* ctl_sh) {
    int& pending_sh = ctl_sh[0];
    int& help_sh = ctl_sh[1];
    int* miss_sh = ctl_sh + 2;
    const uint64_t t0 = wall_clock64();
    uint32_t* sl = slot + td.chunk0;
    uint32_t mx;
    for (;;) {
        mx = 0;
        int missing = 0;
        for (uint32_t q = threadIdx.x; q < td.nchunks; q += kBlock) {
            const uint32_t x = __hip_atomic_load(sl + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            missing |= x == 0u;
            const uint32_t k = x & 0x7FFFFFFFu;
            mx = k > mx ? k : mx;
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
        if (threadIdx.x == 0) pending_sh = 0;
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < td.nchunks; q += kBlock) {
            if (__hip_atomic_load(sl + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
                const int k = atomicAdd(&pending_sh, 1);
                if (k < kHelpBatch) miss_sh[k] = (int)q;
            }
        }
        __syncthreads();
        const int m = pending_sh < kHelpBatch ? pending_sh : kHelpBatch;
        for (int i = 0; i < m; ++i) {
            const uint32_t q = (uint32_t)miss_sh[i];
            const uint32_t mk = chunk_max_key(td, q, sh);
            if (threadIdx.x == 0) {
                uint32_t expected = 0u;
                __hip_atomic_compare_exchange_strong(sl + q, &expected, mk | 0x80000000u, __ATOMIC_RELAXED,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __syncthreads();  // the list is reused by the next pass
    }
    return u2f(block_max_u32(mx, sh));
}
}  // namespace

template <int kBits, int kDT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void quant_onepass(const TDesc* __restrict__ d, int T, uint32_t C, uint64_t seed,
                                                        uint32_t* __restrict__ words, float* __restrict__ scale_out,
                                                        Ws ws, uint32_t wait_ticks) {
    __shared__ uint32_t sh[4];
    __shared__ int ctl_sh[2 + kHelpBatch];
    float vp[kEpt];
    uint32_t validp = 0;
    TDesc tdp{};
    bool prev = false;
    uint32_t jp = 0;
    float mp = 0.f;  // its scale when already known (a single-chunk tensor)
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
        float m_now = 0.f;
        if (have) {
            const int t = tensor_of_chunk(d, T, c);
            j = c - td.chunk0;
            raw_to_v<kDT>(td, td.resid != nullptr, raw, v);
            uint32_t mk = 0;
#pragma unroll
            for (int i = 0; i < kEpt; ++i) {
                const uint32_t k = ((raw.valid >> i) & 1u) ? key_of(v[i]) : 0u;
                mk = k > mk ? k : mk;
            }
            mk = block_max_u32(mk, sh);
            if (td.nchunks == 1) {
                m_now = u2f(mk);
                if (threadIdx.x == 0) scale_out[t] = m_now;
            } else if (threadIdx.x == 0) {
                __hip_atomic_store(ws.q_slot + c, mk | 0x80000000u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        const uint32_t valid_now = raw.valid;
        const uint32_t cn = c + gridDim.x;
        TDesc tdn{};
        if (cn < C) {
            tdn = d[tensor_of_chunk(d, T, cn)];
            load_raw<kDT>(tdn, cn - tdn.chunk0, tdn.resid != nullptr, raw);
        }
        if (prev) {
            float m = mp;
            if (tdp.nchunks > 1) {
                m = quant_onepass_scale(tdp, ws.q_slot, sh, wait_ticks, ctl_sh);
                if (jp == 0 && threadIdx.x == 0) scale_out[tensor_of_chunk(d, T, tdp.chunk0)] = m;
            }
            quantize_chunk<kBits, false>(tdp, jp, m, vp, validp, seed, words);
        }
        if (!have) break;
#pragma unroll
        for (int i = 0; i < kEpt; ++i) vp[i] = v[i];
        validp = valid_now;
        tdp = td;
        prev = true;
        jp = j;
        mp = m_now;
        td = tdn;
    }
}

// Slots of the one-pass kernel, emptied before it runs (a fill kernel).
__global__ void quant_onepass_reset(uint32_t C, Ws ws) {
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += gridDim.x * blockDim.x) ws.q_slot[c] = 0u;
}

__global__ void quant_empty_scales(const TDesc* __restrict__ d, int T, float* __restrict__ scale_out) {
    const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (t < T && d[t].nchunks == 0) scale_out[t] = 0.f;
}

// Residual update from a payload made elsewhere: e <- (g + e) - decode.
// Each thread's four consecutive elements of a round share one word.
template <int kBits>
__global__ __launch_bounds__(kBlock) void quant_residual_update(const TDesc* __restrict__ d, int T,
                                                                const uint32_t* __restrict__ words,
                                                                const float* __restrict__ scale) {
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_v(td, j, true, v, valid);
    const float unit = (float)((double)scale[t] / (double)Quant<kBits>::kLevels);
    const uint32_t* tw = words + td.off;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        const uint32_t e0 = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x;
        const uint32_t wi = e0 / (32u / kBits);
        const uint32_t word = wi < td.k ? gp(tw)[wi] : 0u;
        const uint32_t sh0 = (e0 % (32u / kBits)) * (uint32_t)kBits;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t code = (word >> (sh0 + (uint32_t)(kBits * q))) & Quant<kBits>::kMask;
            v[4 * r + q] = v[4 * r + q] - quant_decode<kBits>(code, unit);
        }
    }
    store_chunk(td.resid, td.n, j, v);
}

// ------------------------------------------------ TernGrad exact aggregate
// 2-bit codes decode to 0 or +-scale, so the TernGrad aggregate is, like
// the sign aggregate, the exact sum rounded once: with at most 64 workers
// whose nonzero scales span at most tern_span_limit(W) binades, every scale
// is an integer multiple of 2^(emin-150) below 2^(24+span), and the sum of
// W of them stays below 2^31: int32 arithmetic is exact.  Workers go in
// groups of four; a group's four 2-bit codes of an element form an 8-bit
// index into a 256-entry table of the group's sums.  Other scale sets (wider
// spans, subnormal or non-finite scales, more than 64 workers) take the
// multi-word exact path of exact_wide.hpp: one definition for every tensor.
namespace {
constexpr int kTernTab = 16 * 256;  // int32 entries per tensor: 16 groups of four workers

// The scale as a multiple of 2^(emin - 150) (zero stays zero).
__device__ __forceinline__ int32_t tern_scale_units(float sv, int emin) {
    const uint32_t b = f2u(sv);
    const int e = (int)((b >> 23) & 255u);
    if (e == 0) return 0;
    return (int32_t)(((b & 0x7FFFFFu) | 0x800000u) << (e - emin));
}

// Contribution of a 2-bit code (level bit 0, sign bit 1) of scale units sv.
__device__ __forceinline__ int32_t tern_code_value(uint32_t code, int32_t sv) {
    return (code & 1u) ? ((code & 2u) ? -sv : sv) : 0;
}
}  // namespace

// One wave per tensor: its form (info[t]: 1 tables, 0 wide exact path; emin in bits
// 8-15) and, for the exact form, its tables: tab[256 g + p] is the sum over
// the four workers 4g + c of the value of code (p >> 2c) & 3, built from two
// two-worker tables of 16 entries.  Workers past W count as zero.
__global__ __launch_bounds__(64) void tern_agg_prep(const ADesc* __restrict__ a, int T,
                                                    const uint64_t* __restrict__ wp, int W, int span_limit,
                                                    uint32_t* __restrict__ info, int32_t* __restrict__ tabs) {
    __shared__ float sc[64];
    __shared__ int32_t sub[16 * 32];
    const int t = blockIdx.x;
    if (a[t].nunits == 0) return;
    const int lane = (int)threadIdx.x;
    int lo = 1000, hi = -1000, bad = W > 64;
    for (int w = lane; w < W && w < 64; w += 64) {
        const float sv = gp((const float*)w_b(wp, W, w))[t];
        sc[w] = sv;
        const int e = (int)((f2u(sv) >> 23) & 255u);
        if (e == 255 || (e == 0 && (f2u(sv) & 0x7FFFFFu))) bad = 1;
        else if (e) {
            lo = e < lo ? e : lo;
            hi = e > hi ? e : hi;
        }
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
        const int lo2 = __shfl_xor(lo, m, 64), hi2 = __shfl_xor(hi, m, 64);
        lo = lo2 < lo ? lo2 : lo;
        hi = hi2 > hi ? hi2 : hi;
        bad |= __shfl_xor(bad, m, 64);
    }
    const int span = hi < lo ? 0 : hi - lo;
    const int form = !bad && span <= span_limit ? 1 : 0;
    const int emin = hi < lo ? 1 : lo;
    if (lane == 0) info[t] = (uint32_t)form | ((uint32_t)emin << 8);
    if (form != 1) return;
    __builtin_amdgcn_wave_barrier();
    // sub[32 g + 16 h + p]: workers 4g + 2h + c, c < 2, with codes (p >> 2c) & 3
    for (int x = lane; x < 16 * 32; x += 64) {
        const int w0 = 4 * (x >> 5) + 2 * ((x >> 4) & 1), pat = x & 15;
        int32_t acc = 0;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int32_t sv = w0 + c < W ? tern_scale_units(sc[w0 + c], emin) : 0;
            acc += tern_code_value((uint32_t)(pat >> (2 * c)) & 3u, sv);
        }
        sub[x] = acc;
    }
    __builtin_amdgcn_wave_barrier();
    int32_t* tt = tabs + (size_t)t * kTernTab;
    for (int x = 4 * lane; x < kTernTab; x += 256) {
        const int g = x >> 8, p0 = x & 255;
        const int32_t hi16 = sub[32 * g + 16 + (p0 >> 4)];
        u32x4 v;
        v.x = (uint32_t)(sub[32 * g + ((p0 + 0) & 15)] + hi16);
        v.y = (uint32_t)(sub[32 * g + ((p0 + 1) & 15)] + hi16);
        v.z = (uint32_t)(sub[32 * g + ((p0 + 2) & 15)] + hi16);
        v.w = (uint32_t)(sub[32 * g + ((p0 + 3) & 15)] + hi16);
        *(BC_GLOBAL u32x4*)(gp(tt) + x) = v;
    }
}

namespace {
// Indices of one group of four workers for the lane's 16 elements: x[k] is
// worker 4g + k's word (element q's code at bits 2q).  v_perm gathers byte j
// of the four words (elements 4j .. 4j+3, one byte per worker) and a 4x4
// transpose of 2-bit fields (two delta swaps) turns byte i into element
// 4j + i's index, worker k's code at bits 2k.
__device__ __forceinline__ void tern_indices(const uint32_t (&x)[4], uint32_t (&y)[4]) {
    const uint32_t p01 = __builtin_amdgcn_perm(x[1], x[0], 0x05010400u);
    const uint32_t q01 = __builtin_amdgcn_perm(x[1], x[0], 0x07030602u);
    const uint32_t r23 = __builtin_amdgcn_perm(x[3], x[2], 0x05010400u);
    const uint32_t s23 = __builtin_amdgcn_perm(x[3], x[2], 0x07030602u);
    y[0] = __builtin_amdgcn_perm(r23, p01, 0x05040100u);
    y[1] = __builtin_amdgcn_perm(r23, p01, 0x07060302u);
    y[2] = __builtin_amdgcn_perm(s23, q01, 0x05040100u);
    y[3] = __builtin_amdgcn_perm(s23, q01, 0x07060302u);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        uint32_t v = y[j];
        uint32_t t = ((v >> 12) ^ v) & 0x0000F0F0u;
        v ^= t ^ (t << 12);
        t = ((v >> 6) ^ v) & 0x00CC00CCu;
        v ^= t ^ (t << 6);
        y[j] = v;
    }
}
}  // namespace

// Aggregate: one workgroup per 4096-element unit of a tensor, lane l of
// the workgroup owning elements 16 l .. 16 l + 15 of the unit (16 kBits
// bits: kBits / 2 consecutive words of every worker's payload).
//
// Decoding in the inner loop is branch-free: the level bits are widened
// (2-bit: a sign-extended one-bit field masks the unit; 4- and 8-bit:
// level * unit) and the code's sign bit is spliced in at bit 31 with a
// bit-field insert.  A level-0 code with its sign bit set (never written
// by the compressor) then decodes to -0.0 rather than +0.0; the running
// sum never holds -0.0 (it starts at +0.0, and x + (-x) rounds to +0.0),
// and adding either zero to a value that is not -0.0 gives the same
// result, so the sums are those of the +0.0 decoding.
//
// 2-bit codes (TernGrad) are summed exactly.  A tensor in the table form
// (info[t] & 255 == 1) takes the table path: the workgroup copies the
// tensor's tables into LDS, loads the words of all (at most 16 kTS) workers
// at once, and adds one table entry per element and group of four workers
// in int32.  Other tensors take the wide exact path.
template <int kBits, int kTS>
__global__ __launch_bounds__(kBlock) void aggregate_quant(const ADesc* __restrict__ a, int T, uint32_t U,
                                                          const uint64_t* __restrict__ wp, int W, float alpha,
                                                          const uint32_t* __restrict__ info,
                                                          const int32_t* __restrict__ tabs) {
    constexpr int kWords = kBits / 2;
    constexpr int kGroup = 8;  // workers whose words are in flight together
    using Q = Quant<kBits>;
    __shared__ float unit_sh[1024];
    __shared__ __attribute__((aligned(16))) int32_t tab_sh[kBits == 2 ? 256 * 4 * kTS : 4];
    static_assert(kBits != 2 || sizeof(tab_sh) >= kWideScratchBytes, "wide-path scratch");
    const uint32_t u = blockIdx.x;
    const int t = unit_owner(wp, W, u);
    const ADesc ad = a[t];
    for (int w = threadIdx.x; w < W; w += kBlock)
        unit_sh[w] = (float)((double)gp(w_b(wp, W, w))[t] / (double)Q::kLevels);
    __syncthreads();
    const uint32_t e_first = (u - ad.unit0) * kSignAggUnit + 16u * threadIdx.x;  // element of the tensor
    const uint32_t w_first = e_first / (32u / kBits);                          // word of the tensor
    // a unit inside the tensor reads each worker's kWords words with one
    // vector load (4-byte aligned: word offsets are arbitrary); the last
    // unit of a tensor reads word by word, words past the tensor's end
    // reading its last word and decoding as zero
    const bool whole = (uint64_t)(u - ad.unit0 + 1u) * kSignAggUnit <= ad.n;
    uint32_t widx[kWords];
    uint32_t wkeep[kWords];
#pragma unroll
    for (int k = 0; k < kWords; ++k) {
        const bool in = w_first + k < ad.k;
        widx[k] = in ? w_first + k : ad.k - 1u;
        wkeep[k] = in ? 0xFFFFFFFFu : 0u;
    }
    auto load_words = [&](const uint32_t* base, uint32_t (&wd)[kWords]) {
        if (whole) {
            typedef uint32_t vec_t __attribute__((ext_vector_type(kWords), aligned(4)));
            const vec_t x = *(const BC_GLOBAL vec_t*)(gp(base) + w_first);
#pragma unroll
            for (int k = 0; k < kWords; ++k) wd[k] = x[k];
        } else {
#pragma unroll
            for (int k = 0; k < kWords; ++k) wd[k] = gp(base)[widx[k]] & wkeep[k];
        }
    };
    float acc[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[q] = 0.f;
    if constexpr (kBits == 2) {
        const uint32_t inf = info[t];
        if ((inf & 255u) != 1u) {
            // scales the int32 tables cannot hold exactly (or more than 64
            // workers): the wide exact path writes the unit's outputs itself
            aggregate_unit_exact_wide<1>(ad, (int64_t)(u - ad.unit0) * kSignAggUnit, wp, W, alpha, unit_sh,
                                         reinterpret_cast<unsigned char*>(tab_sh));
            return;
        }
        {
            const int G4 = (W + 3) / 4;  // <= 4 kTS
            const int32_t* tt = tabs + (size_t)t * kTernTab;
            uint32_t wv[16 * kTS];
#pragma unroll
            for (int k = 0; k < 16 * kTS; ++k) {
                uint32_t wd[1];
                load_words(w_a(wp, k < W ? k : W - 1) + ad.off, wd);
                wv[k] = wd[0];
            }
            for (int x = 4 * (int)threadIdx.x; x < 256 * G4; x += 4 * kBlock)
                *reinterpret_cast<u32x4*>(tab_sh + x) = ldg4u(tt + x);
            __syncthreads();
            int32_t S[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) S[q] = 0;
#pragma unroll
            for (int g = 0; g < 4 * kTS; ++g) {
                if (g < G4) {
                    const uint32_t xw[4] = {wv[4 * g], wv[4 * g + 1], wv[4 * g + 2], wv[4 * g + 3]};
                    uint32_t y[4];
                    tern_indices(xw, y);
                    const int32_t* tg = tab_sh + 256 * g;
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int i = 0; i < 4; ++i) S[4 * j + i] += tg[(y[j] >> (8 * i)) & 255u];
                }
            }
            // exact: |S| < 2^31 and the unit is a power of two
            const double unit = __builtin_ldexp(1.0, (int)((inf >> 8) & 255u) - 150);
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[q] = (float)((double)S[q] * unit);
        }
    }
    auto add_worker = [&](const uint32_t (&wd)[kWords], float un) {
        const uint32_t ub = f2u(un);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            constexpr int kPer = 32 / kBits;
            const uint32_t word = wd[q / kPer];
            const int pos = (q % kPer) * kBits;  // first bit of the code
            float mag;
            if constexpr (kBits == 2) {
                mag = u2f(ub & (uint32_t)__builtin_amdgcn_sbfe((int)word, pos, 1));
            } else {
                mag = (float)__builtin_amdgcn_ubfe(word, pos, kBits - 1) * un;
            }
            const uint32_t sgn = word << (31 - (pos + kBits - 1));  // the code's sign bit at bit 31
            acc[q] += u2f((sgn & 0x80000000u) ^ f2u(mag));
        }
    };
    int w0 = 0;
    if constexpr (kBits == 2) w0 = W;  // summed on the table path
    for (; w0 + kGroup <= W; w0 += kGroup) {
        uint32_t wd[kGroup][kWords];
#pragma unroll
        for (int g = 0; g < kGroup; ++g) load_words(w_a(wp, w0 + g) + ad.off, wd[g]);
#pragma unroll
        for (int g = 0; g < kGroup; ++g) add_worker(wd[g], unit_sh[w0 + g]);
    }
    for (; w0 < W; ++w0) {
        uint32_t wd[kWords];
        load_words(w_a(wp, w0) + ad.off, wd);
        add_worker(wd, unit_sh[w0]);
    }
    float* out = ad.out + e_first;
    if (e_first + 16u <= ad.n) {
#pragma unroll
        for (int q = 0; q < 16; q += 4)
            stg4f(out + q, f32x4{alpha * acc[q], alpha * acc[q + 1], alpha * acc[q + 2], alpha * acc[q + 3]});
    } else {
#pragma unroll
        for (int q = 0; q < 16; ++q)
            if (e_first + q < ad.n) gp(out)[q] = alpha * acc[q];
    }
}

// ------------------------------------------------------------- launchers
namespace {
template <int kBits>
void quant_compress_bits(const TDesc* d, int T, uint32_t C, bool nt, uint64_t seed, uint32_t* words, float* scale,
                         const Ws& ws, hipStream_t s) {
    if (nt) hipLaunchKernelGGL((quant_pass2<kBits, true>), dim3(C), dim3(kBlock), 0, s, d, T, seed, words, scale, ws);
    else hipLaunchKernelGGL((quant_pass2<kBits, false>), dim3(C), dim3(kBlock), 0, s, d, T, seed, words, scale, ws);
}
}  // namespace

namespace {
template <int kBits, int kDT>
uint32_t quant_onepass_capacity(int cus) {
    static int per_cu = -1;
    if (per_cu < 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, quant_onepass<kBits, kDT>, kBlock, 0) != hipSuccess)
            nb = 0;
        per_cu = nb;
    }
    return (uint32_t)per_cu * (uint32_t)(cus > 0 ? cus : 0);
}

template <int kBits, int kDT>
bool quant_onepass_launch(uint64_t seed, const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty,
                          uint32_t* words, float* scale, const Ws& ws, int cus, hipStream_t s) {
    const uint32_t cap = quant_onepass_capacity<kBits, kDT>(cus);
    if (C == 0 || cap == 0 || max_chunks > cap) return false;
    const uint32_t grid = C < cap ? C : cap;
    hipLaunchKernelGGL(quant_onepass_reset, dim3((C + 255) / 256 < 1024 ? (C + 255) / 256 : 1024), dim3(256), 0, s,
                       C, ws);
    (void)launch_timed(kTimedQuantOnepass, quant_onepass<kBits, kDT>, dim3(grid), dim3(kBlock), 0, s, d, T, C, seed,
                       words, scale, ws, onepass_wait_ticks());
    if (any_empty) hipLaunchKernelGGL(quant_empty_scales, dim3((T + 255) / 256), dim3(256), 0, s, d, T, scale);
    return true;
}

template <int kBits>
bool quant_onepass_dt(uint64_t seed, const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty,
                      bool any_f16, bool any_f32, uint32_t* words, float* scale, const Ws& ws, int cus,
                      hipStream_t s) {
    if (any_f16 && any_f32)
        return quant_onepass_launch<kBits, 2>(seed, d, T, C, max_chunks, any_empty, words, scale, ws, cus, s);
    if (any_f16) return quant_onepass_launch<kBits, 1>(seed, d, T, C, max_chunks, any_empty, words, scale, ws, cus, s);
    return quant_onepass_launch<kBits, 0>(seed, d, T, C, max_chunks, any_empty, words, scale, ws, cus, s);
}
}  // namespace

hipError_t launch_quant_compress(int bits, uint64_t seed, const TDesc* d, int T, uint32_t C, uint32_t max_chunks,
                                 bool any_empty, bool any_f16, bool any_f32, uint32_t* words, float* scale,
                                 const Ws& ws, int cus, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    // one pass when every tensor fits the resident grid
    const bool one =
        bits == 2   ? quant_onepass_dt<2>(seed, d, T, C, max_chunks, any_empty, any_f16, any_f32, words, scale, ws, cus, s)
        : bits == 4 ? quant_onepass_dt<4>(seed, d, T, C, max_chunks, any_empty, any_f16, any_f32, words, scale, ws, cus, s)
                    : quant_onepass_dt<8>(seed, d, T, C, max_chunks, any_empty, any_f16, any_f32, words, scale, ws, cus, s);
    if (one) return hipGetLastError();
    const bool nt = C > kNtChunks;
    if (C > 0) {
        if (nt) (void)launch_timed(kTimedQuantPass1, quant_pass1<true>, dim3(C), dim3(kBlock), 0, s, d, T, ws);
        else (void)launch_timed(kTimedQuantPass1, quant_pass1<false>, dim3(C), dim3(kBlock), 0, s, d, T, ws);
    }
    if (max_chunks > kQuantInlineChunks || C == 0 || any_empty)
        hipLaunchKernelGGL(quant_finalize, dim3(T), dim3(kBlock), 0, s, d, scale, ws);
    if (C > 0) {
        if (bits == 2) quant_compress_bits<2>(d, T, C, nt, seed, words, scale, ws, s);
        else if (bits == 4) quant_compress_bits<4>(d, T, C, nt, seed, words, scale, ws, s);
        else quant_compress_bits<8>(d, T, C, nt, seed, words, scale, ws, s);
    }
    return hipGetLastError();
}

hipError_t launch_quant_residual_update(int bits, const TDesc* d, int T, uint32_t C, const uint32_t* words,
                                        const float* scale, hipStream_t s) {
    if (C == 0) return hipSuccess;
    if (bits == 2) hipLaunchKernelGGL(quant_residual_update<2>, dim3(C), dim3(kBlock), 0, s, d, T, words, scale);
    else if (bits == 4) hipLaunchKernelGGL(quant_residual_update<4>, dim3(C), dim3(kBlock), 0, s, d, T, words, scale);
    else hipLaunchKernelGGL(quant_residual_update<8>, dim3(C), dim3(kBlock), 0, s, d, T, words, scale);
    return hipGetLastError();
}

hipError_t launch_aggregate_quant(int bits, const ADesc* a, int T, uint32_t U, const uint64_t* wp, int W,
                                  float alpha, uint32_t* info, int32_t* tabs, hipStream_t s) {
    if (U == 0) return hipSuccess;
    if (W > 1024) return hipErrorInvalidValue;
    const dim3 grid(U), block(kBlock);
    if (bits == 2) {
        // 24 + span + ceil(log2 W4) <= 31, W4 = W rounded up to a multiple of 4
        const int w4 = 4 * ((W + 3) / 4);
        int lg = 0;
        while ((1 << lg) < w4) ++lg;
        hipLaunchKernelGGL(tern_agg_prep, dim3(T), dim3(64), 0, s, a, T, wp, W, 7 - lg, info, tabs);
        const uint32_t* ci = info;
        const int32_t* ct = tabs;
        const int steps = W > 64 ? 1 : (W + 15) / 16;
        if (steps <= 1) return launch_timed(kTimedAggQuant, aggregate_quant<2, 1>, grid, block, 0, s, a, T, U, wp, W, alpha, ci, ct);
        if (steps == 2) return launch_timed(kTimedAggQuant, aggregate_quant<2, 2>, grid, block, 0, s, a, T, U, wp, W, alpha, ci, ct);
        if (steps == 3) return launch_timed(kTimedAggQuant, aggregate_quant<2, 3>, grid, block, 0, s, a, T, U, wp, W, alpha, ci, ct);
        return launch_timed(kTimedAggQuant, aggregate_quant<2, 4>, grid, block, 0, s, a, T, U, wp, W, alpha, ci, ct);
    }
    const uint32_t* nul = nullptr;
    const int32_t* nt = nullptr;
    if (bits == 4)
        return launch_timed(kTimedAggQuant, aggregate_quant<4, 1>, grid, block, 0, s, a, T, U, wp, W, alpha, nul, nt);
    return launch_timed(kTimedAggQuant, aggregate_quant<8, 1>, grid, block, 0, s, a, T, U, wp, W, alpha, nul, nt);
}

}  // namespace bc
