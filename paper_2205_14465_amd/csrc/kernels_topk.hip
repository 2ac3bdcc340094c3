// kernels_topk.hip -- top-k sparsification with error feedback on gfx950:
// exact top-k and the DGC-style sampled-threshold variant (paper Sec. 2.3,
// sparsification; Sec. 5.1, DGC at a 1% rate with error feedback).
//
// Result (both kinds): the k_t entries of v = g + e_old with the largest
// |v| (keys = magnitude bits), ties to the lower index, emitted with
// ascending indices and values v[idx]; residual e_new = v with the chosen
// entries set to +0.0.
//
// Pipeline (all tensors of a call advance together, one launch per step):
//   exact:    stream pass 1 writes e_new = v and a 2048-bin histogram of
//             key bits 30..20 per tensor -> exact bin of the k-th key ->
//             stream pass 2 re-reads v and compacts the candidates (keys at
//             or above that bin) per 4096-element chunk, in index order.
//   sampled:  a seeded 1% sample (runs of 64 elements) histogrammed per
//             tensor -> threshold bin with a margin -> ONE stream pass
//             writes e_new = v and compacts candidates.  If a tensor ends
//             with fewer than k candidates, the exact histogram path runs
//             for that tensor only (reading v back from e_new).
//   both:     radix select over the candidates only (digits of 11, 10 and
//             10 bits, histograms in LDS, merged with integer atomics)
//             finds the k-th key tau and how many tau-ties to keep; a scan
//             over chunks places each chunk's winners; the emit pass writes
//             the payload and zeroes e_new at the winners.
// Trimming or topping up to exactly k in the selection order makes the
// sampled kind return the same entries as the exact kind.
//
// A DGC step (Sec. 5.1) runs inside the same passes: the pass that forms v
// (the exact path's histogram pass, the sampled path's stream pass; the
// sample reads the same values) first takes the velocity step
// u <- fl32(fl32(m * u) + fl32(c * g)) and writes u, then v = fl32(u + e);
// the emit pass writes +0.0 into u as well as e_new at the winners.  The
// call's table then holds u in the gradient's place; the gradients come
// from a second table of the same tensors.
#include "launch.hpp"

namespace bc {

namespace {

enum FindMode : int {
    kFindThrExact = 0,    // histogram of all keys -> bin of the k-th key
    kFindThrSample = 1,   // histogram of sample keys -> threshold with margin
    kFindDigit0 = 2,      // candidates' bits 30..20 (sets t_fb if too few)
    kFindDigit1 = 3,      // bits 19..10
    kFindDigit2 = 4,      // bits 9..0
};

constexpr uint32_t kAllCandidatesBelow = 16u * kChunk;  // small tensors skip the sample

__device__ __forceinline__ bool active(const uint32_t* fb, int t, bool fb_only) {
    return !fb_only || fb[t] != 0u;
}

// The DGC velocity step of a chunk: td holds u (as the fp32 gradient) and
// e, tg the step's gradient; u receives fl32(fl32(m * u) + fl32(c * g))
// (c the clipping factor, or g as widened without clipping) and v fl32(u + e),
// +0.0 past the tensor's end.
template <bool kNT>
__device__ __forceinline__ void load_v_dgc(const TDesc& td, const TDesc& tg, uint32_t j, const DgcFuse& f,
                                           float u[kEpt], float v[kEpt], uint32_t& valid) {
    float g[kEpt], e[kEpt];
    load_v<kNT>(tg, j, false, g, valid);
    load_v<kNT>(td, j, false, u, valid);
    TDesc te = td;
    te.grad = td.resid;
    load_v<kNT>(te, j, false, e, valid);
    if (f.clip) {
        const float cf = *f.clip;
#pragma unroll
        for (int i = 0; i < kEpt; ++i) g[i] = cf * g[i];
    }
#pragma unroll
    for (int i = 0; i < kEpt; ++i) {
        const float mu = f.m * u[i];
        u[i] = mu + g[i];
        v[i] = u[i] + e[i];
    }
}

__device__ __forceinline__ float* vel_of(const TDesc& td) { return (float*)const_cast<void*>(td.grad); }

// Flush a block's LDS histogram into the tensor's global histogram.
__device__ __forceinline__ void flush_hist(const uint32_t* lh, uint32_t* gh, int bins) {
    for (int b = threadIdx.x; b < bins; b += kBlock) {
        const uint32_t x = lh[b];
        if (x) atomicAdd(gh + b, x);
    }
}

}  // namespace

// Stream pass of the exact path: e_new = v (when `write_resid`; kDGC: after
// the velocity step) and the histogram of key bits 30..20.  With `fb_only`
// it re-reads the stored v of tensors flagged for the fallback.
template <bool kDGC>
__global__ __launch_bounds__(kBlock) void topk_hist_pass(const TDesc* __restrict__ d, int T, uint32_t C,
                                                         int write_resid, int fb_only, Ws ws,
                                                         uint64_t* __restrict__ clear_status, int copies,
                                                         DgcFuse f) {
    __shared__ uint32_t lh[kBins0];
    if (fb_only && ws.t_any[0] == 0u) return;  // no tensor fell back
    for (uint32_t c = blockIdx.x; c < C; c += gridDim.x) {
        if (clear_status && threadIdx.x == 0) clear_status[c] = 0ull;
        const int t = tensor_of_chunk(d, T, c);
        if (!active(ws.t_fb, t, fb_only)) continue;
        const TDesc td = d[t];
        const uint32_t j = c - td.chunk0;
        for (int b = threadIdx.x; b < kBins0; b += kBlock) lh[b] = 0;
        float v[kEpt];
        uint32_t valid;
        if (kDGC && write_resid) {
            float u[kEpt];
            load_v_dgc<false>(td, f.dg[t], j, f, u, v, valid);
            store_chunk(vel_of(td), td.n, j, u);
            store_chunk(td.resid, td.n, j, v);
        } else if (write_resid) {
            load_v(td, j, td.resid != nullptr, v, valid);
            if (td.resid) store_chunk(td.resid, td.n, j, v);
        } else {
            load_stored_v(td, j, v, valid);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kEpt; ++i)
            if ((valid >> i) & 1u) atomicAdd(&lh[key_of(v[i]) >> 20], 1u);
        __syncthreads();
        flush_hist(lh, ws.t_hist + ((size_t)(c % (uint32_t)copies) * T + t) * kBins0, kBins0);
        __syncthreads();
    }
}

// Seeded sample: each 4096-element chunk of a tensor larger than
// kAllCandidatesBelow contributes one run of 64 consecutive elements with
// probability 0.64 (an expected 1% of the tensor).  A workgroup covers 16
// consecutive chunks, four per wave: lanes 0..3 of a wave draw its four
// chunks' runs at once, then the wave issues the four runs' loads together;
// when the 16 chunks all belong to one tensor (the usual case) the keys
// are binned in LDS first so the global histogram sees one atomic per
// non-empty bin.
constexpr uint32_t kSampleChunksPerBlock = 16;

template <bool kDGC>
__global__ __launch_bounds__(kBlock) void topk_sample_hist(const TDesc* __restrict__ d, int T,
                                                           uint32_t C, uint64_t seed, int copies, Ws ws,
                                                           DgcFuse f) {
    uint32_t* gh0 = ws.t_hist + (size_t)(blockIdx.x % (uint32_t)copies) * T * kBins0;  // this workgroup's copy
    __shared__ uint32_t lh[kBins0];
    const uint32_t c0 = blockIdx.x * kSampleChunksPerBlock;
    const uint32_t c1 = (c0 + kSampleChunksPerBlock < C) ? c0 + kSampleChunksPerBlock : C;
    const int t0 = tensor_of_chunk(d, T, c0);
    const bool same = tensor_of_chunk(d, T, c1 - 1) == t0;
    if (same && d[t0].n < kAllCandidatesBelow) return;
    if (same)
        for (int b = threadIdx.x; b < kBins0; b += kBlock) lh[b] = 0;
    __syncthreads();
    const int lane = lane_id();
    // lane q < 4: the run of chunk c0 + wave + 4q (start element, tensor; -1: none)
    uint32_t run_start = 0;
    int run_t = -1;
    if (lane < 4) {
        const uint32_t c = c0 + (uint32_t)wave_id() + 4u * (uint32_t)lane;
        if (c < c1) {
            const int t = tensor_of_chunk(d, T, c);
            const TDesc td = d[t];
            const uint32_t j = c - td.chunk0;
            U64x4 ctr = {{(uint64_t)td.tid, (uint64_t)j, 0, 0}};
            const U64x4 r = philox4x64_10(ctr, seed, kStreamSample);
            const uint32_t u = (uint32_t)(r.v[0] >> 32);
            const uint32_t len = (j + 1 == td.nchunks) ? td.n - j * (uint32_t)kChunk : (uint32_t)kChunk;
            if (td.n >= kAllCandidatesBelow && u < 2748779069u && len >= 64) {  // 0.64 * 2^32
                run_start = j * (uint32_t)kChunk + (uint32_t)(r.v[1] % (uint64_t)(len - 63));
                run_t = t;
            }
        }
    }
    float v[4];
    int tq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        tq[q] = __builtin_amdgcn_readlane(run_t, q);
        v[q] = 0.f;
        if (tq[q] < 0) continue;
        const uint32_t i = (uint32_t)__builtin_amdgcn_readlane((int)run_start, q) + (uint32_t)lane;
        const TDesc td = d[tq[q]];
        if constexpr (kDGC) {  // the value the stream pass will form
            const TDesc tg = f.dg[tq[q]];
            float g;
            if (tg.dtype == 0) g = gp((const float*)tg.grad)[i];
            else g = h2f(gp((const uint16_t*)tg.grad)[i]);
            if (f.clip) g = *f.clip * g;
            const float mu = f.m * gp((const float*)td.grad)[i];
            const float uu = mu + g;
            v[q] = uu + gp(td.resid)[i];
        } else {
            float g;
            if (td.dtype == 0) g = gp((const float*)td.grad)[i];
            else g = h2f(gp((const uint16_t*)td.grad)[i]);
            v[q] = td.resid ? g + gp(td.resid)[i] : g;
        }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (tq[q] < 0) continue;
        const uint32_t bin = key_of(v[q]) >> 20;
        if (same) atomicAdd(&lh[bin], 1u);
        else atomicAdd(gh0 + (size_t)tq[q] * kBins0 + bin, 1u);
    }
    if (!same) return;
    __syncthreads();
    flush_hist(lh, gh0 + (size_t)t0 * kBins0, kBins0);
}

// One workgroup per tensor: read (and clear) the tensor's histogram and
// pick the bin / digit the mode asks for.
__global__ __launch_bounds__(kBlock) void topk_find(const TDesc* __restrict__ d, int T, double ratio,
                                                    int mode, int fb_only, int copies, Ws ws) {
    __shared__ uint64_t sh[4];
    __shared__ uint32_t found_bin, found_above, found_total;
    if (fb_only && ws.t_any[0] == 0u) return;  // no tensor fell back
    const int t = blockIdx.x;
    const TDesc td = d[t];
    if (td.k == 0 || !active(ws.t_fb, t, fb_only)) return;
    const int bins = (mode == kFindDigit1 || mode == kFindDigit2) ? kBins12 : kBins0;
    const int per = bins / kBlock;
    uint32_t* gh = ws.t_hist + (size_t)t * kBins0;
    const size_t cs = (size_t)T * kBins0;  // between copies
    // thread i owns bins [bins - (i+1)*per, bins - i*per): thread 0 the top
    const int hi = bins - threadIdx.x * per;
    uint32_t h[8];
    uint32_t mine = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) h[q] = 0;
    // every copy's loads issued together (at most 8 copies)
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        if (r < copies) {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (q < per) h[q] += gh[r * cs + hi - 1 - q];
        }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        if (r < copies) {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (q < per) gh[r * cs + hi - 1 - q] = 0;
        }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) mine += q < per ? h[q] : 0u;
    uint64_t total64;
    const uint64_t above0 = block_excl_scan_u64(mine, sh, total64);
    const uint32_t total = (uint32_t)total64;
    uint32_t target;
    if (mode == kFindThrExact) {
        target = td.k;
    } else if (mode == kFindThrSample) {
        if (td.n < kAllCandidatesBelow || total == 0) {
            if (threadIdx.x == 0) ws.t_thr[t] = 0;
            return;
        }
        // k rule on the sample size, plus a margin so that the candidates
        // usually cover the k-th key of the tensor
        const uint64_t ppm = (uint64_t)llround(ratio * 1e6);
        uint64_t ks = ((uint64_t)total * ppm + 999999u) / 1000000u;
        if (ks < 1) ks = 1;
        uint64_t tg = ks + ks / 4 + 16;
        target = (uint32_t)(tg < total ? tg : total);
    } else if (mode == kFindDigit0) {
        target = td.k;
        if (total < td.k) {  // too few candidates: exact fallback for this tensor
            if (threadIdx.x == 0) {
                ws.t_fb[t] = 1u;
                atomicOr(ws.t_any, 1u);
            }
            return;
        }
        // a tensor that fell back keeps its flag (bytecomp_topk_stats counts them)
        if (threadIdx.x == 0 && !fb_only) ws.t_fb[t] = 0u;
    } else {
        target = ws.t_krem[t];
    }
    if (threadIdx.x == 0) found_total = total;
    uint32_t above = (uint32_t)above0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        if (q < per) {
            if (above < target && target <= above + h[q]) {
                found_bin = (uint32_t)(hi - 1 - q);
                found_above = above;
            }
            above += h[q];
        }
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    const uint32_t b = found_bin;
    switch (mode) {
        case kFindThrExact:
        case kFindThrSample:
            ws.t_thr[t] = b << 20;
            break;
        case kFindDigit0:
            ws.t_prefix[t] = b << 20;
            ws.t_krem[t] = target - found_above;
            break;
        case kFindDigit1:
            ws.t_prefix[t] |= b << 10;
            ws.t_krem[t] = target - found_above;
            break;
        default:
            ws.t_prefix[t] |= b;
            ws.t_krem[t] = target - found_above;
            break;
    }
    (void)found_total;
}

// Candidate compaction.  Stream mode (sampled main pass): v = g + e,
// e_new = v written back (kDGC: after the velocity step, u written back).
// Re-read mode: v from the residual (or g).  Candidates = valid entries
// with key >= t_thr[t], compacted in index order into the chunk's slot of
// t_cand; also the LDS histogram of their key bits 30..20.
template <bool kNT, bool kDGC>
__global__ __launch_bounds__(kBlock) void topk_compact(const TDesc* __restrict__ d, int T, uint32_t C,
                                                       int stream_mode, int fb_only, int copies, Ws ws,
                                                       DgcFuse f) {
    __shared__ uint32_t lh[kBins0];
    __shared__ uint64_t sh[4];
    if (fb_only && ws.t_any[0] == 0u) return;  // no tensor fell back
    for (uint32_t c = blockIdx.x; c < C; c += gridDim.x) {
        const int t = tensor_of_chunk(d, T, c);
        if (!active(ws.t_fb, t, fb_only)) continue;
        const TDesc td = d[t];
        const uint32_t j = c - td.chunk0;
        for (int b = threadIdx.x; b < kBins0; b += kBlock) lh[b] = 0;
        float v[kEpt];
        uint32_t valid;
        if (kDGC && stream_mode) {
            float u[kEpt];
            load_v_dgc<kNT>(td, f.dg[t], j, f, u, v, valid);
            store_chunk<kNT>(vel_of(td), td.n, j, u);
            store_chunk<kNT>(td.resid, td.n, j, v);
        } else if (stream_mode) {
            load_v<kNT>(td, j, td.resid != nullptr, v, valid);
            if (td.resid) store_chunk<kNT>(td.resid, td.n, j, v);
        } else {
            load_stored_v(td, j, v, valid);
        }
        const uint32_t thr = ws.t_thr[t];
        uint32_t pm = 0;
#pragma unroll
        for (int i = 0; i < kEpt; ++i)
            if (((valid >> i) & 1u) && key_of(v[i]) >= thr) pm |= 1u << i;
        uint64_t packed = 0;
#pragma unroll
        for (int r = 0; r < kRounds; ++r) packed |= (uint64_t)__popc((pm >> (4 * r)) & 0xFu) << (16 * r);
        uint64_t tot;
        const uint64_t pre = block_excl_scan_u64(packed, sh, tot);
        uint2* out = ws.t_cand + (size_t)c * kChunk;
        uint32_t base = 0;
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
            uint32_t rank = base + (uint32_t)((pre >> (16 * r)) & 0xFFFFu);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = 4 * r + q;
                if ((pm >> i) & 1u) {
                    const uint32_t e = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x + q;
                    out[rank++] = make_uint2(e, f2u(v[i]));
                    atomicAdd(&lh[key_of(v[i]) >> 20], 1u);
                }
            }
            base += (uint32_t)((tot >> (16 * r)) & 0xFFFFu);
        }
        if (threadIdx.x == 0) ws.t_ccount[c] = base;
        __syncthreads();
        flush_hist(lh, ws.t_hist + ((size_t)(c % (uint32_t)copies) * T + t) * kBins0, kBins0);
        __syncthreads();
    }
}

// Candidate passes.  A chunk holds about 50 candidates at a 1% rate.  The
// histogram pass gives each workgroup a range of `span` chunks (sized so
// that about a thousand workgroups remain), paying the clearing and flushing
// of its LDS histogram once per range; the count and emit passes give each
// wave one chunk.

// Radix pass over the candidates of a chunk range (at most 16 chunks):
// histogram of the next digit among candidates whose higher bits match the
// prefix chosen so far.  A range inside one tensor (the usual case) walks
// its candidates as one flattened list, every thread's loads in flight
// together; a range that crosses tensors walks chunk by chunk and flushes
// the LDS histogram whenever it moves to another tensor.
constexpr uint32_t kCandSpanMax = 16;

__global__ __launch_bounds__(kBlock) void topk_cand_hist(const TDesc* __restrict__ d, int T, uint32_t C,
                                                         uint32_t span, int pass, int copies, Ws ws) {
    __shared__ uint32_t lh[kBins12];
    __shared__ uint32_t pre[kCandSpanMax + 1];
    uint32_t* gh0 = ws.t_hist + (size_t)(blockIdx.x % (uint32_t)copies) * T * kBins0;  // this workgroup's copy
    const int shift = pass == 1 ? 10 : 0;
    const int match_shift = pass == 1 ? 20 : 10;
    const uint32_t c0 = blockIdx.x * span;
    const uint32_t c1 = c0 + span < C ? c0 + span : C;
    for (int b = threadIdx.x; b < kBins12; b += kBlock) lh[b] = 0;
    int t = tensor_of_chunk(d, T, c0);
    if (c1 <= d[t].chunk0 + d[t].nchunks) {
        // one tensor: candidate counts of the range, then the flattened walk
        const uint32_t nc = c1 - c0;
        const uint32_t mine = threadIdx.x < nc ? ws.t_ccount[c0 + threadIdx.x] : 0u;
        const uint32_t pfx = ws.t_prefix[t] >> match_shift;
        if (threadIdx.x < 64) {
            uint32_t inc = mine;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t y = __shfl_up(inc, o, 64);
                if ((int)threadIdx.x >= o) inc += y;
            }
            if (threadIdx.x < nc) pre[threadIdx.x + 1] = inc;
            if (threadIdx.x == 0) pre[0] = 0;
        }
        __syncthreads();
        const uint32_t M = pre[nc];
        constexpr int kU = 4;  // candidates per thread with loads in flight together
        for (uint32_t f0 = 0; f0 < M; f0 += kU * kBlock) {
            uint32_t key[kU];
#pragma unroll
            for (int q = 0; q < kU; ++q) {
                const uint32_t f = f0 + q * kBlock + threadIdx.x;
                key[q] = 0xFFFFFFFFu;
                if (f < M) {
                    uint32_t ci = 0;  // chunk of the range holding flattened entry f
#pragma unroll
                    for (uint32_t b = kCandSpanMax / 2; b >= 1; b >>= 1)
                        if (ci + b <= nc - 1 && pre[ci + b] <= f) ci += b;
                    key[q] = ws.t_cand[(size_t)(c0 + ci) * kChunk + (f - pre[ci])].y & 0x7FFFFFFFu;
                }
            }
#pragma unroll
            for (int q = 0; q < kU; ++q)
                if (key[q] != 0xFFFFFFFFu && (key[q] >> match_shift) == pfx)
                    atomicAdd(&lh[(key[q] >> shift) & (kBins12 - 1)], 1u);
        }
        __syncthreads();
        flush_hist(lh, gh0 + (size_t)t * kBins0, kBins12);
        return;
    }
    __syncthreads();
    uint32_t prefix = ws.t_prefix[t];
    uint32_t tend = d[t].chunk0 + d[t].nchunks;
    for (uint32_t c = c0; c < c1; ++c) {
        if (c >= tend) {  // next tensor: flush this one's counts
            __syncthreads();
            flush_hist(lh, gh0 + (size_t)t * kBins0, kBins12);
            __syncthreads();
            for (int b = threadIdx.x; b < kBins12; b += kBlock) lh[b] = 0;
            __syncthreads();
            t = tensor_of_chunk(d, T, c);
            prefix = ws.t_prefix[t];
            tend = d[t].chunk0 + d[t].nchunks;
        }
        const uint32_t m = ws.t_ccount[c];
        const uint2* cand = ws.t_cand + (size_t)c * kChunk;
        for (uint32_t i = threadIdx.x; i < m; i += kBlock) {
            const uint32_t key = cand[i].y & 0x7FFFFFFFu;
            if ((key >> match_shift) == (prefix >> match_shift))
                atomicAdd(&lh[(key >> shift) & (kBins12 - 1)], 1u);
        }
    }
    __syncthreads();
    flush_hist(lh, gh0 + (size_t)t * kBins0, kBins12);
}

// Per chunk: candidates above tau and equal to tau, counted with ballots;
// each wave takes kCountChunks consecutive chunks, whose loads it issues
// together (one chunk per wave for calls of few chunks, where the wave
// count matters more).
constexpr uint32_t kCountBatchFrom = 4096;  // chunks

template <uint32_t kCountChunks>
__global__ __launch_bounds__(kBlock) void topk_cand_count(const TDesc* __restrict__ d, int T, uint32_t C,
                                                          Ws ws) {
    const int lane = lane_id();
    const uint32_t c0 = (blockIdx.x * (kBlock / 64) + wave_id()) * kCountChunks;
    uint32_t m[kCountChunks], tau[kCountChunks], key[kCountChunks];
#pragma unroll
    for (uint32_t u = 0; u < kCountChunks; ++u) m[u] = c0 + u < C ? ws.t_ccount[c0 + u] : 0u;
#pragma unroll
    for (uint32_t u = 0; u < kCountChunks; ++u)
        tau[u] = c0 + u < C ? ws.t_prefix[tensor_of_chunk(d, T, c0 + u)] : 0u;
#pragma unroll
    for (uint32_t u = 0; u < kCountChunks; ++u)
        key[u] = (uint32_t)lane < m[u] ? ws.t_cand[(size_t)(c0 + u) * kChunk + lane].y & 0x7FFFFFFFu : 0u;
#pragma unroll
    for (uint32_t u = 0; u < kCountChunks; ++u) {
        const uint32_t c = c0 + u;
        if (c >= C) break;
        const bool in = (uint32_t)lane < m[u];
        uint32_t gt = (uint32_t)__popcll(__ballot(in && key[u] > tau[u]));
        uint32_t eq = (uint32_t)__popcll(__ballot(in && key[u] == tau[u]));
        const uint2* cand = ws.t_cand + (size_t)c * kChunk;
        for (uint32_t i0 = 64; i0 < m[u]; i0 += 64) {  // chunks with more than 64 candidates
            const uint32_t i = i0 + lane;
            const uint32_t k2 = i < m[u] ? cand[i].y & 0x7FFFFFFFu : 0u;
            gt += (uint32_t)__popcll(__ballot(i < m[u] && k2 > tau[u]));
            eq += (uint32_t)__popcll(__ballot(i < m[u] && k2 == tau[u]));
        }
        if (lane == 0) {
            ws.t_gt[c] = gt;
            ws.t_eq[c] = eq;
        }
    }
}

// One workgroup per tensor: place every chunk's winners.  eqb[c] = number
// of tau-equal candidates in earlier chunks; a chunk keeps its tau-equal
// candidates while the running count stays below the number needed.  Thread
// i walks a contiguous run of the tensor's chunks; two block scans over the
// runs' totals give every chunk its prefix.  Runs of up to kScanRegs chunks
// (tensors of up to 256 kScanRegs chunks) are read once into registers, all
// loads in flight together; longer runs are read three times,
// kScanBatch chunks at a time.
constexpr uint32_t kScanRegs = 32;
constexpr uint32_t kScanBatch = 8;

namespace {
// Winners of one chunk given the tau-equal candidates before it.
__device__ __forceinline__ uint64_t chunk_winners(uint32_t gt, uint32_t eq, uint64_t eq_before, uint64_t need) {
    const uint64_t left = eq_before < need ? need - eq_before : 0;
    return (uint64_t)gt + (left < eq ? left : eq);
}
}  // namespace

__global__ __launch_bounds__(kBlock) void topk_cand_scan(const TDesc* __restrict__ d, Ws ws) {
    __shared__ uint64_t sh[4];
    const int t = blockIdx.x;
    const TDesc td = d[t];
    if (td.k == 0 || td.nchunks == 0) return;
    const uint64_t need = ws.t_krem[t];
    const uint32_t per = (td.nchunks + kBlock - 1) / kBlock;
    const uint32_t lo = threadIdx.x * per;
    const uint32_t hi = lo + per < td.nchunks ? lo + per : td.nchunks;
    const uint32_t* eqp = ws.t_eq + td.chunk0;
    const uint32_t* gtp = ws.t_gt + td.chunk0;
    uint64_t tot;
    if (per <= kScanRegs) {
        uint32_t eq[kScanRegs], gt[kScanRegs];
#pragma unroll
        for (uint32_t u = 0; u < kScanRegs; ++u) {
            eq[u] = lo + u < hi ? eqp[lo + u] : 0u;
            gt[u] = lo + u < hi ? gtp[lo + u] : 0u;
        }
        uint64_t eq_run = 0;
#pragma unroll
        for (uint32_t u = 0; u < kScanRegs; ++u) eq_run += eq[u];
        const uint64_t eqb0 = block_excl_scan_u64(eq_run, sh, tot);
        uint64_t sel_run = 0, e = eqb0;
#pragma unroll
        for (uint32_t u = 0; u < kScanRegs; ++u) {
            sel_run += chunk_winners(gt[u], eq[u], e, need);
            e += eq[u];
        }
        uint64_t pos = td.off + block_excl_scan_u64(sel_run, sh, tot);
        e = eqb0;
#pragma unroll
        for (uint32_t u = 0; u < kScanRegs; ++u) {
            if (lo + u < hi) {
                const uint32_t c = td.chunk0 + lo + u;
                ws.t_off[c] = pos;
                ws.t_eqb[c] = (uint32_t)(e < 0xFFFFFFFFull ? e : 0xFFFFFFFFull);
                pos += chunk_winners(gt[u], eq[u], e, need);
                e += eq[u];
            }
        }
        return;
    }
    // tau-equal candidates before each run
    uint64_t eq_run = 0;
    for (uint32_t q0 = lo; q0 < hi; q0 += kScanBatch) {
        uint32_t eq[kScanBatch];
#pragma unroll
        for (uint32_t u = 0; u < kScanBatch; ++u) eq[u] = q0 + u < hi ? eqp[q0 + u] : 0u;
#pragma unroll
        for (uint32_t u = 0; u < kScanBatch; ++u) eq_run += eq[u];
    }
    const uint64_t eqb0 = block_excl_scan_u64(eq_run, sh, tot);
    // winners per chunk, and before each run
    uint64_t sel_run = 0;
    {
        uint64_t e = eqb0;
        for (uint32_t q0 = lo; q0 < hi; q0 += kScanBatch) {
            uint32_t eq[kScanBatch], gt[kScanBatch];
#pragma unroll
            for (uint32_t u = 0; u < kScanBatch; ++u) {
                eq[u] = q0 + u < hi ? eqp[q0 + u] : 0u;
                gt[u] = q0 + u < hi ? gtp[q0 + u] : 0u;
            }
#pragma unroll
            for (uint32_t u = 0; u < kScanBatch; ++u) {
                sel_run += chunk_winners(gt[u], eq[u], e, need);
                e += eq[u];
            }
        }
    }
    uint64_t pos = td.off + block_excl_scan_u64(sel_run, sh, tot);
    uint64_t eqb = eqb0;
    for (uint32_t q0 = lo; q0 < hi; q0 += kScanBatch) {
        uint32_t eq[kScanBatch], gt[kScanBatch];
#pragma unroll
        for (uint32_t u = 0; u < kScanBatch; ++u) {
            eq[u] = q0 + u < hi ? eqp[q0 + u] : 0u;
            gt[u] = q0 + u < hi ? gtp[q0 + u] : 0u;
        }
#pragma unroll
        for (uint32_t u = 0; u < kScanBatch; ++u) {
            if (q0 + u < hi) {
                const uint32_t c = td.chunk0 + q0 + u;
                ws.t_off[c] = pos;
                ws.t_eqb[c] = (uint32_t)(eqb < 0xFFFFFFFFull ? eqb : 0xFFFFFFFFull);
                pos += chunk_winners(gt[u], eq[u], eqb, need);
                eqb += eq[u];
            }
        }
    }
}

// Emit the winners of a chunk in index order and clear them in e_new (kDGC:
// and in u), one wave per chunk; ranks come from ballots.
template <bool kDGC>
__global__ __launch_bounds__(kBlock) void topk_emit(const TDesc* __restrict__ d, int T, uint32_t C,
                                                    uint32_t* __restrict__ idx,
                                                    float* __restrict__ val, Ws ws) {
    const int lane = lane_id();
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;  // lanes under this one
    const uint32_t c = blockIdx.x * (kBlock / 64) + wave_id();
    const uint32_t m = c < C ? ws.t_ccount[c] : 0u;
    if (m > 0) {
        const int t = tensor_of_chunk(d, T, c);
        float* resid = d[t].resid;
        const uint64_t end = d[t].off + d[t].k;
        const uint32_t tau = ws.t_prefix[t];
        const uint64_t need = ws.t_krem[t];
        const uint2* cand = ws.t_cand + (size_t)c * kChunk;
        uint64_t eq_seen = ws.t_eqb[c];
        uint64_t pos = ws.t_off[c];
        for (uint32_t i0 = 0; i0 < m; i0 += 64) {
            const uint32_t i = i0 + lane;
            uint2 e = make_uint2(0, 0);
            uint32_t key = 0;
            if (i < m) {
                e = cand[i];
                key = e.y & 0x7FFFFFFFu;
            }
            const bool is_eq = i < m && key == tau;
            const uint64_t meq = __ballot(is_eq);
            const uint64_t eq_rank = eq_seen + (uint64_t)__popcll(meq & below);
            const bool sel = i < m && (key > tau || (is_eq && eq_rank < need));
            const uint64_t msel = __ballot(sel);
            const uint64_t at = pos + (uint64_t)__popcll(msel & below);
            if (sel && at < end) {
                idx[at] = e.x;
                val[at] = u2f(e.y);
                if (resid) gp(resid)[e.x] = 0.f;
                if constexpr (kDGC) gp(vel_of(d[t]))[e.x] = 0.f;
            }
            eq_seen += (uint64_t)__popcll(meq);
            pos += (uint64_t)__popcll(msel);
        }
    }
}

// ------------------------------------------------- few-chunk exact path
// Calls of at most topk_few_chunks_limit() chunks (2048 unless set lower)
// take a path of five launches (the
// general pipeline's per-step launches cost more than the passes themselves
// at these sizes): clear, the histogram pass, then three kernels that each
// redo the previous radix step's bin search from the global histogram in
// every workgroup instead of in a launch of its own:
//   compact:  bin b of the k-th key (digit 0) -> candidates (keys at or
//             above bin b) per chunk, index order; histogram of digit 1
//             among the candidates in bin b;
//   digit 2:  digit 1 -> histogram of digit 2 among the candidates whose
//             digits 0 and 1 match;
//   emit:     digit 2 gives the k-th key tau and how many tau-equal entries
//             to keep; each wave takes one chunk, counts its candidates
//             above and equal to tau, and finds the counts of all earlier
//             chunks of its tensor by looking back over their published
//             counts (decoupled look-back, Merrill and Garland 2016): a
//             chunk's wave publishes its own counts, then its running
//             totals; a wave that finds an earlier chunk unpublished
//             counts that chunk's candidates itself, so no wave waits for
//             another and the pass needs no particular residency.
// Histogram regions: digit 0 in `copies` copies (chunk c adds to copy
// c % copies, which spreads the atomic additions to the busiest bins over
// several addresses; readers add the copies) at t_hist[(r * T + t) * 2048],
// then digit 1 at t_hist[copies * T * 2048 + t * 1024] and digit 2 at
// t_hist[copies * T * 2048 + T * 1024 + t * 1024].
// Look-back words (t_off, cleared by the histogram pass): bit 62 counts
// published, bit 63 running totals published, bits 61..31 entries above
// tau, bits 30..0 entries equal to tau (chunk counts, or totals over the
// tensor's chunks up to and including this one).
constexpr uint64_t kLbCounts = 1ull << 62, kLbTotals = 1ull << 63;
constexpr int kLbPolls = 16;  // re-reads of unpublished look-back words before counting them
constexpr int kFewCopiesMax = 4;
// digit-0 histogram copies of a few-chunk call of T tensors
inline int few_copies(int T) { return T <= 16 ? kFewCopiesMax : 1; }

namespace {

// Bin holding the target-th largest entry of a global histogram, searched
// by the whole workgroup (thread i owns the i-th run of bins from the top);
// *above receives the entries in higher bins.  Needs 1 <= target <= total.
__device__ uint32_t block_hist_select(const uint32_t* __restrict__ gh, int bins, uint32_t target, uint64_t* sh,
                                      uint32_t* res_sh, uint32_t* above, int copies = 1,
                                      size_t copy_stride = 0) {
    const int per = bins / kBlock;  // 8 or 4
    const int hi = bins - (int)threadIdx.x * per;
    uint32_t h[8];
    uint32_t mine = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) h[q] = q < per ? gh[hi - 1 - q] : 0u;
    for (int r = 1; r < copies; ++r)
#pragma unroll
        for (int q = 0; q < 8; ++q) h[q] += q < per ? gh[r * copy_stride + hi - 1 - q] : 0u;
#pragma unroll
    for (int q = 0; q < 8; ++q) mine += h[q];
    uint64_t tot;
    uint32_t a = (uint32_t)block_excl_scan_u64(mine, sh, tot);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        if (q < per && a < target && target <= a + h[q]) {
            res_sh[0] = (uint32_t)(hi - 1 - q);
            res_sh[1] = a;
        }
        a += h[q];
    }
    __syncthreads();
    const uint32_t b = res_sh[0];
    *above = res_sh[1];
    __syncthreads();
    return b;
}

// The same over 1024 bins by one wave (lane i owns the i-th run of 16
// bins from the top).
__device__ uint32_t wave_hist_select(const uint32_t* __restrict__ gh, uint32_t target, uint32_t* above) {
    const int lane = lane_id();
    const int hi = kBins12 - lane * 16;
    uint32_t h[16];
    uint32_t mine = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        h[q] = gh[hi - 1 - q];
        mine += h[q];
    }
    uint32_t inc = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
    }
    uint32_t a = inc - mine;
    int found = -1;
    uint32_t fa = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        if (found < 0 && a < target && target <= a + h[q]) {
            found = hi - 1 - q;
            fa = a;
        }
        a += h[q];
    }
    const uint64_t m = __ballot(found >= 0);
    const int src = m ? (int)__builtin_ctzll(m) : 0;
    *above = (uint32_t)__shfl(fa, src, 64);
    return (uint32_t)__shfl(found, src, 64);
}

__device__ __forceinline__ uint64_t lb_load(const uint64_t* p) {
    return __hip_atomic_load((unsigned long long*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void lb_store(uint64_t* p, uint64_t v) {
    __hip_atomic_store((unsigned long long*)p, (unsigned long long)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t lb_word(uint64_t flag, uint32_t gt, uint32_t eq) {
    return flag | (uint64_t)gt << 31 | (uint64_t)eq;
}

// Candidates of chunk c above and equal to tau, counted by one wave.
__device__ __forceinline__ void wave_count_chunk(const Ws& ws, uint32_t c, uint32_t tau, uint32_t& gt,
                                                 uint32_t& eq) {
    const int lane = lane_id();
    const uint32_t m = ws.t_ccount[c];
    const uint2* cand = ws.t_cand + (size_t)c * kChunk;
    gt = 0;
    eq = 0;
    for (uint32_t i0 = 0; i0 < m; i0 += 64) {
        const uint32_t i = i0 + (uint32_t)lane;
        const uint32_t key = i < m ? cand[i].y & 0x7FFFFFFFu : 0u;
        gt += (uint32_t)__popcll(__ballot(i < m && key > tau));
        eq += (uint32_t)__popcll(__ballot(i < m && key == tau));
    }
}

}  // namespace

// Digit 0 from the histogram pass's counts, then candidate compaction
// (v re-read from the stored e_new, or from g without error feedback) and
// the digit-1 histogram of the candidates in bin b.
__global__ __launch_bounds__(kBlock) void topk_fast_compact(const TDesc* __restrict__ d, int T, uint32_t C,
                                                            int copies, Ws ws) {
    __shared__ uint32_t lh[kBins12];
    __shared__ uint64_t sh[4];
    __shared__ uint32_t res_sh[2];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    float v[kEpt];
    uint32_t valid;
    load_stored_v(td, j, v, valid);  // in flight during the bin search
    for (int b = threadIdx.x; b < kBins12; b += kBlock) lh[b] = 0;
    uint32_t above;
    const uint32_t b0 = block_hist_select(ws.t_hist + (size_t)t * kBins0, kBins0, td.k, sh, res_sh, &above, copies,
                                          (size_t)T * kBins0);
    if (j == 0 && threadIdx.x == 0) {
        ws.t_thr[t] = b0 << 20;
        ws.t_fb[t] = td.k - above;  // entries still to select inside bin b
    }
    const uint32_t thr = b0 << 20;
    uint32_t pm = 0;
#pragma unroll
    for (int i = 0; i < kEpt; ++i)
        if (((valid >> i) & 1u) && key_of(v[i]) >= thr) pm |= 1u << i;
    uint64_t packed = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) packed |= (uint64_t)__popc((pm >> (4 * r)) & 0xFu) << (16 * r);
    uint64_t tot;
    const uint64_t pre = block_excl_scan_u64(packed, sh, tot);
    uint2* out = ws.t_cand + (size_t)c * kChunk;
    uint32_t base = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        uint32_t rank = base + (uint32_t)((pre >> (16 * r)) & 0xFFFFu);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = 4 * r + q;
            if ((pm >> i) & 1u) {
                const uint32_t e = j * (uint32_t)kChunk + 1024u * r + 4u * threadIdx.x + q;
                const uint32_t key = key_of(v[i]);
                out[rank++] = make_uint2(e, f2u(v[i]));
                if ((key >> 20) == b0) atomicAdd(&lh[(key >> 10) & (kBins12 - 1)], 1u);
            }
        }
        base += (uint32_t)((tot >> (16 * r)) & 0xFFFFu);
    }
    if (threadIdx.x == 0) ws.t_ccount[c] = base;
    __syncthreads();
    flush_hist(lh, ws.t_hist + (size_t)copies * T * kBins0 + (size_t)t * kBins12, kBins12);
}

// Digit 1, then the digit-2 histogram of the candidates whose digits 0 and
// 1 match.
__global__ __launch_bounds__(kBlock) void topk_fast_digit2(const TDesc* __restrict__ d, int T, int copies, Ws ws) {
    __shared__ uint32_t lh[kBins12];
    __shared__ uint64_t sh[4];
    __shared__ uint32_t res_sh[2];
    const uint32_t c = blockIdx.x;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    const uint32_t j = c - td.chunk0;
    uint32_t* h1 = ws.t_hist + (size_t)copies * T * kBins0;
    // the chunk's count and first candidates, in flight during the bin search
    // (a slot holds kChunk entries, so the first kBlock are always in bounds)
    const uint32_t m = ws.t_ccount[c];
    const uint2* cand = ws.t_cand + (size_t)c * kChunk;
    const uint32_t key0 = cand[threadIdx.x].y & 0x7FFFFFFFu;
    for (int b = threadIdx.x; b < kBins12; b += kBlock) lh[b] = 0;
    const uint32_t thr = ws.t_thr[t], r0 = ws.t_fb[t];
    uint32_t above;
    const uint32_t d1 = block_hist_select(h1 + (size_t)t * kBins12, kBins12, r0, sh, res_sh, &above);
    const uint32_t prefix = thr | d1 << 10;
    if (j == 0 && threadIdx.x == 0) {
        ws.t_prefix[t] = prefix;
        ws.t_krem[t] = r0 - above;
    }
    if (threadIdx.x < m && (key0 >> 10) == (prefix >> 10)) atomicAdd(&lh[key0 & (kBins12 - 1)], 1u);
    for (uint32_t i = threadIdx.x + kBlock; i < m; i += kBlock) {
        const uint32_t key = cand[i].y & 0x7FFFFFFFu;
        if ((key >> 10) == (prefix >> 10)) atomicAdd(&lh[key & (kBins12 - 1)], 1u);
    }
    __syncthreads();
    flush_hist(lh, h1 + (size_t)T * kBins12 + (size_t)t * kBins12, kBins12);
}

// Digit 2 gives tau; one wave per chunk counts, looks back, and emits its
// winners in index order (clearing them in e_new; kDGC: and in u).
template <bool kDGC>
__global__ __launch_bounds__(kBlock) void topk_fast_emit(const TDesc* __restrict__ d, int T, uint32_t C, int copies,
                                                         uint32_t* __restrict__ idx, float* __restrict__ val,
                                                         Ws ws) {
    const int lane = lane_id();
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    const uint32_t c = blockIdx.x * (kBlock / 64) + wave_id();
    if (c >= C) return;
    const int t = tensor_of_chunk(d, T, c);
    const TDesc td = d[t];
    // the chunk's count and first 64 candidates, in flight during the bin
    // search (always inside the chunk's slot)
    const uint32_t m = ws.t_ccount[c];
    const uint2* cand = ws.t_cand + (size_t)c * kChunk;
    const uint2 first = cand[lane];
    const uint32_t prefix = ws.t_prefix[t], r1 = ws.t_krem[t];
    uint32_t above;
    const uint32_t d2 =
        wave_hist_select(ws.t_hist + (size_t)copies * T * kBins0 + (size_t)(T + t) * kBins12, r1, &above);
    const uint32_t tau = prefix | d2;
    const uint32_t need = r1 - above;  // tau-equal entries to keep, lowest indices first
    uint32_t gt, eq;
    {
        const uint32_t key = (uint32_t)lane < m ? first.y & 0x7FFFFFFFu : 0u;
        gt = (uint32_t)__popcll(__ballot((uint32_t)lane < m && key > tau));
        eq = (uint32_t)__popcll(__ballot((uint32_t)lane < m && key == tau));
        for (uint32_t i0 = 64; i0 < m; i0 += 64) {
            const uint32_t i = i0 + (uint32_t)lane;
            const uint32_t k2 = i < m ? cand[i].y & 0x7FFFFFFFu : 0u;
            gt += (uint32_t)__popcll(__ballot(i < m && k2 > tau));
            eq += (uint32_t)__popcll(__ballot(i < m && k2 == tau));
        }
    }
    uint64_t* lb = ws.t_off;
    if (lane == 0) lb_store(lb + c, lb_word(kLbCounts, gt, eq));
    // totals of the earlier chunks of the tensor
    uint32_t gt_b = 0, eq_b = 0;
    for (int64_t q0 = (int64_t)c - 1; q0 >= (int64_t)td.chunk0; q0 -= 64) {
        const int64_t q = q0 - lane;
        const bool in = q >= (int64_t)td.chunk0;
        uint64_t w = in ? lb_load(lb + q) : 0ull;
        uint64_t tot_m;
        int lim;
        // chunks whose waves run alongside this one publish within a few
        // load latencies: poll those still unpublished a bounded number of
        // times before counting them here
        for (int spin = 0;; ++spin) {
            tot_m = __ballot(in && (w & kLbTotals));
            lim = tot_m ? (int)__builtin_ctzll(tot_m) : 63;  // up to the nearest chunk with totals
            const bool pend = in && lane <= lim && w == 0ull;
            if (!__ballot(pend) || spin == kLbPolls) break;
            __builtin_amdgcn_s_sleep(4);
            if (pend) w = lb_load(lb + q);
        }
        const bool use = in && lane <= lim;
        // unpublished chunks: count them here, one at a time with the whole wave
        uint64_t help = __ballot(use && w == 0ull);
        while (help) {
            const int l = (int)__builtin_ctzll(help);
            help &= help - 1;
            uint32_t hg, he;
            wave_count_chunk(ws, (uint32_t)(q0 - l), tau, hg, he);
            if (lane == l) w = lb_word(kLbCounts, hg, he);
        }
        uint32_t g = use ? (uint32_t)(w >> 31) & 0x7FFFFFFFu : 0u;
        uint32_t e = use ? (uint32_t)w & 0x7FFFFFFFu : 0u;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            g += __shfl_xor(g, o, 64);
            e += __shfl_xor(e, o, 64);
        }
        gt_b += g;
        eq_b += e;
        if (tot_m) break;
    }
    if (lane == 0) lb_store(lb + c, lb_word(kLbCounts | kLbTotals, gt_b + gt, eq_b + eq));
    // emit
    if (m == 0) return;
    float* resid = td.resid;
    const uint64_t end = td.off + td.k;
    uint64_t eq_seen = eq_b;
    uint64_t pos = td.off + gt_b + (eq_b < need ? eq_b : need);
    for (uint32_t i0 = 0; i0 < m; i0 += 64) {
        const uint32_t i = i0 + lane;
        uint2 e = make_uint2(0, 0);
        uint32_t key = 0;
        if (i < m) {
            e = i0 == 0 ? first : cand[i];
            key = e.y & 0x7FFFFFFFu;
        }
        const bool is_eq = i < m && key == tau;
        const uint64_t meq = __ballot(is_eq);
        const uint64_t eq_rank = eq_seen + (uint64_t)__popcll(meq & below);
        const bool sel = i < m && (key > tau || (is_eq && eq_rank < need));
        const uint64_t msel = __ballot(sel);
        const uint64_t at = pos + (uint64_t)__popcll(msel & below);
        if (sel && at < end) {
            idx[at] = e.x;
            val[at] = u2f(e.y);
            if (resid) gp(resid)[e.x] = 0.f;
            if constexpr (kDGC) gp(vel_of(td))[e.x] = 0.f;
        }
        eq_seen += (uint64_t)__popcll(meq);
        pos += (uint64_t)__popcll(msel);
    }
}

// Clear the tensors' histograms (T * 2048 words, a multiple of 4) and the
// fallback flag at the start of a call.
__global__ void topk_zero_hist(uint32_t* h, uint64_t n, uint32_t* any) {
    const uint64_t n4 = n / 4;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (uint64_t)gridDim.x * blockDim.x)
        reinterpret_cast<u32x4*>(h)[i] = u32x4{0u, 0u, 0u, 0u};
    if (blockIdx.x == 0 && threadIdx.x == 0) any[0] = 0u;
}

namespace {

template <bool kDGC>
hipError_t launch_topk_t(int kind, double ratio, uint64_t seed, const TDesc* d, int T, uint32_t C,
                         uint32_t* idx, float* val, const Ws& ws, hipStream_t s, const DgcFuse& f) {
    const dim3 blk(kBlock);
    const DgcFuse none{nullptr, 0.f, nullptr};
    if (C <= topk_few_chunks_limit()) {  // few chunks: the five-launch exact path (both kinds: same result)
        const int copies = few_copies(T);
        const uint64_t hn = (uint64_t)T * ((uint64_t)copies * kBins0 + 2 * kBins12);
        uint32_t zb = (uint32_t)((hn / 4 + 255) / 256);
        if (zb > 4096) zb = 4096;
        hipLaunchKernelGGL(topk_zero_hist, dim3(zb), dim3(256), 0, s, ws.t_hist, hn, ws.t_any);
        (void)launch_timed(kTimedTopkHist, topk_hist_pass<kDGC>, dim3(C), blk, 0, s, d, T, C, 1, 0, ws, ws.t_off,
                           copies, f);
        hipLaunchKernelGGL(topk_fast_compact, dim3(C), blk, 0, s, d, T, C, copies, ws);
        hipLaunchKernelGGL(topk_fast_digit2, dim3(C), blk, 0, s, d, T, copies, ws);
        hipLaunchKernelGGL(topk_fast_emit<kDGC>, dim3((C + kBlock / 64 - 1) / (kBlock / 64)), blk, 0, s, d, T, C,
                           copies, idx, val, ws);
        return hipGetLastError();
    }
    const int R = topk_general_copies(T);
    const uint64_t hn = (uint64_t)T * R * kBins0;
    uint32_t zb = (uint32_t)((hn / 4 + 255) / 256);
    if (zb > 4096) zb = 4096;
    hipLaunchKernelGGL(topk_zero_hist, dim3(zb), dim3(256), 0, s, ws.t_hist, hn, ws.t_any);
    if (kind == 0) {  // exact
        hipLaunchKernelGGL(topk_hist_pass<kDGC>, dim3(C), blk, 0, s, d, T, C, 1, 0, ws, (uint64_t*)nullptr, R, f);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindThrExact, 0, R, ws);
        (void)launch_timed(kTimedTopkCompact, topk_compact<false, false>, dim3(C), blk, 0, s, d, T, C, 0, 0, R, ws,
                           none);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindDigit0, 0, R, ws);
    } else {  // sampled threshold, exact fallback per tensor
        hipLaunchKernelGGL(topk_sample_hist<kDGC>, dim3((C + kSampleChunksPerBlock - 1) / kSampleChunksPerBlock),
                           blk, 0, s, d, T, C, seed, R, ws, f);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindThrSample, 0, R, ws);
        if (C > kNtChunks)
            (void)launch_timed(kTimedTopkCompact, topk_compact<true, kDGC>, dim3(C), blk, 0, s, d, T, C, 1, 0, R, ws,
                               f);
        else
            (void)launch_timed(kTimedTopkCompact, topk_compact<false, kDGC>, dim3(C), blk, 0, s, d, T, C, 1, 0, R,
                               ws, f);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindDigit0, 0, R, ws);
        // fallback passes: small grids that walk the chunks, and return at
        // once when no tensor fell back (the usual case); they re-read the
        // stored v, so a DGC step needs nothing more here
        const dim3 fb_grid(C < 1024u ? C : 1024u);
        hipLaunchKernelGGL(topk_hist_pass<false>, fb_grid, blk, 0, s, d, T, C, 0, 1, ws, (uint64_t*)nullptr, R, none);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindThrExact, 1, R, ws);
        hipLaunchKernelGGL((topk_compact<false, false>), fb_grid, blk, 0, s, d, T, C, 0, 1, R, ws, none);
        hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindDigit0, 1, R, ws);
    }
    uint32_t span = C / 1024u;
    span = span < 1u ? 1u : (span > kCandSpanMax ? kCandSpanMax : span);
    const dim3 hist_grid((C + span - 1) / span);
    hipLaunchKernelGGL(topk_cand_hist, hist_grid, blk, 0, s, d, T, C, span, 1, R, ws);
    hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindDigit1, 0, R, ws);
    hipLaunchKernelGGL(topk_cand_hist, hist_grid, blk, 0, s, d, T, C, span, 2, R, ws);
    hipLaunchKernelGGL(topk_find, dim3(T), blk, 0, s, d, T, ratio, (int)kFindDigit2, 0, R, ws);
    if (C >= kCountBatchFrom)
        hipLaunchKernelGGL(topk_cand_count<4>, dim3((C + 15) / 16), blk, 0, s, d, T, C, ws);
    else
        hipLaunchKernelGGL(topk_cand_count<1>, dim3((C + 3) / 4), blk, 0, s, d, T, C, ws);
    hipLaunchKernelGGL(topk_cand_scan, dim3(T), blk, 0, s, d, ws);
    hipLaunchKernelGGL(topk_emit<kDGC>, dim3((C + kBlock / 64 - 1) / (kBlock / 64)), blk, 0, s, d, T, C, idx, val,
                       ws);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_topk(int kind, double ratio, uint64_t seed, const TDesc* d, int T, uint32_t C,
                       bool, bool, uint32_t* idx, float* val, const Ws& ws, hipStream_t s, const DgcFuse* dgc) {
    if (C == 0) return hipSuccess;
    if (dgc) return launch_topk_t<true>(kind, ratio, seed, d, T, C, idx, val, ws, s, *dgc);
    return launch_topk_t<false>(kind, ratio, seed, d, T, C, idx, val, ws, s, DgcFuse{nullptr, 0.f, nullptr});
}

}  // namespace bc
