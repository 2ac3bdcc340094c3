// kernels_randk.hip -- seeded random-k sparsification with error feedback
// on gfx950 (Randomk at a 1% rate, paper Sec. 5.1; sparsification with
// error feedback, Sec. 2.3).
//
// The k_t indices of tensor t are the images of 0..k_t-1 under the keyed
// pseudorandom permutation of [0, n_t) in randk_perm.hpp (a four-round
// Feistel network with cycle-walking, keyed by (seed, tensor id)).
//
// Instead of sorting the k indices, they are bucketed by runs of 2^S
// consecutive 4096-element chunks (S from the call's chunk count): each
// generating workgroup histograms its indices in LDS and writes one row of
// per-bucket counts, a column pass and a scan give every workgroup its
// position in every bucket, and a second pass places the indices there, so
// no global atomics are used.  The generated indices wait in the payload's
// index buffer (which the streaming pass overwrites in full) and are placed
// into r_tmp.  The streaming pass then takes a run of 2^SP chunks of one
// bucket per workgroup (SP <= S; several workgroups per bucket when the
// indices are sparse enough that each rescanning the bucket's list is
// cheap): it marks the run's indices in an LDS bitmap, and for each chunk
// zeroes them in e_new and emits (index, v) in index order, which is the
// sorted payload.
#include "launch.hpp"
#include "randk_perm.hpp"

#include <mutex>

namespace bc {

namespace {

constexpr int kScanBlock = kBlock * 16;  // bucket sizes per scan block
constexpr int kColBlock = 1024;          // threads of the column pass

// Tensor owning flat payload entry j: largest t with off[t] <= j.

}  // namespace

// Per-call preparation: derive the round keys.
__global__ void randk_prep(const TDesc* __restrict__ d, int T, uint64_t seed, Ws ws) {
    const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (t >= T) return;
    const uint4 rk = randk_round_keys(seed, d[t].tid);
    ws.r_keys[4 * t] = rk.x;
    ws.r_keys[4 * t + 1] = rk.y;
    ws.r_keys[4 * t + 2] = rk.z;
    ws.r_keys[4 * t + 3] = rk.w;
}


// A thread's view of the tensor that owns its current entry: what index
// generation and bucketing need, refreshed only when an entry crosses into
// a later tensor (entries are visited in increasing order).
struct EntryTensor {
    int t;
    uint64_t off, next_off;  // first entry of this tensor and of the next
    uint32_t n, chunk0, h, mask;
    uint4 rk;
};

__device__ __forceinline__ void entry_tensor_load(const TDesc* __restrict__ d, int T, const uint32_t* keys,
                                                  int t, EntryTensor& et) {
    const TDesc td = d[t];
    et.t = t;
    et.off = td.off;
    et.next_off = t + 1 < T ? d[t + 1].off : ~0ull;
    et.n = td.n;
    et.chunk0 = td.chunk0;
    et.h = half_bits(td.n);
    et.mask = et.h >= 32 ? 0xFFFFFFFFu : ((1u << et.h) - 1u);
    et.rk = *reinterpret_cast<const uint4*>(keys + 4 * t);
}

__device__ __forceinline__ void entry_tensor_advance(const TDesc* __restrict__ d, int T, const uint32_t* keys,
                                                     uint64_t j, EntryTensor& et) {
    if (j < et.next_off) return;
    int t = et.t;
    while (t + 1 < T && d[t + 1].off <= j) ++t;
    entry_tensor_load(d, T, keys, t, et);
}

// Generate the indices of kGenEntries consecutive payload entries, keep
// them in gen (the payload's index buffer), and write this workgroup's row
// of bucket counts.  A thread
// takes its entries in turn, but the cycle walks are not aligned across the
// wave: every pass of the loop applies one Feistel evaluation per thread,
// and a thread whose walk has landed in [0, n) records its index and starts
// its next entry in the same pass.  A wave then costs about the largest
// per-thread total of evaluations rather than the sum over entries of the
// largest walk in the wave (walks take 1 to 4 evaluations on average and
// have long tails).
__global__ __launch_bounds__(kGenBlock) void randk_count(const TDesc* __restrict__ d, int T, uint64_t sum_k,
                                                         uint32_t S, uint32_t NB, uint32_t* __restrict__ gen,
                                                         Ws ws) {
    extern __shared__ uint32_t hist[];  // [NB]
    for (uint32_t b = threadIdx.x; b < NB; b += kGenBlock) hist[b] = 0;
    __syncthreads();
    const uint64_t j0 = (uint64_t)blockIdx.x * kGenEntries + threadIdx.x;
    EntryTensor et;
    uint64_t j = j0;
    int q = 0;
    bool live = j0 < sum_k;
    uint32_t cur = 0;  // the value the next evaluation permutes
    if (live) {
        entry_tensor_load(d, T, ws.r_keys, tensor_of_entry(d, T, j0), et);
        cur = (uint32_t)(j - et.off);
    }
    while (__any(live)) {
        if (live) {
            const uint32_t x = feistel(cur, et.h, et.mask, et.rk);
            if (x < et.n) {
                gen[j] = x;
                atomicAdd(&hist[(et.chunk0 + x / (uint32_t)kChunk) >> S], 1u);
                ++q;
                j += (uint64_t)kGenBlock;
                live = q < kGenPerThread && j < sum_k;
                if (live) {
                    entry_tensor_advance(d, T, ws.r_keys, j, et);
                    cur = (uint32_t)(j - et.off);
                }
            } else {
                cur = x;
            }
        }
    }
    __syncthreads();
    uint32_t* row = ws.r_hist + (size_t)blockIdx.x * NB;
    for (uint32_t b = threadIdx.x; b < NB; b += kGenBlock) row[b] = hist[b];
}

// Per-workgroup counts to positions within each bucket: a workgroup of 16
// waves takes 64 buckets (one per lane); wave w sums its share of the
// generating workgroups' rows, the shares are combined in LDS, and each
// wave then writes the exclusive prefix down its rows.  The bucket's size
// goes to r_ccount.
__global__ __launch_bounds__(kColBlock) void randk_columns(uint32_t NB, uint32_t nblk, Ws ws) {
    __shared__ uint32_t part[kColBlock / 64][64];
    const int lane = lane_id();
    const int w = threadIdx.x >> 6;
    const uint32_t bk = blockIdx.x * 64u + (uint32_t)lane;
    const uint32_t per = (nblk + kColBlock / 64 - 1) / (kColBlock / 64);
    const uint32_t g0 = (uint32_t)w * per;
    const uint32_t g1 = g0 + per < nblk ? g0 + per : nblk;
    const bool live = bk < NB;
    uint32_t sum = 0;
    for (uint32_t g = g0; g < g1; ++g) sum += live ? ws.r_hist[(size_t)g * NB + bk] : 0u;
    part[w][lane] = sum;
    __syncthreads();
    uint32_t acc = 0, total = 0;
    for (int q = 0; q < kColBlock / 64; ++q) {
        acc += q < w ? part[q][lane] : 0u;
        total += part[q][lane];
    }
    if (!live) return;
    for (uint32_t g = g0; g < g1; ++g) {
        uint32_t* p = ws.r_hist + (size_t)g * NB + bk;
        const uint32_t c = *p;
        *p = acc;
        acc += c;
    }
    if (w == 0) ws.r_ccount[bk] = total;
}

// Scan, step 1: sum of each block of 4096 bucket sizes.
__global__ __launch_bounds__(kBlock) void randk_scan_sums(uint32_t NB, Ws ws, uint64_t* bsum) {
    __shared__ uint64_t sh[4];
    const uint32_t b0 = blockIdx.x * (uint32_t)kScanBlock;
    uint64_t x = 0;
    for (int q = 0; q < 16; ++q) {
        const uint32_t c = b0 + q * kBlock + threadIdx.x;
        if (c < NB) x += ws.r_ccount[c];
    }
    uint64_t tot;
    block_excl_scan_u64(x, sh, tot);
    if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// Scan, step 2: payload position of each bucket's first entry.
__global__ __launch_bounds__(kBlock) void randk_scan_apply(uint32_t NB, Ws ws, const uint64_t* bsum) {
    __shared__ uint64_t sh[4];
    uint64_t pre = 0;
    for (uint32_t b = threadIdx.x; b < blockIdx.x; b += kBlock) pre += bsum[b];
    uint64_t base;
    block_excl_scan_u64(pre, sh, base);
    // thread i owns 16 consecutive bucket sizes
    const uint32_t c0 = blockIdx.x * (uint32_t)kScanBlock + threadIdx.x * 16u;
    uint32_t cnt[16];
    uint64_t mine = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        cnt[q] = (c0 + q < NB) ? ws.r_ccount[c0 + q] : 0u;
        mine += cnt[q];
    }
    uint64_t tot;
    uint64_t run = base + block_excl_scan_u64(mine, sh, tot);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        if (c0 + q < NB) ws.r_coff[c0 + q] = run;
        run += cnt[q];
    }
    if (c0 < NB && c0 + 16 >= NB) ws.r_coff[NB] = run;  // the thread holding the last size
}

// Place each generated index (gen, in generation order) in its bucket's
// range of r_tmp: the workgroup's position in the bucket (payload start +
// column prefix) plus a rank taken in LDS.  The value stored is the index's
// position within the bucket's 2^S chunks.
__global__ __launch_bounds__(kGenBlock) void randk_place(const TDesc* __restrict__ d, int T, uint64_t sum_k,
                                                         uint32_t S, uint32_t NB,
                                                         const uint32_t* __restrict__ gen, Ws ws) {
    extern __shared__ uint32_t lds[];
    uint32_t* base = lds;       // [NB] this workgroup's first position in each bucket
    uint32_t* rank = lds + NB;  // [NB] entries placed so far
    const uint32_t* row = ws.r_hist + (size_t)blockIdx.x * NB;
    for (uint32_t b = threadIdx.x; b < NB; b += kGenBlock) {
        base[b] = (uint32_t)ws.r_coff[b] + row[b];
        rank[b] = 0;
    }
    __syncthreads();
    const uint64_t j0 = (uint64_t)blockIdx.x * kGenEntries + threadIdx.x;
    EntryTensor et;
    if (j0 < sum_k) entry_tensor_load(d, T, ws.r_keys, tensor_of_entry(d, T, j0), et);
    for (int q = 0; q < kGenPerThread; ++q) {
        const uint64_t j = j0 + (uint64_t)q * kGenBlock;
        if (j >= sum_k) break;
        entry_tensor_advance(d, T, ws.r_keys, j, et);
        const uint32_t x = gen[j];
        const uint32_t gc = et.chunk0 + x / (uint32_t)kChunk;
        const uint32_t b = gc >> S;
        const uint32_t pos = base[b] + atomicAdd(&rank[b], 1u);
        ws.r_tmp[pos] = ((gc - (b << S)) << 12) | (x & (uint32_t)(kChunk - 1));
    }
}

// A run of 2^SP chunks of one bucket per workgroup (the whole bucket when
// SP = S).  The run's indices, read from the bucket's list, are marked in
// an LDS bitmap, and the list's indices below the run are counted; these
// and the per-chunk counts of the bitmap with their prefix give each
// chunk's payload position.  Then every wave streams whole chunks (or, in
// runs of at most 2 chunks, half chunks) on its own (no workgroup
// barrier): lane l holds elements 256 r + 4 l + i (r < 16, i < 4) of the
// chunk, writes e_new (selected entries zeroed) and emits its selected
// (index, v) pairs at positions from a wave prefix over the rounds, which
// is ascending index order.
namespace {
// v = widen(g) + e (or widen(g)) for the 32 elements a lane owns of the
// 2048 elements from `lo` (all inside the tensor): element 256 r + 4 lane + i
// at v[4 r + i].
template <int DT, bool kNT>
__device__ __forceinline__ void half_loads(const TDesc& td, uint32_t lo, int lane, bool use_e, float (&v)[32]) {
    const uint32_t e0 = lo + 4u * (uint32_t)lane;
    f32x4 gf[8];
    u32x2 gh[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        if constexpr (DT == 0) gf[r] = ldg4f_s<kNT>((const float*)td.grad + e0 + 256u * r);
        else gh[r] = ldg2u_s<kNT>((const uint16_t*)td.grad + e0 + 256u * r);
    }
    if (use_e) {
        f32x4 ev[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) ev[r] = ldg4f_s<kNT>(td.resid + e0 + 256u * r);
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[4 * r + i] = g_elem<DT>(gf[r], gh[r], i) + ev[r][i];
    } else {
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[4 * r + i] = g_elem<DT>(gf[r], gh[r], i);
    }
}

// The DGC velocity step over the same 32 elements: td holds u (as the fp32
// gradient) and e, tg the step's gradient; u receives fl32(fl32(m * u) +
// fl32(c * g)) and v fl32(u + e).  `whole`: all 2048 elements inside the
// tensor; else each element is checked, and those past the end read +0.0
// and are left out of `valid`.
template <int DT, bool kNT>
__device__ __forceinline__ void half_loads_dgc(const TDesc& td, const TDesc& tg, uint32_t lo, int lane, bool whole,
                                               const DgcFuse& f, float (&v)[32], float (&u)[32], uint32_t& valid) {
    const uint32_t e0 = lo + 4u * (uint32_t)lane;
    const bool clip = f.clip != nullptr;
    const float cf = clip ? *f.clip : 1.f;
    auto step = [&](float g, float uo, float e, float& un, float& vn) {
        if (clip) g = cf * g;
        const float mu = f.m * uo;
        un = mu + g;
        vn = un + e;
    };
    if (whole) {
        f32x4 gf[8], uf[8], ef[8];
        u32x2 gh[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            if constexpr (DT == 0) gf[r] = ldg4f_s<kNT>((const float*)tg.grad + e0 + 256u * r);
            else gh[r] = ldg2u_s<kNT>((const uint16_t*)tg.grad + e0 + 256u * r);
            uf[r] = ldg4f_s<kNT>((const float*)td.grad + e0 + 256u * r);
            ef[r] = ldg4f_s<kNT>(td.resid + e0 + 256u * r);
        }
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
            for (int i = 0; i < 4; ++i) step(g_elem<DT>(gf[r], gh[r], i), uf[r][i], ef[r][i], u[4 * r + i], v[4 * r + i]);
        valid = 0xFFFFFFFFu;
        return;
    }
    valid = 0;
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t x = e0 + 256u * r + i;
            const bool ok = x < td.n;
            float gx = 0.f, ux = 0.f, ex = 0.f;
            if (ok) {
                gx = DT == 0 ? gp((const float*)tg.grad)[x] : h2f(gp((const uint16_t*)tg.grad)[x]);
                ux = gp((const float*)td.grad)[x];
                ex = gp(td.resid)[x];
            }
            step(gx, ux, ex, u[4 * r + i], v[4 * r + i]);
            valid |= (ok ? 1u : 0u) << (4 * r + i);
        }
}
}  // namespace

// kHalves (runs of at most 2 chunks, not with kDGC): each wave takes half a
// chunk, so that all four waves have work; else each wave takes whole
// chunks.  kDGC: a DGC
// step (d holds u in the gradient's place, f.dg the gradients) whose
// velocity update runs here and whose masking is the zeroing of the
// selected entries of u, written back with e_new.
template <bool kNT, bool kHalves, bool kDGC>
__global__ __launch_bounds__(kBlock) void randk_stream(const TDesc* __restrict__ d, int T, uint32_t C,
                                                       uint32_t S, uint32_t SP, uint32_t NB,
                                                       uint32_t* __restrict__ idx, float* __restrict__ val,
                                                       Ws ws, DgcFuse f) {
    extern __shared__ uint32_t bm[];  // [2^SP * 128] bits of the run's chunks
    __shared__ uint32_t coff[(1u << kRandkMaxShift) + 1];
    __shared__ uint32_t below_sh;
    const int lane = lane_id();
    const int wave = wave_id();
    // the F runs of a bucket take workgroup ids congruent modulo 8 (one XCD,
    // whose L2 then serves the bucket's list to all of them) and are
    // dispatched within 8F ids of each other
    const uint32_t F = 1u << (S - SP);
    const uint32_t b = blockIdx.x / (8u * F) * 8u + blockIdx.x % 8u;
    const uint32_t run = blockIdx.x / 8u % F;
    if (b >= NB) return;
    const uint32_t cb = b << S;
    const uint32_t ncb = (C - cb < (1u << S)) ? C - cb : (1u << S);
    const uint32_t s0 = run << SP;  // the run's first chunk within the bucket
    if (s0 >= ncb) return;
    const uint32_t nc = (ncb - s0 < (1u << SP)) ? ncb - s0 : (1u << SP);
    const uint32_t c0 = cb + s0;
    const uint32_t ylo = s0 << 12, yhi = (s0 + nc) << 12;
    const uint64_t beg = ws.r_coff[b], end = ws.r_coff[b + 1];
    for (uint32_t i = threadIdx.x; i < nc * (uint32_t)kChunkWords; i += kBlock) bm[i] = 0u;
    if (threadIdx.x == 0) below_sh = 0u;
    __syncthreads();
    uint32_t below = 0;
    for (uint64_t i = beg + threadIdx.x; i < end; i += kBlock) {
        const uint32_t y = ws.r_tmp[i];
        if (y < ylo) ++below;
        else if (y < yhi) atomicOr(&bm[(y - ylo) >> 5], 1u << (y & 31));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) below += __shfl_xor(below, o, 64);
    if (lane == 0 && below) atomicAdd(&below_sh, below);
    __syncthreads();
    // selected entries per chunk (one wave per chunk), then their prefix
    for (uint32_t q = (uint32_t)wave; q < nc; q += kBlock / 64) {
        uint32_t c = __popc(bm[q * (uint32_t)kChunkWords + lane]) + __popc(bm[q * (uint32_t)kChunkWords + 64 + lane]);
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
        if (lane == 0) coff[q] = c;
    }
    __syncthreads();
    if (wave == 0) {
        // exclusive prefix of nc <= 256 counts: four per lane
        uint32_t x[4], mine = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t q = 4u * lane + i;
            x[i] = q < nc ? coff[q] : 0u;
            mine += x[i];
        }
        uint32_t inc = mine;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = __shfl_up(inc, o, 64);
            if (lane >= o) inc += y;
        }
        uint32_t at = inc - mine;
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t q = 4u * lane + i;
            if (q <= nc) coff[q] = at;
            at += x[i];
        }
    }
    __syncthreads();
    const uint32_t units = kHalves ? 2 * nc : nc;
    for (uint32_t unit = (uint32_t)wave; unit < units; unit += kBlock / 64) {
        const uint32_t q = kHalves ? unit >> 1 : unit;
        const int tq = tensor_of_chunk(d, T, c0 + q);
        const TDesc td = d[tq];
        const uint32_t j = c0 + q - td.chunk0;
        const bool use_e = td.resid != nullptr;
        uint64_t base = beg + below_sh + coff[q];
        if (kHalves && (unit & 1u)) {  // the second half: after the first half's entries
            uint32_t n0 = __popc(bm[q * (uint32_t)kChunkWords + lane]);
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) n0 += __shfl_xor(n0, o, 64);
            base += n0;
        }
        // the chunk in two halves of 2048 elements, emitted in order (kHalves:
        // this unit's half only)
        for (uint32_t h = 0; h < (kHalves ? 1u : 2u); ++h) {
            const uint32_t half = kHalves ? (unit & 1u) : h;
            const uint32_t lo = j * (uint32_t)kChunk + 2048u * half;
            float v[32];
            float un[kDGC ? 32 : 1];  // kDGC: the velocity after the step
            uint32_t valid = 0;
            const bool whole = (uint64_t)lo + 2048u <= td.n;
            if constexpr (kDGC) {
                const TDesc tg = f.dg[tq];
                if (tg.dtype == 0) half_loads_dgc<0, kNT>(td, tg, lo, lane, whole, f, v, un, valid);
                else half_loads_dgc<1, kNT>(td, tg, lo, lane, whole, f, v, un, valid);
            } else if (whole) {
                // straight-line: every load of the half is issued before any is used
                if (td.dtype == 0) half_loads<0, kNT>(td, lo, lane, use_e, v);
                else half_loads<1, kNT>(td, lo, lane, use_e, v);
                valid = 0xFFFFFFFFu;
            }
#pragma unroll
            for (int r = 0; r < 8 && !(whole || kDGC); ++r) {
                const uint32_t e0 = lo + 256u * r + 4u * (uint32_t)lane;
                float g4[4] = {0.f, 0.f, 0.f, 0.f}, e4[4] = {0.f, 0.f, 0.f, 0.f};
                if (e0 + 3 < td.n) {
                    if (td.dtype == 0) {
                        const f32x4 x = ldg4f_s<kNT>((const float*)td.grad + e0);
                        g4[0] = x.x; g4[1] = x.y; g4[2] = x.z; g4[3] = x.w;
                    } else {
                        const u32x2 h = ldg2u_s<kNT>((const uint16_t*)td.grad + e0);
                        g4[0] = h2f(h.x & 0xFFFFu);
                        g4[1] = h2f(h.x >> 16);
                        g4[2] = h2f(h.y & 0xFFFFu);
                        g4[3] = h2f(h.y >> 16);
                    }
                    if (use_e) {
                        const f32x4 y = ldg4f_s<kNT>(td.resid + e0);
                        e4[0] = y.x; e4[1] = y.y; e4[2] = y.z; e4[3] = y.w;
                    }
                    valid |= 0xFu << (4 * r);
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (e0 + i < td.n) {
                            g4[i] = td.dtype == 0 ? gp((const float*)td.grad)[e0 + i]
                                                  : h2f(gp((const uint16_t*)td.grad)[e0 + i]);
                            if (use_e) e4[i] = gp(td.resid)[e0 + i];
                            valid |= 1u << (4 * r + i);
                        }
                    }
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) v[4 * r + i] = use_e ? g4[i] + e4[i] : g4[i];
            }
            uint32_t pm = 0;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const uint32_t word = bm[q * (uint32_t)kChunkWords + 64u * half + 8 * r + (lane >> 3)];
                pm |= ((word >> (4 * (lane & 7))) & 0xFu) << (4 * r);
            }
            pm &= valid;
            if (use_e) {
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const uint32_t e0 = lo + 256u * r + 4u * (uint32_t)lane;
                    float o[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) o[i] = ((pm >> (4 * r + i)) & 1u) ? 0.f : v[4 * r + i];
                    if (whole || e0 + 3 < td.n) {
                        stg4f_s<kNT>(td.resid + e0, f32x4{o[0], o[1], o[2], o[3]});
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (e0 + i < td.n) gp(td.resid)[e0 + i] = o[i];
                    }
                    if constexpr (kDGC) {  // u with the selected entries masked
                        float* vel = (float*)const_cast<void*>(td.grad);
#pragma unroll
                        for (int i = 0; i < 4; ++i) o[i] = ((pm >> (4 * r + i)) & 1u) ? 0.f : un[4 * r + i];
                        if (whole || e0 + 3 < td.n) {
                            stg4f_s<kNT>(vel + e0, f32x4{o[0], o[1], o[2], o[3]});
                        } else {
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                if (e0 + i < td.n) gp(vel)[e0 + i] = o[i];
                        }
                    }
                }
            }
            // positions: 16-bit per-round counts, four rounds per 64-bit word,
            // scanned over the lanes; a round's base is the sum of earlier rounds
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint64_t packed = 0;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    packed |= (uint64_t)__popc((pm >> (16 * h + 4 * r)) & 0xFu) << (16 * r);
                uint64_t inc = packed;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const uint64_t y = __shfl_up(inc, o, 64);
                    if (lane >= o) inc += y;
                }
                const uint64_t tot = __shfl(inc, 63, 64);
                const uint64_t pre = inc - packed;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int rr = 4 * h + r;
                    uint64_t at = base + ((pre >> (16 * r)) & 0xFFFFu);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (((pm >> (4 * rr + i)) & 1u) && at < end) {  // the bucket's range bounds every write
                            idx[at] = lo + 256u * rr + 4u * (uint32_t)lane + i;
                            val[at] = v[4 * rr + i];
                            ++at;
                        }
                    }
                    base += (tot >> (16 * r)) & 0xFFFFu;
                }
            }
        }
    }
}

bool randk_buckets(uint32_t C, uint32_t* S, uint32_t* NB) {
    uint32_t s = 0;
    while (s < kRandkMaxShift && ((C + (1u << s) - 1) >> s) > kRandkBuckets) ++s;
    const uint32_t nb = (C + (1u << s) - 1) >> s;
    if (S) *S = s;
    if (NB) *NB = nb;
    return nb <= kRandkMaxBuckets;
}

namespace {
// Dynamic LDS beyond 64 KiB must be allowed per kernel; raise a kernel's
// limit to what a call needs (at most 2^8 chunks of bitmap, 128 KiB).
hipError_t need_lds(const void* f, size_t bytes, size_t& allowed) {
    if (bytes <= 64 * 1024 || bytes <= allowed) return hipSuccess;
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) allowed = bytes;
    return e;
}
std::mutex g_lds_mu;
size_t g_lds_place = 0, g_lds_stream[2][2] = {{0, 0}, {0, 0}};  // [non-temporal][DGC]

template <bool kNT, bool kDGC>
hipError_t need_lds_stream(size_t bytes) {
    return need_lds((const void*)randk_stream<kNT, false, kDGC>, bytes, g_lds_stream[kNT][kDGC]);
}
}  // namespace

hipError_t launch_randk(uint64_t seed, const TDesc* d, int T, uint32_t C, uint64_t sum_k, bool,
                        bool, uint32_t* idx, float* val, const Ws& ws, hipStream_t s, const DgcFuse* dgc) {
    if (C == 0 || T == 0) return hipSuccess;
    uint32_t S, NB;
    if (!randk_buckets(C, &S, &NB) || sum_k >= (1ull << 32)) return hipErrorInvalidValue;
    // runs of 2^SP chunks per stream workgroup: shorter runs balance the
    // pass's end better (long-lived workgroups leave the chip part-idle
    // while the last ones finish), but each of a bucket's 2^(S - SP)
    // workgroups reads the whole bucket list, so runs are split only while
    // those re-reads stay under a quarter of the 8 B-per-element input, at
    // most 32 runs per bucket, and never below 2 chunks (half a chunk per
    // wave).  A DGC step keeps whole chunks per wave (its half-chunk form
    // holds too many registers) and so runs of at least 4 chunks.
    uint32_t SP = S;
    const uint32_t sp_min = dgc ? 2u : 1u;
    while (SP > sp_min && S - SP < 5 && ((sum_k << (S - SP + 1)) * 4 <= (uint64_t)C * kChunk * 2)) --SP;
    const size_t lds_place = (size_t)NB * 8, lds_stream = ((size_t)kChunkWords * 4) << SP;
    {
        std::lock_guard<std::mutex> lk(g_lds_mu);
        hipError_t e = need_lds((const void*)randk_place, lds_place, g_lds_place);
        // (runs of more than 2 chunks: 2^SP * 512 bytes, at most 128 KiB)
        if (e == hipSuccess) e = need_lds_stream<false, false>(lds_stream);
        if (e == hipSuccess) e = need_lds_stream<true, false>(lds_stream);
        if (e == hipSuccess) e = need_lds_stream<false, true>(lds_stream);
        if (e == hipSuccess) e = need_lds_stream<true, true>(lds_stream);
        if (e != hipSuccess) return e;
    }
    const dim3 blk(kBlock);
    const uint32_t nscan = (NB + kScanBlock - 1) / kScanBlock;
    uint64_t* bsum = ws.r_coff + (size_t)NB + 1;  // scratch after the bucket offsets
    hipLaunchKernelGGL(randk_prep, dim3((T + 255) / 256), dim3(256), 0, s, d, T, seed, ws);
    const uint32_t nblk = (uint32_t)((sum_k + kGenEntries - 1) / kGenEntries);
    if (nblk) {
        hipLaunchKernelGGL(randk_count, dim3(nblk), dim3(kGenBlock), (size_t)NB * 4, s, d, T, sum_k, S, NB, idx,
                           ws);
    }
    hipLaunchKernelGGL(randk_columns, dim3((NB + 63) / 64), dim3(kColBlock), 0, s, NB, nblk, ws);
    hipLaunchKernelGGL(randk_scan_sums, dim3(nscan), blk, 0, s, NB, ws, bsum);
    hipLaunchKernelGGL(randk_scan_apply, dim3(nscan), blk, 0, s, NB, ws, bsum);
    if (nblk)
        hipLaunchKernelGGL(randk_place, dim3(nblk), dim3(kGenBlock), lds_place, s, d, T, sum_k, S, NB,
                           (const uint32_t*)idx, ws);
    // ids in groups of 8F: 8 buckets' F runs each (a last group may hold
    // fewer buckets: its surplus workgroups return at once)
    const uint32_t F = 1u << (S - SP);
    const dim3 sgrid((NB + 7) / 8 * 8 * F);
    const bool nt = C > kNtChunks, halves = SP <= 1;
    const DgcFuse f = dgc ? *dgc : DgcFuse{nullptr, 0.f, nullptr};
    const auto kern = dgc ? (nt ? randk_stream<true, false, true> : randk_stream<false, false, true>)
                          : (nt ? (halves ? randk_stream<true, true, false> : randk_stream<true, false, false>)
                                : (halves ? randk_stream<false, true, false> : randk_stream<false, false, false>));
    return launch_timed(kTimedRandkStream, kern, sgrid, blk, lds_stream, s, d, T, C, S, SP, NB, idx, val, ws, f);
}

}  // namespace bc
