// kernels_agg_sparse.hip -- sparse decompress-and-aggregate of W workers'
// payloads on gfx950 (paper Sec. 3.1, Reason #2: after the gather each node
// decompresses the N payloads and aggregates them; Sec. 4.2.1, Dimension 3:
// the aggregation of compressed tensors is not associative, so it is not an
// Allreduce).
//
// out_t[i] = alpha * (sum of the workers' values at i, added in ascending
// worker order, one fp32 addition each, starting from +0.0).  No
// floating-point atomics are used, so results are deterministic and match
// that order bit for bit.
//
// Each wave owns a run of 2048-, 4096- or 8192-element output tiles held in
// LDS.
// For every tile it walks the workers in order; worker w's entries for the
// tile are the next ones after its cursor (indices ascending), read 64 at a
// time and added into the tile (indices are unique within a worker, so a
// worker's adds never collide and need no atomics).  Cursors are found by a
// search (lower_bound_guess) only where a wave's run starts inside a
// tensor.  Two forms: a slot pipeline that keeps 8 or 16 workers' next
// windows in flight (any W), and a ring form for 33 to 64 workers that
// keeps every worker's window in registers across the whole run (below).
#include <mutex>

#include "launch.hpp"

namespace bc {

// First position p in [0, k) with idx[p] >= x (k if none) for a tensor of
// n elements, starting at the position the entries would have if they were
// spread evenly over the tensor: a gallop away from that guess (steps of
// 32, 64, ... positions) brackets the answer and a binary search finishes
// inside the bracket.  On evenly spread indices the answer lies within a
// few hundred positions of the guess, so a search reads about seven lines
// of the index array instead of one per halving.
__device__ __forceinline__ uint32_t lower_bound_guess(const uint32_t* idx, uint32_t k, uint32_t n, uint32_t x) {
    if (k == 0) return 0;
    uint32_t g = n ? (uint32_t)(((uint64_t)k * x) / n) : 0u;
    if (g >= k) g = k - 1;
    uint32_t lo, hi;  // the answer lies in [lo, hi]
    if (gp(idx)[g] < x) {
        lo = g + 1;
        hi = k;
        for (uint32_t step = 32;; step *= 2) {
            const uint64_t q = (uint64_t)g + step;
            if (q >= k) break;
            if (gp(idx)[q] >= x) {
                hi = (uint32_t)q;
                break;
            }
            lo = (uint32_t)q + 1;
        }
    } else {
        lo = 0;
        hi = g;
        for (uint32_t step = 32;; step *= 2) {
            if (g < step) break;
            const uint32_t q = g - step;
            if (gp(idx)[q] < x) {
                lo = q + 1;
                break;
            }
            hi = q;
        }
    }
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (gp(idx)[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// Each wave owns a run of consecutive kTS-element tiles held in its own LDS
// slice.  The next 64 kEPL entries of kS workers (a window: lane l holds
// entries l, l + 64, ... of it) are kept in flight in registers
// (slot w % kS holds worker w): as soon as a worker's entries for the tile
// have been added, its slot is refilled with the worker that comes kS
// later, or, when W is a multiple of kS and the next tile continues the
// tensor, with the entries of the slot's first worker (w % kS) for the next
// tile (its cursor is final by then).
//
// kLanes (W <= 64): lane w of a VGPR holds worker w's cursor and its two
// payload pointers (already offset to the tensor), read with readlane, so
// a step touches neither LDS nor the scalar cache for bookkeeping.
// Otherwise the cursors live in LDS after the tiles and the pointers are
// read from the worker table.
//
// kNT: the output tiles are written with the non-temporal hint (outputs
// larger than the last-level cache).
//
// kEPL = 2 (8192-element tiles, for calls with many tiles) halves the
// steps per element of the 4096-element form: each step covers a worker's
// next 128 entries, two per lane.
//
// kRagged (with kLanes): the payloads are parts packed by
// bytecomp_pack_part, so worker w's entries of tensor t start at
// rp_w[t] and number rp_w[t+1] - rp_w[t] (rp[w] is worker w's part-offset
// array); a worker with no entries reads a dummy location rp[Wp] instead.
template <uint32_t kTS, int kS, bool kLanes, bool kRagged, bool kNT, int kEPL>
__global__ __launch_bounds__(kBlock) void aggregate_sparse(const ADesc* __restrict__ a, int T,
                                                           uint32_t U, const uint64_t* __restrict__ wp,
                                                           int W, float alpha, const uint64_t* __restrict__ rp) {
    static_assert(kLanes || !kRagged, "ragged payloads need the lane-held worker state");
    extern __shared__ uint32_t lds[];
    const int wave = wave_id();
    const int lane = lane_id();
    float* tile = reinterpret_cast<float*>(lds) + wave * (int)kTS;
    uint32_t* cur = lds + 4 * kTS + wave * W;  // !kLanes only
    const uint64_t nw = (uint64_t)gridDim.x * 4;
    const uint64_t gw = (uint64_t)blockIdx.x * 4 + wave;
    const uint32_t u_beg = (uint32_t)((gw * U) / nw);
    const uint32_t u_end = (uint32_t)(((gw + 1) * U) / nw);
    const bool cross = (W % kS) == 0;
    // per-lane worker state (kLanes): cursor, payload pointers of the tensor,
    // and (kRagged) the worker's entry count of the tensor
    uint32_t curv = 0;
    uint64_t pav = 0, pbv = 0;
    uint32_t kv = 0;
    auto get_cur = [&](int w) -> uint32_t {
        if constexpr (kLanes) return (uint32_t)__builtin_amdgcn_readlane((int)curv, w);
        else return cur[w];
    };
    auto set_cur = [&](int w, uint32_t c) {
        if constexpr (kLanes) curv = lane == w ? c : curv;
        else if (lane == 0) cur[w] = c;
    };
    // Every slot load is issued unconditionally (index clamped into the
    // tensor's entries) so that the compiler can count the loads in flight
    // exactly and wait only for the one it needs; a dead slot's entries are
    // masked by setting every bit of its index (never below a tile end).
    constexpr uint32_t kWin = 64u * kEPL;  // entries per window
    uint32_t x[kS][kEPL];
    float y[kS][kEPL];
    uint32_t inv[kS][kEPL];
    int t = -1;
    ADesc ad{};
    bool primed = false;  // slots already hold this tile's first entries
    for (uint32_t u = u_beg; u < u_end; ++u) {
        if (t < 0 || u >= ad.unit0 + ad.nunits) {
            t = unit_owner(wp, W, u);
            ad = a[t];
            const uint32_t lo0 = (u - ad.unit0) * kTS;
            if constexpr (kRagged) {
                const int wl = lane < W ? lane : W - 1;
                const uint64_t* po = (const uint64_t*)rp[wl];
                const uint64_t o0 = po[t], o1 = po[t + 1];
                kv = (uint32_t)(o1 - o0);
                pav = kv ? wp[wl] + o0 * 4u : rp[padded_workers(W)];
                pbv = kv ? wp[padded_workers(W) + wl] + o0 * 4u : rp[padded_workers(W)];
                curv = lo0 == 0 ? 0u : lower_bound_guess((const uint32_t*)pav, kv, ad.n, lo0);
            } else if constexpr (kLanes) {
                const int wl = lane < W ? lane : W - 1;
                pav = wp[wl] + ad.off * 4u;
                pbv = wp[padded_workers(W) + wl] + ad.off * 4u;
                curv = lo0 == 0 ? 0u : lower_bound_guess((const uint32_t*)pav, ad.k, ad.n, lo0);
            } else {
                for (int w = lane; w < W; w += 64)
                    cur[w] = lo0 == 0 ? 0u : lower_bound_guess(w_a(wp, w) + ad.off, ad.k, ad.n, lo0);
                __builtin_amdgcn_wave_barrier();
            }
            primed = false;
        }
        // entries of worker w in this tensor (the same for every worker unless
        // the payloads are ragged parts; a part may hold none)
        auto k_of = [&](int w) -> uint32_t {
            if constexpr (kRagged) return (uint32_t)__builtin_amdgcn_readlane((int)kv, w);
            else return ad.k;
        };
        auto load_slot = [&](int q, int w, uint32_t c, bool live) {
            const uint32_t kw = k_of(w);
            const uint32_t* pa;
            const float* pb;
            if constexpr (kLanes) {
                pa = (const uint32_t*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pav >> 32), w) << 32) |
                                       (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pav, w));
                pb = (const float*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pbv >> 32), w) << 32) |
                                    (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pbv, w));
            } else {
                pa = w_a(wp, w) + ad.off;
                pb = w_b(wp, W, w) + ad.off;
            }
#pragma unroll
            for (int e = 0; e < kEPL; ++e) {
                const uint32_t i = c + 64u * e + lane;
                const uint32_t ic = i < kw ? i : (kw ? kw - 1u : 0u);
                x[q][e] = gp(pa)[ic];
                y[q][e] = gp(pb)[ic];
                inv[q][e] = (live && i < kw) ? 0u : 0xFFFFFFFFu;
                asm volatile("" : "+v"(inv[q][e]));  // computed here, not sunk to its use
            }
        };
        if (!primed) {
            // W through an opaque copy: keeps the sixteen per-slot worker
            // numbers and flags from being hoisted into live SGPRs
            int Wq = W;
            asm volatile("" : "+s"(Wq));
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                const int w = q < Wq ? q : Wq - 1;
                load_slot(q, w, get_cur(w), q < Wq);
            }
        }
        const uint32_t lo = (u - ad.unit0) * kTS;
        const uint32_t hi = (lo + kTS < ad.n) ? lo + kTS : ad.n;
        const uint32_t len = hi - lo;
        const bool next_same = cross && u + 1 < u_end && u + 1 < ad.unit0 + ad.nunits;
#pragma unroll
        for (uint32_t r = 0; r < kTS / 256u; ++r)
            *reinterpret_cast<f32x4*>(tile + 256u * r + 4u * lane) = f32x4{0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_wave_barrier();
        // a worker with a whole window or more in the tile (dense payloads)
        // ends the pipelined walk: the rest of the tile, from that worker
        // on, is finished one window at a time below.  Keeping that
        // loop out of the pipelined steps keeps their load waits exact.
        int dw = -1;
        uint32_t dcc = 0;
        for (int w0 = 0; w0 < W; w0 += kS) {
            // all kS steps issue their two loads on every path (the ones
            // past W or after a dense worker are dead), so that the compiler
            // counts the loads in flight the same way on every path
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                const int w = w0 + q;
                // W through an opaque copy per step, so that the per-step
                // flags are computed here rather than hoisted into SGPRs
                int Wq = W;
                asm volatile("" : "+s"(Wq));
                uint32_t cc = 0;
                if (w < Wq && dw < 0) {  // no load in here
                    cc = get_cur(w);
                    uint32_t cnt = 0;
#pragma unroll
                    for (int e = 0; e < kEPL; ++e) {
                        const uint32_t xv = x[q][e] | inv[q][e];
                        cnt += (uint32_t)__popcll(__ballot(xv < hi));
                        // entries below the tile can only come from an unsorted
                        // payload; they are skipped rather than written out of range
                        const uint32_t dd = xv - lo;
                        if (dd < len) tile[dd] += y[q][e];
                    }
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                    if (cnt == kWin) {
                        dw = w;
                        dcc = cc;
                    } else {
                        set_cur(w, cc);
                    }
                }
                // refill the slot: the worker kS later in this tile, or else
                // (W a multiple of kS) worker q's entries for the next tile,
                // its cursor being final here
                const int wn = w + kS;
                const bool later = wn < Wq;
                int wr = later ? wn : wn - Wq;
                wr = wr < Wq ? wr : Wq - 1;
                const bool live = w < Wq && dw < 0 && (later || next_same);
                load_slot(q, wr, later ? get_cur(wn) : (wr == w ? cc : get_cur(wr)), live);
            }
            if (dw >= 0) break;
        }
        if (dw >= 0) {
            for (int w = dw; w < W; ++w) {
                uint32_t cc = w == dw ? dcc : get_cur(w);
                const uint32_t* pa;
                const float* pb;
                if constexpr (kLanes) {
                    pa = (const uint32_t*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pav >> 32), w) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pav, w));
                    pb = (const float*)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(pbv >> 32), w) << 32) |
                                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pbv, w));
                } else {
                    pa = w_a(wp, w) + ad.off;
                    pb = w_b(wp, W, w) + ad.off;
                }
                uint32_t cnt = kWin;
                while (cnt == kWin) {
                    const uint32_t kw = k_of(w);
                    cnt = 0;
#pragma unroll
                    for (int e = 0; e < kEPL; ++e) {
                        const uint32_t i = cc + 64u * e + lane;
                        const bool oki = i < kw;
                        const uint32_t ic = oki ? i : (kw ? kw - 1u : 0u);
                        const uint32_t xi = oki ? gp(pa)[ic] : 0xFFFFFFFFu;
                        const float yi = gp(pb)[ic];
                        cnt += (uint32_t)__popcll(__ballot(xi < hi));
                        const uint32_t dd = xi - lo;
                        if (dd < len) tile[dd] += yi;
                    }
                    cc += cnt;
                    __builtin_amdgcn_wave_barrier();
                }
                set_cur(w, cc);
            }
            primed = false;
        } else {
            primed = next_same;
        }
        float* out = ad.out + lo;
        if (len == kTS) {
#pragma unroll
            for (uint32_t r = 0; r < kTS / 256u; ++r) {
                const uint32_t i = 256u * r + 4u * lane;
                const f32x4 v = *reinterpret_cast<const f32x4*>(tile + i);
                stg4f_s<kNT>(out + i, f32x4{alpha * v[0], alpha * v[1], alpha * v[2], alpha * v[3]});
            }
        } else {
            for (uint32_t i = 4u * lane; i < len; i += 256u) {
                if (i + 3 < len) {
                    stg4f_s<kNT>(out + i, f32x4{alpha * tile[i], alpha * tile[i + 1], alpha * tile[i + 2],
                                         alpha * tile[i + 3]});
                } else {
                    for (uint32_t q = i; q < len; ++q) gp(out)[q] = alpha * tile[q];
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
}


// ------------------------------------------------------ ring-window form
// For W <= 64 and sparse enough payloads: every worker keeps one 64-entry
// window of (index, value) pairs in registers for the wave's whole run of
// tiles, as a ring -- lane l holds the window's entry whose position in the
// worker's payload is congruent to l modulo 64.  The window of worker w
// starts at its cursor c and holds positions [c, c + 64).  A step adds the
// window's entries that fall in the tile (a prefix of the window: indices
// ascend and everything below the tile was consumed before) into the tile,
// then reloads exactly the lanes it consumed with the positions 64 further
// on.  Every payload entry is thus fetched once per call, and a reload has
// a whole round of the other workers' steps to arrive before it is used.
// A worker with more than 64 entries in one tile repeats the step after
// its reload has arrived (rare at the densities this form is chosen for).
//
// Loads go through buffer resources sized to the worker's entry count:
// positions past it read zero without touching memory, and the lanes that
// hold them are masked out of the step by the count, so the windows need
// no clamping.  Each step does one LDS read-add-write: lanes with nothing
// to add address a per-lane dummy word past the tile instead of branching.

__device__ __forceinline__ __amdgpu_buffer_rsrc_t entries_rsrc(uint64_t base, uint32_t k) {
    // raw buffer over k 4-byte entries (gfx9 word 3: 32-bit data format)
    return __builtin_amdgcn_make_buffer_rsrc((void*)(uintptr_t)base, (short)0, (int)(k * 4u), 0x00020000);
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), l) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
}

// Lane state of worker `lane` for tensor t: entry count and the bases of
// its index and value arrays (lanes past W copy worker W - 1; they are
// never read for a worker number >= W).
template <bool kRagged>
__device__ __forceinline__ void ring_lane_state(const ADesc& ad, int t, const uint64_t* __restrict__ wp, int W,
                                                const uint64_t* __restrict__ rp, uint32_t& kv, uint64_t& pav,
                                                uint64_t& pbv) {
    const int lane = lane_id();
    const int wl = lane < W ? lane : W - 1;
    const int Wp = padded_workers(W);
    if constexpr (kRagged) {
        const uint64_t* po = (const uint64_t*)rp[wl];
        const uint64_t o0 = po[t], o1 = po[t + 1];
        kv = (uint32_t)(o1 - o0);
        pav = wp[wl] + o0 * 4u;
        pbv = wp[Wp + wl] + o0 * 4u;
    } else {
        kv = ad.k;
        pav = wp[wl] + ad.off * 4u;
        pbv = wp[Wp + wl] + ad.off * 4u;
    }
}

// kW: worker slots (8, 16, 32 or 64; slots W .. kW - 1 hold no entries and
// their steps add nothing).  kRagged: as in aggregate_sparse (parts packed
// by bytecomp_pack_part).
//
// Every window register has one definition inside the tile loop, the
// step's reload, so that the compiler keeps each window in place and
// tracks its loads exactly: the reload of a tensor's last tile already
// fetches the next tensor's first window (cursor 0), and the windows of
// the run's first tile are fetched before the loop.
template <uint32_t kTS, int kW, bool kRagged, bool kNT>
__global__ __launch_bounds__(kBlock) void aggregate_sparse_ring(const ADesc* __restrict__ a, int T, uint32_t U,
                                                                const uint64_t* __restrict__ wp, int W, float alpha,
                                                                const uint64_t* __restrict__ rp) {
    extern __shared__ uint32_t lds[];
    const int wave = wave_id();
    const int lane = lane_id();
    float* tile = reinterpret_cast<float*>(lds) + wave * (int)(kTS + 64u);
    const uint64_t nw = (uint64_t)gridDim.x * 4;
    const uint64_t gw = (uint64_t)blockIdx.x * 4 + wave;
    const uint32_t u_beg = (uint32_t)((gw * U) / nw);
    const uint32_t u_end = (uint32_t)(((gw + 1) * U) / nw);
    if (u_beg >= u_end) return;
    // the windows: worker w's entries in x[w] (indices) and y[w] (values)
    uint32_t x[kW];
    float y[kW];
    auto fetch = [&](uint64_t pa, uint64_t pb, uint32_t kw, uint32_t pos, uint32_t& xo, float& yo) {
        xo = __builtin_amdgcn_raw_buffer_load_b32(entries_rsrc(pa, kw), (int)(pos * 4u), 0, 0);
        yo = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(entries_rsrc(pb, kw), (int)(pos * 4u), 0, 0));
    };
    // lane w: worker w's cursor, entry count and payload bases for the tensor
    int t = unit_owner(wp, W, u_beg);
    ADesc ad = a[t];
    uint32_t kv, curv;
    uint64_t pav, pbv;
    ring_lane_state<kRagged>(ad, t, wp, W, rp, kv, pav, pbv);
    {
        const uint32_t lo0 = (u_beg - ad.unit0) * kTS;
        curv = 0;
        if (lo0 != 0 && lane < W) curv = lower_bound_guess((const uint32_t*)pav, kv, ad.n, lo0);
        if (lane >= W) kv = curv = 0;  // empty slots
#pragma unroll
        for (int w = 0; w < kW; ++w) {
            const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)curv, w);
            fetch(readlane64(pav, w), readlane64(pbv, w), (uint32_t)__builtin_amdgcn_readlane((int)kv, w),
                  c + (((uint32_t)lane - c) & 63u), x[w], y[w]);
        }
    }
    for (uint32_t u = u_beg; u < u_end; ++u) {
        const uint32_t lo = (u - ad.unit0) * kTS;
        const uint32_t hi = (lo + kTS < ad.n) ? lo + kTS : ad.n;
        const uint32_t len = hi - lo;
        // the next tile starts another tensor: its state, for the reloads
        const bool sw = u + 1 < u_end && u + 1 >= ad.unit0 + ad.nunits;
        int t2 = t;
        ADesc ad2 = ad;
        uint32_t kv2 = kv;
        uint64_t pav2 = pav, pbv2 = pbv;
        if (sw) {
            t2 = unit_owner(wp, W, u + 1);
            ad2 = a[t2];
            ring_lane_state<kRagged>(ad2, t2, wp, W, rp, kv2, pav2, pbv2);
            if (lane >= W) kv2 = 0;
        }
#pragma unroll
        for (uint32_t r = 0; r < kTS / 256u; ++r)
            *reinterpret_cast<f32x4*>(tile + 256u * r + 4u * lane) = f32x4{0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int w = 0; w < kW; ++w) {
            const uint32_t kw = (uint32_t)__builtin_amdgcn_readlane((int)kv, w);
            const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)curv, w);
            // lanes holding positions below the worker's count
            const uint32_t rem = kw - c;
            uint64_t vm = rem >= 64u ? ~0ull : ((1ull << rem) - 1ull);
            const uint32_t sh = c & 63u;
            vm = sh ? (vm << sh) | (vm >> (64u - sh)) : vm;
            const uint32_t dd = x[w] - lo;
            const uint64_t m = __ballot(dd < len) & vm;
            const uint32_t cnt = (uint32_t)__popcll(m);
            const uint32_t at = __builtin_amdgcn_inverse_ballot_w64(m) ? dd : kTS + (uint32_t)lane;
            const float v = tile[at];
            tile[at] = v + y[w];
            uint32_t cf = c + cnt;
            const bool dense = cnt == 64u;
            if (dense) {
                // the whole window was in the tile: continue straight from
                // the payload, 64 positions at a time, until the worker's
                // entries leave the tile
                const uint64_t pa = readlane64(pav, w), pb = readlane64(pbv, w);
                uint32_t more = 64u;
                while (more == 64u) {
                    const uint32_t pos = cf + (uint32_t)lane;
                    uint32_t xi;
                    float yi;
                    fetch(pa, pb, kw, pos, xi, yi);
                    const uint32_t di = xi - lo;
                    const uint64_t mi = __ballot(pos < kw && di < len);
                    more = (uint32_t)__popcll(mi);
                    const uint32_t ai = __builtin_amdgcn_inverse_ballot_w64(mi) ? di : kTS + (uint32_t)lane;
                    const float vi = tile[ai];
                    tile[ai] = vi + yi;
                    cf += more;
                }
            }
            // the window moves to positions [cf, cf + 64) (the next tensor's
            // [0, 64) when the tile ends a tensor): the consumed lanes load
            // their new positions (c + 64 + p is cf's ring slot of lane p),
            // every lane after a dense tile or at a tensor switch
            const uint32_t c2 = sw ? 0u : cf;
            const uint32_t p = ((uint32_t)lane - c) & 63u;
            if (sw || dense || p < cnt)
                fetch(readlane64(sw ? pav2 : pav, w), readlane64(sw ? pbv2 : pbv, w),
                      sw ? (uint32_t)__builtin_amdgcn_readlane((int)kv2, w) : kw,
                      c2 + (((uint32_t)lane - c2) & 63u), x[w], y[w]);
            curv = __builtin_amdgcn_inverse_ballot_w64(1ull << w) ? c2 : curv;
        }
        __builtin_amdgcn_wave_barrier();
        float* out = ad.out + lo;
        if (len == kTS) {
#pragma unroll
            for (uint32_t r = 0; r < kTS / 256u; ++r) {
                const uint32_t i = 256u * r + 4u * lane;
                const f32x4 v = *reinterpret_cast<const f32x4*>(tile + i);
                stg4f_s<kNT>(out + i, f32x4{alpha * v[0], alpha * v[1], alpha * v[2], alpha * v[3]});
            }
        } else {
            for (uint32_t i = 4u * lane; i < len; i += 256u) {
                if (i + 3 < len) {
                    stg4f_s<kNT>(out + i, f32x4{alpha * tile[i], alpha * tile[i + 1], alpha * tile[i + 2],
                                         alpha * tile[i + 3]});
                } else {
                    for (uint32_t q = i; q < len; ++q) gp(out)[q] = alpha * tile[q];
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (sw) {
            t = t2;
            ad = ad2;
            kv = kv2;
            pav = pav2;
            pbv = pbv2;
        }
    }
}

// -------------------------------------------------------------- launchers
uint32_t sparse_agg_tile(uint64_t n_total, uint64_t k_total, int W, bool* ring) {
    // ring form (more than 32 workers; fewer take the slot pipeline below,
    // measured faster there): the largest tile in which a worker holds about
    // 44 entries or fewer on average (its 64-entry window then almost never
    // runs dry inside a tile); entry counts stay below 2^30 for 32-bit byte
    // offsets
    *ring = false;
    if (W > 32 && W <= 64 && k_total < (1ull << 30) - 64u && n_total > 0) {
        for (uint32_t ts = 8192u; ts >= 1024u; ts >>= 1)
            if (k_total * ts <= n_total * 44u) {
                *ring = true;
                return ts;
            }
    }
    // 8192-element tiles (128-entry windows) for calls of at least 2^24
    // elements whose workers hold about 100 entries per such tile or fewer;
    // else 4096-element tiles while a worker holds about 48 entries per tile
    // or fewer (one 64-entry window covers its entries); 2048 otherwise
    if (n_total >= (1ull << 24) && k_total * 8192u <= n_total * 100u) return 8192u;
    return k_total * 4096u <= n_total * 48u ? 4096u : 2048u;
}

namespace {
template <uint32_t kTS, int kS, bool kLanes, bool kRagged, bool kNT>
hipError_t launch_sparse_t(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                           const uint64_t* rp, hipStream_t s) {
    constexpr int kEPL = kTS > 4096u ? 2 : 1;
    const auto kern = aggregate_sparse<kTS, kS, kLanes, kRagged, kNT, kEPL>;
    const size_t lds = (size_t)4 * (kTS * 4 + (kLanes ? 0 : (size_t)W * 4));
    // one round of resident workgroups at this LDS size (more waves with
    // shorter runs measured slower)
    size_t per_cu = (160u * 1024u) / lds;
    if (per_cu < 1) per_cu = 1;
    if (per_cu > 8) per_cu = 8;
    // LDS past 64 KiB per workgroup must be allowed per kernel (once; the
    // largest size this instantiation meets)
    if (lds > 64 * 1024) {
        static std::mutex mu;
        static size_t allowed = 0;
        std::lock_guard<std::mutex> lk(mu);
        if (lds > allowed) {
            const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)lds);
            if (e != hipSuccess) return e;
            allowed = lds;
        }
    }
    uint64_t blocks = (U + 3) / 4;
    const uint64_t cap = per_cu * (uint64_t)(cus > 0 ? cus : 256);
    if (blocks > cap) blocks = cap;
    return launch_timed(kTimedAggSparse, kern, dim3((uint32_t)blocks), dim3(kBlock), lds, s, a, T, U, w, W, alpha,
                        rp);
}
template <uint32_t kTS, bool kRagged, bool kNT>
hipError_t launch_sparse_nt(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                            const uint64_t* rp, hipStream_t s) {
    if constexpr (!kRagged) {
        if (W > 64) return launch_sparse_t<kTS, 16, false, false, kNT>(a, T, U, w, W, alpha, cus, rp, s);
    }
    if (W % 16 == 0 || W % 8 != 0) return launch_sparse_t<kTS, 16, true, kRagged, kNT>(a, T, U, w, W, alpha, cus, rp, s);
    return launch_sparse_t<kTS, 8, true, kRagged, kNT>(a, T, U, w, W, alpha, cus, rp, s);
}
// Outputs past this many tiles (256 MB at 4096 elements) are written with
// the non-temporal hint.
constexpr uint32_t kNtTiles = 16384;
template <uint32_t kTS, bool kRagged>
hipError_t launch_sparse_ts(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                            const uint64_t* rp, hipStream_t s) {
    if ((uint64_t)U * kTS > (uint64_t)kNtTiles * 4096u)
        return launch_sparse_nt<kTS, kRagged, true>(a, T, U, w, W, alpha, cus, rp, s);
    return launch_sparse_nt<kTS, kRagged, false>(a, T, U, w, W, alpha, cus, rp, s);
}
}  // namespace

namespace {
template <uint32_t kTS, int kW, bool kRagged, bool kNT>
hipError_t launch_ring_t(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                         const uint64_t* rp, hipStream_t s) {
    const auto kern = aggregate_sparse_ring<kTS, kW, kRagged, kNT>;
    const size_t lds = (size_t)4 * 4 * (kTS + 64u);
    // one round of resident workgroups (registers and LDS decide how many)
    static int per_cu = 0;
    if (per_cu == 0) {
        int nb = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kBlock, lds);
        if (e != hipSuccess) return e;
        per_cu = nb > 0 ? nb : 1;
    }
    uint64_t blocks = (U + 3) / 4;
    const uint64_t cap = (uint64_t)per_cu * (uint64_t)(cus > 0 ? cus : 256);
    if (blocks > cap) blocks = cap;
    return launch_timed(kTimedAggSparse, kern, dim3((uint32_t)blocks), dim3(kBlock), lds, s, a, T, U, w, W, alpha,
                        rp);
}
template <uint32_t kTS, int kW, bool kRagged>
hipError_t launch_ring_nt(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                          const uint64_t* rp, hipStream_t s) {
    if ((uint64_t)U * kTS > (uint64_t)kNtTiles * 4096u)
        return launch_ring_t<kTS, kW, kRagged, true>(a, T, U, w, W, alpha, cus, rp, s);
    return launch_ring_t<kTS, kW, kRagged, false>(a, T, U, w, W, alpha, cus, rp, s);
}
template <uint32_t kTS, bool kRagged>
hipError_t launch_ring_ts(const ADesc* a, int T, uint32_t U, const uint64_t* w, int W, float alpha, int cus,
                          const uint64_t* rp, hipStream_t s) {
    // (the form is chosen for 33 to 64 workers)
    return launch_ring_nt<kTS, 64, kRagged>(a, T, U, w, W, alpha, cus, rp, s);
}
template <bool kRagged>
hipError_t launch_ring(const ADesc* a, int T, uint32_t U, uint32_t tile, const uint64_t* w, int W, float alpha,
                       int cus, const uint64_t* rp, hipStream_t s) {
    switch (tile) {
        case 8192u: return launch_ring_ts<8192u, kRagged>(a, T, U, w, W, alpha, cus, rp, s);
        case 4096u: return launch_ring_ts<4096u, kRagged>(a, T, U, w, W, alpha, cus, rp, s);
        case 2048u: return launch_ring_ts<2048u, kRagged>(a, T, U, w, W, alpha, cus, rp, s);
        case 1024u: return launch_ring_ts<1024u, kRagged>(a, T, U, w, W, alpha, cus, rp, s);
        default: return hipErrorInvalidValue;
    }
}
}  // namespace

hipError_t launch_aggregate_sparse(const ADesc* a, int T, uint32_t U, uint32_t tile, bool ring, const uint64_t* w,
                                   int W, float alpha, int cus, const uint64_t* rp, hipStream_t s) {
    if (U == 0) return hipSuccess;
    if ((rp || ring) && W > 64) return hipErrorInvalidValue;
    hipError_t e;
    if (ring) {
        e = rp ? launch_ring<true>(a, T, U, tile, w, W, alpha, cus, rp, s)
               : launch_ring<false>(a, T, U, tile, w, W, alpha, cus, nullptr, s);
    } else if (rp) {
        if (tile == 8192u) e = launch_sparse_ts<8192u, true>(a, T, U, w, W, alpha, cus, rp, s);
        else if (tile == 4096u) e = launch_sparse_ts<4096u, true>(a, T, U, w, W, alpha, cus, rp, s);
        else if (tile == 2048u) e = launch_sparse_ts<2048u, true>(a, T, U, w, W, alpha, cus, rp, s);
        else return hipErrorInvalidValue;
    } else {
        if (tile == 8192u) e = launch_sparse_ts<8192u, false>(a, T, U, w, W, alpha, cus, nullptr, s);
        else if (tile == 4096u) e = launch_sparse_ts<4096u, false>(a, T, U, w, W, alpha, cus, nullptr, s);
        else if (tile == 2048u) e = launch_sparse_ts<2048u, false>(a, T, U, w, W, alpha, cus, nullptr, s);
        else return hipErrorInvalidValue;
    }
    return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace bc
