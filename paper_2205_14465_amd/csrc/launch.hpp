// launch.hpp -- host-side launchers of the gfx950 kernels and the
// workspace carve-up they share.  Included by the C-ABI layer only.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "common.hpp"

namespace bc {

// Pointers into the caller's workspace.  Every call clears the counters it
// uses in its first kernel, so the workspace needs no initialisation and may
// be shared by calls of different kinds and shapes (not concurrently).
struct Ws {
    uint32_t* flags;        // header: failure flags
    // BC_SIGN1
    float* s_val;           // [T] published scales
    double* s_partial;      // [C] per-chunk sums of |v|
    uint32_t* s_info;       // [T] TernGrad aggregate: form (bits 0-7), smallest scale
                            // exponent (8-15)
    uint64_t* s_slot;       // [C] one-pass compress: ~bits of each chunk's partial sum once
                            // published, 0 otherwise (emptied before the kernel runs)
    int32_t* s_tab;         // TernGrad aggregate: int32 lookup tables of each tensor, [T * 4096]
    // BC_TERNGRAD, BC_QSGD4, BC_QSGD8 (and s_val)
    uint32_t* q_max;        // [C] largest |v| bits of each chunk
    uint32_t* q_slot;       // [C] one-pass compress: those bits | 1 << 31 once published, 0 otherwise
                            // (emptied before the kernel runs)
    // BC_TOPK, BC_TOPK_SAMPLED
    uint32_t* t_hist;       // [T * 2048] histograms         
    uint32_t* t_thr;        // [T] candidate threshold (key)
    uint32_t* t_prefix;     // [T] radix-select prefix (key)
    uint32_t* t_krem;       // [T] entries still to select
    uint32_t* t_fb;         // [T] 1 = tensor needs the exact-histogram fallback
    uint32_t* t_any;        // [1] nonzero when some tensor of the call needs it
    uint2* t_cand;          // [C * 4096] candidates (local index, value bits)
    uint32_t* t_ccount;     // [C] candidates per chunk
    uint32_t* t_gt;         // [C] candidates above the threshold key
    uint32_t* t_eq;         // [C] candidates equal to the threshold key
    uint64_t* t_off;        // [C] payload position of a chunk's first winner
    uint32_t* t_eqb;        // [C] equal-key candidates in earlier chunks
    // BC_RANDK
    uint32_t* r_keys;       // [T * 4] Feistel round keys
    uint32_t* r_tmp;        // [sum k] generated indices
    uint32_t* r_ccount;     // [NB] indices per bucket
    uint64_t* r_coff;       // [NB + 1] payload position of each bucket, then
                            // [ceil(NB / 4096)] scan block sums
    uint32_t* r_hist;       // [generating workgroups * NB] per-workgroup bucket
                            // counts, then positions within each bucket
    // DGC local clipping (sparse kinds)
    double* d_part;         // [C] sums of squares per chunk
    float* d_factor;        // [1] the clipping factor
};

// Byte offsets of every region for a call shape; `total` is the workspace
// size.  Regions a kind does not use have size 0.
struct WsPlan {
    size_t flags, s_val, s_partial, s_info, s_tab, s_slot, q_max, q_slot;
    size_t t_hist, t_thr, t_prefix, t_krem, t_fb, t_any, t_cand, t_ccount, t_gt, t_eq, t_off, t_eqb;
    size_t r_keys, r_tmp, r_ccount, r_coff, r_hist;
    size_t d_part, d_factor;
    size_t total;
};

// agg_tables false: without the regions only the sign and TernGrad
// aggregates use (a compress-only workspace).
WsPlan plan_workspace(int kind, int T, uint64_t chunks, uint64_t sum_k, bool agg_tables = true);
Ws carve_workspace(void* base, const WsPlan& p);

}  // namespace bc

#include "../../include/bytecomp.h"

namespace bc {

// A compress call checked on the host: its descriptor table (chunk map not
// included), chunk count, largest tensor in chunks, payload entries, dtype
// mix, whether a tensor is empty, and the workspace plan.
struct CompressPrep {
    std::vector<TDesc> d;
    uint32_t C = 0, maxc = 0;
    uint64_t sum_k = 0, ppm = 0;
    bool a16 = false, a32 = false, any_empty = false;
    WsPlan plan{};
};
// BC_OK (T = 0 included: nothing to do) or the call's error status.
int compress_prepare(int kind, double ratio, const bc_tensor* t, int T, const bc_payload& out, bool agg_tables,
                     CompressPrep& p);
// The kind's compress kernels on a device descriptor table (TDesc[T], then
// the chunk -> tensor map) and a carved workspace.
hipError_t compress_launch(int kind, double ratio, uint64_t seed, const CompressPrep& p, const TDesc* dd,
                           const bc_payload& out, const Ws& w, hipStream_t s);

struct DevInfo {
    int cus;
    bool any_empty;      // per call: some tensor has no elements
    int wall_khz;        // rate of the constant-rate counter kernels read (wall_clock64)
};
hipError_t device_info(int dev, DevInfo* out);

// ------------------------------------------------------- kernel timing
// Kernels a caller may ask to have timed (bytecomp_time_next_launch).
enum TimedKernel { kTimedNone = 0, kTimedAggSign, kTimedAggSparse, kTimedRandkStream, kTimedTopkCompact,
                   kTimedSignPass1, kTimedQuantPass1, kTimedAggQuant, kTimedSignOnepass, kTimedQuantOnepass,
                   kTimedTopkHist };
// If a request for kernel `k` is pending, hand over its events and clear it.
bool take_kernel_timer(int k, hipEvent_t* start, hipEvent_t* stop);

// How long (in ticks of the device's constant-rate counter, wall_clock64)
// a one-pass compress workgroup waits for the rest of its tensor's chunk
// partials before it computes the missing ones itself.
uint32_t onepass_wait_ticks();
// Copies of each top-k histogram in the general pipeline for a call of T
// tensors: workgroups add into copy (their index mod copies), which spreads
// the atomic additions to the busiest bins; readers add the copies.
inline int topk_general_copies(int T) { return T <= 256 ? 8 : T <= 1024 ? 2 : 1; }  // at most 8
// A profiler range (roctx) around one C-ABI call: a push at construction,
// the pop at scope exit; without a profiler attached both are plain calls.
struct CallRange {
    explicit CallRange(const char* name);
    ~CallRange();
    CallRange(const CallRange&) = delete;
    CallRange& operator=(const CallRange&) = delete;
};
// Top-k calls of at most this many chunks take the few-chunk path.
constexpr uint32_t kTopkFewChunksMax = 2048;  // 8M elements: its counts fit in 31 bits
uint32_t topk_few_chunks_limit();

// Launch `kernel`, bracketed by the requested events when kernel `k` is to
// be timed.
template <typename F, typename... Args>
inline hipError_t launch_timed(int k, F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                               Args... args) {
    hipEvent_t e0, e1;
    if (take_kernel_timer(k, &e0, &e1))
        hipExtLaunchKernelGGL(kernel, grid, block, (std::uint32_t)lds, s, e0, e1, 0u, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
    return hipGetLastError();
}

// Streaming passes of calls with more chunks than this use non-temporal
// loads and stores: their g and e (6 to 8 bytes per element) outgrow the
// 256 MB last-level cache, which smaller sets keep between passes.
constexpr uint32_t kNtChunks = 8192;

// ------------------------------------------------------------- launchers
// d: device TDesc[T]; C: total chunks.  Return the first HIP error.
hipError_t launch_sign_compress(const TDesc* d, int T, uint32_t C, uint32_t max_chunks, bool any_empty,
                                bool any_f16, bool any_f32, uint32_t* bits, float* scale, const Ws& ws, int cus,
                                hipStream_t s);
// A DGC step folded into the compress passes: the velocity step runs
// inside the stream pass that forms v, the masking inside the pass that
// knows the selection (the top-k emit pass, the random-k stream pass).  The
// call's table d then holds u (as the fp32 gradient) and e; dg holds the
// step's gradients (same tensors, chunks and k); clip is the device
// clipping factor or NULL.
struct DgcFuse {
    const TDesc* dg;
    float m;
    const float* clip;
};
// dgc: NULL for a plain call.
hipError_t launch_topk(int kind, double ratio, uint64_t seed, const TDesc* d, int T, uint32_t C,
                       bool any_f16, bool any_f32, uint32_t* idx, float* val, const Ws& ws,
                       hipStream_t s, const DgcFuse* dgc = nullptr);
hipError_t launch_randk(uint64_t seed, const TDesc* d, int T, uint32_t C, uint64_t sum_k,
                        bool any_f16, bool any_f32, uint32_t* idx, float* val, const Ws& ws,
                        hipStream_t s, const DgcFuse* dgc = nullptr);
hipError_t launch_residual_update(int kind, const TDesc* d, int T, uint32_t C, bool any_f16,
                                  bool any_f32, const uint32_t* idx, const float* val,
                                  const uint32_t* bits, const float* scale, hipStream_t s);
// Sparse aggregate tile (elements per work unit) for a call whose tensors
// hold n_total elements and k_total entries per worker from W workers;
// *ring tells whether the ring-window kernel takes the call.
uint32_t sparse_agg_tile(uint64_t n_total, uint64_t k_total, int W, bool* ring);
// rp: null, or (ragged parts) per-worker part-offset arrays, then a dummy
// readable location, as device pointers [padded_workers(W) + 1].
hipError_t launch_aggregate_sparse(const ADesc* a, int T, uint32_t units, uint32_t tile, bool ring,
                                   const uint64_t* wp, int W, float alpha, int cus, const uint64_t* rp,
                                   hipStream_t s);
hipError_t launch_aggregate_sign(const ADesc* a, int T, uint32_t units, const uint64_t* wp, int W,
                                 float alpha, hipStream_t s);
// Stochastic b-bit quantizers (bits 2, 4 or 8).
hipError_t launch_quant_compress(int bits, uint64_t seed, const TDesc* d, int T, uint32_t C, uint32_t max_chunks,
                                 bool any_empty, bool any_f16, bool any_f32, uint32_t* words, float* scale,
                                 const Ws& ws, int cus, hipStream_t s);
hipError_t launch_quant_residual_update(int bits, const TDesc* d, int T, uint32_t C, const uint32_t* words,
                                        const float* scale, hipStream_t s);
// DGC local clipping: chunk sums of squares of the gradients of table d in
// part[C], the factor in factor[0] and, when given, factor_out[0].
hipError_t launch_dgc_clip(const TDesc* d, int T, uint32_t C, double clip, double* part, float* factor,
                           float* factor_out, hipStream_t s);
// units of kSignAggUnit elements; W <= 1024
// info, tabs: the TernGrad exact form's per-tensor forms and tables (2-bit only).
hipError_t launch_aggregate_quant(int bits, const ADesc* a, int T, uint32_t units, const uint64_t* wp, int W,
                                  float alpha, uint32_t* info, int32_t* tabs, hipStream_t s);

// Random-k bucketing: generating workgroups of kGenBlock threads handle
// kGenEntries payload entries each; a bucket is 2^S consecutive chunks with
// S the smallest shift giving at most kRandkBuckets buckets (S <= 8).  A
// call whose chunk count would need more than kRandkMaxBuckets buckets is
// refused.  randk_buckets returns false for such a call.
constexpr int kGenBlock = 1024;
constexpr int kGenPerThread = 32;
constexpr uint32_t kGenEntries = (uint32_t)kGenBlock * kGenPerThread;
constexpr uint32_t kRandkBuckets = 8192;
constexpr uint32_t kRandkMaxBuckets = 16384;
constexpr uint32_t kRandkMaxShift = 8;
bool randk_buckets(uint32_t C, uint32_t* S, uint32_t* NB);

// Divisible scheme: pack part j of one payload.  word_bits: 0 for the
// sparse kinds, else the code bits per element (1 sign, 2, 4, 8); words:
// the packed words (word kinds); max_entries: an upper bound on the part's
// entries (sparse), which sizes the copy grid.
hipError_t launch_pack_part(int word_bits, const PDesc* p, int T, bc_payload_dev in, bc_payload_dev out,
                            uint64_t* part_off, uint64_t words, uint64_t max_entries, int cus, hipStream_t s);

// Work-unit sizes of the aggregate kernels (elements per unit).

constexpr uint32_t kSignAggUnit = 4096;  // one workgroup: 16 elements per lane

}  // namespace bc
