// api.hip -- the C ABI (include/bytecomp.h): argument validation, payload
// layout, workspace planning, the per-device descriptor cache, and the
// launch sequences of the gfx950 kernels.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <atomic>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/bytecomp.h"
#include "launch.hpp"

#include <rocprofiler-sdk-roctx/roctx.h>

namespace bc {

namespace {

constexpr int kMaxT = 1 << 20;
constexpr int kMaxW = 1024;
constexpr uint64_t kMaxN = (1ull << 32) - 65536;  // uint32 indices, chunk arithmetic headroom

bool debug_mode() {
    static int mode = -1;
    if (mode < 0) {
        const char* e = std::getenv("BYTECOMP_DEBUG");
        mode = (e && e[0] == '1') ? 1 : 0;
    }
    return mode == 1;
}

uint64_t ratio_ppm(double ratio) {
    if (!(ratio > 0.0) || ratio > 1.0) return 0;
    return (uint64_t)std::llround(ratio * 1e6);
}

uint64_t k_of(uint64_t n, uint64_t ppm) {
    if (n == 0) return 0;
    uint64_t k = (n * ppm + 999999u) / 1000000u;
    if (k < 1) k = 1;
    if (k > n) k = n;
    return k;
}

uint64_t words_of(uint64_t n) { return (n + 31u) / 32u; }

bool is_sparse(int kind) { return kind == BC_TOPK || kind == BC_TOPK_SAMPLED || kind == BC_RANDK; }

// Bits per element of the stochastic quantizers (0 for the other kinds).
int quant_bits(int kind) {
    return kind == BC_TERNGRAD ? 2 : kind == BC_QSGD4 ? 4 : kind == BC_QSGD8 ? 8 : 0;
}

// Payload entries (sparse kinds) or 32-bit words (sign, quantizers) of a
// tensor of n elements.
uint64_t count_of(int kind, uint64_t n, uint64_t ppm) {
    if (is_sparse(kind)) return k_of(n, ppm);
    if (const int b = quant_bits(kind)) return (n * (uint64_t)b + 31u) / 32u;
    return words_of(n);
}

size_t align256(size_t x) { return (x + 255u) & ~(size_t)255u; }

// ----------------------------------------------------- descriptor cache
// Device copies of descriptor tables, keyed by their exact bytes and the
// device; a hit costs no copy.  Entries are uploaded from pinned host
// memory on the calling stream; other streams wait on the upload event.
struct Entry {
    int device = -1;
    std::vector<unsigned char> key;
    void* dev = nullptr;
    void* pinned = nullptr;
    size_t cap = 0;
    hipStream_t upload_stream = nullptr;
    hipEvent_t ready = nullptr;
    hipEvent_t used = nullptr;
    hipStream_t last_stream = nullptr;
    bool multi_stream = false;
    uint64_t tick = 0;
};

std::mutex g_mu;
Entry g_cache[32];
uint64_t g_tick = 0;

// The device copy holds the key bytes followed by `extra` bytes derived
// from them (the chunk- or unit-to-tensor maps), built only on a miss.
template <typename Fill>
hipError_t cache_get(const void* bytes, size_t len, size_t extra, Fill fill, hipStream_t s, Entry** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    Entry* victim = nullptr;
    for (Entry& en : g_cache) {
        if (en.device == dev && en.key.size() == len && std::memcmp(en.key.data(), bytes, len) == 0) {
            if (en.upload_stream != s) {
                e = hipStreamWaitEvent(s, en.ready, 0);
                if (e != hipSuccess) return e;
            }
            en.tick = ++g_tick;
            *out = &en;
            return hipSuccess;
        }
        if (!victim || en.tick < victim->tick) victim = &en;
    }
    Entry& en = *victim;
    if (en.device >= 0) {
        // make sure no queued kernel still reads the old table
        if (en.multi_stream) {
            e = hipDeviceSynchronize();
        } else if (en.used) {
            e = hipEventSynchronize(en.used);
        }
        if (e != hipSuccess) return e;
    }
    const size_t total = len + extra;
    if (en.device != dev || en.cap < total) {
        if (en.dev) (void)hipFree(en.dev);
        if (en.pinned) (void)hipHostFree(en.pinned);
        if (en.ready) (void)hipEventDestroy(en.ready);
        if (en.used) (void)hipEventDestroy(en.used);
        en = Entry();
        size_t cap = total < 4096 ? 4096 : total;
        if ((e = hipMalloc(&en.dev, cap)) != hipSuccess) { en = Entry(); return e; }
        if ((e = hipHostMalloc(&en.pinned, cap, hipHostMallocDefault)) != hipSuccess) {
            (void)hipFree(en.dev);
            en = Entry();
            return e;
        }
        (void)hipEventCreateWithFlags(&en.ready, hipEventDisableTiming);
        (void)hipEventCreateWithFlags(&en.used, hipEventDisableTiming);
        en.cap = cap;
        en.device = dev;
    }
    std::memcpy(en.pinned, bytes, len);
    fill((unsigned char*)en.pinned + len);
    en.key.assign((const unsigned char*)bytes, (const unsigned char*)bytes + len);
    e = hipMemcpyAsync(en.dev, en.pinned, total, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipEventRecord(en.ready, s);
    if (e != hipSuccess) { en.key.clear(); return e; }
    en.upload_stream = s;
    en.last_stream = s;
    en.multi_stream = false;
    en.tick = ++g_tick;
    *out = &en;
    return hipSuccess;
}

void cache_mark_used(Entry* en, hipStream_t s) {
    if (en->last_stream != s) en->multi_stream = true;
    en->last_stream = s;
    (void)hipEventRecord(en->used, s);
}

// ------------------------------------------------------------ device info
std::mutex g_dev_mu;
DevInfo g_dev[64];
bool g_dev_ok[64];

}  // namespace


hipError_t device_info(int dev, DevInfo* out) {
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    if (!g_dev_ok[dev]) {
        hipDeviceProp_t p;
        hipError_t e = hipGetDeviceProperties(&p, dev);
        if (e != hipSuccess) return e;
        DevInfo di;
        di.cus = p.multiProcessorCount;
        di.any_empty = false;
        int khz = 0;
        if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) khz = 0;
        di.wall_khz = khz;
        g_dev[dev] = di;
        g_dev_ok[dev] = true;
    }
    *out = g_dev[dev];
    return hipSuccess;
}

// ------------------------------------------------------- kernel timing
namespace {
std::mutex g_timer_mu;
std::atomic<int> g_timer_kernel{kTimedNone};
hipEvent_t g_timer_start = nullptr, g_timer_stop = nullptr;

// Sets (or clears, k = kTimedNone) the request; returns whether a request
// was pending (set and not yet taken by a launch).
bool set_kernel_timer(int k, hipEvent_t start, hipEvent_t stop) {
    std::lock_guard<std::mutex> lk(g_timer_mu);
    const bool pending = g_timer_kernel.load(std::memory_order_relaxed) != kTimedNone;
    g_timer_start = start;
    g_timer_stop = stop;
    g_timer_kernel.store(k, std::memory_order_release);
    return pending;
}
}  // namespace

CallRange::CallRange(const char* name) { roctxRangePushA(name); }
CallRange::~CallRange() { roctxRangePop(); }

// ------------------------------------------------- one-pass wait limit
namespace {
std::atomic<uint32_t> g_wait_us{200};
std::atomic<uint32_t> g_topk_few{kTopkFewChunksMax};
}  // namespace

uint32_t topk_few_chunks_limit() { return g_topk_few.load(std::memory_order_relaxed); }

uint32_t onepass_wait_ticks() {
    int dev = 0;
    DevInfo di;
    uint64_t khz = 100000;  // the usual rate of the counter, if the query fails
    if (hipGetDevice(&dev) == hipSuccess && device_info(dev, &di) == hipSuccess && di.wall_khz > 0)
        khz = (uint64_t)di.wall_khz;
    const uint64_t t = (uint64_t)g_wait_us.load(std::memory_order_relaxed) * khz / 1000u;
    return t > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)t;
}

bool take_kernel_timer(int k, hipEvent_t* start, hipEvent_t* stop) {
    if (g_timer_kernel.load(std::memory_order_acquire) != k) return false;
    std::lock_guard<std::mutex> lk(g_timer_mu);
    if (g_timer_kernel.load(std::memory_order_relaxed) != k) return false;
    *start = g_timer_start;
    *stop = g_timer_stop;
    g_timer_kernel.store(kTimedNone, std::memory_order_relaxed);
    return true;
}

// -------------------------------------------------------------- workspace
WsPlan plan_workspace(int kind, int T, uint64_t C, uint64_t sum_k, bool agg_tables) {
    WsPlan p;
    std::memset(&p, 0, sizeof(p));
    size_t at = 256;  // header
    auto take = [&](size_t& field, size_t bytes) {
        field = bytes ? at : 0;
        at = align256(at + bytes);
    };
    const size_t t = (size_t)T;
    if (kind == BC_SIGN1) {
        take(p.s_val, t * 4);
        take(p.s_partial, (size_t)C * 8);
        take(p.s_slot, (size_t)C * 8);
    } else if (quant_bits(kind)) {
        take(p.s_val, t * 4);
        take(p.q_max, (size_t)C * 4);
        take(p.q_slot, (size_t)C * 4);
        if (kind == BC_TERNGRAD && agg_tables) {
            take(p.s_info, t * 4);
            take(p.s_tab, t * 4096 * 4);
        }
    } else if (kind == BC_TOPK || kind == BC_TOPK_SAMPLED) {
        // the general pipeline: copies of one histogram per tensor; the
        // few-chunk path: up to 4 copies of digit 0, then digits 1 and 2
        {
            size_t per = (size_t)topk_general_copies(T) * kBins0;
            if (C <= kTopkFewChunksMax && per < 4 * kBins0 + 2 * kBins12) per = 4 * kBins0 + 2 * kBins12;
            take(p.t_hist, t * per * 4);
        }
        take(p.t_thr, t * 4);
        take(p.t_prefix, t * 4);
        take(p.t_krem, t * 4);
        take(p.t_fb, t * 4);
        take(p.t_any, 4);
        take(p.t_cand, (size_t)C * kChunk * 8);
        take(p.t_ccount, (size_t)C * 4);
        take(p.t_gt, (size_t)C * 4);
        take(p.t_eq, (size_t)C * 4);
        take(p.t_off, (size_t)C * 8);
        take(p.t_eqb, (size_t)C * 4);
    } else if (kind == BC_RANDK) {
        uint32_t S = 0, NB = 0;
        randk_buckets((uint32_t)(C < 0xFFFFFFFFull ? C : 0xFFFFFFFFull), &S, &NB);
        const size_t nscan = ((size_t)NB + kBlock * 16 - 1) / (kBlock * 16);
        const size_t nblk = (size_t)((sum_k + kGenEntries - 1) / kGenEntries);
        take(p.r_keys, t * 16);
        take(p.r_tmp, (size_t)sum_k * 4);
        take(p.r_ccount, (size_t)NB * 4);
        take(p.r_coff, ((size_t)NB + 1 + nscan) * 8);
        take(p.r_hist, nblk * NB * 4);
    }
    if (kind == BC_TOPK || kind == BC_TOPK_SAMPLED || kind == BC_RANDK) {
        take(p.d_part, (size_t)C * 8);
        take(p.d_factor, 4);
    }
    p.total = at;
    return p;
}

Ws carve_workspace(void* base, const WsPlan& p) {
    char* b = (char*)base;
    auto at = [&](size_t off) -> void* { return off ? (void*)(b + off) : nullptr; };
    Ws w;
    std::memset(&w, 0, sizeof(w));
    w.flags = (uint32_t*)b;
    w.s_val = (float*)at(p.s_val);
    w.s_partial = (double*)at(p.s_partial);
    w.s_info = (uint32_t*)at(p.s_info);
    w.s_tab = (int32_t*)at(p.s_tab);
    w.s_slot = (uint64_t*)at(p.s_slot);
    w.q_max = (uint32_t*)at(p.q_max);
    w.q_slot = (uint32_t*)at(p.q_slot);
    w.t_hist = (uint32_t*)at(p.t_hist);
    w.t_thr = (uint32_t*)at(p.t_thr);
    w.t_prefix = (uint32_t*)at(p.t_prefix);
    w.t_krem = (uint32_t*)at(p.t_krem);
    w.t_fb = (uint32_t*)at(p.t_fb);
    w.t_any = (uint32_t*)at(p.t_any);
    w.t_cand = (uint2*)at(p.t_cand);
    w.t_ccount = (uint32_t*)at(p.t_ccount);
    w.t_gt = (uint32_t*)at(p.t_gt);
    w.t_eq = (uint32_t*)at(p.t_eq);
    w.t_off = (uint64_t*)at(p.t_off);
    w.t_eqb = (uint32_t*)at(p.t_eqb);
    w.r_keys = (uint32_t*)at(p.r_keys);
    w.r_tmp = (uint32_t*)at(p.r_tmp);
    w.r_ccount = (uint32_t*)at(p.r_ccount);
    w.r_coff = (uint64_t*)at(p.r_coff);
    w.r_hist = (uint32_t*)at(p.r_hist);
    w.d_part = (double*)at(p.d_part);
    w.d_factor = (float*)at(p.d_factor);
    return w;
}

hipError_t launch_zero_header(uint32_t* flags, hipStream_t s);

}  // namespace bc

using namespace bc;

namespace {

int hip_status(hipError_t e) { return e == hipSuccess ? BC_OK : BC_E_HIP; }

int finish(int rc, hipStream_t s, void* ws) {
    if (rc != BC_OK || !debug_mode()) return rc;
    if (hipStreamSynchronize(s) != hipSuccess) return BC_E_HIP;
    if (ws) {
        uint32_t f = 0;
        if (hipMemcpy(&f, ws, 4, hipMemcpyDeviceToHost) != hipSuccess) return BC_E_HIP;
        if (f) return BC_E_DEVICE;
    }
    return BC_OK;
}

// Validate a tensor list and build its descriptor table.
int build_tdesc(int kind, uint64_t ppm, const bc_tensor* t, int T, bool need_resid,
                std::vector<TDesc>& d, uint32_t& C, uint32_t& max_chunks, uint64_t& sum_k,
                bool& any16, bool& any32) {
    d.resize((size_t)T);
    uint64_t chunks = 0, off = 0;
    max_chunks = 0;
    any16 = any32 = false;
    for (int i = 0; i < T; ++i) {
        const bc_tensor& x = t[i];
        if (x.dtype != BC_F32 && x.dtype != BC_F16) return BC_E_DTYPE;
        if (x.n >= kMaxN) return BC_E_SIZE;
        if (x.n > 0 && !x.grad) return BC_E_NULL;
        if (need_resid && x.n > 0 && !x.residual) return BC_E_NULL;
        const uintptr_t ga = (uintptr_t)x.grad, ra = (uintptr_t)x.residual;
        if ((x.dtype == BC_F32 && (ga & 15u)) || (x.dtype == BC_F16 && (ga & 7u)) || (ra & 15u))
            return BC_E_ALIGN;
        const uint64_t nc = (x.n + kChunk - 1) / kChunk;
        TDesc& o = d[(size_t)i];
        o.grad = x.grad;
        o.resid = x.n ? x.residual : nullptr;
        o.n = (uint32_t)x.n;
        o.dtype = x.dtype;
        o.tid = x.tensor_id;
        const uint64_t cnt = count_of(kind, x.n, ppm);
        o.k = (uint32_t)cnt;
        o.off = off;
        o.chunk0 = (uint32_t)chunks;
        o.nchunks = (uint32_t)nc;
        off += cnt;
        chunks += nc;
        if (nc > max_chunks) max_chunks = (uint32_t)nc;
        if (x.n) (x.dtype == BC_F16 ? any16 : any32) = true;
    }
    if (chunks >= (1ull << 31)) return BC_E_SIZE;
    C = (uint32_t)chunks;
    sum_k = off;
    return BC_OK;
}

// chunk -> tensor map stored after the descriptor table
void fill_chunk_map(const std::vector<TDesc>& d, uint32_t* m) {
    for (size_t i = 0; i < d.size(); ++i)
        for (uint32_t q = 0; q < d[i].nchunks; ++q) m[d[i].chunk0 + q] = (uint32_t)i;
}

int check_kind_ratio(int kind, double ratio, uint64_t& ppm) {
    if (kind < BC_TOPK || kind > BC_QSGD8) return BC_E_KIND;
    ppm = 1;
    if (is_sparse(kind)) {
        ppm = ratio_ppm(ratio);
        if (ppm == 0) return BC_E_RATIO;
    }
    return BC_OK;
}

}  // namespace

namespace bc {

// Host-side checks and descriptor table of a compress call (everything
// before device memory is needed).  agg_tables: plan the workspace with the
// aggregate's regions (the size bytecomp_workspace_size reports) or
// without them (compress only).
int compress_prepare(int kind, double ratio, const bc_tensor* t, int T, const bc_payload& out, bool agg_tables,
                     CompressPrep& p) {
    int rc = check_kind_ratio(kind, ratio, p.ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!t) return BC_E_NULL;
    if (is_sparse(kind) ? (!out.idx || !out.val) : (!out.bits || !out.scale)) return BC_E_NULL;
    try {
        rc = build_tdesc(kind, p.ppm, t, T, false, p.d, p.C, p.maxc, p.sum_k, p.a16, p.a32);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    if (rc) return rc;
    // random-k: payload positions are 32-bit and the bucket count is bounded
    if (kind == BC_RANDK && (p.sum_k >= (1ull << 32) || !randk_buckets(p.C, nullptr, nullptr))) return BC_E_SIZE;
    p.any_empty = false;
    for (int i = 0; i < T && !p.any_empty; ++i) p.any_empty = t[i].n == 0;
    p.plan = plan_workspace(kind, T, p.C, p.sum_k, agg_tables);
    return BC_OK;
}

// The kind's compress kernels, on descriptor table dd (device) and carved
// workspace w.
hipError_t compress_launch(int kind, double ratio, uint64_t seed, const CompressPrep& p, const TDesc* dd,
                           const bc_payload& out, const Ws& w, hipStream_t s) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    DevInfo di;
    if ((e = device_info(dev, &di)) != hipSuccess) return e;
    const int T = (int)p.d.size();
    switch (kind) {
        case BC_SIGN1:
            return launch_sign_compress(dd, T, p.C, p.maxc, p.any_empty, p.a16, p.a32, out.bits, out.scale, w,
                                        di.cus, s);
        case BC_TOPK:
        case BC_TOPK_SAMPLED:
            return launch_topk(kind == BC_TOPK ? 0 : 1, ratio, seed, dd, T, p.C, p.a16, p.a32, out.idx, out.val, w,
                               s);
        case BC_TERNGRAD:
        case BC_QSGD4:
        case BC_QSGD8:
            return launch_quant_compress(quant_bits(kind), seed, dd, T, p.C, p.maxc, p.any_empty, p.a16, p.a32,
                                         out.bits, out.scale, w, di.cus, s);
        default:
            return launch_randk(seed, dd, T, p.C, p.sum_k, p.a16, p.a32, out.idx, out.val, w, s);
    }
}

}  // namespace bc

namespace {
// One DGC step (bytecomp_compress_dgc, bytecomp_compress_dgc_clip).
int compress_dgc_impl(int kind, double ratio, uint64_t seed, float momentum, bool clipping, double clip_norm,
                      float* clip_factor, const bc_tensor* t, float* const* velocity, int T, bc_payload out,
                      void* ws, size_t ws_bytes, void* stream);
}  // namespace

extern "C" {

const char* bytecomp_strerror(int status) {
    switch (status) {
        case BC_OK: return "ok";
        case BC_E_NULL: return "a required pointer is NULL";
        case BC_E_KIND: return "unknown compression kind";
        case BC_E_DTYPE: return "unknown gradient dtype";
        case BC_E_RATIO: return "ratio outside (0, 1] or below one part per million";
        case BC_E_SIZE: return "tensor or call too large";
        case BC_E_COUNT: return "invalid tensor or worker count";
        case BC_E_WORKSPACE: return "workspace missing or too small";
        case BC_E_HIP: return "HIP runtime error";
        case BC_E_ALIGN: return "dense buffer not aligned (fp32 and outputs 16 B, fp16 8 B)";
        case BC_E_DEVICE: return "a kernel reported a failure";
        default: return "unknown status";
    }
}

int bytecomp_layout(int kind, double ratio, const uint64_t* n, int T, uint64_t* off) {
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT) return BC_E_COUNT;
    if (!off || (T > 0 && !n)) return BC_E_NULL;
    off[0] = 0;
    for (int t = 0; t < T; ++t) {
        if (n[t] >= kMaxN) return BC_E_SIZE;
        off[t + 1] = off[t] + count_of(kind, n[t], ppm);
    }
    return BC_OK;
}

int bytecomp_workspace_size(int kind, double ratio, const uint64_t* n, int T, int W, size_t* bytes) {
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT || W < 1 || W > kMaxW) return BC_E_COUNT;
    if (!bytes || (T > 0 && !n)) return BC_E_NULL;
    uint64_t C = 0, sk = 0;
    for (int t = 0; t < T; ++t) {
        if (n[t] >= kMaxN) return BC_E_SIZE;
        C += (n[t] + kChunk - 1) / kChunk;
        sk += is_sparse(kind) ? k_of(n[t], ppm) : 0;
    }
    *bytes = plan_workspace(kind, T, C, sk).total;
    return BC_OK;
}

int bytecomp_workspace_init(void* ws, size_t ws_bytes, void* stream) {
    if (!ws) return BC_E_NULL;
    if (ws_bytes < 256) return BC_E_WORKSPACE;
    return hip_status(launch_zero_header((uint32_t*)ws, (hipStream_t)stream));
}

int bytecomp_compress(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                      bc_payload out, void* ws, size_t ws_bytes, void* stream) {
    const CallRange range("bytecomp_compress");
    CompressPrep p;
    int rc = compress_prepare(kind, ratio, t, T, out, true, p);
    if (rc || T == 0) return rc;
    if (!ws) return BC_E_WORKSPACE;
    if (ws_bytes < p.plan.total) return BC_E_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    std::lock_guard<std::mutex> lk(g_mu);
    Entry* en = nullptr;
    hipError_t e = cache_get(p.d.data(), p.d.size() * sizeof(TDesc), (size_t)p.C * 4,
                             [&](void* dst) { fill_chunk_map(p.d, (uint32_t*)dst); }, s, &en);
    if (e != hipSuccess) return BC_E_HIP;
    e = compress_launch(kind, ratio, seed, p, (const TDesc*)en->dev, out, carve_workspace(ws, p.plan), s);
    cache_mark_used(en, s);
    return finish(hip_status(e), s, ws);
}

int bytecomp_compress_dgc(int kind, double ratio, uint64_t seed, float momentum, const bc_tensor* t,
                          float* const* velocity, int T, bc_payload out, void* ws, size_t ws_bytes, void* stream) {
    const CallRange range("bytecomp_compress_dgc");
    return compress_dgc_impl(kind, ratio, seed, momentum, false, 0.0, nullptr, t, velocity, T, out, ws, ws_bytes,
                             stream);
}

int bytecomp_compress_dgc_clip(int kind, double ratio, uint64_t seed, float momentum, double clip_norm,
                               const bc_tensor* t, float* const* velocity, int T, bc_payload out,
                               float* clip_factor, void* ws, size_t ws_bytes, void* stream) {
    const CallRange range("bytecomp_compress_dgc_clip");
    if (!(clip_norm >= 0.0)) return BC_E_RATIO;  // NaN or negative
    return compress_dgc_impl(kind, ratio, seed, momentum, true, clip_norm, clip_factor, t, velocity, T, out, ws,
                             ws_bytes, stream);
}

}  // extern "C"

namespace {

int compress_dgc_impl(int kind, double ratio, uint64_t seed, float momentum, bool clipping, double clip_norm,
                      float* clip_factor, const bc_tensor* t, float* const* velocity, int T, bc_payload out,
                      void* ws, size_t ws_bytes, void* stream) {
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (!is_sparse(kind)) return BC_E_KIND;
    if (T < 0 || T > kMaxT) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!t || !velocity || !out.idx || !out.val) return BC_E_NULL;
    if (!ws) return BC_E_WORKSPACE;
    std::vector<bc_tensor> tv, tc;
    std::vector<TDesc> dm, dc;
    uint32_t C, maxc, C2, maxc2;
    uint64_t sum_k, sum_k2;
    bool a16, a32, b16, b32;
    try {
        tv.resize((size_t)T);
        tc.resize((size_t)T);
        for (int i = 0; i < T; ++i) {
            if (t[i].n > 0 && (!velocity[i] || !t[i].residual)) return BC_E_NULL;
            tv[(size_t)i] = t[i];  // dm: the gradients (u in the residual's place, checked like one)
            tv[(size_t)i].residual = velocity[i];
            tc[(size_t)i] = bc_tensor{velocity[i], t[i].residual, t[i].n, BC_F32, t[i].tensor_id};
        }
        // every argument is checked before anything is enqueued
        rc = build_tdesc(kind, ppm, tv.data(), T, true, dm, C, maxc, sum_k, a16, a32);
        if (rc == BC_OK) rc = build_tdesc(kind, ppm, tc.data(), T, true, dc, C2, maxc2, sum_k2, b16, b32);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    if (rc) return rc;
    if (kind == BC_RANDK && (sum_k >= (1ull << 32) || !randk_buckets(C, nullptr, nullptr))) return BC_E_SIZE;
    const WsPlan plan = plan_workspace(kind, T, C, sum_k);
    if (ws_bytes < plan.total) return BC_E_WORKSPACE;
    const Ws w = carve_workspace(ws, plan);
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    // the velocity step and the masking inside the compress passes: dc (u
    // in the gradient's place, e) drives them, dm supplies g
    std::lock_guard<std::mutex> lk(g_mu);
    Entry* em = nullptr;
    Entry* ec = nullptr;
    e = cache_get(dm.data(), dm.size() * sizeof(TDesc), (size_t)C * 4,
                  [&](void* dst) { fill_chunk_map(dm, (uint32_t*)dst); }, s, &em);
    if (e != hipSuccess) return BC_E_HIP;
    if (clipping) {
        e = launch_dgc_clip((const TDesc*)em->dev, T, C, clip_norm, w.d_part, w.d_factor, clip_factor, s);
        if (e != hipSuccess) {
            cache_mark_used(em, s);
            return BC_E_HIP;
        }
    }
    // the newest entry is never the one a miss replaces, so em stays valid
    e = cache_get(dc.data(), dc.size() * sizeof(TDesc), (size_t)C2 * 4,
                  [&](void* dst) { fill_chunk_map(dc, (uint32_t*)dst); }, s, &ec);
    if (e != hipSuccess) {
        cache_mark_used(em, s);
        return BC_E_HIP;
    }
    const DgcFuse f{(const TDesc*)em->dev, momentum, clipping ? w.d_factor : nullptr};
    if (kind == BC_RANDK)
        e = launch_randk(seed, (const TDesc*)ec->dev, T, C2, sum_k2, b16, b32, out.idx, out.val, w, s, &f);
    else
        e = launch_topk(kind == BC_TOPK ? 0 : 1, ratio, seed, (const TDesc*)ec->dev, T, C2, b16, b32, out.idx,
                        out.val, w, s, &f);
    cache_mark_used(em, s);
    cache_mark_used(ec, s);
    return finish(hip_status(e), s, ws);
}

}  // namespace

namespace {

// Decompress-and-aggregate.  part_off == nullptr: W whole payloads in the
// bytecomp_layout layout.  Otherwise (sparse kinds, W <= 64): W packed
// parts, worker w's entries of tensor t at part_off[w][t] ..
// part_off[w][t+1] (device arrays), indices relative to the tensor.
int aggregate_impl(int kind, double ratio, const bc_payload* in, const uint64_t* const* part_off, int W,
                   const uint64_t* n, int T, float* const* out, float alpha, void* ws, size_t ws_bytes,
                   void* stream) {
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT || W < 1 || W > kMaxW) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!in || !n || !out) return BC_E_NULL;
    if (!ws) return BC_E_WORKSPACE;
    if (ws_bytes < 256) return BC_E_WORKSPACE;
    const bool sparse = is_sparse(kind);
    const bool ragged = part_off != nullptr;
    if (ragged) {
        if (!sparse) return BC_E_KIND;
        if (W > 64) return BC_E_COUNT;
        for (int q = 0; q < W; ++q)
            if (!part_off[q]) return BC_E_NULL;
    }
    // ragged parts: [dummy-padded part-offset pointers][ADesc...][workers...]
    const size_t rp_bytes = ragged ? align256((size_t)(padded_workers(W) + 1) * sizeof(uint64_t)) : 0;
    uint32_t unit = kSignAggUnit;
    bool ring = false;
    if (sparse) {
        uint64_t nt = 0, kt = 0;
        for (int i = 0; i < T; ++i) {
            if (n[i] >= kMaxN) return BC_E_SIZE;
            nt += n[i];
            kt += k_of(n[i], ppm);
        }
        unit = sparse_agg_tile(nt, kt, W, &ring);
    }
    std::vector<unsigned char> table;
    try {
        table.resize(rp_bytes + (size_t)T * sizeof(ADesc) + (size_t)2 * padded_workers(W) * sizeof(uint64_t));
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    if (ragged) {
        uint64_t* rp = (uint64_t*)table.data();
        for (int q = 0; q < padded_workers(W); ++q) rp[q] = (uint64_t)(uintptr_t)part_off[q < W ? q : W - 1];
        rp[padded_workers(W)] = (uint64_t)(uintptr_t)ws;  // a readable dummy location
    }
    ADesc* a = (ADesc*)(table.data() + rp_bytes);
    uint64_t* wa = (uint64_t*)(table.data() + rp_bytes + (size_t)T * sizeof(ADesc));
    uint64_t* wb = wa + padded_workers(W);
    uint64_t units = 0, off = 0;
    // sign: a tensor's units start on 128-byte lines of the payloads (worker
    // 0's address decides; the kernel derives the same shift)
    const uint64_t sign_base = kind == BC_SIGN1 && in && in[0].bits ? (uint64_t)(uintptr_t)in[0].bits >> 2 : 0;
    for (int i = 0; i < T; ++i) {
        if (n[i] >= kMaxN) return BC_E_SIZE;
        if (n[i] > 0 && !out[i]) return BC_E_NULL;
        if ((uintptr_t)out[i] & 15u) return BC_E_ALIGN;
        const uint64_t cnt = count_of(kind, n[i], ppm);
        uint64_t nu = (n[i] + unit - 1) / unit;
        if (kind == BC_SIGN1 && cnt) nu = (cnt + ((sign_base + off) & 31u) + kSignAggUnit / 32 - 1) / (kSignAggUnit / 32);
        a[i].out = out[i];
        a[i].n = (uint32_t)n[i];
        a[i].k = (uint32_t)cnt;
        a[i].off = off;
        a[i].unit0 = (uint32_t)units;
        a[i].nunits = (uint32_t)nu;
        off += cnt;
        units += nu;
    }
    if (units >= (1ull << 31)) return BC_E_SIZE;
    if (ragged) {
        for (int i = 0; i < T; ++i) a[i].k = 0;  // per-worker counts come from the parts
        off = 1;                                 // payloads are not addressed by layout
    }
    Ws w{};  // TernGrad: per-tensor forms and lookup tables live in the workspace
    if (kind == BC_TERNGRAD) {
        uint64_t C = 0;
        for (int i = 0; i < T; ++i) C += (n[i] + kChunk - 1) / kChunk;
        const WsPlan plan = plan_workspace(kind, T, C, 0);
        if (ws_bytes < plan.total) return BC_E_WORKSPACE;
        w = carve_workspace(ws, plan);
    }
    // the sign kernel addresses a worker's words with a 32-bit byte offset
    if (!sparse && off >= (1ull << 30)) return BC_E_SIZE;
    for (int q = 0; q < W; ++q) {
        if (sparse) {
            if (off && (!in[q].idx || !in[q].val)) return BC_E_NULL;
            wa[q] = (uint64_t)(uintptr_t)in[q].idx;
            wb[q] = (uint64_t)(uintptr_t)in[q].val;
        } else {
            if (!in[q].bits || !in[q].scale) return BC_E_NULL;
            wa[q] = (uint64_t)(uintptr_t)in[q].bits;
            wb[q] = (uint64_t)(uintptr_t)in[q].scale;
        }
    }
    // descriptors W .. padded_workers(W)-1 repeat the last worker, so that
    // kernels may read worker descriptors sixteen at a time
    for (int q = W; q < padded_workers(W); ++q) {
        wa[q] = wa[W - 1];
        wb[q] = wb[W - 1];
    }
    hipStream_t s = (hipStream_t)stream;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BC_E_HIP;
    DevInfo di;
    if (device_info(dev, &di) != hipSuccess) return BC_E_HIP;
    std::lock_guard<std::mutex> lk(g_mu);
    Entry* en = nullptr;
    hipError_t e = cache_get(table.data(), table.size(), (size_t)units * 4,
                             [&](void* dst) {
                                 uint32_t* m = (uint32_t*)dst;
                                 for (int i = 0; i < T; ++i)
                                     for (uint32_t q = 0; q < a[i].nunits; ++q) m[a[i].unit0 + q] = (uint32_t)i;
                             },
                             s, &en);
    if (e != hipSuccess) return BC_E_HIP;
    const uint64_t* rpd = ragged ? (const uint64_t*)en->dev : nullptr;
    const ADesc* ad = (const ADesc*)((const char*)en->dev + rp_bytes);
    const uint64_t* wdd = (const uint64_t*)((const char*)en->dev + rp_bytes + (size_t)T * sizeof(ADesc));
    if (sparse) {
        e = launch_aggregate_sparse(ad, T, (uint32_t)units, unit, ring, wdd, W, alpha, di.cus, rpd, s);
    } else if (quant_bits(kind)) {
        e = launch_aggregate_quant(quant_bits(kind), ad, T, (uint32_t)units, wdd, W, alpha, w.s_info, w.s_tab, s);
    } else {
        e = launch_aggregate_sign(ad, T, (uint32_t)units, wdd, W, alpha, s);
    }
    cache_mark_used(en, s);
    return finish(hip_status(e), s, ws);
}

}  // namespace

extern "C" {

int bytecomp_decompress_aggregate(int kind, double ratio, const bc_payload* in, int W,
                                  const uint64_t* n, int T, float* const* out, float alpha,
                                  void* ws, size_t ws_bytes, void* stream) {
    const CallRange range("bytecomp_decompress_aggregate");
    return aggregate_impl(kind, ratio, in, nullptr, W, n, T, out, alpha, ws, ws_bytes, stream);
}

int bytecomp_aggregate_part(int kind, double ratio, const bc_payload* in, const uint64_t* const* part_off,
                            int W, const uint64_t* len, int T, float* const* out, float alpha, void* ws,
                            size_t ws_bytes, void* stream) {
    const CallRange range("bytecomp_aggregate_part");
    if (!is_sparse(kind))  // packed sign and quantizer parts have the word layout of the range lengths
        return aggregate_impl(kind, ratio, in, nullptr, W, len, T, out, alpha, ws, ws_bytes, stream);
    if (!part_off) return BC_E_NULL;
    return aggregate_impl(kind, ratio, in, part_off, W, len, T, out, alpha, ws, ws_bytes, stream);
}

int bytecomp_pack_part(int kind, double ratio, const uint64_t* n, int T, bc_payload in, int parts,
                       const uint64_t* bounds, int j, bc_payload out, uint64_t* part_off, void* stream) {
    const CallRange range("bytecomp_pack_part");
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT || parts < 1 || j < 0 || j >= parts) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!n || !bounds || !part_off) return BC_E_NULL;
    const bool sparse = is_sparse(kind);
    if (sparse ? (!in.idx || !in.val || !out.idx || !out.val) : (!in.bits || !in.scale || !out.bits || !out.scale))
        return BC_E_NULL;
    std::vector<PDesc> p;
    try {
        p.resize((size_t)T);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    uint64_t in_off = 0, out_words = 0, max_entries = 0;
    for (int t = 0; t < T; ++t) {
        if (n[t] >= kMaxN) return BC_E_SIZE;
        const uint64_t* b = bounds + (size_t)t * (parts + 1);
        if (b[0] != 0 || b[parts] != n[t]) return BC_E_SIZE;
        for (int q = 0; q < parts; ++q) {
            if (b[q] > b[q + 1]) return BC_E_SIZE;
            if (q > 0 && (b[q] & 31u)) return BC_E_ALIGN;
        }
        const uint64_t cnt = count_of(kind, n[t], ppm);
        PDesc& d = p[(size_t)t];
        d.in_off = in_off;
        d.out_off = out_words;
        d.k = (uint32_t)cnt;
        d.lo = (uint32_t)b[j];
        d.hi = (uint32_t)b[j + 1];
        d.pad = 0;
        in_off += cnt;
        out_words += count_of(kind, b[j + 1] - b[j], ppm);  // words of the range (word kinds)
        max_entries += cnt < b[j + 1] - b[j] ? cnt : b[j + 1] - b[j];
    }
    hipStream_t s = (hipStream_t)stream;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BC_E_HIP;
    DevInfo di;
    if (device_info(dev, &di) != hipSuccess) return BC_E_HIP;
    std::lock_guard<std::mutex> lk(g_mu);
    Entry* en = nullptr;
    hipError_t e = cache_get(p.data(), p.size() * sizeof(PDesc), 0, [](void*) {}, s, &en);
    if (e != hipSuccess) return BC_E_HIP;
    const bc_payload_dev din{in.idx, in.val, in.bits, in.scale};
    const bc_payload_dev dout{out.idx, out.val, out.bits, out.scale};
    e = launch_pack_part(sparse ? 0 : quant_bits(kind) ? quant_bits(kind) : 1, (const PDesc*)en->dev, T, din, dout,
                         part_off, out_words, max_entries, di.cus, s);
    cache_mark_used(en, s);
    return hip_status(e);
}

int bytecomp_residual_update(int kind, double ratio, const bc_tensor* t, int T, bc_payload own,
                             void* stream) {
    const CallRange range("bytecomp_residual_update");
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (T < 0 || T > kMaxT) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!t) return BC_E_NULL;
    if (is_sparse(kind) ? (!own.idx || !own.val) : (!own.bits || !own.scale)) return BC_E_NULL;
    std::vector<TDesc> d;
    uint32_t C, maxc;
    uint64_t sum_k;
    bool a16, a32;
    try {
        rc = build_tdesc(kind, ppm, t, T, true, d, C, maxc, sum_k, a16, a32);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    std::lock_guard<std::mutex> lk(g_mu);
    Entry* en = nullptr;
    hipError_t e = cache_get(d.data(), d.size() * sizeof(TDesc), (size_t)C * 4,
                             [&](void* dst) { fill_chunk_map(d, (uint32_t*)dst); }, s, &en);
    if (e != hipSuccess) return BC_E_HIP;
    if (quant_bits(kind))
        e = launch_quant_residual_update(quant_bits(kind), (const TDesc*)en->dev, T, C, own.bits, own.scale, s);
    else
        e = launch_residual_update(kind, (const TDesc*)en->dev, T, C, a16, a32, own.idx, own.val, own.bits,
                                   own.scale, s);
    cache_mark_used(en, s);
    return finish(hip_status(e), s, nullptr);
}

int bytecomp_time_next_launch(const char* kernel, void* start_event, void* stop_event) {
    if (!start_event && !stop_event) return set_kernel_timer(kTimedNone, nullptr, nullptr) ? 1 : BC_OK;
    if (!kernel || !start_event || !stop_event) return BC_E_NULL;
    static const struct { const char* name; int k; } names[] = {
        {"aggregate_sign", kTimedAggSign},       {"aggregate_sparse", kTimedAggSparse},
        {"randk_stream", kTimedRandkStream},     {"topk_compact", kTimedTopkCompact},
        {"sign_pass1", kTimedSignPass1},         {"quant_pass1", kTimedQuantPass1},
        {"aggregate_quant", kTimedAggQuant},     {"sign_onepass", kTimedSignOnepass},
        {"quant_onepass", kTimedQuantOnepass},   {"topk_hist", kTimedTopkHist}};
    for (const auto& x : names) {
        if (std::strcmp(kernel, x.name) == 0) {
            (void)set_kernel_timer(x.k, (hipEvent_t)start_event, (hipEvent_t)stop_event);
            return BC_OK;
        }
    }
    return BC_E_KIND;
}

int bytecomp_set_wait_limit(uint32_t microseconds) {
    if (microseconds > 10000000u) return BC_E_SIZE;
    g_wait_us.store(microseconds, std::memory_order_relaxed);
    return BC_OK;
}

int bytecomp_set_topk_few_chunks(uint32_t chunks) {
    if (chunks > kTopkFewChunksMax) return BC_E_SIZE;
    g_topk_few.store(chunks, std::memory_order_relaxed);
    return BC_OK;
}

int bytecomp_topk_stats(int kind, double ratio, const uint64_t* n, int T, const void* ws, size_t ws_bytes,
                        void* stream, uint64_t* candidates, uint32_t* fallbacks) {
    uint64_t ppm;
    int rc = check_kind_ratio(kind, ratio, ppm);
    if (rc) return rc;
    if (kind != BC_TOPK && kind != BC_TOPK_SAMPLED) return BC_E_KIND;
    if (T < 0 || T > kMaxT) return BC_E_COUNT;
    if (!candidates || !fallbacks || (T > 0 && !n)) return BC_E_NULL;
    *candidates = 0;
    *fallbacks = 0;
    uint64_t C = 0, sk = 0;
    for (int t = 0; t < T; ++t) {
        if (n[t] >= kMaxN) return BC_E_SIZE;
        C += (n[t] + kChunk - 1) / kChunk;
        sk += k_of(n[t], ppm);
    }
    if (C == 0) return BC_OK;
    if (!ws) return BC_E_NULL;
    const WsPlan plan = plan_workspace(kind, T, C, sk);
    if (ws_bytes < plan.total) return BC_E_WORKSPACE;
    std::vector<uint32_t> cc, fb;
    try {
        cc.resize((size_t)C);
        fb.resize((size_t)T);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    hipStream_t s = (hipStream_t)stream;
    const char* base = (const char*)ws;
    hipError_t e = hipMemcpyAsync(cc.data(), base + plan.t_ccount, (size_t)C * 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(fb.data(), base + plan.t_fb, (size_t)T * 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return BC_E_HIP;
    uint64_t cand = 0;
    for (uint32_t x : cc) cand += x;
    uint32_t nfb = 0;
    // the few-chunk path keeps another per-tensor value in t_fb
    if (kind == BC_TOPK_SAMPLED && C > topk_few_chunks_limit())
        for (uint32_t x : fb) nfb += x != 0u;
    *candidates = cand;
    *fallbacks = nfb;
    return BC_OK;
}

int bytecomp_device_status(void* ws, size_t ws_bytes, void* stream, uint32_t* flags) {
    if (!ws || !flags) return BC_E_NULL;
    if (ws_bytes < 256) return BC_E_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    uint32_t f = 0;
    hipError_t e = hipMemcpyAsync(&f, ws, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = launch_zero_header((uint32_t*)ws, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return BC_E_HIP;
    *flags = f;
    return BC_OK;
}

}  // extern "C"
