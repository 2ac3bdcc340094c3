// cpu_ops.hip -- the compression operators and their aggregates on the
// host CPU, multi-threaded (host code only; no kernel here).
//
// The paper offloads the compression of some tensors from the GPUs to the
// CPUs (Sec. 4.4.3, CPU offloading) and profiles every operation on both
// kinds of compute resource (Sec. 4.3, "Compression time").  These are the
// library's CPU operators for that: the same definitions and payload
// layouts as the GPU path (bytecomp_compress, bytecomp_decompress_aggregate),
// on host memory, so a payload compressed on either side aggregates on
// either side.  Work is split over std::thread workers by tensor and by
// element range.
//
// Results: sparse payloads, residuals and aggregates are identical to the
// GPU path's; a sign scale is the fp64 sum of |v| in range order, rounded
// once (the same value as the GPU's up to the order of the fp64 additions).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <thread>
#include <vector>

#include "../../include/bytecomp.h"
#include "exact_wide.hpp"
#include "launch.hpp"
#include "randk_perm.hpp"

namespace bc {
namespace {

uint32_t hbits(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return u;
}
float hfloat(uint32_t u) {
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}

// Reads v_i = widen(g_i) + e_i (e = 0 without a residual).  Copied into
// each task so that its pointers stay in registers across the task's
// stores.
struct VReader {
    const float* g32;
    const uint16_t* g16;
    const float* e;
    explicit VReader(const bc_tensor& t)
        : g32(t.dtype == BC_F32 ? static_cast<const float*>(t.grad) : nullptr),
          g16(t.dtype == BC_F32 ? nullptr : static_cast<const uint16_t*>(t.grad)),
          e(t.residual) {}
    float operator()(uint64_t i) const {
        const float g = g32 ? g32[i] : (float)__builtin_bit_cast(_Float16, g16[i]);
        return e ? g + e[i] : g;
    }
};

// Runs fn(task) for task = 0 .. tasks-1 on up to `threads` threads.
template <typename F>
void parallel_for(uint64_t tasks, int threads, F fn) {
    if (tasks == 0) return;
    const uint64_t nt = std::min<uint64_t>((uint64_t)(threads > 0 ? threads : 1), tasks);
    if (nt <= 1) {
        for (uint64_t q = 0; q < tasks; ++q) fn(q);
        return;
    }
    std::vector<std::thread> pool;
    pool.reserve(nt);
    for (uint64_t w = 0; w < nt; ++w)
        pool.emplace_back([&, w] {
            for (uint64_t q = w; q < tasks; q += nt) fn(q);
        });
    for (auto& th : pool) th.join();
}

constexpr uint64_t kRange = 1u << 16;  // elements per range task (a multiple of 32)

uint64_t k_rule(uint64_t n, uint64_t ppm) {
    if (n == 0) return 0;
    uint64_t k = (n * ppm + 999999u) / 1000000u;
    return k < 1 ? 1 : (k > n ? n : k);
}

// ------------------------------------------------------------- compress
// Sparse emission: the elements that `pick(i)` selects, indices ascending,
// values v[idx]; the residual is v with the selected entries +0.0.  One
// pass counts each range's picks, a second writes them at the ranges'
// prefix offsets.
template <typename Pick>
void emit_sparse(const bc_tensor& t, Pick pick, uint32_t* idx, float* val, int threads) {
    const uint64_t n = t.n, nr = (n + kRange - 1) / kRange;
    const VReader rd(t);
    std::vector<uint64_t> at(nr + 1, 0);
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        uint64_t c = 0;
        for (uint64_t i = lo; i < hi; ++i) c += pick(i) ? 1u : 0u;
        at[q + 1] = c;
    });
    for (uint64_t q = 0; q < nr; ++q) at[q + 1] += at[q];
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        const VReader v_at = rd;
        float* const res = t.residual;
        uint64_t j = at[q];
        for (uint64_t i = lo; i < hi; ++i) {
            const float v = v_at(i);
            const bool sel = pick(i);
            if (sel) {
                idx[j] = (uint32_t)i;
                val[j] = v;
                ++j;
            }
            if (res) res[i] = sel ? 0.0f : v;
        }
    });
}

// Exact top-k: the first k of the order (|v| bits descending, index
// ascending).  A radix select finds the k-th of that order: a histogram of
// the top 12 key bits (per range, then summed) gives the bin that holds
// it, and the bin's entries are ordered to find the element itself; the
// selection is then every element at or before it in the order.
void compress_topk(const bc_tensor& t, uint64_t k, uint32_t* idx, float* val, int threads) {
    const uint64_t n = t.n, nr = (n + kRange - 1) / kRange;
    if (k >= n) {
        emit_sparse(t, [](uint64_t) { return true; }, idx, val, threads);
        return;
    }
    constexpr int kShift = 19, kBins = 1 << 12;  // keys are 31 bits
    std::vector<uint32_t> key(n);
    std::vector<uint32_t> hist(nr * kBins, 0u);
    const VReader rd(t);
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        const VReader v_at = rd;
        uint32_t* const h = &hist[q * kBins];
        uint32_t* const kq = key.data();
        for (uint64_t i = lo; i < hi; ++i) {
            const uint32_t x = hbits(v_at(i)) & 0x7FFFFFFFu;
            kq[i] = x;
            ++h[x >> kShift];
        }
    });
    std::vector<uint64_t> tot(kBins, 0);
    for (uint64_t q = 0; q < nr; ++q)
        for (int b = 0; b < kBins; ++b) tot[b] += hist[q * kBins + b];
    int b = kBins - 1;
    uint64_t above = 0;
    while (above + tot[b] < k) above += tot[b--];
    // the bin's entries, index ascending, ordered to find the (k - above)-th
    std::vector<uint64_t> at(nr + 1, 0);
    for (uint64_t q = 0; q < nr; ++q) at[q + 1] = at[q] + hist[q * kBins + b];
    std::vector<uint32_t> cand(at[nr]);
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        uint64_t j = at[q];
        for (uint64_t i = lo; i < hi; ++i)
            if ((int)(key[i] >> kShift) == b) cand[j++] = (uint32_t)i;
    });
    auto before = [&](uint32_t x, uint32_t y) { return key[x] != key[y] ? key[x] > key[y] : x < y; };
    const uint64_t need = k - above;  // >= 1
    std::nth_element(cand.begin(), cand.begin() + (int64_t)(need - 1), cand.end(), before);
    const uint32_t kth = cand[need - 1], kkey = key[kth];
    emit_sparse(t, [&](uint64_t i) { return key[i] > kkey || (key[i] == kkey && i <= kth); }, idx, val,
                threads);
}

// Random-k: the images of 0 .. k-1 under the tensor's keyed permutation.
void compress_randk(const bc_tensor& t, uint64_t k, uint64_t seed, uint32_t* idx, float* val, int threads) {
    const uint32_t n = (uint32_t)t.n, h = half_bits(n), mask = (1u << h) - 1u;
    const uint4 rk = randk_round_keys(seed, t.tensor_id);
    std::vector<uint8_t> mark(n, 0);
    parallel_for((k + kRange - 1) / kRange, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(k, lo + kRange);
        for (uint64_t j = lo; j < hi; ++j) {
            uint32_t x = feistel((uint32_t)j, h, mask, rk);
            while (x >= n) x = feistel(x, h, mask, rk);
            mark[x] = 1;  // distinct images: no two threads write one byte
        }
    });
    emit_sparse(t, [&](uint64_t i) { return mark[i] != 0; }, idx, val, threads);
}

// Sign: bits of v, scale = fp64 sum of |v| / n rounded to fp32 (four
// interleaved fp64 partials per range, ranges in order), residual
// v - (bit ? -s : +s).
void compress_sign(const bc_tensor& t, uint32_t* words, float* scale, int threads) {
    const uint64_t n = t.n, nr = (n + kRange - 1) / kRange;
    const VReader rd(t);
    std::vector<double> part(nr, 0.0);
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        const VReader v_at = rd;
        uint32_t* const wq = words;
        double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
        for (uint64_t w = lo / 32; w < (hi + 31) / 32; ++w) {
            uint32_t word = 0;
            const uint64_t i0 = 32 * w;
            if (i0 + 32 <= hi) {
                for (int j = 0; j < 32; j += 4) {
                    const float v0 = v_at(i0 + j), v1 = v_at(i0 + j + 1), v2 = v_at(i0 + j + 2),
                                v3 = v_at(i0 + j + 3);
                    word |= (hbits(v0) >> 31) << j | (hbits(v1) >> 31) << (j + 1) | (hbits(v2) >> 31) << (j + 2) |
                            (hbits(v3) >> 31) << (j + 3);
                    a0 += std::fabs((double)v0);
                    a1 += std::fabs((double)v1);
                    a2 += std::fabs((double)v2);
                    a3 += std::fabs((double)v3);
                }
            } else {
                for (uint64_t i = i0; i < hi; ++i) {
                    const float v = v_at(i);
                    word |= (hbits(v) >> 31) << (i % 32);
                    const double a = std::fabs((double)v);
                    if (i % 4 == 0) a0 += a;
                    else if (i % 4 == 1) a1 += a;
                    else if (i % 4 == 2) a2 += a;
                    else a3 += a;
                }
            }
            wq[w] = word;
        }
        part[q] = (a0 + a1) + (a2 + a3);
    });
    double tot = 0.0;
    for (double p : part) tot += p;
    const float s = n ? (float)(tot / (double)n) : 0.0f;
    *scale = s;
    if (!t.residual) return;
    parallel_for(nr, threads, [&](uint64_t q) {
        const uint64_t lo = q * kRange, hi = std::min(n, lo + kRange);
        const VReader v_at = rd;
        float* const res = t.residual;
        for (uint64_t i = lo; i < hi; ++i) {
            const float v = v_at(i);
            res[i] = v - ((hbits(v) >> 31) ? -s : s);
        }
    });
}

// ------------------------------------------------------------ aggregate
// Sparse: per element, the workers' values in ascending worker order, one
// fp32 addition each from +0.0, then alpha times the sum.
void aggregate_sparse_range(const bc_payload* in, int W, uint64_t off, uint64_t k, uint64_t lo, uint64_t hi,
                            float alpha, float* out) {
    for (uint64_t i = lo; i < hi; ++i) out[i] = 0.0f;
    for (int w = 0; w < W; ++w) {
        const uint32_t* ix = in[w].idx + off;
        const float* vx = in[w].val + off;
        const uint32_t* p = std::lower_bound(ix, ix + k, (uint32_t)lo);
        for (; p != ix + k && *p < hi; ++p) out[*p] = out[*p] + vx[p - ix];
    }
    for (uint64_t i = lo; i < hi; ++i) out[i] = alpha * out[i];
}

// Sign: the order-free exact sum of the decoded values (NaN when one is
// NaN or both infinities occur, an infinity when one occurs, else the
// exact real sum rounded once), times alpha.  Scale sets whose fp64 sums
// are exact (finite normal or zero scales spanning at most
// 29 - ceil(log2 W) binades) add in fp64; others use the 288-bit integer
// limbs of exact_wide.hpp.
struct SignTensorForm {
    bool fp64 = true;
    int emin = 1;
};

SignTensorForm sign_form(const float* sc, int W) {
    SignTensorForm f;
    int lo = 1000, hi = -1000;
    bool bad = false;
    for (int w = 0; w < W; ++w) {
        const uint32_t b = hbits(sc[w]), e = (b >> 23) & 255u;
        if (e == 255u || (e == 0u && (b & 0x7FFFFFu))) bad = true;
        if (e != 255u && (b & 0x7FFFFFFFu)) {
            const int E = e ? (int)e : 1;
            lo = std::min(lo, E);
            hi = std::max(hi, E);
        }
    }
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    f.fp64 = !bad && (hi < lo || hi - lo <= 29 - lg);
    f.emin = hi < lo ? 1 : lo;
    return f;
}

float sign_exact_element(const uint32_t* const* words, const float* sc, int W, const SignTensorForm& f,
                         uint64_t i) {
    if (f.fp64) {
        double acc = 0.0;
        for (int w = 0; w < W; ++w) {
            const bool neg = (words[w][i / 32] >> (i % 32)) & 1u;
            acc += neg ? -(double)sc[w] : (double)sc[w];
        }
        return acc == 0.0 ? 0.0f : (float)acc;  // an exact zero gives +0.0
    }
    int64_t acc[kWideLimbs] = {};
    bool nan = false, pinf = false, ninf = false;
    for (int w = 0; w < W; ++w) {
        const uint32_t sb = hbits(sc[w]);
        const int bk = wide::bucket_of(sb, f.emin);
        if (bk == 9) continue;
        const bool neg = (((words[w][i / 32] >> (i % 32)) ^ (sb >> 31)) & 1u) != 0u;
        if (bk == 8) {
            if (sb & 0x7FFFFFu) nan = true;
            else if (neg) ninf = true;
            else pinf = true;
            continue;
        }
        const uint32_t e = (sb >> 23) & 255u;
        const int r = ((e ? (int)e : 1) - f.emin) & 31;
        const uint64_t c = (uint64_t)((sb & 0x7FFFFFu) | (e ? 0x800000u : 0u)) << r;
        const int64_t lo = (int64_t)(uint32_t)c, hi = (int64_t)(uint32_t)(c >> 32);
        acc[bk] += neg ? -lo : lo;
        acc[bk + 1] += neg ? -hi : hi;
    }
    if (nan || (pinf && ninf)) return hfloat(0x7FC00000u);
    if (pinf) return hfloat(0x7F800000u);
    if (ninf) return hfloat(0xFF800000u);
    return wide::round_total(acc, f.emin);
}

bool is_sparse_kind(int kind) { return kind == BC_TOPK || kind == BC_TOPK_SAMPLED || kind == BC_RANDK; }

}  // namespace
}  // namespace bc

using namespace bc;

extern "C" int bytecomp_cpu_compress(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                                     bc_payload out, int threads) {
    const CallRange range("bytecomp_cpu_compress");
    if (kind < BC_TOPK || kind > BC_QSGD8) return BC_E_KIND;
    if (kind > BC_SIGN1) return BC_E_KIND;  // the quantizers have no CPU form here
    uint64_t ppm = 1;
    if (is_sparse_kind(kind)) {
        if (!(ratio > 0.0) || ratio > 1.0) return BC_E_RATIO;
        ppm = (uint64_t)std::llround(ratio * 1e6);
        if (ppm == 0) return BC_E_RATIO;
    }
    if (T < 0 || T > (1 << 20)) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!t) return BC_E_NULL;
    if (is_sparse_kind(kind) ? (!out.idx || !out.val) : (!out.bits || !out.scale)) return BC_E_NULL;
    std::vector<uint64_t> off((size_t)T + 1, 0);
    for (int i = 0; i < T; ++i) {
        if (t[i].dtype != BC_F32 && t[i].dtype != BC_F16) return BC_E_DTYPE;
        if (t[i].n >= (1ull << 32) - 65536) return BC_E_SIZE;
        if (t[i].n && !t[i].grad) return BC_E_NULL;
        off[i + 1] = off[i] + (is_sparse_kind(kind) ? k_rule(t[i].n, ppm) : (t[i].n + 31) / 32);
    }
    if (threads <= 0) threads = (int)std::max(1u, std::thread::hardware_concurrency());
    try {
        // large tensors spread their work over the threads; the rest share
        // the threads one tensor each
        std::vector<int> big, small;
        for (int i = 0; i < T; ++i) (t[i].n >= 4 * kRange ? big : small).push_back(i);
        auto one = [&](int i, int th) {
            const bc_tensor& x = t[i];
            const uint64_t k = off[i + 1] - off[i];
            if (kind == BC_SIGN1) compress_sign(x, out.bits + off[i], out.scale + i, th);
            else if (kind == BC_RANDK) compress_randk(x, k, seed, out.idx + off[i], out.val + off[i], th);
            else compress_topk(x, k, out.idx + off[i], out.val + off[i], th);  // the sampled kind's result too
        };
        for (int i : big) one(i, threads);
        parallel_for(small.size(), threads, [&](uint64_t q) { one(small[q], 1); });
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    } catch (...) {
        return BC_E_HIP;
    }
    return BC_OK;
}

extern "C" int bytecomp_cpu_decompress_aggregate(int kind, double ratio, const bc_payload* in, int W,
                                                 const uint64_t* n, int T, float* const* out, float alpha,
                                                 int threads) {
    const CallRange range("bytecomp_cpu_decompress_aggregate");
    if (kind < BC_TOPK || kind > BC_SIGN1) return BC_E_KIND;
    uint64_t ppm = 1;
    if (is_sparse_kind(kind)) {
        if (!(ratio > 0.0) || ratio > 1.0) return BC_E_RATIO;
        ppm = (uint64_t)std::llround(ratio * 1e6);
        if (ppm == 0) return BC_E_RATIO;
    }
    if (T < 0 || T > (1 << 20) || W < 1 || W > 1024) return BC_E_COUNT;
    if (T == 0) return BC_OK;
    if (!in || !n || !out) return BC_E_NULL;
    std::vector<uint64_t> off((size_t)T + 1, 0), r0((size_t)T + 1, 0);
    for (int i = 0; i < T; ++i) {
        if (n[i] >= (1ull << 32) - 65536) return BC_E_SIZE;
        if (n[i] && !out[i]) return BC_E_NULL;
        off[i + 1] = off[i] + (is_sparse_kind(kind) ? k_rule(n[i], ppm) : (n[i] + 31) / 32);
        r0[i + 1] = r0[i] + (n[i] + kRange - 1) / kRange;
    }
    for (int w = 0; w < W; ++w)
        if (is_sparse_kind(kind) ? (off[T] && (!in[w].idx || !in[w].val)) : (!in[w].bits || !in[w].scale))
            return BC_E_NULL;
    if (threads <= 0) threads = (int)std::max(1u, std::thread::hardware_concurrency());
    try {
        std::vector<SignTensorForm> form;
        std::vector<float> sc;
        if (kind == BC_SIGN1) {
            form.resize((size_t)T);
            sc.resize((size_t)T * W);
            for (int i = 0; i < T; ++i) {
                for (int w = 0; w < W; ++w) sc[(size_t)i * W + w] = in[w].scale[i];
                form[(size_t)i] = sign_form(&sc[(size_t)i * W], W);
            }
        }
        parallel_for(r0[T], threads, [&](uint64_t q) {
            const int i = (int)(std::upper_bound(r0.begin(), r0.end(), q) - r0.begin()) - 1;
            const uint64_t lo = (q - r0[i]) * kRange, hi = std::min(n[i], lo + kRange);
            if (kind != BC_SIGN1) {
                aggregate_sparse_range(in, W, off[i], off[i + 1] - off[i], lo, hi, alpha, out[i]);
                return;
            }
            std::vector<const uint32_t*> wd((size_t)W);
            for (int w = 0; w < W; ++w) wd[(size_t)w] = in[w].bits + off[i];
            const float* s = &sc[(size_t)i * W];
            if (form[(size_t)i].fp64) {
                // 32 elements (one word per worker) at a time, workers in
                // order; every partial sum is exact, so the order is free
                for (uint64_t w0 = lo / 32; w0 < (hi + 31) / 32; ++w0) {
                    double acc[32] = {};
                    for (int w = 0; w < W; ++w) {
                        const uint32_t word = wd[(size_t)w][w0];
                        const double p = (double)s[w], m = -p;
                        for (int j = 0; j < 32; ++j) acc[j] += ((word >> j) & 1u) ? m : p;
                    }
                    const uint64_t e1 = std::min(hi, 32 * w0 + 32);
                    for (uint64_t e = 32 * w0; e < e1; ++e) {
                        const double a = acc[e - 32 * w0];
                        out[i][e] = alpha * (a == 0.0 ? 0.0f : (float)a);  // an exact zero gives +0.0
                    }
                }
                return;
            }
            for (uint64_t e = lo; e < hi; ++e)
                out[i][e] = alpha * sign_exact_element(wd.data(), s, W, form[(size_t)i], e);
        });
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    } catch (...) {
        return BC_E_HIP;
    }
    return BC_OK;
}
