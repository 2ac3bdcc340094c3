// plan_sim.hip -- the decision algorithm's timeline model and Algorithm 2's
// enumeration on the host (no kernel here): the paper's CPU offloading
// search evaluates the iteration time of every vector of per-group
// offloading counts (Sec. 4.4.3, Algorithm 2 and the Theorem's
// prod(|G_i| + 1) strategies); each evaluation is one run of the timeline
// model of Sec. 4.3 ("Expressing interactions").
//
// Timeline model: a tensor's steps run on four resources (0 GPU, 1 CPU,
// 2 PCIe link, 3 network), each serving one step at a time in order of
// release (earliest release first, then lower tensor index, then earlier
// step).  Step 0 of every tensor is its backward computation on the GPU;
// tensor i's step 0 is released when tensor i-1's step 0 ends; each later
// step of a tensor is released when its previous step ends.  Completions
// are processed in time order (ties in the order they were scheduled);
// after each, idle resources start their next waiting step, in resource
// order.  The iteration time is the end of the last step of any tensor.
// The planner's Python model (planner.simulate) is the same definition; a
// CPU test compares the two on random instances bit for bit.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <functional>
#include <queue>
#include <thread>
#include <vector>

#include "../../include/bytecomp.h"

namespace bc {
namespace {

constexpr int kResources = 4;
constexpr int kOptions = 5;  // none, GPU indivisible, GPU divisible, CPU indivisible, CPU divisible

struct Waiting {
    double t;
    int i, s;
    bool operator>(const Waiting& o) const {
        if (t != o.t) return t > o.t;
        if (i != o.i) return i > o.i;
        return s > o.s;
    }
};
struct Event {
    double t;
    uint64_t seq;
    int r;
    bool operator>(const Event& o) const { return t != o.t ? t > o.t : seq > o.seq; }
};

// The stages of tensor i under option o: [off[i*kOptions+o], off[...+1]).
struct Table {
    int T;
    const double* compute;
    const uint64_t* off;
    const int32_t* res;
    const double* dur;
};

double simulate(const Table& tb, const int32_t* S) {
    const int T = tb.T;
    if (T == 0) return 0.0;
    // step s of tensor i: s = 0 computation, s >= 1 stage s-1 of its option
    auto nstages = [&](int i) -> int {
        const int o = S[i];
        return 1 + (int)(tb.off[i * kOptions + o + 1] - tb.off[i * kOptions + o]);
    };
    auto res_of = [&](int i, int s) -> int { return s == 0 ? 0 : tb.res[tb.off[i * kOptions + S[i]] + s - 1]; };
    auto dur_of = [&](int i, int s) -> double {
        return s == 0 ? tb.compute[i] : tb.dur[tb.off[i * kOptions + S[i]] + s - 1];
    };
    std::priority_queue<Waiting, std::vector<Waiting>, std::greater<Waiting>> waiting[kResources];
    std::priority_queue<Event, std::vector<Event>, std::greater<Event>> events;
    double free_at[kResources] = {0.0, 0.0, 0.0, 0.0};
    bool busy[kResources] = {false, false, false, false};
    int run_i[kResources] = {0, 0, 0, 0}, run_s[kResources] = {0, 0, 0, 0};
    uint64_t seq = 0;
    double last = 0.0;
    auto release = [&](double t, int i, int s) { waiting[res_of(i, s)].push(Waiting{t, i, s}); };
    auto start = [&](int r, double now) {
        if (busy[r] || waiting[r].empty()) return;
        const Waiting w = waiting[r].top();
        waiting[r].pop();
        const double begin = std::max(std::max(now, w.t), free_at[r]);
        const double end = begin + dur_of(w.i, w.s);
        busy[r] = true;
        run_i[r] = w.i;
        run_s[r] = w.s;
        free_at[r] = end;
        events.push(Event{end, seq++, r});
    };
    release(0.0, 0, 0);
    start(0, 0.0);
    while (!events.empty()) {
        const Event ev = events.top();
        events.pop();
        const int r = ev.r, i = run_i[r], s = run_s[r];
        busy[r] = false;
        if (s + 1 < nstages(i)) release(ev.t, i, s + 1);
        else last = std::max(last, ev.t);
        if (s == 0 && i + 1 < T) release(ev.t, i + 1, 0);
        for (int q = 0; q < kResources; ++q) start(q, ev.t);
    }
    return last;
}

bool valid_table(int T, const double* compute, const uint64_t* off, const int32_t* res, const double* dur) {
    if (T < 0) return false;
    if (T == 0) return true;
    if (!compute || !off) return false;
    const uint64_t n = off[(size_t)T * kOptions];
    if (n && (!res || !dur)) return false;
    for (size_t q = 0; q < (size_t)T * kOptions; ++q)
        if (off[q] > off[q + 1]) return false;
    for (uint64_t q = 0; q < n; ++q)
        if (res[q] < 0 || res[q] >= kResources) return false;
    return true;
}

}  // namespace
}  // namespace bc

using namespace bc;

extern "C" int bytecomp_plan_simulate(int T, const double* compute_us, const uint64_t* stage_off,
                                      const int32_t* stage_res, const double* stage_us, const int32_t* option,
                                      double* iteration_us) {
    if (!iteration_us || (T > 0 && !option)) return BC_E_NULL;
    if (!valid_table(T, compute_us, stage_off, stage_res, stage_us)) return BC_E_NULL;
    for (int i = 0; i < T; ++i)
        if (option[i] < 0 || option[i] >= kOptions) return BC_E_KIND;
    *iteration_us = simulate(Table{T, compute_us, stage_off, stage_res, stage_us}, option);
    return BC_OK;
}

extern "C" int bytecomp_plan_enumerate(int T, const double* compute_us, const uint64_t* stage_off,
                                       const int32_t* stage_res, const double* stage_us, const int32_t* option,
                                       int G, const uint64_t* group_off, const int32_t* group_member,
                                       uint64_t max_evals, double eps_us, int threads, int32_t* best_counts,
                                       double* best_us, uint64_t* evals) {
    if (!best_counts || !best_us || !evals || (T > 0 && !option) || G < 0 || (G > 0 && (!group_off || !group_member)))
        return BC_E_NULL;
    if (!valid_table(T, compute_us, stage_off, stage_res, stage_us)) return BC_E_NULL;
    for (int i = 0; i < T; ++i)
        if (option[i] < 0 || option[i] >= kOptions) return BC_E_KIND;
    uint64_t total = 1;
    for (int g = 0; g < G; ++g) {
        if (group_off[g] > group_off[g + 1]) return BC_E_COUNT;
        for (uint64_t q = group_off[g]; q < group_off[g + 1]; ++q) {
            const int32_t i = group_member[q];
            if (i < 0 || i >= T || (option[i] != 1 && option[i] != 2)) return BC_E_KIND;  // GPU options only
        }
        const uint64_t m = group_off[g + 1] - group_off[g] + 1;
        if (total > max_evals / m) return BC_E_SIZE;  // beyond the caller's bound: nothing evaluated
        total *= m;
    }
    const Table tb{T, compute_us, stage_off, stage_res, stage_us};
    std::vector<double> f;
    try {
        f.resize(total);
    } catch (const std::bad_alloc&) {
        return BC_E_SIZE;
    }
    // count vector of index x: mixed radix, the last group varying fastest
    // (the order itertools.product walks)
    auto eval_range = [&](uint64_t lo, uint64_t hi) {
        std::vector<int32_t> S(option, option + T);
        for (uint64_t x = lo; x < hi; ++x) {
            std::copy(option, option + T, S.begin());
            uint64_t rem = x;
            for (int g = G - 1; g >= 0; --g) {
                const uint64_t m = group_off[g + 1] - group_off[g] + 1;
                const uint64_t u = rem % m;
                rem /= m;
                for (uint64_t q = 0; q < u; ++q) {
                    const int32_t i = group_member[group_off[g] + q];
                    S[(size_t)i] = option[i] + 2;  // the same scheme on the CPU
                }
            }
            f[x] = simulate(tb, S.data());
        }
    };
    int nt = threads > 0 ? threads : (int)std::max(1u, std::thread::hardware_concurrency());
    if ((uint64_t)nt > total) nt = (int)total;
    try {
        if (nt <= 1) {
            eval_range(0, total);
        } else {
            std::vector<std::thread> pool;
            for (int w = 0; w < nt; ++w)
                pool.emplace_back(eval_range, total * (uint64_t)w / (uint64_t)nt, total * (uint64_t)(w + 1) / (uint64_t)nt);
            for (auto& th : pool) th.join();
        }
    } catch (...) {
        return BC_E_HIP;
    }
    // the first vector that improves on the best so far by more than eps,
    // in enumeration order (the planner's rule)
    uint64_t best = 0;
    double bf = f[0];
    for (uint64_t x = 1; x < total; ++x)
        if (f[x] < bf - eps_us) {
            bf = f[x];
            best = x;
        }
    // (vector 0 is "no offloading", which the caller's starting point is;
    // a strictly better one replaces it only by more than eps)
    uint64_t rem = best;
    for (int g = G - 1; g >= 0; --g) {
        const uint64_t m = group_off[g + 1] - group_off[g] + 1;
        best_counts[g] = (int32_t)(rem % m);
        rem /= m;
    }
    *best_us = bf;
    *evals = total;
    return BC_OK;
}
