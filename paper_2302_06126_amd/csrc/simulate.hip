// Host simulator of one training iteration under a deployment strategy
// (Section 4.3.2 of the paper, with the auxiliary ops the compiler of
// Section 4.3.1 inserts): the strategy is compiled into tasks (compute per
// replica, model-parallel gather, gradient sync, link transfers), every
// device and every device link runs a FIFO queue, a task enters its queue
// when its inputs are ready, and reference counting of tensors gives each
// device's peak memory.  The rules are listed in include/tag_search.h.
//
// Layout: tasks in flat arrays, dependencies and dependents as CSR built by
// counting sorts that keep insertion order, one ring per resource sized by
// a counting pass, and a binary heap of completions keyed by (finish time,
// task number).  Per-thread scratch makes the batched entry point
// allocation-free after the first simulation of each thread.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <limits>
#include <thread>
#include <vector>

#include "search_internal.hpp"

namespace tag {

struct SimScratch {
    // tasks
    std::vector<int32_t> res, op, dev, src, uses, left;
    std::vector<int8_t> kind;
    std::vector<double> dur, start, finish, size;
    // dependencies (k -> tasks it waits for), dependents (transpose)
    std::vector<int32_t> dep_task, dep_of, dep_off, dep_idx, out_off, out_idx, waiting, cnt;
    // per op
    std::vector<int32_t> dcount, dfirst, comp0, ready0;
    std::vector<int32_t> devlist;
    // resources
    std::vector<int32_t> q_off, q_head, q_tail, q_buf;
    std::vector<char> running;
    std::vector<double> busy;
    std::vector<std::pair<double, int32_t>> heap;
    std::vector<double> cur, peak;
    std::vector<double> gstart, gend, isum;
    std::vector<int32_t> icnt, cons_op;
};

namespace {

constexpr int kAR = 0, kPS = 1, kDUP = 2, kMP = 3;
constexpr double kMemFactor = 4.0;   // weights + gradients + two optimizer moments per parameter byte
enum : int8_t { kC = 0, kG = 1, kS = 2, kX = 3 };
using SimWork = SimScratch;

double bw_min_of(const tag_search_problem *P, const int32_t *D, int r) {
    double m = std::numeric_limits<double>::infinity();
    for (int x = 0; x < r; ++x)
        for (int y = x + 1; y < r; ++y) m = std::min(m, P->bw[(size_t)D[x] * P->M + D[y]]);
    return m;
}

inline int32_t link_res(int M, int a, int b) {
    if (a > b) std::swap(a, b);
    return M + a * M + b;
}

struct SimResult {
    double T = 0.0;
    bool valid = true, oom = false;
    int64_t n_tasks = 0;
};

// One simulation of the full strategy (mask, opt per group).  The output
// arrays may be null.
SimResult simulate_full(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt, SimWork &W,
                        double *g_makespan, double *g_idle, double *d_peak, double *d_idle, double *l_idle) {
    SimResult R;
    const int N = P->N, M = P->M, K = P->K;
    // device sets per op
    W.dcount.assign(N, 0);
    W.dfirst.assign(N + 1, 0);
    W.devlist.clear();
    for (int i = 0; i < N; ++i) {
        const uint64_t m = mask[P->group_of[i]];
        W.dfirst[i] = (int32_t)W.devlist.size();
        for (int j = 0; j < M; ++j)
            if ((m >> j) & 1ull) W.devlist.push_back(j);
        W.dcount[i] = (int32_t)W.devlist.size() - W.dfirst[i];
        if (W.dcount[i] == 0) R.valid = false;
    }
    W.dfirst[N] = (int32_t)W.devlist.size();
    if (!R.valid) {
        R.T = std::numeric_limits<double>::infinity();
        R.oom = true;
        return R;
    }
    auto D = [&](int i) { return W.devlist.data() + W.dfirst[i]; };
    auto has = [&](int i, int j) { return ((mask[P->group_of[i]] >> j) & 1ull) != 0; };
    auto slot = [&](int i, int j) {   // position of device j in op i's device list
        const int32_t *d = D(i);
        return (int)(std::lower_bound(d, d + W.dcount[i], j) - d);
    };
    // ---- tasks ----
    W.res.clear(); W.op.clear(); W.dev.clear(); W.src.clear(); W.uses.clear(); W.kind.clear();
    W.dur.clear(); W.size.clear();
    W.dep_task.clear(); W.dep_of.clear();
    W.comp0.assign(N, 0);
    W.ready0.assign(N, 0);
    auto add = [&](int32_t res, double dur, int8_t kind, int32_t op, int32_t dev, double size) {
        W.res.push_back(res); W.dur.push_back(dur); W.kind.push_back(kind); W.op.push_back(op);
        W.dev.push_back(dev); W.size.push_back(size); W.uses.push_back(0); W.src.push_back(-1);
        return (int32_t)W.res.size() - 1;
    };
    auto dep = [&](int32_t k, int32_t d) { W.dep_task.push_back(k); W.dep_of.push_back(d); };
    for (int i = 0; i < N; ++i) {
        const int r = W.dcount[i], o = opt[P->group_of[i]];
        const int32_t *Di = D(i);
        W.comp0[i] = (int32_t)W.res.size();
        for (int x = 0; x < r; ++x) {
            const int j = Di[x];
            const double du = (o == kDUP || r == 1) ? P->op_flops[i] / P->speed[j] : P->op_flops[i] / (r * P->speed[j]);
            add(j, du, kC, i, j, (o == kDUP || r == 1) ? P->op_bytes[i] : P->op_bytes[i] / r);
        }
        W.ready0[i] = W.comp0[i];
        if (o == kMP && r > 1) {
            const double du = (double)(r - 1) / r * P->op_bytes[i] / bw_min_of(P, Di, r);
            W.ready0[i] = (int32_t)W.res.size();
            for (int x = 0; x < r; ++x) {
                const int32_t k = add(Di[x], du, kG, i, Di[x], P->op_bytes[i]);
                for (int y = 0; y < r; ++y) dep(k, W.comp0[i] + y);
                W.uses[W.comp0[i] + x] += 1;
            }
        }
        if (P->op_params[i] > 0 && r > 1 && (o == kAR || o == kPS)) {
            double du;
            if (o == kAR) {
                du = 2.0 * (r - 1) / r * P->op_params[i] / bw_min_of(P, Di, r);
            } else {
                double bps = std::numeric_limits<double>::infinity();
                for (int x = 1; x < r; ++x) bps = std::min(bps, P->bw[(size_t)Di[0] * M + Di[x]]);
                du = 2.0 * (r - 1) / r * P->op_params[i] / bps;
            }
            for (int x = 0; x < r; ++x) {
                const int32_t k = add(Di[x], du, kS, i, Di[x], 0.0);
                for (int y = 0; y < r; ++y) dep(k, W.comp0[i] + y);
            }
        }
    }
    W.cons_op.clear();
    const size_t E = P->oo_src.size();
    for (size_t e = 0; e < E; ++e) {
        const int p = P->oo_src[e], c = P->oo_dst[e];
        const int rc = W.dcount[c], oc = opt[P->group_of[c]];
        const double share = (oc == kAR || oc == kPS) ? 1.0 / rc : 1.0;
        const int32_t *Dp = D(p), *Dc = D(c);
        const int rp = W.dcount[p];
        for (int x = 0; x < rc; ++x) {
            const int j = Dc[x];
            const int32_t cons = W.comp0[c] + x;
            if (has(p, j)) {
                const int32_t s = W.ready0[p] + slot(p, j);
                dep(cons, s);
                W.uses[s] += 1;
                continue;
            }
            int s = Dp[0];
            for (int y = 1; y < rp; ++y)
                if (P->bw[(size_t)Dp[y] * M + j] > P->bw[(size_t)s * M + j]) s = Dp[y];
            const double nbytes = P->op_bytes[p] * share;
            const int32_t srct = W.ready0[p] + slot(p, s);
            const int32_t k = add(link_res(M, s, j), nbytes / P->bw[(size_t)s * M + j], kX, p, j, nbytes);
            W.src[k] = srct;
            W.uses[k] = 1;
            W.uses[srct] += 1;
            dep(k, srct);
            dep(cons, k);
            W.cons_op.push_back(c);
        }
    }
    const int32_t n = (int32_t)W.res.size();
    R.n_tasks = n;
    // ---- CSR of dependencies (insertion order kept) and dependents ----
    const size_t nd = W.dep_task.size();
    W.dep_off.assign(n + 1, 0);
    W.out_off.assign(n + 1, 0);
    for (size_t t = 0; t < nd; ++t) { W.dep_off[W.dep_task[t] + 1]++; W.out_off[W.dep_of[t] + 1]++; }
    for (int32_t k = 0; k < n; ++k) { W.dep_off[k + 1] += W.dep_off[k]; W.out_off[k + 1] += W.out_off[k]; }
    W.dep_idx.resize(nd);
    W.cnt.assign(n, 0);
    for (size_t t = 0; t < nd; ++t) {
        const int32_t k = W.dep_task[t];
        W.dep_idx[W.dep_off[k] + W.cnt[k]++] = W.dep_of[t];
    }
    // dependents of d in ascending dependent order: walk tasks in order
    W.out_idx.resize(nd);
    W.cnt.assign(n, 0);
    for (int32_t k = 0; k < n; ++k)
        for (int32_t t = W.dep_off[k]; t < W.dep_off[k + 1]; ++t) {
            const int32_t d = W.dep_idx[t];
            W.out_idx[W.out_off[d] + W.cnt[d]++] = k;
        }
    W.waiting.resize(n);
    for (int32_t k = 0; k < n; ++k) W.waiting[k] = W.dep_off[k + 1] - W.dep_off[k];
    // ---- resource rings ----
    const int nres = M + M * M;
    W.q_off.assign(nres + 1, 0);
    for (int32_t k = 0; k < n; ++k) W.q_off[W.res[k] + 1]++;
    for (int r = 0; r < nres; ++r) W.q_off[r + 1] += W.q_off[r];
    W.q_head.assign(W.q_off.begin(), W.q_off.end() - 1);
    W.q_tail = W.q_head;
    W.q_buf.resize(n);
    W.running.assign(nres, 0);
    W.busy.assign(nres, 0.0);
    W.start.assign(n, 0.0);
    W.finish.assign(n, 0.0);
    W.heap.clear();
    auto cmp = [](const std::pair<double, int32_t> &a, const std::pair<double, int32_t> &b) {
        return a.first > b.first || (a.first == b.first && a.second > b.second);   // min-heap
    };
    auto start_next = [&](int r, double now) {
        const int32_t k = W.q_buf[W.q_head[r]++];
        W.start[k] = now;
        W.finish[k] = now + W.dur[k];
        W.busy[r] += W.dur[k];
        W.running[r] = 1;
        W.heap.push_back({W.finish[k], k});
        std::push_heap(W.heap.begin(), W.heap.end(), cmp);
    };
    auto make_ready = [&](int32_t k, double now) {
        const int r = W.res[k];
        W.q_buf[W.q_tail[r]++] = k;
        if (!W.running[r]) start_next(r, now);
    };
    // ---- memory: resident parameters ----
    W.cur.assign(M, 0.0);
    for (int i = 0; i < N; ++i) {
        const int r = W.dcount[i], o = opt[P->group_of[i]];
        const int32_t *Di = D(i);
        for (int x = 0; x < r; ++x)
            W.cur[Di[x]] += kMemFactor * (o == kMP ? P->op_params[i] / r : P->op_params[i]);
    }
    W.peak = W.cur;
    W.left = W.uses;
    // ---- events ----
    for (int32_t k = 0; k < n; ++k)
        if (W.waiting[k] == 0) make_ready(k, 0.0);
    int32_t done = 0;
    while (!W.heap.empty()) {
        std::pop_heap(W.heap.begin(), W.heap.end(), cmp);
        const double now = W.heap.back().first;
        const int32_t k = W.heap.back().second;
        W.heap.pop_back();
        const int r = W.res[k];
        W.running[r] = 0;
        ++done;
        const int d = W.dev[k];
        const int8_t kd = W.kind[k];
        if (kd != kS) {
            W.cur[d] += W.size[k];
            W.peak[d] = std::max(W.peak[d], W.cur[d]);
        }
        // inputs: C and X use their dependencies, G its own partition
        if (kd == kC || kd == kX) {
            for (int32_t t = W.dep_off[k]; t < W.dep_off[k + 1]; ++t) {
                const int32_t q = W.dep_idx[t];
                if (--W.left[q] == 0) W.cur[W.dev[q]] -= W.size[q];
            }
        } else if (kd == kG) {
            const int32_t q = W.comp0[W.op[k]] + slot(W.op[k], d);
            if (--W.left[q] == 0) W.cur[W.dev[q]] -= W.size[q];
        }
        if (kd != kS && W.left[k] == 0) W.cur[d] -= W.size[k];
        for (int32_t t = W.out_off[k]; t < W.out_off[k + 1]; ++t) {
            const int32_t q = W.out_idx[t];
            if (--W.waiting[q] == 0) make_ready(q, now);
        }
        if (!W.running[r] && W.q_head[r] < W.q_tail[r]) start_next(r, now);
    }
    if (done != n) {
        R.valid = false;
        R.n_tasks = -1;   // cycle
        return R;
    }
    double T = 0.0;
    for (int32_t k = 0; k < n; ++k) T = std::max(T, W.finish[k]);
    R.T = T;
    for (int j = 0; j < M; ++j)
        if (W.peak[j] > P->mem[j]) R.oom = true;
    if (g_makespan || g_idle) {
        W.gstart.assign(K, std::numeric_limits<double>::infinity());
        W.gend.assign(K, 0.0);
        W.isum.assign(K, 0.0);
        W.icnt.assign(K, 0);
        size_t xi = 0;
        for (int32_t k = 0; k < n; ++k) {
            const int g = P->group_of[W.op[k]];
            if (W.kind[k] == kC) W.gstart[g] = std::min(W.gstart[g], W.start[k]);
            if (W.kind[k] != kX) W.gend[g] = std::max(W.gend[g], W.finish[k]);
        }
        // transfers were numbered in creation order; cons_op follows the same order
        for (int32_t k = 0; k < n; ++k) {
            if (W.kind[k] != kX) continue;
            const int gp = P->group_of[W.op[k]], gc = P->group_of[W.cons_op[xi++]];
            if (gp != gc) {
                W.isum[gp] += W.start[k] - W.finish[W.src[k]];
                W.icnt[gp] += 1;
            }
        }
        for (int g = 0; g < K; ++g) {
            if (g_makespan) g_makespan[g] = W.gend[g] - W.gstart[g];
            if (g_idle) g_idle[g] = W.icnt[g] ? W.isum[g] / W.icnt[g] : 0.0;
        }
    }
    for (int j = 0; j < M; ++j) {
        if (d_peak) d_peak[j] = W.peak[j];
        if (d_idle) d_idle[j] = T > 0 ? 1.0 - W.busy[j] / T : 0.0;
    }
    if (l_idle)
        for (size_t e = 0; e < P->dd_a.size(); ++e)
            l_idle[e] = T > 0 ? 1.0 - W.busy[link_res(M, P->dd_a[e], P->dd_b[e])] / T : 0.0;
    return R;
}

tag_status check_sim_path(const tag_search_problem *p, const int32_t *path, int32_t depth) {
    if (depth < 0 || depth > p->K) TAG_FAIL(TAG_EINVAL, "depth must be in [0, n_groups]");
    if (depth > 0 && !path) TAG_FAIL(TAG_EINVAL, "path must be non-NULL");
    for (int i = 0; i < depth; ++i)
        if (path[i] < 0 || path[i] >= p->S) TAG_FAIL(TAG_ERANGE, "slice id out of range");
    return TAG_OK;
}

}  // namespace

SimScratch *sim_scratch_new() { return new SimScratch(); }
void sim_scratch_free(SimScratch *w) { delete w; }

bool sim_run(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt, SimScratch *W, double *T,
             bool *valid, bool *oom, double *g_makespan, double *g_idle, double *d_peak, double *d_idle,
             double *l_idle) {
    const SimResult R = simulate_full(P, mask, opt, *W, g_makespan, g_idle, d_peak, d_idle, l_idle);
    *T = R.T;
    *valid = R.valid;
    *oom = R.oom;
    return R.n_tasks >= 0;
}

}  // namespace tag

using namespace tag;

extern "C" tag_status tag_simulate(const tag_search_problem *p, const int32_t *path, int32_t depth, tag_sim_out *out) {
    clear_error();
    if (!p || !out) TAG_FAIL(TAG_EINVAL, "problem and out must be non-NULL");
    tag_status st = check_sim_path(p, path, depth);
    if (st != TAG_OK) return st;
    std::vector<uint64_t> mask(p->K);
    std::vector<int32_t> opt(p->K);
    full_strategy(p, path, depth, mask.data(), opt.data());
    SimWork W;
    const SimResult R = simulate_full(p, mask.data(), opt.data(), W, out->group_makespan, out->group_idle,
                                      out->dev_peak, out->dev_idle, out->link_idle);
    if (R.n_tasks < 0) TAG_FAIL(TAG_EINVAL, "the tensor graph has a cycle");
    out->iter_time = R.T;
    out->valid = R.valid ? 1 : 0;
    out->oom = R.oom ? 1 : 0;
    out->n_tasks = R.n_tasks;
    if (!R.valid) {
        for (int g = 0; g < p->K; ++g) {
            if (out->group_makespan) out->group_makespan[g] = 0.0;
            if (out->group_idle) out->group_idle[g] = 0.0;
        }
        for (int j = 0; j < p->M; ++j) {
            if (out->dev_peak) out->dev_peak[j] = 0.0;
            if (out->dev_idle) out->dev_idle[j] = 0.0;
        }
        if (out->link_idle)
            for (size_t e = 0; e < p->dd_a.size(); ++e) out->link_idle[e] = 0.0;
    }
    return TAG_OK;
}

extern "C" tag_status tag_simulate_batch(const tag_search_problem *p, int32_t B, const int32_t *depth,
                                         const int32_t *path, int32_t path_stride, int32_t n_threads,
                                         double *iter_time, int32_t *oom) {
    clear_error();
    if (!p || !depth || !iter_time || !oom) TAG_FAIL(TAG_EINVAL, "NULL argument");
    if (B < 0 || n_threads < 1 || n_threads > 256) TAG_FAIL(TAG_EINVAL, "need B >= 0 and 1 <= n_threads <= 256");
    if (path_stride < p->K) TAG_FAIL(TAG_EINVAL, "path_stride must be >= n_groups");
    for (int32_t b = 0; b < B; ++b) {
        tag_status st = check_sim_path(p, path ? path + (size_t)b * path_stride : nullptr, depth[b]);
        if (st != TAG_OK) return st;
    }
    std::vector<char> cyc(std::max(B, 1), 0);
    std::atomic<int32_t> next{0};
    auto run = [&](int) {
        SimWork W;
        std::vector<uint64_t> mask(p->K);
        std::vector<int32_t> opt(p->K);
        for (int32_t b = next.fetch_add(1); b < B; b = next.fetch_add(1)) {
            full_strategy(p, path ? path + (size_t)b * path_stride : nullptr, depth[b], mask.data(), opt.data());
            const SimResult R = simulate_full(p, mask.data(), opt.data(), W, nullptr, nullptr, nullptr, nullptr, nullptr);
            iter_time[b] = R.T;
            oom[b] = R.oom ? 1 : 0;
            if (R.n_tasks < 0) cyc[b] = 1;
        }
    };
    const int nt = std::min<int>(n_threads, std::max<int32_t>(B, 1));
    if (nt == 1) {
        run(0);
    } else {
        std::vector<std::thread> th;
        th.reserve(nt);
        for (int t = 0; t < nt; ++t) th.emplace_back(run, t);
        for (auto &x : th) x.join();
    }
    for (int32_t b = 0; b < B; ++b)
        if (cyc[b]) TAG_FAIL(TAG_EINVAL, "the tensor graph has a cycle");
    return TAG_OK;
}
