// Strategy-search service (host side): the search problem, the analytic
// iteration-time model that gives the reward, the PUCT tree with batched
// selection, and the packing of selected leaves into the state records the
// feature kernel expands (Section 4.2.2 of the paper, Monte-Carlo Tree
// Search; the readings are listed in include/tag_search.h).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <limits>
#include <map>
#include <new>
#include <thread>
#include <utility>

#include "search_internal.hpp"

using namespace tag;

namespace tag {

namespace {

constexpr int kAR = 0, kPS = 1, kDUP = 2, kMP = 3;
constexpr double kMemFactor = 4.0;   // weights + gradients + two optimizer moments per parameter byte

double bw_min(const tag_search_problem *P, const int *devs, int r) {
    double m = std::numeric_limits<double>::infinity();
    for (int x = 0; x < r; ++x)
        for (int y = x + 1; y < r; ++y) m = std::min(m, P->bw[(size_t)devs[x] * P->M + devs[y]]);
    return m;
}

}  // namespace

void full_strategy(const tag_search_problem *P, const int32_t *path, int32_t depth, uint64_t *mask, int32_t *opt) {
    const uint64_t all = P->M >= 64 ? ~0ull : ((1ull << P->M) - 1);
    if (depth == 0) {
        for (int g = 0; g < P->K; ++g) { mask[g] = all; opt[g] = kAR; }
        return;
    }
    const uint64_t m0 = P->slice_mask[path[0]] & all;
    const int32_t o0 = P->slice_opt[path[0]];
    for (int g = 0; g < P->K; ++g) { mask[g] = m0; opt[g] = o0; }
    for (int i = 0; i < depth; ++i) {
        const int g = P->order[i];
        mask[g] = P->slice_mask[path[i]] & all;
        opt[g] = P->slice_opt[path[i]];
    }
}

// The model of include/tag_search.h, in the order the reference computes it.
Eval evaluate_strategy(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt) {
    Eval e;
    e.load.assign(P->M, 0.0);
    e.mem.assign(P->M, 0.0);
    e.comp.assign(P->K, 0.0);
    e.sync.assign(P->K, 0.0);
    bool invalid = false;
    int devs[64];
    for (int g = 0; g < P->K; ++g) {
        int r = 0;
        for (int j = 0; j < P->M; ++j)
            if ((mask[g] >> j) & 1ull) devs[r++] = j;
        if (r == 0) { invalid = true; continue; }
        const int o = opt[g];
        double s = 0.0;
        if (r > 1 && o == kAR) {
            s = 2.0 * (r - 1) / r * P->PB[g] / bw_min(P, devs, r);
        } else if (r > 1 && o == kPS) {
            const int p = devs[0];
            double bps = std::numeric_limits<double>::infinity();
            for (int x = 1; x < r; ++x) bps = std::min(bps, P->bw[(size_t)p * P->M + devs[x]]);
            s = 2.0 * (r - 1) / r * P->PB[g] / bps;
        } else if (r > 1) {
            s = (double)(r - 1) / r * P->AB[g] / bw_min(P, devs, r);
        }
        e.sync[g] = s;
        double cmax = 0.0;
        for (int x = 0; x < r; ++x) {
            const int j = devs[x];
            const double c = o == kDUP ? P->FL[g] / P->speed[j] : P->FL[g] / (r * P->speed[j]);
            cmax = std::max(cmax, c);
            e.load[j] += c + s;
            const double wbytes = o == kMP ? P->PB[g] / r : P->PB[g];
            const double abytes = o == kDUP ? P->AB[g] : P->AB[g] / r;
            e.mem[j] += kMemFactor * wbytes + abytes;
        }
        e.comp[g] = cmax;
    }
    double xfer = 0.0;
    for (size_t k = 0; k < P->xpairs.size(); ++k) {
        const uint64_t m1 = mask[P->xpairs[k].first], m2 = mask[P->xpairs[k].second];
        if (m1 == m2 || m1 == 0 || m2 == 0) continue;
        const int p1 = __builtin_ctzll(m1), p2 = __builtin_ctzll(m2);
        xfer += P->xbytes[k] / P->bw[(size_t)p1 * P->M + p2];
    }
    double lmax = 0.0;
    for (int j = 0; j < P->M; ++j) lmax = std::max(lmax, e.load[j]);
    e.T = lmax + xfer;
    e.oom = invalid;
    for (int j = 0; j < P->M; ++j)
        if (e.mem[j] > P->mem[j]) e.oom = true;
    return e;
}

// Iteration time, OOM flag and the runtime feedback of a full strategy
// under the problem's model: group makespan (s) and idle share, device
// memory share and idle share.
//  analytic:  makespan = slowest replica's compute, idle share = sync /
//             (compute + sync), memory = the model's use, idle = 1 - load / T
//  simulator: makespan and memory peak as simulated, group idle share =
//             mean idle before its output transfers / T, device idle share
bool strategy_feedback(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt, SimScratch *W,
                       Feedback *f) {
    f->gms.assign(P->K, 0.0);
    f->gidle.assign(P->K, 0.0);
    f->memf.assign(P->M, 0.0);
    f->didle.assign(P->M, 0.0);
    f->lidle.assign(P->dd_a.size(), 0.0);
    if (P->model == 0) {
        const Eval e = evaluate_strategy(P, mask, opt);
        f->T = e.T;
        f->oom = e.oom;
        for (int g = 0; g < P->K; ++g) {
            const double cs = e.comp[g] + e.sync[g];
            f->gms[g] = e.comp[g];
            f->gidle[g] = cs > 0 ? e.sync[g] / cs : 0.0;
        }
        for (int j = 0; j < P->M; ++j) {
            f->memf[j] = std::min(e.mem[j] / P->mem[j], 1.0);
            f->didle[j] = e.T > 0 ? 1.0 - e.load[j] / e.T : 0.0;
        }
        return true;
    }
    bool valid = true, oom = false;
    f->peak.assign(P->M, 0.0);
    if (!sim_run(P, mask, opt, W, &f->T, &valid, &oom, f->gms.data(), f->gidle.data(), f->peak.data(),
                 f->didle.data(), f->lidle.empty() ? nullptr : f->lidle.data()))
        return false;
    f->oom = oom || !valid;
    if (!valid) {
        std::fill(f->gms.begin(), f->gms.end(), 0.0);
        std::fill(f->gidle.begin(), f->gidle.end(), 0.0);
        std::fill(f->didle.begin(), f->didle.end(), 0.0);
        std::fill(f->lidle.begin(), f->lidle.end(), 0.0);
        return true;
    }
    for (int g = 0; g < P->K; ++g) f->gidle[g] = f->T > 0 ? std::min(f->gidle[g] / f->T, 1.0) : 0.0;
    for (int j = 0; j < P->M; ++j) f->memf[j] = std::min(f->peak[j] / P->mem[j], 1.0);
    return true;
}

}  // namespace tag

// ------------------------------------------------------------------ problem
extern "C" tag_status tag_search_problem_create(const tag_search_problem_desc *d, tag_search_problem **out) {
    clear_error();
    if (!d || !out) TAG_FAIL(TAG_EINVAL, "desc and out must be non-NULL");
    *out = nullptr;
    if (d->n_op < 1 || d->n_dev < 1 || d->n_dev > 64 || d->n_groups < 1 || d->n_slices < 1 ||
        d->n_slices > 4096 || d->e_dd < 0 || d->e_oo < 0 || d->e_od < 0)
        TAG_FAIL(TAG_EINVAL, "need n_op >= 1, 1 <= n_dev <= 64, n_groups >= 1, 1 <= n_slices <= 4096, edge counts >= 0");
    if (d->f_op != 40 && d->f_op != 42) TAG_FAIL(TAG_ESHAPE, "f_op must be 40 or 42");
    if (!d->group_of || !d->op_type || !d->op_flops || !d->op_bytes || !d->op_params || !d->dev_tflops ||
        !d->dev_mem_gb || !d->dev_intra_gbs || !d->slice_mask || !d->slice_option ||
        (d->e_dd && (!d->dd_a || !d->dd_b || !d->dd_gbs)) || (d->e_oo && (!d->oo_src || !d->oo_dst)) ||
        (d->e_od && (!d->od_op || !d->od_dev)))
        TAG_FAIL(TAG_EINVAL, "array arguments must be non-NULL");
    const int N = d->n_op, M = d->n_dev, K = d->n_groups;
    std::vector<char> used(K, 0);
    for (int u = 0; u < N; ++u) {
        if (d->group_of[u] < 0 || d->group_of[u] >= K) TAG_FAIL(TAG_ERANGE, "group id out of range");
        used[d->group_of[u]] = 1;
        if (!(d->op_flops[u] > 0) || !(d->op_bytes[u] > 0) || !(d->op_params[u] >= 0) ||
            !std::isfinite(d->op_flops[u]) || !std::isfinite(d->op_bytes[u]) || !std::isfinite(d->op_params[u]))
            TAG_FAIL(TAG_EINVAL, "op FLOPs and bytes must be positive and finite, parameters >= 0");
    }
    for (int g = 0; g < K; ++g)
        if (!used[g]) TAG_FAIL(TAG_EINVAL, "every group must hold at least one op");
    for (int j = 0; j < M; ++j)
        if (!(d->dev_tflops[j] > 0) || !(d->dev_mem_gb[j] > 0) || !(d->dev_intra_gbs[j] > 0) ||
            !std::isfinite(d->dev_tflops[j]) || !std::isfinite(d->dev_mem_gb[j]) || !std::isfinite(d->dev_intra_gbs[j]))
            TAG_FAIL(TAG_EINVAL, "device speeds, memories and bandwidths must be positive and finite");
    for (int s = 0; s < d->n_slices; ++s)
        if (d->slice_option[s] > 3) TAG_FAIL(TAG_EINVAL, "slice options must be 0..3");

    tag_search_problem *P = new (std::nothrow) tag_search_problem();
    if (!P) TAG_FAIL(TAG_EINVAL, "out of host memory");
    P->N = N; P->M = M; P->K = K; P->S = d->n_slices; P->f_op = d->f_op;
    P->group_of.assign(d->group_of, d->group_of + N);
    P->op_type.assign(d->op_type, d->op_type + N);
    P->op_flops.assign(d->op_flops, d->op_flops + N);
    P->op_bytes.assign(d->op_bytes, d->op_bytes + N);
    P->FL.assign(K, 0.0); P->PB.assign(K, 0.0); P->AB.assign(K, 0.0);
    for (int u = 0; u < N; ++u) {   // plain sums in op order
        const int g = d->group_of[u];
        P->FL[g] += d->op_flops[u];
        P->PB[g] += d->op_params[u];
        P->AB[g] += d->op_bytes[u];
    }
    P->order.resize(K);
    for (int g = 0; g < K; ++g) P->order[g] = g;
    std::stable_sort(P->order.begin(), P->order.end(),
                     [&](int a, int b) { return P->FL[a] > P->FL[b]; });
    P->rep.assign(K, -1);
    std::vector<double> best(K, -1.0);
    for (int u = 0; u < N; ++u) {
        const int g = d->group_of[u];
        if (d->op_flops[u] > best[g]) { best[g] = d->op_flops[u]; P->rep[g] = u; }
    }
    P->speed.resize(M); P->mem.resize(M);
    P->dev_tflops.assign(d->dev_tflops, d->dev_tflops + M);
    P->dev_mem_gb.assign(d->dev_mem_gb, d->dev_mem_gb + M);
    P->dev_intra.assign(d->dev_intra_gbs, d->dev_intra_gbs + M);
    P->bw.assign((size_t)M * M, 0.0);
    for (int j = 0; j < M; ++j) {
        P->speed[j] = d->dev_tflops[j] * 1e12;
        P->mem[j] = d->dev_mem_gb[j] * 1e9;
        P->bw[(size_t)j * M + j] = d->dev_intra_gbs[j] * 1e9;
    }
    for (int64_t e = 0; e < d->e_dd; ++e) {
        const int a = d->dd_a[e], b = d->dd_b[e];
        if (a < 0 || a >= M || b < 0 || b >= M) { delete P; TAG_FAIL(TAG_ERANGE, "device link id out of range"); }
        if (!(d->dd_gbs[e] > 0) || !std::isfinite(d->dd_gbs[e])) { delete P; TAG_FAIL(TAG_EINVAL, "link bandwidths must be positive"); }
        P->bw[(size_t)a * M + b] = P->bw[(size_t)b * M + a] = d->dd_gbs[e] * 1e9;
    }
    for (int a = 0; a < M; ++a)
        for (int b = 0; b < M; ++b)
            if (!(P->bw[(size_t)a * M + b] > 0)) { delete P; TAG_FAIL(TAG_EINVAL, "every device pair needs a link"); }
    std::map<std::pair<int, int>, size_t> idx;
    for (int64_t e = 0; e < d->e_oo; ++e) {
        const int s = d->oo_src[e], t = d->oo_dst[e];
        if (s < 0 || s >= N || t < 0 || t >= N) { delete P; TAG_FAIL(TAG_ERANGE, "tensor op id out of range"); }
        const int gs = d->group_of[s], gd = d->group_of[t];
        if (gs == gd) continue;
        auto it = idx.find({gs, gd});
        if (it == idx.end()) {
            idx[{gs, gd}] = P->xpairs.size();
            P->xpairs.push_back({gs, gd});
            P->xbytes.push_back(0.0);
            it = idx.find({gs, gd});
        }
        P->xbytes[it->second] += d->op_bytes[s];
    }
    P->op_params.assign(d->op_params, d->op_params + N);
    P->oo_src.assign(d->oo_src, d->oo_src + d->e_oo);
    P->oo_dst.assign(d->oo_dst, d->oo_dst + d->e_oo);
    P->dd_a.assign(d->dd_a, d->dd_a + d->e_dd);
    P->dd_b.assign(d->dd_b, d->dd_b + d->e_dd);
    P->dd_gbs.assign(d->dd_gbs, d->dd_gbs + d->e_dd);
    P->od_op.assign(d->od_op, d->od_op + d->e_od);
    P->od_dev.assign(d->od_dev, d->od_dev + d->e_od);
    for (int64_t e = 0; e < d->e_od; ++e)
        if (P->od_op[e] < 0 || P->od_op[e] >= N || P->od_dev[e] < 0 || P->od_dev[e] >= M) {
            delete P;
            TAG_FAIL(TAG_ERANGE, "op-device pair id out of range");
        }
    P->slice_mask.assign(d->slice_mask, d->slice_mask + d->n_slices);
    P->slice_opt.assign(d->slice_option, d->slice_option + d->n_slices);
    {   // baseline iteration time
        std::vector<uint64_t> mk(K);
        std::vector<int32_t> op(K);
        full_strategy(P, nullptr, 0, mk.data(), op.data());
        P->T_base = evaluate_strategy(P, mk.data(), op.data()).T;
    }
    *out = P;
    return TAG_OK;
}

extern "C" void tag_search_problem_destroy(tag_search_problem *p) { delete p; }

extern "C" tag_status tag_search_order(const tag_search_problem *p, int32_t *order, int32_t *rep_op) {
    clear_error();
    if (!p || !order || !rep_op) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    for (int g = 0; g < p->K; ++g) { order[g] = p->order[g]; rep_op[g] = p->rep[g]; }
    return TAG_OK;
}

namespace {
tag_status check_path(const tag_search_problem *p, const int32_t *path, int32_t depth) {
    if (depth < 0 || depth > p->K) TAG_FAIL(TAG_EINVAL, "depth must be in [0, n_groups]");
    if (depth > 0 && !path) TAG_FAIL(TAG_EINVAL, "path must be non-NULL");
    for (int i = 0; i < depth; ++i)
        if (path[i] < 0 || path[i] >= p->S) TAG_FAIL(TAG_ERANGE, "slice id out of range");
    return TAG_OK;
}
}  // namespace

extern "C" tag_status tag_search_evaluate(const tag_search_problem *p, const int32_t *path, int32_t depth,
                                          double *reward, double *iter_time, int32_t *oom) {
    clear_error();
    if (!p || !reward || !iter_time || !oom) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    tag_status st = check_path(p, path, depth);
    if (st != TAG_OK) return st;
    std::vector<uint64_t> mk(p->K);
    std::vector<int32_t> op(p->K);
    full_strategy(p, path, depth, mk.data(), op.data());
    Feedback f;
    SimScratch *W = p->model ? sim_scratch_new() : nullptr;
    const bool ok = strategy_feedback(p, mk.data(), op.data(), W, &f);
    sim_scratch_free(W);
    if (!ok) TAG_FAIL(TAG_EINVAL, "the tensor graph has a cycle");
    *iter_time = f.T;
    *oom = f.oom ? 1 : 0;
    *reward = f.oom ? -1.0 : p->T_base / f.T;
    return TAG_OK;
}

extern "C" tag_status tag_search_set_model(tag_search_problem *p, int32_t model) {
    clear_error();
    if (!p) TAG_FAIL(TAG_EINVAL, "problem must be non-NULL");
    if (model != 0 && model != 1) TAG_FAIL(TAG_EINVAL, "model must be 0 (analytic) or 1 (simulator)");
    const int32_t old = p->model;
    p->model = model;
    std::vector<uint64_t> mk(p->K);
    std::vector<int32_t> op(p->K);
    full_strategy(p, nullptr, 0, mk.data(), op.data());
    Feedback f;
    SimScratch *W = model ? sim_scratch_new() : nullptr;
    const bool ok = strategy_feedback(p, mk.data(), op.data(), W, &f);
    sim_scratch_free(W);
    if (!ok) {
        p->model = old;
        TAG_FAIL(TAG_EINVAL, "the tensor graph has a cycle");
    }
    p->T_base = f.T;
    return TAG_OK;
}

// ------------------------------------------------------------------ packing
extern "C" tag_status tag_search_device_bytes(const tag_search_problem *p, size_t *static_bytes,
                                              size_t *state_bytes) {
    clear_error();
    if (!p || !static_bytes || !state_bytes) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    const StaticLayout sl = static_layout(p);
    *static_bytes = sl.total;
    *state_bytes = state_layout(p).total;
    return TAG_OK;
}

extern "C" tag_status tag_search_upload(const tag_search_problem *p, void *static_dev, size_t bytes,
                                        void *hip_stream) {
    clear_error();
    if (!p || !static_dev) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    const StaticLayout sl = static_layout(p);
    if (bytes < sl.total) TAG_FAIL(TAG_ENOSPACE, "static buffer too small (see tag_search_device_bytes)");
    std::vector<char> h(sl.total, 0);
    int32_t *gof = reinterpret_cast<int32_t *>(h.data() + sl.group_of);
    int32_t *typ = reinterpret_cast<int32_t *>(h.data() + sl.op_type);
    float *lfl = reinterpret_cast<float *>(h.data() + sl.lflops);
    float *lby = reinterpret_cast<float *>(h.data() + sl.lbytes);
    float *dst = reinterpret_cast<float *>(h.data() + sl.dev);
    int32_t *odo = reinterpret_cast<int32_t *>(h.data() + sl.od_op);
    int32_t *odd = reinterpret_cast<int32_t *>(h.data() + sl.od_dev);
    for (int u = 0; u < p->N; ++u) {
        gof[u] = p->group_of[u];
        typ[u] = p->op_type[u];
        lfl[u] = (float)(std::log10(p->op_flops[u]) - 8.0);
        lby[u] = (float)(std::log10(p->op_bytes[u]) - 6.0);
    }
    for (int j = 0; j < p->M; ++j) {
        dst[4 * j + 0] = (float)(p->dev_tflops[j] / 10.0);
        dst[4 * j + 1] = (float)(p->dev_mem_gb[j] / 32.0);
        dst[4 * j + 2] = 1.0f;
        dst[4 * j + 3] = (float)std::log10(p->dev_intra[j]);
    }
    for (size_t e = 0; e < p->od_op.size(); ++e) { odo[e] = p->od_op[e]; odd[e] = p->od_dev[e]; }
    float *lbw = reinterpret_cast<float *>(h.data() + sl.dd_lbw);
    for (size_t e = 0; e < p->dd_a.size(); ++e) lbw[e] = (float)(std::log10(p->dd_gbs[e]) - 1.0);
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    TAG_HIP_CHECK(hipMemcpyAsync(static_dev, h.data(), sl.total, hipMemcpyHostToDevice, st));
    TAG_HIP_CHECK(hipStreamSynchronize(st));
    return TAG_OK;
}

extern "C" tag_status tag_search_pack(const tag_search_problem *p, int32_t B, const int32_t *depth,
                                      const int32_t *path, int32_t path_stride, void *states,
                                      double *rewards, int32_t *query_op) {
    clear_error();
    if (!p || !depth || !path || !states || !rewards || !query_op) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (B < 1 || path_stride < p->K) TAG_FAIL(TAG_EINVAL, "need B >= 1 and path_stride >= n_groups");
    for (int b = 0; b < B; ++b) {
        tag_status st = check_path(p, path + (size_t)b * path_stride, depth[b]);
        if (st != TAG_OK) return st;
    }
    const StateLayout L = state_layout(p);
    // workers claim leaves from a shared counter; the simulator model spreads
    // the leaves over host threads (each leaf writes only its own records)
    std::atomic<int> next{0};
    auto work = [&](char *cycle) {
        std::vector<uint64_t> mk(p->K);
        std::vector<int32_t> op(p->K);
        Feedback f;
        SimScratch *W = p->model ? sim_scratch_new() : nullptr;
        for (int b = next.fetch_add(1); b < B; b = next.fetch_add(1)) {
            const int32_t *pb = path + (size_t)b * path_stride;
            const int d = depth[b];
            full_strategy(p, pb, d, mk.data(), op.data());
            if (!strategy_feedback(p, mk.data(), op.data(), W, &f)) {
                *cycle = 1;
                break;
            }
            rewards[b] = f.oom ? -1.0 : p->T_base / f.T;
            char *rec = static_cast<char *>(states) + (size_t)b * L.total;
            int32_t *hdr = reinterpret_cast<int32_t *>(rec);
            uint64_t *msk = reinterpret_cast<uint64_t *>(rec + L.mask);
            int32_t *opt = reinterpret_cast<int32_t *>(rec + L.option);
            int32_t *dec = reinterpret_cast<int32_t *>(rec + L.decided);
            float *gf = reinterpret_cast<float *>(rec + L.gfeat);
            float *df = reinterpret_cast<float *>(rec + L.dfeat);
            const int nxt = d < p->K ? p->order[d] : -1;
            hdr[0] = nxt;
            hdr[1] = 0;
            query_op[b] = nxt >= 0 ? p->rep[nxt] : 0;
            for (int g = 0; g < p->K; ++g) { dec[g] = 0; msk[g] = mk[g]; opt[g] = op[g]; gf[2 * g] = gf[2 * g + 1] = 0.f; }
            for (int i = 0; i < d; ++i) {
                const int g = p->order[i];
                dec[g] = 1;
                gf[2 * g] = (float)std::log10(std::max(f.gms[g], 1e-12) * 1e3);
                gf[2 * g + 1] = (float)f.gidle[g];
            }
            for (int j = 0; j < p->M; ++j) {
                df[2 * j] = (float)f.memf[j];
                df[2 * j + 1] = (float)f.didle[j];
            }
            float *lf = reinterpret_cast<float *>(rec + L.lfeat);
            for (size_t e = 0; e < f.lidle.size(); ++e) lf[e] = (float)f.lidle[e];
        }
        sim_scratch_free(W);
    };
    const int hw = std::max(1u, std::thread::hardware_concurrency());
    const int nt = p->model ? std::min({B, kPackThreads, hw}) : 1;
    std::vector<char> cycle(nt, 0);
    if (nt == 1) {
        work(cycle.data());
    } else {
        std::vector<std::thread> th;
        th.reserve(nt);
        for (int t = 0; t < nt; ++t) th.emplace_back(work, cycle.data() + t);
        for (auto &x : th) x.join();
    }
    for (char c : cycle)
        if (c) TAG_FAIL(TAG_EINVAL, "the tensor graph has a cycle");
    return TAG_OK;
}

// ------------------------------------------------------------------ tree
struct tag_mcts {
    int32_t L = 0, S = 0;
    double c = 1.0, vl = 0.0;
    struct Vertex {
        int32_t depth;
        int32_t edges;   // offset of the vertex's edge arrays, -1 until expanded
    };
    std::vector<Vertex> v;
    // edge arrays of expanded vertices, S entries each
    std::vector<int32_t> N, VL, child;
    std::vector<double> Q, G;
    int64_t expanded = 0;

    int32_t add_vertex(int32_t depth) {
        v.push_back({depth, -1});
        return (int32_t)v.size() - 1;
    }
    void expand(int32_t vid, const float *pr) {
        const int32_t off = (int32_t)(N.size());
        N.resize(off + S, 0); VL.resize(off + S, 0); child.resize(off + S, -1);
        Q.resize(off + S, 0.0); G.resize(off + S, 0.0);
        for (int a = 0; a < S; ++a) G[off + a] = (double)pr[a];
        v[vid].edges = off;
        ++expanded;
    }
    int32_t pick(int32_t vid) const {
        const int32_t o = v[vid].edges;
        int64_t total = 0;
        for (int a = 0; a < S; ++a) total += N[o + a] + VL[o + a];
        const double sq = std::sqrt((double)total);
        double best = -std::numeric_limits<double>::infinity();
        int32_t arg = 0;
        for (int a = 0; a < S; ++a) {
            const int64_t n = N[o + a], l = VL[o + a], ne = n + l;
            const double q = ne > 0 ? ((double)n * Q[o + a] + (double)l * vl) / (double)ne : 0.0;
            const double u = q + c * G[o + a] * sq / (1.0 + (double)ne);
            if (u > best) { best = u; arg = a; }
        }
        return arg;
    }
};

extern "C" tag_status tag_mcts_create(int32_t n_levels, int32_t n_actions, double c_puct, double vl_value,
                                      tag_mcts **out) {
    clear_error();
    if (!out) TAG_FAIL(TAG_EINVAL, "out must be non-NULL");
    *out = nullptr;
    if (n_levels < 1 || n_actions < 1 || n_actions > 4096) TAG_FAIL(TAG_EINVAL, "need n_levels >= 1, 1 <= n_actions <= 4096");
    if (!(c_puct >= 0) || !std::isfinite(c_puct) || !std::isfinite(vl_value)) TAG_FAIL(TAG_EINVAL, "c_puct must be >= 0, values finite");
    tag_mcts *t = new (std::nothrow) tag_mcts();
    if (!t) TAG_FAIL(TAG_EINVAL, "out of host memory");
    t->L = n_levels; t->S = n_actions; t->c = c_puct; t->vl = vl_value;
    t->add_vertex(0);
    *out = t;
    return TAG_OK;
}

extern "C" void tag_mcts_destroy(tag_mcts *t) { delete t; }

extern "C" tag_status tag_mcts_select(tag_mcts *t, int32_t B, int32_t *leaf, int32_t *depth, int32_t *path) {
    clear_error();
    if (!t || !leaf || !depth || !path) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (B < 1) TAG_FAIL(TAG_EINVAL, "B must be >= 1");
    for (int b = 0; b < B; ++b) {
        int32_t vid = 0, d = 0;
        int32_t *pb = path + (size_t)b * t->L;
        while (t->v[vid].edges >= 0 && t->v[vid].depth < t->L) {
            const int32_t a = t->pick(vid);
            const int32_t o = t->v[vid].edges + a;
            t->VL[o] += 1;
            pb[d++] = a;
            if (t->child[o] < 0) {
                const int32_t c = t->add_vertex(t->v[vid].depth + 1);
                t->child[t->v[vid].edges + a] = c;   // (edges vector unchanged by add_vertex)
            }
            vid = t->child[t->v[vid].edges + a];
        }
        leaf[b] = vid;
        depth[b] = d;
    }
    return TAG_OK;
}

extern "C" tag_status tag_mcts_update(tag_mcts *t, int32_t B, const int32_t *leaf, const int32_t *depth,
                                      const int32_t *path, const float *priors, const double *rewards) {
    clear_error();
    if (!t || !leaf || !depth || !path || !rewards) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (B < 1) TAG_FAIL(TAG_EINVAL, "B must be >= 1");
    // validate every path against the tree before changing anything
    for (int b = 0; b < B; ++b) {
        if (depth[b] < 0 || depth[b] > t->L) TAG_FAIL(TAG_EINVAL, "depth out of range");
        if (!std::isfinite(rewards[b])) TAG_FAIL(TAG_EINVAL, "rewards must be finite");
        int32_t vid = 0;
        for (int i = 0; i < depth[b]; ++i) {
            const int32_t a = path[(size_t)b * t->L + i];
            if (t->v[vid].edges < 0 || a < 0 || a >= t->S) TAG_FAIL(TAG_EINVAL, "path does not match the tree");
            const int32_t o = t->v[vid].edges + a;
            if (t->VL[o] < 1 || t->child[o] < 0) TAG_FAIL(TAG_EINVAL, "path holds no in-flight visit");
            vid = t->child[o];
        }
        if (vid != leaf[b]) TAG_FAIL(TAG_EINVAL, "leaf does not match its path");
        if (t->v[vid].depth < t->L && t->v[vid].edges < 0) {
            if (!priors) TAG_FAIL(TAG_EINVAL, "priors are needed to expand a leaf");
            for (int a = 0; a < t->S; ++a) {
                const float x = priors[(size_t)b * t->S + a];
                if (!(x >= 0.f) || !std::isfinite(x)) TAG_FAIL(TAG_EINVAL, "priors must be finite and >= 0");
            }
        }
    }
    for (int b = 0; b < B; ++b) {
        const int32_t lv = leaf[b];
        if (t->v[lv].depth < t->L && t->v[lv].edges < 0) t->expand(lv, priors + (size_t)b * t->S);
        int32_t vid = 0;
        const double r = rewards[b];
        for (int i = 0; i < depth[b]; ++i) {
            const int32_t o = t->v[vid].edges + path[(size_t)b * t->L + i];
            t->VL[o] -= 1;
            t->N[o] += 1;
            t->Q[o] += (r - t->Q[o]) / (double)t->N[o];
            vid = t->child[o];
        }
    }
    return TAG_OK;
}

extern "C" tag_status tag_mcts_root_stats(const tag_mcts *t, int32_t *visits, double *q) {
    clear_error();
    if (!t || !visits || !q) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    const int32_t o = t->v[0].edges;
    for (int a = 0; a < t->S; ++a) {
        visits[a] = o >= 0 ? t->N[o + a] : 0;
        q[a] = o >= 0 ? t->Q[o + a] : 0.0;
    }
    return TAG_OK;
}

extern "C" tag_status tag_mcts_best_path(const tag_mcts *t, int32_t *path, int32_t *depth) {
    clear_error();
    if (!t || !path || !depth) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    int32_t vid = 0, d = 0;
    while (t->v[vid].edges >= 0 && t->v[vid].depth < t->L) {
        const int32_t o = t->v[vid].edges;
        int32_t a = 0;
        for (int x = 1; x < t->S; ++x)
            if (t->N[o + x] > t->N[o + a]) a = x;
        if (t->N[o + a] == 0 || t->child[o + a] < 0) break;
        path[d++] = a;
        vid = t->child[o + a];
    }
    *depth = d;
    return TAG_OK;
}

extern "C" tag_status tag_mcts_size(const tag_mcts *t, int64_t *vertices, int64_t *expanded) {
    clear_error();
    if (!t || !vertices || !expanded) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    *vertices = (int64_t)t->v.size();
    *expanded = t->expanded;
    return TAG_OK;
}
