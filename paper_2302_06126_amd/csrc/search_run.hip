// Native search rounds (include/tag_search.h, tag_search_run): the host
// tree work of round k+1 overlaps the GPU evaluation of round k when
// pipelined.  All device memory comes from the caller's workspace; the
// per-round host staging (states + query ops out, priors in) is double
// buffered in the caller's pinned buffer.
#include "search_internal.hpp"

using namespace tag;

namespace {

struct RunLayout {
    // device
    size_t stat, states, qop, qrep, qgraph, x_op, x_dev, x_od, x_dd, fwd_ws, E_op, E_dev, dec_ws, argmax, best, prior;
    size_t fwd_bytes, dec_bytes, dev_total;
    // host (pinned): two stages of [states | qop] and of [prior]
    size_t h_stage, h_prior, host_total;
};

tag_status run_layout(const tag_search_problem *p, const tag_graph *g, const tag_model_dims *dims, int32_t B,
                      RunLayout *L) {
    size_t sb = 0, rb = 0;
    tag_status st = tag_search_device_bytes(p, &sb, &rb);
    if (st != TAG_OK) return st;
    st = tag_gnn_workspace(g, dims, B, &L->fwd_bytes);
    if (st != TAG_OK) return st;
    st = tag_gnn_decide_workspace(g, dims, B, p->S, B, &L->dec_bytes);
    if (st != TAG_OK) return st;
    const size_t F = (size_t)dims->f, N = p->N, M = p->M, E = std::max<size_t>(p->od_op.size(), 1);
    size_t o = 0;
    auto put = [&](size_t bytes) { const size_t r = o; o = align_up(o + std::max<size_t>(bytes, 1), 256); return r; };
    L->stat = put(sb);
    L->states = put((size_t)B * rb);
    L->qop = put(4 * (size_t)B);
    L->qrep = put(4 * (size_t)B);
    L->qgraph = put(4 * (size_t)B);
    L->x_op = put(4 * (size_t)B * N * p->f_op);
    L->x_dev = put(4 * (size_t)B * M * 8);
    L->x_od = put((size_t)B * E);
    L->x_dd = put(p->model ? 8 * (size_t)B * p->dd_a.size() : 0);   // per-leaf link rows (simulator)
    L->fwd_ws = put(L->fwd_bytes);
    L->E_op = put(4 * (size_t)B * N * F);
    L->E_dev = put(4 * (size_t)B * M * F);
    L->dec_ws = put(L->dec_bytes);
    L->argmax = put(4 * (size_t)B);
    L->best = put(4 * (size_t)B);
    L->prior = put(4 * (size_t)B * p->S);
    L->dev_total = o;
    L->h_stage = align_up((size_t)B * rb + 4 * (size_t)B, 256);
    L->h_prior = align_up(4 * (size_t)B * p->S, 256);
    L->host_total = 2 * (L->h_stage + L->h_prior);
    return TAG_OK;
}

}  // namespace

extern "C" tag_status tag_search_run_workspace(const tag_search_problem *p, const tag_graph *g,
                                               const tag_model_dims *dims, int32_t batch, size_t *dev_bytes,
                                               size_t *host_bytes) {
    clear_error();
    if (!p || !g || !dims || !dev_bytes || !host_bytes) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (batch < 1) TAG_FAIL(TAG_EINVAL, "batch must be >= 1");
    RunLayout L;
    tag_status st = run_layout(p, g, dims, batch, &L);
    if (st != TAG_OK) return st;
    clear_error();
    *dev_bytes = L.dev_total;
    *host_bytes = L.host_total;
    return TAG_OK;
}

extern "C" tag_status tag_search_run(const tag_search_run_args *a, void *hip_stream) {
    clear_error();
    if (!a || !a->problem || !a->tree || !a->graph || !a->dims || !a->weights || !a->slices || !a->workspace ||
        !a->host_buf || (a->graph->e_oo && !a->x_oo) || (a->graph->e_dd && !a->x_dd))
        TAG_FAIL(TAG_EINVAL, "problem, tree, graph, dims, weights, slices, buffers and shared features must be non-NULL");
    const tag_search_problem *p = a->problem;
    const int32_t B = a->batch, K = p->K, S = p->S;
    if (B < 1 || a->rounds < 1) TAG_FAIL(TAG_EINVAL, "batch and rounds must be >= 1");
    if (a->dims->f_op != p->f_op) TAG_FAIL(TAG_ESHAPE, "dims->f_op must equal the problem's op feature width");
    if (a->graph->G != 1 || a->graph->n_op != p->N || a->graph->n_dev != p->M ||
        a->graph->e_od != (int64_t)p->od_op.size())
        TAG_FAIL(TAG_ESHAPE, "the graph must be the problem's single topology");
    if (a->slices->n_slices != S) TAG_FAIL(TAG_ESHAPE, "the slice table must be the problem's");
    int64_t tv = 0, te = 0;
    {
        tag_status st = tag_mcts_size(a->tree, &tv, &te);
        if (st != TAG_OK) return st;
    }
    RunLayout L;
    tag_status st = run_layout(p, a->graph, a->dims, B, &L);
    if (st != TAG_OK) return st;
    clear_error();
    if (a->ws_bytes < L.dev_total) TAG_FAIL(TAG_ENOSPACE, "workspace too small (see tag_search_run_workspace)");
    if (a->host_bytes < L.host_total) TAG_FAIL(TAG_ENOSPACE, "host buffer too small (see tag_search_run_workspace)");
    if ((reinterpret_cast<uintptr_t>(a->workspace) | reinterpret_cast<uintptr_t>(a->host_buf)) & 255)
        TAG_FAIL(TAG_EINVAL, "workspace and host_buf must be 256-byte aligned");
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    char *W = static_cast<char *>(a->workspace);
    char *H = static_cast<char *>(a->host_buf);
    size_t sb = 0, rb = 0;
    tag_search_device_bytes(p, &sb, &rb);

    st = tag_search_upload(p, W + L.stat, sb, hip_stream);
    if (st != TAG_OK) return st;
    {   // constant query columns: replica b, topology 0
        std::vector<int32_t> qr(B), qg(B, 0);
        for (int b = 0; b < B; ++b) qr[b] = b;
        TAG_HIP_CHECK(hipMemcpyAsync(W + L.qrep, qr.data(), 4 * (size_t)B, hipMemcpyHostToDevice, stream));
        TAG_HIP_CHECK(hipMemcpyAsync(W + L.qgraph, qg.data(), 4 * (size_t)B, hipMemcpyHostToDevice, stream));
        TAG_HIP_CHECK(hipStreamSynchronize(stream));
    }
    tag_features feats{};
    feats.n_replicas = B;
    feats.x_op = reinterpret_cast<const float *>(W + L.x_op);
    feats.x_dev = reinterpret_cast<const float *>(W + L.x_dev);
    feats.x_oo = a->x_oo;
    // the simulator's link idle shares make the link rows per leaf
    const bool own_dd = p->model != 0 && !p->dd_a.empty();
    feats.x_dd = own_dd ? reinterpret_cast<const float *>(W + L.x_dd) : a->x_dd;
    feats.x_od = reinterpret_cast<const uint8_t *>(W + L.x_od);
    feats.stride_oo = 0;
    feats.stride_dd = own_dd ? 2 * (int64_t)p->dd_a.size() : 0;
    feats.stride_od = (int64_t)p->od_op.size();

    hipEvent_t done[2];
    TAG_HIP_CHECK(hipEventCreateWithFlags(&done[0], hipEventDisableTiming));
    if (hipEventCreateWithFlags(&done[1], hipEventDisableTiming) != hipSuccess) {
        (void)hipEventDestroy(done[0]);
        TAG_FAIL(TAG_EHIP, "hipEventCreate failed");
    }
    struct Round {
        std::vector<int32_t> leaf, depth, path;
        std::vector<double> reward;
    } R[2];
    for (auto &r : R) { r.leaf.resize(B); r.depth.resize(B); r.path.assign((size_t)B * K, 0); r.reward.resize(B); }
    auto stage = [&](int k) { return H + (size_t)(k & 1) * (L.h_stage + L.h_prior); };
    auto hprior = [&](int k) { return reinterpret_cast<float *>(stage(k) + L.h_stage); };

    // host part of round k: select, rewards + packed states (into stage k)
    auto prepare = [&](int k) -> tag_status {
        Round &r = R[k & 1];
        tag_status s2 = tag_mcts_select(a->tree, B, r.leaf.data(), r.depth.data(), r.path.data());
        if (s2 != TAG_OK) return s2;
        char *sg = stage(k);
        return tag_search_pack(p, B, r.depth.data(), r.path.data(), K, sg, r.reward.data(),
                               reinterpret_cast<int32_t *>(sg + (size_t)B * rb));
    };
    // device part of round k: copy in, features, forward, decide, copy priors out
    auto launch = [&](int k) -> tag_status {
        char *sg = stage(k);
        if (hipMemcpyAsync(W + L.states, sg, (size_t)B * rb, hipMemcpyHostToDevice, stream) != hipSuccess ||
            hipMemcpyAsync(W + L.qop, sg + (size_t)B * rb, 4 * (size_t)B, hipMemcpyHostToDevice, stream) != hipSuccess)
            TAG_FAIL(TAG_EHIP, "hipMemcpyAsync (search states) failed");
        tag_status s2 = tag_search_features(p, B, W + L.stat, W + L.states, reinterpret_cast<float *>(W + L.x_op),
                                            reinterpret_cast<float *>(W + L.x_dev),
                                            reinterpret_cast<uint8_t *>(W + L.x_od), hip_stream);
        if (s2 != TAG_OK) return s2;
        if (own_dd) {
            s2 = tag_search_link_features(p, B, W + L.stat, W + L.states, reinterpret_cast<float *>(W + L.x_dd),
                                          hip_stream);
            if (s2 != TAG_OK) return s2;
        }
        s2 = tag_gnn_forward(a->graph, a->dims, a->weights, &feats, W + L.fwd_ws, L.fwd_bytes,
                             reinterpret_cast<float *>(W + L.E_op), reinterpret_cast<float *>(W + L.E_dev), hip_stream);
        if (s2 != TAG_OK) return s2;
        s2 = tag_gnn_decide(a->graph, a->dims, a->weights, B, reinterpret_cast<const float *>(W + L.E_op),
                            reinterpret_cast<const float *>(W + L.E_dev), a->slices, B,
                            reinterpret_cast<const int32_t *>(W + L.qrep), reinterpret_cast<const int32_t *>(W + L.qgraph),
                            reinterpret_cast<const int32_t *>(W + L.qop), reinterpret_cast<int32_t *>(W + L.argmax),
                            reinterpret_cast<float *>(W + L.best), reinterpret_cast<float *>(W + L.prior), nullptr,
                            W + L.dec_ws, L.dec_bytes, hip_stream);
        if (s2 != TAG_OK) return s2;
        if (hipMemcpyAsync(hprior(k), W + L.prior, 4 * (size_t)B * S, hipMemcpyDeviceToHost, stream) != hipSuccess ||
            hipEventRecord(done[k & 1], stream) != hipSuccess)
            TAG_FAIL(TAG_EHIP, "hipMemcpyAsync / hipEventRecord (priors) failed");
        return TAG_OK;
    };
    auto finish = [&](int k) -> tag_status {
        if (hipEventSynchronize(done[k & 1]) != hipSuccess) TAG_FAIL(TAG_EHIP, "hipEventSynchronize failed");
        Round &r = R[k & 1];
        const float *pr = hprior(k);
        if (a->depth_out) std::copy(r.depth.begin(), r.depth.end(), a->depth_out + (size_t)k * B);
        if (a->path_out) std::copy(r.path.begin(), r.path.end(), a->path_out + (size_t)k * B * K);
        if (a->reward_out) std::copy(r.reward.begin(), r.reward.end(), a->reward_out + (size_t)k * B);
        if (a->prior_out) std::copy(pr, pr + (size_t)B * S, a->prior_out + (size_t)k * B * S);
        return tag_mcts_update(a->tree, B, r.leaf.data(), r.depth.data(), r.path.data(), pr, r.reward.data());
    };

    tag_status rs = prepare(0);
    if (rs == TAG_OK) rs = launch(0);
    for (int k = 0; rs == TAG_OK && k < a->rounds; ++k) {
        const bool more = k + 1 < a->rounds;
        if (a->pipelined && more) {
            rs = prepare(k + 1);               // round k's edges still hold their in-flight visits
            if (rs == TAG_OK) rs = launch(k + 1);
        }
        if (rs == TAG_OK) rs = finish(k);
        if (rs == TAG_OK && !a->pipelined && more) {
            rs = prepare(k + 1);
            if (rs == TAG_OK) rs = launch(k + 1);
        }
    }
    // drain: no work may stay queued on the caller's buffers after an error
    (void)hipStreamSynchronize(stream);
    (void)hipEventDestroy(done[0]);
    (void)hipEventDestroy(done[1]);
    return rs;
}
