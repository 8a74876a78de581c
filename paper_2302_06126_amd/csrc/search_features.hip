// GNN inputs of a batch of search states (op / device / placement-edge
// features, Section 4.2.1 input table: raw features, the strategy encoding,
// runtime feedback and the search progress) expanded on the GPU from the
// packed state records tag_search_pack writes.  Element-parallel and
// store-bound: consecutive threads write consecutive feature words.
#include "search_internal.hpp"

namespace tag {
namespace {

struct FeatArgs {
    int32_t B, N, M, K, f_op;
    int64_t E;
    const int32_t *group_of, *op_type, *od_op, *od_dev;
    const float *lflops, *lbytes, *dev;
    const char *states;
    StateLayout L;
    float *x_op, *x_dev;
    uint8_t *x_od;
};

__global__ void __launch_bounds__(256) feat_op(FeatArgs a) {
    const int64_t total = (int64_t)a.B * a.N * a.f_op;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / a.f_op;
        const int c = (int)(i - row * a.f_op);
        const int b = (int)(row / a.N);
        const int u = (int)(row - (int64_t)b * a.N);
        const char *rec = a.states + (size_t)b * a.L.total;
        const int g = a.group_of[u];
        const int nxt = reinterpret_cast<const int32_t *>(rec)[0];
        const bool dec = reinterpret_cast<const int32_t *>(rec + a.L.decided)[g] != 0;
        float v = 0.f;
        if (c < 32) v = (a.op_type[u] & 31) == c ? 1.f : 0.f;
        else if (c == 32) v = a.lflops[u];
        else if (c == 33) v = a.lbytes[u];
        else if (c < 38) v = (dec && reinterpret_cast<const int32_t *>(rec + a.L.option)[g] == c - 34) ? 1.f : 0.f;
        else if (c == 38) v = dec ? 1.f : 0.f;
        else if (c == 39) v = g == nxt ? 1.f : 0.f;
        else v = dec ? reinterpret_cast<const float *>(rec + a.L.gfeat)[2 * g + (c - 40)] : 0.f;
        a.x_op[i] = v;
    }
}

__global__ void __launch_bounds__(256) feat_dev(FeatArgs a) {
    const int64_t total = (int64_t)a.B * a.M * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / 8;
        const int c = (int)(i & 7);
        const int b = (int)(row / a.M);
        const int j = (int)(row - (int64_t)b * a.M);
        const char *rec = a.states + (size_t)b * a.L.total;
        float v = 0.f;
        if (c < 4) v = a.dev[4 * j + c];
        else if (c < 6) v = reinterpret_cast<const float *>(rec + a.L.dfeat)[2 * j + (c - 4)];
        a.x_dev[i] = v;
    }
}

__global__ void __launch_bounds__(256) feat_od(FeatArgs a) {
    const int64_t total = (int64_t)a.B * a.E;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int b = (int)(i / a.E);
        const int64_t e = i - (int64_t)b * a.E;
        const char *rec = a.states + (size_t)b * a.L.total;
        const int g = a.group_of[a.od_op[e]];
        const bool dec = reinterpret_cast<const int32_t *>(rec + a.L.decided)[g] != 0;
        const uint64_t m = reinterpret_cast<const uint64_t *>(rec + a.L.mask)[g];
        a.x_od[i] = (dec && ((m >> a.od_dev[e]) & 1ull)) ? 1 : 0;
    }
}

// link rows of every state: log10(GB/s) - 1 and the link's idle share
__global__ void __launch_bounds__(256) feat_dd(int32_t B, int64_t E, const float *lbw, const char *states,
                                               StateLayout L, float *x_dd) {
    const int64_t total = (int64_t)B * E * 2;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / 2;
        const int b = (int)(row / E);
        const int64_t e = row - (int64_t)b * E;
        x_dd[i] = (i & 1) ? reinterpret_cast<const float *>(states + (size_t)b * L.total + L.lfeat)[e] : lbw[e];
    }
}

unsigned grid_for(int64_t n) {
    const int64_t g = (n + 255) / 256;
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(g, 65536));
}

}  // namespace
}  // namespace tag

using namespace tag;

extern "C" tag_status tag_search_features(const tag_search_problem *p, int32_t B, const void *static_dev,
                                          const void *states_dev, float *x_op, float *x_dev, uint8_t *x_od,
                                          void *hip_stream) {
    clear_error();
    if (!p || !static_dev || !states_dev || !x_op || !x_dev || (!x_od && !p->od_op.empty()))
        TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (B < 1) TAG_FAIL(TAG_EINVAL, "B must be >= 1");
    if ((reinterpret_cast<uintptr_t>(static_dev) | reinterpret_cast<uintptr_t>(states_dev)) & 15)
        TAG_FAIL(TAG_EINVAL, "static_dev and states_dev must be 16-byte aligned");
    const StaticLayout sl = static_layout(p);
    const char *sd = static_cast<const char *>(static_dev);
    FeatArgs a;
    a.B = B; a.N = p->N; a.M = p->M; a.K = p->K; a.f_op = p->f_op;
    a.E = (int64_t)p->od_op.size();
    a.group_of = reinterpret_cast<const int32_t *>(sd + sl.group_of);
    a.op_type = reinterpret_cast<const int32_t *>(sd + sl.op_type);
    a.lflops = reinterpret_cast<const float *>(sd + sl.lflops);
    a.lbytes = reinterpret_cast<const float *>(sd + sl.lbytes);
    a.dev = reinterpret_cast<const float *>(sd + sl.dev);
    a.od_op = reinterpret_cast<const int32_t *>(sd + sl.od_op);
    a.od_dev = reinterpret_cast<const int32_t *>(sd + sl.od_dev);
    a.states = static_cast<const char *>(states_dev);
    a.L = state_layout(p);
    a.x_op = x_op; a.x_dev = x_dev; a.x_od = x_od;
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    feat_op<<<grid_for((int64_t)B * p->N * p->f_op), 256, 0, st>>>(a);
    feat_dev<<<grid_for((int64_t)B * p->M * 8), 256, 0, st>>>(a);
    if (a.E > 0) feat_od<<<grid_for((int64_t)B * a.E), 256, 0, st>>>(a);
    return launch_status("tag_search_features");
}

extern "C" tag_status tag_search_link_features(const tag_search_problem *p, int32_t B, const void *static_dev,
                                               const void *states_dev, float *x_dd, void *hip_stream) {
    clear_error();
    if (!p || !static_dev || !states_dev || (!x_dd && !p->dd_a.empty())) TAG_FAIL(TAG_EINVAL, "arguments must be non-NULL");
    if (B < 1) TAG_FAIL(TAG_EINVAL, "B must be >= 1");
    if ((reinterpret_cast<uintptr_t>(static_dev) | reinterpret_cast<uintptr_t>(states_dev)) & 15)
        TAG_FAIL(TAG_EINVAL, "static_dev and states_dev must be 16-byte aligned");
    const int64_t E = (int64_t)p->dd_a.size();
    if (E == 0) return TAG_OK;
    const StaticLayout sl = static_layout(p);
    feat_dd<<<grid_for((int64_t)B * E * 2), 256, 0, static_cast<hipStream_t>(hip_stream)>>>(
        B, E, reinterpret_cast<const float *>(static_cast<const char *>(static_dev) + sl.dd_lbw),
        static_cast<const char *>(states_dev), state_layout(p), x_dd);
    return launch_status("tag_search_link_features");
}
