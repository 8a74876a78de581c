// Decision head (Section 4.2.1, the decoder after the GNN; Section 4.2, the
// placement matrix P and the four replication options O).
//
// For query op i and slice a = (mask, option):
//   x     = [ sum_{j in mask} E_dev[j] ; E_op[i] ; onehot(option) ]
//   score = w2 . ReLU(W1 x + b1) + b2   (H > 0)  or  w2 . x + b2  (H = 0)
// W1 x splits exactly into a per-slice part and a per-query part:
//   W1 x = sum_{j in mask} (W1_dev E_dev[j]) + W1_opt[:, option] + W1_op E_op[i]
// so the kernels compute t_j = W1_dev E_dev[j] once per device, the slice
// part u_a once per (candidate, slice), v_i once per query, and then only
// the ReLU readout per (query, slice).  The softmax over the slice table
// gives the priors; the argmax (lowest index among equal maxima) is decoded
// into placement, replica count, sync scheme and the compression (SFB) flag.
#include <algorithm>
#include <mutex>
#include <string>

#include "tag_internal.hpp"

namespace tag {
namespace {

struct DecArgs {
    int32_t R, G, S, Q, F, H, Hx;
    int64_t n_op, n_dev;
    const int32_t *op_off, *dev_off;   // [G+1]
    const float *E_op, *E_dev;
    const uint64_t *mask;
    const uint8_t *option;
    const float *P;      // projection rows [Hx][2F+4] (W1, or w2 for the linear head)
    const float *b1, *w2, *b2;
    const int32_t *q_rep, *q_graph, *q_op;
    float *t;            // [R*n_dev][Hx]
    float *u;            // [R*G][Hx][S]
    float *v;            // [Q][Hx]
    int32_t *argmax;
    float *best, *prior;
    tag_decision *dec;
};

// u[rg][h][a] = sum_{j in mask_a} t[dev(rg, j)][h] + P[h][2F + opt_a] (+ b1[h])
// One block per (candidate graph rg, chunk of kSliceH hidden units): the
// chunk of the graph's device rows t and the option columns sit in LDS; each
// thread walks the set bits of its slices' masks in ascending device order.
constexpr int kSliceH = 8;
__global__ void __launch_bounds__(256) dec_slice(DecArgs A) {
    __shared__ float tl[64][kSliceH + 1];
    __shared__ float po[4][kSliceH];
    const int nch = (A.Hx + kSliceH - 1) / kSliceH;
    const int64_t rg = blockIdx.x / nch;
    const int h0 = (int)(blockIdx.x % nch) * kSliceH;
    const int32_t r = (int32_t)(rg / A.G), g = (int32_t)(rg % A.G);
    const int32_t d0 = A.dev_off[g], nd = A.dev_off[g + 1] - d0;
    const int din = 2 * A.F + 4;
    for (int i = threadIdx.x; i < nd * kSliceH; i += blockDim.x) {
        const int j = i / kSliceH, hh = i % kSliceH;
        tl[j][hh] = h0 + hh < A.Hx ? A.t[((int64_t)r * A.n_dev + d0 + j) * A.Hx + h0 + hh] : 0.f;
    }
    for (int i = threadIdx.x; i < 4 * kSliceH; i += blockDim.x) {
        const int o = i / kSliceH, hh = i % kSliceH, h = h0 + hh;
        po[o][hh] = h < A.Hx ? A.P[(size_t)h * din + 2 * A.F + o] + (A.H > 0 ? A.b1[h] : 0.f) : 0.f;
    }
    __syncthreads();
    const uint64_t keep = nd >= 64 ? ~0ull : ((1ull << nd) - 1ull);
    for (int32_t a = threadIdx.x; a < A.S; a += blockDim.x) {
        uint64_t m = A.mask[a] & keep;
        const int opt = min((int)A.option[a], 3);
        float acc[kSliceH];
#pragma unroll
        for (int hh = 0; hh < kSliceH; ++hh) acc[hh] = po[opt][hh];
        while (m) {
            const int j = __builtin_ctzll(m);
            m &= m - 1;
#pragma unroll
            for (int hh = 0; hh < kSliceH; ++hh) acc[hh] += tl[j][hh];
        }
        float *u = A.u + (rg * A.Hx + h0) * A.S + a;
#pragma unroll
        for (int hh = 0; hh < kSliceH; ++hh)
            if (h0 + hh < A.Hx) u[(int64_t)hh * A.S] = acc[hh];
    }
}

__device__ __forceinline__ bool query_valid(const DecArgs &A, int32_t q, int32_t *r, int32_t *g, int32_t *op) {
    *r = A.q_rep[q]; *g = A.q_graph[q]; *op = A.q_op[q];
    if (*r < 0 || *r >= A.R || *g < 0 || *g >= A.G) return false;
    return *op >= 0 && *op < A.op_off[*g + 1] - A.op_off[*g];
}

// row of E_op read by each query (-1: invalid query)
__global__ void dec_query_rows(DecArgs A, int32_t *qrow) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < A.Q; q += (int64_t)gridDim.x * blockDim.x) {
        int32_t r, g, op;
        qrow[q] = query_valid(A, (int32_t)q, &r, &g, &op) ? (int32_t)((int64_t)r * A.n_op + A.op_off[g] + op) : -1;
    }
}

constexpr int kScoreThreads = 256;

__device__ __forceinline__ float slice_score(const DecArgs &A, const float *urg, const float *vq,
                                             const float *w2s, int32_t a) {
    if (A.H == 0) return A.b2[0] + urg[a] + vq[0];
    // independent loads in batches of 16 hidden units, summed in order
    float s = 0.f;
    int h = 0;
    for (; h + 16 <= A.H; h += 16) {
        float uu[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) uu[k] = urg[(int64_t)(h + k) * A.S + a];
#pragma unroll
        for (int k = 0; k < 16; ++k) s = fmaf(w2s[h + k], fmaxf(uu[k] + vq[h + k], 0.f), s);
    }
    for (; h < A.H; ++h) s = fmaf(w2s[h], fmaxf(urg[(int64_t)h * A.S + a] + vq[h], 0.f), s);
    return A.b2[0] + s;
}

// Max (lowest index on ties) and sum of exponentials over the block's
// per-thread partials, then the prior, argmax and decoded decision of query
// q whose raw scores are already in A.prior (when it is given).
__device__ void finish_query(const DecArgs &A, int32_t q, int32_t g, float m, int32_t im, float z,
                             float *red_m, int32_t *red_i, float *red_z) {
    red_m[threadIdx.x] = m; red_i[threadIdx.x] = im; red_z[threadIdx.x] = z;
    __syncthreads();
    for (int off = kScoreThreads / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) {
            float m1 = red_m[threadIdx.x], m2 = red_m[threadIdx.x + off];
            int32_t i1 = red_i[threadIdx.x], i2 = red_i[threadIdx.x + off];
            float z1 = red_z[threadIdx.x], z2 = red_z[threadIdx.x + off];
            float M = fmaxf(m1, m2);
            float zz = (m1 == -INFINITY ? 0.f : z1 * __expf(m1 - M)) + (m2 == -INFINITY ? 0.f : z2 * __expf(m2 - M));
            int32_t ii = (m2 > m1 || (m2 == m1 && i2 < i1)) ? i2 : i1;
            red_m[threadIdx.x] = M; red_i[threadIdx.x] = ii; red_z[threadIdx.x] = zz;
        }
        __syncthreads();
    }
    const float M = red_m[0], Z = red_z[0];
    const int32_t best = red_i[0];
    __syncthreads();   // the reduction arrays are reused by the next query
    if (A.prior) {
        const float inv = 1.f / Z;
        for (int32_t a = threadIdx.x; a < A.S; a += blockDim.x) {
            float s = A.prior[(int64_t)q * A.S + a];
            A.prior[(int64_t)q * A.S + a] = __expf(s - M) * inv;
        }
    }
    if (threadIdx.x == 0) {
        if (best < 0 || best >= A.S) {   // no comparable score (NaN inputs)
            A.argmax[q] = -1;
            A.best[q] = __builtin_nanf("");
            if (A.dec) A.dec[q] = tag_decision{0, 0, 0, 0, 0};
            return;
        }
        A.argmax[q] = best;
        A.best[q] = M;
        if (A.dec) {
            const int32_t nd = A.dev_off[g + 1] - A.dev_off[g];
            const uint64_t valid = nd >= 64 ? ~0ull : ((1ull << nd) - 1ull);
            const uint64_t msk = A.mask[best] & valid;
            const int o = min((int)A.option[best], 3);
            const int pc = __popcll(msk);
            A.dec[q] = tag_decision{msk, o, o == 3 ? 1 : pc, o == 0 ? 0 : (o == 1 ? 1 : 2), o == 2 ? 1 : 0};
        }
    }
}

__device__ void invalid_query(const DecArgs &A, int32_t q) {
    if (threadIdx.x == 0) {
        A.argmax[q] = -1;
        A.best[q] = __builtin_nanf("");
        if (A.dec) A.dec[q] = tag_decision{0, 0, 0, 0, 0};
    }
    if (A.prior)
        for (int32_t a = threadIdx.x; a < A.S; a += blockDim.x) A.prior[(int64_t)q * A.S + a] = 0.f;
}

// QB consecutive queries per block: scores, softmax prior, argmax, decoded
// decision.  When the block's queries are all valid and read one
// candidate's slice terms u (consecutive queries usually do), every u value
// is loaded once for all QB of them; otherwise the queries are taken one by
// one.  Consecutive blocks run on one XCD, so a candidate's u is fetched into
// one L2 rather than all eight.
template <int QB>
__global__ void __launch_bounds__(kScoreThreads) dec_score(DecArgs A) {
    extern __shared__ float sh[];   // v[QB][Hx] | w2[H]
    __shared__ float red_m[kScoreThreads];
    __shared__ int32_t red_i[kScoreThreads];
    __shared__ float red_z[kScoreThreads];
    const int32_t q0 = (int32_t)xcd_swizzle(blockIdx.x, gridDim.x) * QB;
    const int32_t nq = min(QB, A.Q - q0);
    float *w2s = sh + QB * A.Hx;
    for (int h = threadIdx.x; h < A.H; h += blockDim.x) w2s[h] = A.w2[h];
    int32_t rq[QB], gq[QB];
    bool shared = nq == QB;
#pragma unroll
    for (int i = 0; i < QB; ++i) {
        int32_t op;
        const bool ok = i < nq && query_valid(A, q0 + i, &rq[i], &gq[i], &op);
        shared = shared && ok && rq[i] == rq[0] && gq[i] == gq[0];
    }
    if (shared && QB > 1) {
        for (int i = 0; i < QB; ++i)
            for (int h = threadIdx.x; h < A.Hx; h += blockDim.x) sh[i * A.Hx + h] = A.v[(int64_t)(q0 + i) * A.Hx + h];
        __syncthreads();
        const float *urg = A.u + ((int64_t)rq[0] * A.G + gq[0]) * A.Hx * A.S;
        float m[QB], z[QB];
        int32_t im[QB];
#pragma unroll
        for (int i = 0; i < QB; ++i) { m[i] = -INFINITY; z[i] = 0.f; im[i] = INT32_MAX; }
        for (int32_t a = threadIdx.x; a < A.S; a += blockDim.x) {
            float sc[QB];
            if (A.H == 0) {
#pragma unroll
                for (int i = 0; i < QB; ++i) sc[i] = A.b2[0] + urg[a] + sh[i * A.Hx];
            } else {
                // independent loads in batches of 16 hidden units, summed in order
#pragma unroll
                for (int i = 0; i < QB; ++i) sc[i] = 0.f;
                int h = 0;
                for (; h + 16 <= A.H; h += 16) {
                    float uu[16];
#pragma unroll
                    for (int k = 0; k < 16; ++k) uu[k] = urg[(int64_t)(h + k) * A.S + a];
#pragma unroll
                    for (int k = 0; k < 16; ++k)
#pragma unroll
                        for (int i = 0; i < QB; ++i)
                            sc[i] = fmaf(w2s[h + k], fmaxf(uu[k] + sh[i * A.Hx + h + k], 0.f), sc[i]);
                }
                for (; h < A.H; ++h) {
                    const float uu = urg[(int64_t)h * A.S + a];
#pragma unroll
                    for (int i = 0; i < QB; ++i) sc[i] = fmaf(w2s[h], fmaxf(uu + sh[i * A.Hx + h], 0.f), sc[i]);
                }
#pragma unroll
                for (int i = 0; i < QB; ++i) sc[i] += A.b2[0];
            }
#pragma unroll
            for (int i = 0; i < QB; ++i) {
                if (A.prior) A.prior[(int64_t)(q0 + i) * A.S + a] = sc[i];
                if (sc[i] > m[i]) { z[i] = z[i] * __expf(m[i] - sc[i]) + 1.f; m[i] = sc[i]; im[i] = a; }
                else z[i] += __expf(sc[i] - m[i]);
            }
        }
        for (int i = 0; i < QB; ++i) finish_query(A, q0 + i, gq[0], m[i], im[i], z[i], red_m, red_i, red_z);
        return;
    }
    for (int i = 0; i < nq; ++i) {
        const int32_t q = q0 + i;
        int32_t r, g, op;
        if (!query_valid(A, q, &r, &g, &op)) {
            invalid_query(A, q);
            continue;
        }
        float *vq = sh;
        __syncthreads();   // the previous query's reads of v are done
        for (int h = threadIdx.x; h < A.Hx; h += blockDim.x) vq[h] = A.v[(int64_t)q * A.Hx + h];
        __syncthreads();
        const float *urg = A.u + ((int64_t)r * A.G + g) * A.Hx * A.S;
        // max (lowest index on ties) and the running sum of exponentials
        float m = -INFINITY, z = 0.f;
        int32_t im = INT32_MAX;
        for (int32_t a = threadIdx.x; a < A.S; a += blockDim.x) {
            float s = slice_score(A, urg, vq, w2s, a);
            if (A.prior) A.prior[(int64_t)q * A.S + a] = s;
            if (s > m) { z = z * __expf(m - s) + 1.f; m = s; im = a; }
            else z += __expf(s - m);
        }
        finish_query(A, q, g, m, im, z, red_m, red_i, red_z);
    }
}

struct DecLayout {
    float *t, *u, *v;
    int32_t *qrow;
};

size_t carve_dec(const tag_graph *g, int32_t Hx, int32_t R, int32_t S, int32_t Q, void *base, DecLayout *L) {
    Carver c(base);
    L->t = c.take<float>((size_t)R * g->n_dev * Hx);
    L->u = c.take<float>((size_t)R * g->G * Hx * S);
    L->v = c.take<float>((size_t)std::max(Q, 1) * Hx);
    L->qrow = c.take<int32_t>((size_t)std::max(Q, 1));
    return c.used;
}

inline unsigned grid_for(int64_t n) {
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 1 << 20));
}

}  // namespace

void launch_slice_terms(int32_t R, int32_t G, int32_t S, int32_t F, int32_t H, int64_t n_dev, const int32_t *dev_off,
                        const float *t, const float *W1, const float *b1, const uint64_t *mask,
                        const uint8_t *option, float *u, hipStream_t st) {
    DecArgs A{};
    A.R = R; A.G = G; A.S = S; A.F = F; A.H = H; A.Hx = std::max(H, 1);
    A.n_dev = n_dev;
    A.dev_off = dev_off;
    A.t = const_cast<float *>(t); A.P = W1; A.b1 = b1;
    A.mask = mask; A.option = option;
    A.u = u;
    dec_slice<<<(unsigned)((int64_t)R * G * ((A.Hx + kSliceH - 1) / kSliceH)), 256, 0, st>>>(A);
}

}  // namespace tag

using namespace tag;

extern "C" tag_status tag_gnn_decide_workspace(const tag_graph *g, const tag_model_dims *dims, int32_t n_replicas,
                                               int32_t n_slices, int32_t n_query, size_t *bytes) {
    clear_error();
    if (!g || !dims || !bytes) TAG_FAIL(TAG_EINVAL, "graph, dims and bytes must be non-NULL");
    if (n_replicas < 1 || n_slices < 1 || n_query < 0) TAG_FAIL(TAG_EINVAL, "need n_replicas >= 1, n_slices >= 1, n_query >= 0");
    if (dims->dec_hidden < 0 || dims->dec_hidden > 1024) TAG_FAIL(TAG_ESHAPE, "dec_hidden must be in [0, 1024]");
    DecLayout L;
    *bytes = carve_dec(g, std::max(dims->dec_hidden, 1), n_replicas, n_slices, n_query, nullptr, &L);
    return TAG_OK;
}

namespace tag {
namespace {

// The body of tag_gnn_decide over a workspace of ws_bytes at `workspace`
// (the caller's buffer, or the library's static scratch).
tag_status decide_run(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w, int32_t n_replicas,
                      const float *E_op, const float *E_dev, const tag_slices *slices, int32_t n_query,
                      const int32_t *query_rep, const int32_t *query_graph, const int32_t *query_op,
                      int32_t *argmax, float *best_score, float *prior, tag_decision *decision, void *workspace,
                      size_t ws_bytes, void *hip_stream, const char *ws_what) {
    if (!g || !dims || !w || !E_op || !E_dev || !slices) TAG_FAIL(TAG_EINVAL, "NULL argument");
    if (dims->f != 64 && dims->f != 128 && dims->f != 256) TAG_FAIL(TAG_ESHAPE, "f must be 64, 128 or 256");
    if (dims->dec_hidden < 0 || dims->dec_hidden > 1024) TAG_FAIL(TAG_ESHAPE, "dec_hidden must be in [0, 1024]");
    if (n_replicas < 1) TAG_FAIL(TAG_EINVAL, "n_replicas must be >= 1");
    if (slices->n_slices < 1 || !slices->mask || !slices->option) TAG_FAIL(TAG_EINVAL, "empty or NULL slice table");
    if (n_query < 0) TAG_FAIL(TAG_EINVAL, "n_query must be >= 0");
    if (n_query == 0) return TAG_OK;
    if (!query_rep || !query_graph || !query_op || !argmax || !best_score)
        TAG_FAIL(TAG_EINVAL, "query arrays, argmax and best_score must be non-NULL");
    if (!w->dec_w2 || !w->dec_b2 || (dims->dec_hidden > 0 && (!w->dec_w1 || !w->dec_b1)))
        TAG_FAIL(TAG_EINVAL, "decoder weights must be non-NULL");
    if (!workspace) TAG_FAIL(TAG_EINVAL, "workspace must be non-NULL");
    const int32_t H = dims->dec_hidden, Hx = std::max(H, 1);
    DecLayout L;
    const size_t need = carve_dec(g, Hx, n_replicas, slices->n_slices, n_query, nullptr, &L);
    if (need > ws_bytes)
        TAG_FAIL(TAG_ENOSPACE, std::string(ws_what) + ": needs " + std::to_string(need) + " bytes, has " +
                                   std::to_string(ws_bytes));
    carve_dec(g, Hx, n_replicas, slices->n_slices, n_query, workspace, &L);
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    DecArgs A{};
    A.R = n_replicas; A.G = g->G; A.S = slices->n_slices; A.Q = n_query; A.F = dims->f; A.H = H; A.Hx = Hx;
    A.n_op = g->n_op; A.n_dev = g->n_dev;
    A.op_off = g->op_off_d; A.dev_off = g->dev_off_d;
    A.E_op = E_op; A.E_dev = E_dev;
    A.mask = slices->mask; A.option = slices->option;
    A.P = H > 0 ? w->dec_w1 : w->dec_w2;
    A.b1 = w->dec_b1; A.w2 = w->dec_w2; A.b2 = w->dec_b2;
    A.q_rep = query_rep; A.q_graph = query_graph; A.q_op = query_op;
    A.t = L.t; A.u = L.u; A.v = L.v;
    A.argmax = argmax; A.best = best_score; A.prior = prior; A.dec = decision;
    const int din = 2 * A.F + 4;
    prof_begin(TAG_STAGE_DECIDE, stream);
    // t = E_dev W1_dev^T and v = E_op[query rows] W1_op^T as MFMA GEMMs
    launch_small_gemm(SmallGemm{E_dev, A.F, (int64_t)A.R * A.n_dev, nullptr, A.F, A.P, din, Hx, nullptr, 0,
                                A.t, Hx, 0}, stream);
    dec_query_rows<<<grid_for(A.Q), 256, 0, stream>>>(A, L.qrow);
    launch_small_gemm(SmallGemm{E_op, A.F, A.Q, L.qrow, A.F, A.P + A.F, din, Hx, nullptr, 0, A.v, Hx, 0}, stream);
    dec_slice<<<(unsigned)((int64_t)A.R * A.G * ((Hx + kSliceH - 1) / kSliceH)), 256, 0, stream>>>(A);
    // four queries per block once there are enough blocks to fill the GPU
    if (A.Q >= 8192)
        dec_score<4><<<(unsigned)((A.Q + 3) / 4), kScoreThreads, sizeof(float) * (4 * Hx + H), stream>>>(A);
    else
        dec_score<1><<<(unsigned)A.Q, kScoreThreads, sizeof(float) * (Hx + H), stream>>>(A);
    prof_end(TAG_STAGE_DECIDE, stream);
    return launch_status("tag_gnn_decide");
}

// Static scratch of the allocation-free entry point: one copy per GPU the
// library runs on, held until the process ends.  Host code never passes the
// symbol itself to a kernel (on the host it only names the variable); it
// passes the device address hipGetSymbolAddress returns for the current
// device, looked up once per device.
constexpr size_t kDecideScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kDecideScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

tag_status scratch_for_current_device(void **out) {
    int dev = -1;
    TAG_HIP_CHECK(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) TAG_FAIL(TAG_EINVAL, "device index out of range for the static scratch");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        TAG_HIP_CHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) TAG_FAIL(TAG_EHIP, "hipGetSymbolAddress returned NULL for the static scratch");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TAG_OK;
}

}  // namespace
}  // namespace tag

extern "C" tag_status tag_gnn_decide(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                     int32_t n_replicas, const float *E_op, const float *E_dev,
                                     const tag_slices *slices, int32_t n_query, const int32_t *query_rep,
                                     const int32_t *query_graph, const int32_t *query_op, int32_t *argmax,
                                     float *best_score, float *prior, tag_decision *decision, void *workspace,
                                     size_t ws_bytes, void *hip_stream) {
    clear_error();
    return decide_run(g, dims, w, n_replicas, E_op, E_dev, slices, n_query, query_rep, query_graph, query_op,
                      argmax, best_score, prior, decision, workspace, ws_bytes, hip_stream,
                      "decide workspace too small (see tag_gnn_decide_workspace)");
}

extern "C" size_t tag_gnn_decide_noalloc_max_bytes(void) { return kDecideScratchBytes; }

extern "C" tag_status tag_gnn_decide_noalloc(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                             int32_t n_replicas, const float *E_op, const float *E_dev,
                                             const tag_slices *slices, int32_t n_query, const int32_t *query_rep,
                                             const int32_t *query_graph, const int32_t *query_op,
                                             int32_t *argmax, float *best_score, float *prior,
                                             tag_decision *decision, void *hip_stream) {
    clear_error();
    void *ws = nullptr;
    const tag_status st = scratch_for_current_device(&ws);
    if (st != TAG_OK) return st;
    return decide_run(g, dims, w, n_replicas, E_op, E_dev, slices, n_query, query_rep, query_graph, query_op,
                      argmax, best_score, prior, decision, ws, kDecideScratchBytes, hip_stream,
                      "problem exceeds the static decide scratch (tag_gnn_decide_noalloc_max_bytes)");
}

// ------------------------------------------------------------ full enumeration
// Every non-empty device mask of the query's topology (n_dev <= 16) with each
// of the four options: slice a = 4 (mask - 1) + option.  Wavefronts walk
// Gray-code ranges of masks, so consecutive masks differ in one device and
// the device part of the pre-activation changes by one row of t; lanes hold
// hidden units (HPL per lane) and a wavefront sum per option gives the
// score.  Per-block (max, sum, argmax) records are merged per query in block
// order; priors are normalised in a second pass.
namespace tag {
namespace {

struct FullArgs {
    DecArgs A;
    int32_t NB;            // blocks per query
    int32_t S_full;        // 4 (2^max_dev - 1): prior row stride
    float *rec;            // [Q][NB][4]: max, sum, argmax (as float bits), valid
};

__device__ __forceinline__ float wave_sum(float v) {
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

template <int HPL>
__global__ void __launch_bounds__(256) dec_full(FullArgs FA) {
    const DecArgs &A = FA.A;
    extern __shared__ float sh[];   // t rows [16][Hx] | base [4][Hx] | w2 [Hx]
    __shared__ float rm[4], rz[4];
    __shared__ int32_t ri[4];
    const int32_t q = blockIdx.x / FA.NB, c = blockIdx.x % FA.NB;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int Hx = A.Hx;
    int32_t r, g, op;
    float *rec = FA.rec + ((int64_t)q * FA.NB + c) * 4;
    if (!query_valid(A, q, &r, &g, &op)) {
        if (threadIdx.x == 0) { rec[0] = -INFINITY; rec[1] = 0.f; rec[2] = __int_as_float(INT32_MAX); rec[3] = 0.f; }
        return;
    }
    const int32_t d0 = A.dev_off[g], nd = A.dev_off[g + 1] - d0;
    float *tl = sh, *base = sh + 16 * Hx, *w2s = base + 4 * Hx;
    const int din = 2 * A.F + 4;
    for (int i = threadIdx.x; i < nd * Hx; i += blockDim.x)
        tl[i] = A.t[((int64_t)r * A.n_dev + d0 + i / Hx) * Hx + i % Hx];
    for (int i = threadIdx.x; i < 4 * Hx; i += blockDim.x) {
        const int o = i / Hx, h = i % Hx;
        base[i] = A.P[(int64_t)h * din + 2 * A.F + o] + (A.H > 0 ? A.b1[h] : 0.f) + A.v[(int64_t)q * Hx + h];
    }
    for (int h = threadIdx.x; h < Hx; h += blockDim.x) w2s[h] = A.H > 0 ? A.w2[h] : 0.f;
    __syncthreads();
    // this wavefront's Gray range
    const int64_t total = (int64_t)1 << nd;
    const int64_t W = (int64_t)FA.NB * 4, wid = (int64_t)c * 4 + wv;
    const int64_t len = (total + W - 1) / W;
    const int64_t g0 = wid * len, g1 = g0 + len < total ? g0 + len : total;
    float m = -INFINITY, z = 0.f;
    int32_t im = INT32_MAX;
    if (g0 < g1) {
        float ds[HPL];
        uint32_t mask = (uint32_t)(g0 ^ (g0 >> 1));
#pragma unroll
        for (int i = 0; i < HPL; ++i) {
            const int h = lane + 64 * i;
            float s = 0.f;
            for (int j = 0; j < nd; ++j)
                if ((mask >> j) & 1u) s += h < Hx ? tl[j * Hx + h] : 0.f;
            ds[i] = s;
        }
        for (int64_t gi = g0; gi < g1; ++gi) {
            if (gi > g0) {
                const int j = __builtin_ctzll((unsigned long long)gi);
                mask ^= 1u << j;
                const float sg = ((mask >> j) & 1u) ? 1.f : -1.f;
#pragma unroll
                for (int i = 0; i < HPL; ++i) {
                    const int h = lane + 64 * i;
                    if (h < Hx) ds[i] = fmaf(sg, tl[j * Hx + h], ds[i]);
                }
            }
            if (mask == 0) continue;
#pragma unroll
            for (int o = 0; o < 4; ++o) {
                float s;
                if (A.H == 0) {   // linear head: Hx = 1, lane 0 holds the sums
                    s = A.b2[0] + __shfl(ds[0] + base[o], 0, 64);
                } else {
                    float p = 0.f;
#pragma unroll
                    for (int i = 0; i < HPL; ++i) {
                        const int h = lane + 64 * i;
                        if (h < Hx) p = fmaf(w2s[h], fmaxf(ds[i] + base[o * Hx + h], 0.f), p);
                    }
                    s = A.b2[0] + wave_sum(p);
                }
                const int32_t a = (int32_t)(4 * (mask - 1) + o);
                if (A.prior && lane == 0) A.prior[(int64_t)q * FA.S_full + a] = s;
                if (s > m) { z = z * __expf(m - s) + 1.f; m = s; im = a; }
                else { z += __expf(s - m); if (s == m && a < im) im = a; }
            }
        }
    }
    if (lane == 0) { rm[wv] = m; rz[wv] = z; ri[wv] = im; }
    __syncthreads();
    if (threadIdx.x == 0) {
        float M = -INFINITY, Z = 0.f;
        int32_t I = INT32_MAX;
        for (int k = 0; k < 4; ++k) {
            const float m2 = rm[k];
            if (m2 == -INFINITY) continue;
            const float nm = fmaxf(M, m2);
            Z = (M == -INFINITY ? 0.f : Z * __expf(M - nm)) + rz[k] * __expf(m2 - nm);
            if (m2 > M || (m2 == M && ri[k] < I)) I = ri[k];
            M = nm;
        }
        rec[0] = M; rec[1] = Z; rec[2] = __int_as_float(I); rec[3] = 1.f;
    }
}

// One lane per run of kFullRun consecutive Gray indices from an aligned
// start (H <= 128): the device part of the pre-activation lives in the
// lane's registers, and since all lanes sit at the same offset inside
// their runs, every step toggles the same device j = ctz(step) in all
// lanes; the t row of j, the option bases and w2 are wave-uniform LDS reads.
constexpr int kFullRun = 16;

struct FullTpm {
    FullArgs FA;
    const float *base;     // [Q][4][HP]: W1_opt + b1 + v_q (zero past H)
    const float *w2p;      // [HP] (zero past H)
};

template <int HP>
__global__ void __launch_bounds__(256) dec_full_tpm(FullTpm T) {
    const FullArgs &FA = T.FA;
    const DecArgs &A = FA.A;
    __shared__ float rm[4], rz[4];
    __shared__ int32_t ri[4];
    const int32_t q = blockIdx.x / FA.NB, c = blockIdx.x % FA.NB;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    int32_t r, g, op;
    float *rec = FA.rec + ((int64_t)q * FA.NB + c) * 4;
    if (!query_valid(A, q, &r, &g, &op)) {
        if (threadIdx.x == 0) { rec[0] = -INFINITY; rec[1] = 0.f; rec[2] = __int_as_float(INT32_MAX); rec[3] = 0.f; }
        return;
    }
    const int32_t d0 = A.dev_off[g], nd = A.dev_off[g + 1] - d0;
    const int H = A.Hx;
    const int64_t total = (int64_t)1 << nd;
    const int run = total < kFullRun ? (int)total : kFullRun;
    const int64_t g0 = ((int64_t)c * 256 + threadIdx.x) * run;
    // the query's option bases, w2 and the topology's t rows (zero past H), read
    // as LDS broadcasts in the inner loops
    __shared__ float sbq[4 * HP], sw2[HP], strow[16 * HP];
    for (int i = threadIdx.x; i < 4 * HP; i += 256) sbq[i] = T.base[(int64_t)q * 4 * HP + i];
    for (int i = threadIdx.x; i < HP; i += 256) sw2[i] = T.w2p[i];
    for (int i = threadIdx.x; i < nd * HP; i += 256) {
        const int j = i / HP, h = i % HP;
        strow[i] = h < H ? A.t[((int64_t)r * A.n_dev + d0 + j) * H + h] : 0.f;
    }
    __syncthreads();
    const float *trow = strow;
    const float *bq = sbq;
    float m = -INFINITY, z = 0.f;
    int32_t im = INT32_MAX;
    if (g0 < total) {
        uint32_t mask = (uint32_t)(g0 ^ (g0 >> 1));
        float ds[HP];
#pragma unroll
        for (int h = 0; h < HP; ++h) ds[h] = 0.f;
        for (int j = 0; j < nd; ++j) {
            if (!((mask >> j) & 1u)) continue;
#pragma unroll
            for (int h = 0; h < HP; ++h)
                ds[h] += trow[j * HP + h];
        }
        for (int st = 0; st < run; ++st) {
            // read the LDS constants afresh for every mask: held in registers across
            // the loop they would take 640 of them (one wavefront per SIMD, spills)
            asm volatile("" ::: "memory");
            if (st > 0) {
                const int j = __builtin_ctz((unsigned)st);   // same in every lane
                mask ^= 1u << j;
                const float sg = ((mask >> j) & 1u) ? 1.f : -1.f;
#pragma unroll
                for (int h = 0; h < HP; ++h)
                    ds[h] = fmaf(sg, trow[j * HP + h], ds[h]);
            }
            if (mask == 0) continue;
            float s[4];
#pragma unroll
            for (int o = 0; o < 4; ++o) {
                float acc = 0.f;
#pragma unroll
                for (int h = 0; h < HP; ++h) acc = fmaf(sw2[h], fmaxf(ds[h] + bq[o * HP + h], 0.f), acc);
                s[o] = A.b2[0] + acc;
            }
            const int32_t a0 = (int32_t)(4 * (mask - 1));
            if (A.prior)
                *reinterpret_cast<float4 *>(A.prior + (int64_t)q * FA.S_full + a0) = float4{s[0], s[1], s[2], s[3]};
#pragma unroll
            for (int o = 0; o < 4; ++o) {
                if (s[o] > m) { z = z * __expf(m - s[o]) + 1.f; m = s[o]; im = a0 + o; }
                else { z += __expf(s[o] - m); if (s[o] == m && a0 + o < im) im = a0 + o; }
            }
        }
    }
    // wavefront merge of the lanes' (max, sum, argmax), then the block's four
    for (int o = 32; o >= 1; o >>= 1) {
        const float m2 = __shfl_xor(m, o, 64), z2 = __shfl_xor(z, o, 64);
        const int32_t i2 = __shfl_xor(im, o, 64);
        const float nm = fmaxf(m, m2);
        if (nm != -INFINITY) {
            z = (m == -INFINITY ? 0.f : z * __expf(m - nm)) + (m2 == -INFINITY ? 0.f : z2 * __expf(m2 - nm));
            if (m2 > m || (m2 == m && i2 < im)) im = i2;
            m = nm;
        }
    }
    if (lane == 0) { rm[wv] = m; rz[wv] = z; ri[wv] = im; }
    __syncthreads();
    if (threadIdx.x == 0) {
        float M = -INFINITY, Z = 0.f;
        int32_t I = INT32_MAX;
        for (int k = 0; k < 4; ++k) {
            const float m2 = rm[k];
            if (m2 == -INFINITY) continue;
            const float nm = fmaxf(M, m2);
            Z = (M == -INFINITY ? 0.f : Z * __expf(M - nm)) + rz[k] * __expf(m2 - nm);
            if (m2 > M || (m2 == M && ri[k] < I)) I = ri[k];
            M = nm;
        }
        rec[0] = M; rec[1] = Z; rec[2] = __int_as_float(I); rec[3] = 1.f;
    }
}

// option bases of every query and the padded readout
__global__ void dec_full_base(DecArgs A, int HP, float *base, float *w2p) {
    const int din = 2 * A.F + 4;
    const int64_t total = (int64_t)A.Q * 4 * HP;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int h = (int)(i % HP), o = (int)((i / HP) % 4);
        const int64_t q = i / (4 * HP);
        base[i] = h < A.H ? A.P[(int64_t)h * din + 2 * A.F + o] + A.b1[h] + A.v[q * A.Hx + h] : 0.f;
        if (i < HP) w2p[i] = i < A.H ? A.w2[i] : 0.f;
    }
}

// per query: merge the block records in order, decode the argmax, then
// normalise the priors of the query's slices (zeros beyond them)
__global__ void __launch_bounds__(256) dec_full_merge(FullArgs FA) {
    const DecArgs &A = FA.A;
    __shared__ float sM, sZ;
    const int32_t q = blockIdx.x;
    int32_t r, g, op;
    const bool ok = query_valid(A, q, &r, &g, &op);
    const int32_t nd = ok ? A.dev_off[g + 1] - A.dev_off[g] : 0;
    const int32_t S_q = ok ? 4 * ((1 << nd) - 1) : 0;
    if (threadIdx.x == 0) {
        float M = -INFINITY, Z = 0.f;
        int32_t I = INT32_MAX;
        for (int32_t c = 0; c < FA.NB; ++c) {
            const float *rec = FA.rec + ((int64_t)q * FA.NB + c) * 4;
            const float m2 = rec[0];
            if (!(rec[3] > 0.f) || m2 == -INFINITY) continue;
            const float nm = fmaxf(M, m2);
            Z = (M == -INFINITY ? 0.f : Z * __expf(M - nm)) + rec[1] * __expf(m2 - nm);
            const int32_t i2 = __float_as_int(rec[2]);
            if (m2 > M || (m2 == M && i2 < I)) I = i2;
            M = nm;
        }
        sM = M;
        sZ = Z;
        if (!ok || I == INT32_MAX) {
            A.argmax[q] = -1;
            A.best[q] = __builtin_nanf("");
            if (A.dec) A.dec[q] = tag_decision{0, 0, 0, 0, 0};
        } else {
            A.argmax[q] = I;
            A.best[q] = M;
            if (A.dec) {
                const uint64_t msk = (uint64_t)(I / 4 + 1);
                const int o = I % 4;
                const int pc = __popcll(msk);
                A.dec[q] = tag_decision{msk, o, o == 3 ? 1 : pc, o == 0 ? 0 : (o == 1 ? 1 : 2), o == 2 ? 1 : 0};
            }
        }
    }
    __syncthreads();
    if (!A.prior) return;
    const float M = sM, inv = sZ > 0.f ? 1.f / sZ : 0.f;
    float *row = A.prior + (int64_t)q * FA.S_full;
    for (int32_t a = threadIdx.x; a < FA.S_full; a += blockDim.x)
        row[a] = a < S_q && ok ? __expf(row[a] - M) * inv : 0.f;
}

struct FullLayout {
    float *t, *v, *rec, *base, *w2p;
    int32_t *qrow;
};

// padded hidden width of the lane-per-mask kernel (0: lanes over hidden units)
int full_hp(int32_t H) { return H == 0 || H > 128 ? 0 : (H <= 32 ? 32 : (H <= 64 ? 64 : 128)); }

int32_t full_blocks(int32_t Q, int32_t max_dev, int32_t H) {
    const int64_t masks = (int64_t)1 << max_dev;
    if (full_hp(H))   // one lane per run of kFullRun masks
        return (int32_t)std::max<int64_t>(1, (masks / kFullRun + 255) / 256);
    // enough blocks to fill the chip, at least 64 masks per wavefront
    const int64_t by_work = std::max<int64_t>(1, masks / (4 * 64));
    const int64_t by_fill = std::max<int64_t>(1, 2048 / std::max(Q, 1));
    return (int32_t)std::min(by_work, by_fill);
}

size_t carve_full(const tag_graph *g, int32_t H, int32_t R, int32_t Q, void *base, FullLayout *L) {
    Carver c(base);
    const int32_t Hx = std::max(H, 1);
    L->t = c.take<float>((size_t)R * g->n_dev * Hx);
    L->v = c.take<float>((size_t)std::max(Q, 1) * Hx);
    L->rec = c.take<float>((size_t)std::max(Q, 1) * full_blocks(Q, g->max_dev, H) * 4);
    L->qrow = c.take<int32_t>((size_t)std::max(Q, 1));
    const int hp = full_hp(H);
    L->base = hp ? c.take<float>((size_t)std::max(Q, 1) * 4 * hp) : nullptr;
    L->w2p = hp ? c.take<float>((size_t)hp) : nullptr;
    return c.used;
}

}  // namespace
}  // namespace tag

extern "C" tag_status tag_gnn_decide_full_workspace(const tag_graph *g, const tag_model_dims *dims,
                                                    int32_t n_replicas, int32_t n_query, size_t *bytes) {
    clear_error();
    if (!g || !dims || !bytes) TAG_FAIL(TAG_EINVAL, "graph, dims and bytes must be non-NULL");
    if (n_replicas < 1 || n_query < 0) TAG_FAIL(TAG_EINVAL, "need n_replicas >= 1, n_query >= 0");
    if (dims->dec_hidden < 0 || dims->dec_hidden > 512) TAG_FAIL(TAG_ESHAPE, "full enumeration needs dec_hidden <= 512");
    if (g->max_dev > 16) TAG_FAIL(TAG_ESHAPE, "full enumeration needs at most 16 devices per topology");
    FullLayout L;
    *bytes = carve_full(g, dims->dec_hidden, n_replicas, n_query, nullptr, &L);
    return TAG_OK;
}

extern "C" tag_status tag_gnn_decide_full(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                          int32_t n_replicas, const float *E_op, const float *E_dev,
                                          int32_t n_query, const int32_t *query_rep, const int32_t *query_graph,
                                          const int32_t *query_op, int32_t *argmax, float *best_score,
                                          float *prior, tag_decision *decision, void *workspace, size_t ws_bytes,
                                          void *hip_stream) {
    clear_error();
    if (!g || !dims || !w || !E_op || !E_dev) TAG_FAIL(TAG_EINVAL, "NULL argument");
    if (dims->f != 64 && dims->f != 128 && dims->f != 256) TAG_FAIL(TAG_ESHAPE, "f must be 64, 128 or 256");
    if (dims->dec_hidden < 0 || dims->dec_hidden > 512) TAG_FAIL(TAG_ESHAPE, "full enumeration needs dec_hidden <= 512");
    if (g->max_dev > 16) TAG_FAIL(TAG_ESHAPE, "full enumeration needs at most 16 devices per topology");
    if (n_replicas < 1) TAG_FAIL(TAG_EINVAL, "n_replicas must be >= 1");
    if (n_query < 0) TAG_FAIL(TAG_EINVAL, "n_query must be >= 0");
    if (n_query == 0) return TAG_OK;
    if (!query_rep || !query_graph || !query_op || !argmax || !best_score)
        TAG_FAIL(TAG_EINVAL, "query arrays, argmax and best_score must be non-NULL");
    if (!w->dec_w2 || !w->dec_b2 || (dims->dec_hidden > 0 && (!w->dec_w1 || !w->dec_b1)))
        TAG_FAIL(TAG_EINVAL, "decoder weights must be non-NULL");
    if (!workspace) TAG_FAIL(TAG_EINVAL, "workspace must be non-NULL");
    const int32_t H = dims->dec_hidden, Hx = std::max(H, 1);
    FullLayout L;
    if (carve_full(g, H, n_replicas, n_query, nullptr, &L) > ws_bytes)
        TAG_FAIL(TAG_ENOSPACE, "workspace too small (see tag_gnn_decide_full_workspace)");
    carve_full(g, H, n_replicas, n_query, workspace, &L);
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    FullArgs FA{};
    DecArgs &A = FA.A;
    A.R = n_replicas; A.G = g->G; A.S = 0; A.Q = n_query; A.F = dims->f; A.H = H; A.Hx = Hx;
    A.n_op = g->n_op; A.n_dev = g->n_dev;
    A.op_off = g->op_off_d; A.dev_off = g->dev_off_d;
    A.E_op = E_op; A.E_dev = E_dev;
    A.P = H > 0 ? w->dec_w1 : w->dec_w2;
    A.b1 = w->dec_b1; A.w2 = w->dec_w2; A.b2 = w->dec_b2;
    A.q_rep = query_rep; A.q_graph = query_graph; A.q_op = query_op;
    A.t = L.t; A.v = L.v;
    A.argmax = argmax; A.best = best_score; A.prior = prior; A.dec = decision;
    FA.NB = full_blocks(n_query, g->max_dev, H);
    FA.S_full = 4 * ((1 << std::max(g->max_dev, 1)) - 1);
    FA.rec = L.rec;
    const int din = 2 * A.F + 4;
    launch_small_gemm(SmallGemm{E_dev, A.F, (int64_t)A.R * A.n_dev, nullptr, A.F, A.P, din, Hx, nullptr, 0,
                                A.t, Hx, 0}, stream);
    dec_query_rows<<<grid_for(A.Q), 256, 0, stream>>>(A, L.qrow);
    launch_small_gemm(SmallGemm{E_op, A.F, A.Q, L.qrow, A.F, A.P + A.F, din, Hx, nullptr, 0, A.v, Hx, 0}, stream);
    const unsigned grid = (unsigned)((int64_t)n_query * FA.NB);
    const int hp = full_hp(H);
    if (hp) {
        dec_full_base<<<grid_for((int64_t)n_query * 4 * hp), 256, 0, stream>>>(A, hp, L.base, L.w2p);
        FullTpm T{FA, L.base, L.w2p};
        if (hp == 32) dec_full_tpm<32><<<grid, 256, 0, stream>>>(T);
        else if (hp == 64) dec_full_tpm<64><<<grid, 256, 0, stream>>>(T);
        else dec_full_tpm<128><<<grid, 256, 0, stream>>>(T);
        dec_full_merge<<<(unsigned)n_query, 256, 0, stream>>>(FA);
        return launch_status("tag_gnn_decide_full");
    }
    const size_t sh = sizeof(float) * (size_t)21 * Hx;
    const int hpl = (Hx + 63) / 64;
    if (hpl <= 1) dec_full<1><<<grid, 256, sh, stream>>>(FA);
    else if (hpl <= 2) dec_full<2><<<grid, 256, sh, stream>>>(FA);
    else if (hpl <= 4) dec_full<4><<<grid, 256, sh, stream>>>(FA);
    else dec_full<8><<<grid, 256, sh, stream>>>(FA);
    dec_full_merge<<<(unsigned)n_query, 256, 0, stream>>>(FA);
    return launch_status("tag_gnn_decide_full");
}
