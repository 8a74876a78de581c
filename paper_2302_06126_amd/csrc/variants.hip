// Readings of the layer equation of Section 4.2.1 that the paper leaves open,
// on a generic fp32 path:
//  * five directed relations: op<-op along the tensor (row = consumer),
//    op<-op against it (row = producer), op<-device, device<-op and
//    device<-device, each with its own W = [W^h | W^e], b, a, adst and
//    softmax (the default reading has three undirected link types);
//  * ReLU after the fully connected edge encoders (default: affine);
//  * K attention heads over all f channels, each with its own attention
//    vectors, averaged (default: K concatenated heads of f/K channels).
// Per layer: W^h h of every node for every relation that touches its type
// (MFMA GEMMs, no folded bias), the edge terms W^e e + b of every link as
// tables, then one wavefront per destination row walks each incoming
// relation's entries with an online softmax per head and writes
// h' = sum_r gamma_r agg_r once.
#include <algorithm>

#include "agg_common.hpp"
#include "fwd_internal.hpp"
#include "transform.hpp"

namespace tag {
namespace {

constexpr int kVarMaxAvgHeads = 8;

__global__ void fill_zero(float *p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0.f;
}

// ------------------------------------------------------------ edge terms
// te[row][c] = b[c] + sum_k W^e[c][k] act(A[k] . x_row + cA[k]); one block
// per table row, the encoded edge vector staged in LDS.
struct EdgeTermArgs {
    const float *We;      // W of the relation: row c at We + c * 2F, W^e = columns [F, 2F)
    const float *b;       // [F]
    const float *A;       // encoder [F][d]
    const float *cA;      // encoder bias [F]
    int d, F, relu;
    // raw feature of table row i: od (d = 1, two rows): x = i; otherwise
    // x = feat[(i / n_links) * stride + (i % n_links) * d + t]
    const float *feat;
    int64_t n_links, stride;
    int bits;             // 1: the rows are the placement bits 0 and 1
    float *te;            // [rows][F]
};

__global__ void __launch_bounds__(256) var_edge_terms(EdgeTermArgs a) {
    __shared__ float enc[256];
    const int64_t i = blockIdx.x;
    const int F = a.F;
    float x0, x1 = 0.f;
    if (a.bits) {
        x0 = (float)i;
    } else {
        const float *xr = a.feat + (i / a.n_links) * a.stride + (i % a.n_links) * a.d;
        x0 = xr[0];
        if (a.d == 2) x1 = xr[1];
    }
    for (int k = threadIdx.x; k < F; k += blockDim.x) {
        float e = a.cA[k] + a.A[(size_t)k * a.d] * x0;
        if (a.d == 2) e = fmaf(a.A[(size_t)k * a.d + 1], x1, e);
        enc[k] = a.relu ? fmaxf(e, 0.f) : e;
    }
    __syncthreads();
    for (int c = threadIdx.x; c < F; c += blockDim.x) {
        const float *wr = a.We + (size_t)c * 2 * F + F;
        float s = a.b[c];
        for (int k = 0; k < F; ++k) s = fmaf(wr[k], enc[k], s);
        a.te[i * F + c] = s;
    }
}

// ------------------------------------------------------------ aggregation
struct VarRel {
    int bucket;              // CSR bucket holding the destination rows
    int dir;                 // bucket 0 only: 0 every entry, 1 forward (row = consumer), 2 backward
    const float *ysrc;       // W^h h of the sources: row (rep * n_src + v) at ysrc + row * ldy
    const float *ydst;       // W^h h of the destinations: row (rep * n_dst + u)
    int64_t n_src;
    int ldy;
    const float *te;         // edge terms: [rows][F]
    int te_bits;             // 1: two rows, selected by the link's placement bit
    int64_t te_rep;          // replica stride of te in rows (0: shared)
    const float *as, *ad;    // attention vectors ([F], or [K][F] for averaged heads)
    float gamma;
};

struct VarArgs {
    int R, F, K, avg;
    float slope;
    int64_t n_dst;           // destination rows per replica
    const int32_t *rp[4], *col[4], *eid[4];
    const int32_t *oo_head;
    const uint8_t *x_od;
    int64_t s_od;
    int n_rel;
    VarRel rel[3];
    float *out;              // [R * n_dst][F]
};

__device__ __forceinline__ float group_sum(float v, int width) {
    for (int o = width / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One wavefront per (replica, destination row); lane l owns channels
// [l CPL, (l + 1) CPL).  Concatenated heads: head k = channels of lanes
// [k 64/K, (k+1) 64/K); averaged heads: every head spans all lanes.
template <int CPL>
__global__ void __launch_bounds__(256) agg_var(VarArgs A) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (int64_t)A.R * A.n_dst) return;
    const int32_t rep = (int32_t)(w / A.n_dst);
    const int32_t u = (int32_t)(w % A.n_dst);
    const int F = A.F, K = A.K;
    const int c0 = lane * CPL;
    const int lph = 64 / K;               // concatenated heads: lanes per head
    const int nh = A.avg ? K : 1;         // heads this lane tracks
    float out[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) out[c] = 0.f;
    for (int ri = 0; ri < A.n_rel; ++ri) {
        const VarRel &V = A.rel[ri];
        const int32_t beg = A.rp[V.bucket][u], end = A.rp[V.bucket][u + 1];
        if (beg == end) continue;
        float yd[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) yd[c] = V.ydst[((int64_t)rep * A.n_dst + u) * V.ldy + c0 + c];
        // destination terms (exp2 domain)
        float qd[kVarMaxAvgHeads];
        for (int k = 0; k < nh; ++k) {
            const float *ad = V.ad + (A.avg ? (size_t)k * F : 0);
            float q = 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) q = fmaf(ad[c0 + c], yd[c], q);
            qd[k] = A.avg ? group_sum(q, 64) : group_sum(q, lph);
        }
        float mx[kVarMaxAvgHeads], den[kVarMaxAvgHeads], acc[kVarMaxAvgHeads][CPL];
        for (int k = 0; k < nh; ++k) {
            mx[k] = -INFINITY;
            den[k] = 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) acc[k][c] = 0.f;
        }
        const uint8_t *xb = A.x_od + (int64_t)rep * A.s_od;
        for (int32_t e = beg; e < end; ++e) {
            const int32_t v = A.col[V.bucket][e], id = A.eid[V.bucket][e];
            if (V.dir) {
                const bool fwd = A.oo_head[id] == u;
                if (fwd != (V.dir == 1)) continue;
            }
            const float *te = V.te + ((V.te_bits ? (xb[id] ? 1 : 0) : id) + (int64_t)rep * V.te_rep) * F;
            float m[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                m[c] = fmaxf(V.ysrc[((int64_t)rep * V.n_src + v) * V.ldy + c0 + c] + te[c0 + c], 0.f);
            for (int k = 0; k < nh; ++k) {
                const float *as = V.as + (A.avg ? (size_t)k * F : 0);
                float part = 0.f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) part = fmaf(as[c0 + c], m[c], part);
                const float s = (A.avg ? group_sum(part, 64) : group_sum(part, lph)) + qd[k];
                const float s2 = (s > 0.f ? s : A.slope * s) * kLog2e;
                const float nm = fmaxf(mx[k], s2);
                const float sc = __builtin_amdgcn_exp2f(mx[k] - nm);
                const float p = __builtin_amdgcn_exp2f(s2 - nm);
                den[k] = fmaf(den[k], sc, p);
#pragma unroll
                for (int c = 0; c < CPL; ++c) acc[k][c] = fmaf(acc[k][c], sc, p * m[c]);
                mx[k] = nm;
            }
        }
        const float g = A.avg ? V.gamma / K : V.gamma;
        for (int k = 0; k < nh; ++k) {
            if (den[k] <= 0.f) continue;   // no entry of this direction
            const float inv = g / den[k];
#pragma unroll
            for (int c = 0; c < CPL; ++c) out[c] = fmaf(acc[k][c], inv, out[c]);
        }
    }
    float *o = A.out + ((int64_t)rep * A.n_dst + u) * F + c0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[c] = out[c];
}

// ------------------------------------------------------------ planning
struct VarLayout {
    float *H_op[2], *H_dev[2];
    float *zero;                 // [F] zeros (no bias added by the transform)
    float *Y_opA, *Y_opB, *Y_devA, *Y_devB;   // [rows][2F]
    float *te_oo[2], *te_od[2], *te_dd;
};

size_t carve_var(const tag_graph *g, const tag_model_dims *d, int32_t R, int64_t reps_oo, int64_t reps_dd,
                 void *base, VarLayout *L) {
    Carver c(base);
    const size_t F = d->f, N = (size_t)R * g->n_op, M = (size_t)R * g->n_dev;
    for (int i = 0; i < 2; ++i) {
        L->H_op[i] = c.take<float>(N * F + 1);
        L->H_dev[i] = c.take<float>(M * F + 1);
    }
    L->zero = c.take<float>(F);
    L->Y_opA = c.take<float>(N * 2 * F + 1);
    L->Y_opB = c.take<float>(N * 2 * F + 1);
    L->Y_devA = c.take<float>(M * 2 * F + 1);
    L->Y_devB = c.take<float>(M * 2 * F + 1);
    for (int i = 0; i < 2; ++i) {
        L->te_oo[i] = c.take<float>((size_t)reps_oo * g->e_oo * F + 1);
        L->te_od[i] = c.take<float>(2 * F);
    }
    L->te_dd = c.take<float>((size_t)reps_dd * g->e_dd * F + 1);
    return c.used;
}

// Y = H [W_first ; W_second]^T (W^h blocks of two relations) into [rows][2F], no bias
void var_transform(const tag_model_dims *d, const float *H, int64_t rows, const float *W1, const float *W2,
                   float *Y, const float *zero, hipStream_t st) {
    if (rows == 0) return;
    const int F = d->f;
    GemmArgs ga{};
    ga.F = F;
    ga.prep.jph = 0;
    ga.prep.K = d->heads;
    ga.prep.cp_same[0] = ga.prep.cp_same[1] = zero;
    ga.prep.cp_od = zero;
    ga.tiles0 = transform_row_tiles(rows);
    ga.side[0] = GemmSide{H, rows, W1, W2, 2 * F, Y};
    ga.side[1] = GemmSide{nullptr, 0, W1, W2, 2 * F, nullptr};
    launch_transform(ga, false, st);
}

void var_edge_table(const tag_model_dims *d, const float *W, const float *b, const float *A, const float *cA, int dr,
                    const float *feat, int64_t n_links, int64_t stride, int64_t reps, bool bits, float *te,
                    hipStream_t st) {
    const int64_t rows = bits ? 2 : reps * n_links;
    if (rows == 0) return;
    EdgeTermArgs a{W, b, A, cA, dr, d->f, d->edge_act == 1 ? 1 : 0, feat, std::max<int64_t>(n_links, 1), stride,
                   bits ? 1 : 0, te};
    var_edge_terms<<<(unsigned)rows, 256, 0, st>>>(a);
}

template <int CPL>
void launch_agg_var(const VarArgs &A, hipStream_t st) {
    const int64_t waves = (int64_t)A.R * A.n_dst;
    if (waves == 0) return;
    agg_var<CPL><<<(unsigned)((waves + 3) / 4), 256, 0, st>>>(A);
}

void dispatch_agg_var(int F, const VarArgs &A, hipStream_t st) {
    if (F == 64) launch_agg_var<1>(A, st);
    else if (F == 128) launch_agg_var<2>(A, st);
    else launch_agg_var<4>(A, st);
}

}  // namespace

bool is_variant(const tag_model_dims *d) {
    return (d->relations != 0 && d->relations != 3) || d->edge_act != 0 || d->head_mode != 0;
}

tag_status check_variant(const tag_model_dims *d) {
    if (d->relations != 0 && d->relations != 3 && d->relations != 5) TAG_FAIL(TAG_EINVAL, "relations must be 3 or 5");
    if (d->edge_act != 0 && d->edge_act != 1) TAG_FAIL(TAG_EINVAL, "edge_act must be 0 or 1");
    if (d->head_mode != 0 && d->head_mode != 1) TAG_FAIL(TAG_EINVAL, "head_mode must be 0 or 1");
    if (!is_variant(d)) return TAG_OK;
    if (d->dtype != TAG_F32) TAG_FAIL(TAG_ESHAPE, "the relations / edge_act / head_mode variants run in fp32");
    if (d->sigma != 0) TAG_FAIL(TAG_ESHAPE, "the relations / edge_act / head_mode variants use ReLU messages");
    if (d->head_mode == 1 && d->heads > kVarMaxAvgHeads) TAG_FAIL(TAG_ESHAPE, "averaged heads: at most 8 heads");
    return TAG_OK;
}

size_t variant_workspace(const tag_graph *g, const tag_model_dims *d, int32_t R) {
    VarLayout L;
    // edge tables sized for per-replica features (the caller's strides decide at run time)
    return carve_var(g, d, R, R, R, nullptr, &L);
}

tag_status forward_variant(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                           const tag_features *x, void *workspace, size_t ws_bytes, float *E_op, float *E_dev,
                           hipStream_t stream) {
    const int32_t R = x->n_replicas;
    VarLayout L;
    if (carve_var(g, dims, R, R, R, nullptr, &L) > ws_bytes)
        TAG_FAIL(TAG_ENOSPACE, "workspace too small (see tag_gnn_workspace)");
    carve_var(g, dims, R, R, R, workspace, &L);
    const int F = dims->f, K = dims->heads, NL = dims->layers;
    const int NR = dims->relations == 5 ? 5 : 3;
    const size_t asz = (size_t)(dims->head_mode == 1 ? K : 1) * F;
    const int64_t N = (int64_t)R * g->n_op, M = (int64_t)R * g->n_dev;
    const int64_t reps_oo = x->stride_oo ? R : 1, reps_dd = x->stride_dd ? R : 1;
    fill_zero<<<1, 256, 0, stream>>>(L.zero, F);   // a kernel, not a memset node, so the call stays capturable

    // encoders: h0 = ReLU(A x + c) (fp32)
    SmallGemm eo{x->x_op, dims->f_op, N, nullptr, dims->f_op, w->enc_op_w, dims->f_op, F, w->enc_op_b, 1, L.H_op[0], F, 0};
    SmallGemm ed{x->x_dev, dims->f_dev, M, nullptr, dims->f_dev, w->enc_dev_w, dims->f_dev, F, w->enc_dev_b, 1,
                 L.H_dev[0], F, 0};
    prof_begin(TAG_STAGE_ENCODE, stream);
    launch_small_gemm(eo, stream);
    launch_small_gemm(ed, stream);
    prof_end(TAG_STAGE_ENCODE, stream);

    VarArgs base{};
    base.R = R; base.F = F; base.K = K; base.avg = dims->head_mode == 1 ? 1 : 0;
    base.slope = dims->leaky_slope;
    for (int b = 0; b < 4; ++b) { base.rp[b] = g->rowptr[b]; base.col[b] = g->col[b]; base.eid[b] = g->eid[b]; }
    base.oo_head = g->oo_head;
    base.x_od = x->x_od; base.s_od = x->stride_od;
    for (int l = 0; l < NL; ++l) {
        const float *W[5], *bb[5], *as[5], *ad[5];
        for (int r = 0; r < NR; ++r) {
            W[r] = w->layer_w + ((size_t)l * NR + r) * F * 2 * F;
            bb[r] = w->layer_b + ((size_t)l * NR + r) * F;
            as[r] = w->att_src + ((size_t)l * NR + r) * asz;
            ad[r] = w->att_dst + ((size_t)l * NR + r) * asz;
        }
        const float *Hop = L.H_op[l & 1], *Hdev = L.H_dev[l & 1];
        // relation indices: op<-op (one or two), op<-device, device<-op, device<-device
        const int r_f = 0, r_b = NR == 5 ? 1 : 0, r_od = NR == 5 ? 2 : 1, r_do = NR == 5 ? 3 : 1, r_dd = NR == 5 ? 4 : 2;
        prof_begin(TAG_STAGE_TRANSFORM, stream);
        var_transform(dims, Hop, N, W[r_f], W[r_b], L.Y_opA, L.zero, stream);     // op sources/destinations of op<-op
        var_transform(dims, Hop, N, W[r_od], W[r_do], L.Y_opB, L.zero, stream);   // op destination of op<-dev, source of dev<-op
        var_transform(dims, Hdev, M, W[r_dd], W[r_od], L.Y_devA, L.zero, stream); // dev<-dev; device source of op<-dev
        var_transform(dims, Hdev, M, W[r_do], W[r_do], L.Y_devB, L.zero, stream); // device destination of dev<-op
        prof_end(TAG_STAGE_TRANSFORM, stream);
        // edge-term tables
        var_edge_table(dims, W[r_f], bb[r_f], w->enc_edge_w[0], w->enc_edge_b[0], 1, x->x_oo, g->e_oo, x->stride_oo,
                       reps_oo, false, L.te_oo[0], stream);
        if (NR == 5)
            var_edge_table(dims, W[r_b], bb[r_b], w->enc_edge_w[0], w->enc_edge_b[0], 1, x->x_oo, g->e_oo,
                           x->stride_oo, reps_oo, false, L.te_oo[1], stream);
        var_edge_table(dims, W[r_od], bb[r_od], w->enc_edge_w[1], w->enc_edge_b[1], 1, nullptr, 0, 0, 1, true,
                       L.te_od[0], stream);
        if (NR == 5)
            var_edge_table(dims, W[r_do], bb[r_do], w->enc_edge_w[1], w->enc_edge_b[1], 1, nullptr, 0, 0, 1, true,
                           L.te_od[1], stream);
        var_edge_table(dims, W[r_dd], bb[r_dd], w->enc_edge_w[2], w->enc_edge_b[2], 2, x->x_dd, g->e_dd, x->stride_dd,
                       reps_dd, false, L.te_dd, stream);
        const bool last = l == NL - 1;
        float *out_op = last ? E_op : L.H_op[(l + 1) & 1];
        float *out_dev = last ? E_dev : L.H_dev[(l + 1) & 1];
        const int ld2 = 2 * F;
        const float *te_b = NR == 5 ? L.te_oo[1] : L.te_oo[0];
        const float *te_do = NR == 5 ? L.te_od[1] : L.te_od[0];
        // op destinations
        VarArgs A = base;
        A.n_dst = g->n_op;
        A.out = out_op;
        int n = 0;
        if (NR == 5) {
            A.rel[n++] = VarRel{0, 1, L.Y_opA, L.Y_opA, g->n_op, ld2, L.te_oo[0], 0, reps_oo > 1 ? g->e_oo : 0,
                                as[r_f], ad[r_f], dims->gamma_same};
            A.rel[n++] = VarRel{0, 2, L.Y_opA + F, L.Y_opA + F, g->n_op, ld2, te_b, 0, reps_oo > 1 ? g->e_oo : 0,
                                as[r_b], ad[r_b], dims->gamma_same};
        } else {
            A.rel[n++] = VarRel{0, 0, L.Y_opA, L.Y_opA, g->n_op, ld2, L.te_oo[0], 0, reps_oo > 1 ? g->e_oo : 0,
                                as[r_f], ad[r_f], dims->gamma_same};
        }
        A.rel[n++] = VarRel{1, 0, L.Y_devA + F, L.Y_opB, g->n_dev, ld2, L.te_od[0], 1, 0, as[r_od], ad[r_od],
                            dims->gamma_cross};
        A.n_rel = n;
        prof_begin(TAG_STAGE_AGG_OP_OP, stream);
        dispatch_agg_var(F, A, stream);
        prof_end(TAG_STAGE_AGG_OP_OP, stream);
        // device destinations
        VarArgs B = base;
        B.n_dst = g->n_dev;
        B.out = out_dev;
        B.rel[0] = VarRel{2, 0, L.Y_opB + F, L.Y_devB, g->n_op, ld2, te_do, 1, 0, as[r_do], ad[r_do], dims->gamma_cross};
        B.rel[1] = VarRel{3, 0, L.Y_devA, L.Y_devA, g->n_dev, ld2, L.te_dd, 0, reps_dd > 1 ? g->e_dd : 0, as[r_dd],
                          ad[r_dd], dims->gamma_same};
        B.n_rel = 2;
        prof_begin(TAG_STAGE_AGG_DEV_MERGE, stream);
        dispatch_agg_var(F, B, stream);
        prof_end(TAG_STAGE_AGG_DEV_MERGE, stream);
    }
    return launch_status("tag_gnn_forward");
}

}  // namespace tag
