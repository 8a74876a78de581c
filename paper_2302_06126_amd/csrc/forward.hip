// Forward pass of the heterogeneous GNN (Section 4.2.1 of the paper).
//
// Layer l, link type r, destination u, neighbour v (edge feature e_uv):
//   m_uv  = ReLU(W^h h_v + W^e e_uv + b)                W = [W^h | W^e]
//   s_uvk = LeakyReLU(a^(k) . m_uv^(k) + adst^(k) . (W^h h_u)^(k))
//   h'_u  = sum_r gamma_r sum_v softmax_v(s_uvk) m_uv^(k)   (heads concatenated)
//
// GPU formulation (exact algebra, only rounding differs from the plain
// definition):
//  * Edge encoders are affine and have no activation, so W^e e + b is folded
//    once per call into U_{l,r} = W^e A_r (f x d_r) and c'_{l,r} = W^e c_r + b;
//    the per-entry edge term is U x + c' (d_r <= 2 multiply-adds per channel).
//  * W^h h is computed once per node (not per entry) by an MFMA GEMM per
//    side: op rows get [W^h_oo ; W^h_od], device rows [W^h_dd ; W^h_od],
//    written as Y [rows][2f] (first half: same-type relation, second: od).
//  * Aggregation runs one wavefront per destination row (per candidate),
//    lanes own f/64 consecutive channels, head scores are reduced over the
//    64/K lanes of a head, and the softmax is an online (running-max)
//    softmax in the exp2 domain.  Long device<-op rows are split into
//    chunks whose (max, denominator, accumulator) partials are merged in a
//    fixed order, so results do not depend on scheduling.
#include <algorithm>

#include "agg_common.hpp"
#include "fwd_internal.hpp"
#include "transform.hpp"

namespace tag {
namespace {

// ------------------------------------------------------------------ folding
// U[l][r][c][t] = sum_k W^e[c][k] A_r[k][t];  cp[l][r][c] = b[c] + sum_k W^e[c][k] c_r[k]
struct FoldArgs {
    const float *layer_w, *layer_b;
    const float *A[3], *c[3];
    float *U, *cp;
    int F;
};

// one wavefront per (layer, relation, output channel); lanes split the k sum
__global__ void __launch_bounds__(64) fold_edge_terms(FoldArgs a) {
    const int F = a.F;
    const int lr = blockIdx.x / F, c = blockIdx.x % F;   // lr = l*3 + r
    const int r = lr % 3;
    const int d = (r == 2) ? 2 : 1;
    const float *W = a.layer_w + (size_t)lr * F * 2 * F + (size_t)c * 2 * F + F;   // row c of W^e
    float u0 = 0.f, u1 = 0.f, s = 0.f;
    for (int k = threadIdx.x; k < F; k += 64) {
        const float we = W[k];
        u0 = fmaf(we, a.A[r][(size_t)k * d + 0], u0);
        if (d == 2) u1 = fmaf(we, a.A[r][(size_t)k * d + 1], u1);
        s = fmaf(we, a.c[r][k], s);
    }
    for (int o = 32; o >= 1; o >>= 1) {
        u0 += __shfl_xor(u0, o, 64);
        u1 += __shfl_xor(u1, o, 64);
        s += __shfl_xor(s, o, 64);
    }
    if (threadIdx.x == 0) {
        a.U[((size_t)lr * F + c) * 2 + 0] = u0;
        a.U[((size_t)lr * F + c) * 2 + 1] = u1;
        a.cp[(size_t)lr * F + c] = a.layer_b[(size_t)lr * F + c] + s;
    }
}

// W^h of every (layer, relation) to bf16: Wb[l][r][n][k] = bf16(W[l][r][n][k]), k < F
__global__ void convert_wh_bf16(const float *layer_w, uint16_t *Wb, int F, int LR) {
    int64_t total = (int64_t)LR * F * F;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t lr = i / ((int64_t)F * F);
        int64_t rem = i % ((int64_t)F * F);
        int64_t n = rem / F, k = rem % F;
        Wb[i] = f2bf(layer_w[(lr * F + n) * 2 * F + k]);
    }
}

// op destinations: B0 (op<-op) and B1 (op<-dev)
template <int F, int K, bool BF, bool ELU = false>
__global__ void __launch_bounds__(256) agg_op(AggArgs A) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    if (w >= (int64_t)A.R * A.n_op) return;
    const int32_t rep = (int32_t)(w / A.n_op);
    const int32_t u = (int32_t)(w % A.n_op);
    const int c0 = lane * CPL;
    const int64_t yrow_u = ((int64_t)rep * A.n_op + u) * 2 * F;
    float out[CPL];
    for (int c = 0; c < CPL; ++c) out[c] = 0.f;
    {   // B0: op <- op, relation oo
        RelConst<CPL> k; k.load(A, 0, F, c0);
        float yd[CPL]; load_ch<CPL, BF>(A.Y_op, yrow_u + c0, yd);
        float q = 0.f;
        for (int c = 0; c < CPL; ++c) q = fmaf(k.ad[c], stored_dst<BF>(yd[c], k.cp[c]), q);
        q = head_sum<LPH>(q);
        Online<CPL> o; o.init();
        const int32_t beg = A.rp[0][u], end = A.rp[0][u + 1];
        const float *xo = A.x_oo + (int64_t)rep * A.s_oo;
        for (int32_t e = beg; e < end; ++e) {
            const int32_t v = A.col[0][e];
            const float x0 = xo[A.eid[0][e]];
            float y[CPL]; load_ch<CPL, BF>(A.Y_op, ((int64_t)rep * A.n_op + v) * 2 * F + c0, y);
            float m[CPL];
            float s2 = entry_score<CPL, LPH, ELU, BF>(y, x0, 0.f, k, q, A.slope, m);
            o.push(s2, m);
        }
        if (end > beg) {
            float inv = A.g_same / o.den;
            for (int c = 0; c < CPL; ++c) out[c] = o.acc[c] * inv;
        }
    }
    {   // B1: op <- device, relation od
        RelConst<CPL> k; k.load(A, 1, F, c0);
        float yd[CPL]; load_ch<CPL, BF>(A.Y_op, yrow_u + F + c0, yd);
        float q = 0.f;
        for (int c = 0; c < CPL; ++c) q = fmaf(k.ad[c], stored_dst<BF>(yd[c], k.cp[c]), q);
        q = head_sum<LPH>(q);
        Online<CPL> o; o.init();
        const int32_t beg = A.rp[1][u], end = A.rp[1][u + 1];
        const uint8_t *xb = A.x_od + (int64_t)rep * A.s_od;
        for (int32_t e = beg; e < end; ++e) {
            const int32_t j = A.col[1][e];
            const float x0 = xb[A.eid[1][e]] ? 1.f : 0.f;
            float y[CPL]; load_ch<CPL, BF>(A.Y_dev, ((int64_t)rep * A.n_dev + j) * 2 * F + F + c0, y);
            float m[CPL];
            float s2 = entry_score<CPL, LPH, ELU, BF>(y, x0, 0.f, k, q, A.slope, m);
            o.push(s2, m);
        }
        if (end > beg) {
            float inv = A.g_cross / o.den;
            for (int c = 0; c < CPL; ++c) out[c] = fmaf(o.acc[c], inv, out[c]);
        }
    }
    store_row<CPL, BF>(A.H_op, ((int64_t)rep * A.n_op + u) * F + c0, A.out_f32 != 0, out);
}

// device <- op partials over chunks of kChunk entries
template <int F, int K, bool BF, bool ELU = false>
__global__ void __launch_bounds__(256) agg_dev_part(AggArgs A) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const uint32_t nblk = gridDim.x;
    const uint32_t lb = xcd_swizzle(blockIdx.x, nblk);
    // logical wave id: (rep, chunk, device) with the device fastest
    const int64_t w = (int64_t)lb * kWaves + (threadIdx.x >> 6);
    const int64_t total = (int64_t)A.R * A.maxc * A.n_dev;
    if (w >= total) return;
    const int32_t j = (int32_t)(w % A.n_dev);
    const int32_t c = (int32_t)((w / A.n_dev) % A.maxc);
    const int32_t rep = (int32_t)(w / ((int64_t)A.n_dev * A.maxc));
    const int32_t rbeg = A.rp[2][j], rend = A.rp[2][j + 1];
    const int32_t beg = rbeg + c * kChunk;
    if (beg >= rend) return;
    const int32_t end = min(beg + kChunk, rend);
    const int c0 = lane * CPL;
    RelConst<CPL> k; k.load(A, 1, F, c0);
    float yd[CPL]; load_ch<CPL, BF>(A.Y_dev, ((int64_t)rep * A.n_dev + j) * 2 * F + F + c0, yd);
    float q = 0.f;
    for (int cc = 0; cc < CPL; ++cc) q = fmaf(k.ad[cc], stored_dst<BF>(yd[cc], k.cp[cc]), q);
    q = head_sum<LPH>(q);
    Online<CPL> o; o.init();
    const uint8_t *xb = A.x_od + (int64_t)rep * A.s_od;
    for (int32_t e = beg; e < end; ++e) {
        const int32_t u = A.col[2][e];
        const float x0 = xb[A.eid[2][e]] ? 1.f : 0.f;
        float y[CPL]; load_ch<CPL, BF>(A.Y_op, ((int64_t)rep * A.n_op + u) * 2 * F + F + c0, y);
        float m[CPL];
        float s2 = entry_score<CPL, LPH, ELU, BF>(y, x0, 0.f, k, q, A.slope, m);
        o.push(s2, m);
    }
    // partial record: [mx per head][den per head][acc F]
    float *p = A.part + (((int64_t)rep * A.n_dev + j) * A.maxc + c) * (F + 2 * K);
    const int head = lane / LPH;
    if ((lane % LPH) == 0) { p[head] = o.mx; p[K + head] = o.den; }
    for (int cc = 0; cc < CPL; ++cc) p[2 * K + c0 + cc] = o.acc[cc];
}

// device destinations: merge B2 partials, then B3 (dev <- dev)
template <int F, int K, bool BF, bool ELU = false>
__global__ void __launch_bounds__(256) agg_dev_final(AggArgs A) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    if (w >= (int64_t)A.R * A.n_dev) return;
    const int32_t rep = (int32_t)(w / A.n_dev);
    const int32_t j = (int32_t)(w % A.n_dev);
    const int c0 = lane * CPL;
    const int head = lane / LPH;
    float out[CPL];
    for (int c = 0; c < CPL; ++c) out[c] = 0.f;
    {   // B2 merge in record order (records with a zero sum hold no links),
        // one online pass: records are read sixteen at a time so their loads
        // overlap, and the running sums are rescaled to each batch's maximum
        constexpr int RB = 16;
        const int32_t deg = A.rp[2][j + 1] - A.rp[2][j];
        int32_t nch = (deg + kChunk - 1) / kChunk;
        if (A.rec_mode) {
            int32_t lo = 0, hi = A.G;
            while (hi - lo > 1) {
                const int32_t mid = (lo + hi) >> 1;
                if (A.dev_off[mid] <= j) lo = mid; else hi = mid;
            }
            nch = A.group_off[lo + 1] - A.group_off[lo];
        }
        if (deg > 0 && nch > 0) {
            constexpr int REC = F + 2 * K;
            const float *p0 = A.part + ((int64_t)rep * A.n_dev + j) * A.maxc * REC;
            float M = -INFINITY, den = 0.f, acc[CPL];
            for (int cc = 0; cc < CPL; ++cc) acc[cc] = 0.f;
            for (int32_t c = 0; c < nch; c += RB) {
                float mv[RB], dv[RB], av[RB][CPL];
#pragma unroll
                for (int i = 0; i < RB; ++i) {
                    const float *p = p0 + (int64_t)(c + i) * REC;
                    if (c + i < nch) {
                        mv[i] = p[head];
                        dv[i] = p[K + head];
                        load_ch<CPL, false>(p, 2 * K + c0, av[i]);
                    } else {
                        mv[i] = -INFINITY;
                        dv[i] = 0.f;
                        for (int cc = 0; cc < CPL; ++cc) av[i][cc] = 0.f;
                    }
                }
                float Mb = M;
#pragma unroll
                for (int i = 0; i < RB; ++i) Mb = fmaxf(Mb, mv[i]);
                // records without links (maximum -inf) weigh nothing
                const float r = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - Mb);
                den *= r;
                for (int cc = 0; cc < CPL; ++cc) acc[cc] *= r;
#pragma unroll
                for (int i = 0; i < RB; ++i) {
                    const float sc = mv[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mv[i] - Mb);
                    den = fmaf(dv[i], sc, den);
                    for (int cc = 0; cc < CPL; ++cc) acc[cc] = fmaf(av[i][cc], sc, acc[cc]);
                }
                M = Mb;
            }
            float inv = A.g_cross / den;
            for (int cc = 0; cc < CPL; ++cc) out[cc] = acc[cc] * inv;
        }
    }
    {   // B3: dev <- dev, relation dd, EB entries per step
        constexpr int EB = 16;
        RelConst<CPL> k; k.load(A, 2, F, c0);
        float yd[CPL]; load_ch<CPL, BF>(A.Y_dev, ((int64_t)rep * A.n_dev + j) * 2 * F + c0, yd);
        float q = 0.f;
        for (int c = 0; c < CPL; ++c) q = fmaf(k.ad[c], stored_dst<BF>(yd[c], k.cp[c]), q);
        q = head_sum<LPH>(q);
        Online<CPL> o; o.init();
        const int32_t beg = A.rp[3][j], end = A.rp[3][j + 1];
        const float *xd = A.x_dd + (int64_t)rep * A.s_dd;
        for (int32_t e = beg; e < end; e += EB) {
            const int n = min(EB, end - e);
            int32_t v[EB], id[EB];
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                v[i] = i < n ? A.col[3][e + i] : 0;
                id[i] = i < n ? A.eid[3][e + i] : 0;
            }
            float x0[EB], x1[EB], y[EB][CPL];
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                x0[i] = i < n ? xd[(int64_t)id[i] * 2] : 0.f;
                x1[i] = i < n ? xd[(int64_t)id[i] * 2 + 1] : 0.f;
                load_ch<CPL, BF>(A.Y_dev, ((int64_t)rep * A.n_dev + v[i]) * 2 * F + c0, y[i]);
            }
            float s2[EB], m[EB][CPL];
#pragma unroll
            for (int i = 0; i < EB; ++i) s2[i] = entry_score<CPL, LPH, ELU, BF>(y[i], x0[i], x1[i], k, q, A.slope, m[i]);
            o.template push_n<EB>(s2, m, n);
        }
        if (end > beg) {
            float inv = A.g_same / o.den;
            for (int c = 0; c < CPL; ++c) out[c] = fmaf(o.acc[c], inv, out[c]);
        }
    }
    store_row<CPL, BF>(A.H_dev, ((int64_t)rep * A.n_dev + j) * F + c0, A.out_f32 != 0, out);
}

template <int F, int K, bool BF, bool ELU = false>
void launch_agg(const AggArgs &A, hipStream_t st) {
    const int64_t op_waves = (int64_t)A.R * A.n_op;
    const int64_t part_waves = (int64_t)A.R * A.maxc * A.n_dev;
    const int64_t dev_waves = (int64_t)A.R * A.n_dev;
    prof_begin(TAG_STAGE_AGG_OP_OP, st);
    agg_op<F, K, BF, ELU><<<(unsigned)((op_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_OP_OP, st);
    prof_begin(TAG_STAGE_AGG_DEV_OP, st);
    agg_dev_part<F, K, BF, ELU><<<(unsigned)((part_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_DEV_OP, st);
    (void)dev_waves;
}

template <int F, int K, bool BF, bool ELU = false>
void launch_dev_final(const AggArgs &A, hipStream_t st) {
    const int64_t dev_waves = (int64_t)A.R * A.n_dev;
    prof_begin(TAG_STAGE_AGG_DEV_MERGE, st);
    agg_dev_final<F, K, BF, ELU><<<(unsigned)((dev_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_DEV_MERGE, st);
}

// first-version aggregation (used when heads are narrower than 16 channels),
// then the device merge + dev<-dev pass shared by both paths
template <int F, int K, bool BF, bool ELU = false>
void launch_layer(bool mfma, const AggArgs &A, hipStream_t st) {
    if (!mfma) launch_agg<F, K, BF, ELU>(A, st);
    else launch_agg_mfma(F, K, BF, A, st);   // takes every layer the layout was planned for
    launch_dev_final<F, K, BF, ELU>(A, st);
}

template <int F, bool BF, bool ELU = false>
tag_status dispatch_heads(int K, bool mfma, const AggArgs &A, hipStream_t st) {
    switch (K) {
        case 1: launch_layer<F, 1, BF, ELU>(mfma, A, st); break;
        case 2: launch_layer<F, 2, BF, ELU>(mfma, A, st); break;
        case 4: launch_layer<F, 4, BF, ELU>(mfma, A, st); break;
        case 8: launch_layer<F, 8, BF, ELU>(mfma, A, st); break;
        case 16: launch_layer<F, 16, BF, ELU>(mfma, A, st); break;
        case 32: launch_layer<F, 32, BF, ELU>(mfma, A, st); break;
        case 64: launch_layer<F, 64, BF, ELU>(mfma, A, st); break;
        default: TAG_FAIL(TAG_ESHAPE, "unsupported head count");
    }
    return TAG_OK;
}

tag_status dispatch_agg(int F, int K, bool bf, bool mfma, const AggArgs &A, hipStream_t st) {
    if (A.elu) {   // the ELU variant runs in fp32
        if (bf) TAG_FAIL(TAG_ESHAPE, "the ELU variant needs the fp32 variant");
        if (F == 64) return dispatch_heads<64, false, true>(K, mfma, A, st);
        if (F == 128) return dispatch_heads<128, false, true>(K, mfma, A, st);
        return dispatch_heads<256, false, true>(K, mfma, A, st);
    }
    if (F == 64) return bf ? dispatch_heads<64, true>(K, mfma, A, st) : dispatch_heads<64, false>(K, mfma, A, st);
    if (F == 128) return bf ? dispatch_heads<128, true>(K, mfma, A, st) : dispatch_heads<128, false>(K, mfma, A, st);
    return bf ? dispatch_heads<256, true>(K, mfma, A, st) : dispatch_heads<256, false>(K, mfma, A, st);
}

}  // namespace

// ------------------------------------------------------------------ planning
tag_status check_dims(const tag_model_dims *d) {
    if (!d) TAG_FAIL(TAG_EINVAL, "dims is NULL");
    if (d->f != 64 && d->f != 128 && d->f != 256) TAG_FAIL(TAG_ESHAPE, "f must be 64, 128 or 256");
    if (d->heads < 1 || d->heads > 64 || (d->heads & (d->heads - 1)))
        TAG_FAIL(TAG_ESHAPE, "heads must be a power of two in [1, 64]");
    if (d->layers < 1 || d->layers > 16) TAG_FAIL(TAG_ESHAPE, "layers must be in [1, 16]");
    if (d->f_op < 1 || d->f_op > 64 || d->f_dev < 1 || d->f_dev > 64)
        TAG_FAIL(TAG_ESHAPE, "f_op and f_dev must be in [1, 64]");
    if (d->dec_hidden < 0 || d->dec_hidden > 1024) TAG_FAIL(TAG_ESHAPE, "dec_hidden must be in [0, 1024]");
    if (d->dtype != TAG_F32 && d->dtype != TAG_BF16) TAG_FAIL(TAG_EINVAL, "dtype must be TAG_F32 or TAG_BF16");
    if (!(d->gamma_same == d->gamma_same) || !(d->gamma_cross == d->gamma_cross))
        TAG_FAIL(TAG_EINVAL, "gamma must not be NaN");
    if (!(d->leaky_slope >= 0.f && d->leaky_slope <= 1.f))
        TAG_FAIL(TAG_EINVAL, "leaky_slope must be in [0, 1]");
    if (d->sigma != 0 && d->sigma != 1) TAG_FAIL(TAG_EINVAL, "sigma must be 0 (ReLU) or 1 (ELU)");
    if (d->sigma == 1 && d->dtype != TAG_F32) TAG_FAIL(TAG_ESHAPE, "the ELU variant needs the fp32 variant");
    return check_variant(d);
}

size_t carve_fwd(const tag_graph *g, const tag_model_dims *d, int32_t R, void *base, FwdLayout *L) {
    Carver c(base);
    const int F = d->f;
    const size_t es = d->dtype == TAG_BF16 ? 2 : 4;
    L->U = c.take<float>((size_t)d->layers * 3 * F * 2);
    L->cp = c.take<float>((size_t)d->layers * 3 * F);
    L->Wb = d->dtype == TAG_BF16 ? c.take<uint16_t>((size_t)d->layers * 3 * F * F) : nullptr;
    for (int i = 0; i < 2; ++i) {
        L->H_op[i] = c.take<char>((size_t)R * g->n_op * F * es);
        L->H_dev[i] = c.take<char>((size_t)R * g->n_dev * F * es);
    }
    L->Y_op = c.take<char>((size_t)R * g->n_op * 2 * F * es);
    L->Y_dev = c.take<char>((size_t)R * g->n_dev * 2 * F * es);
    L->mfma = mfma_path_supported(F, d->heads, g->n_op, R, g->n_dev, (int)es);
    L->maxc = L->mfma ? std::max<int32_t>(1, g->max_groups)
                      : std::max<int32_t>(1, (g->max_degree[2] + kChunk - 1) / kChunk);
    L->part = c.take<float>((size_t)R * g->n_dev * L->maxc * (F + 2 * d->heads));
    if (L->mfma) {
        L->omask = c.take<uint64_t>((size_t)R * g->n_op * 2);
        L->Sdev = c.take<float>((size_t)R * g->n_dev * 4 * d->heads);
        // fp32 message table [R n_dev][2][F], or its three bf16 split parts [3][R n_dev][F]
        L->T = c.take<float>((size_t)R * g->n_dev * 3 * F);
        L->Sop = c.take<float>((size_t)R * g->n_op * 4 * d->heads);
        L->tile_ext = c.take<int32_t>((size_t)std::max<int32_t>(g->n_tiles, 1) * 8);
        L->xcsr = c.take<float>((size_t)R * std::max<int64_t>(g->nnz[0], 1));
    } else {
        L->omask = nullptr;
        L->Sdev = L->T = L->Sop = nullptr;
        L->tile_ext = nullptr;
        L->xcsr = nullptr;
    }
    return c.used;
}

}  // namespace tag

using namespace tag;

extern "C" tag_status tag_gnn_workspace(const tag_graph *g, const tag_model_dims *dims, int32_t n_replicas,
                                        size_t *bytes) {
    clear_error();
    if (!g || !bytes) TAG_FAIL(TAG_EINVAL, "graph and bytes must be non-NULL");
    tag_status st = check_dims(dims);
    if (st != TAG_OK) return st;
    if (n_replicas < 1) TAG_FAIL(TAG_EINVAL, "n_replicas must be >= 1");
    if (is_variant(dims)) {
        *bytes = variant_workspace(g, dims, n_replicas);
        return TAG_OK;
    }
    FwdLayout L;
    *bytes = carve_fwd(g, dims, n_replicas, nullptr, &L);
    return TAG_OK;
}

extern "C" tag_status tag_gnn_forward(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                      const tag_features *x, void *workspace, size_t ws_bytes, float *E_op,
                                      float *E_dev, void *hip_stream) {
    clear_error();
    return forward_run(g, dims, w, x, workspace, ws_bytes, E_op, E_dev, static_cast<hipStream_t>(hip_stream),
                       nullptr);
}

namespace tag {

// Relation transforms of layer l (Y = W^h h + c', attention terms, device
// message table) for the hidden rows H_op / H_dev, into the layout's buffers.
void launch_layer_transform(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                            const FwdLayout &L, int32_t R, int l, const void *H_op, const void *H_dev,
                            hipStream_t stream) {
    const int F = dims->f, K = dims->heads;
    const bool bf = dims->dtype == TAG_BF16;
    const int64_t rows_op = (int64_t)R * g->n_op, rows_dev = (int64_t)R * g->n_dev;
    const int D = F / K;
    const int jph = (L.mfma && D <= 64) ? D / 16 : 0;
    const float *att_src = w->att_src + (size_t)l * 3 * F, *att_dst = w->att_dst + (size_t)l * 3 * F;
    const float *U = L.U + (size_t)l * 3 * F * 2, *cp = L.cp + (size_t)l * 3 * F;
    GemmArgs ga{};
    ga.F = F;
    ga.prep.jph = jph;
    ga.prep.K = K;
    ga.prep.elu = dims->sigma == 1 ? 1 : 0;
    ga.prep.a_od = att_src + F;
    ga.prep.ad_od = att_dst + F;
    ga.prep.cp_od = cp + F;
    ga.prep.u_od = U + 2 * F;
    ga.prep.cp_same[0] = cp;
    ga.prep.cp_same[1] = cp + 2 * F;
    ga.prep.ad_same[0] = att_dst;
    ga.prep.ad_same[1] = att_dst + 2 * F;
    ga.prep.S[0] = L.Sop;
    ga.prep.S[1] = L.Sdev;
    ga.prep.T = L.T;
    ga.tiles0 = transform_row_tiles(rows_op);
    if (bf) {
        const uint16_t *Wl = L.Wb + (size_t)l * 3 * F * F;
        ga.side[0] = GemmSide{H_op, rows_op, Wl + 0 * F * F, Wl + 1 * F * F, F, L.Y_op};
        ga.side[1] = GemmSide{H_dev, rows_dev, Wl + 2 * F * F, Wl + 1 * F * F, F, L.Y_dev};
    } else {
        const float *Wl = w->layer_w + (size_t)l * 3 * F * 2 * F;
        ga.side[0] = GemmSide{H_op, rows_op, Wl + 0 * F * 2 * F, Wl + 1 * F * 2 * F, 2 * F, L.Y_op};
        ga.side[1] = GemmSide{H_dev, rows_dev, Wl + 2 * F * 2 * F, Wl + 1 * F * 2 * F, 2 * F, L.Y_dev};
    }
    prof_begin(TAG_STAGE_TRANSFORM, stream);
    launch_transform(ga, bf, stream);
    prof_end(TAG_STAGE_TRANSFORM, stream);
}

tag_status forward_run(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w, const tag_features *x,
                       void *workspace, size_t ws_bytes, float *E_op, float *E_dev, hipStream_t stream,
                       const FwdSave *save) {
    if (!g || !w || !x || !E_op || !E_dev || !workspace)
        TAG_FAIL(TAG_EINVAL, "graph, weights, features, outputs and workspace must be non-NULL");
    tag_status st = check_dims(dims);
    if (st != TAG_OK) return st;
    const int32_t R = x->n_replicas;
    if (R < 1) TAG_FAIL(TAG_EINVAL, "n_replicas must be >= 1");
    if (!x->x_op || !x->x_dev || (g->e_oo && !x->x_oo) || (g->e_dd && !x->x_dd) || (g->e_od && !x->x_od))
        TAG_FAIL(TAG_EINVAL, "feature arrays must be non-NULL");
    if (x->stride_oo < 0 || x->stride_dd < 0 || x->stride_od < 0) TAG_FAIL(TAG_EINVAL, "strides must be >= 0");
    if (!w->enc_op_w || !w->enc_op_b || !w->enc_dev_w || !w->enc_dev_b || !w->layer_w || !w->layer_b ||
        !w->att_src || !w->att_dst)
        TAG_FAIL(TAG_EINVAL, "weight arrays must be non-NULL");
    for (int r = 0; r < 3; ++r)
        if (!w->enc_edge_w[r] || !w->enc_edge_b[r]) TAG_FAIL(TAG_EINVAL, "edge encoder weights must be non-NULL");
    if ((reinterpret_cast<uintptr_t>(x->x_op) | reinterpret_cast<uintptr_t>(E_op) |
         reinterpret_cast<uintptr_t>(E_dev) | reinterpret_cast<uintptr_t>(w->layer_w) |
         reinterpret_cast<uintptr_t>(workspace)) & 15)
        TAG_FAIL(TAG_EINVAL, "x_op, E_op, E_dev, layer_w and workspace must be 16-byte aligned");
    if (is_variant(dims)) {
        if (save) TAG_FAIL(TAG_ESHAPE, "saved activations need the default readings");
        return forward_variant(g, dims, w, x, workspace, ws_bytes, E_op, E_dev, stream);
    }
    FwdLayout L;
    if (carve_fwd(g, dims, R, nullptr, &L) > ws_bytes) TAG_FAIL(TAG_ENOSPACE, "workspace too small (see tag_gnn_workspace)");
    carve_fwd(g, dims, R, workspace, &L);
    const int F = dims->f, K = dims->heads, NL = dims->layers;
    const bool bf = dims->dtype == TAG_BF16;
    if (save && bf) TAG_FAIL(TAG_ESHAPE, "saved activations need the fp32 variant");
    // hidden rows of layer l: the ping-pong buffers, or the caller's slots
    auto h_op = [&](int l) -> void * { return save ? static_cast<void *>(save->H_op[l]) : L.H_op[l & 1]; };
    auto h_dev = [&](int l) -> void * { return save ? static_cast<void *>(save->H_dev[l]) : L.H_dev[l & 1]; };

    FoldArgs fa{w->layer_w, w->layer_b, {w->enc_edge_w[0], w->enc_edge_w[1], w->enc_edge_w[2]},
                {w->enc_edge_b[0], w->enc_edge_b[1], w->enc_edge_b[2]}, L.U, L.cp, F};
    fold_edge_terms<<<NL * 3 * F, 64, 0, stream>>>(fa);
    if (bf) convert_wh_bf16<<<256, 256, 0, stream>>>(w->layer_w, L.Wb, F, NL * 3);

    // encoders: hidden h0 in the working precision
    const int64_t rows_op = (int64_t)R * g->n_op, rows_dev = (int64_t)R * g->n_dev;
    {
        // h0 = ReLU(A x + c) as a small-K MFMA GEMM per node type
        SmallGemm eo{x->x_op, dims->f_op, rows_op, nullptr, dims->f_op, w->enc_op_w, dims->f_op, F,
                     w->enc_op_b, 1, h_op(0), F, bf ? 1 : 0};
        SmallGemm ed{x->x_dev, dims->f_dev, rows_dev, nullptr, dims->f_dev, w->enc_dev_w, dims->f_dev, F,
                     w->enc_dev_b, 1, h_dev(0), F, bf ? 1 : 0};
        prof_begin(TAG_STAGE_ENCODE, stream);
        launch_small_gemm(eo, stream);
        launch_small_gemm(ed, stream);
        prof_end(TAG_STAGE_ENCODE, stream);
    }
    AggArgs A{};
    A.R = R;
    A.n_op = g->n_op; A.n_dev = g->n_dev;
    for (int b = 0; b < 4; ++b) { A.rp[b] = g->rowptr[b]; A.col[b] = g->col[b]; A.eid[b] = g->eid[b]; }
    A.Y_op = L.Y_op; A.Y_dev = L.Y_dev;
    A.x_oo = x->x_oo; A.s_oo = x->stride_oo;
    A.x_dd = x->x_dd; A.s_dd = x->stride_dd;
    A.x_od = x->x_od; A.s_od = x->stride_od;
    A.g_same = dims->gamma_same; A.g_cross = dims->gamma_cross; A.slope = dims->leaky_slope;
    A.elu = dims->sigma == 1 ? 1 : 0;
    A.part = L.part; A.maxc = L.maxc;
    A.G = g->G; A.n_tiles = g->n_tiles;
    A.tiles = g->tiles_d; A.tile_off = g->tile_off_d; A.op_off = g->op_off_d; A.dev_off = g->dev_off_d;
    A.n_groups = g->n_groups; A.groups = g->groups_d; A.group_off = g->group_off_d;
    A.omask = L.omask; A.Sdev = L.Sdev; A.T = L.T; A.Sop = L.Sop;
    A.rec_mode = L.mfma ? 1 : 0;
    A.tile_ext = L.tile_ext;
    A.xcsr = L.xcsr;
    A.s_xcsr = x->stride_oo ? g->nnz[0] : 0;
    if (L.mfma) {
        launch_pack_masks(A, stream);
        launch_prep_tiles_x(A, g->nnz[0], stream);
    }

    // the transform epilogue forms the attention terms when a head fits one
    // wavefront's 64 columns
    const int D = F / K;
    const int jph = (L.mfma && D <= 64) ? D / 16 : 0;
    A.prep_done = jph > 0 ? 1 : 0;
    for (int l = 0; l < NL; ++l) {
        const bool last = (l == NL - 1);
        A.att_src = w->att_src + (size_t)l * 3 * F;
        A.att_dst = w->att_dst + (size_t)l * 3 * F;
        A.U = L.U + (size_t)l * 3 * F * 2;
        A.cp = L.cp + (size_t)l * 3 * F;
        // relation transforms: op rows [W^h_oo ; W^h_od], device rows [W^h_dd ; W^h_od]
        FwdLayout Ll = L;
        if (save) { Ll.Y_op = save->Y_op[l]; Ll.Y_dev = save->Y_dev[l]; }
        A.Y_op = Ll.Y_op; A.Y_dev = Ll.Y_dev;
        launch_layer_transform(g, dims, w, Ll, R, l, h_op(l), h_dev(l), stream);
        A.H_op = last ? static_cast<void *>(E_op) : h_op(l + 1);
        A.H_dev = last ? static_cast<void *>(E_dev) : h_dev(l + 1);
        A.out_f32 = last ? 1 : (bf ? 0 : 1);
        st = dispatch_agg(F, K, bf, L.mfma, A, stream);
        if (st != TAG_OK) return st;
    }
    return launch_status("tag_gnn_forward");
}

}  // namespace tag
