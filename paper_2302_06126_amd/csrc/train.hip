// Training step of the GNN (Section 4.2.2: the prior G(s, a) of the decoder
// is trained toward the search's selection probabilities pi(s, a) by
// minimising their cross entropy), fp32.
//
//   loss = -(1/Q) sum_q sum_a target[q][a] log softmax_a(score[q][a])
//
// Forward: the forward pass of forward.hip with every layer's input rows H^l
// and relation transforms Y^l = W^h H^l + c' kept (no recomputation).
//
// Backward, per layer from the last to the first, with dO_u = gamma_r dH'_u
// the gradient reaching destination u's gamma-weighted sum of relation r:
//   scores   (per entry e = (u <- v), per head k)
//              s_e = LeakyReLU(a . m_e + adst . (Y_u - c')),  m_e = sigma(Y_v + U x_e)
//              (sigma: ReLU, or ELU for the variant)
//              dalpha_e = dO_u . m_e
//   softmax  (per destination row) alpha_e = softmax(s), c_u = sum_e alpha_e dalpha_e,
//              dz_e = alpha_e (dalpha_e - c_u) LeakyReLU'(s_e),  Z_u = sum_e dz_e
//   messages (per source row v, over the entries it feeds)
//              dm_e = alpha_e dO_u + dz_e a,  dpre_e = dm_e sigma'(pre_e)
//              dY_v = sum_e dpre_e + Z_v adst      (Z_v: v as a destination)
//            and the parameter sums d a = sum dz m, d adst = sum Z (Y - c'),
//            dU = sum dpre x^T, dc' = sum dpre
//   GEMMs    dH = dY [W^h ; W^h'] (both relations of a node type in one
//            K = 2f contraction), dW^h = dY^T H (split-K, partials summed in
//            a fixed order)
// then the node encoders (ReLU mask, dA = dpre^T x, dc = column sums) and
// the folded edge encoders (U = W^e A_r, c' = W^e c_r + b):
//   dW^e = dU A_r^T + dc' c_r^T,  db = dc',  dA_r = sum_l W^e^T dU,  dc_r = sum_l W^e^T dc'.
// Per-entry scalars live in slots the source-side pass can find through the
// transposed bucket: undirected links (op-op, device-device) are keyed by
// edge id with the direction bit (destination id > source id) and found
// through the row's own bucket; op-device links (both directions) are keyed
// by the entry's position in the op<-device bucket, which the
// device<-op bucket reaches through a position map built at the start of the
// step.
//
// Every reduction runs in a fixed order (per-block partials summed by one
// thread per output), so the step is bitwise repeatable.
#include <algorithm>

#include "../../include/tag_train.h"
#include "agg_common.hpp"
#include "fwd_internal.hpp"

namespace tag {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- GEMM
// C_z (+)= sum_{k in split z} A(m, k) B(k, n) on MFMA 16x16x4 (fp32).
// A(m, k) = A[m lda + k] (a_kc) or A[k lda + m]; B(k, n) = B[n ldb + k]
// (b_kc) or B[k ldb + n].  Column ones_col of an n-contiguous B reads 1
// (it turns the product into column sums of A).  64 x 64 block tiles of
// four 32 x 32 wavefront tiles, k-chunks of 16 staged through LDS with the
// next chunk's loads in flight.
struct Gemm {
    const float *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    int64_t M, N, K;
    int64_t ones_col;
    float *C;
    int64_t ldc, c_split;
    int64_t k_per;
    int accumulate;
};

constexpr int GM = 64, GN = 64, GK = 16;

template <bool AKC, bool BKC>
__global__ void __launch_bounds__(256) gemm_f32(Gemm G) {
    __shared__ float As[GK][GM + 4];
    __shared__ float Bs[GK][GN + 4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.x * GM, n0 = (int64_t)blockIdx.y * GN;
    const int64_t kb = (int64_t)blockIdx.z * G.k_per, ke = std::min<int64_t>(G.K, kb + G.k_per);
    f4 acc[2][2];
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    float ra[4], rb[4];
    auto gload = [&](int64_t k0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (AKC) {
                const int64_t m = m0 + (tid >> 4) + 16 * q, k = k0 + (tid & 15);
                ra[q] = (m < G.M && k < ke) ? G.A[m * G.lda + k] : 0.f;
            } else {
                const int64_t m = m0 + (tid & 63), k = k0 + (tid >> 6) + 4 * q;
                ra[q] = (m < G.M && k < ke) ? G.A[k * G.lda + m] : 0.f;
            }
            if (BKC) {
                const int64_t n = n0 + (tid >> 4) + 16 * q, k = k0 + (tid & 15);
                rb[q] = (n < G.N && k < ke) ? G.B[n * G.ldb + k] : 0.f;
            } else {
                const int64_t n = n0 + (tid & 63), k = k0 + (tid >> 6) + 4 * q;
                rb[q] = (k < ke && n < G.N) ? (n == G.ones_col ? 1.f : G.B[k * G.ldb + n]) : 0.f;
            }
        }
    };
    if (kb < ke) gload(kb);
    for (int64_t k0 = kb; k0 < ke; k0 += GK) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (AKC) As[tid & 15][(tid >> 4) + 16 * q] = ra[q];
            else As[(tid >> 6) + 4 * q][tid & 63] = ra[q];
            if (BKC) Bs[tid & 15][(tid >> 4) + 16 * q] = rb[q];
            else Bs[(tid >> 6) + 4 * q][tid & 63] = rb[q];
        }
        __syncthreads();
        if (k0 + GK < ke) gload(k0 + GK);
#pragma unroll
        for (int kk = 0; kk < GK; kk += 4) {
            float a[2], b[2];
            for (int i = 0; i < 2; ++i) a[i] = As[kk + (lane >> 4)][wm * 32 + i * 16 + (lane & 15)];
            for (int j = 0; j < 2; ++j) b[j] = Bs[kk + (lane >> 4)][wn * 32 + j * 16 + (lane & 15)];
            for (int i = 0; i < 2; ++i)
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }
    float *C = G.C + (int64_t)blockIdx.z * G.c_split;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 32 + j * 16 + (lane & 15);
            if (n >= G.N) continue;
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * 32 + i * 16 + 4 * (lane >> 4) + v;
                if (m >= G.M) continue;
                float *p = C + m * G.ldc + n;
                *p = G.accumulate ? *p + acc[i][j][v] : acc[i][j][v];
            }
        }
}

// split count for a k-range of K rows over `tiles` output tiles: enough
// blocks to fill the chip, at least 4 k-chunks per split
int64_t split_k_per(int64_t K, int64_t tiles, int64_t *splits) {
    int64_t s = std::max<int64_t>(1, std::min<int64_t>(1024 / std::max<int64_t>(tiles, 1), (K + 63) / 64));
    int64_t per = ((K + s - 1) / s + GK - 1) / GK * GK;
    per = std::max<int64_t>(per, GK);
    *splits = std::max<int64_t>(1, (K + per - 1) / per);
    return per;
}

void launch_gemm(Gemm G, bool a_kc, bool b_kc, int64_t splits, hipStream_t st) {
    if (G.M <= 0 || G.N <= 0) return;
    dim3 grid((unsigned)((G.M + GM - 1) / GM), (unsigned)((G.N + GN - 1) / GN), (unsigned)splits);
    if (a_kc && b_kc) gemm_f32<true, true><<<grid, 256, 0, st>>>(G);
    else if (a_kc) gemm_f32<true, false><<<grid, 256, 0, st>>>(G);
    else if (b_kc) gemm_f32<false, true><<<grid, 256, 0, st>>>(G);
    else gemm_f32<false, false><<<grid, 256, 0, st>>>(G);
}

// out[m ldo + n] (+)= sum_z P[z ps + m ldp + n], z in order
// out[m][n] (+)= sum over the nz split partials P[z][m][n] in a fixed order:
// a block takes 256 / GS consecutive outputs and splits the partials into GS
// contiguous groups (one per thread of an output, eight loads in flight); the
// group sums are added in group order.  GS = 16 for launches with few outputs.
template <int GS>
__global__ void __launch_bounds__(256) sum_splits(const float *P, int64_t ps, int64_t ldp, int32_t nz, int64_t M,
                                                  int64_t N, float *out, int64_t ldo, int accumulate) {
    constexpr int OUT = 256 / GS;
    __shared__ float red[GS][OUT];
    const int o = threadIdx.x % OUT, q = threadIdx.x / OUT;
    const int64_t i = (int64_t)blockIdx.x * OUT + o;
    const bool ok = i < M * N;
    const int64_t m = ok ? i / N : 0, n = ok ? i % N : 0;
    const int32_t per = (nz + GS - 1) / GS, z0 = min(nz, q * per), z1 = min(nz, z0 + per);
    float s = 0.f;
    if (ok) {
        const float *p = P + m * ldp + n;
#pragma unroll 8
        for (int32_t z = z0; z < z1; ++z) s += p[(int64_t)z * ps];
    }
    red[q][o] = s;
    __syncthreads();
    if (q == 0 && ok) {
        float t = 0.f;
#pragma unroll
        for (int g = 0; g < GS; ++g) t += red[g][o];
        float *op = out + m * ldo + n;
        *op = accumulate ? *op + t : t;
    }
}

// launches with at most kFewOutputs outputs use 16 split groups per output
constexpr int64_t kFewOutputs = 8192;
void launch_sum_splits(const float *P, int64_t ps, int64_t ldp, int32_t nz, int64_t M, int64_t N, float *out,
                       int64_t ldo, int accumulate, hipStream_t st) {
    const int64_t outputs = M * N;
    if (outputs <= 0) return;
    if (outputs <= kFewOutputs)
        sum_splits<16><<<(unsigned)((outputs + 15) / 16), 256, 0, st>>>(P, ps, ldp, nz, M, N, out, ldo, accumulate);
    else
        sum_splits<4><<<(unsigned)((outputs + 63) / 64), 256, 0, st>>>(P, ps, ldp, nz, M, N, out, ldo, accumulate);
}

inline unsigned grid_for(int64_t n, int per = 256) {
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>((n + per - 1) / per, 1 << 20));
}

// dW = A^T B over K rows (A: [K][M] rows of stride lda, B: [K][nb] of stride
// ldb, optional ones column at nb), summed over splits into out
// ([M][nb] of stride ldo) and, with a ones column, bias_out [M].
void weight_grad(const float *A, int64_t lda, const float *B, int64_t ldb, int64_t M, int64_t nb, bool ones,
                 int64_t K, float *P, float *out, int64_t ldo, float *bias_out, int accumulate, hipStream_t st,
                 int stage = -1) {
    const int64_t N = nb + (ones ? 1 : 0);
    const int64_t tiles = ((M + GM - 1) / GM) * ((N + GN - 1) / GN);
    int64_t splits;
    const int64_t per = split_k_per(K, tiles, &splits);
    Gemm g{A, lda, B, ldb, M, N, K, ones ? nb : -1, P, N, M * N, per, 0};
    prof_begin(stage, st);
    launch_gemm(g, false, false, splits, st);
    prof_end(stage, st);
    launch_sum_splits(P, M * N, N, (int32_t)splits, M, nb, out, ldo, accumulate, st);
    if (ones) launch_sum_splits(P + nb, M * N, N, (int32_t)splits, M, 1, bias_out, 1, accumulate, st);
}

// ------------------------------------------------------------- layer backward
struct BwdLayer {
    int32_t R;
    int F;
    const float *att_src, *att_dst;   // [3][F] of the layer
    const float *U, *cp;              // [3][F][2], [3][F]
    const float *x_oo; int64_t s_oo;
    const float *x_dd; int64_t s_dd;
    const uint8_t *x_od; int64_t s_od;
    float slope;
};

// One destination bucket of the forward pass.
struct BwdBucket {
    const int32_t *rp, *col, *eid;
    int64_t n_dst, n_src;             // rows per replica
    const float *Ydst; int ydst_off;  // saved Y rows ([R*n][2F]) and the relation's half
    const float *Ysrc; int ysrc_off;
    const float *dO; float gamma;     // gradient rows of the destinations [R*n_dst][F]
    int rel, xkind, twin;             // xkind 0 oo (log size), 1 od (bit), 2 dd (two values)
    float *SA, *SD;                   // [R][n_slots][K]
    int64_t n_slots;
    int32_t chunks;                   // kChunkA-entry chunks per row (max degree)
    float *Z; int zsel;               // [R*n_dst][2][K] per-destination dz sums
    int spos;                         // slot = the entry's position in this bucket
    const int32_t *smap;              // else, if set: slot = smap[position]
};

constexpr int kChunkA = 32;     // entries per score item
constexpr int kChunkB = 128;    // entries per message item
constexpr int kPersist = 2048;  // blocks of the passes that sum parameter gradients
constexpr int kLongRow = 256;   // buckets with rows this long (max degree) take the entry-per-lane softmax

__device__ __forceinline__ void edge_x(const BwdLayer &P, int xkind, int32_t rep, int32_t id, float &x0, float &x1) {
    if (xkind == 0) {
        x0 = P.x_oo[(int64_t)rep * P.s_oo + id];
        x1 = 0.f;
    } else if (xkind == 1) {
        x0 = P.x_od[(int64_t)rep * P.s_od + id] ? 1.f : 0.f;
        x1 = 0.f;
    } else {
        const float *p = P.x_dd + (int64_t)rep * P.s_dd + 2 * (int64_t)id;
        x0 = p[0];
        x1 = p[1];
    }
}

// sum over the LPH lanes of a head (DPP inside 16-lane rows, then shuffles)
template <int LPH>
__device__ __forceinline__ float hsum(float v) {
    v = row_sum<(LPH < 16 ? LPH : 16)>(v);
    if constexpr (LPH >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (LPH >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

__device__ __forceinline__ int64_t slot_of(int twin, int32_t id, int32_t dst, int32_t src) {
    return twin ? 2 * (int64_t)id + (dst > src ? 1 : 0) : (int64_t)id;
}

// slot of the entry at position e of a bucket walk
__device__ __forceinline__ int64_t entry_slot(int spos, const int32_t *smap, int32_t e, int twin, int32_t id,
                                              int32_t dst, int32_t src) {
    return spos ? (int64_t)e : (smap ? (int64_t)smap[e] : slot_of(twin, id, dst, src));
}

// scores: one wavefront per (replica, destination row, chunk of kChunkA
// entries); lanes own F/64 channels; writes s and dalpha per (entry, head)
template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_scores(BwdLayer P, BwdBucket B) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t rows = (int64_t)P.R * B.n_dst;
    if (w >= rows * B.chunks) return;
    const int64_t ru = w / B.chunks;
    const int32_t ch = (int32_t)(w % B.chunks);
    const int32_t rep = (int32_t)(ru / B.n_dst), u = (int32_t)(ru % B.n_dst);
    const int32_t beg = B.rp[u] + ch * kChunkA, end = min(B.rp[u + 1], beg + kChunkA);
    if (beg >= end) return;
    const int c0 = lane * CPL;
    const int r = B.rel;
    float a[CPL], u0[CPL], u1[CPL], yd[CPL], dO[CPL];
    load_ch<CPL, false>(B.Ydst, ru * 2 * F + B.ydst_off + c0, yd);
    load_ch<CPL, false>(B.dO, ru * F + c0, dO);
    float q = 0.f;
    for (int c = 0; c < CPL; ++c) {
        a[c] = P.att_src[r * F + c0 + c];
        u0[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 0];
        u1[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 1];
        q = fmaf(P.att_dst[r * F + c0 + c], yd[c] - P.cp[r * F + c0 + c], q);
        dO[c] *= B.gamma;
    }
    q = hsum<LPH>(q);
    const int64_t sbase = (int64_t)rep * B.n_slots;
    constexpr int EB = 4;
    for (int32_t e0 = beg; e0 < end; e0 += EB) {
        float ys[EB][CPL], x0[EB], x1[EB];
        int32_t vv[EB], id[EB];
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            const int32_t e = min(e0 + i, end - 1);
            vv[i] = B.col[e];
            id[i] = B.eid[e];
        }
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            load_ch<CPL, false>(B.Ysrc, ((int64_t)rep * B.n_src + vv[i]) * 2 * F + B.ysrc_off + c0, ys[i]);
            edge_x(P, B.xkind, rep, id[i], x0[i], x1[i]);
        }
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            float pa = 0.f, pd = 0.f;
            for (int c = 0; c < CPL; ++c) {
                const float m = msg_act<ELU>(ys[i][c] + fmaf(u0[c], x0[i], u1[c] * x1[i]));
                pa = fmaf(a[c], m, pa);
                pd = fmaf(dO[c], m, pd);
            }
            pa = hsum<LPH>(pa);
            pd = hsum<LPH>(pd);
            const float s = leaky(pa + q, P.slope);
            if (e0 + i < end && (lane & (LPH - 1)) == 0) {
                const int64_t slot = entry_slot(B.spos, B.smap, e0 + i, B.twin, id[i], u, vv[i]);
                const int64_t idx = (sbase + slot) * K + lane / LPH;
                B.SA[idx] = s;
                B.SD[idx] = pd;
            }
        }
    }
}

// scores of short rows (buckets whose rows fit one kChunkA chunk): four
// rows per wavefront, 16 lanes per row with F/16 channels per lane (heads of
// at least F/16 channels); the same values as bwd_scores
template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_scores_short(BwdLayer P, BwdBucket B) {
    constexpr int CPE = F / 16, LPH = 16 / K, EB = 4;
    static_assert(K <= 16, "16-lane rows need heads of at least f/16 channels");
    const int lane = threadIdx.x & 63, grp = lane >> 4, jl = lane & 15;
    const int64_t ru = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 4 + grp;
    const int64_t rows = (int64_t)P.R * B.n_dst;
    const bool have = ru < rows;
    const int32_t rep = have ? (int32_t)(ru / B.n_dst) : 0, u = have ? (int32_t)(ru % B.n_dst) : 0;
    const int32_t beg = have ? B.rp[u] : 0, n = have ? B.rp[u + 1] - beg : 0;
    const int c0 = jl * CPE, h = c0 / (F / K);
    const int r = B.rel;
    float a[CPE], u0[CPE], u1[CPE], yd[CPE], dO[CPE];
    load_ch<CPE, false>(B.Ydst, (have ? ru : 0) * 2 * F + B.ydst_off + c0, yd);
    load_ch<CPE, false>(B.dO, (have ? ru : 0) * F + c0, dO);
    float q = 0.f;
    for (int c = 0; c < CPE; ++c) {
        a[c] = P.att_src[r * F + c0 + c];
        u0[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 0];
        u1[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 1];
        q = fmaf(P.att_dst[r * F + c0 + c], yd[c] - P.cp[r * F + c0 + c], q);
        dO[c] *= B.gamma;
    }
    q = row_sum<LPH>(q);
    int32_t nmax = n;   // the wavefront's longest row
    nmax = max(nmax, __shfl_xor(nmax, 16, 64));
    nmax = max(nmax, __shfl_xor(nmax, 32, 64));
    const int64_t sbase = (int64_t)rep * B.n_slots;
    for (int32_t i0 = 0; i0 < nmax; i0 += EB) {
        float ys[EB][CPE], x0[EB], x1[EB];
        int32_t vv[EB], id[EB];
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            const int32_t e = i0 + i < n ? beg + i0 + i : 0;   // rows past their end read entry 0
            vv[i] = B.col[e];
            id[i] = B.eid[e];
        }
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            load_ch<CPE, false>(B.Ysrc, ((int64_t)rep * B.n_src + vv[i]) * 2 * F + B.ysrc_off + c0, ys[i]);
            edge_x(P, B.xkind, rep, id[i], x0[i], x1[i]);
        }
#pragma unroll
        for (int i = 0; i < EB; ++i) {
            float pa = 0.f, pd = 0.f;
            for (int c = 0; c < CPE; ++c) {
                const float m = msg_act<ELU>(ys[i][c] + fmaf(u0[c], x0[i], u1[c] * x1[i]));
                pa = fmaf(a[c], m, pa);
                pd = fmaf(dO[c], m, pd);
            }
            pa = row_sum<LPH>(pa);
            pd = row_sum<LPH>(pd);
            const float sv = leaky(pa + q, P.slope);
            if (i0 + i < n && (jl % LPH) == 0) {
                const int32_t e = beg + i0 + i;
                const int64_t slot = entry_slot(B.spos, B.smap, e, B.twin, id[i], u, vv[i]);
                const int64_t idx = (sbase + slot) * K + h;
                B.SA[idx] = sv;
                B.SD[idx] = pd;
            }
        }
    }
}

// online softmax statistics: fold logit s with weight d into (max, sum, weighted sum)
__device__ __forceinline__ void softmax_fold(float s, float d, float &mx, float &den, float &num) {
    if (s > mx) {
        const float sc = __expf(mx - s);
        den = fmaf(den, sc, 1.f);
        num = fmaf(num, sc, d);
        mx = s;
    } else {
        const float p = __expf(s - mx);
        den += p;
        num = fmaf(p, d, num);
    }
}

// merge another lane's (max, sum, weighted sum) into this lane's
__device__ __forceinline__ void softmax_merge(float m2, float d2, float n2, float &mx, float &den, float &num) {
    const float M = fmaxf(mx, m2);
    if (M == -INFINITY) return;
    const float s1 = mx == -INFINITY ? 0.f : __expf(mx - M), s2 = m2 == -INFINITY ? 0.f : __expf(m2 - M);
    den = den * s1 + d2 * s2;
    num = num * s1 + n2 * s2;
    mx = M;
}

// Softmax backward of one long row (rows of hundreds of entries): lanes over
// entries, each lane all K heads of its entry, two 64-entry rounds of loads
// in flight; returns the row's Z per head in every lane.
template <int K>
__device__ void softmax_row_long(const BwdLayer &P, const BwdBucket &B, int32_t u, int32_t beg, int32_t end,
                                 int64_t sbase, int lane, float (&Z)[K]) {
    constexpr int U = 2;
    auto slot_at = [&](int32_t e) -> int64_t {
        return B.spos ? (int64_t)e : (B.smap ? (int64_t)B.smap[e] : slot_of(B.twin, B.eid[e], u, B.col[e]));
    };
    float mx[K], den[K], num[K];
#pragma unroll
    for (int k = 0; k < K; ++k) { mx[k] = -INFINITY; den[k] = num[k] = 0.f; }
    for (int32_t e0 = beg; e0 < end; e0 += 64 * U) {
        int64_t sl[U];
        bool ok[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int32_t e = e0 + 64 * j + lane;
            ok[j] = e < end;
            sl[j] = ok[j] ? slot_at(e) : 0;
        }
        float sv[U][K], dv[U][K];
#pragma unroll
        for (int j = 0; j < U; ++j)
#pragma unroll
            for (int k = 0; k < K; ++k) {
                sv[j][k] = ok[j] ? B.SA[(sbase + sl[j]) * K + k] : 0.f;
                dv[j][k] = ok[j] ? B.SD[(sbase + sl[j]) * K + k] : 0.f;
            }
#pragma unroll
        for (int j = 0; j < U; ++j)
            if (ok[j])
#pragma unroll
                for (int k = 0; k < K; ++k) softmax_fold(sv[j][k], dv[j][k], mx[k], den[k], num[k]);
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1)
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float m2 = __shfl_xor(mx[k], o, 64), d2 = __shfl_xor(den[k], o, 64), n2 = __shfl_xor(num[k], o, 64);
            softmax_merge(m2, d2, n2, mx[k], den[k], num[k]);
        }
    float inv[K], cc[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        inv[k] = den[k] > 0.f ? 1.f / den[k] : 0.f;
        cc[k] = num[k] * inv[k];
        Z[k] = 0.f;
    }
    for (int32_t e0 = beg; e0 < end; e0 += 64 * U) {
        int64_t sl[U];
        bool ok[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int32_t e = e0 + 64 * j + lane;
            ok[j] = e < end;
            sl[j] = ok[j] ? slot_at(e) : 0;
        }
        float sv[U][K], dv[U][K];
#pragma unroll
        for (int j = 0; j < U; ++j)
#pragma unroll
            for (int k = 0; k < K; ++k) {
                sv[j][k] = ok[j] ? B.SA[(sbase + sl[j]) * K + k] : 0.f;
                dv[j][k] = ok[j] ? B.SD[(sbase + sl[j]) * K + k] : 0.f;
            }
#pragma unroll
        for (int j = 0; j < U; ++j)
            if (ok[j])
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const float s = sv[j][k];
                    const float al = __expf(s - mx[k]) * inv[k];
                    const float dz = al * (dv[j][k] - cc[k]) * (s > 0.f ? 1.f : P.slope);
                    B.SA[(sbase + sl[j]) * K + k] = al;
                    B.SD[(sbase + sl[j]) * K + k] = dz;
                    Z[k] += dz;
                }
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1)
#pragma unroll
        for (int k = 0; k < K; ++k) Z[k] += __shfl_xor(Z[k], o, 64);
}

// softmax backward: one wavefront per (replica, destination row), lanes
// over (entry, head) pairs (LONG: lanes over entries, see softmax_row_long);
// turns (s, dalpha) into (alpha, dz) in place, writes Z_u and sums
// d adst = Z_u (Y_u - c') per block
template <int F, int K, bool LONG>
__global__ void __launch_bounds__(256) bwd_softmax(BwdLayer P, BwdBucket B, float *part_ad) {
    constexpr int CPL = F / 64, EPS = 64 / K, D = F / K;
    __shared__ float red[4][F];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int ei = lane / K, k = lane % K;
    const int c0 = lane * CPL;
    const int r = B.rel;
    float acc[CPL], ad[CPL], cp[CPL];
    for (int c = 0; c < CPL; ++c) {
        acc[c] = 0.f;
        ad[c] = P.att_dst[r * F + c0 + c];
        cp[c] = P.cp[r * F + c0 + c];
    }
    const int64_t rows = (int64_t)P.R * B.n_dst;
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t ru = (int64_t)blockIdx.x * 4 + wv; ru < rows; ru += nw) {
        const int32_t rep = (int32_t)(ru / B.n_dst), u = (int32_t)(ru % B.n_dst);
        const int32_t beg = B.rp[u], end = B.rp[u + 1];
        const int64_t sbase = (int64_t)rep * B.n_slots;
        float zh;
        if constexpr (LONG) {
            float Zk[K];
            softmax_row_long<K>(P, B, u, beg, end, sbase, lane, Zk);
            zh = 0.f;
#pragma unroll
            for (int kk = 0; kk < K; ++kk) {
                if (kk == c0 / D) zh = Zk[kk];
                if (lane == kk) B.Z[(ru * 2 + B.zsel) * K + kk] = Zk[kk];
            }
        } else {
            float mx = -INFINITY, den = 0.f, num = 0.f;
            for (int32_t e0 = beg; e0 < end; e0 += EPS) {
                const int32_t e = e0 + ei;
                if (e < end) {
                    const int64_t slot = B.spos ? (int64_t)e
                                                : (B.smap ? (int64_t)B.smap[e] : slot_of(B.twin, B.eid[e], u, B.col[e]));
                    const int64_t idx = (sbase + slot) * K + k;
                    softmax_fold(B.SA[idx], B.SD[idx], mx, den, num);
                }
            }
            for (int o = K; o < 64; o <<= 1) {
                const float m2 = __shfl_xor(mx, o, 64), d2 = __shfl_xor(den, o, 64), n2 = __shfl_xor(num, o, 64);
                softmax_merge(m2, d2, n2, mx, den, num);
            }
            const float inv = den > 0.f ? 1.f / den : 0.f;
            const float cc = num * inv;
            float zs = 0.f;
            for (int32_t e0 = beg; e0 < end; e0 += EPS) {
                const int32_t e = e0 + ei;
                if (e < end) {
                    const int64_t slot = B.spos ? (int64_t)e
                                                : (B.smap ? (int64_t)B.smap[e] : slot_of(B.twin, B.eid[e], u, B.col[e]));
                    const int64_t idx = (sbase + slot) * K + k;
                    const float s = B.SA[idx], da = B.SD[idx];
                    const float al = __expf(s - mx) * inv;
                    const float dz = al * (da - cc) * (s > 0.f ? 1.f : P.slope);
                    B.SA[idx] = al;
                    B.SD[idx] = dz;
                    zs += dz;
                }
            }
            for (int o = K; o < 64; o <<= 1) zs += __shfl_xor(zs, o, 64);
            if (ei == 0) B.Z[(ru * 2 + B.zsel) * K + k] = zs;
            zh = __shfl(zs, c0 / D, 64);   // lane h < K holds head h
        }
        if (end > beg) {
            float yd[CPL];
            load_ch<CPL, false>(B.Ydst, ru * 2 * F + B.ydst_off + c0, yd);
            for (int c = 0; c < CPL; ++c) acc[c] = fmaf(zh, yd[c] - cp[c], acc[c]);
        }
    }
    for (int c = 0; c < CPL; ++c) red[wv][c0 + c] = acc[c];
    __syncthreads();
    for (int c = threadIdx.x; c < F; c += 256)
        part_ad[(int64_t)blockIdx.x * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
}

// softmax backward of short rows (single-chunk buckets): persistent
// wavefronts over quads of destination rows, 16 lanes per row over (entry,
// head) pairs for the statistics and over F/16 channels for d adst; the same
// values as bwd_softmax
template <int F, int K>
__global__ void __launch_bounds__(256) bwd_softmax_short(BwdLayer P, BwdBucket B, float *part_ad) {
    constexpr int CPE = F / 16, EPS = 16 / K, D = F / K;
    static_assert(K <= 16, "16-lane rows need heads of at least f/16 channels");
    __shared__ float red[4][F];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4, jl = lane & 15;
    const int ei = jl / K, k = jl % K;
    const int c0 = jl * CPE;
    const int r = B.rel;
    float acc[CPE], cp[CPE];
    for (int c = 0; c < CPE; ++c) {
        acc[c] = 0.f;
        cp[c] = P.cp[r * F + c0 + c];
    }
    const int64_t rows = (int64_t)P.R * B.n_dst;
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t qd = (int64_t)blockIdx.x * 4 + wv; qd * 4 < rows; qd += nw) {
        const int64_t ru = qd * 4 + grp;
        const bool have = ru < rows;
        const int32_t rep = have ? (int32_t)(ru / B.n_dst) : 0, u = have ? (int32_t)(ru % B.n_dst) : 0;
        const int32_t beg = have ? B.rp[u] : 0, end = have ? B.rp[u + 1] : 0;
        int32_t nmax = end - beg;   // the wavefront's longest row
        nmax = max(nmax, __shfl_xor(nmax, 16, 64));
        nmax = max(nmax, __shfl_xor(nmax, 32, 64));
        const int64_t sbase = (int64_t)rep * B.n_slots;
        auto slot_at = [&](int32_t e) -> int64_t {
            return B.spos ? (int64_t)e : (B.smap ? (int64_t)B.smap[e] : slot_of(B.twin, B.eid[e], u, B.col[e]));
        };
        float mx = -INFINITY, den = 0.f, num = 0.f;
        for (int32_t j0 = 0; j0 < nmax; j0 += EPS) {
            const int32_t e = beg + j0 + ei;
            if (e < end) {
                const int64_t idx = (sbase + slot_at(e)) * K + k;
                softmax_fold(B.SA[idx], B.SD[idx], mx, den, num);
            }
        }
        for (int o = K; o < 16; o <<= 1) {
            const float m2 = __shfl_xor(mx, o, 64), d2 = __shfl_xor(den, o, 64), n2 = __shfl_xor(num, o, 64);
            softmax_merge(m2, d2, n2, mx, den, num);
        }
        const float inv = den > 0.f ? 1.f / den : 0.f, cc = num * inv;
        float zs = 0.f;
        for (int32_t j0 = 0; j0 < nmax; j0 += EPS) {
            const int32_t e = beg + j0 + ei;
            if (e < end) {
                const int64_t idx = (sbase + slot_at(e)) * K + k;
                const float sv = B.SA[idx], da = B.SD[idx];
                const float al = __expf(sv - mx) * inv;
                const float dz = al * (da - cc) * (sv > 0.f ? 1.f : P.slope);
                B.SA[idx] = al;
                B.SD[idx] = dz;
                zs += dz;
            }
        }
        for (int o = K; o < 16; o <<= 1) zs += __shfl_xor(zs, o, 64);
        if (have && ei == 0) B.Z[(ru * 2 + B.zsel) * K + k] = zs;
        const float zh = __shfl(zs, grp * 16 + c0 / D, 64);   // lane h of the group holds head h
        if (have && end > beg) {
            float yd[CPE];
            load_ch<CPE, false>(B.Ydst, ru * 2 * F + B.ydst_off + c0, yd);
            for (int c = 0; c < CPE; ++c) acc[c] = fmaf(zh, yd[c] - cp[c], acc[c]);
        }
    }
    // the four row groups' sums, then the wavefronts' in order
    for (int c = 0; c < CPE; ++c) {
        acc[c] += __shfl_xor(acc[c], 16, 64);
        acc[c] += __shfl_xor(acc[c], 32, 64);
    }
    if (grp == 0)
        for (int c = 0; c < CPE; ++c) red[wv][c0 + c] = acc[c];
    __syncthreads();
    for (int c = threadIdx.x; c < F; c += 256)
        part_ad[(int64_t)blockIdx.x * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
}

// Rows of one node type as sources: the entries they feed, listed by the
// bucket in which the row is the destination of the same relation.
struct BwdSrc {
    const int32_t *rp, *col, *eid;
    int64_t n_self, n_nbr;
    const float *Yself; int yoff;
    const float *dOn; float gamma;    // gradient rows of the neighbours (forward destinations)
    const float *SA, *SD;             // (alpha, dz) of the forward bucket nbr <- self
    int64_t n_slots;
    int twin, rel, xkind;
    const float *Z; int zsel;         // Z of the row as a destination of the relation
    float *dY; int dyoff;             // [R*n_self][2F]
    float *PB;                        // [R*n_self][chunks][F] chunk partials (chunks > 1)
    int32_t chunks;
    int spos;                         // slot = the entry's position in this bucket
    const int32_t *smap;              // else, if set: slot = smap[position]
};

// messages: persistent wavefronts over (replica, source row, chunk of
// kChunkB entries); dY rows (or chunk partials) and per-block sums of
// d a, dU (two columns) and dc'
template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_messages(BwdLayer P, BwdSrc S, float *part) {
    constexpr int CPL = F / 64, D = F / K;
    __shared__ float red[4][F];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c0 = lane * CPL, h = c0 / D;
    const int r = S.rel;
    float a[CPL], ad[CPL], u0[CPL], u1[CPL];
    float ga[CPL], gu0[CPL], gu1[CPL], gcp[CPL];
    for (int c = 0; c < CPL; ++c) {
        a[c] = P.att_src[r * F + c0 + c];
        ad[c] = P.att_dst[r * F + c0 + c];
        u0[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 0];
        u1[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 1];
        ga[c] = gu0[c] = gu1[c] = gcp[c] = 0.f;
    }
    const int64_t items = (int64_t)P.R * S.n_self * S.chunks;
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t it = (int64_t)blockIdx.x * 4 + wv; it < items; it += nw) {
        const int64_t rv = it / S.chunks;
        const int32_t ch = (int32_t)(it % S.chunks);
        const int32_t rep = (int32_t)(rv / S.n_self), v = (int32_t)(rv % S.n_self);
        const int32_t beg = S.rp[v] + ch * kChunkB, end = min(S.rp[v + 1], beg + kChunkB);
        if (ch > 0 && beg >= end) continue;
        float ys[CPL], dys[CPL];
        load_ch<CPL, false>(S.Yself, rv * 2 * F + S.yoff + c0, ys);
        for (int c = 0; c < CPL; ++c) dys[c] = 0.f;
        const int64_t sbase = (int64_t)rep * S.n_slots;
        constexpr int EB = 4;
        for (int32_t e0 = beg; e0 < end; e0 += EB) {
            float dou[EB][CPL], x0[EB], x1[EB], al[EB], dz[EB];
            int32_t uu[EB], id[EB];
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                const int32_t e = min(e0 + i, end - 1);
                uu[i] = S.col[e];
                id[i] = S.eid[e];
            }
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                load_ch<CPL, false>(S.dOn, ((int64_t)rep * S.n_nbr + uu[i]) * F + c0, dou[i]);
                edge_x(P, S.xkind, rep, id[i], x0[i], x1[i]);
                const int64_t slot = entry_slot(S.spos, S.smap, min(e0 + i, end - 1), S.twin, id[i], uu[i], v);
                const int64_t idx = (sbase + slot) * K + h;
                al[i] = S.SA[idx];
                dz[i] = S.SD[idx];
            }
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                if (e0 + i >= end) break;
                for (int c = 0; c < CPL; ++c) {
                    const float pre = ys[c] + fmaf(u0[c], x0[i], u1[c] * x1[i]);
                    const float m = msg_act<ELU>(pre);
                    const float dm = fmaf(al[i] * S.gamma, dou[i][c], dz[i] * a[c]);
                    // sigma'(pre): ReLU 1 / 0, ELU 1 / e^pre (= m + 1)
                    const float dp = pre > 0.f ? dm : (ELU ? dm * (m + 1.f) : 0.f);
                    dys[c] += dp;
                    ga[c] = fmaf(dz[i], m, ga[c]);
                    gu0[c] = fmaf(dp, x0[i], gu0[c]);
                    gu1[c] = fmaf(dp, x1[i], gu1[c]);
                    gcp[c] += dp;
                }
            }
        }
        if (S.chunks == 1) {
            const float zv = S.Z[(rv * 2 + S.zsel) * K + h];
            float *o = S.dY + rv * 2 * F + S.dyoff + c0;
            for (int c = 0; c < CPL; ++c) o[c] = fmaf(zv, ad[c], dys[c]);
        } else {
            float *o = S.PB + (rv * S.chunks + ch) * F + c0;
            for (int c = 0; c < CPL; ++c) o[c] = dys[c];
        }
    }
    float *q[4] = {ga, gu0, gu1, gcp};
    for (int t = 0; t < 4; ++t) {
        for (int c = 0; c < CPL; ++c) red[wv][c0 + c] = q[t][c];
        __syncthreads();
        for (int c = threadIdx.x; c < F; c += 256)
            part[((int64_t)t * gridDim.x + blockIdx.x) * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
        __syncthreads();
    }
}

// messages of short source rows (single-chunk buckets): persistent
// wavefronts over quads of source rows, 16 lanes per row with F/16 channels
// per lane (heads of at least F/16 channels), four entries in flight (two
// at F = 256); the
// same values and block sums as bwd_messages
template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_messages_short(BwdLayer P, BwdSrc S, float *part) {
    constexpr int CPE = F / 16, D = F / K, EB = F >= 256 ? 2 : 4;   // entries in flight (register budget)
    static_assert(K <= 16, "16-lane rows need heads of at least f/16 channels");
    __shared__ float red[4][F];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4, jl = lane & 15;
    const int c0 = jl * CPE, h = c0 / D;
    const int r = S.rel;
    float a[CPE], ad[CPE], u0[CPE], u1[CPE];
    float ga[CPE], gu0[CPE], gu1[CPE], gcp[CPE];
    for (int c = 0; c < CPE; ++c) {
        a[c] = P.att_src[r * F + c0 + c];
        ad[c] = P.att_dst[r * F + c0 + c];
        u0[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 0];
        u1[c] = P.U[((int64_t)r * F + c0 + c) * 2 + 1];
        ga[c] = gu0[c] = gu1[c] = gcp[c] = 0.f;
    }
    const int64_t rows = (int64_t)P.R * S.n_self;
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t qd = (int64_t)blockIdx.x * 4 + wv; qd * 4 < rows; qd += nw) {
        const int64_t rv = qd * 4 + grp;
        const bool have = rv < rows;
        const int32_t rep = have ? (int32_t)(rv / S.n_self) : 0, v = have ? (int32_t)(rv % S.n_self) : 0;
        const int32_t beg = have ? S.rp[v] : 0, n = have ? S.rp[v + 1] - beg : 0;
        int32_t nmax = n;   // the wavefront's longest row
        nmax = max(nmax, __shfl_xor(nmax, 16, 64));
        nmax = max(nmax, __shfl_xor(nmax, 32, 64));
        float ys[CPE], dys[CPE];
        load_ch<CPE, false>(S.Yself, (have ? rv : 0) * 2 * F + S.yoff + c0, ys);
        for (int c = 0; c < CPE; ++c) dys[c] = 0.f;
        const int64_t sbase = (int64_t)rep * S.n_slots;
        for (int32_t i0 = 0; i0 < nmax; i0 += EB) {
            float dou[EB][CPE], x0[EB], x1[EB], al[EB], dz[EB];
            int32_t uu[EB], id[EB];
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                const int32_t e = i0 + i < n ? beg + i0 + i : 0;   // rows past their end read entry 0
                uu[i] = S.col[e];
                id[i] = S.eid[e];
            }
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                const int32_t e = i0 + i < n ? beg + i0 + i : 0;
                load_ch<CPE, false>(S.dOn, ((int64_t)rep * S.n_nbr + uu[i]) * F + c0, dou[i]);
                edge_x(P, S.xkind, rep, id[i], x0[i], x1[i]);
                const int64_t slot = entry_slot(S.spos, S.smap, e, S.twin, id[i], uu[i], v);
                const int64_t idx = (sbase + slot) * K + h;
                al[i] = S.SA[idx];
                dz[i] = S.SD[idx];
            }
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                if (i0 + i >= n) continue;
                for (int c = 0; c < CPE; ++c) {
                    const float pre = ys[c] + fmaf(u0[c], x0[i], u1[c] * x1[i]);
                    const float m = msg_act<ELU>(pre);
                    const float dm = fmaf(al[i] * S.gamma, dou[i][c], dz[i] * a[c]);
                    const float dp = pre > 0.f ? dm : (ELU ? dm * (m + 1.f) : 0.f);
                    dys[c] += dp;
                    ga[c] = fmaf(dz[i], m, ga[c]);
                    gu0[c] = fmaf(dp, x0[i], gu0[c]);
                    gu1[c] = fmaf(dp, x1[i], gu1[c]);
                    gcp[c] += dp;
                }
            }
        }
        if (have) {
            const float zv = S.Z[(rv * 2 + S.zsel) * K + h];
            float *o = S.dY + rv * 2 * F + S.dyoff + c0;
            for (int c = 0; c < CPE; ++c) o[c] = fmaf(zv, ad[c], dys[c]);
        }
    }
    // the four row groups' sums, then the wavefronts' in order
    auto flush = [&](int t, float (&qv)[CPE]) {
        for (int c = 0; c < CPE; ++c) {
            qv[c] += __shfl_xor(qv[c], 16, 64);
            qv[c] += __shfl_xor(qv[c], 32, 64);
        }
        if (grp == 0)
            for (int c = 0; c < CPE; ++c) red[wv][c0 + c] = qv[c];
        __syncthreads();
        for (int c = threadIdx.x; c < F; c += 256)
            part[((int64_t)t * gridDim.x + blockIdx.x) * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
        __syncthreads();
    };
    flush(0, ga);
    flush(1, gu0);
    flush(2, gu1);
    flush(3, gcp);
}

// dY rows of sources with several chunks: the row's chunk partials summed
// in order, plus Z adst (heads of D = F / K channels)
__global__ void bwd_combine(BwdLayer P, BwdSrc S, int K) {
    const int F = P.F, D = F / K;
    const int r = S.rel;
    const int64_t total = (int64_t)P.R * S.n_self * F;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t rv = i / F;
        const int c = (int)(i % F);
        const int32_t v = (int32_t)(rv % S.n_self);
        const int32_t deg = S.rp[v + 1] - S.rp[v];
        const int32_t nch = max(1, (deg + kChunkB - 1) / kChunkB);
        float s = 0.f;
        for (int32_t ch = 0; ch < nch; ++ch) s += S.PB[(rv * S.chunks + ch) * F + c];
        S.dY[rv * 2 * F + S.dyoff + c] = fmaf(S.Z[(rv * 2 + S.zsel) * K + c / D], P.att_dst[r * F + c], s);
    }
}

// ------------------------------------------------------- op-device tiles
// Op-device links carry only the placement bit, so a device row's message
// has two forms (bit 0 / 1).  One block per (replica, tile of consecutive
// ops of one topology) stages the topology's device message rows, gradient
// rows and attention terms in LDS and walks the tile's ops: op rows are
// read once, and both directions of every op-device link are handled from
// the op's side (the long device rows are never walked).
struct OdTile {
    const int32_t *tiles;          // [n_tiles][3]: first op (global), op count, topology
    const int32_t *dev_off;        // [G+1]
    const int32_t *rp, *col, *eid; // op<-device bucket (rows: ops)
    int64_t n_op, n_dev, n_slots;
    const float *Y_op, *Y_dev;     // saved Y rows, od half at +F
    const float *dO_op, *dO_dev;   // gradient rows of the layer outputs
    float gamma;
    float *SA1, *SD1, *SA2, *SD2;  // slots of op<-device and device<-op entries
    float *Zop, *Zdev;             // [rows][2][K]; od at 1 (written by the tile kernels)
    float *dY_op, *dY_dev;         // od halves: dY_op + F, dY_dev + 0
    float *PD;                     // [R][n_tiles][max_dev][F] device partials
    int32_t max_dev, n_tiles;
    const int32_t *tile_off;       // [G+1]
    float *part;                   // [4][nb][F] parameter partials (da, dU0, dU1, dc')
    // softmax of both op-device directions inside the tile kernels
    float *part_a1;                // [R*n_tiles][F] d adst sums over the tile's op rows
    float *drec;                   // [R*n_tiles][max_dev][K][3] device<-op records (max, sum, weighted sum)
    float *dstat;                  // [R*n_dev][K][3] merged device statistics (max, 1/sum, c)
    float *zrec;                   // [R*n_tiles][max_dev][K] sums of dz over the tile's device<-op entries
    float *part_a2;                // [ceil(R*n_dev/4)][F] d adst sums over device rows
};

// LDS row stride of the staged device rows (+4 floats: the four entry
// groups of a wavefront read different rows at the same channels)
template <int F>
constexpr int od_stride() { return F + 4; }

// Block set-up of the tile kernels: the tile's row pointers, one byte per
// tile entry (local device index | placement bit << 7, read coalesced from
// the entry range of the tile), and the device rows of the tile's topology:
// messages for both bits, gamma dO rows and (TERMS) attention logit terms
// and destination terms.
template <int F, int K, bool ELU, bool TERMS>
__device__ void od_stage(const BwdLayer &P, const OdTile &T, int32_t rep, int32_t u0, int32_t n, int32_t d0,
                         int32_t nd, float *md, float *dod, float *pd, float *qdd, int32_t *rps, uint8_t *ent) {
    constexpr int D = F / K, FS = od_stride<F>();
    constexpr int RU = 8, EU = 4;   // loads issued together per thread (rows, entries)
    const float *a = P.att_src + F, *ad = P.att_dst + F, *cp = P.cp + F;
    const int tid = threadIdx.x, nt = blockDim.x;
    for (int i = tid; i <= n; i += nt) rps[i] = T.rp[u0 + i];
    const int32_t e0 = T.rp[u0], ne = T.rp[u0 + n] - e0;
    const uint8_t *xb = P.x_od + (int64_t)rep * P.s_od;
    for (int i0 = tid; i0 < ne; i0 += EU * nt) {
        int32_t cl[EU], id[EU];
#pragma unroll
        for (int j = 0; j < EU; ++j) {
            const int i = min(i0 + j * nt, ne - 1);
            cl[j] = T.col[e0 + i];
            id[j] = T.eid[e0 + i];
        }
        uint8_t xv[EU];
#pragma unroll
        for (int j = 0; j < EU; ++j) xv[j] = xb[id[j]];
#pragma unroll
        for (int j = 0; j < EU; ++j)
            if (i0 + j * nt < ne) ent[i0 + j * nt] = (uint8_t)((cl[j] - d0) | (xv[j] ? 0x80 : 0));
    }
    const int total = nd * F;
    for (int i0 = tid; i0 < total; i0 += RU * nt) {
        float y[RU], g[RU], u[RU];
#pragma unroll
        for (int j = 0; j < RU; ++j) {
            const int i = min(i0 + j * nt, total - 1);
            const int v = i / F, c = i % F;
            const int64_t row = (int64_t)rep * T.n_dev + d0 + v;
            y[j] = T.Y_dev[row * 2 * F + F + c];
            g[j] = T.dO_dev[row * F + c];
            u[j] = P.U[((int64_t)F + c) * 2 + 0];
        }
#pragma unroll
        for (int j = 0; j < RU; ++j) {
            const int i = i0 + j * nt;
            if (i < total) {
                const int v = i / F, c = i % F;
                md[(v * 2 + 0) * FS + c] = msg_act<ELU>(y[j]);
                md[(v * 2 + 1) * FS + c] = msg_act<ELU>(y[j] + u[j]);
                dod[v * FS + c] = T.gamma * g[j];
            }
        }
    }
    if constexpr (TERMS) {
        __syncthreads();
        for (int i = tid; i < nd * 3 * K; i += nt) {
            const int v = i / (3 * K), r = i % (3 * K), x = r / K, k = r % K;
            float t = 0.f;
            if (x < 2) {
                for (int c = k * D; c < (k + 1) * D; ++c) t = fmaf(a[c], md[(v * 2 + x) * FS + c], t);
                pd[(v * 2 + x) * K + k] = t;
            } else {
                const float *y = T.Y_dev + ((int64_t)rep * T.n_dev + d0 + v) * 2 * F + F;
                for (int c = k * D; c < (k + 1) * D; ++c) t = fmaf(ad[c], y[c] - cp[c], t);
                qdd[v * K + k] = t;
            }
        }
    }
    __syncthreads();
}

// Lane layout of the tile kernels: a wavefront takes four entries of an op
// at a time, 16 lanes per entry, f/16 consecutive channels per lane; a
// head spans 16/K lanes (K <= 16).  Each wavefront walks ops u0 + wv,
// u0 + wv + 4, ... and reads the rows of its next op while it works on the
// current one.  Slots of op-device entries are keyed by their position in
// the op<-device bucket.
// max over aligned groups of 16 lanes (DPP inside a 16-lane row)
__device__ __forceinline__ float row_max16(float v) {
    auto dpp = [](float x, auto ctrl) {
        return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), decltype(ctrl)::value, 0xf, 0xf, true));
    };
    v = fmaxf(v, dpp(v, std::integral_constant<int, 0xB1>{}));    // quad_perm [1,0,3,2]
    v = fmaxf(v, dpp(v, std::integral_constant<int, 0x4E>{}));    // quad_perm [2,3,0,1]
    v = fmaxf(v, dpp(v, std::integral_constant<int, 0x141>{}));   // row_half_mirror
    v = fmaxf(v, dpp(v, std::integral_constant<int, 0x140>{}));   // row_mirror
    return v;
}

// Scores on the matrix cores (topologies of at most 16 devices): wavefront w
// takes the tile's ops 16 w .. 16 w + 15; per head and placement bit b the
// logit gradients dO_u . m_b(v) (op <- device) and dO_v . m_b(u) (device <-
// op) are fp32 MFMA 16x16x4 products over the head's channels, lane l
// supplying op 16 w + l % 16 (A) and device l % 16 (B) at channel slice
// l / 16.  Result register r of lane l is op 16 w + 4 (l / 16) + r, device
// l % 16: an op row's entries lie in the 16 lanes of one lane group, so its
// softmax (op <- device) reduces over those lanes; the device<-op records
// fold per lane over its four ops, then over lane groups and wavefronts in order.
template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_od_scores(BwdLayer P, OdTile T) {
    constexpr int D = F / K, FS = od_stride<F>(), CPL = F / 64;
    constexpr int HG = K >= 2 ? 2 : 1;   // heads per pass over the channels (register budget)
    static_assert(K <= 16 && D >= 16, "the op-device tile path needs heads of at least 16 channels");
    extern __shared__ float sh[];
    __shared__ int32_t rps[kOpTile + 1];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float zop[kOpTile][K];   // Z of the tile's op rows (op <- device)
    __shared__ float red[4][F];
    __shared__ float cst[4][F];         // U (bit column), a, a~, c' of the relation
    const int32_t t = blockIdx.x, rep = blockIdx.y;
    const int32_t u0 = T.tiles[3 * t], n = T.tiles[3 * t + 1], g = T.tiles[3 * t + 2];
    const int32_t d0 = T.dev_off[g], nd = T.dev_off[g + 1] - d0;
    const int MD = T.max_dev;
    float *md = sh, *dod = md + 2 * MD * FS, *pd = dod + MD * FS, *qdd = pd + 2 * MD * K;
    float *dst = qdd + MD * K;           // [4][16][K][3] device<-op records per wavefront
    uint8_t *ent = reinterpret_cast<uint8_t *>(dst + 4 * 16 * K * 3);
    for (int i = threadIdx.x; i < 4 * 16 * K; i += blockDim.x) {
        dst[3 * i] = -INFINITY;
        dst[3 * i + 1] = dst[3 * i + 2] = 0.f;
    }
    for (int i = threadIdx.x; i < F; i += blockDim.x) {
        cst[0][i] = P.U[((int64_t)F + i) * 2 + 0];
        cst[1][i] = P.att_src[F + i];
        cst[2][i] = P.att_dst[F + i];
        cst[3][i] = P.cp[F + i];
    }
    od_stage<F, K, ELU, true>(P, T, rep, u0, n, d0, nd, md, dod, pd, qdd, rps, ent);
    // link and placement-bit masks of the tile's ops over the topology's devices
    if (threadIdx.x < kOpTile) {
        uint64_t pr = 0ull, bt = 0ull;
        if ((int)threadIdx.x < n)
            for (int32_t e = rps[threadIdx.x]; e < rps[threadIdx.x + 1]; ++e) {
                const int eb = ent[e - rps[0]];
                pr |= 1ull << (eb & 0x7f);
                if (eb >> 7) bt |= 1ull << (eb & 0x7f);
            }
        pres[threadIdx.x] = pr;
        bits[threadIdx.x] = bt;
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, lr = lane & 15, lg = lane >> 4;
    const int ua = 16 * wv + lr;                       // op this lane supplies (A rows)
    const bool aok = ua < n;
    const int64_t rowa = (int64_t)rep * T.n_op + u0 + (aok ? ua : 0);
    const float *ya = T.Y_op + rowa * 2 * F + F, *da = T.dO_op + rowa * F;
    const bool vok = lr < nd;                          // device of this lane's column (B, results)
    const int64_t sbase = (int64_t)rep * T.n_slots;
    for (int hg = 0; hg < K; hg += HG) {
        f4 d1[HG][2], d2[HG][2];
        float qv[HG], p0v[HG], p1v[HG];                // this lane's parts of the op's head terms
#pragma unroll
        for (int j = 0; j < HG; ++j) {
            d1[j][0] = d1[j][1] = d2[j][0] = d2[j][1] = f4{0.f, 0.f, 0.f, 0.f};
            qv[j] = p0v[j] = p1v[j] = 0.f;
        }
        // one pass over the channels of heads hg .. hg + HG - 1
#pragma unroll
        for (int kk = 0; kk < HG * D / 4; ++kk) {
            const int j = kk / (D / 4);
            const int c = hg * D + 4 * kk + lg;
            const float y = aok ? ya[c] : 0.f;
            const float gd = aok ? T.gamma * da[c] : 0.f;
            const float m0 = aok ? msg_act<ELU>(y) : 0.f;
            const float m1 = aok ? msg_act<ELU>(y + cst[0][c]) : 0.f;
            const float as = cst[1][c];
            qv[j] = fmaf(cst[2][c], y - cst[3][c], qv[j]);
            p0v[j] = fmaf(as, m0, p0v[j]);
            p1v[j] = fmaf(as, m1, p1v[j]);
            const float bm0 = vok ? md[(lr * 2 + 0) * FS + c] : 0.f, bm1 = vok ? md[(lr * 2 + 1) * FS + c] : 0.f;
            const float bd = vok ? dod[lr * FS + c] : 0.f;
            d1[j][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(gd, bm0, d1[j][0], 0, 0, 0);
            d1[j][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(gd, bm1, d1[j][1], 0, 0, 0);
            d2[j][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(m0, bd, d2[j][0], 0, 0, 0);
            d2[j][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(m1, bd, d2[j][1], 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < HG; ++j) {
        const int h = hg + j;
        // the op's head terms: sums over the four channel slices (lane groups)
        float qp = qv[j], p0p = p0v[j], p1p = p1v[j];
        qp += __shfl_xor(qp, 16, 64); qp += __shfl_xor(qp, 32, 64);
        p0p += __shfl_xor(p0p, 16, 64); p0p += __shfl_xor(p0p, 32, 64);
        p1p += __shfl_xor(p1p, 16, 64); p1p += __shfl_xor(p1p, 32, 64);
        float dmx = -INFINITY, dden = 0.f, dnum = 0.f;   // device<-op record of this lane's device
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int u = 16 * wv + 4 * lg + r;          // the op of result register r
            const int src = 4 * lg + r;                  // a lane supplying op u
            const float qu = __shfl(qp, src, 64), p0u = __shfl(p0p, src, 64), p1u = __shfl(p1p, src, 64);
            const uint64_t pr = u < n ? pres[u] : 0ull, bt = u < n ? bits[u] : 0ull;
            const bool ok = vok && ((pr >> lr) & 1ull);
            const int x = (int)((bt >> lr) & 1ull);
            const float dd1 = x ? d1[j][1][r] : d1[j][0][r], dd2 = x ? d2[j][1][r] : d2[j][0][r];
            const float s1 = ok ? leaky(pd[(lr * 2 + x) * K + h] + qu, P.slope) : -INFINITY;   // op <- device
            const float s2 = leaky((x ? p1u : p0u) + (vok ? qdd[lr * K + h] : 0.f), P.slope);   // device <- op
            const int32_t e = ok ? rps[u] + __popcll(pr & ((1ull << lr) - 1ull)) : 0;
            if (ok) {
                const int64_t idx = (sbase + e) * K + h;
                T.SA2[idx] = s2;
                T.SD2[idx] = dd2;
                softmax_fold(s2, dd2, dmx, dden, dnum);
            }
            // softmax of op u's row over its devices (the lane group)
            const float mx = row_max16(s1);
            const float ex = ok ? __expf(s1 - mx) : 0.f;
            const float den = row_sum<16>(ex), num = row_sum<16>(ex * dd1);
            const float inv = den > 0.f ? 1.f / den : 0.f, cc = num * inv;
            const float al = ex * inv;
            const float dz = ok ? al * (dd1 - cc) * (s1 > 0.f ? 1.f : P.slope) : 0.f;
            if (ok) {
                const int64_t idx = (sbase + e) * K + h;
                T.SA1[idx] = al;
                T.SD1[idx] = dz;
            }
            const float zs = row_sum<16>(dz);
            if (lr == 0 && u < n) {
                zop[u][h] = zs;
                T.Zop[(((int64_t)rep * T.n_op + u0 + u) * 2 + 1) * K + h] = zs;
            }
        }
        // this wavefront's record of device lr: its lane groups in order
        for (int o = 16; o < 64; o <<= 1) {
            const float m2 = __shfl_xor(dmx, o, 64), d2v = __shfl_xor(dden, o, 64), n2 = __shfl_xor(dnum, o, 64);
            softmax_merge(m2, d2v, n2, dmx, dden, dnum);
        }
        if (lg == 0) {
            float *st = dst + ((wv * 16 + lr) * K + h) * 3;
            st[0] = dmx; st[1] = dden; st[2] = dnum;
        }
        }
    }
    // d adst of the op rows: sum over the wavefront's ops of Z_u (Y_u - c'), lanes over channels
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    {
        float acc[CPL];
        for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
        const int cc0 = lane * CPL, hh = cc0 / D;
        for (int uu = 0; uu < 16; ++uu) {
            const int u = 16 * wv + uu;
            if (u >= n) break;
            float y[CPL];
            load_ch<CPL, false>(T.Y_op, ((int64_t)rep * T.n_op + u0 + u) * 2 * F + F + cc0, y);
            const float z = zop[u][hh];
            for (int c = 0; c < CPL; ++c) acc[c] = fmaf(z, y[c] - cst[3][cc0 + c], acc[c]);
        }
        for (int c = 0; c < CPL; ++c) red[wv][cc0 + c] = acc[c];
    }
    __syncthreads();
    // the tile's sums of d adst (op rows) and device<-op records, wavefronts in order
    const int64_t tb = (int64_t)rep * T.n_tiles + t;
    for (int c = threadIdx.x; c < F; c += 256) T.part_a1[tb * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
    for (int i = threadIdx.x; i < nd * K; i += blockDim.x) {
        float mx = dst[3 * i], den = dst[3 * i + 1], num = dst[3 * i + 2];
        for (int w = 1; w < 4; ++w) {
            const float *o = dst + ((size_t)w * 16 * K + i) * 3;
            softmax_merge(o[0], o[1], o[2], mx, den, num);
        }
        float *r = T.drec + ((tb * MD) * K + i) * 3;
        r[0] = mx; r[1] = den; r[2] = num;
    }
}

// device<-op softmax statistics: per (candidate, device, head) the tiles'
// records of the device's topology merged in tile order
__global__ void bwd_od_dev_stats(BwdLayer P, OdTile T, const int32_t *dev_topo, int K) {
    const int64_t total = (int64_t)P.R * T.n_dev * K;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / K;
        const int h = (int)(i % K);
        const int32_t rep = (int32_t)(row / T.n_dev), d = (int32_t)(row % T.n_dev);
        const int32_t g = dev_topo[d], v = d - T.dev_off[g];
        float mx = -INFINITY, den = 0.f, num = 0.f;
        for (int32_t t = T.tile_off[g]; t < T.tile_off[g + 1]; ++t) {
            const float *r = T.drec + ((((int64_t)rep * T.n_tiles + t) * T.max_dev + v) * K + h) * 3;
            softmax_merge(r[0], r[1], r[2], mx, den, num);
        }
        const float inv = den > 0.f ? 1.f / den : 0.f;
        T.dstat[i * 3 + 0] = mx;
        T.dstat[i * 3 + 1] = inv;
        T.dstat[i * 3 + 2] = num * inv;
    }
}

// derivative of sigma from its output: ReLU [m > 0]; ELU 1 or e^z = m + 1
template <bool ELU>
__device__ __forceinline__ float dact(float m) { return m > 0.f ? 1.f : (ELU ? m + 1.f : 0.f); }

// The (alpha, dz) scalars of an op's entries come in chunks of 64 / K
// entries, lane i holding entry i / K, head i % K of the chunk (one
// coalesced read per array); the first chunk of the next op is read ahead.
// Op side per entry (the wavefront's op is the source of device<-op links):
// dY of the op row and the op's parts of d a, dU0 and dc'.  Device side
// (op<-device links, the devices are the sources): each entry's alpha goes
// into a dense per-head matrix aw[h][device][op] (the placement bit in the
// sign bit; alpha >= 0) and its dz into per-bit sums; after the tile's ops,
// sum_u alpha_uv gamma dO_u[c] for each placement bit is a (devices x 64 ops)
// by (64 ops x channels) product on the matrix cores, and sigma' of the
// device's message, the a Z terms and the device parts of d a, dU0 and dc'
// are applied once per (device, channel).
constexpr int kAS = 68;   // row stride of aw: the 16 x 4 operand reads fall on distinct banks

template <int F, int K, bool ELU>
__global__ void __launch_bounds__(256) bwd_od_messages(BwdLayer P, OdTile T) {
    constexpr int CPE = F / 16, FS = od_stride<F>(), EPC = 64 / K, D = F / K;
    constexpr bool AHEAD = CPE <= 8;   // read the next op's rows ahead (register budget)
    static_assert(K <= 16 && D >= 16, "the op-device tile path needs heads of at least 16 channels");
    extern __shared__ float sh[];
    __shared__ float red[4][F];
    __shared__ float dpart[3][F];      // device side of d a, dU0, dc' per channel
    __shared__ int32_t rps[kOpTile + 1];
    const int32_t t = blockIdx.x, rep = blockIdx.y;
    const int32_t u0 = T.tiles[3 * t], n = T.tiles[3 * t + 1], g = T.tiles[3 * t + 2];
    const int32_t d0 = T.dev_off[g], nd = T.dev_off[g + 1] - d0;
    const int MD = T.max_dev, MDP = (MD + 15) & ~15;
    float *md = sh, *dod = md + 2 * MD * FS;
    float *aw = dod + MD * FS;          // [K][MDP][kAS] alpha of op<-device entries, sign bit = placement bit
    float *dsm = aw + K * MDP * kAS;    // [MD][K][3] device<-op statistics (max, 1/sum, c)
    float *zacc = dsm + 3 * MD * K;     // [4][MD][K] sums of dz over device<-op entries per wavefront
    float *z1 = zacc + 4 * MD * K;      // [4][2][K][MDP] sums of dz over op<-device entries per wavefront and bit
    uint8_t *ent = reinterpret_cast<uint8_t *>(z1 + 8 * K * MDP);
    for (int i = threadIdx.x; i < K * MDP * kAS; i += blockDim.x) aw[i] = 0.f;
    for (int i = threadIdx.x; i < 4 * MD * K; i += blockDim.x) zacc[i] = 0.f;
    for (int i = threadIdx.x; i < 8 * K * MDP; i += blockDim.x) z1[i] = 0.f;
    {
        const float *src = T.dstat + ((int64_t)rep * T.n_dev + d0) * K * 3;
        for (int i = threadIdx.x; i < nd * K * 3; i += blockDim.x) dsm[i] = src[i];
    }
    od_stage<F, K, ELU, false>(P, T, rep, u0, n, d0, nd, md, dod, nullptr, nullptr, rps, ent);
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int grp = lane >> 4, jl = lane & 15;
    const int c0 = jl * CPE, h = c0 / D;
    float a[CPE], ad[CPE], u0c[CPE], ga[CPE], gu0[CPE], gcp[CPE];
    for (int c = 0; c < CPE; ++c) {
        a[c] = P.att_src[F + c0 + c];
        ad[c] = P.att_dst[F + c0 + c];
        u0c[c] = P.U[((int64_t)F + c0 + c) * 2 + 0];
        ga[c] = gu0[c] = gcp[c] = 0.f;
    }
    float *zw = zacc + (size_t)wv * MD * K, *z1w = z1 + (size_t)wv * 2 * K * MDP;
    const int64_t sbase = (int64_t)rep * T.n_slots * K;
    const int32_t ebase = rps[0];
    auto scalars = [&](int32_t cs, int32_t end, float (&m)[4]) {
        if (cs + lane / K < end) {
            const int64_t i = sbase + (int64_t)cs * K + lane;
            m[0] = T.SA1[i]; m[1] = T.SD1[i]; m[2] = T.SA2[i]; m[3] = T.SD2[i];
        } else {
            m[0] = m[1] = m[2] = m[3] = 0.f;
        }
    };
    // per entry and head (the lanes of a chunk hold distinct (device, head)
    // pairs): op<-device alpha into aw and dz into the per-bit sums;
    // device<-op (s, dalpha) -> (alpha, dz) with the device's merged
    // statistics, and the dz sums per (device, head)
    auto to_alpha = [&](int32_t cs, int32_t end, int32_t ui, float (&m)[4]) {
        const int32_t e = cs + lane / K;
        if (e < end) {
            const int eb = ent[e - ebase];
            const int v = eb & 0x7f, x = eb >> 7, k = lane % K;
            aw[(k * MDP + v) * kAS + ui] = __int_as_float(__float_as_int(m[0]) | (x << 31));
            z1w[(x * K + k) * MDP + v] += m[1];
            const float *st = dsm + (v * K + k) * 3;
            const float sv = m[2];
            const float al = __expf(sv - st[0]) * st[1];
            const float dz = al * (m[3] - st[2]) * (sv > 0.f ? 1.f : P.slope);
            m[2] = al;
            m[3] = dz;
            zw[v * K + k] += dz;
        }
    };
    float nyo[CPE], ndO[CPE], nm[4];
    auto fetch = [&](int32_t ui) {
        if constexpr (AHEAD) {
            const int64_t row = (int64_t)rep * T.n_op + u0 + ui;
            load_ch<CPE, false>(T.Y_op, row * 2 * F + F + c0, nyo);
        }
        scalars(rps[ui], rps[ui + 1], nm);
    };
    if (wv < n) fetch(wv);
    for (int32_t ui = wv; ui < n; ui += 4) {
        const int64_t row = (int64_t)rep * T.n_op + u0 + ui;
        float yo[CPE], m0[CPE], m1[CPE], dys[CPE], sc[4];
        if constexpr (AHEAD) {
            for (int c = 0; c < CPE; ++c) yo[c] = nyo[c];
        } else {
            load_ch<CPE, false>(T.Y_op, row * 2 * F + F + c0, yo);
        }
        for (int i = 0; i < 4; ++i) sc[i] = nm[i];
        const int32_t beg = rps[ui], end = rps[ui + 1];
        if (ui + 4 < n) fetch(ui + 4);
        if (beg < end) to_alpha(beg, end, ui, sc);
        for (int c = 0; c < CPE; ++c) {
            m0[c] = msg_act<ELU>(yo[c]);
            m1[c] = msg_act<ELU>(yo[c] + u0c[c]);
            dys[c] = 0.f;
        }
        for (int32_t cs = beg; cs < end; cs += EPC) {
            if (cs != beg) {   // rows longer than one chunk
                scalars(cs, end, sc);
                to_alpha(cs, end, ui, sc);
            }
            const int32_t ce = min(end, cs + EPC);
            for (int32_t e0 = cs; e0 < ce; e0 += 4) {
                const int32_t e = e0 + grp;
                const int src = (e - cs) * K + h;   // < 64: e - cs < EPC
                const float al2 = __shfl(sc[2], src, 64), dz2 = __shfl(sc[3], src, 64);   // device v <- op u
                if (e < ce) {
                    const int eb = ent[e - ebase];
                    const int v = eb & 0x7f, x = eb >> 7;
                    const float *dv = dod + v * FS + c0;
                    for (int c = 0; c < CPE; ++c) {
                        const float mo = x ? m1[c] : m0[c];
                        const float dpo = dact<ELU>(mo) * fmaf(al2, dv[c], dz2 * a[c]);
                        dys[c] += dpo;
                        ga[c] = fmaf(dz2, mo, ga[c]);
                        if (x) gu0[c] += dpo;
                        gcp[c] += dpo;
                    }
                }
            }
        }
        // the four entry groups' sums, in order
        for (int c = 0; c < CPE; ++c) {
            dys[c] += __shfl_xor(dys[c], 16, 64);
            dys[c] += __shfl_xor(dys[c], 32, 64);
        }
        if (grp == 0) {
            const float zo = T.Zop[(row * 2 + 1) * K + h];
            float *o = T.dY_op + row * 2 * F + F + c0;
            for (int c = 0; c < CPE; ++c) o[c] = fmaf(zo, ad[c], dys[c]);
        }
    }
    for (int c = 0; c < CPE; ++c) {
        ga[c] += __shfl_xor(ga[c], 16, 64);  ga[c] += __shfl_xor(ga[c], 32, 64);
        gu0[c] += __shfl_xor(gu0[c], 16, 64); gu0[c] += __shfl_xor(gu0[c], 32, 64);
        gcp[c] += __shfl_xor(gcp[c], 16, 64); gcp[c] += __shfl_xor(gcp[c], 32, 64);
    }
    __syncthreads();
    // device side on the matrix cores: wavefront w takes the 16-channel column
    // blocks w, w + 4, ...; lane l supplies aw[h][rb + l % 16][ks + l / 16]
    // (A, by bit) and gamma dO[ks + l / 16][column] (B); result register r of
    // lane l is device rb + 4 (l / 16) + r, channel cb 16 + l % 16
    float *pdst = T.PD + (((int64_t)rep * T.n_tiles + t) * MD) * F;
    for (int cb = wv; cb < F / 16; cb += 4) {
        const int cl = cb * 16 + (lane & 15), hc = cl / D;
        const float ac = P.att_src[F + cl];
        float sga = 0.f, sgu = 0.f, sgc = 0.f;
        float bo[kOpTile / 4];   // this lane's B operands, one per k step
#pragma unroll
        for (int ks = 0; ks < kOpTile / 4; ++ks) {
            const int uk = 4 * ks + (lane >> 4);
            bo[ks] = uk < n ? T.gamma * T.dO_op[((int64_t)rep * T.n_op + u0 + uk) * F + cl] : 0.f;
        }
        for (int rb = 0; rb < MDP; rb += 16) {
            f4 t0 = f4{0.f, 0.f, 0.f, 0.f}, t1 = f4{0.f, 0.f, 0.f, 0.f};
            const float *arow = aw + (hc * MDP + rb + (lane & 15)) * kAS + (lane >> 4);
#pragma unroll
            for (int ks = 0; ks < kOpTile / 4; ++ks) {
                const float w = arow[4 * ks];
                const bool bit = __float_as_int(w) < 0;
                const float wa = fabsf(w);
                t0 = __builtin_amdgcn_mfma_f32_16x16x4f32(bit ? 0.f : wa, bo[ks], t0, 0, 0, 0);
                t1 = __builtin_amdgcn_mfma_f32_16x16x4f32(bit ? wa : 0.f, bo[ks], t1, 0, 0, 0);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int v = rb + 4 * (lane >> 4) + r;
                if (v < nd) {
                    float zb0 = 0.f, zb1 = 0.f;   // the wavefronts' dz sums in order
                    for (int w = 0; w < 4; ++w) {
                        zb0 += z1[((w * 2 + 0) * K + hc) * MDP + v];
                        zb1 += z1[((w * 2 + 1) * K + hc) * MDP + v];
                    }
                    const float mb0 = md[(v * 2 + 0) * FS + cl], mb1 = md[(v * 2 + 1) * FS + cl];
                    const float p0 = dact<ELU>(mb0) * fmaf(ac, zb0, t0[r]);
                    const float p1 = dact<ELU>(mb1) * fmaf(ac, zb1, t1[r]);
                    pdst[(int64_t)v * F + cl] = p0 + p1;
                    sga = fmaf(mb0, zb0, fmaf(mb1, zb1, sga));
                    sgu += p1;
                    sgc += p0 + p1;
                }
            }
        }
        // the column's sums over the four lane groups (device rows)
        sga += __shfl_xor(sga, 16, 64); sga += __shfl_xor(sga, 32, 64);
        sgu += __shfl_xor(sgu, 16, 64); sgu += __shfl_xor(sgu, 32, 64);
        sgc += __shfl_xor(sgc, 16, 64); sgc += __shfl_xor(sgc, 32, 64);
        if (lane < 16) { dpart[0][cl] = sga; dpart[1][cl] = sgu; dpart[2][cl] = sgc; }
    }
    // this tile's dz sums of device<-op entries: the four wavefronts' sums in order
    float *zdst = T.zrec + (((int64_t)rep * T.n_tiles + t) * MD) * K;
    for (int i = threadIdx.x; i < nd * K; i += blockDim.x) {
        const size_t st = (size_t)MD * K;
        zdst[i] = (zacc[i] + zacc[st + i]) + (zacc[2 * st + i] + zacc[3 * st + i]);
    }
    // parameter partials of the block: the wavefronts' op-side sums in order, then the device side
    const int64_t nb = (int64_t)gridDim.x * gridDim.y, b = (int64_t)rep * gridDim.x + t;
    auto flush = [&](int qq, int slot, const float (&qv)[CPE]) {
        if (grp == 0)
            for (int c = 0; c < CPE; ++c) red[wv][c0 + c] = qv[c];
        __syncthreads();
        for (int c = threadIdx.x; c < F; c += 256)
            T.part[((int64_t)slot * nb + b) * F + c] = ((red[0][c] + red[1][c]) + (red[2][c] + red[3][c])) + dpart[qq][c];
        __syncthreads();
    };
    flush(0, 0, ga);
    flush(1, 1, gu0);
    flush(2, 3, gcp);
    for (int c = threadIdx.x; c < F; c += 256) T.part[((int64_t)2 * nb + b) * F + c] = 0.f;   // no dU1 for od
}

// device od rows, one wavefront per row: Z = the tiles' dz sums in tile
// order, dY = the tiles' partials in tile order + Z adst, and per-block sums
// of d adst = Z (Y - c') over the block's four rows
template <int F, int K>
__global__ void __launch_bounds__(256) bwd_od_devices(BwdLayer P, OdTile T, const int32_t *dev_topo) {
    constexpr int CPL = F / 64, D = F / K;
    __shared__ float red[4][F];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t row = (int64_t)blockIdx.x * 4 + wv;
    const int c0 = lane * CPL;
    float acc[CPL];
    for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
    if (row < (int64_t)P.R * T.n_dev) {
        const int32_t rep = (int32_t)(row / T.n_dev), d = (int32_t)(row % T.n_dev);
        const int32_t g = dev_topo[d], v = d - T.dev_off[g];
        const int32_t t0 = T.tile_off[g], t1 = T.tile_off[g + 1];
        const int64_t tb = (int64_t)rep * T.n_tiles;
        float z = 0.f;
        if (lane < K)
            for (int32_t t = t0; t < t1; ++t) z += T.zrec[((tb + t) * T.max_dev + v) * K + lane];
        if (lane < K) T.Zdev[(row * 2 + 1) * K + lane] = z;
        const float zh = __shfl(z, c0 / D, 64);
        for (int c = 0; c < CPL; ++c) {
            float s = 0.f;
            for (int32_t t = t0; t < t1; ++t) s += T.PD[((tb + t) * T.max_dev + v) * F + c0 + c];
            T.dY_dev[row * 2 * F + c0 + c] = fmaf(zh, P.att_dst[F + c0 + c], s);
            acc[c] = zh * (T.Y_dev[row * 2 * F + F + c0 + c] - P.cp[F + c0 + c]);
        }
    }
    for (int c = 0; c < CPL; ++c) red[wv][c0 + c] = acc[c];
    __syncthreads();
    for (int c = threadIdx.x; c < F; c += 256)
        T.part_a2[(int64_t)blockIdx.x * F + c] = (red[0][c] + red[1][c]) + (red[2][c] + red[3][c]);
}

// slot keys of the op-device links: pos_of[eid] = position in the op<-device
// bucket, then m21[q] = pos_of[eid of position q of the device<-op bucket]
__global__ void od_positions(const int32_t *eid, int64_t n, int32_t *pos_of) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x)
        pos_of[eid[p]] = (int32_t)p;
}
__global__ void od_map(const int32_t *eid, int64_t n, const int32_t *pos_of, int32_t *m21) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n; q += (int64_t)gridDim.x * blockDim.x)
        m21[q] = pos_of[eid[q]];
}

// topology of every device row
__global__ void dev_topology(const int32_t *dev_off, int32_t G, int64_t n_dev, int32_t *out) {
    for (int64_t d = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; d < n_dev; d += (int64_t)gridDim.x * blockDim.x) {
        int32_t g = 0;
        while (g + 1 < G && dev_off[g + 1] <= d) ++g;
        out[d] = g;
    }
}

// Parameter sums of one layer from the per-block partials:
//   att_dst grad (scores' softmax passes), att_src grad, dU, dc' (message passes)
struct ParamReduce {
    const float *pa[4];     // bwd_softmax partials of buckets 0..3: [nb][F]
    const float *pm[4];     // bwd_messages partials of the four source passes: [4][nb][F]
    int32_t nb_a[4], nb_m[4];
    int F;
    float *g_att_src, *g_att_dst;   // [3][F] of the layer
    float *dU, *dcp;                // [3][F][2], [3][F] of the layer
};

// block (relation r, quantity, 16 columns); thread (column, row group of
// 16) sums its rows of every partial array of the relation, then the 16
// groups are added in order
__global__ void __launch_bounds__(256) bwd_params(ParamReduce R) {
    __shared__ float red[16][17];
    const int rel_of[4] = {0, 1, 1, 2};
    const int F = R.F;
    const int cb = (F + 15) / 16;
    const int rq = blockIdx.x / cb, c = (blockIdx.x % cb) * 16 + (threadIdx.x & 15), grp = threadIdx.x >> 4;
    const int r = rq / 5, qty = rq % 5;
    float s = 0.f;
    if (c < F) {
        for (int p = 0; p < 4; ++p) {
            if (rel_of[p] != r) continue;
            const float *base;
            int32_t nb;
            if (qty == 0) { base = R.pa[p]; nb = R.nb_a[p]; }
            else { base = R.pm[p] + (int64_t)(qty - 1) * R.nb_m[p] * F; nb = R.nb_m[p]; }
#pragma unroll 8
            for (int32_t b = grp; b < nb; b += 16) s += base[(int64_t)b * F + c];
        }
    }
    red[grp][threadIdx.x & 15] = s;
    __syncthreads();
    if (grp != 0 || c >= F) return;
    float t = 0.f;
    for (int g = 0; g < 16; ++g) t += red[g][threadIdx.x & 15];
    if (qty == 0) R.g_att_dst[r * F + c] = t;
    else if (qty == 1) R.g_att_src[r * F + c] = t;
    else if (qty == 2) R.dU[((int64_t)r * F + c) * 2 + 0] = t;
    else if (qty == 3) R.dU[((int64_t)r * F + c) * 2 + 1] = t;
    else R.dcp[r * F + c] = t;
}

// ReLU mask of the encoders: g = H0 > 0 ? g : 0
__global__ void relu_mask(float *g, const float *h, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        if (!(h[i] > 0.f)) g[i] = 0.f;
}

// Folded edge encoders, per layer l and relation r (d_r = 1, 1, 2):
//   grad layer_b = dc';  grad W^e[o][k] = sum_t dU[o][t] A_r[k][t] + dc'[o] c_r[k]
struct FoldBwd {
    const float *layer_w;
    const float *A[3], *c[3];
    const float *dU, *dcp;   // [L][3][F][2], [L][3][F]
    float *g_layer_w, *g_layer_b;
    float *g_A[3], *g_c[3];
    int F, L;
};

__global__ void fold_bwd_we(FoldBwd a) {
    const int F = a.F;
    const int64_t total = (int64_t)a.L * 3 * F * F;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t lr = i / ((int64_t)F * F);
        const int o = (int)((i / F) % F), k = (int)(i % F);
        const int r = (int)(lr % 3), d = r == 2 ? 2 : 1;
        const float *du = a.dU + (lr * F + o) * 2;
        float s = a.dcp[lr * F + o] * a.c[r][k];
        for (int t = 0; t < d; ++t) s = fmaf(du[t], a.A[r][(int64_t)k * d + t], s);
        a.g_layer_w[(lr * F + o) * 2 * F + F + k] = s;
        if (k == 0) a.g_layer_b[lr * F + o] = a.dcp[lr * F + o];
    }
}

// grad A_r[k][t] = sum_l sum_o W^e_{l,r}[o][k] dU_{l,r}[o][t];  grad c_r[k] likewise with dc'.
// Block (relation, 64 k); thread (k, o group of 4) sums its o over the
// layers, then the groups are added in order.
__global__ void __launch_bounds__(256) fold_bwd_enc(FoldBwd a) {
    // block (relation r, 16 encoder outputs k); thread (k, output group of 16):
    // sums its outputs o of every layer, then the 16 groups are added in order
    __shared__ float red[3][16][17];
    const int F = a.F;
    const int kb = (F + 15) / 16;
    const int r = blockIdx.x / kb, kk = threadIdx.x & 15, grp = threadIdx.x >> 4;
    const int k = (blockIdx.x % kb) * 16 + kk;
    const int d = r == 2 ? 2 : 1;
    float s0 = 0.f, s1 = 0.f, sc = 0.f;
    if (k < F) {
        for (int l = 0; l < a.L; ++l) {
            const int64_t lr = (int64_t)l * 3 + r;
#pragma unroll 4
            for (int o = grp; o < F; o += 16) {
                const float we = a.layer_w[(lr * F + o) * 2 * F + F + k];
                s0 = fmaf(we, a.dU[(lr * F + o) * 2 + 0], s0);
                s1 = fmaf(we, a.dU[(lr * F + o) * 2 + 1], s1);
                sc = fmaf(we, a.dcp[lr * F + o], sc);
            }
        }
    }
    red[0][grp][kk] = s0;
    red[1][grp][kk] = s1;
    red[2][grp][kk] = sc;
    __syncthreads();
    if (grp != 0 || k >= F) return;
    float t0 = 0.f, t1 = 0.f, tc = 0.f;
    for (int gq = 0; gq < 16; ++gq) { t0 += red[0][gq][kk]; t1 += red[1][gq][kk]; tc += red[2][gq][kk]; }
    a.g_A[r][(int64_t)k * d + 0] = t0;
    if (d == 2) a.g_A[r][(int64_t)k * d + 1] = t1;
    a.g_c[r][k] = tc;
}

// ------------------------------------------------------------------ decoder
// With t = E_dev W1_dev^T, the slice part u[rg][h][a] = sum_{j in mask_a}
// t_j[h] + W1_opt[h][option_a] + b1[h] (shared by every query of the
// candidate graph rg) and v_q = W1_op E_op[i_q], the hidden pre-activation
// is u[rg][h][a] + v_q[h].  Backward, per candidate graph, with
// dpre_qah = dscore_qa w2_h [pre > 0] and D_ah = sum_{q of rg} dpre_qah:
//   dT_j = sum_{a: j in mask_a} D_a   (then dE_dev = dT W1_dev, dW1_dev = dT^T E_dev)
//   dv_q = sum_a dpre_qa             (then dE_op = dv W1_op, dW1_op = dv^T E_op[i_q])
//   dW1_opt[o] = sum_{a: option o} D_a, db1 = sum_a D_a, dw2 = sum dscore ReLU(pre),
//   db2 = sum dscore.
struct DecTrain {
    int32_t R, G, S, Q, F, H, RG;
    int64_t n_op, n_dev;
    const int32_t *op_off, *dev_off;
    const uint64_t *mask;
    const uint8_t *option;
    const float *w2, *b2;
    const int32_t *q_rep, *q_graph, *q_op;
    const float *target;
    const float *u;          // [RG][H][S]
    const float *v;          // [Q][H]
    int32_t *qrow;           // [Q] E_op row of each query (-1: invalid)
    int32_t *qcnt, *qoff, *qlist;   // queries per candidate graph: [RG], [RG+1], [Q]
    float inv_q;
    float *ds;               // [Q][S] d loss / d score
    float *loss_q, *db2q;    // [Q]
    float *dvq;              // [Q][H]
    float *dT;               // [R n_dev][H]
    float *dopt_part;        // [RG][4][H]
    float *dw2_part;         // [RG][H]
};

__device__ __forceinline__ bool dec_query(const DecTrain &A, int32_t q, int32_t *r, int32_t *g, int32_t *op) {
    *r = A.q_rep[q]; *g = A.q_graph[q]; *op = A.q_op[q];
    if (*r < 0 || *r >= A.R || *g < 0 || *g >= A.G) return false;
    return *op >= 0 && *op < A.op_off[*g + 1] - A.op_off[*g];
}

__global__ void dec_rows(DecTrain A) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < A.Q; q += (int64_t)gridDim.x * blockDim.x) {
        int32_t r, g, op;
        A.qrow[q] = dec_query(A, (int32_t)q, &r, &g, &op) ? (int32_t)((int64_t)r * A.n_op + A.op_off[g] + op) : -1;
    }
}

// query lists per candidate graph, in query order: counts, offsets, lists
__global__ void dec_count(DecTrain A, int fill) {
    for (int64_t rg = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; rg < A.RG; rg += (int64_t)gridDim.x * blockDim.x) {
        int32_t n = 0;
        int32_t *out = fill ? A.qlist + A.qoff[rg] : nullptr;
        for (int32_t q = 0; q < A.Q; ++q) {
            if (A.qrow[q] < 0 || (int64_t)A.q_rep[q] * A.G + A.q_graph[q] != rg) continue;
            if (fill) out[n] = q;
            ++n;
        }
        if (!fill) A.qcnt[rg] = n;
    }
}

__global__ void __launch_bounds__(256) dec_scan(DecTrain A) {
    __shared__ int32_t part[256];
    const int t = threadIdx.x;
    const int64_t per = (A.RG + 255) / 256, b = t * per, e = b + per < A.RG ? b + per : A.RG;
    int32_t s = 0;
    for (int64_t i = b; i < e; ++i) s += A.qcnt[i];
    part[t] = s;
    __syncthreads();
    if (t == 0) {
        int32_t run = 0;
        for (int i = 0; i < 256; ++i) { const int32_t x = part[i]; part[i] = run; run += x; }
        A.qoff[A.RG] = run;
    }
    __syncthreads();
    int32_t run = part[t];
    for (int64_t i = b; i < e; ++i) { A.qoff[i] = run; run += A.qcnt[i]; }
}

// one block per query: scores of every slice, softmax, loss term and dscore
__global__ void __launch_bounds__(256) dec_scores(DecTrain A) {
    extern __shared__ float sh[];   // sc[S] | v[H] | w2[H]
    __shared__ float red[256], red2[256];
    const int tid = threadIdx.x;
    const int32_t q = blockIdx.x;
    int32_t r, g, op;
    if (!dec_query(A, q, &r, &g, &op)) {
        for (int32_t a = tid; a < A.S; a += 256) A.ds[(int64_t)q * A.S + a] = 0.f;
        if (tid == 0) { A.loss_q[q] = 0.f; A.db2q[q] = 0.f; }
        return;
    }
    const int H = A.H;
    float *sc = sh, *vq = sh + A.S, *w2s = vq + H;
    for (int h = tid; h < H; h += 256) { vq[h] = A.v[(int64_t)q * H + h]; w2s[h] = A.w2[h]; }
    __syncthreads();
    const float *urg = A.u + ((int64_t)r * A.G + g) * H * A.S;
    float mx = -INFINITY;
    for (int32_t a = tid; a < A.S; a += 256) {
        float s = 0.f;
        int h = 0;
        for (; h + 8 <= H; h += 8) {
            float uu[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) uu[k] = urg[(int64_t)(h + k) * A.S + a];
#pragma unroll
            for (int k = 0; k < 8; ++k) s = fmaf(w2s[h + k], fmaxf(uu[k] + vq[h + k], 0.f), s);
        }
        for (; h < H; ++h) s = fmaf(w2s[h], fmaxf(urg[(int64_t)h * A.S + a] + vq[h], 0.f), s);
        s += A.b2[0];
        sc[a] = s;
        mx = fmaxf(mx, s);
    }
    red[tid] = mx;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red[tid] = fmaxf(red[tid], red[tid + o]);
        __syncthreads();
    }
    const float M0 = red[0];
    __syncthreads();
    const float *tg = A.target + (int64_t)q * A.S;
    float z = 0.f, tt = 0.f;
    for (int32_t a = tid; a < A.S; a += 256) {
        z += __expf(sc[a] - M0);
        tt += tg[a];
    }
    red[tid] = z;
    red2[tid] = tt;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) { red[tid] += red[tid + o]; red2[tid] += red2[tid + o]; }
        __syncthreads();
    }
    const float Z = red[0], T = red2[0];
    const float logZ = __logf(Z);
    __syncthreads();
    float lt = 0.f, db = 0.f;
    for (int32_t a = tid; a < A.S; a += 256) {
        const float ls = sc[a] - M0 - logZ;          // log prior
        const float d = A.inv_q * (__expf(ls) * T - tg[a]);
        lt = fmaf(tg[a], ls, lt);
        A.ds[(int64_t)q * A.S + a] = d;
        db += d;
    }
    red[tid] = lt;
    red2[tid] = db;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) { red[tid] += red[tid + o]; red2[tid] += red2[tid + o]; }
        __syncthreads();
    }
    if (tid == 0) { A.loss_q[q] = -A.inv_q * red[0]; A.db2q[q] = red2[0]; }
}

constexpr int kDecHC = 32;    // hidden units per gradient block
constexpr int kDecSC = 256;   // slices per LDS chunk

// One block per (candidate graph, 32 hidden units); thread (hh, grp) walks
// the graph's queries in order over its slices a = grp (mod 8) of each
// 256-slice chunk, keeping D[a][h] in registers; then D goes through LDS
// into dT[j][h] (thread owns j = grp (mod 8)) and the option sums.
__global__ void __launch_bounds__(256) dec_grad(DecTrain A) {
    __shared__ float buf[kDecSC * (kDecHC + 1)];      // u chunk [32][257], then D chunk [256][33]
    __shared__ uint64_t mk[kDecSC];
    __shared__ uint8_t op[kDecSC];
    __shared__ float red[8][kDecHC];
    const int tid = threadIdx.x, hh = tid & (kDecHC - 1), grp = tid >> 5;
    const int nch = (A.H + kDecHC - 1) / kDecHC;
    const int64_t rg = blockIdx.x / nch;
    const int h0 = (int)(blockIdx.x % nch) * kDecHC, h = h0 + hh, H = A.H;
    const bool live = h < H;
    const int32_t r = (int32_t)(rg / A.G), g = (int32_t)(rg % A.G);
    const int32_t d0 = A.dev_off[g], nd = A.dev_off[g + 1] - d0;
    const uint64_t keep = nd >= 64 ? ~0ull : ((1ull << nd) - 1ull);
    const int32_t nq = A.qcnt[rg];
    const int32_t *list = A.qlist + A.qoff[rg];
    const float w2h = live ? A.w2[h] : 0.f;
    const float *urg = A.u + rg * H * A.S;
    float dT[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float dopt = 0.f, dw2 = 0.f;
    for (int32_t a0 = 0; a0 < A.S; a0 += kDecSC) {
        __syncthreads();
        for (int i = tid; i < kDecHC * kDecSC; i += 256) {
            const int c = i / kDecSC, a = i % kDecSC;
            buf[c * (kDecSC + 1) + a] = (h0 + c < H && a0 + a < A.S) ? urg[(int64_t)(h0 + c) * A.S + a0 + a] : 0.f;
        }
        for (int a = tid; a < kDecSC; a += 256) {
            mk[a] = a0 + a < A.S ? A.mask[a0 + a] & keep : 0ull;
            op[a] = a0 + a < A.S ? (uint8_t)min((int)A.option[a0 + a], 3) : 4;
        }
        __syncthreads();
        float D[kDecSC / 8];
#pragma unroll
        for (int i = 0; i < kDecSC / 8; ++i) D[i] = 0.f;
        for (int32_t k = 0; k < nq; ++k) {
            const int32_t q = list[k];
            const float vqh = live ? A.v[(int64_t)q * H + h] : 0.f;
            const float *dsq = A.ds + (int64_t)q * A.S + a0;
            float dv = 0.f;
#pragma unroll
            for (int i = 0; i < kDecSC / 8; ++i) {
                const int a = grp + 8 * i;
                if (a0 + a < A.S) {
                    const float pre = buf[hh * (kDecSC + 1) + a] + vqh;
                    const float d = dsq[a];
                    const float dp = pre > 0.f ? d * w2h : 0.f;
                    D[i] += dp;
                    dv += dp;
                    dw2 = fmaf(d, fmaxf(pre, 0.f), dw2);
                }
            }
            red[grp][hh] = dv;
            __syncthreads();
            if (grp == 0 && live) {
                float sum = 0.f;
                for (int gg = 0; gg < 8; ++gg) sum += red[gg][hh];
                float *o = A.dvq + (int64_t)q * H + h;
                *o = a0 == 0 ? sum : *o + sum;
            }
            __syncthreads();
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kDecSC / 8; ++i) buf[(grp + 8 * i) * (kDecHC + 1) + hh] = D[i];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int j = grp + 8 * i;
            if (j >= nd) continue;
            float sum = 0.f;
            for (int a = 0; a < kDecSC; ++a)
                if ((mk[a] >> j) & 1ull) sum += buf[a * (kDecHC + 1) + hh];
            dT[i] += sum;
        }
        if (grp < 4) {
            float sum = 0.f;
            for (int a = 0; a < kDecSC; ++a)
                if (op[a] == grp) sum += buf[a * (kDecHC + 1) + hh];
            dopt += sum;
        }
    }
    if (live) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int j = grp + 8 * i;
            if (j < nd) A.dT[((int64_t)r * A.n_dev + d0 + j) * H + h] = dT[i];
        }
        if (grp < 4) A.dopt_part[(rg * 4 + grp) * H + h] = dopt;
    }
    __syncthreads();
    red[grp][hh] = dw2;
    __syncthreads();
    if (grp == 0 && live) {
        float sum = 0.f;
        for (int gg = 0; gg < 8; ++gg) sum += red[gg][hh];
        A.dw2_part[rg * H + h] = sum;
    }
}

// rows of E_op read by the queries (zero rows for invalid ones)
__global__ void dec_gather_rows(const float *E_op, const int32_t *qrow, int32_t Q, int F, float *Eq) {
    const int64_t total = (int64_t)Q * F;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t row = qrow[i / F];
        Eq[i] = row >= 0 ? E_op[(int64_t)row * F + i % F] : 0.f;
    }
}

// dE_op rows of the queries: the first query of each row sums, in query
// order, the dE rows of every query reading that row
__global__ void dec_grad_op(const int32_t *qrow, int32_t Q, int F, const float *dEq, float *g_op) {
    const int32_t q = blockIdx.x;
    const int32_t row = qrow[q];
    if (row < 0) return;
    for (int32_t p = 0; p < q; ++p)
        if (qrow[p] == row) return;
    for (int c = threadIdx.x; c < F; c += blockDim.x) {
        float s = 0.f;
        for (int32_t p = q; p < Q; ++p)
            if (qrow[p] == row) s += dEq[(int64_t)p * F + c];
        g_op[(int64_t)row * F + c] = s;
    }
}

// decoder parameter sums over candidate graphs (W1 option columns, b1, w2)
__global__ void dec_params(DecTrain A, float *g_w1, float *g_b1, float *g_w2) {
    const int din = 2 * A.F + 4, H = A.H;
    for (int h = blockIdx.x * blockDim.x + threadIdx.x; h < H; h += gridDim.x * blockDim.x) {
        float o4[4] = {0.f, 0.f, 0.f, 0.f}, w2 = 0.f;
        for (int32_t rg = 0; rg < A.RG; ++rg) {
            for (int o = 0; o < 4; ++o) o4[o] += A.dopt_part[((int64_t)rg * 4 + o) * H + h];
            w2 += A.dw2_part[(int64_t)rg * H + h];
        }
        float b1 = 0.f;
        for (int o = 0; o < 4; ++o) {
            g_w1[(int64_t)h * din + 2 * A.F + o] = o4[o];
            b1 += o4[o];
        }
        g_b1[h] = b1;
        g_w2[h] = w2;
    }
}

// loss and output-bias gradient: fixed-order block sums over the queries
__global__ void __launch_bounds__(256) dec_totals(const float *loss_q, const float *db2q, int32_t Q, float *loss,
                                                  float *g_b2) {
    __shared__ float r1[256], r2[256];
    const int t = threadIdx.x;
    float a = 0.f, b = 0.f;
    for (int32_t q = t; q < Q; q += 256) { a += loss_q[q]; b += db2q[q]; }
    r1[t] = a;
    r2[t] = b;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (t < o) { r1[t] += r1[t + o]; r2[t] += r2[t + o]; }
        __syncthreads();
    }
    if (t == 0) { loss[0] = r1[0]; g_b2[0] = r2[0]; }
}

__global__ void fill_zero(float *p, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = 0.f;
}

// ------------------------------------------------------------------ update
struct SgdList {
    float *w[18];
    const float *g[18];
    int64_t n[18];
    int count;
    float lr;
};

__global__ void sgd_update(SgdList L) {
    const int a = blockIdx.y;
    if (a >= L.count) return;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < L.n[a]; i += (int64_t)gridDim.x * blockDim.x)
        L.w[a][i] = fmaf(-L.lr, L.g[a][i], L.w[a][i]);
}

// ------------------------------------------------------------------ layout
struct TrainLayout {
    void *fwd;
    size_t fwd_bytes;
    float *H_op[16], *H_dev[16], *Y_op[16], *Y_dev[16];
    float *E_op, *E_dev, *G_op, *G_dev, *dY_op, *dY_dev;
    float *SA[4], *SD[4];
    float *Zop, *Zdev;
    float *PB;
    float *part_a[4], *part_m[4];
    int32_t nb_a[4], nb_m[4];
    float *dU, *dcp;
    float *P0, *P1;
    float *PD, *part_od;     // op-device tile path: device partials, parameter partials
    float *part_a1, *drec, *dstat, *zrec, *part_a2;   // ... and its softmax records and d adst sums
    int32_t nb_dev4;         // blocks of bwd_od_devices (four device rows each)
    int32_t *dev_topo;
    int32_t *pos_of, *m21;   // op-device links: edge id -> op<-device position; device<-op position -> same
    // decoder
    float *t, *u, *v, *ds, *loss_q, *db2q, *dvq, *dT, *dopt_part, *dw2_part, *Eq, *dEq;
    int32_t *qrow, *qcnt, *qoff, *qlist;
};

int32_t chunks_of(int32_t max_degree, int per) { return std::max<int32_t>(1, (max_degree + per - 1) / per); }

int64_t n_slots(const tag_graph *g, int b) {
    return b == 0 ? 2 * g->e_oo : (b == 3 ? 2 * g->e_dd : g->e_od);
}

// the op-device tile path needs the topology's device rows in LDS
// dynamic LDS bytes of the tile kernels: float rows, then one byte per tile entry
size_t od_scores_lds(int F, int K, int max_dev) {
    return sizeof(float) * ((size_t)3 * max_dev * (F + 4) + (size_t)3 * max_dev * K + (size_t)4 * 16 * K * 3) +
           (size_t)kOpTile * max_dev;
}
size_t od_messages_lds(int F, int K, int max_dev) {
    const size_t mdp = (size_t)(max_dev + 15) / 16 * 16;
    return sizeof(float) * ((size_t)3 * max_dev * (F + 4) + (size_t)K * mdp * kAS + (size_t)7 * max_dev * K +
                            (size_t)8 * K * mdp) + (size_t)kOpTile * max_dev;
}

// (heads of at least 16 channels and at least f/16: one head inside a 16-lane
// entry group and inside a 16-channel column block of the device-side products)
bool od_tiles_fit(const tag_graph *g, int F, int K) {
    // dynamic rows + the static reduction rows and row pointers of the messages kernel
    // static LDS of the two kernels: row pointers, reduction and constant rows, op masks and Z
    const size_t rp = sizeof(int32_t) * (kOpTile + 1);
    const size_t stat_m = sizeof(float) * 7 * F + rp;
    const size_t stat_s = sizeof(float) * (8 * F + (size_t)kOpTile * K) + 2 * sizeof(uint64_t) * kOpTile + rp;
    return g->n_tiles > 0 && g->max_dev <= 16 && K <= 16 && F / K >= 16 &&
           od_messages_lds(F, K, g->max_dev) + stat_m <= 64 * 1024 &&
           od_scores_lds(F, K, g->max_dev) + stat_s <= 64 * 1024;
}

int32_t persist_blocks(int64_t items) {
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(kPersist, (items + 3) / 4));
}

// size of the split-K partials of every weight gradient
int64_t split_floats(const tag_graph *g, const tag_model_dims *d, int32_t R, int32_t Q) {
    const int64_t F = d->f;
    auto one = [&](int64_t M, int64_t N, int64_t K) {
        int64_t s;
        split_k_per(K, ((M + GM - 1) / GM) * ((N + GN - 1) / GN), &s);
        return s * M * N;
    };
    int64_t m = one(2 * F, F, (int64_t)R * g->n_op);
    m = std::max(m, one(2 * F, F, (int64_t)R * g->n_dev));
    m = std::max(m, one(F, d->f_op + 1, (int64_t)R * g->n_op));
    m = std::max(m, one(F, d->f_dev + 1, (int64_t)R * g->n_dev));
    const int64_t H = std::max(d->dec_hidden, 1);
    m = std::max(m, one(H, F, (int64_t)R * g->n_dev));
    m = std::max(m, one(H, F, std::max(Q, 1)));
    return m;
}

size_t carve_train(const tag_graph *g, const tag_model_dims *d, int32_t R, int32_t S, int32_t Q, void *base,
                   TrainLayout *L) {
    FwdLayout fl;
    const size_t fb = carve_fwd(g, d, R, nullptr, &fl);
    Carver c(base);
    L->fwd = c.take<char>(fb);
    L->fwd_bytes = fb;
    const int64_t F = d->f, K = d->heads, ro = (int64_t)R * g->n_op, rd = (int64_t)R * g->n_dev;
    for (int l = 0; l < 16; ++l) L->H_op[l] = L->H_dev[l] = L->Y_op[l] = L->Y_dev[l] = nullptr;
    for (int l = 0; l < d->layers; ++l) {
        L->H_op[l] = c.take<float>(ro * F);
        L->H_dev[l] = c.take<float>(rd * F);
        L->Y_op[l] = c.take<float>(ro * 2 * F);
        L->Y_dev[l] = c.take<float>(rd * 2 * F);
    }
    L->E_op = c.take<float>(ro * F);
    L->E_dev = c.take<float>(rd * F);
    L->G_op = c.take<float>(ro * F);
    L->G_dev = c.take<float>(rd * F);
    L->dY_op = c.take<float>(ro * 2 * F);
    L->dY_dev = c.take<float>(rd * 2 * F);
    for (int b = 0; b < 4; ++b) {
        L->SA[b] = c.take<float>((size_t)R * n_slots(g, b) * K);
        L->SD[b] = c.take<float>((size_t)R * n_slots(g, b) * K);
    }
    L->Zop = c.take<float>(ro * 2 * K);
    L->Zdev = c.take<float>(rd * 2 * K);
    int64_t pb = 0;
    for (int b = 0; b < 4; ++b) {
        const int64_t rows = (b < 2) ? ro : rd;
        const int32_t ch = chunks_of(g->max_degree[b], kChunkB);
        if (ch > 1) pb = std::max(pb, rows * ch * F);
    }
    L->PB = c.take<float>(std::max<int64_t>(pb, 1));
    for (int b = 0; b < 4; ++b) {
        const int64_t rows = (b < 2) ? ro : rd;
        L->nb_a[b] = persist_blocks(rows);
        L->nb_m[b] = persist_blocks(rows * chunks_of(g->max_degree[b], kChunkB));
        L->part_a[b] = c.take<float>((size_t)L->nb_a[b] * F);
        L->part_m[b] = c.take<float>((size_t)4 * L->nb_m[b] * F);
    }
    if (od_tiles_fit(g, (int)F, (int)K)) {
        const int64_t nb = (int64_t)R * g->n_tiles;
        L->PD = c.take<float>((size_t)nb * g->max_dev * F);
        L->part_od = c.take<float>((size_t)4 * nb * F);
        L->part_a1 = c.take<float>((size_t)nb * F);
        L->drec = c.take<float>((size_t)nb * g->max_dev * K * 3);
        L->dstat = c.take<float>((size_t)std::max<int64_t>(rd, 1) * K * 3);
        L->zrec = c.take<float>((size_t)nb * g->max_dev * K);
        L->nb_dev4 = (int32_t)std::max<int64_t>(1, (rd + 3) / 4);
        L->part_a2 = c.take<float>((size_t)L->nb_dev4 * F);
        L->dev_topo = c.take<int32_t>((size_t)std::max<int64_t>(g->n_dev, 1));
    } else {
        L->PD = L->part_od = nullptr;
        L->part_a1 = L->drec = L->dstat = L->zrec = L->part_a2 = nullptr;
        L->nb_dev4 = 0;
        L->dev_topo = nullptr;
    }
    L->pos_of = c.take<int32_t>((size_t)std::max<int64_t>(g->e_od, 1));
    L->m21 = c.take<int32_t>((size_t)std::max<int64_t>(g->e_od, 1));
    L->dU = c.take<float>((size_t)d->layers * 3 * F * 2);
    L->dcp = c.take<float>((size_t)d->layers * 3 * F);
    const int64_t sp = split_floats(g, d, R, Q);
    L->P0 = c.take<float>(sp);
    L->P1 = c.take<float>(sp);
    const int64_t H = std::max(d->dec_hidden, 1), Qm = std::max(Q, 1), RG = (int64_t)R * g->G;
    L->t = c.take<float>(rd * H);
    L->u = c.take<float>(RG * H * S);
    L->v = c.take<float>(Qm * H);
    L->ds = c.take<float>(Qm * S);
    L->loss_q = c.take<float>(Qm);
    L->db2q = c.take<float>(Qm);
    L->dvq = c.take<float>(Qm * H);
    L->dT = c.take<float>(rd * H);
    L->dopt_part = c.take<float>(RG * 4 * H);
    L->dw2_part = c.take<float>(RG * H);
    L->Eq = c.take<float>(Qm * F);
    L->dEq = c.take<float>(Qm * F);
    L->qrow = c.take<int32_t>(Qm);
    L->qcnt = c.take<int32_t>(RG);
    L->qoff = c.take<int32_t>(RG + 1);
    L->qlist = c.take<int32_t>(Qm);
    return c.used;
}

// LDS floats of the op-device tile kernels

template <int F, int K, bool ELU>
void launch_layer_bwd(const BwdLayer &P, BwdBucket (&B)[4], BwdSrc (&S)[4], const ParamReduce &pr, const OdTile *od,
                      const int32_t *dev_topo, hipStream_t st) {
    const dim3 tgrid(od ? (unsigned)od->n_tiles : 1u, (unsigned)P.R);
    if (od) {
        prof_begin(TAG_STAGE_BWD_SCORES, st);
        if constexpr (K <= 16 && F / K >= 16)
            bwd_od_scores<F, K, ELU><<<tgrid, 256, od_scores_lds(F, K, od->max_dev), st>>>(P, *od);
        prof_end(TAG_STAGE_BWD_SCORES, st);
    }
    for (int b = 0; b < 4; ++b) {
        const int64_t waves = (int64_t)P.R * B[b].n_dst * B[b].chunks;
        if (waves <= 0 || (od && (b == 1 || b == 2))) continue;
        prof_begin(TAG_STAGE_BWD_SCORES, st);
        bool short_rows = false;
        if constexpr (K <= 16) short_rows = B[b].chunks == 1;
        if (short_rows) {
            if constexpr (K <= 16)
                bwd_scores_short<F, K, ELU><<<(unsigned)((waves + 15) / 16), 256, 0, st>>>(P, B[b]);
        } else {
            bwd_scores<F, K, ELU><<<(unsigned)((waves + 3) / 4), 256, 0, st>>>(P, B[b]);
        }
        prof_end(TAG_STAGE_BWD_SCORES, st);
    }
    for (int b = 0; b < 4; ++b) {
        if (od && (b == 1 || b == 2)) continue;   // inside the tile kernels
        prof_begin(TAG_STAGE_BWD_SOFTMAX, st);
        float *pa = const_cast<float *>(pr.pa[b]);
        bool long_rows = false, short_rows = false;
        if constexpr (K <= 16) {
            long_rows = B[b].chunks * kChunkA >= kLongRow;
            short_rows = B[b].chunks == 1;
        }
        if (long_rows) {
            if constexpr (K <= 16) bwd_softmax<F, K, true><<<pr.nb_a[b], 256, 0, st>>>(P, B[b], pa);
        } else if (short_rows) {
            if constexpr (K <= 16) bwd_softmax_short<F, K><<<pr.nb_a[b], 256, 0, st>>>(P, B[b], pa);
        } else {
            bwd_softmax<F, K, false><<<pr.nb_a[b], 256, 0, st>>>(P, B[b], pa);
        }
        prof_end(TAG_STAGE_BWD_SOFTMAX, st);
    }
    if (od) {
        prof_begin(TAG_STAGE_BWD_SOFTMAX, st);
        bwd_od_dev_stats<<<grid_for((int64_t)P.R * od->n_dev * K), 256, 0, st>>>(P, *od, dev_topo, K);
        prof_end(TAG_STAGE_BWD_SOFTMAX, st);
        prof_begin(TAG_STAGE_BWD_MESSAGES, st);
        if constexpr (K <= 16 && F / K >= 16)
            bwd_od_messages<F, K, ELU><<<tgrid, 256, od_messages_lds(F, K, od->max_dev), st>>>(P, *od);
        prof_end(TAG_STAGE_BWD_MESSAGES, st);
        bwd_od_devices<F, K><<<(unsigned)(((int64_t)P.R * od->n_dev + 3) / 4), 256, 0, st>>>(P, *od, dev_topo);
    }
    for (int s = 0; s < 4; ++s) {
        if (od && (s == 1 || s == 2)) continue;
        prof_begin(TAG_STAGE_BWD_MESSAGES, st);
        bool short_rows = false;
        if constexpr (K <= 16) short_rows = S[s].chunks == 1;
        if (short_rows) {
            if constexpr (K <= 16)
                bwd_messages_short<F, K, ELU><<<pr.nb_m[s], 256, 0, st>>>(P, S[s], const_cast<float *>(pr.pm[s]));
        } else {
            bwd_messages<F, K, ELU><<<pr.nb_m[s], 256, 0, st>>>(P, S[s], const_cast<float *>(pr.pm[s]));
        }
        prof_end(TAG_STAGE_BWD_MESSAGES, st);
        if (S[s].chunks > 1) bwd_combine<<<grid_for((int64_t)P.R * S[s].n_self * F), 256, 0, st>>>(P, S[s], K);
    }
    bwd_params<<<15 * ((F + 15) / 16), 256, 0, st>>>(pr);
}

template <int F, bool ELU>
bool dispatch_layer_bwd_f(int K, const BwdLayer &P, BwdBucket (&B)[4], BwdSrc (&S)[4], const ParamReduce &pr,
                          const OdTile *od, const int32_t *dt, hipStream_t st) {
    switch (K) {
        case 1: launch_layer_bwd<F, 1, ELU>(P, B, S, pr, od, dt, st); return true;
        case 2: launch_layer_bwd<F, 2, ELU>(P, B, S, pr, od, dt, st); return true;
        case 4: launch_layer_bwd<F, 4, ELU>(P, B, S, pr, od, dt, st); return true;
        case 8: launch_layer_bwd<F, 8, ELU>(P, B, S, pr, od, dt, st); return true;
        case 16: launch_layer_bwd<F, 16, ELU>(P, B, S, pr, od, dt, st); return true;
        case 32: launch_layer_bwd<F, 32, ELU>(P, B, S, pr, od, dt, st); return true;
        case 64: launch_layer_bwd<F, 64, ELU>(P, B, S, pr, od, dt, st); return true;
    }
    return false;
}

bool dispatch_layer_bwd(int F, int K, bool elu, const BwdLayer &P, BwdBucket (&B)[4], BwdSrc (&S)[4],
                        const ParamReduce &pr, const OdTile *od, const int32_t *dt, hipStream_t st) {
    if (F == 64) return elu ? dispatch_layer_bwd_f<64, true>(K, P, B, S, pr, od, dt, st)
                            : dispatch_layer_bwd_f<64, false>(K, P, B, S, pr, od, dt, st);
    if (F == 128) return elu ? dispatch_layer_bwd_f<128, true>(K, P, B, S, pr, od, dt, st)
                             : dispatch_layer_bwd_f<128, false>(K, P, B, S, pr, od, dt, st);
    if (F == 256) return elu ? dispatch_layer_bwd_f<256, true>(K, P, B, S, pr, od, dt, st)
                             : dispatch_layer_bwd_f<256, false>(K, P, B, S, pr, od, dt, st);
    return false;
}


tag_status check_train(const tag_graph *g, const tag_model_dims *dims, int32_t R, int32_t S, int32_t Q) {
    if (!g || !dims) TAG_FAIL(TAG_EINVAL, "graph and dims must be non-NULL");
    tag_status st = check_dims(dims);
    if (st != TAG_OK) return st;
    if (dims->dtype != TAG_F32) TAG_FAIL(TAG_ESHAPE, "training supports the fp32 variant only");
    if (is_variant(dims)) TAG_FAIL(TAG_ESHAPE, "training supports the default readings (3 relations, affine "
                                               "edge encoders, concatenated heads) only");
    if (dims->dec_hidden < 1) TAG_FAIL(TAG_ESHAPE, "training needs the MLP decoder (dec_hidden >= 1)");
    if (R < 1 || S < 1 || Q < 1) TAG_FAIL(TAG_EINVAL, "need n_replicas, n_slices and n_query >= 1");
    if (S > 4096) TAG_FAIL(TAG_ESHAPE, "training supports at most 4096 slices");
    return TAG_OK;
}

}  // namespace
}  // namespace tag

using namespace tag;

extern "C" tag_status tag_train_workspace(const tag_graph *g, const tag_model_dims *dims, int32_t n_replicas,
                                          int32_t n_slices, int32_t n_query, size_t *bytes) {
    clear_error();
    if (!bytes) TAG_FAIL(TAG_EINVAL, "bytes must be non-NULL");
    tag_status st = check_train(g, dims, n_replicas, n_slices, n_query);
    if (st != TAG_OK) return st;
    TrainLayout L;
    *bytes = carve_train(g, dims, n_replicas, n_slices, n_query, nullptr, &L);
    return TAG_OK;
}

extern "C" tag_status tag_train_step(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                     const tag_features *x, const tag_slices *slices, const tag_train_batch *batch,
                                     const tag_grads *gr, float lr, float *loss, void *workspace, size_t ws_bytes,
                                     void *hip_stream) {
    clear_error();
    if (!w || !x || !slices || !batch || !gr || !loss || !workspace)
        TAG_FAIL(TAG_EINVAL, "weights, features, slices, batch, grads, loss and workspace must be non-NULL");
    const int32_t R = x->n_replicas, S = slices->n_slices, Q = batch->n_query;
    tag_status st = check_train(g, dims, R, S, Q);
    if (st != TAG_OK) return st;
    if (!slices->mask || !slices->option) TAG_FAIL(TAG_EINVAL, "NULL slice table");
    if (!batch->query_rep || !batch->query_graph || !batch->query_op || !batch->target)
        TAG_FAIL(TAG_EINVAL, "query arrays and targets must be non-NULL");
    if (!w->dec_w1 || !w->dec_b1 || !w->dec_w2 || !w->dec_b2) TAG_FAIL(TAG_EINVAL, "decoder weights must be non-NULL");
    const float *gp[] = {gr->enc_op_w, gr->enc_op_b, gr->enc_dev_w, gr->enc_dev_b, gr->enc_edge_w[0],
                         gr->enc_edge_w[1], gr->enc_edge_w[2], gr->enc_edge_b[0], gr->enc_edge_b[1],
                         gr->enc_edge_b[2], gr->layer_w, gr->layer_b, gr->att_src, gr->att_dst,
                         gr->dec_w1, gr->dec_b1, gr->dec_w2, gr->dec_b2};
    for (const float *p : gp)
        if (!p) TAG_FAIL(TAG_EINVAL, "gradient arrays must be non-NULL");
    if (!(lr >= 0.f) || lr == INFINITY) TAG_FAIL(TAG_EINVAL, "lr must be finite and >= 0");
    TrainLayout L;
    if (carve_train(g, dims, R, S, Q, nullptr, &L) > ws_bytes)
        TAG_FAIL(TAG_ENOSPACE, "training workspace too small (see tag_train_workspace)");
    carve_train(g, dims, R, S, Q, workspace, &L);
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    const int F = dims->f, K = dims->heads, NL = dims->layers, H = dims->dec_hidden;
    const int64_t ro = (int64_t)R * g->n_op, rd = (int64_t)R * g->n_dev;

    // forward with saved activations
    FwdSave save{};
    for (int l = 0; l < NL; ++l) {
        save.H_op[l] = L.H_op[l]; save.H_dev[l] = L.H_dev[l];
        save.Y_op[l] = L.Y_op[l]; save.Y_dev[l] = L.Y_dev[l];
    }
    st = forward_run(g, dims, w, x, L.fwd, L.fwd_bytes, L.E_op, L.E_dev, stream, &save);
    if (st != TAG_OK) return st;
    FwdLayout FL;
    carve_fwd(g, dims, R, L.fwd, &FL);   // folded edge terms U, c' of every layer

    // decoder: loss, its parameter gradients and dE
    DecTrain D{};
    D.R = R; D.G = g->G; D.S = S; D.Q = Q; D.F = F; D.H = H; D.RG = R * g->G;
    D.n_op = g->n_op; D.n_dev = g->n_dev;
    D.op_off = g->op_off_d; D.dev_off = g->dev_off_d;
    D.mask = slices->mask; D.option = slices->option;
    D.w2 = w->dec_w2; D.b2 = w->dec_b2;
    D.q_rep = batch->query_rep; D.q_graph = batch->query_graph; D.q_op = batch->query_op;
    D.target = batch->target;
    D.u = L.u; D.v = L.v; D.qrow = L.qrow;
    D.qcnt = L.qcnt; D.qoff = L.qoff; D.qlist = L.qlist;
    D.inv_q = 1.f / (float)Q;
    D.ds = L.ds; D.loss_q = L.loss_q; D.db2q = L.db2q; D.dvq = L.dvq; D.dT = L.dT;
    D.dopt_part = L.dopt_part; D.dw2_part = L.dw2_part;
    const int din = 2 * F + 4;
    const int64_t RG = (int64_t)R * g->G;
    prof_begin(TAG_STAGE_BWD_DECODER, stream);
    launch_small_gemm(SmallGemm{L.E_dev, F, rd, nullptr, F, w->dec_w1, din, H, nullptr, 0, L.t, H, 0}, stream);
    dec_rows<<<grid_for(Q), 256, 0, stream>>>(D);
    launch_small_gemm(SmallGemm{L.E_op, F, Q, L.qrow, F, w->dec_w1 + F, din, H, nullptr, 0, L.v, H, 0}, stream);
    launch_slice_terms(R, g->G, S, F, H, g->n_dev, g->dev_off_d, L.t, w->dec_w1, w->dec_b1, slices->mask,
                       slices->option, L.u, stream);
    dec_count<<<grid_for(RG), 256, 0, stream>>>(D, 0);
    dec_scan<<<1, 256, 0, stream>>>(D);
    dec_count<<<grid_for(RG), 256, 0, stream>>>(D, 1);
    dec_scores<<<Q, 256, sizeof(float) * (S + 2 * H), stream>>>(D);
    fill_zero<<<grid_for((int64_t)Q * H), 256, 0, stream>>>(L.dvq, (int64_t)Q * H);
    dec_grad<<<(unsigned)(RG * ((H + kDecHC - 1) / kDecHC)), 256, 0, stream>>>(D);
    dec_totals<<<1, 256, 0, stream>>>(L.loss_q, L.db2q, Q, loss, gr->dec_b2);
    dec_params<<<grid_for(H), 256, 0, stream>>>(D, gr->dec_w1, gr->dec_b1, gr->dec_w2);
    // device side: dE_dev = dT W1_dev, dW1_dev = dT^T E_dev
    launch_gemm(Gemm{L.dT, H, w->dec_w1, din, rd, F, H, -1, L.G_dev, F, 0, H, 0}, true, false, 1, stream);
    weight_grad(L.dT, H, L.E_dev, F, H, F, false, rd, L.P0, gr->dec_w1, din, nullptr, 0, stream);
    // op side: dE_op rows of the queries = dv W1_op, dW1_op = dv^T E_op[query rows]
    dec_gather_rows<<<grid_for((int64_t)Q * F), 256, 0, stream>>>(L.E_op, L.qrow, Q, F, L.Eq);
    weight_grad(L.dvq, H, L.Eq, F, H, F, false, Q, L.P1, gr->dec_w1 + F, din, nullptr, 0, stream);
    launch_gemm(Gemm{L.dvq, H, w->dec_w1 + F, din, Q, F, H, -1, L.dEq, F, 0, H, 0}, true, false, 1, stream);
    fill_zero<<<grid_for(ro * F), 256, 0, stream>>>(L.G_op, ro * F);
    dec_grad_op<<<Q, 256, 0, stream>>>(L.qrow, Q, F, L.dEq, L.G_op);
    prof_end(TAG_STAGE_BWD_DECODER, stream);

    // layers, last to first
    if (L.dev_topo) dev_topology<<<grid_for(g->n_dev), 256, 0, stream>>>(g->dev_off_d, g->G, g->n_dev, L.dev_topo);
    if (g->e_od > 0) {
        od_positions<<<grid_for(g->e_od), 256, 0, stream>>>(g->eid[1], g->e_od, L.pos_of);
        od_map<<<grid_for(g->e_od), 256, 0, stream>>>(g->eid[2], g->e_od, L.pos_of, L.m21);
    }
    BwdLayer P{};
    P.R = R; P.F = F;
    P.x_oo = x->x_oo; P.s_oo = x->stride_oo;
    P.x_dd = x->x_dd; P.s_dd = x->stride_dd;
    P.x_od = x->x_od; P.s_od = x->stride_od;
    P.slope = dims->leaky_slope;
    const float gs = dims->gamma_same, gc = dims->gamma_cross;
    for (int l = NL - 1; l >= 0; --l) {
        P.att_src = w->att_src + (size_t)l * 3 * F;
        P.att_dst = w->att_dst + (size_t)l * 3 * F;
        P.U = FL.U + (size_t)l * 3 * F * 2;
        P.cp = FL.cp + (size_t)l * 3 * F;
        const float *Yo = L.Y_op[l], *Yd = L.Y_dev[l];
        // forward buckets: Y_op = [oo | od], Y_dev = [dd | od]
        BwdBucket B[4];
        B[0] = BwdBucket{g->rowptr[0], g->col[0], g->eid[0], g->n_op, g->n_op, Yo, 0, Yo, 0, L.G_op, gs, 0, 0, 1,
                         L.SA[0], L.SD[0], n_slots(g, 0), chunks_of(g->max_degree[0], kChunkA), L.Zop, 0};
        B[1] = BwdBucket{g->rowptr[1], g->col[1], g->eid[1], g->n_op, g->n_dev, Yo, F, Yd, F, L.G_op, gc, 1, 1, 0,
                         L.SA[1], L.SD[1], n_slots(g, 1), chunks_of(g->max_degree[1], kChunkA), L.Zop, 1};
        B[2] = BwdBucket{g->rowptr[2], g->col[2], g->eid[2], g->n_dev, g->n_op, Yd, F, Yo, F, L.G_dev, gc, 1, 1, 0,
                         L.SA[2], L.SD[2], n_slots(g, 2), chunks_of(g->max_degree[2], kChunkA), L.Zdev, 1};
        B[3] = BwdBucket{g->rowptr[3], g->col[3], g->eid[3], g->n_dev, g->n_dev, Yd, 0, Yd, 0, L.G_dev, gs, 2, 2, 1,
                         L.SA[3], L.SD[3], n_slots(g, 3), chunks_of(g->max_degree[3], kChunkA), L.Zdev, 0};
        // source passes; dY_op = [oo | od], dY_dev = [od | dd]
        BwdSrc Sx[4];
        Sx[0] = BwdSrc{g->rowptr[0], g->col[0], g->eid[0], g->n_op, g->n_op, Yo, 0, L.G_op, gs, L.SA[0], L.SD[0],
                       n_slots(g, 0), 1, 0, 0, L.Zop, 0, L.dY_op, 0, L.PB, chunks_of(g->max_degree[0], kChunkB)};
        Sx[1] = BwdSrc{g->rowptr[1], g->col[1], g->eid[1], g->n_op, g->n_dev, Yo, F, L.G_dev, gc, L.SA[2], L.SD[2],
                       n_slots(g, 2), 0, 1, 1, L.Zop, 1, L.dY_op, F, L.PB, chunks_of(g->max_degree[1], kChunkB)};
        Sx[2] = BwdSrc{g->rowptr[2], g->col[2], g->eid[2], g->n_dev, g->n_op, Yd, F, L.G_op, gc, L.SA[1], L.SD[1],
                       n_slots(g, 1), 0, 1, 1, L.Zdev, 1, L.dY_dev, 0, L.PB, chunks_of(g->max_degree[2], kChunkB)};
        Sx[3] = BwdSrc{g->rowptr[3], g->col[3], g->eid[3], g->n_dev, g->n_dev, Yd, 0, L.G_dev, gs, L.SA[3], L.SD[3],
                       n_slots(g, 3), 1, 2, 2, L.Zdev, 0, L.dY_dev, F, L.PB, chunks_of(g->max_degree[3], kChunkB)};
        // op-device slots: positions of the op<-device bucket
        B[1].spos = 1; B[2].smap = L.m21;
        Sx[1].spos = 1; Sx[2].smap = L.m21;
        ParamReduce pr{};
        for (int b = 0; b < 4; ++b) {
            pr.pa[b] = L.part_a[b]; pr.nb_a[b] = L.nb_a[b];
            pr.pm[b] = L.part_m[b]; pr.nb_m[b] = L.nb_m[b];
        }
        pr.F = F;
        OdTile od{};
        const bool use_od = L.PD != nullptr;
        if (use_od) {
            od.tiles = g->tiles_d; od.dev_off = g->dev_off_d;
            od.rp = g->rowptr[1]; od.col = g->col[1]; od.eid = g->eid[1];
            od.n_op = g->n_op; od.n_dev = g->n_dev; od.n_slots = n_slots(g, 1);
            od.Y_op = Yo; od.Y_dev = Yd; od.dO_op = L.G_op; od.dO_dev = L.G_dev; od.gamma = gc;
            od.SA1 = L.SA[1]; od.SD1 = L.SD[1]; od.SA2 = L.SA[2]; od.SD2 = L.SD[2];
            od.Zop = L.Zop; od.Zdev = L.Zdev; od.dY_op = L.dY_op; od.dY_dev = L.dY_dev;
            od.PD = L.PD; od.max_dev = std::max(g->max_dev, 1); od.n_tiles = g->n_tiles;
            od.tile_off = g->tile_off_d; od.part = L.part_od;
            od.part_a1 = L.part_a1; od.drec = L.drec; od.dstat = L.dstat; od.zrec = L.zrec; od.part_a2 = L.part_a2;
            pr.pm[1] = L.part_od; pr.nb_m[1] = R * g->n_tiles;   // both op-device source passes
            pr.nb_m[2] = 0;
            pr.pa[1] = L.part_a1; pr.nb_a[1] = R * g->n_tiles;   // both op-device softmaxes
            pr.pa[2] = L.part_a2; pr.nb_a[2] = L.nb_dev4;
        }
        pr.g_att_src = gr->att_src + (size_t)l * 3 * F;
        pr.g_att_dst = gr->att_dst + (size_t)l * 3 * F;
        pr.dU = L.dU + (size_t)l * 3 * F * 2;
        pr.dcp = L.dcp + (size_t)l * 3 * F;
        if (!dispatch_layer_bwd(F, K, dims->sigma == 1, P, B, Sx, pr, use_od ? &od : nullptr, L.dev_topo, stream))
            TAG_FAIL(TAG_ESHAPE, "unsupported f / heads");
        const float *Wl = w->layer_w + (size_t)l * 3 * F * 2 * F;
        float *gW = gr->layer_w + (size_t)l * 3 * F * 2 * F;
        // dW^h: op side rows [oo ; od], device side rows [od ; dd]
        weight_grad(L.dY_op, 2 * F, L.H_op[l], F, 2 * F, F, false, ro, L.P0, gW, 2 * F, nullptr, 0, stream,
                    TAG_STAGE_BWD_DW);
        {
            int64_t splits;
            const int64_t per = split_k_per(rd, ((2 * F + GM - 1) / GM) * ((F + GN - 1) / GN), &splits);
            Gemm gd{L.dY_dev, 2 * F, L.H_dev[l], F, 2 * F, F, rd, -1, L.P1, F, 2 * F * F, per, 0};
            prof_begin(TAG_STAGE_BWD_DW, stream);
            launch_gemm(gd, false, false, splits, stream);
            prof_end(TAG_STAGE_BWD_DW, stream);
            float *g1 = gW + (size_t)F * 2 * F;
            launch_sum_splits(L.P1, 2 * F * F, F, (int32_t)splits, F, F, g1, 2 * F, 1, stream);
            launch_sum_splits(L.P1 + (size_t)F * F, 2 * F * F, F, (int32_t)splits, F, F, g1 + (size_t)F * 2 * F, 2 * F,
                              0, stream);
        }
        // dH = dY [W^h ; W^h'] (overwrites the layer-output gradients, no longer needed)
        prof_begin(TAG_STAGE_BWD_DH, stream);
        launch_gemm(Gemm{L.dY_op, 2 * F, Wl, 2 * F, ro, F, 2 * F, -1, L.G_op, F, 0, 2 * F, 0}, true, false, 1, stream);
        prof_end(TAG_STAGE_BWD_DH, stream);
        prof_begin(TAG_STAGE_BWD_DH, stream);
        launch_gemm(Gemm{L.dY_dev, 2 * F, Wl + (size_t)F * 2 * F, 2 * F, rd, F, 2 * F, -1, L.G_dev, F, 0, 2 * F, 0},
                    true, false, 1, stream);
        prof_end(TAG_STAGE_BWD_DH, stream);
    }

    // node encoders: h0 = ReLU(A x + c)
    relu_mask<<<grid_for(ro * F), 256, 0, stream>>>(L.G_op, L.H_op[0], ro * F);
    relu_mask<<<grid_for(rd * F), 256, 0, stream>>>(L.G_dev, L.H_dev[0], rd * F);
    weight_grad(L.G_op, F, x->x_op, dims->f_op, F, dims->f_op, true, ro, L.P0, gr->enc_op_w, dims->f_op,
                gr->enc_op_b, 0, stream);
    weight_grad(L.G_dev, F, x->x_dev, dims->f_dev, F, dims->f_dev, true, rd, L.P1, gr->enc_dev_w, dims->f_dev,
                gr->enc_dev_b, 0, stream);
    // folded edge encoders
    FoldBwd fb{w->layer_w, {w->enc_edge_w[0], w->enc_edge_w[1], w->enc_edge_w[2]},
               {w->enc_edge_b[0], w->enc_edge_b[1], w->enc_edge_b[2]}, L.dU, L.dcp, gr->layer_w, gr->layer_b,
               {gr->enc_edge_w[0], gr->enc_edge_w[1], gr->enc_edge_w[2]},
               {gr->enc_edge_b[0], gr->enc_edge_b[1], gr->enc_edge_b[2]}, F, NL};
    fold_bwd_we<<<grid_for((int64_t)NL * 3 * F * F), 256, 0, stream>>>(fb);
    fold_bwd_enc<<<3 * ((F + 15) / 16), 256, 0, stream>>>(fb);

    if (lr > 0.f) {
        SgdList sl{};
        const int64_t fo = dims->f_op, fd = dims->f_dev, Hd = H;
        float *wp[18] = {const_cast<float *>(w->enc_op_w), const_cast<float *>(w->enc_op_b),
                         const_cast<float *>(w->enc_dev_w), const_cast<float *>(w->enc_dev_b),
                         const_cast<float *>(w->enc_edge_w[0]), const_cast<float *>(w->enc_edge_w[1]),
                         const_cast<float *>(w->enc_edge_w[2]), const_cast<float *>(w->enc_edge_b[0]),
                         const_cast<float *>(w->enc_edge_b[1]), const_cast<float *>(w->enc_edge_b[2]),
                         const_cast<float *>(w->layer_w), const_cast<float *>(w->layer_b),
                         const_cast<float *>(w->att_src), const_cast<float *>(w->att_dst),
                         const_cast<float *>(w->dec_w1), const_cast<float *>(w->dec_b1),
                         const_cast<float *>(w->dec_w2), const_cast<float *>(w->dec_b2)};
        const int64_t n[18] = {F * fo, F, F * fd, F, F, F, 2 * F, F, F, F, (int64_t)NL * 3 * F * 2 * F,
                               (int64_t)NL * 3 * F, (int64_t)NL * 3 * F, (int64_t)NL * 3 * F, Hd * din, Hd, Hd, 1};
        for (int i = 0; i < 18; ++i) {
            sl.w[i] = wp[i];
            sl.g[i] = gp[i];
            sl.n[i] = n[i];
        }
        sl.count = 18;
        sl.lr = lr;
        sgd_update<<<dim3(64, 18), 256, 0, stream>>>(sl);
    }
    return launch_status("tag_train_step");
}
