// Attention aggregation on the matrix cores (heads of at least 16 channels).
//
// The placement links between ops and devices carry only a bit, so every
// op<->device message is one of two rows per source node:
//   m_b[v] = ReLU(W^h_od h_v + c'_od + b U_od),  b in {0, 1}
// and its attention logit a . m_b[v] is a per-(source, bit, head) scalar.
// Both op<->device aggregations are therefore dense contractions over a
// 64-op tile of one topology:
//   device <- op:  acc[j][c] = sum_{u, b} alpha_k(j, u, b) m_b[u][c]   (M x 128) x (128 x f)
//   op <- device:  acc[u][c] = sum_{j, b} alpha_k(u, j, b) m_b[j][c]   (64 x 2M) x (2M x f)
// with alpha = 0 unless (u, j) is a placement link whose bit is b.  They run
// as fp32 MFMA 16x16x4 products; the attention weights are formed in
// registers as the A operand.  device <- op tiles write (max, sum, partial)
// records that a merge pass combines in tile order; op <- device rows are
// complete inside one tile and are normalised directly; the same kernel
// gathers the tile's op <- op rows and writes each op row once.
#include "agg_common.hpp"

namespace tag {
namespace {

// omask[r][u] = (present, bits) over the local devices of u's topology.
// One block per (op tile, candidate): the tile's op<-dev entries are one
// contiguous CSR range, read coalesced and OR-ed into LDS masks.
__global__ void __launch_bounds__(256) pack_op_masks(AggArgs A) {
    __shared__ int32_t rp[kOpTile + 1];
    __shared__ unsigned long long pres[kOpTile], bits[kOpTile];
    const int32_t t = blockIdx.x, r = blockIdx.y;
    const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
    const int32_t d0 = A.dev_off[g];
    for (int i = threadIdx.x; i <= nu; i += blockDim.x) rp[i] = A.rp[1][u0 + i];
    for (int i = threadIdx.x; i < kOpTile; i += blockDim.x) { pres[i] = 0ull; bits[i] = 0ull; }
    __syncthreads();
    const uint8_t *xb = A.x_od + (int64_t)r * A.s_od;
    for (int32_t e = rp[0] + threadIdx.x; e < rp[nu]; e += blockDim.x) {
        int lo = 0, hi = nu;   // last local row with rp[row] <= e
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (rp[mid] <= e) lo = mid; else hi = mid;
        }
        const unsigned long long m = 1ull << (A.col[1][e] - d0);
        atomicOr(&pres[lo], m);
        if (xb[A.eid[1][e]]) atomicOr(&bits[lo], m);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nu; i += blockDim.x) {
        const int64_t mi = 2 * ((int64_t)r * A.n_op + u0 + i);
        A.omask[mi] = pres[i];
        A.omask[mi + 1] = bits[i];
    }
}

// per device row: message table T (bit 0 / 1), their logits p0, p1, and the
// destination terms q_od, q_dd
template <int F, int K, bool BF>
__global__ void __launch_bounds__(256) dev_prep(AggArgs A) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    if (i >= (int64_t)A.R * A.n_dev) return;
    const int c0 = lane * CPL;
    RelConst<CPL> od; od.load(A, 1, F, c0);
    RelConst<CPL> dd; dd.load(A, 2, F, c0);
    float yo[CPL], yd[CPL];
    load_ch<CPL, BF>(A.Y_dev, i * 2 * F + F + c0, yo);
    load_ch<CPL, BF>(A.Y_dev, i * 2 * F + c0, yd);
    float p0 = 0.f, p1 = 0.f, qo = 0.f, qd = 0.f;
    for (int c = 0; c < CPL; ++c) {
        const float yc = yo[c] + od.cp[c];
        const float t0 = fmaxf(yc, 0.f), t1 = fmaxf(yc + od.u0[c], 0.f);
        A.T[(i * 2 + 0) * F + c0 + c] = t0;
        A.T[(i * 2 + 1) * F + c0 + c] = t1;
        p0 = fmaf(od.a[c], t0, p0);
        p1 = fmaf(od.a[c], t1, p1);
        qo = fmaf(od.ad[c], yo[c], qo);
        qd = fmaf(dd.ad[c], yd[c], qd);
    }
    p0 = head_sum<LPH>(p0); p1 = head_sum<LPH>(p1);
    qo = head_sum<LPH>(qo); qd = head_sum<LPH>(qd);
    if ((lane % LPH) == 0) {
        const int h = lane / LPH;
        float *S = A.Sdev + i * 4 * K;
        S[h] = p0; S[K + h] = p1; S[2 * K + h] = qo; S[3 * K + h] = qd;
    }
}

// device <- op over one 64-op tile: partial (max, sum, accumulator) records
template <int F, int K, bool BF>
__global__ void __launch_bounds__(256) agg_b2(AggArgs A) {
    constexpr int D = F / K;                       // head width (>= 16 here)
    constexpr int WC = F / 4;                      // columns per wavefront
    constexpr int NCB = WC / 16;                   // 16-column blocks per wavefront
    constexpr int HPW = WC >= D ? WC / D : 1;      // heads per wavefront
    constexpr int YS = F + 4;                      // padded LDS row
    __shared__ float Ys[kOpTile * YS];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float pb[kOpTile][2][K];
    __shared__ float qd[64][K], mxS[64][K];
    __shared__ float cpS[F], US[F], aS[F], adS[F];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t t = blockIdx.x, r = blockIdx.y;
    const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
    const int32_t d0 = A.dev_off[g], Mg = A.dev_off[g + 1] - d0;
    const int32_t chunk = t - A.tile_off[g];

    for (int i = tid; i < F; i += 256) {
        cpS[i] = A.cp[F + i];
        US[i] = A.U[(size_t)(F + i) * 2];
        aS[i] = A.att_src[F + i];
        adS[i] = A.att_dst[F + i];
    }
    for (int i = tid; i < kOpTile; i += 256) {
        const bool ok = i < nu;
        const int64_t mi = 2 * ((int64_t)r * A.n_op + u0 + i);
        pres[i] = ok ? A.omask[mi] : 0ull;
        bits[i] = ok ? A.omask[mi + 1] : 0ull;
    }
    for (int i = tid; i < 64 * K; i += 256) {
        const int j = i / K, h = i % K;
        qd[j][h] = j < Mg ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + 2 * K + h] * kLog2e : 0.f;
    }
    for (int i = tid; i < kOpTile * (F / 4); i += 256) {
        const int u = i / (F / 4), c = (i % (F / 4)) * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (u < nu) load_ch<4, BF>(A.Y_op, ((int64_t)r * A.n_op + u0 + u) * 2 * F + F + c, v);
        for (int q = 0; q < 4; ++q) Ys[u * YS + c + q] = v[q];
    }
    __syncthreads();
    // op-side logits of both message variants, and q_od of the op rows
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        float p0 = 0.f, p1 = 0.f, q = 0.f;
        for (int c = h * D; c < (h + 1) * D; ++c) {
            const float y = Ys[u * YS + c];
            const float yc = y + cpS[c];
            p0 = fmaf(aS[c], fmaxf(yc, 0.f), p0);
            p1 = fmaf(aS[c], fmaxf(yc + US[c], 0.f), p1);
            q = fmaf(adS[c], y, q);
        }
        pb[u][0][h] = p0 * kLog2e;   // exp2-domain logits
        pb[u][1][h] = p1 * kLog2e;
        if (u < nu) A.qop[((int64_t)r * A.n_op + u0 + u) * K + h] = q;
    }
    __syncthreads();
    // per (device, head): exact max of the logit over the tile's links
    // (LeakyReLU is monotone, so it is LeakyReLU of the largest pre-activation)
    for (int i = tid; i < Mg * K; i += 256) {
        const int j = i / K, h = i % K;
        float mx = -INFINITY;
        for (int u = 0; u < nu; ++u) {
            const uint64_t pr = pres[u], bt = bits[u];
            const float v = ((bt >> j) & 1ull) ? pb[u][1][h] : pb[u][0][h];
            mx = ((pr >> j) & 1ull) ? fmaxf(mx, v) : mx;
        }
        const float x = mx + qd[j][h];
        mxS[j][h] = mx == -INFINITY ? -INFINITY : fmaxf(x, A.slope * x);
    }
    __syncthreads();

    const int cbase = wave * WC;
    const int h0 = cbase / D;
    constexpr int CPH = NCB / HPW;                 // column blocks per head inside a wavefront
    float cpv[NCB], Uv[NCB];
    for (int cb = 0; cb < NCB; ++cb) {
        const int col = cbase + cb * 16 + (lane & 15);
        cpv[cb] = cpS[col];
        Uv[cb] = US[col];
    }
    const int NRB = (Mg + 15) / 16;
    f4 acc[4][NCB];
    float zl[4][HPW];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) zl[rb][hh] = 0.f;
    }
    const int b = (lane >> 4) & 1;
    const float slope = A.slope;
    // per-lane constants of the lane's device rows j = rb*16 + l%16
    float q2[4][HPW], m2[4][HPW];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        const int j = rb * 16 + (lane & 15);
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            q2[rb][hh] = qd[j][h0 + hh];
            m2[rb][hh] = j < Mg ? mxS[j][h0 + hh] : 0.f;
        }
    }
    for (int s = 0; s < kOpTile / 2; ++s) {
        const int ul = 2 * s + (lane >> 5);
        const uint64_t pr = pres[ul], bt = b ? bits[ul] : ~bits[ul];   // bt bit j: link bit equals b
        float bv[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const float yc = Ys[ul * YS + cbase + cb * 16 + (lane & 15)] + cpv[cb];
            bv[cb] = fmaxf(b ? yc + Uv[cb] : yc, 0.f);
        }
        float pu[HPW];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) pu[hh] = pb[ul][b][h0 + hh];
        const uint64_t sel = pr & bt;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            if (rb < NRB) {
                const int j = rb * 16 + (lane & 15);
                const bool on = (sel >> j) & 1ull;   // j < Mg holds for every set bit
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    const int h = h0 + hh;
                    const float x = pu[hh] + q2[rb][hh];
                    const float af = on ? __builtin_amdgcn_exp2f(fmaxf(x, slope * x) - m2[rb][hh]) : 0.f;
                    zl[rb][hh] += af;
#pragma unroll
                    for (int c2 = 0; c2 < CPH; ++c2)
                        acc[rb][hh * CPH + c2] =
                            __builtin_amdgcn_mfma_f32_16x16x4f32(af, bv[hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
                }
            }
        }
    }
    const int REC = F + 2 * K;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = rb * 16 + 4 * (lane >> 4) + v;
            if (rb < NRB && j < Mg) {
                float *rec = A.part + (((int64_t)r * A.n_dev + d0 + j) * A.maxc + chunk) * REC + 2 * K;
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) rec[cbase + cb * 16 + (lane & 15)] = acc[rb][cb][v];
            }
        }
    // softmax sums: lanes l, l+16, l+32, l+48 hold parts of device row l % 16
    const bool head_owner = (cbase % D) == 0;   // first wavefront covering its heads
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            float z = zl[rb][hh];
            z += __shfl_xor(z, 16, 64);
            z += __shfl_xor(z, 32, 64);
            const int j = rb * 16 + (lane & 15);
            if (head_owner && lane < 16 && rb < NRB && j < Mg) {
                float *rec = A.part + (((int64_t)r * A.n_dev + d0 + j) * A.maxc + chunk) * REC;
                rec[h0 + hh] = mxS[j][h0 + hh];
                rec[K + h0 + hh] = z;
            }
        }
}

// Op destinations of one 64-op tile.  op <- op: each wavefront gathers 16 of
// the tile's rows, four at a time (16 lanes and f/16 channels per row), into
// an LDS tile.  op <- device: MFMA contraction of the attention weights with
// the device message table.  Both are combined and written once.
template <int F, int K, bool BF>
__global__ void __launch_bounds__(256) agg_op_tile(AggArgs A) {
    constexpr int D = F / K;
    constexpr int WC = F / 4;
    constexpr int NCB = WC / 16;
    constexpr int HPW = WC >= D ? WC / D : 1;
    constexpr int CPL = F / 16;              // op<-op channels per lane
    constexpr int LPH = 16 / K;              // op<-op lanes per head (K <= 16 on this path)
    constexpr int EB = CPL >= 16 ? 2 : 4;    // neighbour rows loaded together
    constexpr int OS = F + 4;                // LDS tile row stride
    __shared__ float Ot[kOpTile * OS];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float qo[kOpTile][K], mxS[kOpTile][K];
    __shared__ float P[64][2][K];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t t = blockIdx.x, r = blockIdx.y;
    const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
    const int32_t d0 = A.dev_off[g], Mg = A.dev_off[g + 1] - d0;
    for (int i = tid; i < kOpTile; i += 256) {
        const bool ok = i < nu;
        const int64_t mi = 2 * ((int64_t)r * A.n_op + u0 + i);
        pres[i] = ok ? A.omask[mi] : 0ull;
        bits[i] = ok ? A.omask[mi + 1] : 0ull;
    }
    // logits in the exp2 domain: LeakyReLU commutes with the positive factor log2(e)
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        qo[u][h] = u < nu ? A.qop[((int64_t)r * A.n_op + u0 + u) * K + h] * kLog2e : 0.f;
    }
    for (int i = tid; i < 64 * 2 * K; i += 256) {
        const int j = i / (2 * K), bh = i % (2 * K);
        P[j][bh / K][bh % K] = j < Mg ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + bh] * kLog2e : 0.f;
    }
    __syncthreads();
    // op <- device softmax maxima (LeakyReLU of the largest pre-activation)
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        const uint64_t pr = pres[u], bt = bits[u];
        float mx = -INFINITY;
        for (int j = 0; j < Mg; ++j)
            if ((pr >> j) & 1ull) mx = fmaxf(mx, P[j][(bt >> j) & 1ull][h]);
        const float x = mx + qo[u][h];
        mxS[u][h] = mx == -INFINITY ? -INFINITY : fmaxf(x, A.slope * x);
    }
    // op <- op into the LDS tile (gamma_same applied)
    {
        const int li = lane & 15;
        const int c0 = li * CPL;
        float a[CPL], u0c[CPL], cp[CPL], ad[CPL];
        for (int c = 0; c < CPL; ++c) {
            a[c] = A.att_src[c0 + c];
            u0c[c] = A.U[(size_t)(c0 + c) * 2];
            cp[c] = A.cp[c0 + c];
            ad[c] = A.att_dst[c0 + c];
        }
        const float *xo = A.x_oo + (int64_t)r * A.s_oo;
        const int64_t ybase = (int64_t)r * A.n_op * 2 * F + c0;
        for (int it = 0; it < 4; ++it) {
            const int ul = wave * 16 + it * 4 + (lane >> 4);
            const bool live = ul < nu;
            const int32_t u = u0 + (live ? ul : 0);
            float q = 0.f;
            {
                float yd[CPL];
                load_ch<CPL, BF>(A.Y_op, ybase + (int64_t)u * 2 * F, yd);
                for (int c = 0; c < CPL; ++c) q = fmaf(ad[c], yd[c], q);
            }
            q = head_sum<LPH>(q);
            Online<CPL> o; o.init();
            const int32_t beg = A.rp[0][u], end = A.rp[0][u + 1];
            for (int32_t e = beg; e < end; e += EB) {
                const int n = min(EB, end - e);
                int32_t v[EB], id[EB];
                for (int i = 0; i < EB; ++i) {
                    v[i] = i < n ? A.col[0][e + i] : 0;
                    id[i] = i < n ? A.eid[0][e + i] : 0;
                }
                float x[EB], y[EB][CPL];
                for (int i = 0; i < EB; ++i) {
                    x[i] = i < n ? xo[id[i]] : 0.f;
                    if (i < n) load_ch<CPL, BF>(A.Y_op, ybase + (int64_t)v[i] * 2 * F, y[i]);
                }
                for (int i = 0; i < EB; ++i) {
                    if (i < n) {
                        float m[CPL], part = 0.f;
                        for (int c = 0; c < CPL; ++c) {
                            m[c] = fmaxf(y[i][c] + fmaf(u0c[c], x[i], cp[c]), 0.f);
                            part = fmaf(a[c], m[c], part);
                        }
                        const float s2 = leaky(head_sum<LPH>(part) + q, A.slope) * kLog2e;
                        o.push(s2, m);
                    }
                }
            }
            const float inv = end > beg ? A.g_same / o.den : 0.f;
            if (live)
                for (int c = 0; c < CPL; ++c) Ot[ul * OS + c0 + c] = o.acc[c] * inv;
        }
    }
    __syncthreads();

    const int cbase = wave * WC;
    const int h0 = cbase / D;
    constexpr int CPH = NCB / HPW;
    f4 acc[4][NCB];
    float zl[4][HPW];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) zl[rb][hh] = 0.f;
    }
    const float *Tb = A.T + ((int64_t)r * A.n_dev + d0) * 2 * F;
    const int steps = (Mg + 1) / 2;
    const int b = (lane >> 4) & 1;
    // per-lane constants of the lane's op rows u = rb*16 + l%16; the masks are
    // pre-shifted to this lane's first device (j = l/32) and advance two per step
    uint64_t prs[4], bts[4];
    float q2[4][HPW], m2[4][HPW];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        const int u = rb * 16 + (lane & 15);
        prs[rb] = pres[u] >> (lane >> 5);
        bts[rb] = bits[u] >> (lane >> 5);
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            q2[rb][hh] = qo[u][h0 + hh];
            m2[rb][hh] = mxS[u][h0 + hh];
        }
    }
    const float slope = A.slope;
    for (int s = 0; s < steps; ++s) {
        const int j = 2 * s + (lane >> 5);
        const bool jok = j < Mg;
        float bv[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
            bv[cb] = jok ? Tb[((int64_t)j * 2 + b) * F + cbase + cb * 16 + (lane & 15)] : 0.f;
        float pj[HPW];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) pj[hh] = P[j][b][h0 + hh];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            const bool on = jok && (prs[rb] & 1ull) && ((int)(bts[rb] & 1ull) == b);
            prs[rb] >>= 2;
            bts[rb] >>= 2;
#pragma unroll
            for (int hh = 0; hh < HPW; ++hh) {
                const float x = pj[hh] + q2[rb][hh];
                const float af = on ? __builtin_amdgcn_exp2f(fmaxf(x, slope * x) - m2[rb][hh]) : 0.f;
                zl[rb][hh] += af;
#pragma unroll
                for (int c2 = 0; c2 < CPH; ++c2)
                    acc[rb][hh * CPH + c2] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(af, bv[hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
            }
        }
    }
    // softmax sums of op row rb*16 + l%16 are spread over lanes l, l+16,
    // l+32, l+48; the output row of register v in lane l is rb*16 + 4(l/16) + v
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        float scale[HPW][4];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            float z = zl[rb][hh];
            z += __shfl_xor(z, 16, 64);
            z += __shfl_xor(z, 32, 64);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float zv = __shfl(z, 4 * (lane >> 4) + v, 64);
                scale[hh][v] = zv > 0.f ? A.g_cross / zv : 0.f;
            }
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int u = rb * 16 + 4 * (lane >> 4) + v;
            if (u >= nu) continue;
            const int64_t row = (int64_t)r * A.n_op + u0 + u;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int col = cbase + cb * 16 + (lane & 15);
                const float val = fmaf(scale[cb / CPH][v], acc[rb][cb][v], Ot[u * OS + col]);
                if (A.out_f32) static_cast<float *>(A.H_op)[row * F + col] = val;
                else static_cast<uint16_t *>(A.H_op)[row * F + col] = f2bf(val);
            }
        }
    }
}

template <int F, int K, bool BF>
void launch_mfma(const AggArgs &A, hipStream_t st) {
    const int64_t op_waves = (int64_t)A.R * A.n_op;
    const int64_t dev_waves = (int64_t)A.R * A.n_dev;
    const dim3 tiles((unsigned)A.n_tiles, (unsigned)A.R);
    prof_begin(TAG_STAGE_DEV_PREP, st);
    dev_prep<F, K, BF><<<(unsigned)((dev_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A);
    prof_end(TAG_STAGE_DEV_PREP, st);
    prof_begin(TAG_STAGE_AGG_DEV_OP, st);
    agg_b2<F, K, BF><<<tiles, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_DEV_OP, st);
    prof_begin(TAG_STAGE_AGG_OP_DEV, st);
    agg_op_tile<F, K, BF><<<tiles, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_OP_DEV, st);
    (void)op_waves;
}

template <int F, bool BF>
bool dispatch_mfma_heads(int K, const AggArgs &A, hipStream_t st) {
    switch (K) {
        case 1: launch_mfma<F, 1, BF>(A, st); return true;
        case 2: launch_mfma<F, 2, BF>(A, st); return true;
        case 4: launch_mfma<F, 4, BF>(A, st); return true;
        case 8: if (F / 8 >= 16) { launch_mfma<F, (F / 8 >= 16 ? 8 : 4), BF>(A, st); return true; } return false;
        case 16: if (F / 16 >= 16) { launch_mfma<F, (F / 16 >= 16 ? 16 : 4), BF>(A, st); return true; } return false;
        default: return false;
    }
}

}  // namespace

bool mfma_path_supported(int F, int K) { return K >= 1 && F / K >= 16 && K <= 16; }

void launch_pack_masks(const AggArgs &A, hipStream_t st) {
    pack_op_masks<<<dim3((unsigned)A.n_tiles, (unsigned)A.R), 256, 0, st>>>(A);
}

bool launch_agg_mfma(int F, int K, bool bf, const AggArgs &A, hipStream_t st) {
    if (!mfma_path_supported(F, K)) return false;
    if (F == 64) return bf ? dispatch_mfma_heads<64, true>(K, A, st) : dispatch_mfma_heads<64, false>(K, A, st);
    if (F == 128) return bf ? dispatch_mfma_heads<128, true>(K, A, st) : dispatch_mfma_heads<128, false>(K, A, st);
    return bf ? dispatch_mfma_heads<256, true>(K, A, st) : dispatch_mfma_heads<256, false>(K, A, st);
}

}  // namespace tag
