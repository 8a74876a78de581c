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
#include <type_traits>

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

// Attention terms of node rows when the transform epilogue cannot form them
// (heads wider than 64 channels): per row, S = (p0, p1, q_od, q_same) and, for
// device rows, the message table T (bit 0 / 1).  One wavefront per row.
template <int F, int K, bool BF>
__global__ void __launch_bounds__(256) prep_rows(AggArgs A, int dev_side) {
    constexpr int CPL = F / 64, LPH = 64 / K;
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    const int64_t rows = (int64_t)A.R * (dev_side ? A.n_dev : A.n_op);
    if (i >= rows) return;
    const void *Y = dev_side ? A.Y_dev : A.Y_op;
    float *Sr = dev_side ? A.Sdev : A.Sop;
    const int c0 = lane * CPL;
    RelConst<CPL> od; od.load(A, 1, F, c0);
    RelConst<CPL> same; same.load(A, dev_side ? 2 : 0, F, c0);
    float yo[CPL], ys[CPL];
    load_ch<CPL, BF>(Y, i * 2 * F + F + c0, yo);
    load_ch<CPL, BF>(Y, i * 2 * F + c0, ys);
    float p0 = 0.f, p1 = 0.f, qo = 0.f, qs = 0.f;
    for (int c = 0; c < CPL; ++c) {
        const float yc = yo[c];   // stored rows hold Y + c'
        const float t0 = fmaxf(yc, 0.f), t1 = fmaxf(yc + od.u0[c], 0.f);
        if (dev_side) {
            if (BF) {
                reinterpret_cast<unsigned *>(A.T)[i * F + c0 + c] = pack_bf2(t0, t1);
            } else {
                A.T[(i * 2 + 0) * F + c0 + c] = t0;
                A.T[(i * 2 + 1) * F + c0 + c] = t1;
            }
        }
        p0 = fmaf(od.a[c], t0, p0);
        p1 = fmaf(od.a[c], t1, p1);
        qo = fmaf(od.ad[c], yo[c] - od.cp[c], qo);
        qs = fmaf(same.ad[c], ys[c] - same.cp[c], qs);
    }
    p0 = head_sum<LPH>(p0); p1 = head_sum<LPH>(p1);
    qo = head_sum<LPH>(qo); qs = head_sum<LPH>(qs);
    if ((lane % LPH) == 0) {
        const int h = lane / LPH;
        float *S = Sr + i * 4 * K;
        S[h] = p0; S[K + h] = p1; S[2 * K + h] = qo; S[3 * K + h] = qs;
    }
}

// order-preserving float <-> int keys (LDS integer max atomics on floats)
__device__ __forceinline__ int fkey(float x) {
    const int i = __float_as_int(x);
    return i < 0 ? i ^ 0x7fffffff : i;
}
__device__ __forceinline__ float fdekey(int k) { return __int_as_float(k < 0 ? k ^ 0x7fffffff : k); }

// device <- op over one group of consecutive 64-op tiles of a topology.  A
// first pass takes the exact softmax maxima of the group's links (every
// (op, head) raises the maxima of its linked devices); the MFMA passes then
// accumulate every tile against those fixed maxima, so the device-row
// accumulators stay in registers across the group, and one (max, sum,
// partial) record per device row is written at the end.
template <int F, int K, bool BF>
__global__ void __launch_bounds__(256) agg_b2(AggArgs A) {
    constexpr int D = F / K;                       // head width (>= 16 here)
    constexpr int WC = F / 4;                      // columns per wavefront
    constexpr int NCB = WC / 16;                   // 16-column blocks per wavefront
    constexpr int HPW = WC >= D ? WC / D : 1;      // heads per wavefront
    constexpr int CPH = NCB / HPW;                 // column blocks per head inside a wavefront
    constexpr int YS = BF ? F + 8 : F + 4;         // padded LDS row (bf16 rows stay 16-byte aligned)
    typedef typename std::conditional<BF, uint16_t, float>::type YT;
    __shared__ __attribute__((aligned(16))) YT Ys[kOpTile * YS];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float pb[kOpTile][2][K];
    __shared__ int mxk[64][K];
    __shared__ float qd[64][K], mrun[64][K];
    __shared__ float US[F];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t r = blockIdx.y;
    const int32_t t0 = A.groups[2 * blockIdx.x];
    const int32_t t1 = t0 + A.groups[2 * blockIdx.x + 1];
    const int32_t g = A.tiles[3 * t0 + 2];
    const int32_t d0 = A.dev_off[g], Mg = A.dev_off[g + 1] - d0;
    const int32_t chunk = (int32_t)blockIdx.x - A.group_off[g];
    const float *Sop = A.Sop + (int64_t)r * A.n_op * 4 * K;
    const uint64_t *om = A.omask + (int64_t)r * A.n_op * 2;
    const float slope = A.slope;

    for (int i = tid; i < F; i += 256) {
        US[i] = A.U[(size_t)(F + i) * 2];
    }
    for (int i = tid; i < 64 * K; i += 256) {
        const int j = i / K, h = i % K;
        qd[j][h] = j < Mg ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + 2 * K + h] * kLog2e : 0.f;
        mxk[j][h] = INT_MIN;
    }
    __syncthreads();
    for (int32_t t = t0; t < t1; ++t) {
        const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1];
        for (int i = tid; i < nu * K; i += 256) {
            const int64_t u = u0 + i / K;
            const int h = i % K;
            uint64_t pr = om[2 * u];
            const uint64_t bt = om[2 * u + 1];
            const int k0 = fkey(Sop[u * 4 * K + h]), k1 = fkey(Sop[u * 4 * K + K + h]);
            while (pr) {
                const int j = __builtin_ctzll(pr);
                pr &= pr - 1;
                atomicMax(&mxk[j][h], ((bt >> j) & 1ull) ? k1 : k0);
            }
        }
    }
    __syncthreads();
    // LeakyReLU is monotone: the largest logit is LeakyReLU of the largest
    // pre-activation (exp2 domain)
    for (int i = tid; i < 64 * K; i += 256) {
        const int j = i / K, h = i % K;
        const int key = mxk[j][h];
        const float x = key == INT_MIN ? 0.f : fdekey(key) * kLog2e + qd[j][h];
        mrun[j][h] = key == INT_MIN ? -INFINITY : fmaxf(x, slope * x);
    }

    const int cbase = wave * WC;
    const int h0 = cbase / D;
    const int NRB = (Mg + 15) / 16;
    const int b = (lane >> 4) & 1;
    float Uv[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const int col = cbase + cb * 16 + (lane & 15);
        Uv[cb] = US[col];
    }
    f4 acc[4][NCB];
    float zl[4][HPW], q2[4][HPW], m2[4][HPW];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) zl[rb][hh] = 0.f;
    }

    for (int32_t t = t0; t < t1; ++t) {
        const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1];
        for (int i = tid; i < kOpTile; i += 256) {
            const bool ok = i < nu;
            pres[i] = ok ? om[2 * (int64_t)(u0 + i)] : 0ull;
            bits[i] = ok ? om[2 * (int64_t)(u0 + i) + 1] : 0ull;
        }
        for (int i = tid; i < kOpTile * 2 * K; i += 256) {
            const int u = i / (2 * K), bh = i % (2 * K);
            pb[u][bh / K][bh % K] = u < nu ? Sop[(int64_t)(u0 + u) * 4 * K + bh] * kLog2e : 0.f;
        }
        if constexpr (BF) {
            for (int i = tid; i < kOpTile * (F / 8); i += 256) {
                const int u = i / (F / 8), c = (i % (F / 8)) * 8;
                u4v v = u4v{0u, 0u, 0u, 0u};
                if (u < nu)
                    v = *reinterpret_cast<const u4v *>(static_cast<const uint16_t *>(A.Y_op) +
                                                       ((int64_t)r * A.n_op + u0 + u) * 2 * F + F + c);
                *reinterpret_cast<u4v *>(&Ys[u * YS + c]) = v;
            }
        } else {
            for (int i = tid; i < kOpTile * (F / 4); i += 256) {
                const int u = i / (F / 4), c = (i % (F / 4)) * 4;
                float v[4] = {0.f, 0.f, 0.f, 0.f};
                if (u < nu) load_ch<4, false>(A.Y_op, ((int64_t)r * A.n_op + u0 + u) * 2 * F + F + c, v);
                for (int q = 0; q < 4; ++q) Ys[u * YS + c + q] = v[q];
            }
        }
        __syncthreads();
        if (t == t0) {
            // per-lane constants of the lane's device rows j = rb*16 + l%16
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const int j = rb * 16 + (lane & 15);
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    q2[rb][hh] = qd[j][h0 + hh];
                    m2[rb][hh] = j < Mg ? mrun[j][h0 + hh] : 0.f;
                }
            }
        }
        if constexpr (BF) {
            // bf16 16x16x32 products: k = 2u + b over the tile's 64 ops; lane l
            // supplies k = 8(l/16) .. 8(l/16)+7 of a 32-wide step, i.e. ops
            // ub .. ub+3 with both bits
#pragma unroll 1
            for (int ks = 0; ks < kOpTile / 16; ++ks) {
                const int ub = 16 * ks + 4 * (lane >> 4);
                bf8 bop[NCB];
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const int c = cbase + cb * 16 + (lane & 15);
                    unsigned w[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float yc = bf2f(Ys[(ub + q) * YS + c]);
                        w[q] = pack_bf2(fmaxf(yc, 0.f), fmaxf(yc + Uv[cb], 0.f));
                    }
                    bop[cb] = as_bf8(w[0], w[1], w[2], w[3]);
                }
                uint64_t prq[4], btq[4];
                float p0q[4][HPW], p1q[4][HPW];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    prq[q] = pres[ub + q];
                    btq[q] = bits[ub + q];
#pragma unroll
                    for (int hh = 0; hh < HPW; ++hh) {
                        p0q[q][hh] = pb[ub + q][0][h0 + hh];
                        p1q[q][hh] = pb[ub + q][1][h0 + hh];
                    }
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    if (rb < NRB) {
                        const int j = rb * 16 + (lane & 15);
#pragma unroll
                        for (int hh = 0; hh < HPW; ++hh) {
                            unsigned w[4];
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const bool on = (prq[q] >> j) & 1ull;
                                const bool bit = (btq[q] >> j) & 1ull;
                                const float x = (bit ? p1q[q][hh] : p0q[q][hh]) + q2[rb][hh];
                                const float af = on ? __builtin_amdgcn_exp2f(fmaxf(x, slope * x) - m2[rb][hh]) : 0.f;
                                zl[rb][hh] += af;
                                w[q] = pack_bf2(bit ? 0.f : af, bit ? af : 0.f);
                            }
                            const bf8 aop = as_bf8(w[0], w[1], w[2], w[3]);
#pragma unroll
                            for (int c2 = 0; c2 < CPH; ++c2)
                                acc[rb][hh * CPH + c2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    aop, bop[hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
                        }
                    }
                }
            }
        } else
        for (int s = 0; s < kOpTile / 2; ++s) {
            const int ul = 2 * s + (lane >> 5);
            const uint64_t pr = pres[ul], bt = b ? bits[ul] : ~bits[ul];   // bt bit j: link bit equals b
            float bv[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const float yc = static_cast<float>(Ys[ul * YS + cbase + cb * 16 + (lane & 15)]);
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
                        const float x = pu[hh] + q2[rb][hh];
                        const float af = on ? __builtin_amdgcn_exp2f(fmaxf(x, slope * x) - m2[rb][hh]) : 0.f;
                        zl[rb][hh] += af;
#pragma unroll
                        for (int c2 = 0; c2 < CPH; ++c2)
                            acc[rb][hh * CPH + c2] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                af, bv[hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();   // the next tile overwrites the LDS tile and masks
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
                rec[h0 + hh] = mrun[j][h0 + hh];
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
    constexpr int EB = (CPL >= 16 || (CPL == 8 && !BF)) ? 2 : 4;   // neighbour rows per batch
    constexpr int OS = F + 4;                // LDS tile row stride
    constexpr int ECAP = F >= 256 ? 512 : 192;   // op<-op entries of the tile staged in LDS (the rest
                                                 // are read from the CSR; 192 keeps four blocks per CU at f = 128)
    __shared__ float Ot[kOpTile * OS];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float qo[kOpTile][K], mxS[kOpTile][K];
    __shared__ float P[64][2][K];
    __shared__ int32_t Erp[kOpTile + 1], Ecol[ECAP];
    __shared__ float Ex[ECAP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t t = blockIdx.x, r = blockIdx.y;
    const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
    const int32_t d0 = A.dev_off[g], Mg = A.dev_off[g + 1] - d0;
    const float *xo = A.x_oo + (int64_t)r * A.s_oo;
    // the tile's op <- op entries are one contiguous CSR range
    const int32_t eb = A.rp[0][u0];
    const int32_t ne = min(A.rp[0][u0 + nu] - eb, ECAP);
    for (int i = tid; i <= nu; i += 256) Erp[i] = A.rp[0][u0 + i] - eb;
    for (int i = tid; i < ne; i += 256) {
        Ecol[i] = A.col[0][eb + i];
        Ex[i] = xo[A.eid[0][eb + i]];
    }
    for (int i = tid; i < kOpTile; i += 256) {
        const bool ok = i < nu;
        const int64_t mi = 2 * ((int64_t)r * A.n_op + u0 + i);
        pres[i] = ok ? A.omask[mi] : 0ull;
        bits[i] = ok ? A.omask[mi + 1] : 0ull;
    }
    // logits in the exp2 domain: LeakyReLU commutes with the positive factor log2(e)
    const float *Sop = A.Sop + (int64_t)r * A.n_op * 4 * K;
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        qo[u][h] = u < nu ? Sop[(int64_t)(u0 + u) * 4 * K + 2 * K + h] * kLog2e : 0.f;
    }
    for (int i = tid; i < 64 * 2 * K; i += 256) {
        const int j = i / (2 * K), bh = i % (2 * K);
        P[j][bh / K][bh % K] = j < Mg ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + bh] * kLog2e : 0.f;
    }
    __syncthreads();
    // op <- device softmax maxima (LeakyReLU of the largest pre-activation)
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        uint64_t pr = pres[u];
        const uint64_t bt = bits[u];
        float mx = -INFINITY;
        while (pr) {
            const int j = __builtin_ctzll(pr);
            pr &= pr - 1;
            mx = fmaxf(mx, P[j][(bt >> j) & 1ull][h]);
        }
        const float x = mx + qo[u][h];
        mxS[u][h] = mx == -INFINITY ? -INFINITY : fmaxf(x, A.slope * x);
    }
    // op <- op into the LDS tile (gamma_same applied).  Each 16-lane group
    // streams four consecutive tile rows (one contiguous entry range) batch
    // by batch, so groups whose rows are short move on instead of idling.
    {
        const int li = lane & 15;
        const int c0 = li * CPL;
        float a[CPL], u0c[CPL];
        for (int c = 0; c < CPL; ++c) {
            a[c] = A.att_src[c0 + c];
            u0c[c] = A.U[(size_t)(c0 + c) * 2];
        }
        const int64_t ybase = (int64_t)r * A.n_op * 2 * F + c0;
        const float slope = A.slope;
        const int gr0 = wave * 16 + (lane >> 4) * 4;   // the group's first tile row
        auto rbeg = [&](int i) -> int32_t { return Erp[min(gr0 + i, nu)]; };   // rows >= nu are empty
        float qv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ul = gr0 + i;
            qv[i] = ul < nu ? Sop[(int64_t)(u0 + ul) * 4 * K + 3 * K + c0 / (F / K)] : 0.f;
            if (ul < nu)
                for (int c = 0; c < CPL; ++c) Ot[ul * OS + c0 + c] = 0.f;   // rows without entries stay zero
        }
        // (row, first entry, row end) of the group's batches; ri == 4: done
        auto first_from = [&](int i, int &ri, int32_t &e, int32_t &rend) {
            while (i < 4 && rbeg(i + 1) == rbeg(i)) ++i;
            ri = i;
            e = i < 4 ? rbeg(i) : 0;
            rend = i < 4 ? rbeg(i + 1) : 0;
        };
        RowRaw<CPL, BF> buf[EB];
        float xx[EB];
        auto fetch = [&](int32_t e, int32_t end) {
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                const int32_t le = e + i;
                int32_t v = u0;
                xx[i] = 0.f;
                if (le < end) {
                    if (le < ECAP) { v = Ecol[le]; xx[i] = Ex[le]; }
                    else { v = A.col[0][eb + le]; xx[i] = xo[A.eid[0][eb + le]]; }
                }
                buf[i].load(A.Y_op, ybase + (int64_t)v * 2 * F);   // a tile row when past the end
            }
        };
        int ri;
        int32_t e, rend;
        first_from(0, ri, e, rend);
        Online<CPL> o; o.init();
        if (ri < 4) fetch(e, rend);
        // one batch per iteration: the batch's messages are formed from buf,
        // then buf is refilled with the following batch (possibly of a later
        // row) while scores and the softmax update of this one proceed
        while (ri < 4) {
            const int n = min(EB, rend - e);
            int nri = ri;
            int32_t ne = e + n, nrend = rend;
            if (ne >= rend) first_from(ri + 1, nri, ne, nrend);
            float m[EB][CPL];
#pragma unroll
            for (int i = 0; i < EB; ++i)
#pragma unroll
                for (int c = 0; c < CPL; ++c) m[i][c] = fmaxf(fmaf(u0c[c], xx[i], buf[i].get(c)), 0.f);
            if (nri < 4) fetch(ne, nrend);
            const float q = ri == 0 ? qv[0] : (ri == 1 ? qv[1] : (ri == 2 ? qv[2] : qv[3]));
            float s2[EB];
#pragma unroll
            for (int i = 0; i < EB; ++i) {
                float part = 0.f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) part = fmaf(a[c], m[i][c], part);
                const float sv = head_sum<LPH>(part) + q;
                s2[i] = fmaxf(sv, slope * sv) * kLog2e;
            }
            o.template push_n<EB>(s2, m, n);
            if (nri != ri) {   // row ri complete
                const float inv = A.g_same / o.den;
                for (int c = 0; c < CPL; ++c) Ot[(gr0 + ri) * OS + c0 + c] = o.acc[c] * inv;
                o.init();
            }
            ri = nri; e = ne; rend = nrend;
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
    const float slope = A.slope;
    if constexpr (BF) {
        // bf16 16x16x32 products: k = 2j + b over the tile's devices; lane l
        // supplies devices jb .. jb+3 (both bits) of a 32-wide step
        const unsigned *Tp = reinterpret_cast<const unsigned *>(A.T) + ((int64_t)r * A.n_dev + d0) * F;
        uint64_t prs[4], bts[4];
        float q2[4][HPW], m2[4][HPW];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            const int u = rb * 16 + (lane & 15);
            prs[rb] = pres[u];
            bts[rb] = bits[u];
#pragma unroll
            for (int hh = 0; hh < HPW; ++hh) {
                q2[rb][hh] = qo[u][h0 + hh];
                m2[rb][hh] = mxS[u][h0 + hh];
            }
        }
        const int ksteps = (Mg + 15) / 16;
        bf8 bops[4][NCB];   // every step's message operands, loaded together
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int jb = 16 * ks + 4 * (lane >> 4);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int c = cbase + cb * 16 + (lane & 15);
                unsigned w[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) w[q] = jb + q < Mg ? Tp[(int64_t)(jb + q) * F + c] : 0u;
                bops[ks][cb] = as_bf8(w[0], w[1], w[2], w[3]);
            }
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (ks >= ksteps) break;
            const int jb = 16 * ks + 4 * (lane >> 4);
            const bf8 (&bop)[NCB] = bops[ks];
            float p0q[4][HPW], p1q[4][HPW];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    p0q[q][hh] = P[jb + q][0][h0 + hh];
                    p1q[q][hh] = P[jb + q][1][h0 + hh];
                }
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    unsigned w[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const bool on = (prs[rb] >> (jb + q)) & 1ull;    // never set for jb + q >= Mg
                        const bool bit = (bts[rb] >> (jb + q)) & 1ull;
                        const float x = (bit ? p1q[q][hh] : p0q[q][hh]) + q2[rb][hh];
                        const float af = on ? __builtin_amdgcn_exp2f(fmaxf(x, slope * x) - m2[rb][hh]) : 0.f;
                        zl[rb][hh] += af;
                        w[q] = pack_bf2(bit ? 0.f : af, bit ? af : 0.f);
                    }
                    const bf8 aop = as_bf8(w[0], w[1], w[2], w[3]);
#pragma unroll
                    for (int c2 = 0; c2 < CPH; ++c2)
                        acc[rb][hh * CPH + c2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            aop, bop[hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
                }
            }
        }
    } else {
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
    const dim3 groups((unsigned)A.n_groups, (unsigned)A.R);
    if (!A.prep_done) {
        prof_begin(TAG_STAGE_DEV_PREP, st);
        prep_rows<F, K, BF><<<(unsigned)((op_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A, 0);
        prep_rows<F, K, BF><<<(unsigned)((dev_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A, 1);
        prof_end(TAG_STAGE_DEV_PREP, st);
    }
    prof_begin(TAG_STAGE_AGG_DEV_OP, st);
    agg_b2<F, K, BF><<<groups, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_DEV_OP, st);
    prof_begin(TAG_STAGE_AGG_OP_DEV, st);
    agg_op_tile<F, K, BF><<<tiles, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_OP_DEV, st);
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
