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
// with alpha = 0 unless (u, j) is a placement link whose bit is b, so each
// (row, source) pair of k = 2 source + b holds at most one nonzero weight:
// the 2:4 structure of the sparse 16x16x64 bf16 products, which take both
// operands as exact three-way bf16 splits (six part products, an fp32
// contraction up to fp32 rounding).  fp32 op <- device at F <= 128 runs on
// fp32 16x16x4 products instead (fewer registers, four blocks per CU).  The
// attention weights are formed in registers as the A operand.  device <- op
// tiles write (max, sum, partial)
// records that a merge pass combines in tile order; op <- device rows are
// complete inside one tile and are normalised directly; the same kernel
// gathers the tile's op <- op rows and writes each op row once.
#include <type_traits>

#include "agg_common.hpp"

namespace tag {
namespace {

// omask[r][u] = (present, bits) over the local devices of u's topology.
// One block per (op tile, kMaskCands candidates): the tile's op<-dev CSR range
// is read once for the group; four lanes per op row walk its entries and OR
// device bits in registers, and the four partial masks meet by shuffles.
constexpr int kMaskCands = 4;
static_assert(kMaskCands == 4 && kOpTile * 4 == 256, "one lane per quarter row and per stored candidate");

__global__ void __launch_bounds__(256) pack_op_masks(AggArgs A) {
    typedef unsigned long long u64;
    const int32_t t = blockIdx.x, r0 = blockIdx.y * kMaskCands;
    const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
    const int32_t d0 = A.dev_off[g];
    const int i = threadIdx.x >> 2, q = threadIdx.x & 3;   // op row of the tile, quarter
    u64 pres = 0ull, bits[kMaskCands];
#pragma unroll
    for (int k = 0; k < kMaskCands; ++k) bits[k] = 0ull;
    if (i < nu) {
        const int32_t e1 = A.rp[1][u0 + i + 1];
        for (int32_t e = A.rp[1][u0 + i] + q; e < e1; e += 4) {
            const u64 m = 1ull << (A.col[1][e] - d0);
            const int64_t id = A.eid[1][e];
            pres |= m;
#pragma unroll
            for (int k = 0; k < kMaskCands; ++k)
                if (r0 + k < A.R && A.x_od[(int64_t)(r0 + k) * A.s_od + id]) bits[k] |= m;
        }
    }
    // lanes 4i .. 4i + 3 of one wavefront hold the quarters of row i
#pragma unroll
    for (int o = 1; o < 4; o <<= 1) {
        pres |= __shfl_xor(pres, o);
#pragma unroll
        for (int k = 0; k < kMaskCands; ++k) bits[k] |= __shfl_xor(bits[k], o);
    }
    if (i < nu && r0 + q < A.R) {   // lane q stores candidate r0 + q
        u64 b = bits[0];
#pragma unroll
        for (int k = 1; k < kMaskCands; ++k) b = q == k ? bits[k] : b;
        const int64_t mi = 2 * ((int64_t)(r0 + q) * A.n_op + u0 + i);
        A.omask[mi] = pres;
        A.omask[mi + 1] = b;
    }
}

// Attention terms of node rows when the transform epilogue cannot form them
// (heads wider than 64 channels): per row, S = (p0, p1, q_od, q_same) and, for
// device rows, the message table T (bit 0 / 1; fp32, or its exact bf16
// splits in the bf16 variant).  One wavefront per row.
// Once per forward pass: the op tiles' descriptors (so an op-destination block
// finds its CSR range and device group in one load round) and the op<-op
// edge features in CSR order (so it loads them without the edge-id gather).
__global__ void __launch_bounds__(256) prep_tiles_x(AggArgs A, int64_t nnz0, int32_t xrep) {
    const int64_t n = (int64_t)A.n_tiles + (int64_t)xrep * nnz0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
        if (i < A.n_tiles) {
            const int32_t t = (int32_t)i;
            const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1], g = A.tiles[3 * t + 2];
            const int32_t eb = A.rp[0][u0], d0 = A.dev_off[g];
            int32_t *o = A.tile_ext + 8 * (int64_t)t;
            o[0] = u0; o[1] = nu; o[2] = g; o[3] = eb; o[4] = A.rp[0][u0 + nu] - eb;
            o[5] = d0; o[6] = A.dev_off[g + 1] - d0; o[7] = 0;
        } else {
            const int64_t j = i - A.n_tiles, r = j / nnz0, e = j % nnz0;
            A.xcsr[j] = A.x_oo[r * A.s_oo + A.eid[0][e]];
        }
    }
}

template <int F, int K, bool BF, bool ELU = false>
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
        const float yc = BF ? yo[c] + od.cp[c] : yo[c];   // Y + c' (fp32 rows store it, bf16 rows store Y)
        const float t0 = msg_act<ELU>(yc), t1 = msg_act<ELU>(yc + od.u0[c]);
        if (dev_side) {
            if constexpr (BF || F >= 256) {   // exact three-way bf16 splits, (bit 0, bit 1) pairs
                unsigned sp[3];
                split3(t0, t1, sp);
                unsigned *Tu = reinterpret_cast<unsigned *>(A.T);
                for (int q = 0; q < 3; ++q) Tu[q * rows * F + i * F + c0 + c] = sp[q];
            } else {
                A.T[(i * 2 + 0) * F + c0 + c] = t0;
                A.T[(i * 2 + 1) * F + c0 + c] = t1;
            }
        }
        p0 = fmaf(od.a[c], t0, p0);
        p1 = fmaf(od.a[c], t1, p1);
        qo = fmaf(od.ad[c], stored_dst<BF>(yo[c], od.cp[c]), qo);
        qs = fmaf(same.ad[c], stored_dst<BF>(ys[c], same.cp[c]), qs);
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
template <int F, int K, bool BF, bool ELU = false>
__global__ void __launch_bounds__(256) agg_b2(AggArgs A) {
    constexpr int D = F / K;                       // head width (>= 16 here)
    constexpr int WC = F / 4;                      // columns per wavefront
    constexpr int NCB = WC / 16;                   // 16-column blocks per wavefront
    constexpr int HPW = WC >= D ? WC / D : 1;      // heads per wavefront
    constexpr int CPH = NCB / HPW;                 // column blocks per head inside a wavefront
    // op tiles double-buffered and filled by direct global -> LDS loads,
    // rows unpadded with their 16-byte chunks XOR-swizzled (see ys_off);
    // fp32 rows at F = 256 take 2 x 64 KiB (one block per CU)
    typedef typename std::conditional<BF, uint16_t, float>::type YT;
    // (two separate arrays per buffer, so that the compiler sees that the
    // loads into one buffer do not alias the reads of the other)
    __shared__ __attribute__((aligned(16))) YT Ys0[kOpTile * F], Ys1[kOpTile * F];
    __shared__ __attribute__((aligned(16))) uint64_t MK0[kOpTile][2], MK1[kOpTile][2];   // (present, bit) per op
    __shared__ float pb0[kOpTile][2][K], pb1[kOpTile][2][K];
    __shared__ int mxk[64][K];
    __shared__ float qd[64][K], mrun[64][K];
    __shared__ float US[F], CS[F];

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

    // element (op u, column col) of a tile: 16-byte chunk col / EPC of
    // row u (EPC elements per chunk), XORed with ((u / 4) % 4) times the
    // chunks that sixteen lanes read, so that the four lane groups of a
    // message read (rows 4 apart) fall on different banks
    constexpr int EPC = 16 / sizeof(YT), GSW = 16 / EPC;
    auto ys_off = [](int u, int col) {
        return u * F + ((((col / EPC) ^ (GSW * ((u >> 2) & 3))) * EPC) | (col % EPC));
    };
    // tile t into the given buffers, all by direct loads into LDS: the op
    // rows' second halves, the masks and the raw attention terms (rows
    // past the tile repeat op u0: their weights are zero)
    auto stage = [&](int32_t t, auto &ys, auto &mk, auto &pbn) {
        const int32_t u0 = A.tiles[3 * t], nu = A.tiles[3 * t + 1];
        const YT *Yr = static_cast<const YT *>(A.Y_op) + ((int64_t)r * A.n_op + u0) * 2 * F + F;
        constexpr int NI = kOpTile * F / EPC / 256;   // 16-byte chunks per thread
        const int wv = __builtin_amdgcn_readfirstlane(wave);   // (wave-uniform LDS addresses)
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int P = (wv * NI + i) * 64 + lane;   // physical chunk; the wave fills 1 KB
            const int u = P / (F / EPC), k = (P % (F / EPC)) ^ (GSW * ((u >> 2) & 3));
            load_lds<16>(Yr + (int64_t)(u < nu ? u : 0) * 2 * F + EPC * k, &ys[(wv * NI + i) * 64 * EPC]);
        }
        if (wv == 0)
            load_lds<16>(om + 2 * (int64_t)(u0 + (lane < nu ? lane : 0)), &mk[0][0]);
        // an op's 2K attention terms (8K bytes) in PC-byte lanes
        constexpr int PC = 8 * K >= 16 ? 16 : 4, PCO = 8 * K / PC, PNI = kOpTile * PCO / 64;
#pragma unroll
        for (int j = 0; j < (PNI + 3) / 4; ++j) {
            const int i = wv + 4 * j;
            if (i >= PNI) break;
            const int P = i * 64 + lane, u = P / PCO;
            load_lds<PC>(Sop + (int64_t)(u0 + (u < nu ? u : 0)) * 4 * K + (P % PCO) * (PC / 4),
                         &pbn[0][0][0] + i * 64 * (PC / 4));
        }
    };
    stage(t0, Ys0, MK0, pb0);   // the first tile lands while the maxima are taken
    for (int i = tid; i < F; i += 256) {
        US[i] = A.U[(size_t)(F + i) * 2];
        CS[i] = A.cp[F + i];
    }
    for (int i = tid; i < 64 * K; i += 256) {
        const int j = i / K, h = i % K;
        qd[j][h] = j < Mg ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + 2 * K + h] * kLog2e : 0.f;
        mxk[j][h] = INT_MIN;
    }
    __syncthreads();
    {
        // (op, head) items of the block's tiles, which cover the contiguous
        // ops ub .. ue - 1; MB items per thread have their loads in flight
        // together before their LDS maxima are taken
        const int32_t ub = A.tiles[3 * t0], ue = A.tiles[3 * (t1 - 1)] + A.tiles[3 * (t1 - 1) + 1];
        const int32_t n_items = (ue - ub) * K;
        constexpr int MB = 4;
        for (int32_t base = tid; base < n_items; base += 256 * MB) {
            uint64_t prv[MB], btv[MB];
            float s0v[MB], s1v[MB];
#pragma unroll
            for (int q = 0; q < MB; ++q) {
                const int32_t i = base + 256 * q;
                const int64_t u = ub + (i < n_items ? i : 0) / K;
                const int h = i % K;
                prv[q] = i < n_items ? om[2 * u] : 0ull;
                btv[q] = om[2 * u + 1];
                s0v[q] = Sop[u * 4 * K + h];
                s1v[q] = Sop[u * 4 * K + K + h];
            }
#pragma unroll
            for (int q = 0; q < MB; ++q) {
                const int h = (base + 256 * q) % K;
                const int k0 = fkey(s0v[q]), k1 = fkey(s1v[q]);
                uint64_t pr = prv[q];
                while (pr) {
                    const int j = __builtin_ctzll(pr);
                    pr &= pr - 1;
                    atomicMax(&mxk[j][h], ((btv[q] >> j) & 1ull) ? k1 : k0);
                }
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
    float Uv[NCB], Cv[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const int col = cbase + cb * 16 + (lane & 15);
        Uv[cb] = US[col];
        Cv[cb] = CS[col];
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

    __syncthreads();   // the maxima are in place
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
    // tile t from the current buffers while tile t + 1 lands in the others
    auto run = [&](int32_t t, auto &ysc, auto &mkc, auto &pbc, auto &ysn, auto &mkn, auto &pbn) {
        const int32_t nu = A.tiles[3 * t + 1];
        if (t + 1 < t1) stage(t + 1, ysn, mkn, pbn);
            // sparse 16x16x64 bf16 products (smfmac_split3) over the exact
            // three-way splits of the fp32 attention weights and messages:
            // k = 2u + b over 32 ops per step.  A link carries one bit, so a
            // device row has at most one nonzero weight in each op's pair of
            // k (the 2:4 structure).  Lane group g = l / 16 gives the weights
            // of ops 8g .. 8g+7 of a step (value v at position 2 (v % 2) +
            // bit of its op pair's four k) and the messages of ops 4g .. 4g+3
            // and 16+4g .. 16+4g+3 (both bits).
#pragma unroll 1
            for (int ks = 0; ks < kOpTile / 32; ++ks) {
                const int ua = 32 * ks + 8 * (lane >> 4);
                const int ubm = 32 * ks + 4 * (lane >> 4);
                uint64_t prq[8], btq[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    // rows past the tile hold another op's masks: their presence
                    // is cleared (the loads stay unconditional: ua + q < 64)
                    const uint64_t p = mkc[ua + q][0], b = mkc[ua + q][1];
                    prq[q] = ua + q < nu ? p : 0ull;
                    btq[q] = b;
                }
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    float p0q[8], p1q[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        p0q[q] = pbc[ua + q][0][h0 + hh];
                        p1q[q] = pbc[ua + q][1][h0 + hh];
                    }
                    bf8 aop[4][3];
                    int idx[4];
#pragma unroll
                    for (int rb = 0; rb < 4; ++rb) {
                        if (rb < NRB) {
                            const int j = rb * 16 + (lane & 15);
                            unsigned w[3][4], sb = 0u;
#pragma unroll
                            for (int pr = 0; pr < 4; ++pr) {
                                float af2[2];
#pragma unroll
                                for (int e = 0; e < 2; ++e) {
                                    const int q = 2 * pr + e;
                                    // (device j's flags sit in the low mask word for rb < 2)
                                    const uint32_t pw = (uint32_t)(rb < 2 ? prq[q] : prq[q] >> 32);
                                    const uint32_t bw = (uint32_t)(rb < 2 ? btq[q] : btq[q] >> 32);
                                    const bool on = (pw >> (j & 31)) & 1u;
                                    const unsigned bit = (bw >> (j & 31)) & 1u;
                                    const float x = fmaf(bit ? p1q[q] : p0q[q], kLog2e, q2[rb][hh]);   // raw terms
                                    // (no link: exp2(-inf) = 0, without a branch)
                                    const float y = fmaxf(x, slope * x) - m2[rb][hh];
                                    af2[e] = __builtin_amdgcn_exp2f(on ? y : -INFINITY);
                                    zl[rb][hh] += af2[e];
                                    sb |= bit << (2 * q);
                                }
                                unsigned sp[3];
                                split3(af2[0], af2[1], sp);
#pragma unroll
                                for (int z = 0; z < 3; ++z) w[z][pr] = sp[z];
                            }
#pragma unroll
                            for (int z = 0; z < 3; ++z) aop[rb][z] = as_bf8(w[z][0], w[z][1], w[z][2], w[z][3]);
                            idx[rb] = (int)(0x8888u | sb);
                        }
                    }
#pragma unroll
                    for (int c2 = 0; c2 < CPH; ++c2) {
                        const int cb = hh * CPH + c2;
                        const int col = cbase + cb * 16 + (lane & 15);
                        unsigned w[3][8];
#pragma unroll
                        for (int q = 0; q < 8; ++q) {
                            const int u = ubm + (q < 4 ? q : 12 + q);
                            float yc;   // Y + c' (bf16 rows hold Y, fp32 rows Y + c')
                            if constexpr (BF) yc = bf2f(ysc[ys_off(u, col)]) + Cv[cb];
                            else yc = ysc[ys_off(u, col)];
                            unsigned sp[3];
                            split3(msg_act<ELU>(yc), msg_act<ELU>(yc + Uv[cb]), sp);
#pragma unroll
                            for (int z = 0; z < 3; ++z) w[z][q] = sp[z];
                        }
                        const bf16x16 bo[3] = {as_bf16x16(w[0]), as_bf16x16(w[1]), as_bf16x16(w[2])};
#pragma unroll
                        for (int rb = 0; rb < 4; ++rb)
                            if (rb < NRB) acc[rb][cb] = smfmac_split3(aop[rb], bo, idx[rb], acc[rb][cb]);
                    }
                }
            }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();   // the next tile is in place; this one is free again
    };
    __builtin_amdgcn_s_waitcnt(0);   // the first tile (staged before the maxima)
    __syncthreads();
    for (int32_t t = t0; t < t1; t += 2) {
        run(t, Ys0, MK0, pb0, Ys1, MK1, pb1);
        if (t + 1 < t1) run(t + 1, Ys1, MK1, pb1, Ys0, MK0, pb0);
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

// Op destinations of one 64-op tile of one candidate.
//  * op <- op: each 16-lane group streams the entries of four consecutive
//    tile rows (one contiguous CSR range, staged in LDS as (source, edge
//    feature) pairs, ECAP at a time) with EB neighbour rows always in
//    flight: a slot is refilled as soon as its row has been read, and the
//    refill reads only LDS, so the row loads never wait on each other.  Each
//    row's softmax is taken relative to its first logit (exact; a logit more
//    than 64 above the reference moves it up), so an entry costs one
//    multiply-add per channel for the aggregate.  Rows land in an LDS tile.
//  * op <- device: MFMA contraction of the attention weights (formed in
//    registers) with the device message table.
// Both parts are combined and each op row is written once.
template <int F, int K, bool BF, bool ELU = false>
__global__ void __launch_bounds__(256, (F >= 256 && K >= 8) ? 1 : 2) agg_op_tile(AggArgs A) {
    constexpr int D = F / K;
    constexpr int WC = F / 4;
    constexpr int NCB = WC / 16;
    constexpr int HPW = WC >= D ? WC / D : 1;
    constexpr int CPH = NCB / HPW;
    constexpr int CPL = F / 16;              // op<-op channels per lane
    constexpr int LPH = 16 / K;              // op<-op lanes per head (K <= 16 on this path)
    // neighbour rows in flight per 16-lane group (a slot holds CPL or CPL/2 words)
    constexpr int EB = BF ? (F >= 256 && K >= 8 ? 4 : 8) : (F >= 256 ? 2 : 4);
    constexpr int OS = F + 4;                // LDS tile row stride
    constexpr int ECAP = F >= 256 ? 512 : 192;   // op<-op entries staged in LDS per chunk (192 keeps
                                                 // four blocks per CU at f = 128)
    __shared__ __attribute__((aligned(16))) float Ot[kOpTile * OS];
    __shared__ uint64_t pres[kOpTile], bits[kOpTile];
    __shared__ float qo[kOpTile][K], mxS[kOpTile][K];
    // op<-op destination terms: staged per tile row where the LDS budget
    // allows (f = 256); smaller f keeps the group's four rows in registers
    // (four blocks per CU at f = 128 leave no room for the array)
    constexpr bool kQL = F >= 256;
    __shared__ float qoo[kQL ? kOpTile : 1][kQL ? K : 1];
    // op<-op per-channel constants (a log2 e, U_0, c') staged once per block
    // where the LDS budget allows (f = 256); smaller f loads them per lane
    constexpr bool kCS = F >= 256;
    __shared__ __attribute__((aligned(16))) float CA[kCS ? 3 : 1][kCS ? F : 4];
    __shared__ float P[64][2][K];
    __shared__ int32_t Erp[kOpTile + 1];
    __shared__ int2 Ecx[ECAP];             // staged entries: (source op, edge feature bits)
    __shared__ uint8_t Erw[ECAP];          // tile row of each staged entry

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // XCD-aware order: the hardware deals blocks to the XCDs round-robin; the
    // swizzle gives each XCD a contiguous run of (candidate, tile) pairs, so a
    // candidate's consecutive tiles -- whose op<-op sources overlap -- and its
    // device message table share one L2
    const uint32_t lb = xcd_swizzle(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
    const int32_t t = (int32_t)(lb % gridDim.x), r = (int32_t)(lb / gridDim.x);
    const int4 te0 = *reinterpret_cast<const int4 *>(A.tile_ext + 8 * (int64_t)t);
    const int4 te1 = *reinterpret_cast<const int4 *>(A.tile_ext + 8 * (int64_t)t + 4);
    const int32_t u0 = te0.x, nu = te0.y;
    const int32_t d0 = te1.y, Mg = te1.z;
    const float *xc = A.xcsr + (int64_t)r * A.s_xcsr;   // op<-op edge features in CSR order
    const float *Sop = A.Sop + (int64_t)r * A.n_op * 4 * K;
    const float slope = A.slope;
    const int cbase = wave * WC;
    const int h0 = cbase / D;

    // this lane's op<-op channels c0 .. c0+CPL-1 of the group's four rows
    const int c0 = (lane & 15) * CPL;
    const int gr0 = wave * 16 + (lane >> 4) * 4;   // the group's first tile row
    float qv[4];                                   // (kQL false) the group's op<-op destination terms
    if constexpr (!kQL) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            qv[i] = gr0 + i < nu ? Sop[(int64_t)(u0 + gr0 + i) * 4 * K + 3 * K + c0 / D] : 0.f;
    }
    float a[CPL], u0c[CPL], cpc[CPL];
    static_assert(!kCS || F == 256, "one staged constant per thread");
    float ca3[3];
    if constexpr (kCS) {
        ca3[0] = A.att_src[tid] * kLog2e;
        ca3[1] = A.U[(size_t)tid * 2];
        ca3[2] = BF ? A.cp[tid] : 0.f;
    }

    // ---- prologue: every global load is issued before the first LDS store
    // (the logits go to the exp2 domain: LeakyReLU commutes with log2(e) > 0)
    const int32_t eb = te0.w;
    const int32_t ntot = te1.x;                    // the tile's op<-op entries: one CSR range
    const int32_t ne = min(ntot, ECAP);
    {
        constexpr int NQ = (kOpTile * K + 255) / 256, NP = (64 * 2 * K + 255) / 256, NE = (ECAP + 255) / 256;
        int32_t rp0 = 0, rp1 = 0;
        uint64_t om0 = 0, om1 = 0;
        float q2v[NQ], q3v[NQ], pv[NP], exv[NE];
        int32_t ecv[NE];
        if (tid <= nu) rp0 = A.rp[0][u0 + tid] - eb;
        if (tid < nu) rp1 = A.rp[0][u0 + tid + 1] - eb;
        if (tid < nu) {
            const int64_t mi = 2 * ((int64_t)r * A.n_op + u0 + tid);
            om0 = A.omask[mi];
            om1 = A.omask[mi + 1];
        }
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            const int i = tid + 256 * k, u = i / K, h = i % K;
            const bool ok = i < kOpTile * K && u < nu;
            q2v[k] = ok ? Sop[(int64_t)(u0 + u) * 4 * K + 2 * K + h] : 0.f;   // op <- device
            q3v[k] = kQL && ok ? Sop[(int64_t)(u0 + u) * 4 * K + 3 * K + h] : 0.f;   // op <- op
        }
#pragma unroll
        for (int k = 0; k < NP; ++k) {
            const int i = tid + 256 * k, j = i / (2 * K), bh = i % (2 * K);
            pv[k] = (i < 64 * 2 * K && j < Mg) ? A.Sdev[((int64_t)r * A.n_dev + d0 + j) * 4 * K + bh] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < NE; ++k) {
            const int i = tid + 256 * k;
            ecv[k] = i < ne ? A.col[0][eb + i] : 0;
            exv[k] = i < ne ? xc[eb + i] : 0.f;
        }
        if (tid <= nu) Erp[tid] = rp0;
        if (tid < kOpTile) { pres[tid] = om0; bits[tid] = om1; }
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            const int i = tid + 256 * k;
            if (i < kOpTile * K) {
                qo[i / K][i % K] = q2v[k] * kLog2e;
                if constexpr (kQL) qoo[i / K][i % K] = q3v[k] * kLog2e;
            }
        }
#pragma unroll
        for (int k = 0; k < NP; ++k) {
            const int i = tid + 256 * k;
            if (i < 64 * 2 * K) P[i / (2 * K)][(i % (2 * K)) / K][i % K] = pv[k] * kLog2e;
        }
#pragma unroll
        for (int k = 0; k < NE; ++k) {
            const int i = tid + 256 * k;
            if (i < ne) Ecx[i] = int2{ecv[k], __float_as_int(exv[k])};
        }
        if (tid < nu)
            for (int32_t i = rp0; i < min(rp1, ECAP); ++i) Erw[i] = (uint8_t)tid;
        if constexpr (kCS) {
#pragma unroll
            for (int z = 0; z < 3; ++z) CA[z][tid] = ca3[z];
        }
    }
    __syncthreads();
    // op <- device softmax maxima (LeakyReLU of the largest pre-activation)
    for (int i = tid; i < kOpTile * K; i += 256) {
        const int u = i / K, h = i % K;
        uint64_t pr = pres[u];
        const uint64_t bt = bits[u];
        float mx = -INFINITY;
        while (pr) {   // four linked devices per round, their LDS reads issued together
            float v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int j = pr ? __builtin_ctzll(pr) : 0;
                v[q] = pr ? P[j][(bt >> j) & 1ull][h] : -INFINITY;
                pr &= pr - 1;
            }
            mx = fmaxf(mx, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
        }
        const float x = mx + qo[u][h];
        mxS[u][h] = mx == -INFINITY ? -INFINITY : fmaxf(x, slope * x);
    }

    // ---- op <- op into the LDS tile (gamma_same applied)
    {
        const int hd = c0 / D;                          // this lane's head
        // the candidate's relation transforms (a wave-uniform base; a row's
        // offset from it fits 32 bits, which the host checks)
        const void *Yc = static_cast<const char *>(A.Y_op) + (size_t)r * A.n_op * 2 * F * (BF ? 2 : 4);
        if constexpr (kCS) {
#pragma unroll
            for (int c = 0; c < CPL; c += 4) {
                const float4 x = *reinterpret_cast<const float4 *>(&CA[0][c0 + c]);
                const float4 y = *reinterpret_cast<const float4 *>(&CA[1][c0 + c]);
                const float4 z = *reinterpret_cast<const float4 *>(&CA[2][c0 + c]);
                a[c] = x.x; a[c + 1] = x.y; a[c + 2] = x.z; a[c + 3] = x.w;
                u0c[c] = y.x; u0c[c + 1] = y.y; u0c[c + 2] = y.z; u0c[c + 3] = y.w;
                cpc[c] = z.x; cpc[c + 1] = z.y; cpc[c + 2] = z.z; cpc[c + 3] = z.w;
            }
        } else {
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                a[c] = A.att_src[c0 + c] * kLog2e;
                u0c[c] = A.U[(size_t)(c0 + c) * 2];
                cpc[c] = BF ? A.cp[c0 + c] : 0.f;
            }
        }
        // the group's entries (rows >= nu are empty)
        const int32_t ebeg = Erp[min(gr0, nu)], eend = Erp[min(gr0 + 4, nu)];
        if constexpr (!kQL) {
#pragma unroll
            for (int i = 0; i < 4; ++i) qv[i] *= kLog2e;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (gr0 + i < nu)
                for (int c = 0; c < CPL; ++c) Ot[(gr0 + i) * OS + c0 + c] = 0.f;   // rows without entries stay zero
        const float gs = A.g_same;
        int ri = -1;                  // row being accumulated (-1: none yet)
        float mref = 0.f, den = 0.f, acc[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
        auto finish = [&]() {
            const float inv = gs * __builtin_amdgcn_rcpf(den);
#pragma unroll
            for (int c = 0; c < CPL; ++c) Ot[ri * OS + c0 + c] = acc[c] * inv;
        };
        for (int32_t cb0 = 0; cb0 < ntot; cb0 += ECAP) {
            if (cb0 > 0) {   // next chunk of the tile's entries (block-uniform)
                __syncthreads();
                const int32_t n = min(ntot - cb0, ECAP);
                for (int i = tid; i < n; i += 256) {
                    Ecx[i] = int2{A.col[0][eb + cb0 + i], __float_as_int(xc[eb + cb0 + i])};
                }
                if (tid < nu)
                    for (int32_t i = max(Erp[tid], cb0); i < min(Erp[tid + 1], cb0 + n); ++i)
                        Erw[i - cb0] = (uint8_t)tid;
                __syncthreads();
            }
            // the group's entries of this chunk, in chunk-local indices
            const int32_t lo = max(ebeg, cb0) - cb0, hi = min(eend, cb0 + ECAP) - cb0;
            const int32_t hm = max(hi - 1, 0);
            // two halves of EB / 2 row slots: while one half is consumed the
            // other half's rows are in flight; a half is refilled as a whole
            // right after it has been consumed (past hi a slot is refilled
            // with the tile's first row under the group's last entry's tile
            // row; the last loop round consumes such slots at weight 0)
            constexpr int HB = EB / 2;
            RowRaw<CPL, BF> sa[HB], sb[HB];
            float xa[HB], xb[HB];
            int la[HB], lb2[HB];
            auto fetch = [&](RowRaw<CPL, BF> &sl, float &xv, int &rl, int32_t le) {
                const int32_t lc = min(le, hm);
                const int2 cx = Ecx[lc];
                rl = (int)Erw[lc];                    // past hi: the row of the group's last entry
                xv = __int_as_float(cx.y);
                const int32_t v = le < hi ? cx.x : u0;
                sl.load32(Yc, ((uint32_t)v * (2 * F) + c0) * (BF ? 2u : 4u));
            };
            auto consume = [&](const RowRaw<CPL, BF> &sl, float xv, int rl, int32_t e) {
                float m[CPL];
                float part = 0.f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    // fp32 rows hold Y + c'; bf16 rows hold Y and get the edge term U x + c' whole
                    const float z = BF ? sl.get(c) + fmaf(u0c[c], xv, cpc[c]) : fmaf(u0c[c], xv, sl.get(c));
                    m[c] = msg_act<ELU>(z);
                    part = fmaf(a[c], m[c], part);
                }
                float qd;   // the destination term of row rl
                if constexpr (kQL) qd = qoo[rl][hd];
                else {
                    const int i = rl - gr0;
                    const float qa = (i & 1) ? qv[1] : qv[0], qb = (i & 1) ? qv[3] : qv[2];
                    qd = (i & 2) ? qb : qa;
                }
                const float sv = row_sum<LPH>(part) + qd;
                // a slot past hi gets weight exp2(-inf) = 0 (its row is the one
                // in progress, so it neither starts nor finishes a row)
                const float s2 = fmaxf(sv, slope * sv) + (e < hi ? 0.f : -INFINITY);
                if (rl != ri) {   // first entry of row rl: finish row ri
                    if (ri >= 0) finish();
                    ri = rl;
                    mref = s2;
                    den = 0.f;
#pragma unroll
                    for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
                }
                float d = s2 - mref;
                if (d > 64.f) {   // keep the weights finite: move the reference up
                    const float sc = __builtin_amdgcn_exp2f(-d);
                    den *= sc;
#pragma unroll
                    for (int c = 0; c < CPL; ++c) acc[c] *= sc;
                    mref = s2;
                    d = 0.f;
                }
                const float p = __builtin_amdgcn_exp2f(d);
                den += p;
#pragma unroll
                for (int c = 0; c < CPL; ++c) acc[c] = fmaf(p, m[c], acc[c]);
            };
#pragma unroll
            for (int s = 0; s < HB; ++s) fetch(sa[s], xa[s], la[s], lo + s);
#pragma unroll
            for (int s = 0; s < HB; ++s) fetch(sb[s], xb[s], lb2[s], lo + HB + s);
            for (int32_t base = lo; base < hi; base += EB) {
#pragma unroll
                for (int s = 0; s < HB; ++s) consume(sa[s], xa[s], la[s], base + s);
#pragma unroll
                for (int s = 0; s < HB; ++s) fetch(sa[s], xa[s], la[s], base + EB + s);
#pragma unroll
                for (int s = 0; s < HB; ++s) consume(sb[s], xb[s], lb2[s], base + HB + s);
#pragma unroll
                for (int s = 0; s < HB; ++s) fetch(sb[s], xb[s], lb2[s], base + EB + HB + s);
            }
        }
        if (ri >= 0) finish();
    }

    // ---- op <- device on the matrix cores.  bf16, and fp32 at F = 256:
    // sparse 16x16x64 bf16 products (smfmac_split3) over the exact three-way
    // splits of the fp32 attention weights and message table: k = 2j + b
    // over 32 devices per step.  An
    // (op, device) link carries one bit, so each device's pair of k holds at
    // most one nonzero weight: the 2:4 structure the sparse products take.
    // Lane group g = l / 16 gives the weights of devices 8g .. 8g+7 of a step
    // (value v at position 2 (v % 2) + bit of its device pair's four k) and
    // the table entries of devices 4g .. 4g+3 and 16+4g .. 16+4g+3 (both
    // bits).  The tile's four row blocks go in two halves of two (halving the
    // registers that hold weights and accumulators); per step the weights of
    // one head are formed first, then the table parts stream one 16-column
    // block at a time, the next block's loads in flight while the current one
    // is used.  The first table loads are issued before the barrier, so their
    // latency overlaps the slowest op<-op group.
    constexpr bool kSparseDev = BF || F >= 256;   // (fp32 at F <= 128: see below)
    if constexpr (kSparseDev) {
        // table words by 32-bit byte offsets from the table's (wave-uniform)
        // start; the host checks that the table fits 4 GiB.  Devices past the
        // group read its last device (their weights are zero).
        const char *Tb = reinterpret_cast<const char *>(A.T);
        const uint32_t tpart = (uint32_t)A.R * (uint32_t)A.n_dev * F * 4u;   // bytes between the three parts
        const uint32_t trow = ((uint32_t)r * (uint32_t)A.n_dev + (uint32_t)d0) * F * 4u + (cbase + (lane & 15)) * 4u;
        const int ksteps = (Mg + 31) / 32;   // <= 2: a tile group holds at most 64 devices
        // (the part and column block go into a wave-uniform base, so that a
        // load needs only the lane's row offset)
        auto load_b = [&](int ks, int cb, bf16x16 (&bo)[3]) {
            const int jb = 32 * ks + 4 * (lane >> 4);
            uint32_t off[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) off[q] = trow + (uint32_t)(min(jb + (q < 4 ? q : 12 + q), Mg - 1) * F) * 4u;
#pragma unroll
            for (int z = 0; z < 3; ++z) {
                const char *bz = Tb + (size_t)z * tpart + cb * 64;
                unsigned w[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) w[q] = *reinterpret_cast<const unsigned *>(bz + off[q]);
                bo[z] = as_bf16x16(w);
            }
        };
        bf16x16 bops[2][3];
        if (ksteps > 0) load_b(0, 0, bops[0]);
        __syncthreads();
#pragma unroll 1
        for (int half = 0; half < 2; ++half) {
            f4 acc[2][NCB];
            float zl[2][HPW], q2[2][HPW], m2[2][HPW];
            uint64_t prs[2], bts[2];
#pragma unroll
            for (int b2 = 0; b2 < 2; ++b2) {
                const int u = (2 * half + b2) * 16 + (lane & 15);
                prs[b2] = pres[u];
                bts[b2] = bits[u];
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    q2[b2][hh] = qo[u][h0 + hh];
                    m2[b2][hh] = mxS[u][h0 + hh];
                    zl[b2][hh] = 0.f;
                }
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) acc[b2][cb] = f4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll 1
            for (int ks = 0; ks < ksteps; ++ks) {
                const int jb = 32 * ks + 8 * (lane >> 4);
                unsigned on8[2], bit8[2];
                int idx[2];
#pragma unroll
                for (int b2 = 0; b2 < 2; ++b2) {
                    // the lane's eight presence and bit flags (never set for jb + q >= Mg)
                    on8[b2] = (unsigned)(prs[b2] >> jb) & 0xffu;
                    bit8[b2] = (unsigned)(bts[b2] >> jb) & 0xffu;
                    // position of value q: 2 (q % 2) + bit, in bits 2q+1..2q
                    unsigned sb = (bit8[b2] | (bit8[b2] << 4)) & 0x0f0fu;
                    sb = (sb | (sb << 2)) & 0x3333u;
                    sb = (sb | (sb << 1)) & 0x5555u;
                    idx[b2] = (int)(0x8888u | sb);
                }
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    float p0q[8], p1q[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        p0q[q] = P[jb + q][0][h0 + hh];
                        p1q[q] = P[jb + q][1][h0 + hh];
                    }
                    bf8 aop[2][3];
#pragma unroll
                    for (int b2 = 0; b2 < 2; ++b2) {
                        unsigned w[3][4];
#pragma unroll
                        for (int pr = 0; pr < 4; ++pr) {
                            float af2[2];
#pragma unroll
                            for (int e = 0; e < 2; ++e) {
                                const int q = 2 * pr + e;
                                const bool on = (on8[b2] >> q) & 1u;
                                const bool bit = (bit8[b2] >> q) & 1u;
                                const float x = (bit ? p1q[q] : p0q[q]) + q2[b2][hh];
                                const float y = fmaxf(x, slope * x) - m2[b2][hh];
                                af2[e] = __builtin_amdgcn_exp2f(on ? y : -INFINITY);   // (no link: 0)
                                zl[b2][hh] += af2[e];
                            }
                            unsigned sp[3];
                            split3(af2[0], af2[1], sp);
#pragma unroll
                            for (int z = 0; z < 3; ++z) w[z][pr] = sp[z];
                        }
#pragma unroll
                        for (int z = 0; z < 3; ++z) aop[b2][z] = as_bf8(w[z][0], w[z][1], w[z][2], w[z][3]);
                    }
#pragma unroll
                    for (int c2 = 0; c2 < CPH; ++c2) {
                        const int cb = hh * CPH + c2;
                        // the next (step, column block) pair's table parts
                        // (after the first half's last pair: the first pair
                        // again), into the buffer this pair does not use; with
                        // one column block (NCB = 1) every pair uses bops[0], so
                        // the next step's parts are loaded after its products
                        auto prefetch = [&]() {
                            if (cb + 1 < NCB) load_b(ks, cb + 1, bops[(cb + 1) & 1]);
                            else if (ks + 1 < ksteps) load_b(ks + 1, 0, bops[0]);
                            else if (half == 0) load_b(0, 0, bops[0]);
                        };
                        constexpr bool kAlt = NCB % 2 == 0;   // consecutive pairs alternate buffers
                        if (kAlt || cb + 1 < NCB) prefetch();
#pragma unroll
                        for (int b2 = 0; b2 < 2; ++b2)
                            acc[b2][cb] = smfmac_split3(aop[b2], bops[cb & 1], idx[b2], acc[b2][cb]);
                        if (!kAlt && cb + 1 == NCB) prefetch();
                    }
                }
            }
            // softmax sums of op row rb*16 + l%16 are spread over lanes l,
            // l+16, l+32, l+48; the output row of register v in lane l is
            // rb*16 + 4(l/16) + v; the op<-device part is added into the LDS
            // tile in place (each (row, column) belongs to one lane)
#pragma unroll
            for (int b2 = 0; b2 < 2; ++b2) {
                const int rb = 2 * half + b2;
                float scale[HPW][4];
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) {
                    float z = zl[b2][hh];
                    z += __shfl_xor(z, 16, 64);
                    z += __shfl_xor(z, 32, 64);
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float zv = __shfl(z, 4 * (lane >> 4) + v, 64);
                        scale[hh][v] = zv > 0.f ? A.g_cross * __builtin_amdgcn_rcpf(zv) : 0.f;
                    }
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int u = rb * 16 + 4 * (lane >> 4) + v;
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) {
                        const int col = cbase + cb * 16 + (lane & 15);
                        Ot[u * OS + col] = fmaf(scale[cb / CPH][v], acc[b2][cb][v], Ot[u * OS + col]);
                    }
                }
            }
        }
    } else {
        // fp32 at F <= 128: fp32 16x16x4 products over the fp32 message table
        // [rows][2][F], k = 4 (device, bit) pairs per step, two devices per
        // step (half of each step's k is zero, but the narrower register
        // footprint keeps four blocks per CU, which measured faster here than
        // the sparse products at two); the table loads of SB steps are issued
        // together
        constexpr int SB = 4;
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
        float bv[SB][NCB];
        auto load_batch = [&](int s0) {
#pragma unroll
            for (int k = 0; k < SB; ++k) {
                const int j = 2 * (s0 + k) + (lane >> 5);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    bv[k][cb] = j < Mg ? Tb[((int64_t)j * 2 + b) * F + cbase + cb * 16 + (lane & 15)] : 0.f;
            }
        };
        load_batch(0);
        __syncthreads();
        // per-lane constants of the lane's op rows u = rb*16 + l%16
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
        for (int s0 = 0; s0 < steps; s0 += SB) {
            float bc[SB][NCB];
#pragma unroll
            for (int k = 0; k < SB; ++k)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) bc[k][cb] = bv[k][cb];
            if (s0 + SB < steps) load_batch(s0 + SB);
#pragma unroll
            for (int k = 0; k < SB; ++k) {
                const int j = 2 * (s0 + k) + (lane >> 5);
                if (2 * (s0 + k) >= Mg) break;
                const bool jok = j < Mg;
                float pj[HPW];
#pragma unroll
                for (int hh = 0; hh < HPW; ++hh) pj[hh] = P[j][b][h0 + hh];
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const bool on = jok && ((prs[rb] >> j) & 1ull) && ((int)((bts[rb] >> j) & 1ull) == b);
#pragma unroll
                    for (int hh = 0; hh < HPW; ++hh) {
                        const float x = pj[hh] + q2[rb][hh];
                        const float y = fmaxf(x, slope * x) - m2[rb][hh];
                        const float af = __builtin_amdgcn_exp2f(on ? y : -INFINITY);   // (no link: 0)
                        zl[rb][hh] += af;
#pragma unroll
                        for (int c2 = 0; c2 < CPH; ++c2)
                            acc[rb][hh * CPH + c2] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                af, bc[k][hh * CPH + c2], acc[rb][hh * CPH + c2], 0, 0, 0);
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
                    scale[hh][v] = zv > 0.f ? A.g_cross * __builtin_amdgcn_rcpf(zv) : 0.f;
                }
            }
            // the op<-device part is added into the LDS tile in place (each
            // (row, column) belongs to one lane)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int u = rb * 16 + 4 * (lane >> 4) + v;
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const int col = cbase + cb * 16 + (lane & 15);
                    Ot[u * OS + col] = fmaf(scale[cb / CPH][v], acc[rb][cb][v], Ot[u * OS + col]);
                }
            }
        }
    }
    __syncthreads();
    // whole rows leave in 16-byte stores: 4 floats (last layer) or 8 bf16
    if (A.out_f32) {
        float *out = static_cast<float *>(A.H_op) + ((int64_t)r * A.n_op + u0) * F;
        for (int idx = tid; idx < nu * (F / 4); idx += 256) {
            const int u = idx / (F / 4), c = (idx % (F / 4)) * 4;
            *reinterpret_cast<float4 *>(out + (int64_t)u * F + c) = *reinterpret_cast<const float4 *>(&Ot[u * OS + c]);
        }
    } else {
        uint16_t *out = static_cast<uint16_t *>(A.H_op) + ((int64_t)r * A.n_op + u0) * F;
        for (int idx = tid; idx < nu * (F / 8); idx += 256) {
            const int u = idx / (F / 8), c = (idx % (F / 8)) * 8;
            const float4 a = *reinterpret_cast<const float4 *>(&Ot[u * OS + c]);
            const float4 b = *reinterpret_cast<const float4 *>(&Ot[u * OS + c + 4]);
            *reinterpret_cast<u4v *>(out + (int64_t)u * F + c) =
                u4v{pack_bf2(a.x, a.y), pack_bf2(a.z, a.w), pack_bf2(b.x, b.y), pack_bf2(b.z, b.w)};
        }
    }
}

template <int F, int K, bool BF, bool ELU = false>
void launch_mfma(const AggArgs &A, hipStream_t st) {
    const int64_t op_waves = (int64_t)A.R * A.n_op;
    const int64_t dev_waves = (int64_t)A.R * A.n_dev;
    const dim3 tiles((unsigned)A.n_tiles, (unsigned)A.R);
    const dim3 groups((unsigned)A.n_groups, (unsigned)A.R);
    if (!A.prep_done) {
        prof_begin(TAG_STAGE_DEV_PREP, st);
        prep_rows<F, K, BF, ELU><<<(unsigned)((op_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A, 0);
        prep_rows<F, K, BF, ELU><<<(unsigned)((dev_waves + kWaves - 1) / kWaves), 256, 0, st>>>(A, 1);
        prof_end(TAG_STAGE_DEV_PREP, st);
    }
    prof_begin(TAG_STAGE_AGG_DEV_OP, st);
    agg_b2<F, K, BF, ELU><<<groups, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_DEV_OP, st);
    prof_begin(TAG_STAGE_AGG_OP_DEV, st);
    agg_op_tile<F, K, BF, ELU><<<tiles, 256, 0, st>>>(A);
    prof_end(TAG_STAGE_AGG_OP_DEV, st);
}

template <int F, bool BF, bool ELU = false>
bool dispatch_mfma_heads(int K, const AggArgs &A, hipStream_t st) {
    switch (K) {
        case 1: launch_mfma<F, 1, BF, ELU>(A, st); return true;
        case 2: launch_mfma<F, 2, BF, ELU>(A, st); return true;
        case 4: launch_mfma<F, 4, BF, ELU>(A, st); return true;
        case 8: if (F / 8 >= 16) { launch_mfma<F, (F / 8 >= 16 ? 8 : 4), BF, ELU>(A, st); return true; } return false;
        case 16: if (F / 16 >= 16) { launch_mfma<F, (F / 16 >= 16 ? 16 : 4), BF, ELU>(A, st); return true; } return false;
        default: return false;
    }
}

}  // namespace

// heads of at least 16 channels, at most 16 heads, and a candidate's relation
// transforms within 32-bit byte offsets of its base (the op<-op gathers)
bool mfma_path_supported(int F, int K, int64_t n_op, int64_t R, int64_t n_dev, int esz) {
    return K >= 1 && F / K >= 16 && K <= 16 && n_op * 2 * F * esz < (int64_t(1) << 32) &&
           R * n_dev * F * 12 < (int64_t(1) << 32);
}

void launch_prep_tiles_x(const AggArgs &A, int64_t nnz0, hipStream_t st) {
    const int32_t xrep = A.s_xcsr ? A.R : 1;
    const int64_t n = (int64_t)A.n_tiles + (int64_t)xrep * nnz0;
    if (n == 0) return;
    const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 4096);
    prep_tiles_x<<<blocks, 256, 0, st>>>(A, nnz0, xrep);
}

void launch_pack_masks(const AggArgs &A, hipStream_t st) {
    pack_op_masks<<<dim3((unsigned)A.n_tiles, (unsigned)((A.R + kMaskCands - 1) / kMaskCands)), 256, 0, st>>>(A);
}

bool launch_agg_mfma(int F, int K, bool bf, const AggArgs &A, hipStream_t st) {
    if (!mfma_path_supported(F, K, A.n_op, A.R, A.n_dev, bf ? 2 : 4)) return false;
    if (A.elu) {   // the ELU variant runs in fp32
        if (bf) return false;
        if (F == 64) return dispatch_mfma_heads<64, false, true>(K, A, st);
        if (F == 128) return dispatch_mfma_heads<128, false, true>(K, A, st);
        return dispatch_mfma_heads<256, false, true>(K, A, st);
    }
    if (F == 64) return bf ? dispatch_mfma_heads<64, true>(K, A, st) : dispatch_mfma_heads<64, false>(K, A, st);
    if (F == 128) return bf ? dispatch_mfma_heads<128, true>(K, A, st) : dispatch_mfma_heads<128, false>(K, A, st);
    return bf ? dispatch_mfma_heads<256, true>(K, A, st) : dispatch_mfma_heads<256, false>(K, A, st);
}

}  // namespace tag
