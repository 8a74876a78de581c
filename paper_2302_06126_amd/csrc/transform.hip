// Relation transforms (Section 4.2.1 layer equation, the W^h h part):
//   op rows:     Y = H [W^h_oo ; W^h_od]^T     device rows: Y = H [W^h_dd ; W^h_od]^T
// The fp32 kernel stores Y with the folded bias c' of each relation added
// (Y + c' starts every message ReLU(Y + c' + U x)); the bf16 kernel stores
// bf16(Y) alone, the rounded product of the bf16 variant, and the message
// kernels add c' in fp32.  The attention destination terms use Y itself.
// One launch covers both row sets of a layer, in 128 x 128 block tiles whose
// k-chunks pass through LDS with the next chunk's global loads in flight
// while the current one feeds the matrix cores.  The 1-D block order is
// XCD-swizzled so the column tiles of one row tile (which re-read the same
// rows of H) land on the same XCD and share its L2.
//
// Both kernels run on 16x16x32 bf16 MFMAs; the fp32 kernel contracts exact
// three-way bf16 splits of its fp32 operands.  Operand layout: lane l
// supplies row/column l % 16 of A/B and the 8-wide k-slice l / 16; result
// register v of lane l holds row 4 (l / 16) + v, column l % 16.  The fp32
// kernel feeds the weights as the first operand and the hidden rows as the
// second, so its result blocks are tiles of Y^T (see store_rows); the bf16
// kernel takes Y = H W^T directly (store_tile_bf16).
#include "tag_internal.hpp"
#include "transform.hpp"

namespace tag {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef u4v u4;

constexpr int BM = 128, BN = 128;
constexpr int kBkBf16 = 32;   // k-chunk of the bf16 kernel (a multiple of 32)

struct Tile {
    int sd;
    int64_t m0;
    int n0;
};

template <int TM = BM>
__device__ __forceinline__ Tile tile_of(const GemmArgs &G) {
    const uint32_t lb = xcd_swizzle(blockIdx.x, gridDim.x);
    const int ct = 2 * G.F / BN;
    const int64_t rt = lb / ct;
    Tile t;
    t.n0 = (int)(lb % ct) * BN;
    t.sd = rt < G.tiles0 ? 0 : 1;
    t.m0 = (rt - (t.sd ? G.tiles0 : 0)) * TM;
    return t;
}

// Sums of 4 row values over the 16 lanes of a lane group: after two exchange
// steps and a two-step butterfly, lanes k with k / 4 = v hold the total of row v.
__device__ __forceinline__ float xpose_sum4(const float (&v)[4], int lane) {
    const bool b3 = lane & 8, b2 = lane & 4;
    float w2[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const float keep = b3 ? v[i + 2] : v[i], send = b3 ? v[i] : v[i + 2];
        w2[i] = keep + __shfl_xor(send, 8, 64);
    }
    float w = (b2 ? w2[1] : w2[0]) + __shfl_xor(b2 ? w2[0] : w2[1], 4, 64);
    w += __shfl_xor(w, 2, 64);
    w += __shfl_xor(w, 1, 64);
    return w;
}

// Epilogue of the bf16 kernel, whose products are taken as Y = H W^T: result
// register v of block (i, j) in lane l holds row 16 i + 4 (l / 16) + v and
// column 16 j + l % 16 of the wavefront's 64 x 64 tile.  The stored row is
// bf16(W^h h) without c'; the attention terms and the device message table
// use that rounded value plus c' in fp32, and the table holds the exact
// three-way bf16 splits of the fp32 messages (the operands of the op <-
// device contraction).  The k loop's LDS buffers are reused: the block's
// per-column constants are staged first (so no global load follows a store),
// the rounded 128 x 128 tile is written to LDS, and whole rows leave in
// 16-byte stores.
constexpr int kTileStride = BN + 8;   // bf16 elements per LDS tile row (272 bytes)

template <int JPH, int MB>
__device__ void store_tile_bf16(const GemmArgs &G, const Tile &t, int wm, int wn, int lane, const f4 (&acc)[4][4],
                                uint16_t *sm) {
    constexpr int NT = 2 * MB;                     // threads per block
    constexpr int HW = JPH > 0 ? 4 / JPH : 1;      // heads per wavefront
    const GemmPrep &P = G.prep;
    const int64_t rows = t.sd ? G.side[1].rows : G.side[0].rows;
    const int F = G.F, K = P.K, D = 16 * (JPH > 0 ? JPH : 1);
    const int64_t ldy = 2 * F;
    uint16_t *Yp = static_cast<uint16_t *>(t.sd ? G.side[1].Y : G.side[0].Y);
    uint16_t *tile = sm;                                            // [MB][kTileStride]
    float *cst = reinterpret_cast<float *>(sm + MB * kTileStride);  // [4][BN]: c', a, a~, U
    const int tid = threadIdx.x;
    if (tid < BN) {   // constants of block column n0 + tid (same-type half: a = U = 0)
        const int n = t.n0 + tid;
        const bool od = n >= F;
        const int c = od ? n - F : n;
        cst[tid] = od ? P.cp_od[c] : P.cp_same[t.sd][c];
        cst[BN + tid] = (JPH > 0 && od) ? P.a_od[c] : 0.f;
        cst[2 * BN + tid] = JPH > 0 ? (od ? P.ad_od[c] : P.ad_same[t.sd][c]) : 0.f;
        cst[3 * BN + tid] = (JPH > 0 && od) ? P.u_od[2 * c] : 0.f;
    }
    __syncthreads();
    const int col0 = t.n0 + wn * 64;
    const bool od = col0 >= F;
    const int cw = od ? col0 - F : col0;           // first channel of the relation
    const int k = lane & 15;
    const int rt0 = wm * 64 + 4 * (lane >> 4);     // this lane's first row in the block tile
    const int64_t rbase = t.m0 + rt0;
    const bool writer = (k & 3) == 0;
    const bool dev_od = od && t.sd == 1;
    float *S = P.S[t.sd];
    float c3[4], c1[4], c2[4], c4[4];   // c', a, a~, U of the lane's four columns
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int cl = wn * 64 + j * 16 + k;
        c3[j] = cst[cl]; c1[j] = cst[BN + cl]; c2[j] = cst[2 * BN + cl]; c4[j] = cst[3 * BN + cl];
    }
    unsigned *Tu = reinterpret_cast<unsigned *>(P.T);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float yv[4][4];   // [j][v]: the rounded product W^h h as stored
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int v = 0; v < 4; v += 2) {
                const unsigned pr = pack_bf2(acc[i][j][v], acc[i][j][v + 1]);
                yv[j][v] = __uint_as_float(pr << 16);
                yv[j][v + 1] = __uint_as_float(pr & 0xffff0000u);
                const int cl = wn * 64 + j * 16 + k;
                tile[(rt0 + i * 16 + v) * kTileStride + cl] = static_cast<uint16_t>(pr & 0xffffu);
                tile[(rt0 + i * 16 + v + 1) * kTileStride + cl] = static_cast<uint16_t>(pr >> 16);
            }
        }
        // device message rows, bit 0 / 1, as exact bf16 splits (the table exists
        // only with the attention-term epilogue, JPH > 0)
        if (JPH > 0 && dev_od) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t rv = rbase + i * 16 + v;
                if (rv >= rows) continue;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float ys = yv[j][v] + c3[j];
                    unsigned sp[3];
                    split3(fmaxf(ys, 0.f), fmaxf(ys + c4[j], 0.f), sp);
#pragma unroll
                    for (int q = 0; q < 3; ++q) Tu[q * rows * F + rv * F + cw + j * 16 + k] = sp[q];
                }
            }
        }
        if constexpr (JPH == 0) continue;
        const int64_t row = rbase + i * 16 + (k >> 2);   // row of this lane's totals
#pragma unroll
        for (int hw = 0; hw < HW; ++hw) {
            const int h = cw / D + hw;
            if (od) {
                float p0[4], p1[4], q[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    p0[v] = p1[v] = q[v] = 0.f;
#pragma unroll
                    for (int jj = 0; jj < JPH; ++jj) {
                        const int j = hw * JPH + jj;
                        const float ys = yv[j][v] + c3[j];
                        p0[v] = fmaf(c1[j], fmaxf(ys, 0.f), p0[v]);
                        p1[v] = fmaf(c1[j], fmaxf(ys + c4[j], 0.f), p1[v]);
                        q[v] = fmaf(c2[j], yv[j][v], q[v]);
                    }
                }
                const float s0 = xpose_sum4(p0, lane), s1 = xpose_sum4(p1, lane), s2 = xpose_sum4(q, lane);
                if (writer && row < rows) {
                    S[row * 4 * K + h] = s0;
                    S[row * 4 * K + K + h] = s1;
                    S[row * 4 * K + 2 * K + h] = s2;
                }
            } else {
                float q[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    q[v] = 0.f;
#pragma unroll
                    for (int jj = 0; jj < JPH; ++jj) q[v] = fmaf(c2[hw * JPH + jj], yv[hw * JPH + jj][v], q[v]);
                }
                const float s2 = xpose_sum4(q, lane);
                if (writer && row < rows) S[row * 4 * K + 3 * K + h] = s2;
            }
        }
    }
    __syncthreads();
    // whole rows of the block's 128 columns: 16 threads per row, 16 bytes each
#pragma unroll
    for (int it = 0; it < MB * BN / 8 / NT; ++it) {
        const int idx = it * NT + tid;
        const int rr = idx >> 4, ch = idx & 15;
        const int64_t m = t.m0 + rr;
        if (m < rows) {
            const u4 v = *reinterpret_cast<const u4 *>(&tile[rr * kTileStride + ch * 8]);
            *reinterpret_cast<u4 *>(Yp + m * ldy + t.n0 + ch * 8) = v;
        }
    }
}

// Epilogue of the fp32 kernel.  The products are taken as Y^T = W H^T
// (weights as the first MFMA operand), so result register v of block (j, i)
// in lane l holds output row 16 i + l % 16 and output column 16 j + 4 (l / 16)
// + v of a 64-column slab: each lane owns four consecutive columns of one row
// per block, staged with one 16-byte LDS write, and a head's attention sums
// reduce inside the lane and then over the four lanes l % 16 + {0, 16, 32, 48}.
//
// The per-column constants are read from LDS (`cst[kind * CS + column]`,
// kinds c', a, a~, U; CS columns per kind), staged before any store is
// issued: on this GPU a wait for an outstanding load also waits for earlier
// stores, so no global load may follow the first store.
//
// One call covers NI row blocks of 16 (rows rbase + 16 i, rbase carrying the
// lane's l % 16) and the 64 columns col0 .. col0 + 63, which lie in one
// relation half (F is a multiple of 64), from accumulator blocks
// acc[J0 .. J0 + 3][0 .. NI - 1].  The Y rows go through the wavefront's
// LDS slice `stage` (16 NI rows of kStageStride floats) and leave as whole
// 256-byte row segments, four rows per store instruction (stored from the
// accumulator layout, each instruction would cover half of sixteen lines).
constexpr int kStageStride = 64 + 4;
template <int JPH, bool ELU, int NI, int CS, int J0, int NJ, bool TSP>
__device__ void store_rows(const GemmArgs &G, const Tile &t, int64_t rbase, int col0, int lane,
                           const f4 (&acc)[NJ][NI], const float *cst, float *stage) {
    static_assert(J0 + 4 <= NJ, "four column blocks");
    const GemmPrep &P = G.prep;
    const int64_t rows = t.sd ? G.side[1].rows : G.side[0].rows;
    const int F = G.F, K = P.K, D = 16 * (JPH > 0 ? JPH : 1);
    const int64_t ldy = 2 * F;
    void *Yp = t.sd ? G.side[1].Y : G.side[0].Y;
    const bool od = col0 >= F;
    const int cw = od ? col0 - F : col0;           // first channel of the relation
    const int g = lane >> 4;
    const bool dev_od = od && t.sd == 1;           // device rows also get the message table
    float *S = P.S[t.sd];
    // row blocks outer, column blocks inner
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int64_t m = rbase + 16 * i;
        const bool mok = m < rows;
        float p0 = 0.f, p1 = 0.f, q = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = cw + 16 * j + 4 * g;         // the lane's first channel in this block
            const int cc = 16 * j + 4 * g;             // ... within the slab's columns
            float c3[4], c1[4], c2[4], c4[4];           // c'; od: a, a~, U; same-type: a~
            {
                const float4 x3 = *reinterpret_cast<const float4 *>(cst + cc);
                const float4 x1 = *reinterpret_cast<const float4 *>(cst + CS + cc);
                const float4 x2 = *reinterpret_cast<const float4 *>(cst + 2 * CS + cc);
                const float4 x4 = *reinterpret_cast<const float4 *>(cst + 3 * CS + cc);
                c3[0] = x3.x; c3[1] = x3.y; c3[2] = x3.z; c3[3] = x3.w;
                c1[0] = x1.x; c1[1] = x1.y; c1[2] = x1.z; c1[3] = x1.w;
                c2[0] = x2.x; c2[1] = x2.y; c2[2] = x2.z; c2[3] = x2.w;
                c4[0] = x4.x; c4[1] = x4.y; c4[2] = x4.z; c4[3] = x4.w;
            }
            {
                float ys[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) ys[v] = acc[J0 + j][i][v] + c3[v];
                *reinterpret_cast<float4 *>(stage + (16 * i + (lane & 15)) * kStageStride + cc) =
                    make_float4(ys[0], ys[1], ys[2], ys[3]);
            }
            if (mok) {
                float ys[4], yv[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) { ys[v] = acc[J0 + j][i][v] + c3[v]; yv[v] = acc[J0 + j][i][v]; }
                if constexpr (JPH > 0) {
                    if (od) {
                        float t0[4], t1[4];
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            t0[v] = msg_act<ELU>(ys[v]);
                            t1[v] = msg_act<ELU>(ys[v] + c4[v]);
                            p0 = fmaf(c1[v], t0[v], p0);
                            p1 = fmaf(c1[v], t1[v], p1);
                            q = fmaf(c2[v], yv[v], q);
                        }
                        if (TSP && dev_od) {   // message rows of bit 0 / 1 as exact splits, (bit 0, bit 1) pairs
                            unsigned sp[4][3];
#pragma unroll
                            for (int v = 0; v < 4; ++v) split3(t0[v], t1[v], sp[v]);
                            unsigned *Tu = reinterpret_cast<unsigned *>(P.T);
#pragma unroll
                            for (int z = 0; z < 3; ++z)
                                *reinterpret_cast<u4 *>(Tu + z * rows * F + m * F + c) =
                                    u4{sp[0][z], sp[1][z], sp[2][z], sp[3][z]};
                        } else if (!TSP && dev_od) {   // fp32 message rows of bit 0 / 1
                            *reinterpret_cast<float4 *>(P.T + (m * 2 + 0) * F + c) = make_float4(t0[0], t0[1], t0[2], t0[3]);
                            *reinterpret_cast<float4 *>(P.T + (m * 2 + 1) * F + c) = make_float4(t1[0], t1[1], t1[2], t1[3]);
                        }
                    } else {
#pragma unroll
                        for (int v = 0; v < 4; ++v) q = fmaf(c2[v], yv[v], q);
                    }
                }
            }
            if constexpr (JPH > 0) {
                if ((j + 1) % JPH == 0) {   // the head of blocks j+1-JPH .. j is complete for row m
                    const int h = (cw + 16 * (j + 1 - JPH)) / D;
                    p0 += __shfl_xor(p0, 16, 64); p0 += __shfl_xor(p0, 32, 64);
                    p1 += __shfl_xor(p1, 16, 64); p1 += __shfl_xor(p1, 32, 64);
                    q += __shfl_xor(q, 16, 64); q += __shfl_xor(q, 32, 64);
                    if (g == 0 && mok) {
                        if (od) {
                            S[m * 4 * K + h] = p0;
                            S[m * 4 * K + K + h] = p1;
                            S[m * 4 * K + 2 * K + h] = q;
                        } else {
                            S[m * 4 * K + 3 * K + h] = q;
                        }
                    }
                    p0 = p1 = q = 0.f;
                }
            }
        }
    }
    // the staged rows, four per instruction (a wavefront's own LDS slice:
    // its writes above are ordered before these reads)
    const int64_t r0 = rbase - (lane & 15);
#pragma unroll
    for (int it = 0; it < 4 * NI; ++it) {
        const int rr = 4 * it + (lane >> 4);
        const float4 v = *reinterpret_cast<const float4 *>(stage + rr * kStageStride + 4 * (lane & 15));
        if (r0 + rr < rows)
            *reinterpret_cast<float4 *>(static_cast<float *>(Yp) + (r0 + rr) * ldy + col0 + 4 * (lane & 15)) = v;
    }
}

// The four per-column constants of output column n (c'; od: a, a~, U;
// same-type: a~; zero where a kind does not apply)
template <int JPH>
__device__ __forceinline__ void column_consts(const GemmArgs &G, int sd, int n, float (&v)[4]) {
    const GemmPrep &P = G.prep;
    const bool od = n >= G.F;
    const int c = od ? n - G.F : n;
    v[0] = od ? P.cp_od[c] : P.cp_same[sd][c];
    v[1] = v[2] = v[3] = 0.f;
    if (JPH > 0) {
        if (od) { v[1] = P.a_od[c]; v[2] = P.ad_od[c]; v[3] = P.u_od[2 * c]; }
        else v[2] = P.ad_same[sd][c];
    }
}

// fp32 relation transform on the bf16 matrix cores: both operands are split
// exactly into three bf16 parts (split3) as they are loaded, and each 16 x 16
// output block takes the six part products a_i b_j with i + j <= 2 on 16x16x32
// bf16 MFMAs with fp32 accumulation.  Every part product is exact in fp32;
// the three dropped ones add up to at most (2^-23 + 2^-32) |a b|, one fp32
// rounding of the product, so the result is the fp32 contraction up to fp32
// rounding.  At the matrix cores' rates (bf16 16 times fp32) the six
// 16x16x32 products of a 16 x 16 x 32 contraction take 3/8 of the time of
// its eight 16x16x4 fp32 products.
//
// 128 x 128 block tiles, four wavefronts of 32 rows x 128 columns, so each
// hidden row is loaded and split by one wavefront only: lanes read their H
// operands straight from global memory into registers (row l % 16 of a row
// block, k-slice 8 (l / 16) of the 32-wide step) and split them there.  The
// weights of the block's 128 columns pass through LDS as split planes, one
// 32-wide k-step at a time, double-buffered, rows unpadded with XOR-swizzled
// 16-byte chunks (as in gemm_bf16).  The next step's global loads are in
// flight while the current step's 96 products per wavefront run.
template <int JPH, bool ELU, bool TSP>
__global__ void __launch_bounds__(256) gemm_f32s(GemmArgs G) {
    constexpr int BK = 32;
    __shared__ __attribute__((aligned(16))) uint16_t Ws[2][3][BN * BK];
    __shared__ __attribute__((aligned(16))) float cst[4 * BN];   // column constants, 4 kinds x 128
    auto sw = [](int r) { return ((r >> 1) ^ (r >> 2)) & 3; };
    const Tile t = tile_of(G);
    const GemmSide S = t.sd ? G.side[1] : G.side[0];
    const float *__restrict__ H = static_cast<const float *>(S.H);
    const int F = G.F;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid < BN) {
        float v[4];
        column_consts<JPH>(G, t.sd, t.n0 + tid, v);
#pragma unroll
        for (int q = 0; q < 4; ++q) cst[q * BN + tid] = v[q];
    }
    // weight loader: thread -> rows tid/4 and tid/4 + 64 of the block's
    // columns, 8-wide k-chunk tid % 4 of the step
    const int lc = tid & 3;
    const float *brow[2];
    int loff[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int lr = (tid >> 2) + 64 * q;
        const int gn = t.n0 + lr;
        brow[q] = (gn < F ? static_cast<const float *>(S.B0) + (size_t)gn * S.ldb
                          : static_cast<const float *>(S.B1) + (size_t)(gn - F) * S.ldb) + 8 * lc;
        loff[q] = lr * BK + 8 * (lc ^ sw(lr));
    }
    // hidden-row operands: row blocks i = 0, 1 of the wavefront's 32 rows
    const int64_t rbase = t.m0 + wave * 32 + (lane & 15);
    const float *hrow[2];
    bool hok[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        hok[i] = rbase + 16 * i < S.rows;
        hrow[i] = H + (hok[i] ? rbase + 16 * i : 0) * F + 8 * (lane >> 4);
    }
    int boff[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int r = j * 16 + (lane & 15);
        boff[j] = r * BK + 8 * ((lane >> 4) ^ sw(r));
    }
    float4 rb[2][2], rh[2][2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            rb[q][0] = *reinterpret_cast<const float4 *>(brow[q] + k0);
            rb[q][1] = *reinterpret_cast<const float4 *>(brow[q] + k0 + 4);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {   // rows past the end read row 0 (zeroed when split)
            rh[i][0] = *reinterpret_cast<const float4 *>(hrow[i] + k0);
            rh[i][1] = *reinterpret_cast<const float4 *>(hrow[i] + k0 + 4);
        }
    };
    // eight fp32 values -> their three bf16 planes, 16 bytes each
    auto split8 = [](const float4 (&x)[2], u4 (&o)[3]) {
        unsigned p[4][3];
        split3(x[0].x, x[0].y, p[0]);
        split3(x[0].z, x[0].w, p[1]);
        split3(x[1].x, x[1].y, p[2]);
        split3(x[1].z, x[1].w, p[3]);
#pragma unroll
        for (int z = 0; z < 3; ++z) o[z] = u4{p[0][z], p[1][z], p[2][z], p[3][z]};
    };
    auto wstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            u4 o[3];
            split8(rb[q], o);
#pragma unroll
            for (int z = 0; z < 3; ++z) *reinterpret_cast<u4 *>(&Ws[buf][z][loff[q]]) = o[z];
        }
    };
    bf8 ah[2][3];
    auto hsplit = [&]() {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            u4 o[3];
            split8(rh[i], o);
#pragma unroll
            for (int z = 0; z < 3; ++z) ah[i][z] = __builtin_bit_cast(bf8, hok[i] ? o[z] : u4{0u, 0u, 0u, 0u});
        }
    };
    f4 acc[8][2];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[j][i] = f4{0.f, 0.f, 0.f, 0.f};
    gload(0);
    wstore(0);
    hsplit();
    __syncthreads();
    const int nk = F / BK;
    for (int kc = 0; kc < nk; ++kc) {
        const int buf = kc & 1;
        if (kc + 1 < nk) gload((kc + 1) * BK);
        // two column blocks at a time: 24 products over four accumulators,
        // part products outer so that no two consecutive ones share one
#pragma unroll
        for (int jp = 0; jp < 4; ++jp) {
            bf8 bw[2][3];
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                for (int z = 0; z < 3; ++z)
                    bw[jj][z] = *reinterpret_cast<const bf8 *>(&Ws[buf][z][boff[2 * jp + jj]]);
            constexpr int PW[6] = {2, 1, 0, 1, 0, 0}, PH[6] = {0, 1, 2, 0, 1, 0};   // smallest first
#pragma unroll
            for (int pp = 0; pp < 6; ++pp)
#pragma unroll
                for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                    for (int i = 0; i < 2; ++i)
                        acc[2 * jp + jj][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            bw[jj][PW[pp]], ah[i][PH[pp]], acc[2 * jp + jj][i], 0, 0, 0);
        }
        if (kc + 1 < nk) {
            wstore(buf ^ 1);
            hsplit();
        }
        __syncthreads();
    }
    // the k-step buffers are free (the loop ends with a barrier): one row
    // stage per wavefront
    float *stage = reinterpret_cast<float *>(&Ws[0][0][0]) + wave * 32 * kStageStride;
    static_assert(4 * 32 * kStageStride * 4 <= sizeof(Ws), "row stages must fit the k-step buffers");
    store_rows<JPH, ELU, 2, BN, 0, 8, TSP>(G, t, rbase, t.n0, lane, acc, cst, stage);
    store_rows<JPH, ELU, 2, BN, 4, 8, TSP>(G, t, rbase, t.n0 + 64, lane, acc, cst + 64, stage);
}

template <int JPH, int MB>
__global__ void __launch_bounds__(2 * MB) gemm_bf16(GemmArgs G) {
    // MB x 128 block tiles, MB / 32 wavefronts of 64 x 64 (two per column
    // half): a taller block reads each k-chunk of the weights for more rows
    constexpr int BK = kBkBf16, NT = 2 * MB;
    static_assert(BK == 32, "four 16-byte chunks per LDS row");
    static_assert(MB == 128 || MB == 256, "two or four row wavefronts");
    // k-chunk buffers As[2][MB * BK], Bs[2][BN * BK]: unpadded rows whose four
    // 16-byte chunks are XOR-swizzled (chunk c of row r at c ^ sw(r)) so that
    // neither the loader's stores (4 threads per row) nor the operand reads
    // (16 rows, one chunk) meet a bank twice; the epilogue reuses the space
    // for the output tile and the column constants
    constexpr int SMK = 2 * MB * BK + 2 * BN * BK, SME = (MB * kTileStride * 2 + 4 * BN * 4) / 2;
    constexpr int SM = SMK > SME ? SMK : SME;
    __shared__ __attribute__((aligned(16))) uint16_t sm[SM];
    uint16_t (*As)[MB * BK] = reinterpret_cast<uint16_t (*)[MB * BK]>(sm);
    uint16_t (*Bs)[BN * BK] = reinterpret_cast<uint16_t (*)[BN * BK]>(sm + 2 * MB * BK);
    auto sw = [](int r) { return ((r >> 1) ^ (r >> 2)) & 3; };
    const Tile t = tile_of<MB>(G);
    const GemmSide S = t.sd ? G.side[1] : G.side[0];
    const uint16_t *__restrict__ H = static_cast<const uint16_t *>(S.H);
    const int F = G.F;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // loader: 16-byte chunk tid % 4 of rows tid/4 + (NT/4) q; the A tile's MB
    // rows take two per thread, the B tile's 128 rows 512 / NT
    constexpr int QB = 4 * BN / NT;
    const int lc = tid & 3;
    const uint16_t *arow[2], *brow[QB];
    bool aok[2];
    int loffa[2], loffb[QB];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int lr = (tid >> 2) + (NT / 4) * q;
        const int64_t gm = t.m0 + lr;
        aok[q] = gm < S.rows;
        arow[q] = H + (aok[q] ? gm : 0) * F + 8 * lc;
        loffa[q] = lr * BK + 8 * (lc ^ sw(lr));
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) {
        const int lr = (tid >> 2) + (NT / 4) * q;
        const int gn = t.n0 + lr;
        brow[q] = (gn < F ? static_cast<const uint16_t *>(S.B0) + (size_t)gn * S.ldb
                          : static_cast<const uint16_t *>(S.B1) + (size_t)(gn - F) * S.ldb) + 8 * lc;
        loffb[q] = lr * BK + 8 * (lc ^ sw(lr));
    }
    u4 ra[2], rb[QB];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
            ra[q] = aok[q] ? *reinterpret_cast<const u4 *>(arow[q] + k0) : u4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int q = 0; q < QB; ++q) rb[q] = *reinterpret_cast<const u4 *>(brow[q] + k0);
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) *reinterpret_cast<u4 *>(&As[buf][loffa[q]]) = ra[q];
#pragma unroll
        for (int q = 0; q < QB; ++q) *reinterpret_cast<u4 *>(&Bs[buf][loffb[q]]) = rb[q];
    };
    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    gload(0);
    sstore(0);
    __syncthreads();
    const int nk = F / BK;
    const int kc4 = lane >> 4;   // this lane's chunk of a 32-wide step
    int aoff[4], boff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ra_ = wm * 64 + i * 16 + (lane & 15), rb_ = wn * 64 + i * 16 + (lane & 15);
        aoff[i] = ra_ * BK + 8 * (kc4 ^ sw(ra_));
        boff[i] = rb_ * BK + 8 * (kc4 ^ sw(rb_));
    }
    for (int kc = 0; kc < nk; ++kc) {
        const int buf = kc & 1;
        if (kc + 1 < nk) gload((kc + 1) * BK);
        bf8 a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const bf8 *>(&As[buf][aoff[i]]);
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = *reinterpret_cast<const bf8 *>(&Bs[buf][boff[j]]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        if (kc + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }
    store_tile_bf16<JPH, MB>(G, t, wm, wn, lane, acc, sm);
}

}  // namespace

int64_t transform_row_tiles(int64_t rows) { return (rows + BM - 1) / BM; }

constexpr int kBf16Rows = 128;   // rows per bf16 block tile (256 measured no faster)

template <int JPH>
void launch_gemm(const GemmArgs &G, bool bf, unsigned blocks, hipStream_t st) {
    // the device message table: split planes at F = 256, fp32 rows below
    if (bf) gemm_bf16<JPH, kBf16Rows><<<blocks, 2 * kBf16Rows, 0, st>>>(G);
    else if (G.F >= 256) {
        if (G.prep.elu) gemm_f32s<JPH, true, true><<<blocks, 256, 0, st>>>(G);
        else gemm_f32s<JPH, false, true><<<blocks, 256, 0, st>>>(G);
    } else {
        if (G.prep.elu) gemm_f32s<JPH, true, false><<<blocks, 256, 0, st>>>(G);
        else gemm_f32s<JPH, false, false><<<blocks, 256, 0, st>>>(G);
    }
}

void launch_transform(const GemmArgs &G0, bool bf, hipStream_t st) {
    GemmArgs G = G0;
    const int64_t bm = bf ? kBf16Rows : BM;   // rows per block tile
    G.tiles0 = (G.side[0].rows + bm - 1) / bm;
    const int64_t tiles1 = (G.side[1].rows + bm - 1) / bm;
    const unsigned blocks = (unsigned)((G.tiles0 + tiles1) * (2 * G.F / BN));
    switch (G.prep.jph) {
        case 1: launch_gemm<1>(G, bf, blocks, st); break;
        case 2: launch_gemm<2>(G, bf, blocks, st); break;
        case 4: launch_gemm<4>(G, bf, blocks, st); break;
        default: launch_gemm<0>(G, bf, blocks, st); break;
    }
}

}  // namespace tag
