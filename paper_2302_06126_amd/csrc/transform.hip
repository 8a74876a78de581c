// Relation transforms (Section 4.2.1 layer equation, the W^h h part):
//   op rows:     Y = H [W^h_oo ; W^h_od]^T     device rows: Y = H [W^h_dd ; W^h_od]^T
// One launch covers both row sets of a layer.  128 x 128 block tiles, four
// wavefronts of 64 x 64, k-chunks staged through LDS with the next chunk's
// global loads in flight while the current one feeds the matrix cores.  The
// 1-D block order is XCD-swizzled so the column tiles of one row tile (which
// re-read the same rows of H) land on the same XCD and share its L2.
//
// MFMA 16x16 operand layout: lane l supplies row/column l % 16 of A/B and
// k-slice l / 16 (4 k per slice for fp32 16x16x4, 8 for bf16 16x16x32);
// result register v of lane l holds row 4 (l / 16) + v, column l % 16.
#include "tag_internal.hpp"
#include "transform.hpp"

namespace tag {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128;

struct Tile {
    int sd;
    int64_t m0;
    int n0;
};

__device__ __forceinline__ Tile tile_of(const GemmArgs &G) {
    const uint32_t lb = xcd_swizzle(blockIdx.x, gridDim.x);
    const int ct = 2 * G.F / BN;
    const int64_t rt = lb / ct;
    Tile t;
    t.n0 = (int)(lb % ct) * BN;
    t.sd = rt < G.tiles0 ? 0 : 1;
    t.m0 = (rt - (t.sd ? G.tiles0 : 0)) * BM;
    return t;
}

__global__ void __launch_bounds__(256) gemm_f32(GemmArgs G) {
    constexpr int BK = 16, LS = BM + 16;   // k-major LDS rows, stride = 16 (mod 64) banks
    __shared__ float As[2][BK * LS];
    __shared__ float Bs[2][BK * LS];
    const Tile t = tile_of(G);
    const GemmSide S = t.sd ? G.side[1] : G.side[0];
    const float *__restrict__ H = static_cast<const float *>(S.H);
    float *__restrict__ Y = static_cast<float *>(S.Y);
    const int F = G.F;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // loader: thread -> (row lr, 8 consecutive k at lk)
    const int lr = tid >> 1, lk = (tid & 1) * 8;
    const int64_t gm = t.m0 + lr;
    const bool aok = gm < S.rows;
    const float *arow = H + (aok ? gm : 0) * F;
    const int gn = t.n0 + lr;
    const float *brow = gn < F ? static_cast<const float *>(S.B0) + (size_t)gn * S.ldb
                               : static_cast<const float *>(S.B1) + (size_t)(gn - F) * S.ldb;
    float4 ra[2], rb[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            ra[q] = aok ? *reinterpret_cast<const float4 *>(arow + k0 + lk + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
            rb[q] = *reinterpret_cast<const float4 *>(brow + k0 + lk + 4 * q);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int k = lk + 4 * q;
            As[buf][(k + 0) * LS + lr] = ra[q].x; As[buf][(k + 1) * LS + lr] = ra[q].y;
            As[buf][(k + 2) * LS + lr] = ra[q].z; As[buf][(k + 3) * LS + lr] = ra[q].w;
            Bs[buf][(k + 0) * LS + lr] = rb[q].x; Bs[buf][(k + 1) * LS + lr] = rb[q].y;
            Bs[buf][(k + 2) * LS + lr] = rb[q].z; Bs[buf][(k + 3) * LS + lr] = rb[q].w;
        }
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
    for (int kc = 0; kc < nk; ++kc) {
        const int buf = kc & 1;
        if (kc + 1 < nk) gload((kc + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            const int krow = (kk + (lane >> 4)) * LS;
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[buf][krow + wm * 64 + i * 16 + (lane & 15)];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[buf][krow + wn * 64 + j * 16 + (lane & 15)];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kc + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }
    const int ldy = 2 * F;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t m = t.m0 + wm * 64 + i * 16 + 4 * (lane >> 4) + v;
            if (m >= S.rows) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) Y[m * ldy + t.n0 + wn * 64 + j * 16 + (lane & 15)] = acc[i][j][v];
        }
}

__global__ void __launch_bounds__(256) gemm_bf16(GemmArgs G) {
    constexpr int BK = 32, LS = BK + 8;    // row-major LDS rows of 40 bf16 (80 B)
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LS];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LS];
    const Tile t = tile_of(G);
    const GemmSide S = t.sd ? G.side[1] : G.side[0];
    const uint16_t *__restrict__ H = static_cast<const uint16_t *>(S.H);
    uint16_t *__restrict__ Y = static_cast<uint16_t *>(S.Y);
    const int F = G.F;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = tid >> 1, lk = (tid & 1) * 16;
    const int64_t gm = t.m0 + lr;
    const bool aok = gm < S.rows;
    const uint16_t *arow = H + (aok ? gm : 0) * F;
    const int gn = t.n0 + lr;
    const uint16_t *brow = gn < F ? static_cast<const uint16_t *>(S.B0) + (size_t)gn * S.ldb
                                  : static_cast<const uint16_t *>(S.B1) + (size_t)(gn - F) * S.ldb;
    u4 ra[2], rb[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            ra[q] = aok ? *reinterpret_cast<const u4 *>(arow + k0 + lk + 8 * q) : u4{0u, 0u, 0u, 0u};
            rb[q] = *reinterpret_cast<const u4 *>(brow + k0 + lk + 8 * q);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            *reinterpret_cast<u4 *>(&As[buf][lr * LS + lk + 8 * q]) = ra[q];
            *reinterpret_cast<u4 *>(&Bs[buf][lr * LS + lk + 8 * q]) = rb[q];
        }
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
    for (int kc = 0; kc < nk; ++kc) {
        const int buf = kc & 1;
        if (kc + 1 < nk) gload((kc + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            const int koff = kk + 8 * (lane >> 4);
            bf8 a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a[i] = *reinterpret_cast<const bf8 *>(&As[buf][(wm * 64 + i * 16 + (lane & 15)) * LS + koff]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                b[j] = *reinterpret_cast<const bf8 *>(&Bs[buf][(wn * 64 + j * 16 + (lane & 15)) * LS + koff]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kc + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }
    const int ldy = 2 * F;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t m = t.m0 + wm * 64 + i * 16 + 4 * (lane >> 4) + v;
            if (m >= S.rows) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) Y[m * ldy + t.n0 + wn * 64 + j * 16 + (lane & 15)] = f2bf(acc[i][j][v]);
        }
}

}  // namespace

int64_t transform_row_tiles(int64_t rows) { return (rows + BM - 1) / BM; }

void launch_transform(const GemmArgs &G, bool bf, hipStream_t st) {
    const int64_t tiles1 = transform_row_tiles(G.side[1].rows);
    const unsigned blocks = (unsigned)((G.tiles0 + tiles1) * (2 * G.F / BN));
    if (bf) gemm_bf16<<<blocks, 256, 0, st>>>(G);
    else gemm_f32<<<blocks, 256, 0, st>>>(G);
}

}  // namespace tag
