// Row-gathered fp32 GEMM with bias/ReLU epilogue on MFMA 16x16x4:
//   C[m][n] = act(bias[n] + sum_k A[row(m)][k] B[n][k]),  row(m) = row_map ? row_map[m] : m
// Used where the contraction is small and dense: the node encoders
// (K = raw feature width) and the decoder projections (K = f).  Any K and N
// (guarded loads); a negative row_map entry reads a zero row.
#include "tag_internal.hpp"

namespace tag {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
constexpr int SM = 64, SN = 64, SK = 16;

__global__ void __launch_bounds__(256) small_gemm(SmallGemm G) {
    __shared__ float As[SM][SK + 1];
    __shared__ float Bs[SN][SK + 1];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.x * SM;
    const int n0 = blockIdx.y * SN;
    f4 acc[2][2];
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int64_t gm = m0 + lr;
    int64_t arow = -1;
    if (gm < G.rows) arow = G.row_map ? G.row_map[gm] : gm;
    const int gn = n0 + lr;
    // the next chunk's operands are loaded into registers while the current
    // one feeds the matrix cores
    float ra[4], rb[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + lk + q;
            ra[q] = (arow >= 0 && k < G.K) ? G.A[arow * G.lda + k] : 0.f;
            rb[q] = (gn < G.N && k < G.K) ? G.B[(int64_t)gn * G.ldb + k] : 0.f;
        }
    };
    gload(0);
    for (int k0 = 0; k0 < G.K; k0 += SK) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            As[lr][lk + q] = ra[q];
            Bs[lr][lk + q] = rb[q];
        }
        __syncthreads();
        if (k0 + SK < G.K) gload(k0 + SK);
#pragma unroll
        for (int kk = 0; kk < SK; kk += 4) {
            float a[2], b[2];
            for (int i = 0; i < 2; ++i) a[i] = As[wm * 32 + i * 16 + (lane & 15)][kk + (lane >> 4)];
            for (int j = 0; j < 2; ++j) b[j] = Bs[wn * 32 + j * 16 + (lane & 15)][kk + (lane >> 4)];
            for (int i = 0; i < 2; ++i)
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn * 32 + j * 16 + (lane & 15);
            if (n >= G.N) continue;
            const float bias = G.bias ? G.bias[n] : 0.f;
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * 32 + i * 16 + 4 * (lane >> 4) + v;
                if (m >= G.rows) continue;
                float x = acc[i][j][v] + bias;
                if (G.relu) x = fmaxf(x, 0.f);
                if (G.c_bf16) static_cast<uint16_t *>(G.C)[m * G.ldc + n] = f2bf(x);
                else static_cast<float *>(G.C)[m * G.ldc + n] = x;
            }
        }
}

}  // namespace

void launch_small_gemm(const SmallGemm &G, hipStream_t st) {
    if (G.rows <= 0 || G.N <= 0) return;
    dim3 grid((unsigned)((G.rows + SM - 1) / SM), (unsigned)((G.N + SN - 1) / SN));
    small_gemm<<<grid, 256, 0, st>>>(G);
}

}  // namespace tag
