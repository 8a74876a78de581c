// Row-gathered fp32 GEMM with bias/ReLU epilogue on MFMA 16x16x4:
//   C[m][n] = act(bias[n] + sum_k A[row(m)][k] B[n][k]),  row(m) = row_map ? row_map[m] : m
// Used where the contraction is small and dense: the node encoders
// (K = raw feature width) and the decoder projections (K = f).  Any K and N
// (guarded loads); a negative row_map entry reads a zero row.
//
// In the op encoder C (rows x f) is the largest stream.  A block covers 128
// columns (all of C's row for f <= 128, so A is read once), and the epilogue
// stages the finished tile in LDS and writes whole rows with 16-byte stores
// when C's pitch and alignment allow.
#include "tag_internal.hpp"

namespace tag {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
constexpr int SN = 128;                               // columns per block
constexpr int CP = SN + 4;                            // staged row pitch (floats)

// SM rows per block, k-chunks of SK; 4 waves as WM x (4 / WM)
template <int SM, int SK, int WM>
struct Tile {
    static constexpr int WN = 4 / WM;
    static constexpr int TI = SM / WM / 16, TJ = SN / WN / 16;   // 16x16 tiles per wave
    static constexpr int NA = SM * SK / 256, NB = SN * SK / 256; // operand floats per thread
    static constexpr int LDS = SM * CP > (SM + SN) * (SK + 1) ? SM * CP : (SM + SN) * (SK + 1);
    static_assert(TI >= 1 && TJ >= 1 && SM * SK % 256 == 0 && SK % 4 == 0, "tile shape");
};

// write a staged SM x SN tile (pitch CP) to C rows m0 .. m0 + mr, columns
// n0 .. n0 + nc: 16-byte stores when vec, else one element at a time
template <int SM>
__device__ __forceinline__ void store_tile(const SmallGemm &G, int vec, const float *Cs, int64_t m0, int64_t mr,
                                           int n0, int nc) {
    const int tid = threadIdx.x;
    if (vec && !G.c_bf16) {
        // 4 floats per 16-byte store; a row of the tile is 32 stores
        float *C = static_cast<float *>(G.C);
        for (int e = tid; e < SM * SN / 4; e += 256) {
            const int r = e >> 5, c = (e & 31) * 4;
            if (r >= mr || c >= nc) continue;
            *reinterpret_cast<f4 *>(C + (m0 + r) * G.ldc + n0 + c) = *reinterpret_cast<const f4 *>(Cs + r * CP + c);
        }
    } else if (vec) {
        // 8 bf16 per 16-byte store; a row of the tile is 16 stores
        uint16_t *C = static_cast<uint16_t *>(G.C);
        for (int e = tid; e < SM * SN / 8; e += 256) {
            const int r = e >> 4, c = (e & 15) * 8;
            if (r >= mr || c >= nc) continue;
            const f4 lo = *reinterpret_cast<const f4 *>(Cs + r * CP + c);
            const f4 hi = *reinterpret_cast<const f4 *>(Cs + r * CP + c + 4);
            const u4v p{pack_bf2(lo[0], lo[1]), pack_bf2(lo[2], lo[3]), pack_bf2(hi[0], hi[1]), pack_bf2(hi[2], hi[3])};
            *reinterpret_cast<u4v *>(C + (m0 + r) * G.ldc + n0 + c) = p;
        }
    } else {
        for (int e = tid; e < SM * SN; e += 256) {
            const int r = e / SN, c = e % SN;
            if (r >= mr || c >= nc) continue;
            const float x = Cs[r * CP + c];
            if (G.c_bf16) static_cast<uint16_t *>(G.C)[(m0 + r) * G.ldc + n0 + c] = f2bf(x);
            else static_cast<float *>(G.C)[(m0 + r) * G.ldc + n0 + c] = x;
        }
    }
}

template <int SM, int SK, int WM>
__global__ void __launch_bounds__(256) small_gemm(SmallGemm G, int vec) {
    using T = Tile<SM, SK, WM>;
    constexpr int WN = T::WN, TI = T::TI, TJ = T::TJ, NA = T::NA, NB = T::NB;
    // the operand chunks, and after the main loop the output tile
    __shared__ __align__(16) float lds[T::LDS];
    float (*As)[SK + 1] = reinterpret_cast<float (*)[SK + 1]>(lds);
    float (*Bs)[SK + 1] = reinterpret_cast<float (*)[SK + 1]>(lds + SM * (SK + 1));
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int64_t m0 = (int64_t)blockIdx.x * SM;
    const int n0 = blockIdx.y * SN;
    f4 acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    // operand element e = tid + 256 q of a chunk sits at row e / SK, column
    // e % SK: consecutive threads read contiguous bytes of one row
    int32_t arow[NA];   // row of A (int32, as row_map entries are)
#pragma unroll
    for (int q = 0; q < NA; ++q) {
        const int64_t gm = m0 + (tid + 256 * q) / SK;
        arow[q] = gm < G.rows ? (G.row_map ? G.row_map[gm] : (int32_t)gm) : -1;
    }
    // the next chunk's operands are loaded into registers while the current
    // one feeds the matrix cores
    float ra[NA], rb[NB];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < NA; ++q) {
            const int k = k0 + (tid + 256 * q) % SK;
            ra[q] = (arow[q] >= 0 && k < G.K) ? G.A[(int64_t)arow[q] * G.lda + k] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < NB; ++q) {
            const int gn = n0 + (tid + 256 * q) / SK, k = k0 + (tid + 256 * q) % SK;
            rb[q] = (gn < G.N && k < G.K) ? G.B[(int64_t)gn * G.ldb + k] : 0.f;
        }
    };
    gload(0);
    for (int k0 = 0; k0 < G.K; k0 += SK) {
#pragma unroll
        for (int q = 0; q < NA; ++q) As[(tid + 256 * q) / SK][(tid + 256 * q) % SK] = ra[q];
#pragma unroll
        for (int q = 0; q < NB; ++q) Bs[(tid + 256 * q) / SK][(tid + 256 * q) % SK] = rb[q];
        __syncthreads();
        if (k0 + SK < G.K) gload(k0 + SK);
#pragma unroll 4
        for (int kk = 0; kk < SK; kk += 4) {
            float a[TI], b[TJ];
#pragma unroll
            for (int i = 0; i < TI; ++i) a[i] = As[wm * (SM / WM) + i * 16 + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
            for (int j = 0; j < TJ; ++j) b[j] = Bs[wn * (SN / WN) + j * 16 + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int j = 0; j < TJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }
    // epilogue: bias and activation into the staged tile (lane l holds rows
    // 4 (l / 16) + v, column l % 16 of each 16x16 tile)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
        const int nl = wn * (SN / WN) + j * 16 + (lane & 15);
        const float bias = (G.bias && n0 + nl < G.N) ? G.bias[n0 + nl] : 0.f;
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float x = acc[i][j][v] + bias;
                if (G.relu) x = fmaxf(x, 0.f);
                lds[(wm * (SM / WM) + i * 16 + 4 * (lane >> 4) + v) * CP + nl] = x;
            }
    }
    __syncthreads();
    const int64_t mr = G.rows - m0 < SM ? G.rows - m0 : SM;
    const int nc = G.N - n0 < SN ? G.N - n0 : SN;
    store_tile<SM>(G, vec, lds, m0, mr, n0, nc);
}

template <int SM, int SK, int WM>
void launch_tile(const SmallGemm &G, int vec, hipStream_t st) {
    dim3 grid((unsigned)((G.rows + SM - 1) / SM), (unsigned)((G.N + SN - 1) / SN));
    small_gemm<SM, SK, WM><<<grid, 256, 0, st>>>(G, vec);
}

}  // namespace

void launch_small_gemm(const SmallGemm &G, hipStream_t st) {
    if (G.rows <= 0 || G.N <= 0) return;
    // 16-byte row stores need every stored vector inside C's row and aligned
    const int per = G.c_bf16 ? 8 : 4;
    const int vec = (G.N % per == 0 && G.ldc % per == 0 && reinterpret_cast<uintptr_t>(G.C) % 16 == 0) ? 1 : 0;
    // fewer than 256 blocks of 64 rows (the decoder projections, the device
    // encoder): 16-row blocks and 32-wide k-chunks, so that more compute units
    // work and fewer dependent load rounds separate the chunks
    if ((G.rows + 63) / 64 < 256) launch_tile<16, 32, 1>(G, vec, st);
    else launch_tile<64, 16, 2>(G, vec, st);
}

}  // namespace tag
