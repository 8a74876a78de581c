// Internal declarations shared by the translation units of libtag.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/tag.h"
#include "../../include/tag_profile.h"

namespace tag {

// ------------------------------------------------------------------ errors
void set_error(const std::string &msg);
void clear_error();

#define TAG_FAIL(code, msg)          \
    do {                             \
        ::tag::set_error(msg);       \
        return (code);               \
    } while (0)

#define TAG_HIP_CHECK(expr)                                                            \
    do {                                                                               \
        hipError_t e_ = (expr);                                                        \
        if (e_ != hipSuccess)                                                          \
            TAG_FAIL(TAG_EHIP, std::string(#expr ": ") + hipGetErrorString(e_));       \
    } while (0)

// Check for a launch error right after enqueueing kernels.
tag_status launch_status(const char *what);

// Optional per-stage event timing (stage ids from include/tag_profile.h).
void prof_begin(int stage, hipStream_t s);
void prof_end(int stage, hipStream_t s);

// ------------------------------------------------------------ memory plans
inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// A bump allocator over a caller buffer (or a size counter when base == null).
struct Carver {
    char *base;
    size_t used = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    template <typename T>
    T *take(size_t count) {
        size_t off = used;
        used = align_up(used + count * sizeof(T));
        return base ? reinterpret_cast<T *>(base + off) : nullptr;
    }
};

}  // namespace tag

// ------------------------------------------------------------ graph handle
struct tag_graph {
    int32_t G = 0;
    int32_t max_dev = 0;
    int64_t n_op = 0, n_dev = 0, e_oo = 0, e_dd = 0, e_od = 0;
    std::vector<int64_t> op_off, dev_off;     // host [G+1]
    int64_t rows[4] = {0, 0, 0, 0}, nnz[4] = {0, 0, 0, 0};
    int32_t max_degree[4] = {0, 0, 0, 0};
    // device arrays inside the caller's csr buffer
    const int32_t *rowptr[4] = {nullptr, nullptr, nullptr, nullptr};
    const int32_t *col[4] = {nullptr, nullptr, nullptr, nullptr};
    const int32_t *eid[4] = {nullptr, nullptr, nullptr, nullptr};
    const int32_t *oo_head = nullptr;    // [E_oo] global id of each tensor link's consumer
    const int32_t *op_off_d = nullptr;   // [G+1]
    const int32_t *dev_off_d = nullptr;  // [G+1]
    // op tiles: runs of at most kOpTile consecutive ops of one topology
    int32_t n_tiles = 0;                 // total over topologies
    int32_t max_tiles = 0;               // largest per-topology tile count
    const int32_t *tiles_d = nullptr;    // [n_tiles][3] = (first op (global), op count, topology)
    const int32_t *tile_off_d = nullptr; // [G+1] first tile of each topology
    // tile groups: runs of consecutive tiles of one topology handled by one
    // device<-op block (at most kMaxDevRecords groups per topology)
    int32_t n_groups = 0;
    int32_t max_groups = 0;
    const int32_t *groups_d = nullptr;   // [n_groups][2] = (first tile, tile count)
    const int32_t *group_off_d = nullptr; // [G+1] first group of each topology
    int device = 0;
};

namespace tag {
constexpr int kOpTile = 64;
constexpr int kMaxDevRecords = 8;    // device<-op partial records per device row

// tiles per group for a topology of nt op tiles
inline int32_t tiles_per_group(int64_t nt) {
    return nt <= kMaxDevRecords ? 1 : (int32_t)((nt + kMaxDevRecords - 1) / kMaxDevRecords);
}

// C[m][n] = act(bias[n] + sum_k A[row(m)][k] * B[n][k]) on MFMA (gemm_small.hip)
struct SmallGemm {
    const float *A;
    int64_t lda, rows;
    const int32_t *row_map;   // optional gather of A rows (negative: zero row)
    int K;
    const float *B;
    int64_t ldb;
    int N;
    const float *bias;        // optional
    int relu;
    void *C;
    int64_t ldc;
    int c_bf16;
};
void launch_small_gemm(const SmallGemm &G, hipStream_t st);

// Slice part of the decoder's hidden pre-activation for every candidate
// graph rg = r G + g (decide.hip): u[rg][h][a] = sum_{j in mask_a} t[dev(rg, j)][h]
// + W1[h][2F + option_a] + b1[h], with t = E_dev W1_dev^T ([R n_dev][H]).
void launch_slice_terms(int32_t R, int32_t G, int32_t S, int32_t F, int32_t H, int64_t n_dev, const int32_t *dev_off,
                        const float *t, const float *W1, const float *b1, const uint64_t *mask,
                        const uint8_t *option, float *u, hipStream_t st);
}

// ----------------------------------------------------------- device helpers
namespace tag {

__device__ __forceinline__ float leaky(float x, float slope) { return x > 0.f ? x : slope * x; }

// message non-linearity sigma of the layer equation: ReLU, or ELU (alpha = 1)
template <bool ELU>
__device__ __forceinline__ float msg_act(float z) {
    if constexpr (ELU) return z > 0.f ? z : __expf(z) - 1.f;
    // max(z, 0) as one integer max of the bits (a set sign bit gives +0), so
    // that no quieting of z is needed first
    else return __int_as_float(max(__float_as_int(z), 0));
}

typedef unsigned u4v __attribute__((ext_vector_type(4)));

// two floats -> packed bf16 pair (round to nearest even, one gfx950
// conversion instruction), lo in the low half
__device__ __forceinline__ unsigned pack_bf2(float lo, float hi) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(unsigned, __builtin_convertvector(f2{lo, hi}, b2));
}
// round-to-nearest-even fp32 -> bf16 bits
__device__ __forceinline__ uint16_t f2bf(float x) { return static_cast<uint16_t>(pack_bf2(x, 0.f) & 0xffffu); }
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// Exact three-way bf16 split of two fp32 values, packed pairwise (lo in the
// low halves): x = part0 + part1 + part2, each part a bf16 value.  Each step
// rounds to nearest even and the residual it leaves is exact in fp32; the
// last residual has at most 8 significant bits, so part2 holds it exactly
// (values far below 2^-100 may lose their smallest parts as denormals).
// Products of two parts are exact in fp32.
__device__ __forceinline__ void split3(float lo, float hi, unsigned (&p)[3]) {
    p[0] = pack_bf2(lo, hi);
    float rl = lo - __uint_as_float(p[0] << 16), rh = hi - __uint_as_float(p[0] & 0xffff0000u);
    p[1] = pack_bf2(rl, rh);
    rl -= __uint_as_float(p[1] << 16);
    rh -= __uint_as_float(p[1] & 0xffff0000u);
    p[2] = pack_bf2(rl, rh);
}

// XCD-aware block order: the hardware deals consecutive workgroups to the
// 8 XCDs round-robin; remap so that logically consecutive blocks share an
// XCD (and its L2).  Bijective on [0, n).
__device__ __forceinline__ uint32_t xcd_swizzle(uint32_t bid, uint32_t n) {
    constexpr uint32_t X = 8;
    uint32_t per = n / X, rem = n % X;
    uint32_t x = bid % X, k = bid / X;
    // blocks bid >= X*per (the ragged tail) keep their order after the full part
    if (k >= per) return bid;
    (void)rem;
    return x * per + k;
}

}  // namespace tag
