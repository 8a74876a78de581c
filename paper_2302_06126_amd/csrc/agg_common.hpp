// Device helpers shared by the aggregation kernels (first-version path in
// forward.hip, MFMA path in agg_mfma.hip).
#pragma once

#include <type_traits>

#include "tag_internal.hpp"

namespace tag {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kWaves = 4;        // wavefronts per aggregation block
constexpr int kChunk = 256;      // entries per device<-op partial (first-version path)

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bf8 as_bf8(unsigned w0, unsigned w1, unsigned w2, unsigned w3) {
    return __builtin_bit_cast(bf8, u4v{w0, w1, w2, w3});
}

// acc += A B for fp32 operands given as exact three-way bf16 splits
// (split3, round-to-nearest-even parts: |a_1| <= 2^-8 |a|, |a_2| <= 2^-16 |a|):
// the six part products a_i b_j with i + j <= 2 on 16x16x32 bf16 MFMAs,
// smallest first.  Each part product is exact in fp32; the dropped terms
// a_1 b_2, a_2 b_1 and a_2 b_2 add up to at most (2^-23 + 2^-32) |a b|, the
// size of one fp32 rounding of the product, so the result is an fp32
// contraction of A and B up to fp32 rounding.
__device__ __forceinline__ f4 mfma_split3(const bf8 (&a)[3], const bf8 (&b)[3], f4 acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[2], b[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1], b[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1], b[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[1], acc, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[0], acc, 0, 0, 0);
}

// SZ bytes per lane from global memory straight into LDS (global_load_lds,
// dword or dwordx4): lane l of the wavefront writes lds + SZ l, lds being
// wave-uniform; counted by vmcnt like any global load.  The builtin exists in
// the device pass only.
template <int SZ = 16>
__device__ __forceinline__ void load_lds(const void *src, void *lds) {
    static_assert(SZ == 4 || SZ == 16, "4- or 16-byte lanes");
#if defined(__HIP_DEVICE_COMPILE__)
    if constexpr (SZ == 16) __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
    else __builtin_amdgcn_global_load_lds(src, lds, 4, 0, 0);
#endif
}

// Sparse 16x16x64 bf16 products (v_smfmac_f32_16x16x64_bf16).  A is 16 x 64
// with at most two nonzeros in every four consecutive k, given as its eight
// nonzero values per lane plus 2-bit positions; B is dense 64 x 16.  Lane
// layout, lane l, g = l / 16: A row l % 16, value v at k = 16g + 4(v/2) + i_v
// with i_v = bits 2v+1..2v of the index operand; B column l % 16, element t
// at k = 8g + t (t < 8) or 32 + 8g + t - 8 (t >= 8); the result as for the
// dense 16x16 products (row 4g + i in register i).
typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));
typedef unsigned u8v __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bf16x16 as_bf16x16(const unsigned (&w)[8]) {
    return __builtin_bit_cast(bf16x16, u8v{w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]});
}
// mfma_split3 on the sparse products: the same six part products, with the
// index operand shared by the three parts of A
__device__ __forceinline__ f4 smfmac_split3(const bf8 (&a)[3], const bf16x16 (&b)[3], int idx, f4 acc) {
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[2], b[0], acc, idx, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[1], b[1], acc, idx, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[0], b[2], acc, idx, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[1], b[0], acc, idx, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[0], b[1], acc, idx, 0, 0);
    return __builtin_amdgcn_smfmac_f32_16x16x64_bf16(a[0], b[0], acc, idx, 0, 0);
}

// -------------------------------------------------------------- aggregation
struct AggArgs {
    int32_t R;
    int64_t n_op, n_dev;
    const int32_t *rp[4], *col[4], *eid[4];
    const void *Y_op, *Y_dev;         // [R*n][2F]
    const float *x_oo; int64_t s_oo;
    const float *x_dd; int64_t s_dd;
    const uint8_t *x_od; int64_t s_od;
    const float *att_src, *att_dst;   // [3][F] of this layer
    const float *U;                   // [3][F][2] of this layer
    const float *cp;                  // [3][F] of this layer
    float g_same, g_cross, slope;
    void *H_op, *H_dev;               // outputs (bf16 hidden or fp32)
    int out_f32;
    int32_t elu;                      // message non-linearity: 0 ReLU, 1 ELU (fp32 only)
    float *part;                      // device<-op partials
    int32_t maxc;                     // partial records per device row
    // MFMA path
    int32_t G, n_tiles;
    const int32_t *tiles, *tile_off, *op_off, *dev_off;
    uint64_t *omask;                  // [R*n_op][2]: present / placement-bit masks over local devices
    float *Sdev;                      // [R*n_dev][4][K]: p0, p1, q_od, q_dd of device rows
    float *T;                         // fp32 variant: [R*n_dev][2][F] device messages for bit 0 / 1;
                                      // bf16 variant: [3][R*n_dev][F] the exact three-way bf16 splits
                                      // (split3) of the same fp32 messages, packed (bit 0, bit 1)
    float *Sop;                       // [R*n_op][4][K]: p0, p1, q_od, q_oo of op rows
    int32_t prep_done;                // Sop, Sdev and T already written by the transform
    int32_t rec_mode;                 // 0: records per 256-entry chunk, 1: per tile group
    int32_t n_groups;
    const int32_t *groups, *group_off;   // tile groups of the device<-op blocks
    // written once per forward pass by prep_tiles_x: per op tile (first op,
    // op count, topology, first op<-op CSR entry, op<-op entries, first
    // device, device count, 0), and the op<-op edge features in CSR order
    int32_t *tile_ext;                // [n_tiles][8]
    float *xcsr; int64_t s_xcsr;      // [xrep][nnz of B0], xrep = 1 (shared features) or R
};

// MFMA path (agg_mfma.hip)
// whether the tile path takes a layer: heads of 16 to F channels (K <= 16),
// and the per-candidate transform rows (n_op 2F elements of esz bytes) and
// the device message table (three parts of R n_dev F words) addressed by
// 32-bit byte offsets
bool mfma_path_supported(int F, int K, int64_t n_op, int64_t R, int64_t n_dev, int esz);
void launch_pack_masks(const AggArgs &A, hipStream_t st);
void launch_prep_tiles_x(const AggArgs &A, int64_t nnz0, hipStream_t st);
bool launch_agg_mfma(int F, int K, bool bf, const AggArgs &A, hipStream_t st);

// CPL consecutive channels starting at element `off` (fp32 or bf16 storage);
// CPL is 1, 2 or a multiple of 4, and `off` is a multiple of min(CPL, 4).
template <int CPL, bool BF>
__device__ __forceinline__ void load_ch(const void *base, int64_t off, float (&v)[CPL]) {
    static_assert(CPL == 1 || CPL == 2 || CPL % 4 == 0, "unsupported channels per lane");
    if constexpr (BF) {
        const uint16_t *p = static_cast<const uint16_t *>(base) + off;
        if constexpr (CPL % 4 == 0) {
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) {
                const uint2 q = reinterpret_cast<const uint2 *>(p)[i];
                v[4 * i + 0] = bf2f(q.x & 0xffff); v[4 * i + 1] = bf2f(q.x >> 16);
                v[4 * i + 2] = bf2f(q.y & 0xffff); v[4 * i + 3] = bf2f(q.y >> 16);
            }
        } else if constexpr (CPL == 2) {
            const uint32_t q = *reinterpret_cast<const uint32_t *>(p);
            v[0] = bf2f(q & 0xffff); v[1] = bf2f(q >> 16);
        } else {
            v[0] = bf2f(p[0]);
        }
    } else {
        const float *p = static_cast<const float *>(base) + off;
        if constexpr (CPL % 4 == 0) {
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) {
                const float4 q = reinterpret_cast<const float4 *>(p)[i];
                v[4 * i + 0] = q.x; v[4 * i + 1] = q.y; v[4 * i + 2] = q.z; v[4 * i + 3] = q.w;
            }
        } else if constexpr (CPL == 2) {
            const float2 q = *reinterpret_cast<const float2 *>(p);
            v[0] = q.x; v[1] = q.y;
        } else {
            v[0] = p[0];
        }
    }
}

// CPL consecutive channels of one row kept as loaded (bf16 pairs or fp32
// words); get(c) widens channel c
template <int CPL, bool BF>
struct RowRaw {
    static constexpr int NW = BF ? CPL / 2 : CPL;
    unsigned w[NW];
    __device__ __forceinline__ void load(const void *base, int64_t off) {
        static_assert(CPL % 4 == 0, "RowRaw needs a multiple of 4 channels");
        if constexpr (BF) {
            const uint2 *p = reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(base) + off);
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) { const uint2 q = p[i]; w[2 * i] = q.x; w[2 * i + 1] = q.y; }
        } else {
            const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const float *>(base) + off);
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) {
                const uint4 q = p[i];
                w[4 * i] = q.x; w[4 * i + 1] = q.y; w[4 * i + 2] = q.z; w[4 * i + 3] = q.w;
            }
        }
    }
    // the same from a wave-uniform base and a 32-bit byte offset
    __device__ __forceinline__ void load32(const void *base, uint32_t byte_off) {
        const char *b = static_cast<const char *>(base) + byte_off;
        if constexpr (BF) {
            const uint2 *p = reinterpret_cast<const uint2 *>(b);
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) { const uint2 q = p[i]; w[2 * i] = q.x; w[2 * i + 1] = q.y; }
        } else {
            const uint4 *p = reinterpret_cast<const uint4 *>(b);
#pragma unroll
            for (int i = 0; i < CPL / 4; ++i) {
                const uint4 q = p[i];
                w[4 * i] = q.x; w[4 * i + 1] = q.y; w[4 * i + 2] = q.z; w[4 * i + 3] = q.w;
            }
        }
    }
    __device__ __forceinline__ float get(int c) const {
        if constexpr (BF) return __uint_as_float((c & 1) ? (w[c >> 1] & 0xffff0000u) : (w[c >> 1] << 16));
        else return __uint_as_float(w[c]);
    }
};

template <int LPH>
__device__ __forceinline__ float head_sum(float v) {
#pragma unroll
    for (int o = LPH / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Sum over aligned groups of LPH <= 16 lanes with DPP moves inside a 16-lane
// row (quad swaps, then the half-row and row mirrors pair the remaining
// lanes); every lane of a group ends with the group's total.
template <int LPH>
__device__ __forceinline__ float row_sum(float v) {
    static_assert(LPH >= 1 && LPH <= 16 && (LPH & (LPH - 1)) == 0, "LPH must be a power of two <= 16");
    auto dpp = [](float x, auto ctrl) {
        return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), decltype(ctrl)::value, 0xf, 0xf, true));
    };
    if constexpr (LPH >= 2) v += dpp(v, std::integral_constant<int, 0xB1>{});    // quad_perm [1,0,3,2]
    if constexpr (LPH >= 4) v += dpp(v, std::integral_constant<int, 0x4E>{});    // quad_perm [2,3,0,1]
    if constexpr (LPH >= 8) v += dpp(v, std::integral_constant<int, 0x141>{});   // row_half_mirror
    if constexpr (LPH >= 16) v += dpp(v, std::integral_constant<int, 0x140>{});  // row_mirror
    return v;
}

// per-lane constants of one relation
template <int CPL>
struct RelConst {
    float a[CPL], ad[CPL], u0[CPL], u1[CPL], cp[CPL];
    __device__ void load(const AggArgs &A, int r, int F, int c0) {
        for (int c = 0; c < CPL; ++c) {
            a[c] = A.att_src[r * F + c0 + c];
            ad[c] = A.att_dst[r * F + c0 + c];
            u0[c] = A.U[((size_t)r * F + c0 + c) * 2 + 0];
            u1[c] = A.U[((size_t)r * F + c0 + c) * 2 + 1];
            cp[c] = A.cp[(size_t)r * F + c0 + c];
        }
    }
};

template <int CPL>
struct Online {
    float mx, den, acc[CPL];
    __device__ void init() {
        mx = -INFINITY; den = 0.f;
        for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
    }
    // s2: score already multiplied by log2(e)
    __device__ void push(float s2, const float (&m)[CPL]) {
        float nm = fmaxf(mx, s2);
        float sc = __builtin_amdgcn_exp2f(mx - nm);
        float p = __builtin_amdgcn_exp2f(s2 - nm);
        den = fmaf(den, sc, p);
        for (int c = 0; c < CPL; ++c) acc[c] = fmaf(acc[c], sc, p * m[c]);
        mx = nm;
    }
    // the first n of EB entries, one rescale for the batch
    template <int EB>
    __device__ void push_n(const float (&s2)[EB], const float (&m)[EB][CPL], int n) {
        float nm = mx;
#pragma unroll
        for (int i = 0; i < EB; ++i)
            if (i < n) nm = fmaxf(nm, s2[i]);
        const float sc = __builtin_amdgcn_exp2f(mx - nm);
        float p[EB];
#pragma unroll
        for (int i = 0; i < EB; ++i) p[i] = i < n ? __builtin_amdgcn_exp2f(s2[i] - nm) : 0.f;
        float ps = 0.f;
#pragma unroll
        for (int i = 0; i < EB; ++i) ps += p[i];
        den = fmaf(den, sc, ps);
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            float a = acc[c] * sc;
#pragma unroll
            for (int i = 0; i < EB; ++i) a = fmaf(p[i], m[i][c], a);
            acc[c] = a;
        }
        mx = nm;
    }
};

// Stored relation rows Y: the fp32 variant stores W^h h + c' (c' of the
// column's relation), the bf16 variant stores bf16(W^h h) -- only the
// transform's product is rounded, and c' is added in fp32 where a message is
// formed.  stored_dst gives W^h h (attention destination terms).
template <bool BF>
__device__ __forceinline__ float stored_dst(float stored, float cp) { return BF ? stored : stored - cp; }

// message + score of one entry; returns the log2-domain score
template <int CPL, int LPH, bool ELU = false, bool BF = false>
__device__ __forceinline__ float entry_score(const float (&y)[CPL], float x0, float x1, const RelConst<CPL> &k,
                                             float qd, float slope, float (&m)[CPL]) {
    float part = 0.f;
    for (int c = 0; c < CPL; ++c) {
        // fp32 rows hold Y + c'; bf16 rows hold Y, and the edge term U x + c' is added whole
        const float z = BF ? y[c] + fmaf(k.u0[c], x0, fmaf(k.u1[c], x1, k.cp[c]))
                           : y[c] + fmaf(k.u0[c], x0, k.u1[c] * x1);
        m[c] = msg_act<ELU>(z);
        part = fmaf(k.a[c], m[c], part);
    }
    float s = head_sum<LPH>(part) + qd;
    return leaky(s, slope) * kLog2e;
}

template <int CPL, bool BF>
__device__ __forceinline__ void store_row(void *base, int64_t off, bool f32, const float (&v)[CPL]) {
    if (f32) {
        float *p = static_cast<float *>(base) + off;
        for (int c = 0; c < CPL; ++c) p[c] = v[c];
    } else {
        uint16_t *p = static_cast<uint16_t *>(base) + off;
        for (int c = 0; c < CPL; ++c) p[c] = f2bf(v[c]);
    }
}


}  // namespace tag
