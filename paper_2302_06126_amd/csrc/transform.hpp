// Relation-transform GEMM interface (transform.hip).
#pragma once

#include "tag_internal.hpp"

namespace tag {

// One launch covers both row sets of a layer: row tiles [0, tiles0) take the
// op rows (side 0), the rest the device rows (side 1).
struct GemmSide {
    const void *H;       // [rows][F] hidden rows (fp32 or bf16)
    int64_t rows;
    const void *B0, *B1; // weights of output channels [0, F) and [F, 2F), B[n][k], row stride ldb
    int ldb;
    void *Y;             // [rows][2F]
};
// fp32: Y is stored as W^h h + c' (c' of the column's relation: same-type
// half or od half); bf16: Y is stored as bf16(W^h h), the only rounded
// quantity besides the operands, and consumers add c' in fp32.
// Optional epilogue: per-(row, head) attention terms of the layer, taken
// from the output rows while they are still in registers (heads of 16, 32
// or 64 channels, so one head lies inside one wavefront's 64 columns):
//   S[row][0][h] = a_od . sigma(Y_od + c'_od)         logit of message bit 0
//   S[row][1][h] = a_od . sigma(Y_od + c'_od + U_od)  logit of message bit 1
// (with Y the unbiased W^h h)
//   S[row][2][h] = a~_od . Y_od                       destination term, od
//   S[row][3][h] = a~_same . Y_same                   destination term, oo / dd
// and, for device rows, the two message rows T[row][b] = sigma(Y_od + c'_od + b U_od)
// (sigma: ReLU, or ELU for the variant): as exact three-way bf16 splits in
// the bf16 variant and at F = 256, as fp32 rows otherwise.
struct GemmPrep {
    int jph;             // 16-column blocks per head (1, 2, 4); 0: no attention terms
    int K;
    int elu;             // message non-linearity of the terms: 0 ReLU, 1 ELU
    const float *cp_same[2];             // [F]: folded bias c' of oo (side 0) / dd (side 1), added to Y
    const float *a_od, *ad_od, *cp_od;   // [F]
    const float *u_od;                   // U_od[c] at u_od[2c]
    const float *ad_same[2];             // [F]: oo (side 0), dd (side 1)
    float *S[2];                         // [rows][4][K]
    float *T;                            // device rows: [3][rows][F] packed (bit 0, bit 1) pairs
                                         // of the split3 parts (bf16, or F = 256), else fp32 [rows][2][F]
};
struct GemmArgs {
    GemmSide side[2];
    int64_t tiles0;      // row tiles of side 0
    int F;
    GemmPrep prep;
};

int64_t transform_row_tiles(int64_t rows);
void launch_transform(const GemmArgs &G, bool bf, hipStream_t st);

}  // namespace tag
