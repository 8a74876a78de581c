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
struct GemmArgs {
    GemmSide side[2];
    int64_t tiles0;      // row tiles of side 0
    int F;
};

int64_t transform_row_tiles(int64_t rows);
void launch_transform(const GemmArgs &G, bool bf, hipStream_t st);

}  // namespace tag
