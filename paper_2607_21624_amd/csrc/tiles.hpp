// tiles.hpp -- R-Tile shape table for gfx950.
//
// The paper prunes tile-shape candidates with three progressive filters
// (section 4.2, step 1, and the supplementary candidate-generation algorithm):
// C1 computation alignment (warp size, ISA), C2 memory alignment (cache
// capacity, cache-line boundaries), C3 tensor-shape compatibility (padding at
// most 10%).  On gfx950 the same three filters read:
//   C1  rows a multiple of 32 (one MFMA 32x32 operand block per wavefront
//       half) and columns a multiple of 16 (one MFMA k-chunk);
//   C2  a staged K+V tile pair, rows padded by 16 bytes against LDS bank
//       conflicts, fits in half of the 160 KB LDS (two workgroups per CU),
//       and each row is a whole number of 16-byte vector loads;
//   C3  padding of the sequence to whole tiles at most 10% when S is known.
// tile_rows() returns the row count the forward kernel stages, which is the
// largest C1/C2 survivor up to 64 rows.
#pragma once

#include <stdint.h>

namespace fbl {

constexpr int64_t kLdsBytes = 160 * 1024;

constexpr bool tile_c1(int64_t rows, int64_t cols) { return rows % 32 == 0 && cols % 16 == 0; }

constexpr bool tile_c2(int64_t rows, int64_t cols, int64_t elem) {
    return (cols * elem) % 16 == 0 && 2 * rows * (cols * elem + 16) <= kLdsBytes / 2;
}

constexpr bool tile_c3(int64_t rows, int64_t seq) {
    if (seq <= 0) return true;
    const int64_t padded = (seq + rows - 1) / rows * rows;
    return (padded - seq) * 10 <= seq;
}

inline int32_t tile_rows(int64_t D, int32_t dtype) {
    const int64_t elem = dtype == 1 ? 2 : 4;
    int32_t best = 32;
    for (int64_t rows = 32; rows <= 64; rows += 32)
        if (tile_c1(rows, D) && tile_c2(rows, D, elem)) best = (int32_t)rows;
    return best;
}

}  // namespace fbl
