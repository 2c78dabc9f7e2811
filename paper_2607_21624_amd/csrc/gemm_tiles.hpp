// gemm_tiles.hpp -- the output-tile configurations of the projection products
// (host and device).  A configuration fixes the workgroup's output tile
// (bm x bn), the contraction depth staged per step (bk) and the number of LDS
// stages (ns), and how the wavefronts share the tile: a wm x wn grid of
// wavefront tiles, each computed by wk wavefronts that split every step's
// contraction and add their partial sums at the end.
#pragma once

namespace fbl {

struct GemmTile {
    int bm, bn, bk, ns, wm, wn, wk;
};

// Index = the tile id of the C ABI.  Ids 0-3 are the named FBL_GEMM_TILE_*
// shapes.
constexpr GemmTile kGemmTiles[] = {
    {128, 128, 32, 3, 2, 2, 1},  // 0
    {128, 64, 32, 3, 2, 2, 1},   // 1
    {64, 128, 32, 3, 2, 2, 1},   // 2
    {64, 64, 32, 3, 2, 2, 1},    // 3
    {128, 128, 64, 3, 2, 2, 1},  // 4
    {128, 64, 64, 3, 2, 2, 1},   // 5
    {64, 128, 64, 3, 2, 2, 1},   // 6
    {64, 64, 64, 3, 2, 2, 1},    // 7
    {128, 128, 64, 4, 2, 2, 2},  // 8: 8 wavefronts, each 64 x 64 on half of every step
    {64, 64, 128, 3, 1, 1, 4},   // 9: 4 wavefronts, each the whole 64 x 64 on a quarter
    {128, 64, 128, 3, 2, 1, 4},  // 10: 8 wavefronts, each 64 x 64 on a quarter
    {256, 128, 64, 3, 2, 2, 2},  // 11: 8 wavefronts, each 128 x 64 on half
    {128, 256, 64, 3, 2, 2, 2},  // 12: 8 wavefronts, each 64 x 128 on half
    // narrow outputs (LoRA ranks): 32 columns or rows
    {128, 32, 64, 3, 4, 1, 1},   // 13
    {64, 32, 128, 3, 2, 1, 2},   // 14: each wavefront 32 x 32 on half
    {32, 128, 64, 3, 1, 4, 1},   // 15
    {32, 32, 128, 3, 1, 1, 4},   // 16: each wavefront the whole 32 x 32 on a quarter
    // large products: 4 wavefronts of 128 x 128 (the accumulators fill the AGPRs)
    {256, 256, 32, 4, 2, 2, 1},  // 17
    {256, 256, 64, 2, 2, 2, 1},  // 18
    // large products, 8 wavefronts (two per SIMD) of 128 x 64 or 64 x 128
    {256, 256, 64, 2, 2, 4, 1},  // 19
    {256, 256, 64, 2, 4, 2, 1},  // 20
};
constexpr int kGemmTileCount = (int)(sizeof(kGemmTiles) / sizeof(kGemmTiles[0]));

constexpr int gemm_waves(const GemmTile& t) { return t.wm * t.wn * t.wk; }

// LDS bytes of one workgroup: the stages, or the partial sums of the
// wavefronts that split the contraction, whichever is larger.
constexpr int gemm_lds_bytes(const GemmTile& t) {
    const int stages = t.ns * (t.bm + t.bn) * t.bk * 2;
    const int partial = (t.wk - 1) * t.bm * t.bn * 4;
    return stages > partial ? stages : partial;
}

}  // namespace fbl

namespace fbl {

// Candidate filter for the tile of one product (the three progressive filters
// of section 4.2, step 1, and the supplementary candidate-generation
// algorithm), read for gfx950:
//   C1 compute alignment: wavefront tiles of whole 32x32 MFMA blocks, each
//      step split into whole 16-deep MFMA chunks per wavefront;
//   C2 memory alignment: the workgroup's LDS fits in the 160 KB of a CU, and
//      every staged row is a whole number of 128-byte cache lines (a row-read
//      operand stages bk elements per row, a transposed one bm or bn) or
//      spans the operand's whole stored row (narrower than a line);
//   C3 shape: padding the output rows, columns and the contraction to whole
//      tiles adds at most 10% to each; when no tile meets that, the tiles of
//      least padded volume are kept.
constexpr int kGemmLdsBytes = 160 * 1024;
constexpr int kCacheLineBytes = 128;

constexpr bool gemm_c1(const GemmTile& t) {
    return t.bm % (32 * t.wm) == 0 && t.bn % (32 * t.wn) == 0 && (t.bk / 16) % t.wk == 0 &&
           (gemm_waves(t) == 4 || gemm_waves(t) == 8);
}
// a_kmajor / b_nmajor: how the product stores its operands (see proj_gemm.hip);
// a_width / b_width: elements per stored row of A and B
constexpr bool gemm_c2(const GemmTile& t, bool a_kmajor, bool b_nmajor, long long a_width, long long b_width) {
    const long long a_row = (a_kmajor ? t.bm : t.bk) * 2, b_row = (b_nmajor ? t.bk : t.bn) * 2;
    return gemm_lds_bytes(t) <= kGemmLdsBytes && (a_row % kCacheLineBytes == 0 || a_row >= 2 * a_width) &&
           (b_row % kCacheLineBytes == 0 || b_row >= 2 * b_width);
}
constexpr long long gemm_padded(long long n, int tile) { return (n + tile - 1) / tile * tile; }
constexpr bool gemm_c3(const GemmTile& t, long long rows, long long cols, long long kc) {
    return 10 * (gemm_padded(rows, t.bm) - rows) <= rows && 10 * (gemm_padded(cols, t.bn) - cols) <= cols &&
           10 * (gemm_padded(kc, t.bk) - kc) <= kc;
}
// padded volume (C3's fallback ranking)
constexpr double gemm_padded_volume(const GemmTile& t, long long rows, long long cols, long long kc) {
    return (double)gemm_padded(rows, t.bm) * (double)gemm_padded(cols, t.bn) * (double)gemm_padded(kc, t.bk);
}

}  // namespace fbl
