// attn_tiles.hpp -- tile configurations of the attention kernels (host and
// device), and the three progressive candidate filters of the paper's R-Tile
// shape generation (section 4.2, step 1, and the supplementary
// candidate-generation algorithm) read for gfx950.
//
// Each attention pass stages one kind of row tile of a token-major tensor
// into LDS -- the R-Tile of section 4.2, (tile rows x head dim) -- and gives
// each wavefront a block of rows it keeps in registers:
//   forward   K/V tiles of `cols` keys; each wavefront owns `per_wave`
//             queries (Q in registers), `waves` wavefronts per workgroup;
//   kv pass   Q/dO tiles of `cols` queries; each wavefront owns 32 keys (K, V
//             and the dK, dV accumulators in registers);
//   dQ pass   K tiles of 32 keys and the matching dS blocks; each wavefront
//             owns 32 queries; `bufs` LDS buffers (bufs - 1 steps in flight).
// The index into kAttnTiles is the tile id of the C ABI.
#pragma once

#include <stdint.h>

namespace fbl {

enum AttnPass { kAttnFwd = 0, kAttnKv = 1, kAttnDq = 2 };

struct AttnTile {
    int pass;
    int per_wave;  // rows a wavefront owns: queries (forward, dQ) or keys (kv)
    int cols;      // rows of the staged tile: keys (forward, dQ) or queries (kv)
    int waves;     // wavefronts per workgroup
    int occ;       // workgroups per CU the kernel is built for; 0: by head dim (attn_occ)
    int bufs;      // LDS buffers of the staged tiles
};

constexpr AttnTile kAttnTiles[] = {
    // forward: rows per workgroup = per_wave * waves
    {kAttnFwd, 32, 64, 4, 2, 2},  // 0: 128 queries, 64-key tiles, two workgroups per CU
    {kAttnFwd, 64, 32, 4, 1, 2},  // 1: 256 queries, 64 per wavefront (each K/V fragment feeds two products)
    {kAttnFwd, 32, 32, 4, 2, 2},  // 2: 128 queries, 32-key tiles
    {kAttnFwd, 32, 64, 8, 1, 2},  // 3: 256 queries over 8 wavefronts (two per SIMD share each tile)
    {kAttnFwd, 64, 32, 2, 2, 2},  // 4: 128 queries, 64 per wavefront, two workgroups per CU
    // kv pass: 128 keys per workgroup, 32 per wavefront
    {kAttnKv, 32, 32, 4, 0, 4},  // 5: 32-query Q/dO tiles
    {kAttnKv, 32, 64, 4, 1, 4},  // 6: 64-query Q/dO tiles
    // dQ pass from the stored dS: 32 * waves queries per workgroup
    {kAttnDq, 32, 32, 4, 0, 4},  // 7
    {kAttnDq, 32, 32, 8, 0, 4},  // 8
    {kAttnDq, 32, 32, 4, 0, 3},  // 9
    // kv pass, 64 keys per workgroup: two independent workgroups per CU
    {kAttnKv, 32, 32, 2, 0, 4},  // 10
};
constexpr int kAttnTileCount = (int)(sizeof(kAttnTiles) / sizeof(kAttnTiles[0]));

constexpr int attn_rows(const AttnTile& t) { return t.per_wave * t.waves; }

// LDS bytes of one workgroup at head dim D (bf16 tiles); the kernels
// static_assert that their layouts take exactly this much.
constexpr int attn_lds_bytes(const AttnTile& t, int D) {
    if (t.pass == kAttnFwd) return 4 * t.cols * D * 2;  // K0 K1 V0 V1
    if (t.pass == kAttnKv)  // per buffer a Q and a dO tile and 512 bytes of row statistics; a 256-byte sink
        return t.bufs * (2 * t.cols * D * 2 + 512) + 256;
    // dQ: per buffer each wavefront's 32x32 dS block and one 32-key K tile; a
    // 1 KB sink when the K tile has fewer 1 KB loads than there are wavefronts
    const int kinst = 32 * D * 2 / 1024;
    return t.bufs * (t.waves * 2048 + 32 * D * 2) + (kinst < t.waves ? 1024 : 0);
}

constexpr int kLdsPerCu = 160 * 1024;

// Workgroups per CU the kernel is built for.
constexpr int attn_occ(const AttnTile& t, int D) {
    if (t.occ) return t.occ;
    if (t.pass == kAttnKv)  // one wavefront per SIMD (two at D = 64 with 32-query tiles: the state fits 256 registers)
        return ((D == 64 && t.cols == 32) ? 2 : 1) * 4 / t.waves;
    return (2 * attn_lds_bytes(t, D) <= kLdsPerCu && t.waves == 4) ? 2 : 1;
}

// Registers per lane a wavefront of the tile needs at head dim D: the
// register-resident operands and accumulators plus the fragments in flight
// (a model of the kernels' allocation, used by the capacity filter C2).
// Also returned: the part the vector ALUs read (not MFMA accumulators), which
// must fit the 256 architectural VGPRs.
struct RegModel { int total, arch; };
constexpr RegModel attn_regs(const AttnTile& t, int D) {
    if (t.pass == kAttnFwd) {
        const int qt = t.per_wave / 32, kt = t.cols / 32;
        const int q = qt * D / 4, o = qt * D / 2, s = 2 * kt * qt * 16, p = kt * qt * 8;
        const int arch = q + s + p + 32 + 40;  // + fragments in flight, addresses and softmax state
        return {arch + o, arch};
    }
    if (t.pass == kAttnKv) {
        const int nqt = t.cols / 32;
        const int kv = D / 2, acc = D, sdp = 2 * nqt * 16, rowf = nqt * D / 4, trf = nqt * D / 4;
        const int arch = kv + sdp + rowf + trf + 40;
        return {arch + acc, arch};
    }
    const int acc = D / 2;  // dQ^T of 32 queries
    const int arch = 2 * D / 8 + 40;
    return {arch + acc, arch};
}

// ---- candidate filters (section 4.2, step 1), read for gfx950
// C1 compute alignment: whole 32x32 MFMA blocks per wavefront and per staged
//    tile, whole 16-deep MFMA chunks over the head dim, 2 to 8 wavefronts.
constexpr bool attn_c1(const AttnTile& t, int D) {
    return t.per_wave % 32 == 0 && t.cols % 32 == 0 && D % 16 == 0 && t.waves >= 2 && t.waves <= 8;
}
// C2 memory alignment and capacity: the workgroups a CU holds fit its 160 KB
//    of LDS; every staged row is whole 16-byte vector loads and every staged
//    tile whole 1 KB wavefront loads, spread evenly over the wavefronts; the
//    per-lane registers fit the register file share of a wavefront (512 per
//    SIMD lane, divided among the wavefronts a SIMD holds) with the vector
//    operands inside the 256 architectural registers.
constexpr bool attn_c2(const AttnTile& t, int D) {
    const int occ = attn_occ(t, D);
    const int per_simd = (t.waves * occ + 3) / 4;
    const RegModel r = attn_regs(t, D);
    const int tile_loads = t.cols * D * 2 / 1024;
    const bool even = t.pass == kAttnDq || (tile_loads >= t.waves ? tile_loads % t.waves == 0 : t.pass == kAttnFwd);
    return attn_lds_bytes(t, D) * occ <= kLdsPerCu && (D * 2) % 16 == 0 && (t.cols * D * 2) % 1024 == 0 && even &&
           r.total <= 512 / per_simd && r.arch <= 256;
}
// C3 shape: padding the sequence to whole workgroup row blocks (queries for
//    the forward and dQ passes, keys for the kv pass) and to whole staged
//    tiles adds at most 10%.
constexpr long long attn_padded(long long n, int tile) { return (n + tile - 1) / tile * tile; }
constexpr bool attn_c3(const AttnTile& t, long long Sq, long long Skv) {
    const long long rows_seq = t.pass == kAttnKv ? Skv : Sq, cols_seq = t.pass == kAttnKv ? Sq : Skv;
    const int rows = attn_rows(t);
    return 10 * (attn_padded(rows_seq, rows) - rows_seq) <= rows_seq &&
           10 * (attn_padded(cols_seq, t.cols) - cols_seq) <= cols_seq;
}
// padded work volume (C3's ranking when no tile meets the 10% bound)
constexpr double attn_padded_volume(const AttnTile& t, long long Sq, long long Skv) {
    const long long rows_seq = t.pass == kAttnKv ? Skv : Sq, cols_seq = t.pass == kAttnKv ? Sq : Skv;
    const int rows = attn_rows(t);
    return (double)attn_padded(rows_seq, rows) * (double)attn_padded(cols_seq, t.cols);
}

}  // namespace fbl
