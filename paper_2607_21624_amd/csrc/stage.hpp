// stage.hpp -- R-Tile staging of token-major rows into LDS on gfx950.
//
// A tile is ROWS token rows of one head (D contiguous elements each, read at
// row_base + r*ss) placed in LDS without padding.  Each row is CPR 16-byte
// chunks; chunk c of row r is stored in slot c ^ swz(r).  The XOR swizzle is
// the intra-tile placement of the paper's R-Tile (section 4.2, intra-tile
// mapping): it is chosen so that both ways the kernels read a tile hit every
// LDS bank once per 256 bytes --
//   row reads      16 consecutive rows at one chunk (MFMA operands whose
//                  contraction runs along d), and
//   transposed     4 consecutive rows x 4 consecutive chunks per 32 lanes
//   reads          (ds_read_b64_tr_b16, operands contracted along tokens),
// which is the tile invariance of section 4.2 carried to the LDS banks.
//
// Tiles are filled with buffer_load_dwordx4 ... lds: each lane moves 16 bytes
// from global memory straight into LDS (no registers), so the next tile can be
// in flight while the current one is consumed.  The buffer resource covers
// exactly the rows of one (batch, head); rows beyond the sequence read as
// zeros, so ragged tails need no branches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "cdna4.hpp"

namespace fbl {

template <typename T, int D>
struct TileGeom {
    static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
    static constexpr int CPR = D / EPC;              // chunks per row

    // Chunk XOR of row r (values < CPR).
    static FBL_DEV int swz(int r) {
        if constexpr (sizeof(T) == 2) {
            if constexpr (CPR == 16) return ((r & 3) << 2) | ((r >> 2) & 3);
            else if constexpr (CPR == 8) return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
            else return (r >> 2) & 3;
        } else {
            if constexpr (CPR >= 16) return r & 15;
            else return (r >> 1) & 7;
        }
    }
    // Element offset of (row r, column col) inside a tile.
    static FBL_DEV int off(int r, int col) { return r * D + (((col / EPC) ^ swz(r)) * EPC) + (col % EPC); }
};

// Buffer resource (four SGPRs) over `bytes` bytes from `base`: raw, no
// swizzle, stride 0; loads past the end return zeros and touch no memory.
typedef int Rsrc __attribute__((ext_vector_type(4)));
FBL_DEV Rsrc make_rsrc(const void* base, uint32_t bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    return Rsrc{(int)(uint32_t)p, (int)((p >> 32) & 0xffffu), (int)bytes, 0x00020000};
}

// LDS DMA: every lane moves 16 (dma16) or 4 (dma4) bytes from buffer offset
// voff + soff straight into LDS at byte address lds + lane * size (the LDS
// address goes in M0).
//
// Issued as inline assembly on purpose.  The compiler cannot tell which LDS
// bytes a DMA writes, so after one of its own it makes the next LDS read of
// any address wait for every outstanding global load -- which would expose
// the full latency of the prefetch of the next tile in every loop iteration.
// The kernels order these writes against their reads themselves: they wait
// for their own loads (s_waitcnt vmcnt) and then meet at a workgroup barrier
// before any wave reads the tile.  Extra loads the compiler does not know of
// only make its own vmcnt waits stricter (loads retire in order).
// Wait states: s_nop 0 after the M0 write (1 before an LDS DMA); the first
// load of a batch also gets s_nop 4, for an SGPR operand written by a vector
// instruction just before it (5 wait states).  Later loads of the batch reuse
// operands the first one has already read.
template <bool FIRST = true>
FBL_DEV void dma16(Rsrc rs, uint32_t lds, uint32_t voff, uint32_t soff) {
    if constexpr (FIRST)
        asm volatile("s_nop 4\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                     :
                     : "v"(voff), "s"(rs), "s"(soff), "{m0}"(lds)
                     : "memory");
    else
        asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                     :
                     : "v"(voff), "s"(rs), "s"(soff), "{m0}"(lds)
                     : "memory");
}
// dma16 for data read exactly once: the non-temporal hint keeps it from
// displacing reused tiles in L2.
FBL_DEV void dma16_stream(Rsrc rs, uint32_t lds, uint32_t voff, uint32_t soff) {
    asm volatile("s_nop 4\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen nt lds"
                 :
                 : "v"(voff), "s"(rs), "s"(soff), "{m0}"(lds)
                 : "memory");
}
FBL_DEV void dma4(Rsrc rs, uint32_t lds, uint32_t voff, uint32_t soff) {
    asm volatile("s_nop 4\n\ts_nop 0\n\tbuffer_load_dword %0, %1, %2 offen lds"
                 :
                 : "v"(voff), "s"(rs), "s"(soff), "{m0}"(lds)
                 : "memory");
}

// Wait until at most N vector-memory loads of this wave are outstanding.
template <int N>
FBL_DEV void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4]=7 | lgkmcnt[11:8]=15 | vmcnt[5:4]<<14
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Row fragment (8 consecutive elements from column `col`, col % 8 == 0) of
// row r of a staged tile.
template <int D>
FBL_DEV void tile_row_frag(Frag<bf16>& f, const bf16* tile, int r, int col) {
    using G = TileGeom<bf16, D>;
    f.v = *(const FBL_LDS bf16x8*)(tile + G::off(r, col));
}
template <int D>
FBL_DEV void tile_row_frag(Frag<float>& f, const float* tile, int r, int col) {
    using G = TileGeom<float, D>;
    const f32x4 a = *(const FBL_LDS f32x4*)(tile + G::off(r, col));
    const f32x4 b = *(const FBL_LDS f32x4*)(tile + G::off(r, col + 4));
#pragma unroll
    for (int e = 0; e < 4; ++e) { f.v[e] = a[e]; f.v[4 + e] = b[e]; }
}

// Transposed fragment: lane l gets column col0 + (l % 32) at rows
// row0 + [0..3] (elements 0..3) and row1 + [0..3] (elements 4..7).
// row0/row1 are multiples of 4 and uniform over each 16-lane group.
template <int D>
FBL_DEV void tile_tr_frag(Frag<bf16>& f, const bf16* tile, int row0, int row1, int col0, int lane) {
    using G = TileGeom<bf16, D>;
    const int t = lane & 15;
    const int col = col0 + 16 * ((lane >> 4) & 1) + 4 * (t & 3);
    const bf16* p0 = tile + G::off(row0 + (t >> 2), col);
    const bf16* p1 = tile + G::off(row1 + (t >> 2), col);
    const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FBL_LDS bf16x4*)p0);
    const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FBL_LDS bf16x4*)p1);
    f.v = bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}
template <int D>
FBL_DEV void tile_tr_frag(Frag<float>& f, const float* tile, int row0, int row1, int col0, int lane) {
    using G = TileGeom<float, D>;
    const int col = col0 + (lane & 31);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f.v[e] = tile[G::off(row0 + e, col)];
        f.v[4 + e] = tile[G::off(row1 + e, col)];
    }
}

// Per-lane LDS byte addresses of the bf16 fragment reads of a staged tile,
// computed once so every LDS read in the loops is "lane address +
// compile-time constant" (the constant goes into the instruction's
// immediate field).  Valid for any 16-row-aligned block of the tile because
// swz() depends on r mod 16 only.
//   row[c]     row fragment: row (lane % 32), columns 16c + 8g .. +7
//   tr[t][h]   transposed fragment: column 32t + (lane % 32), rows 8h + 4g + [0..3]
template <int D>
struct LaneOffsets {
    static constexpr int NC = D / 16;
    static constexpr int ND = D / 32;
    uint32_t row[NC];
    uint32_t tr[ND][2];
    FBL_DEV void init(uint32_t tile_base, int lane) {
        using G = TileGeom<bf16, D>;
        const int g = lane >> 5, c32 = lane & 31, t = lane & 15;
#pragma unroll
        for (int c = 0; c < NC; ++c) row[c] = tile_base + 2u * (uint32_t)G::off(c32, 16 * c + 8 * g);
#pragma unroll
        for (int tt = 0; tt < ND; ++tt)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int r = 8 * h + 4 * g + (t >> 2);
                const int col = 32 * tt + 16 * ((lane >> 4) & 1) + 4 * (t & 3);
                tr[tt][h] = tile_base + 2u * (uint32_t)G::off(r, col);
            }
    }
};

// LDS byte address of a shared-memory object (its offset in the workgroup's LDS).
FBL_DEV uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(const FBL_LDS void*)p; }

FBL_DEV bf16x8 lds_b128(uint32_t addr, uint32_t const_off) {
    return *(const FBL_LDS bf16x8*)(uintptr_t)(addr + const_off);
}
FBL_DEV bf16x4 lds_tr(uint32_t addr, uint32_t const_off) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FBL_LDS bf16x4*)(uintptr_t)(addr + const_off));
}

// DMA of a ROWS-row tile with per-lane global offsets computed once:
// voff[j] is the byte offset (relative to the tile's first row) of the chunk
// lane `lane` of wave `wave` moves in its j-th load.  The row origin goes in
// the scalar offset of each load.
template <typename T, int D, int ROWS, int NWAVES>
struct DmaPlan {
    using G = TileGeom<T, D>;
    static constexpr int INSTS = ROWS * G::CPR / 64;
    static constexpr int PER_WAVE = (INSTS + NWAVES - 1) / NWAVES;
    static_assert(INSTS >= 1, "a tile is at least one 1 KB load");
    uint32_t voff[PER_WAVE];
    FBL_DEV void init(uint32_t row_bytes, int wave, int lane) {
#pragma unroll
        for (int j = 0; j < PER_WAVE; ++j) {
            const int q = ((j * NWAVES + wave) % INSTS) * 64 + lane;
            const int r = q / G::CPR;
            const int c = (q % G::CPR) ^ G::swz(r);
            voff[j] = (uint32_t)r * row_bytes + (uint32_t)c * 16u;
        }
    }
    // Loads rows row0.. of the tile at LDS byte address `tile`.
    FBL_DEV void issue(uint32_t tile, Rsrc rs, uint32_t row0_bytes, int wave) const {
#pragma unroll
        for (int j = 0; j < PER_WAVE; ++j) {
            const int i = j * NWAVES + wave;
            if (INSTS % NWAVES == 0 || i < INSTS) {
                if (j == 0) dma16<true>(rs, tile + (uint32_t)i * 1024u, voff[j], row0_bytes);
                else dma16<false>(rs, tile + (uint32_t)i * 1024u, voff[j], row0_bytes);
            }
        }
    }
};

// Workgroup order for (rank, head) work items whose cost falls with rank (the
// causal schedule: rank 0 = heaviest block).  With at least 8 heads, XCD x
// (ids are dealt round-robin over the 8 XCDs, each with its own L2) serves
// heads x, x+8, x+16, ... and walks them rank-major -- rank 0 of all its
// heads, then rank 1, ... -- so the heaviest blocks of every head start first
// (longest-first list scheduling) while each head's tiles stay in one L2.
// With fewer heads, plain rank-major order over all XCDs.  Grid size:
// rank_major_grid(); returns false for padding ids.
FBL_DEV bool rank_major_item(int id, int nrank, int nhead, int& rank, int& head) {
    if (nhead < 8) {
        rank = id / nhead;
        head = id % nhead;
        return rank < nrank;
    }
    const int x = id % 8, i = id / 8;
    const int nh = (nhead - x + 7) / 8;  // heads served by XCD x
    rank = i / nh;
    head = x + 8 * (i % nh);
    return rank < nrank;
}
inline int rank_major_grid(int nrank, int nhead) {
    return nhead < 8 ? nrank * nhead : 8 * ((nhead + 7) / 8) * nrank;
}

// Map a linear workgroup id so that consecutive ids of the logical order land
// on the same XCD (ids are dealt round-robin over the 8 XCDs, each with its own
// L2): logical = (id % 8) * per_xcd + id / 8.  Returns -1 for padding ids.
FBL_DEV int xcd_logical_id(int id, int total, int padded_total) {
    const int per_xcd = padded_total / 8;
    const int logical = (id % 8) * per_xcd + id / 8;
    return logical < total ? logical : -1;
}

// f(integral_constant<int, I>) for I = 0, 1, ..., in order: a loop over LDS
// buffers whose index stays a compile-time constant (buffer offsets become
// instruction immediates).
template <int... I, typename F>
FBL_DEV __attribute__((always_inline)) void unroll_steps(std::integer_sequence<int, I...>, F&& f) {
    (f(std::integral_constant<int, I>{}), ...);
}

}  // namespace fbl
