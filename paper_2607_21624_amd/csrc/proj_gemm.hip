// proj_gemm.hip -- projection matrix products on token-major operands, bf16,
// gfx950.
//
// One kernel template computes C[M, N] = sum_k A(m, k) B(k, n) (fp32
// accumulation, bf16 result) for the three products of a linear layer:
//   forward          Y  = X W      A = X  [M, K] rows,   B = W  [K, N] rows
//   data gradient    dX = dY W^T   A = dY [M, N] rows,   B = W read as [N, K]
//   weight gradient  dW = X^T dY   A = X read as [K, M], B = dY [M, N] rows
// Section 4.1 classes these as forward-tensor-dependent: the gradients read
// the stored X, W and dY along other axes than the forward (section 4.2: the
// forward reduces along K, the gradients along N and along the tokens M).
// No operand is ever transposed in memory.  Each operand tile is staged once
// into LDS by DMA in its stored orientation (the R-Tile of section 4.2, with
// the XOR swizzle of stage.hpp) and read back either
//   row-wise      (ds_read_b128: 8 consecutive elements of one stored row)
//                 when the contraction runs along the stored rows, or
//   transposed    (ds_read_b64_tr_b16: one element of each of 4 stored rows)
//                 when it runs down the stored columns.
// Both read kinds hand lane group g (lane / 32) contraction elements
// 8g .. 8g+7 of a 16-element chunk, in order, so any pair of them forms a
// consistent MFMA operand pair.
//
// Extents need not be multiples of the tile.  Operand rows past the end of
// an operand read as zeros (buffer resources bound each operand's span);
// columns past an operand's width read whatever follows in memory, which
// only ever meets output rows/columns that are not stored -- and, along the
// contraction, the positions of a partial last step, which are zeroed in LDS
// before that step's products.
//
// Workgroup (gemm_tiles.hpp): a WM x WN grid of wavefront tiles over a
// BM x BN output tile, each computed by WK wavefronts that split every step's
// contraction; BK-deep steps through NS LDS stages (NS - 1 in flight).  The
// WK partial sums of a wavefront tile are added through LDS at the end, in a
// fixed order.  The products accumulate C^T tiles (lane <-> m, in-lane n), so
// each lane stores four consecutive outputs of a row.
#include <array>
#include <type_traits>
#include <utility>

#include "cdna4.hpp"
#include "gemm_tiles.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace fbl {

namespace {

// LDS tile of ROWS stored rows of COLS bf16 elements (swizzled as in stage.hpp),
// loaded by NW wavefronts.
template <int ROWS, int COLS, int NW>
struct GTile {
    using G = TileGeom<bf16, COLS>;
    using Dma = DmaPlan<bf16, COLS, ROWS, NW>;
    static constexpr int BYTES = ROWS * COLS * 2;
    // every wavefront issues the same number of loads, so one vmcnt count fits all
    static_assert(Dma::INSTS % NW == 0, "whole 1 KB loads per wavefront");
    // row read: stored row r (lane % 32 + 32 * tile), columns 16c + 8g .. +7
    static FBL_DEV uint32_t row_addr(int lane, int c) {
        return 2u * (uint32_t)G::off(lane & 31, 16 * c + 8 * (lane >> 5));
    }
    // transposed read, natural order: stored rows 8g + 4h + [0..3] (plus 16kc),
    // column 32t + lane % 32
    static FBL_DEV uint32_t tr_addr(int lane, int t, int h) {
        const int q = lane & 15;
        const int r = 8 * (lane >> 5) + 4 * h + (q >> 2);
        const int col = 32 * t + 16 * ((lane >> 4) & 1) + 4 * (q & 3);
        return 2u * (uint32_t)G::off(r, col);
    }
};

// AT: A stored k-major ([K, M] rows); BT: B stored n-major ([N, K] rows).
template <int BM, int BN, int BK, int NS, int WM, int WN, int WK, bool AT, bool BT>
struct GemmCfg {
    static constexpr int NW = WM * WN * WK;
    using TA = GTile<AT ? BK : BM, AT ? BM : BK, NW>;
    using TB = GTile<BT ? BN : BK, BT ? BK : BN, NW>;
    static constexpr int TM = BM / (32 * WM), TN = BN / (32 * WN);  // 32x32 tiles per wavefront
    static constexpr int NKC = BK / 16;                              // 16-deep MFMA chunks per step
    static constexpr int KCW = NKC / WK;                             // chunks per wavefront per step
    static constexpr int SA = TA::BYTES, SB = TB::BYTES;
    static constexpr int STAGE = SA + SB;
    static constexpr int BYTES = gemm_lds_bytes(GemmTile{BM, BN, BK, NS, WM, WN, WK});
    static constexpr int LOADS = TA::Dma::PER_WAVE + TB::Dma::PER_WAVE;
    static constexpr int PART = TM * TN * 4096;  // bytes of one wavefront's partial sums
    static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "wavefront tiles of whole 32x32 blocks");
    static_assert(BK % 32 == 0 && NKC % WK == 0 && NS >= 2, "whole chunks per wavefront, at least double buffered");
    static_assert(NW == 4 || NW == 8, "4 or 8 wavefronts");
    // stage offsets are added at run time; the read immediates are tile offsets within a stage
    static_assert((TM - 1) * 32 * BK * 2 < 65536 && (TN - 1) * 32 * BK * 2 < 65536 &&
                      (KCW - 1) * 16 * (BM > BN ? BM : BN) * 2 + 128 < 65536,
                  "LDS read immediates fit 16 bits");
    static_assert(BYTES <= 160 * 1024 && NS * STAGE <= BYTES && (WK - 1) * WM * WN * PART <= BYTES, "LDS");
    static_assert((NS - 1) * LOADS < 64, "vmcnt range");
    static constexpr int OCC = (NW == 4 && BYTES <= 80 * 1024) ? 2 : 1;
};

template <int BM, int BN, int BK, int NS, int WM, int WN, int WK, bool AT, bool BT>
__global__ __launch_bounds__(64 * WM * WN * WK, (GemmCfg<BM, BN, BK, NS, WM, WN, WK, AT, BT>::OCC)) void
proj_gemm_bf16(GemmArgs p) {
    using C = GemmCfg<BM, BN, BK, NS, WM, WN, WK, AT, BT>;
    using TA = typename C::TA;
    using TB = typename C::TB;
    constexpr int TM = C::TM, TN = C::TN, KCW = C::KCW;
    extern __shared__ __attribute__((aligned(1024))) unsigned char gemm_smem[];
    const uint32_t lds = lds_addr(gemm_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    // wavefront position: (wm, wn) in the tile grid, wk = its share of each step
    const int wm = wave % WM, wn = (wave / WM) % WN, wk = wave / (WM * WN);
    const int mt = (p.M + BM - 1) / BM, nt = (p.N + BN - 1) / BN;
    // consecutive ids share a column block of B (the weight) and land on one XCD
    const int logical = xcd_logical_id(blockIdx.x, mt * nt, gridDim.x);
    if (logical < 0) return;
    const int m0 = (logical % mt) * BM, n0 = (logical / mt) * BN;
    const int nk = (p.K + BK - 1) / BK;

    // ---- DMA: each stage holds the A and B tiles of one BK-deep step
    const Rsrc ra = make_rsrc(p.a, p.a_bytes), rb = make_rsrc(p.b, p.b_bytes);
    typename TA::Dma da;
    typename TB::Dma db;
    da.init((uint32_t)(p.lda * 2), wave, lane);
    db.init((uint32_t)(p.ldb * 2), wave, lane);
    auto issue = [&](int s, int buf) __attribute__((always_inline)) {
        const int k0 = s * BK;
        const uint32_t sa = (uint32_t)((AT ? (int64_t)k0 * p.lda + m0 : (int64_t)m0 * p.lda + k0) * 2);
        const uint32_t sb = (uint32_t)((BT ? (int64_t)n0 * p.ldb + k0 : (int64_t)k0 * p.ldb + n0) * 2);
        da.issue(lds + buf * C::STAGE, ra, sa, wave);
        db.issue(lds + buf * C::STAGE + C::SA, rb, sb, wave);
    };

    // ---- per-lane LDS read addresses (stage 0, the wavefront's first chunk)
    const int kc0 = wk * KCW;
    uint32_t aaddr[AT ? TM : KCW][2], baddr[BT ? KCW : TN][2];
    if constexpr (AT) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                aaddr[tm][h] = lds + TA::tr_addr(lane, wm * TM + tm, h) + (uint32_t)(kc0 * 16 * BM * 2);
    } else {
#pragma unroll
        for (int j = 0; j < KCW; ++j) aaddr[j][0] = lds + TA::row_addr(lane, kc0 + j);
    }
    if constexpr (BT) {
#pragma unroll
        for (int j = 0; j < KCW; ++j) baddr[j][0] = lds + C::SA + TB::row_addr(lane, kc0 + j);
    } else {
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                baddr[tn][h] = lds + C::SA + TB::tr_addr(lane, wn * TN + tn, h) + (uint32_t)(kc0 * 16 * BN * 2);
    }
    const uint32_t arow = (uint32_t)(wm * TM * 32 * BK * 2), brow = (uint32_t)(wn * TN * 32 * BK * 2);
    // fragment of A for m-tile tm, the wavefront's chunk j, from the stage at
    // byte offset `stage` (a run-time, wave-uniform value added to the address)
    auto frag_a = [&](uint32_t stage, int tm, int j) __attribute__((always_inline)) {
        Frag<bf16> f;
        if constexpr (AT) {
            const uint32_t off = j * 16 * BM * 2;
            const bf16x4 x = lds_tr(aaddr[tm][0] + stage, off), y = lds_tr(aaddr[tm][1] + stage, off);
            f.v = bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
        } else {
            f.v = lds_b128(aaddr[j][0] + stage + arow, tm * 32 * BK * 2);
        }
        return f;
    };
    auto frag_b = [&](uint32_t stage, int tn, int j) __attribute__((always_inline)) {
        Frag<bf16> f;
        if constexpr (BT) {
            f.v = lds_b128(baddr[j][0] + stage + brow, tn * 32 * BK * 2);
        } else {
            const uint32_t off = j * 16 * BN * 2;
            const bf16x4 x = lds_tr(baddr[tn][0] + stage, off), y = lds_tr(baddr[tn][1] + stage, off);
            f.v = bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
        }
        return f;
    };

    // C^T accumulators: acc[tn][tm] rows = n (acc_row), columns = m (lane)
    f32x16 acc[TN][TM];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) acc[tn][tm] = f32x16{};

    // Step s: wait until step s has landed (the NS - 2 later steps may still
    // be in flight), meet, refill the stage step s-1 used with step s+NS-1,
    // then contract the wavefront's chunks of step s.
    auto wait_step = [&](int s) __attribute__((always_inline)) {
        const int later = min(NS - 2, nk - 1 - s);  // steps issued after step s
        if constexpr (NS >= 5) {
            if (later >= 3) { wait_vmcnt<(NS >= 5 ? 3 : 0) * C::LOADS>(); return; }
        }
        if constexpr (NS >= 4) {
            if (later == 2) { wait_vmcnt<(NS >= 4 ? 2 : 0) * C::LOADS>(); return; }
        }
        if constexpr (NS >= 3) {
            if (later == 1) { wait_vmcnt<C::LOADS>(); return; }
        }
        wait_vmcnt<0>();
    };
    static_assert(NS <= 5, "wait_step covers at most three steps in flight behind the awaited one");
    for (int s = 0; s < NS - 1 && s < nk; ++s) issue(s, s);
    // The last step may hold the end of the contraction (krem < BK elements
    // left, a multiple of 8).  Once its tiles have landed, the workgroup
    // zeroes their contraction positions krem .. BK-1 in LDS (whatever the
    // loads brought there: zeros past an operand's last row, or the next
    // row's elements past its width), so the products run unchanged.
    auto zero_tail = [&](uint32_t stage, int krem) __attribute__((always_inline)) {
        const int tid = threadIdx.x;
        constexpr int NT = 64 * C::NW;
        const f32x4 z = f32x4{};
        // operand tile with the contraction along its stored rows (AT / not BT): whole rows
        auto rows = [&](uint32_t tile, int cols) __attribute__((always_inline)) {
            const int n16 = (BK - krem) * cols / 8;  // 16-byte chunks past row krem
            for (int i = tid; i < n16; i += NT)
                *(FBL_LDS f32x4*)(uintptr_t)(tile + (uint32_t)(krem * cols * 2 + i * 16)) = z;
        };
        // operand tile with the contraction along its stored columns: chunks krem/8 .. of every row
        auto cols = [&](uint32_t tile, int nrows, auto geom) __attribute__((always_inline)) {
            using G = decltype(geom);
            const int per = (BK - krem) / 8;
            for (int i = tid; i < nrows * per; i += NT) {
                const int r = i / per, c = krem / 8 + i % per;
                *(FBL_LDS f32x4*)(uintptr_t)(tile + 2u * (uint32_t)G::off(r, 8 * c)) = z;
            }
        };
        const uint32_t ta = lds + stage, tb = lds + stage + C::SA;
        if constexpr (AT) rows(ta, BM);
        else cols(ta, BM, typename TA::G{});
        if constexpr (BT) cols(tb, BN, typename TB::G{});
        else rows(tb, BN);
    };
    int buf = 0;
    const int nfull = p.K / BK;  // steps wholly inside the contraction
    for (int s = 0; s < nk; ++s) {
        wait_step(s);
        __syncthreads();
        if (s + NS - 1 < nk) issue(s + NS - 1, buf == 0 ? NS - 1 : buf - 1);
        const uint32_t stage = (uint32_t)buf * C::STAGE;
        if (s == nfull) {  // the partial last step (every load of it has landed: nothing is in flight)
            zero_tail(stage, p.K - s * BK);
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < KCW; ++j) {
            Frag<bf16> fa[TM], fb[TN];
#pragma unroll
            for (int tm = 0; tm < TM; ++tm) fa[tm] = frag_a(stage, tm, j);
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) fb[tn] = frag_b(stage, tn, j);
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm) mma(acc[tn][tm], fb[tn], fa[tm]);
        }
        buf = buf + 1 == NS ? 0 : buf + 1;
    }

    if constexpr (WK > 1) {
        // Partial sums: wavefront (wm, wn, wk > 0) parks its accumulators in LDS
        // (the stages are free once every wavefront has passed the barrier
        // after its last step, whose loads it waited for in full); the wk = 0
        // wavefront of the tile adds them in the order wk = 1, 2, ... and stores.
        // Layout per wavefront: [tn][tm][quad][lane] x 16 bytes.
        __syncthreads();
        const uint32_t part0 = lds + (uint32_t)((wn * WM + wm) * C::PART);
        constexpr uint32_t kSlot = (uint32_t)(WM * WN * C::PART);
        if (wk > 0) {
            const uint32_t mine = part0 + (uint32_t)(wk - 1) * kSlot;
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm)
#pragma unroll
                    for (int qd = 0; qd < 4; ++qd) {
                        const uint32_t a = mine + (uint32_t)((((tn * TM + tm) * 4 + qd) * 64 + lane) * 16);
                        *(FBL_LDS f32x4*)(uintptr_t)a = f32x4{acc[tn][tm][4 * qd], acc[tn][tm][4 * qd + 1],
                                                              acc[tn][tm][4 * qd + 2], acc[tn][tm][4 * qd + 3]};
                    }
        }
        __syncthreads();
        if (wk > 0) return;
#pragma unroll
        for (int w = 1; w < WK; ++w) {
            const uint32_t theirs = part0 + (uint32_t)(w - 1) * kSlot;
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm)
#pragma unroll
                    for (int qd = 0; qd < 4; ++qd) {
                        const uint32_t a = theirs + (uint32_t)((((tn * TM + tm) * 4 + qd) * 64 + lane) * 16);
                        const f32x4 v = *(const FBL_LDS f32x4*)(uintptr_t)a;
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[tn][tm][4 * qd + e] += v[e];
                    }
        }
    }

    // C[m][n .. n+3]: lane <-> m, four consecutive n per store (N is a
    // multiple of 4, so a store is wholly inside or wholly outside).  Stores
    // outside the output go to an offset past the buffer's range, which the
    // hardware drops -- no divergent branches around the stores.
    using i32x2 = int __attribute__((ext_vector_type(2)));
    const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(p.c, 0, (int)p.c_bytes, 0x00020000);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
        const int m = m0 + (wm * TM + tm) * 32 + (lane & 31);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int n = n0 + (wn * TN + tn) * 32 + 8 * rr + 4 * g;
                const uint32_t off = m < p.M && n < p.N ? (uint32_t)(((int64_t)m * p.ldc + n) * 2) : 0x80000000u;
                const bf16x4 v = bf16x4{(bf16)acc[tn][tm][4 * rr], (bf16)acc[tn][tm][4 * rr + 1],
                                        (bf16)acc[tn][tm][4 * rr + 2], (bf16)acc[tn][tm][4 * rr + 3]};
                __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(i32x2, v), crs, off, 0, 0);
            }
    }
}

template <int I, bool AT, bool BT>
hipError_t launch_id(const GemmArgs& p, hipStream_t stream) {
    constexpr GemmTile t = kGemmTiles[I];
    using C = GemmCfg<t.bm, t.bn, t.bk, t.ns, t.wm, t.wn, t.wk, AT, BT>;
    constexpr auto kernel = &proj_gemm_bf16<t.bm, t.bn, t.bk, t.ns, t.wm, t.wn, t.wk, AT, BT>;
    const hipError_t once = ensure_dynamic_lds<kernel>(C::BYTES);
    if (once != hipSuccess) return once;
    const int tiles = ((p.M + t.bm - 1) / t.bm) * ((p.N + t.bn - 1) / t.bn);
    hipLaunchKernelGGL(kernel, dim3((tiles + 7) / 8 * 8), dim3(64 * C::NW), C::BYTES, stream, p);
    return hipGetLastError();
}

using Launcher = hipError_t (*)(const GemmArgs&, hipStream_t);

template <bool AT, bool BT, int... I>
constexpr std::array<Launcher, sizeof...(I)> launchers(std::integer_sequence<int, I...>) {
    return {&launch_id<I, AT, BT>...};
}

template <bool AT, bool BT>
hipError_t launch_tile(int tile, const GemmArgs& p, hipStream_t stream) {
    static constexpr auto table = launchers<AT, BT>(std::make_integer_sequence<int, kGemmTileCount>{});
    return table[tile](p, stream);
}

}  // namespace

hipError_t launch_proj_gemm(int a_kmajor, int b_nmajor, int tile, const GemmArgs& p, hipStream_t stream) {
    if (tile < 0 || tile >= kGemmTileCount) return hipErrorInvalidValue;
    if (a_kmajor) return b_nmajor ? launch_tile<true, true>(tile, p, stream) : launch_tile<true, false>(tile, p, stream);
    return b_nmajor ? launch_tile<false, true>(tile, p, stream) : launch_tile<false, false>(tile, p, stream);
}

}  // namespace fbl
