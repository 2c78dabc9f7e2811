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
// Workgroup: 4 wavefronts in a 2 x 2 grid over a BM x BN output tile, 32-deep
// contraction steps, three LDS stages (two in flight), two workgroups per CU.
// The products accumulate C^T tiles (lane <-> m, in-lane n), so each lane
// stores four consecutive outputs of a row.
#include <type_traits>

#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace fbl {

namespace {

constexpr int kGemmBK = 32;  // contraction elements per step
constexpr int kGemmStages = 3;

// LDS tile of ROWS stored rows of COLS bf16 elements (swizzled as in stage.hpp).
template <int ROWS, int COLS>
struct GTile {
    using G = TileGeom<bf16, COLS>;
    using Dma = DmaPlan<bf16, COLS, ROWS, 4>;
    static constexpr int BYTES = ROWS * COLS * 2;
    static_assert(Dma::INSTS % 4 == 0, "whole 1 KB loads per wavefront");
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
template <int BM, int BN, bool AT, bool BT>
struct GemmCfg {
    using TA = GTile<AT ? kGemmBK : BM, AT ? BM : kGemmBK>;
    using TB = GTile<BT ? BN : kGemmBK, BT ? kGemmBK : BN>;
    static constexpr int TM = BM / 64, TN = BN / 64;  // 32x32 tiles per wavefront
    static constexpr int SA = TA::BYTES, SB = TB::BYTES;
    static constexpr int STAGE = SA + SB;
    static constexpr int BYTES = kGemmStages * STAGE;
    static constexpr int LOADS = TA::Dma::PER_WAVE + TB::Dma::PER_WAVE;
    static_assert(BM % 64 == 0 && BN % 64 == 0, "2 x 2 wavefronts of 32-multiples");
    static_assert(kGemmStages * STAGE < 65536, "stage offsets fit the 16-bit LDS immediate");
};

template <int BM, int BN, bool AT, bool BT>
__global__ __launch_bounds__(256, 2) void proj_gemm_bf16(GemmArgs p) {
    using C = GemmCfg<BM, BN, AT, BT>;
    using TA = typename C::TA;
    using TB = typename C::TB;
    constexpr int TM = C::TM, TN = C::TN;
    extern __shared__ __attribute__((aligned(1024))) unsigned char gemm_smem[];
    const uint32_t lds = lds_addr(gemm_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int wm = wave & 1, wn = wave >> 1;  // wavefront position in the 2 x 2 grid
    const int mt = p.M / BM, nt = p.N / BN;
    // consecutive ids share a column block of B (the weight) and land on one XCD
    const int logical = xcd_logical_id(blockIdx.x, mt * nt, gridDim.x);
    if (logical < 0) return;
    const int m0 = (logical % mt) * BM, n0 = (logical / mt) * BN;
    const int nk = p.K / kGemmBK;

    // ---- DMA: each stage holds the A and B tiles of one 32-deep step
    const Rsrc ra = make_rsrc(p.a, p.a_bytes), rb = make_rsrc(p.b, p.b_bytes);
    typename TA::Dma da;
    typename TB::Dma db;
    da.init((uint32_t)(p.lda * 2), wave, lane);
    db.init((uint32_t)(p.ldb * 2), wave, lane);
    auto issue = [&](int s, int buf) __attribute__((always_inline)) {
        const int k0 = s * kGemmBK;
        const uint32_t sa = (uint32_t)((AT ? (int64_t)k0 * p.lda + m0 : (int64_t)m0 * p.lda + k0) * 2);
        const uint32_t sb = (uint32_t)((BT ? (int64_t)n0 * p.ldb + k0 : (int64_t)k0 * p.ldb + n0) * 2);
        da.issue(lds + buf * C::STAGE, ra, sa, wave);
        db.issue(lds + buf * C::STAGE + C::SA, rb, sb, wave);
    };

    // ---- per-lane LDS read addresses (stage 0, contraction chunk 0)
    uint32_t aaddr[AT ? TM : 2][2], baddr[BT ? 2 : TN][2];
    if constexpr (AT) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int h = 0; h < 2; ++h) aaddr[tm][h] = lds + TA::tr_addr(lane, wm * TM + tm, h);
    } else {
#pragma unroll
        for (int c = 0; c < 2; ++c) aaddr[c][0] = lds + TA::row_addr(lane, c);
    }
    if constexpr (BT) {
#pragma unroll
        for (int c = 0; c < 2; ++c) baddr[c][0] = lds + C::SA + TB::row_addr(lane, c);
    } else {
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int h = 0; h < 2; ++h) baddr[tn][h] = lds + C::SA + TB::tr_addr(lane, wn * TN + tn, h);
    }
    // fragment of A for m-tile tm, contraction chunk kc, from stage buffer B
    auto frag_a = [&](auto buf_c, int tm, int kc) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        Frag<bf16> f;
        if constexpr (AT) {
            const uint32_t off = B * C::STAGE + kc * 16 * BM * 2;
            const bf16x4 x = lds_tr(aaddr[tm][0], off), y = lds_tr(aaddr[tm][1], off);
            f.v = bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
        } else {
            f.v = lds_b128(aaddr[kc][0], B * C::STAGE + (wm * TM + tm) * 32 * kGemmBK * 2);
        }
        return f;
    };
    auto frag_b = [&](auto buf_c, int tn, int kc) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        Frag<bf16> f;
        if constexpr (BT) {
            f.v = lds_b128(baddr[kc][0], B * C::STAGE + (wn * TN + tn) * 32 * kGemmBK * 2);
        } else {
            const uint32_t off = B * C::STAGE + kc * 16 * BN * 2;
            const bf16x4 x = lds_tr(baddr[tn][0], off), y = lds_tr(baddr[tn][1], off);
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

    auto step = [&](auto buf_c, int s) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        if (s + 1 < nk) wait_vmcnt<C::LOADS>();  // step s landed; step s+1 may be in flight
        else wait_vmcnt<0>();
        __syncthreads();
        if (s + 2 < nk) issue(s + 2, (B + 2) % kGemmStages);
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            Frag<bf16> fa[TM], fb[TN];
#pragma unroll
            for (int tm = 0; tm < TM; ++tm) fa[tm] = frag_a(buf_c, tm, kc);
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) fb[tn] = frag_b(buf_c, tn, kc);
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                for (int tm = 0; tm < TM; ++tm) mma(acc[tn][tm], fb[tn], fa[tm]);
        }
    };

    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    issue(0, 0);
    if (nk > 1) issue(1, 1);
    for (int s = 0; s < nk; s += 3) {
        step(S0{}, s);
        if (s + 1 < nk) step(S1{}, s + 1);
        if (s + 2 < nk) step(S2{}, s + 2);
    }

    // C[m][n .. n+3]: lane <-> m, four consecutive n per store
    bf16* cbase = static_cast<bf16*>(p.c);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
        const int m = m0 + (wm * TM + tm) * 32 + (lane & 31);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int n = n0 + (wn * TN + tn) * 32 + 8 * rr + 4 * g;
                store4(cbase + (int64_t)m * p.ldc + n, acc[tn][tm][4 * rr], acc[tn][tm][4 * rr + 1],
                       acc[tn][tm][4 * rr + 2], acc[tn][tm][4 * rr + 3]);
            }
    }
}

template <int BM, int BN, bool AT, bool BT>
hipError_t launch_cfg(const GemmArgs& p, hipStream_t stream) {
    using C = GemmCfg<BM, BN, AT, BT>;
    const int tiles = (p.M / BM) * (p.N / BN);
    hipLaunchKernelGGL((proj_gemm_bf16<BM, BN, AT, BT>), dim3((tiles + 7) / 8 * 8), dim3(256), C::BYTES, stream, p);
    return hipGetLastError();
}

template <bool AT, bool BT>
hipError_t launch_tile(int tile, const GemmArgs& p, hipStream_t stream) {
    switch (tile) {
        case kGemmTile128x128: return launch_cfg<128, 128, AT, BT>(p, stream);
        case kGemmTile128x64: return launch_cfg<128, 64, AT, BT>(p, stream);
        case kGemmTile64x128: return launch_cfg<64, 128, AT, BT>(p, stream);
        default: return launch_cfg<64, 64, AT, BT>(p, stream);
    }
}

}  // namespace

int gemm_tile_rows(int tile) { return tile == kGemmTile128x128 || tile == kGemmTile128x64 ? 128 : 64; }
int gemm_tile_cols(int tile) { return tile == kGemmTile128x128 || tile == kGemmTile64x128 ? 128 : 64; }

hipError_t launch_proj_gemm(int a_kmajor, int b_nmajor, int tile, const GemmArgs& p, hipStream_t stream) {
    if (a_kmajor) return b_nmajor ? launch_tile<true, true>(tile, p, stream) : launch_tile<true, false>(tile, p, stream);
    return b_nmajor ? launch_tile<false, true>(tile, p, stream) : launch_tile<false, false>(tile, p, stream);
}

}  // namespace fbl
