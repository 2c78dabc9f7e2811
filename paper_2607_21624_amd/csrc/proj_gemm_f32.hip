// proj_gemm_f32.hip -- the projection products for fp32 storage, gfx950.
//
// The same three products as proj_gemm.hip (Y = X W, dX = dY W^T,
// dW = X^T dY; section 4.1's matrix-product gradients, no operand transposed
// in memory) for tensors stored in fp32, with fp32 accumulation on
// v_mfma_f32_32x32x2_f32 (eight per 16-deep chunk, cdna4.hpp's fragment
// convention).  fp32 storage is the small-configuration path, so the kernel
// is the plain form: a 64 x 64 output tile per workgroup of 4 wavefronts
// (2 x 2, one 32 x 32 tile each), 16-deep steps staged through LDS by
// coalesced element loads in each operand's stored orientation, every load
// and store bounds-checked (any extents, any leading dimensions).
#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace fbl {

namespace {

constexpr int kF32Tile = 64;  // output rows and columns per workgroup
constexpr int kF32K = 16;     // contraction elements per step
constexpr int kF32Pad = 1;    // LDS row padding (floats) against bank conflicts

// AT: A stored k-major ([K, M] rows); BT: B stored n-major ([N, K] rows).
template <bool AT, bool BT>
__global__ __launch_bounds__(256) void proj_gemm_f32(GemmArgs p) {
    // LDS: As[m][k] and Bs[k][n], padded rows
    __shared__ float As[kF32Tile][kF32K + kF32Pad];
    __shared__ float Bs[kF32K][kF32Tile + kF32Pad];
    const float* A = static_cast<const float*>(p.a);
    const float* Bm = static_cast<const float*>(p.b);
    float* Cm = static_cast<float*>(p.c);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = lane >> 5;
    const int wm = wave & 1, wn = wave >> 1;
    const int mt = (p.M + kF32Tile - 1) / kF32Tile, nt = (p.N + kF32Tile - 1) / kF32Tile;
    const int logical = xcd_logical_id(blockIdx.x, mt * nt, gridDim.x);
    if (logical < 0) return;
    const int m0 = (logical % mt) * kF32Tile, n0 = (logical / mt) * kF32Tile;

    f32x16 acc = f32x16{};
    for (int k0 = 0; k0 < p.K; k0 += kF32K) {
        // stage A (64 x 16) and B (16 x 64): 1024 elements each, 4 per thread,
        // consecutive threads on the operand's contiguous axis
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = tid + 256 * u;
            int m, k;
            if constexpr (AT) { k = e / kF32Tile; m = e % kF32Tile; }   // rows of A^T are k
            else { m = e / kF32K; k = e % kF32K; }
            const int gm = m0 + m, gk = k0 + k;
            float x = 0.f;
            if (gm < p.M && gk < p.K) x = AT ? A[(int64_t)gk * p.lda + gm] : A[(int64_t)gm * p.lda + gk];
            As[m][k] = x;
            int n;
            if constexpr (BT) { n = e / kF32K; k = e % kF32K; }          // rows of B^T are n
            else { k = e / kF32Tile; n = e % kF32Tile; }
            const int gn = n0 + n;
            const int gk2 = k0 + k;
            float y = 0.f;
            if (gn < p.N && gk2 < p.K) y = BT ? Bm[(int64_t)gn * p.ldb + gk2] : Bm[(int64_t)gk2 * p.ldb + gn];
            Bs[k][n] = y;
        }
        __syncthreads();
        // one 16-deep chunk: lane group g holds contraction elements 8g .. 8g+7
        Frag<float> fa, fb;
        const int row = wm * 32 + (lane & 31), col = wn * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            fa.v[e] = As[row][8 * g + e];
            fb.v[e] = Bs[8 * g + e][col];
        }
        // accumulator rows = n (acc_row), columns = m (lane): C^T, as in the bf16 kernel
        mma(acc, fb, fa);
        __syncthreads();
    }
    const int m = m0 + wm * 32 + (lane & 31);
    if (m < p.M) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int n = n0 + wn * 32 + acc_row(r, g);
            if (n < p.N) Cm[(int64_t)m * p.ldc + n] = acc[r];
        }
    }
}

template <bool AT, bool BT>
hipError_t launch_f32(const GemmArgs& p, hipStream_t stream) {
    const int tiles = ((p.M + kF32Tile - 1) / kF32Tile) * ((p.N + kF32Tile - 1) / kF32Tile);
    hipLaunchKernelGGL((proj_gemm_f32<AT, BT>), dim3((tiles + 7) / 8 * 8), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_proj_gemm_f32(int a_kmajor, int b_nmajor, const GemmArgs& p, hipStream_t stream) {
    if (a_kmajor) return b_nmajor ? launch_f32<true, true>(p, stream) : launch_f32<true, false>(p, stream);
    return b_nmajor ? launch_f32<false, true>(p, stream) : launch_f32<false, false>(p, stream);
}

}  // namespace fbl
