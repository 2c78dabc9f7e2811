// cdna4.hpp -- gfx950 building blocks shared by the attention kernels:
// MFMA 32x32 tiles for bf16 and fp32 storage, operand-fragment loads from LDS
// (row reads and transposed reads), bf16 packing, and the cross-half
// exchange of a 64-wide wavefront.
//
// Fragment convention (both storage types).  A 32x32xK16 "k-chunk" is
// contracted by one bf16 MFMA (v_mfma_f32_32x32x16_bf16) or by eight fp32
// MFMAs (v_mfma_f32_32x32x2_f32).  In a fragment, lane l serves row/column
// l % 32 of its operand and holds 8 contraction elements; which 8 is fixed
// per call site so that the A and B fragments of one product always agree.
// The accumulator of a 32x32 tile holds, in lane l and register r, the
// element at row (r % 4) + 8 * (r / 4) + 4 * (l / 32) and column l % 32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fbl {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

#define FBL_DEV __device__ __forceinline__
#define FBL_LDS __attribute__((address_space(3)))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------- fragments
template <typename T> struct Frag;
template <> struct Frag<bf16> { bf16x8 v; };
template <> struct Frag<float> { float v[8]; };

// Accumulator row held by register r of lane group g (= lane / 32).
FBL_DEV constexpr int acc_row(int r, int g) { return (r & 3) + 8 * (r >> 2) + 4 * g; }

// D += A * B over one 16-deep k-chunk.
FBL_DEV void mma(f32x16& acc, const Frag<bf16>& a, const Frag<bf16>& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc, 0, 0, 0);
}
FBL_DEV void mma(f32x16& acc, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[e], b.v[e], acc, 0, 0, 0);
}

// Row fragment from LDS: 8 consecutive elements starting at `p` (16-byte
// aligned for bf16, 32-byte for fp32).
FBL_DEV void lds_row_frag(Frag<bf16>& f, const bf16* p) {
    f.v = *reinterpret_cast<const FBL_LDS bf16x8*>(reinterpret_cast<uintptr_t>(p));
}
FBL_DEV void lds_row_frag(Frag<float>& f, const float* p) {
    const FBL_LDS f32x4* q = reinterpret_cast<const FBL_LDS f32x4*>(reinterpret_cast<uintptr_t>(p));
    f32x4 a = q[0], b = q[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) { f.v[e] = a[e]; f.v[4 + e] = b[e]; }
}

// Transposed fragment from an LDS tile stored row-major (row pitch `pitch`
// elements): lane l receives column `col0 + (l % 32)` at the eight rows
// rows(h) + [0..3] for h = 0, 1, i.e. element e of the fragment is
// tile[row_h(e/4) + e%4][col].  row0/row1 are the per-lane-group first rows of
// the two runs of four.
//
// bf16 uses ds_read_b64_tr_b16: inside each group of 16 lanes, source lane s
// reads 4 consecutive elements of row (base_row + s/4) at column
// (base_col + 4*(s%4)), and the hardware hands lane t the 4 elements of
// column base_col + t from those 4 rows.
FBL_DEV void lds_tr_frag(Frag<bf16>& f, const bf16* tile, int pitch, int row0, int row1, int col0, int lane) {
    const int t = lane & 15;
    const int colg = col0 + 16 * ((lane >> 4) & 1);   // this 16-lane group's 16 columns
    const int srow = t >> 2, scol = colg + 4 * (t & 3);
    const bf16* p0 = tile + (row0 + srow) * pitch + scol;
    const bf16* p1 = tile + (row1 + srow) * pitch + scol;
    bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FBL_LDS bf16x4*)(reinterpret_cast<uintptr_t>(p0)));
    bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FBL_LDS bf16x4*)(reinterpret_cast<uintptr_t>(p1)));
    f.v = bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}
FBL_DEV void lds_tr_frag(Frag<float>& f, const float* tile, int pitch, int row0, int row1, int col0, int lane) {
    const int col = col0 + (lane & 31);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f.v[e] = tile[(row0 + e) * pitch + col];
        f.v[4 + e] = tile[(row1 + e) * pitch + col];
    }
}

// Fragment from 8 fp32 values (accumulator registers), rounded to storage type.
FBL_DEV void pack_frag(Frag<bf16>& f, const float* x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) f.v[e] = (bf16)x[e];
}
FBL_DEV void pack_frag(Frag<float>& f, const float* x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) f.v[e] = x[e];
}

// Value of `x` held by lane (l ^ 32).
FBL_DEV float other_half(float x) {
    auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const bool lo = (threadIdx.x & 32) == 0;
    return __uint_as_float(lo ? p[1] : p[0]);
}

FBL_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------- global <-> LDS copies
// 16-byte global load; rows outside [0, nrows) read as zeros.
FBL_DEV uint4 load16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

template <typename T> FBL_DEV void store_out(T* p, float x);
template <> FBL_DEV void store_out<float>(float* p, float x) { *p = x; }
template <> FBL_DEV void store_out<bf16>(bf16* p, float x) { *p = (bf16)x; }

// Four consecutive output elements.
FBL_DEV void store4(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<f32x4*>(p) = f32x4{a, b, c, d};
}
FBL_DEV void store4(bf16* p, float a, float b, float c, float d) {
    *reinterpret_cast<bf16x4*>(p) = bf16x4{(bf16)a, (bf16)b, (bf16)c, (bf16)d};
}

}  // namespace fbl
