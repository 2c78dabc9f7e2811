// tokmap.hpp -- the device side of the token-major index map.
//
// The reshape (B,S,D) -> (B,S,H,HD) and transpose -> (B,H,S,HD) of the
// multi-head attention chain (paper section 4.3.1) only move whole head-dim
// rows, so their composition (section 4.3.2, f3 o f2 o f1) is one affine map
//   offset(b, h, s, i) = b*sb + s*ss + h*sh + i        (sd == 1)
// evaluated once per tile origin; rows of a staged tile then sit ss elements
// apart.  The strides arrive as kernel arguments, already validated on the
// host (sd == 1, head-aligned tiles, 16-byte aligned rows).
#pragma once

#include <stdint.h>

#include "cdna4.hpp"

namespace fbl {

struct TokMap {
    int64_t sb, ss, sh;

    __device__ __host__ __forceinline__ int64_t head_base(int b, int h) const {
        return (int64_t)b * sb + (int64_t)h * sh;
    }
    __device__ __host__ __forceinline__ int64_t offset(int b, int h, int s, int i) const {
        return (int64_t)b * sb + (int64_t)s * ss + (int64_t)h * sh + i;
    }
};

struct MaskArgs {
    int causal;             // key j allowed only for query i >= j
    const int32_t* kv_len;  // nullptr, or device [B]: key j allowed only if j < kv_len[b]
};

struct FwdArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;
    TokMap mq, mk, mv, mo;
    int B, S, Hq, Hkv;  // S: query tokens
    int Skv;            // key/value tokens (S for self-attention)
    float scale_log2;  // softmax scale times log2(e)
    MaskArgs mask;
};

struct BwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const void* o;
    const void* dout;
    const float* lse;
    void* dq;
    void* dk;
    void* dv;
    float* stats;      // workspace [B, Hq, 2, S]: rows LSE * log2(e) and sum_k dO*O per query
    void* ds;          // nullptr, or workspace [B, Hq, nk32, nq32] blocks of 32x32 bf16 dS
    int nq32, nk32;    // ceil(S / 32), ceil(Skv / 32)
    TokMap mq, mk, mv, mo, mdo, mdq, mdk, mdv;
    int B, S, Hq, Hkv;  // S: query tokens
    int Skv;            // key/value tokens (S for self-attention)
    float scale;       // softmax scale
    float scale_log2;  // scale * log2(e)
    MaskArgs mask;
    // Key/value pass split: each key block's query iterations are shared by
    // kv_split workgroups, which write fp32 partial dK (times scale) and dV to
    // dkv_part, [2][kv_split][B, Skv, Hkv, D] (dK planes, then dV); a reduction
    // adds them in split order.  1: no split, dK and dV written directly.
    float* dkv_part = nullptr;
    int kv_split = 1;
    // tile ids (attn_tiles.hpp) of the bf16 key/value and dQ passes
    int kv_tile = 5;
    int dq_tile = 7;
};

// Matrix product C[M, N] = sum_k A(m, k) B(k, n), bf16 operands, row-major
// storage with leading dimensions in elements.  A is stored [M, K] (or [K, M]
// when read k-major), B [K, N] (or [N, K] when read n-major); a_bytes/b_bytes
// bound the bytes the buffer resources may touch.
struct GemmArgs {
    const void* a;
    const void* b;
    void* c;
    int64_t lda, ldb, ldc;
    int M, N, K;
    uint32_t a_bytes, b_bytes, c_bytes;  // spans of the operands and the result (< 2 GiB)
};

}  // namespace fbl
