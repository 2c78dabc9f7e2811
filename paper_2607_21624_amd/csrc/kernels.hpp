// kernels.hpp -- launchers of the attention kernels (host-callable).
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>

#include "attn_tiles.hpp"
#include "gemm_tiles.hpp"
#include "tokmap.hpp"

namespace fbl {

// Raise a kernel's dynamic-LDS limit before its first launch on each device
// (the attribute is held per device).  One flag word per kernel; devices 64
// and up set the attribute on every launch.
template <auto Kernel>
hipError_t ensure_dynamic_lds(int bytes) {
    static std::atomic<uint64_t> done{0};  // bit d: set on device d
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev >= 0 && dev < 64 ? (uint64_t(1) << dev) : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(Kernel), hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
    return e;
}

typedef __bf16 bf16;

// Forward for fp32 storage: O and LSE from Q, K, V; D in {32, 64, 128}.
template <int D>
hipError_t launch_attn_fwd_f32(const FwdArgs& a, hipStream_t stream);

// Forward for bf16 storage with forward tile `tile` of kAttnTiles.
template <int D>
hipError_t launch_attn_fwd_bf16(const FwdArgs& a, int tile, hipStream_t stream);

// Backward: per-row statistics (LSE * log2(e), D = rowsum(dO * O)), then the
// key/value-major pass (dK, dV) and the query-major pass (dQ).
// `phases`: bit 0 statistics, bit 1 kv pass, bit 2 q pass.
template <typename T, int D>
hipError_t launch_attn_bwd(const BwdArgs& a, unsigned phases, hipStream_t stream);

// The whole backward in one launch, for key/value sequences of at most 128
// tokens (one key block per (batch, kv head)): row statistics, dK, dV and dQ.
template <typename T, int D>
hipError_t launch_attn_bwd_fused(const BwdArgs& a, hipStream_t stream);

// Key/value-major backward pass for bf16 storage (software-pipelined kernel)
// with kv tile `tile` of kAttnTiles (its split is a.kv_split).
template <int D>
hipError_t launch_attn_bwd_kv_bf16(const BwdArgs& a, int tile, hipStream_t stream);

// Query-major backward pass (dQ) for bf16 storage (software-pipelined kernel),
// recomputing S and dP.
template <int D>
hipError_t launch_attn_bwd_q_bf16(const BwdArgs& a, hipStream_t stream);

// dQ for bf16 storage from the dS blocks the key/value-major pass stored in
// the workspace (a.ds != nullptr), with dQ tile `tile` of kAttnTiles.
template <int D>
hipError_t launch_attn_bwd_dq_bf16(const BwdArgs& a, int tile, hipStream_t stream);

// Projection matrix products (proj_gemm.hip).  Output tile shapes:
// `tile` indexes kGemmTiles (gemm_tiles.hpp).
// a_kmajor: A stored [K, M]; b_nmajor: B stored [N, K].
hipError_t launch_proj_gemm(int a_kmajor, int b_nmajor, int tile, const GemmArgs& p, hipStream_t stream);
// The same products for fp32 storage (proj_gemm_f32.hip): one tile shape.
hipError_t launch_proj_gemm_f32(int a_kmajor, int b_nmajor, const GemmArgs& p, hipStream_t stream);

// Diagnostic: offsets of a token-major tensor computed by the device index map.
hipError_t launch_layout_map(const TokMap& m, int B, int H, int S, int D, int64_t* out, hipStream_t stream);

}  // namespace fbl
