// kernels.hpp -- launchers of the attention kernels (host-callable).
#pragma once

#include <hip/hip_runtime.h>

#include "tokmap.hpp"

namespace fbl {

typedef __bf16 bf16;

// Forward: O and LSE from Q, K, V.  T is float or __bf16; D in {32, 64, 128}.
template <typename T, int D>
hipError_t launch_attn_fwd(const FwdArgs& a, hipStream_t stream);

// Backward: row statistic D = rowsum(dO * O) and zeroed dQ accumulator,
// then the key/value-major main pass (dK, dV, dQ accumulation), then the
// dQ conversion to the storage type.  Three launches on `stream`.
// `phases`: bit 0 pre, bit 1 main, bit 2 dQ conversion.
template <typename T, int D>
hipError_t launch_attn_bwd(const BwdArgs& a, unsigned phases, hipStream_t stream);

// Diagnostic: offsets of a token-major tensor computed by the device index map.
hipError_t launch_layout_map(const TokMap& m, int B, int H, int S, int D, int64_t* out, hipStream_t stream);

}  // namespace fbl
