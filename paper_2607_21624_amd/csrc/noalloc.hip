// noalloc.hip -- the attention backward for callers that cannot allocate
// device memory (code under HIP graph capture, serving loops that forbid
// allocation): the backward's scratch (per-row statistics, the dS blocks, the
// split pass's partial sums) lives in one library-owned device array instead
// of a caller-provided workspace.
//
// The array is a file-scope __device__ variable: every GPU the library runs
// on holds its own copy, FBL_NOALLOC_SCRATCH_BYTES long, until the process
// ends.  Its device address is looked up once per device with
// hipGetSymbolAddress (the array's name in host code is only a stand-in for
// the lookup) and kept in a per-device table; kernels receive that address as
// their workspace pointer.  Every call on a device shares the array, so
// calls that can run at the same time on one device (different streams with
// no ordering between them) race; nothing in it needs to start at zero (each
// call writes every byte it later reads).
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/fbl.h"

static __device__ __align__(256) unsigned char scratch[FBL_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up

// Device address of the scratch array on the current device; looked up on
// the first call per device, with that device current.
fbl_status scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return FBL_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return FBL_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FBL_ERR_HIP;
        if ((reinterpret_cast<uintptr_t>(p) & 255u) != 0) return FBL_ERR_ALIGN;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return FBL_OK;
}

}  // namespace

extern "C" {

fbl_status fbl_attn_bwd_noalloc(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                                const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                                const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                                const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk,
                                const fbl_layout* ldv, void* dv, void* stream) {
    // the smallest workspace the backward accepts must fit the array
    size_t need = 0;
    fbl_status st = fbl_attn_bwd_workspace_min(lq, lk, &need);
    if (st != FBL_OK) return st;
    if (need > (size_t)FBL_NOALLOC_SCRATCH_BYTES) return FBL_ERR_WORKSPACE;
    void* ws = nullptr;
    if ((st = scratch_address(&ws)) != FBL_OK) return st;
    // The whole array as the workspace: fbl_attn_bwd picks the stored-dS
    // path (and the split key/value pass) exactly when their parts fit.
    return fbl_attn_bwd(lq, q, lk, k, lv, v, lo, o, ldo, dO, lse, scale, mask, ldq, dq, ldk, dk, ldv, dv, ws,
                        (size_t)FBL_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
