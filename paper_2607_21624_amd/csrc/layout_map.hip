// layout_map.hip -- diagnostic kernel evaluating the device index map.
#include "kernels.hpp"

namespace fbl {

namespace {

__global__ __launch_bounds__(256) void layout_map_kernel(TokMap m, int B, int H, int S, int D, int64_t* out) {
    const int64_t n = (int64_t)B * H * S * D;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int i = (int)(idx % D);
        const int s = (int)((idx / D) % S);
        const int h = (int)((idx / ((int64_t)D * S)) % H);
        const int b = (int)(idx / ((int64_t)D * S * H));
        out[idx] = m.offset(b, h, s, i);
    }
}

}  // namespace

hipError_t launch_layout_map(const TokMap& m, int B, int H, int S, int D, int64_t* out, hipStream_t stream) {
    const int64_t n = (int64_t)B * H * S * D;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65535) blocks = 65535;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(layout_map_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, m, B, H, S, D, out);
    return hipGetLastError();
}

}  // namespace fbl
