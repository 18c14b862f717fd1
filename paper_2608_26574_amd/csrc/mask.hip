// State-specific attention mask (Sec. 3.2, Eq. 2-3): one "take x" bit per
// (query row, block position).  One workgroup per sequence; the block's states
// and confidences are staged in LDS, each thread builds whole 64-bit words.
#include "common.h"
#include "launch.h"

namespace dard {

__global__ __launch_bounds__(256) void build_state_mask_kernel(const uint8_t* __restrict__ state,
                                                               const float* __restrict__ conf,
                                                               int B, uint32_t flags,
                                                               uint64_t* __restrict__ sel) {
    __shared__ uint8_t st[128];
    __shared__ float cf[128];
    const int s = blockIdx.x;
    for (int j = threadIdx.x; j < B; j += blockDim.x) {
        st[j] = state[(size_t)s * B + j];
        cf[j] = conf[(size_t)s * B + j];
    }
    __syncthreads();
    const int W = (B + 63) / 64;
    for (int t = threadIdx.x; t < 2 * B * W; t += blockDim.x) {
        const int r = t / W, w = t % W;
        const int i = r % B;
        const bool shadow = r >= B;
        uint64_t word = 0;
        const int j0 = w * 64, j1 = min(B, j0 + 64);
        for (int j = j0; j < j1; ++j)
            if (take_x(st[i], st[j], cf[i], cf[j], shadow, i == j, flags))
                word |= 1ull << (j - j0);
        sel[((size_t)s * 2 * B + r) * W + w] = word;
    }
}

hipError_t launch_build_state_mask(const uint8_t* state, const float* conf, int b, int B,
                                   uint32_t flags, uint64_t* sel, hipStream_t s) {
    hipLaunchKernelGGL(build_state_mask_kernel, dim3(b), dim3(256), 0, s, state, conf, B, flags,
                       sel);
    return hipGetLastError();
}

}  // namespace dard
