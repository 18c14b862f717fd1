// State-specific attention mask (Sec. 3.2, Eq. 2-3): one "take x" bit per
// (query row, block position).  One workgroup of 4 waves per sequence; each
// wave builds whole rows with ballots (row_take_x), so the kernel holds no
// per-bit loops.
#include "common.h"
#include "launch.h"

namespace dard {

__global__ __launch_bounds__(256) void build_state_mask_kernel(const uint8_t* __restrict__ state,
                                                               const float* __restrict__ conf,
                                                               int B, uint32_t flags,
                                                               uint64_t* __restrict__ sel) {
    const int s = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int W = (B + 63) / 64;
    const BlockView v = load_block_view(state + (size_t)s * B, conf + (size_t)s * B, B);
    for (int r = wave; r < 2 * B; r += 4) {
        uint64_t x[kBlockWords];
        row_take_x(v, r, B, flags, x);
        uint64_t mine = x[0];
#pragma unroll
        for (int q = 1; q < kBlockWords; ++q) mine = lane == q ? x[q] : mine;
        if (lane < W) sel[((size_t)s * 2 * B + r) * W + lane] = mine;
    }
}

// Codes outside {0, 1, 2}: their number and the first index.  One workgroup
// walks all n codes, so nothing has to be initialised beforehand.
__global__ __launch_bounds__(256) void check_states_kernel(const uint8_t* __restrict__ state, int n,
                                                           int32_t* __restrict__ status) {
    __shared__ int cnt, first;
    if (threadIdx.x == 0) { cnt = 0; first = 0x7fffffff; }
    __syncthreads();
    int c = 0, f = 0x7fffffff;
    for (int i = threadIdx.x; i < n; i += 256)
        if (state[i] > DARD_STATE_U) { ++c; f = min(f, i); }
    if (c) { atomicAdd(&cnt, c); atomicMin(&first, f); }
    __syncthreads();
    if (threadIdx.x == 0) {
        status[0] = cnt;
        status[1] = cnt ? first : -1;
    }
}

hipError_t launch_check_states(const uint8_t* state, int n, int32_t* status, hipStream_t s) {
    launch(check_states_kernel, dim3(1), dim3(256), 0, s, state, n, status);
    return hipGetLastError();
}

hipError_t launch_build_state_mask(const uint8_t* state, const float* conf, int b, int B,
                                   uint32_t flags, uint64_t* sel, hipStream_t s) {
    launch(build_state_mask_kernel, dim3(b), dim3(256), 0, s, state, conf, B, flags,
                       sel);
    return hipGetLastError();
}

}  // namespace dard
