// The LM-head stage of a step on the rows the decisions read (Alg. 1; Eq. 1
// and Eq. 7):
//   - lm_select_kernel lists the rows: with logit mixing, the shadow row of
//     every position and the x row of every M position (B + |M| per
//     sequence, not 2B); with hidden-state mixing, first the shadow rows of
//     the candidates (their confidences give the guidance weights), then the
//     shadow rows of U positions and one mixed row per M position (B per
//     sequence over the two passes).  Each listed row carries a code: its
//     logit row (sequence * 2B + row), whether its logits are stored, and
//     where its merged confidence partial goes.
//   - lm_gather_kernel copies the listed rows of the final-normalised
//     activations into a compact matrix (fragment-major for bf16); a mixed
//     row is w * x + (1 - w) * s of the position's two rows (Eq. 7 applied
//     to the hidden state: the head is linear without bias, so in exact
//     arithmetic this equals mixing the logits), each operation rounded once
//     in fp32, then rounded to the storage type as every GEMM input is.
//   - lm_merge_kernel folds the per-column-tile (max, first argmax, sum of
//     exp(l - max)) partials that the fused LM-head epilogue writes into the
//     per-8192-logit-chunk partials the decision kernel reads, in column order.
// The row count is device data (it depends on the states): every kernel is
// launched for the largest possible count and skips the rows beyond it.
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr int kSelThreads = 1024;

// Exclusive prefix sum over the workgroup (kSelThreads threads); returns the
// total through `total`.
__device__ int block_scan(int v, int* buf, int* total) {
    const int t = threadIdx.x;
    buf[t] = v;
    __syncthreads();
    for (int o = 1; o < kSelThreads; o <<= 1) {
        const int add = t >= o ? buf[t - o] : 0;
        __syncthreads();
        buf[t] += add;
        __syncthreads();
    }
    const int incl = buf[t];
    *total = buf[kSelThreads - 1];
    __syncthreads();
    return incl - v;
}

// mode 0 (logit mixing): rowmap0 = [shadow rows of all positions] + [x rows
// of M positions], count[0].  mode 1 (hidden-state mixing): rowmap0 = shadow
// rows of C positions (count[0]); rowmap1 = shadow rows of U positions and
// mixed rows of M positions in position order (count[1]).  fused: the C / U
// shadow rows hand their confidence partials to the merge instead of storing
// their logits (M rows of mode 0 are always stored: the mixing reads them).
__global__ __launch_bounds__(kSelThreads) void lm_select_kernel(const uint8_t* __restrict__ state, int b, int B,
                                                                int mode, int fused, int32_t* __restrict__ rowmap0,
                                                                int32_t* __restrict__ rowmap1,
                                                                int32_t* __restrict__ count) {
    __shared__ int buf[kSelThreads];
    const int n = b * B;
    const int per = (n + kSelThreads - 1) / kSelThreads;   // contiguous positions per thread
    const int p0 = threadIdx.x * per, p1 = min(n, p0 + per);
    auto dest = [&](int p, bool shadow) { return (p / B) * 2 * B + (shadow ? B : 0) + p % B; };
    int total = 0;
    if (mode == 0) {
        // shadow rows: fixed places 0 .. n-1
        for (int p = p0; p < p1; ++p) {
            const int st = state[p];
            int code = dest(p, true);
            if (st == DARD_STATE_M) code |= kLmStore;
            else code |= fused ? (st == DARD_STATE_C ? kLmToV : kLmToM) : kLmStore;
            rowmap0[p] = code;
        }
        int c = 0;
        for (int p = p0; p < p1; ++p) c += state[p] == DARD_STATE_M;
        int off = block_scan(c, buf, &total);
        for (int p = p0; p < p1; ++p)
            if (state[p] == DARD_STATE_M) rowmap0[n + off++] = dest(p, false) | kLmStore;
        if (threadIdx.x == 0) { count[0] = n + total; count[1] = 0; }
        return;
    }
    int c = 0;
    for (int p = p0; p < p1; ++p) c += state[p] == DARD_STATE_C;
    int off = block_scan(c, buf, &total);
    for (int p = p0; p < p1; ++p)
        if (state[p] == DARD_STATE_C) rowmap0[off++] = dest(p, true) | (fused ? kLmToV : kLmStore);
    if (threadIdx.x == 0) count[0] = total;
    c = 0;
    for (int p = p0; p < p1; ++p) c += state[p] != DARD_STATE_C;
    off = block_scan(c, buf, &total);
    for (int p = p0; p < p1; ++p) {
        const int st = state[p];
        if (st == DARD_STATE_C) continue;
        rowmap1[off++] = dest(p, true) | (fused ? kLmToM : kLmStore) | (st == DARD_STATE_M ? kLmMix : 0);
    }
    if (threadIdx.x == 0) count[1] = total;
}

// One thread per 8 consecutive elements of a listed row.
template <typename T>
__global__ void lm_gather_kernel(const T* __restrict__ xn, int d, int frag, const int32_t* __restrict__ rowmap,
                                 const int32_t* __restrict__ count, int max_rows, const float* __restrict__ w,
                                 int B, T* __restrict__ out) {
    const int per_row = d / 8;
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (size_t)max_rows * per_row) return;
    const int r = (int)(t / per_row), k = (int)(t % per_row) * 8;
    if (r >= *count) return;
    const int code = rowmap[r];
    const int src = code & kLmRowMask;
    auto off = [&](int row) { return frag ? frag_off(row, k, d) : (size_t)row * d + k; };
    T* dst = out + off(r);
    const T* sp = xn + off(src);
    if (!(code & kLmMix)) {
        if constexpr (sizeof(T) == 2) {
            *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(sp);
        } else {
            reinterpret_cast<float4*>(dst)[0] = reinterpret_cast<const float4*>(sp)[0];
            reinterpret_cast<float4*>(dst)[1] = reinterpret_cast<const float4*>(sp)[1];
        }
        return;
    }
    // mixed row of an M position: the shadow row is `src`, its x row src - B
    const int seq = src / (2 * B), i = src % (2 * B) - B;
    const float wv = w[seq * B + i];
    const float omw = __fsub_rn(1.f, wv);
    const T* xp = xn + off(src - B);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma clang fp contract(off)
        const float a = wv * St<T>::ld(xp + e);
        const float c = omw * St<T>::ld(sp + e);
        St<T>::st(dst + e, a + c);
    }
}

// One wave per (listed row, 8192-logit chunk): lane l merges tile l of the
// chunk (tiles_per_chunk <= 64), then a butterfly over the wave.
__global__ __launch_bounds__(64) void lm_merge_kernel(const float* __restrict__ lpart, int ntile, int tiles_per_chunk,
                                                      const int32_t* __restrict__ rowmap,
                                                      const int32_t* __restrict__ count, int B, int nchunk,
                                                      float* __restrict__ part_v, float* __restrict__ part_m) {
    const int r = blockIdx.x, c = blockIdx.y, lane = threadIdx.x;
    if (r >= *count) return;
    const int code = rowmap[r];
    float* dst = (code & kLmToV) ? part_v : ((code & kLmToM) ? part_m : nullptr);
    if (!dst) return;
    const int tile = c * tiles_per_chunk + lane;
    SmPart p{-INFINITY, 0x7fffffff, 0.f};
    if (lane < tiles_per_chunk && tile < ntile) {
        const float* q = lpart + ((size_t)r * ntile + tile) * 3;
        p = SmPart{q[0], __float_as_int(q[1]), q[2]};
    }
    // butterfly: smpart_merge is symmetric, so every lane ends with the same value
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const SmPart y{__shfl_xor(p.m, o, 64), __shfl_xor(p.a, o, 64), __shfl_xor(p.s, o, 64)};
        p = smpart_merge(p, y);
    }
    if (lane == 0) {
        const int src = code & kLmRowMask;
        const int pos = (src / (2 * B)) * B + src % B;
        float* o = dst + ((size_t)pos * nchunk + c) * kConfStride;
        o[0] = p.m;
        o[1] = __int_as_float(p.a);
        o[2] = p.s;
    }
}

}  // namespace

hipError_t launch_lm_select(const uint8_t* state, int b, int B, int mode, bool fused, int32_t* rowmap0,
                            int32_t* rowmap1, int32_t* count, hipStream_t s) {
    if (b < 1 || B < 1 || B > kMaxBlock) return hipErrorInvalidValue;
    launch(lm_select_kernel, dim3(1), dim3(kSelThreads), 0, s, state, b, B, mode, (int)fused, rowmap0, rowmap1,
           count);
    return hipGetLastError();
}

hipError_t launch_lm_gather(int dtype, const void* xn, int d, bool frag, const int32_t* rowmap, const int32_t* count,
                            int max_rows, const float* w, int B, void* out, hipStream_t s) {
    if (d % 8 || max_rows < 1) return hipErrorInvalidValue;
    const size_t n = (size_t)max_rows * (d / 8);
    const dim3 grid((unsigned)((n + 255) / 256)), blk(256);
    if (dtype == DARD_DTYPE_BF16)
        launch(lm_gather_kernel<bf16_t>, grid, blk, 0, s, (const bf16_t*)xn, d, (int)frag, rowmap, count, max_rows, w,
               B, (bf16_t*)out);
    else
        launch(lm_gather_kernel<float>, grid, blk, 0, s, (const float*)xn, d, 0, rowmap, count, max_rows, w, B,
               (float*)out);
    return hipGetLastError();
}

hipError_t launch_lm_merge(const float* lpart, int ntile, int tile_cols, const int32_t* rowmap, const int32_t* count,
                           int max_rows, int B, int V, float* part_v, float* part_m, hipStream_t s) {
    const int chunk = kConfChunk;
    if (tile_cols < 1 || chunk % tile_cols || chunk / tile_cols > 64 || max_rows < 1) return hipErrorInvalidValue;
    const int nchunk = conf_chunks(V);
    launch(lm_merge_kernel, dim3(max_rows, nchunk), dim3(64), 0, s, lpart, ntile, chunk / tile_cols, rowmap, count,
           B, nchunk, part_v, part_m);
    return hipGetLastError();
}

}  // namespace dard
