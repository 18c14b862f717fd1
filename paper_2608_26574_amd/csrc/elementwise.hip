// Row-wise kernels: embedding gather of the augmented block / prefix with the
// first RMSNorm fused, the RMSNorm between sub-layers, and the row copies
// used to pack the weight image.
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

__device__ __forceinline__ float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = 0.f;
    const int nw = blockDim.x >> 6;
    for (int i = 0; i < nw; ++i) t += red[i];
    __syncthreads();
    return t;
}

// Offset of element (row, c) of a [rows][d] activation, row-major or fragment-major.
__device__ __forceinline__ size_t act_off(int row, int c, int d, bool frag) {
    return frag ? frag_off(row, c, d) : (size_t)row * d + c;
}

// xn[row] = h / sqrt(mean(h^2) + eps) * gain, rounded to T.
template <typename T>
__device__ void norm_row(const float* h, const T* gain, int d, float eps, T* xn, int row, bool frag, float* red) {
    float ss = 0.f;
    for (int c = threadIdx.x; c < d; c += blockDim.x) ss += h[c] * h[c];
    ss = block_sum(ss, red);
    const float inv = rsqrtf(ss / (float)d + eps);
    for (int c = threadIdx.x; c < d; c += blockDim.x)
        St<T>::st(xn + act_off(row, c, d, frag), h[c] * inv * St<T>::ld(gain + c));
}

template <typename T>
__global__ __launch_bounds__(256) void embed_norm_kernel(const int32_t* __restrict__ ids, const T* __restrict__ embeds,
                                                         const T* __restrict__ table, const T* __restrict__ gain,
                                                         int d, int vocab, float eps, int step_B, int mask_id,
                                                         float* __restrict__ h, T* __restrict__ xn, int frag) {
    __shared__ float red[8];
    const size_t row = blockIdx.x;
    int id;
    if (step_B > 0) {
        const int s = row / (2 * step_B), r = row % (2 * step_B);
        id = r < step_B ? ids[(size_t)s * step_B + r] : mask_id;
    } else {
        id = ids[row];
    }
    // ids are device data: keep every read inside its table
    if (id >= vocab || (id < 0 && embeds == nullptr)) id = id < 0 ? 0 : vocab - 1;
    const T* src = id >= 0 ? table + (size_t)id * d : embeds + row * d;
    float* hr = h + row * d;
    for (int c = threadIdx.x; c < d; c += blockDim.x) hr[c] = St<T>::ld(src + c);
    __syncthreads();
    norm_row<T>(hr, gain, d, eps, xn, (int)row, frag != 0, red);
}

// h[row] += sum_s part[s][row] (split-K partials of the preceding projection,
// added in split order), then xn[row] = RMSNorm(h[row]) * gain.  One
// workgroup of 512 threads per row, each thread holding up to kVec float4 of the row.
constexpr int kVec = 4;   // d <= 512 * 4 * kVec

// NS is the split count (0 = no partials); all loads of a thread are issued
// before the first add so that the row costs one memory round trip.
template <typename T, int NS>
__global__ __launch_bounds__(512) void resid_norm_kernel(float* __restrict__ h, const float* __restrict__ part,
                                                         size_t split_stride, const T* __restrict__ gain,
                                                         int d, float eps, T* __restrict__ xn, int frag) {
    __shared__ float red[8];
    const size_t row = blockIdx.x;
    float4* hr = reinterpret_cast<float4*>(h + row * d);
    const int n4 = d / 4;
    float4 v[kVec];
    float4 p[NS > 0 ? NS : 1][kVec];
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
        const int c4 = threadIdx.x + 512 * q;
        v[q] = c4 < n4 ? hr[c4] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int s = 0; s < NS; ++s)
            p[s][q] = c4 < n4 ? reinterpret_cast<const float4*>(part + s * split_stride + row * d)[c4]
                              : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float ss = 0.f;
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
        const int c4 = threadIdx.x + 512 * q;
        float4 x = v[q];
#pragma unroll
        for (int s = 0; s < NS; ++s) { x.x += p[s][q].x; x.y += p[s][q].y; x.z += p[s][q].z; x.w += p[s][q].w; }
        if (NS > 0 && c4 < n4) hr[c4] = x;
        v[q] = x;
        ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) tot += red[w];
    const float inv = rsqrtf(tot / (float)d + eps);
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
        const int c4 = threadIdx.x + 512 * q;
        if (c4 < n4) {
            const int c = 4 * c4;   // c..c+3 stay inside one 8-element group of the fragment layout
            T* out = xn + act_off((int)row, c, d, frag != 0);
            St<T>::st(out, v[q].x * inv * St<T>::ld(gain + c));
            St<T>::st(out + 1, v[q].y * inv * St<T>::ld(gain + c + 1));
            St<T>::st(out + 2, v[q].z * inv * St<T>::ld(gain + c + 2));
            St<T>::st(out + 3, v[q].w * inv * St<T>::ld(gain + c + 3));
        }
    }
}

__global__ void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n16) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

// Packed weight rows.  mode 0: identity; mode 1: per head of `dh` rows, packed
// row 2t <- row t and 2t+1 <- row t + dh/2 (rotary pairs adjacent); mode 2:
// packed row 2t <- row t of src0 (gate), 2t+1 <- row t of src1 (up).
__global__ void pack_rows_kernel(const uint8_t* __restrict__ src0, const uint8_t* __restrict__ src1,
                                 uint8_t* __restrict__ dst, int nrows, int rowbytes, int mode, int dh) {
    const int rd = blockIdx.x;
    if (rd >= nrows) return;
    const uint8_t* src;
    if (mode == 1) {
        const int head = rd / dh, e = rd % dh, t = e / 2;
        src = src0 + (size_t)(head * dh + ((e & 1) ? t + dh / 2 : t)) * rowbytes;
    } else if (mode == 2) {
        src = ((rd & 1) ? src1 : src0) + (size_t)(rd / 2) * rowbytes;
    } else {
        src = src0 + (size_t)rd * rowbytes;
    }
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    uint4* d4 = reinterpret_cast<uint4*>(dst + (size_t)rd * rowbytes);
    for (int i = threadIdx.x; i < rowbytes / 16; i += blockDim.x) d4[i] = s4[i];
}

}  // namespace

hipError_t launch_pack_rows(const void* src0, const void* src1, void* dst, int nrows, int rowbytes, int mode,
                            int dh, hipStream_t s) {
    launch(pack_rows_kernel, dim3(nrows), dim3(128), 0, s, (const uint8_t*)src0,
                       (const uint8_t*)src1, (uint8_t*)dst, nrows, rowbytes, mode, dh);
    return hipGetLastError();
}

hipError_t launch_embed_norm(int dtype, const int32_t* ids, const void* embeds, const void* table,
                             const void* gain, int rows, int d, int vocab, float eps, int step_B,
                             int mask_id, float* h, void* xn, bool frag, hipStream_t s) {
    TraceScope ts(DARD_K_NORM, s);
    if (frag && !frag_rows(dtype, rows)) return hipErrorInvalidValue;
    if (dtype == DARD_DTYPE_BF16)
        launch(embed_norm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, ids,
                           (const bf16_t*)embeds, (const bf16_t*)table, (const bf16_t*)gain, d, vocab, eps, step_B,
                           mask_id, h, (bf16_t*)xn, (int)frag);
    else
        launch(embed_norm_kernel<float>, dim3(rows), dim3(256), 0, s, ids, (const float*)embeds,
                           (const float*)table, (const float*)gain, d, vocab, eps, step_B, mask_id, h, (float*)xn, 0);
    return hipGetLastError();
}

hipError_t launch_resid_norm(int dtype, float* h, const float* part, int nsplit, int rows, int d,
                             const void* gain, float eps, void* xn, bool frag, hipStream_t s) {
    TraceScope ts(DARD_K_NORM, s);
    if (frag && !frag_rows(dtype, rows)) return hipErrorInvalidValue;
    const size_t stride = (size_t)rows * d;
    if (nsplit < 0 || nsplit > 8 || d > 512 * 4 * kVec) return hipErrorInvalidValue;
#define DARD_RN(T, NS)                                                                                 \
    launch((resid_norm_kernel<T, NS>), dim3(rows), dim3(512), 0, s, h, part, stride,      \
                       (const T*)gain, d, eps, (T*)xn, (int)frag)
#define DARD_RN_ALL(T)                                                                                 \
    switch (nsplit) {                                                                                  \
    case 0: DARD_RN(T, 0); break; case 1: DARD_RN(T, 1); break; case 2: DARD_RN(T, 2); break;          \
    case 3: DARD_RN(T, 3); break; case 4: DARD_RN(T, 4); break; case 5: DARD_RN(T, 5); break;          \
    case 6: DARD_RN(T, 6); break; case 7: DARD_RN(T, 7); break; default: DARD_RN(T, 8); break;         \
    }
    if (dtype == DARD_DTYPE_BF16) {
        DARD_RN_ALL(bf16_t)
    } else {
        DARD_RN_ALL(float)
    }
#undef DARD_RN_ALL
#undef DARD_RN
    return hipGetLastError();
}

hipError_t launch_copy_rows(const void* src, void* dst, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    const size_t blocks = (n16 + 255) / 256;
    launch(copy_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, s,
                       (const uint4*)src, (uint4*)dst, n16);
    return hipGetLastError();
}

// ---------------------------------------------------------------- full-sequence rows
__global__ void full_rows_kernel(const int32_t* __restrict__ seq, int N, int blk, int B, int mask_id,
                                 int32_t* __restrict__ row_ids, int32_t* __restrict__ tok) {
    const int s = blockIdx.y, R = N + B, Nc = N - B;
    const int32_t* sq = seq + (size_t)s * N;
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < R; r += gridDim.x * blockDim.x) {
        int id;
        if (r < Nc) id = sq[r < blk ? r : r + B];
        else if (r < N) id = sq[blk + (r - Nc)];
        else id = mask_id;
        row_ids[(size_t)s * R + r] = id;
        if (r >= Nc && r < N) tok[(size_t)s * B + (r - Nc)] = id;
    }
}

hipError_t launch_full_rows(const int32_t* seq, int b, int N, int blk, int B, int mask_id, int32_t* row_ids,
                            int32_t* tok, hipStream_t s) {
    if (b < 1 || B < 1 || N < B || blk < 0 || blk + B > N) return hipErrorInvalidValue;
    launch(full_rows_kernel, dim3((N + B + 255) / 256, b), dim3(256), 0, s, seq, N, blk, B, mask_id, row_ids, tok);
    return hipGetLastError();
}

// One thread per 16 bytes of a destination row.  In the fragment-major layout
// the 8 bf16 values k..k+7 (k % 8 == 0) of a row are contiguous.
template <typename T>
__global__ void gather_rows_kernel(const T* __restrict__ src, int R, int first, int count, int d, int frag,
                                   T* __restrict__ dst, size_t n16) {
    constexpr int E = 16 / sizeof(T);
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n16) return;
    const int per_row = d / E;
    const int mo = (int)(t / per_row), k = (int)(t % per_row) * E;
    const int s = mo / count, mi = s * R + first + mo % count;
    const size_t so = frag ? frag_off(mi, k, d) : (size_t)mi * d + k;
    const size_t dO = frag ? frag_off(mo, k, d) : (size_t)mo * d + k;
    *reinterpret_cast<uint4*>(dst + dO) = *reinterpret_cast<const uint4*>(src + so);
}

hipError_t launch_gather_rows(int dtype, const void* src, int b, int R, int first, int count, int d, bool frag,
                              void* dst, hipStream_t s) {
    if (b < 1 || count < 1 || first < 0 || first + count > R || d % (dtype == DARD_DTYPE_BF16 ? 64 : 4))
        return hipErrorInvalidValue;
    if (frag && !frag_rows(dtype, b * R)) return hipErrorInvalidValue;
    const size_t es = dtype == DARD_DTYPE_BF16 ? 2 : 4;
    const size_t n16 = (size_t)b * count * d * es / 16;
    const unsigned blocks = (unsigned)((n16 + 255) / 256);
    if (dtype == DARD_DTYPE_BF16)
        launch(gather_rows_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, (const bf16_t*)src, R, first, count, d,
               (int)frag, (bf16_t*)dst, n16);
    else
        launch(gather_rows_kernel<float>, dim3(blocks), dim3(256), 0, s, (const float*)src, R, first, count, d, 0,
               (float*)dst, n16);
    return hipGetLastError();
}

}  // namespace dard
