// Projection GEMMs Y = X * W^T (X [M][K] activations, W [N][K] weights, both
// K-contiguous) with fused epilogues:
//   STORE_F32  plain fp32 store (LM head logits, dard_linear)
//   RESID      fp32 residual add into the residual stream (O and down proj.)
//   SWIGLU     silu(gate) * up on interleaved gate/up rows, stored as dtype
//   QKV        rotary embedding on adjacent (t, t + dh/2) pairs, Q to its
//              buffer, K and V straight into the KV cache at the rows' keys
//
// bf16 kernels use v_mfma_f32_16x16x32_bf16 with W as the A operand (16 output
// columns) and X as the B operand (16 tokens), so that each lane ends with 4
// consecutive output columns of one token -- exactly what the epilogues need.
//   gemm_skinny: M <= 64 tokens (a decoding step).  The weight matrix streams
//     from HBM straight into registers, 16-byte loads, each 4-lane group reads
//     128 contiguous bytes of a weight row; the few activation rows are re-read
//     from L2.  The waves of a workgroup split K and are summed in LDS in a
//     fixed order (deterministic).
//   gemm_tiled: 128x128 tiles through LDS for large M (prefill, big batches).
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

template <typename T>
__device__ __forceinline__ void store4(T* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
    const uint32_t w0 = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
    const uint32_t w1 = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
    *reinterpret_cast<uint2*>(p) = make_uint2(w0, w1);
}

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

// Epilogue for output columns n..n+3 (n % 4 == 0) of token row m.
template <typename T>
__device__ __forceinline__ void epilogue(const EpiArgs& e, int m, int n, floatx4 v) {
    switch (e.kind) {
    case EPI_STORE_F32:
        *reinterpret_cast<float4*>(e.y + (size_t)m * e.ldy + n) = make_float4(v[0], v[1], v[2], v[3]);
        break;
    case EPI_RESID: {
        float4* p = reinterpret_cast<float4*>(e.y + (size_t)m * e.ldy + n);
        float4 h = *p;
        h.x += v[0]; h.y += v[1]; h.z += v[2]; h.w += v[3];
        *p = h;
        break;
    }
    case EPI_SWIGLU: {
        T* a = reinterpret_cast<T*>(e.act) + (size_t)m * e.ld_act + n / 2;
        const float r0 = silu(v[0]) * v[1];
        const float r1 = silu(v[2]) * v[3];
        St<T>::st(a, r0);
        St<T>::st(a + 1, r1);
        break;
    }
    case EPI_QKV: {
        const int s = m / e.rows_per_seq, r = m % e.rows_per_seq;
        const int pos = e.step ? e.P + (r % e.B) : r;
        const int cidx = e.step ? e.P + r : r;
        const int qd = e.Hq * e.dh, kd = e.Hkv * e.dh;
        if (n < qd + kd) {
            // rotary pairs (v0, v1) and (v2, v3): natural dims (t, t + dh/2)
            const int ein = (n < qd ? n : n - qd) % e.dh;
            const float2 cs0 = *reinterpret_cast<const float2*>(e.rope + ((size_t)pos * (e.dh / 2) + ein / 2) * 2);
            const float2 cs1 = *reinterpret_cast<const float2*>(e.rope + ((size_t)pos * (e.dh / 2) + ein / 2 + 1) * 2);
            const float a0 = v[0] * cs0.x - v[1] * cs0.y, b0 = v[1] * cs0.x + v[0] * cs0.y;
            const float a1 = v[2] * cs1.x - v[3] * cs1.y, b1 = v[3] * cs1.x + v[2] * cs1.y;
            if (n < qd) {
                store4<T>(reinterpret_cast<T*>(e.q) + (size_t)m * e.ldq + n, a0, b0, a1, b1);
            } else {
                const int kvh = (n - qd) / e.dh;
                T* kc = reinterpret_cast<T*>(e.kc) + (((size_t)s * e.Hkv + kvh) * e.cap + cidx) * e.dh + ein;
                store4<T>(kc, a0, b0, a1, b1);
            }
        } else {
            const int nv = n - qd - kd;
            const int kvh = nv / e.dh, ein = nv % e.dh;
            T* vc = reinterpret_cast<T*>(e.vc) + (((size_t)s * e.Hkv + kvh) * e.cap + cidx) * e.dh + ein;
            store4<T>(vc, v[0], v[1], v[2], v[3]);
        }
        break;
    }
    }
}

// ---------------------------------------------------------------- skinny
template <int NW, int KSPLIT>
__global__ __launch_bounds__(64 * KSPLIT) void gemm_skinny_bf16(const bf16_t* __restrict__ X, int M, int K,
                                                              int ldx, const bf16_t* __restrict__ W, int N,
                                                              EpiArgs e) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * 16 * NW;
    const int m0 = blockIdx.y * 64;

    const bf16_t* wp[NW];
#pragma unroll
    for (int j = 0; j < NW; ++j) wp[j] = W + (size_t)min(n0 + 16 * j + lr, N - 1) * K + 16 * g;
    const bf16_t* xp[4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) xp[mb] = X + (size_t)min(m0 + 16 * mb + lr, M - 1) * ldx + 16 * g;

    floatx4 acc[NW][4];
#pragma unroll
    for (int j = 0; j < NW; ++j)
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) acc[j][mb] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nu = K / 64;
    bf16x8 wa[2][NW], xb[2][4];
    int u = wave;
    if (u < nu) {
#pragma unroll
        for (int j = 0; j < NW; ++j) { wa[0][j] = ld_bf16x8(wp[j] + u * 64); wa[1][j] = ld_bf16x8(wp[j] + u * 64 + 8); }
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) { xb[0][mb] = ld_bf16x8(xp[mb] + u * 64); xb[1][mb] = ld_bf16x8(xp[mb] + u * 64 + 8); }
    }
    for (; u < nu; u += KSPLIT) {
        bf16x8 wn[2][NW], xn[2][4];
        const int un = u + KSPLIT;
        if (un < nu) {
#pragma unroll
            for (int j = 0; j < NW; ++j) { wn[0][j] = ld_bf16x8(wp[j] + un * 64); wn[1][j] = ld_bf16x8(wp[j] + un * 64 + 8); }
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) { xn[0][mb] = ld_bf16x8(xp[mb] + un * 64); xn[1][mb] = ld_bf16x8(xp[mb] + un * 64 + 8); }
        }
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int j = 0; j < NW; ++j)
#pragma unroll
                for (int mb = 0; mb < 4; ++mb) acc[j][mb] = mfma16x16x32(wa[hh][j], xb[hh][mb], acc[j][mb]);
        if (un < nu) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
                for (int j = 0; j < NW; ++j) wa[hh][j] = wn[hh][j];
#pragma unroll
                for (int mb = 0; mb < 4; ++mb) xb[hh][mb] = xn[hh][mb];
            }
        }
    }

    if constexpr (KSPLIT > 1) {
        __shared__ floatx4 red[KSPLIT - 1][NW * 4][64];
        if (wave > 0) {
#pragma unroll
            for (int j = 0; j < NW; ++j)
#pragma unroll
                for (int mb = 0; mb < 4; ++mb) red[wave - 1][j * 4 + mb][lane] = acc[j][mb];
        }
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int w = 0; w < KSPLIT - 1; ++w)
#pragma unroll
            for (int j = 0; j < NW; ++j)
#pragma unroll
                for (int mb = 0; mb < 4; ++mb) acc[j][mb] += red[w][j * 4 + mb][lane];
    }
#pragma unroll
    for (int j = 0; j < NW; ++j) {
        const int n = n0 + 16 * j + 4 * g;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            const int m = m0 + 16 * mb + lr;
            if (m < M && n < N) epilogue<bf16_t>(e, m, n, acc[j][mb]);
        }
    }
}

// ---------------------------------------------------------------- tiled
constexpr int TBM = 128, TBN = 128, TBK = 64, TPAD = TBK + 8;

__global__ __launch_bounds__(256) void gemm_tiled_bf16(const bf16_t* __restrict__ X, int M, int K, int ldx,
                                                       const bf16_t* __restrict__ W, int N, EpiArgs e,
                                                       int tiles_m, int tiles_n) {
    __shared__ __attribute__((aligned(16))) bf16_t Ws[TBN * TPAD];
    __shared__ __attribute__((aligned(16))) bf16_t Xs[TBM * TPAD];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, g = lane >> 4;
    // XCD-aware order: workgroups are dealt round-robin to the 8 XCDs, so give
    // each XCD a contiguous run of tiles (m fastest: tiles sharing a weight
    // panel then share that XCD's L2).
    const int total = tiles_m * tiles_n;
    int bid = blockIdx.x;
    if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
    const int tm = bid % tiles_m, tn = bid / tiles_m;
    const int n0 = tn * TBN, m0 = tm * TBM;
    const int wn = wave & 1, wm = wave >> 1;

    floatx4 acc[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = floatx4{0.f, 0.f, 0.f, 0.f};

    bf16x8 wr[4], xr[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int c = threadIdx.x + 256 * it;
            const int row = c >> 3, c8 = c & 7;
            wr[it] = ld_bf16x8(W + (size_t)min(n0 + row, N - 1) * K + k0 + c8 * 8);
            xr[it] = ld_bf16x8(X + (size_t)min(m0 + row, M - 1) * ldx + k0 + c8 * 8);
        }
    };
    auto sstore = [&]() {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int c = threadIdx.x + 256 * it;
            const int row = c >> 3, c8 = c & 7;
            *reinterpret_cast<bf16x8*>(&Ws[row * TPAD + c8 * 8]) = wr[it];
            *reinterpret_cast<bf16x8*>(&Xs[row * TPAD + c8 * 8]) = xr[it];
        }
    };
    const int nk = K / TBK;
    gload(0);
    for (int kt = 0; kt < nk; ++kt) {
        __syncthreads();
        sstore();
        __syncthreads();
        if (kt + 1 < nk) gload((kt + 1) * TBK);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            bf16x8 af[4], bfr[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                af[j] = *reinterpret_cast<const bf16x8*>(&Ws[(wn * 64 + 16 * j + lr) * TPAD + 32 * hh + 8 * g]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                bfr[i] = *reinterpret_cast<const bf16x8*>(&Xs[(wm * 64 + 16 * i + lr) * TPAD + 32 * hh + 8 * g]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[j][i] = mfma16x16x32(af[j], bfr[i], acc[j][i]);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + 16 * j + 4 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = m0 + wm * 64 + 16 * i + lr;
            if (m < M && n < N) epilogue<bf16_t>(e, m, n, acc[j][i]);
        }
    }
}

// ---------------------------------------------------------------- fp32
// One thread per (token, 4 output columns); 16 tokens x 16 column-quads per
// workgroup with the K loop staged through LDS in 32-wide slices.
__global__ __launch_bounds__(256) void gemm_f32(const float* __restrict__ X, int M, int K, int ldx,
                                                const float* __restrict__ W, int N, EpiArgs e) {
    __shared__ float xs[16][33];
    __shared__ float ws[64][33];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int m = blockIdx.y * 16 + ty;
    const int n = blockIdx.x * 64 + tx * 4;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < K; k0 += 32) {
        for (int t = threadIdx.x; t < 16 * 32; t += 256) {
            const int r = t / 32, c = t % 32;
            const int mm = blockIdx.y * 16 + r;
            xs[r][c] = (mm < M && k0 + c < K) ? X[(size_t)mm * ldx + k0 + c] : 0.f;
        }
        for (int t = threadIdx.x; t < 64 * 32; t += 256) {
            const int r = t / 32, c = t % 32;
            const int nn = blockIdx.x * 64 + r;
            ws[r][c] = (nn < N && k0 + c < K) ? W[(size_t)nn * K + k0 + c] : 0.f;
        }
        __syncthreads();
        for (int c = 0; c < 32; ++c) {
            const float xv = xs[ty][c];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] += xv * ws[tx * 4 + i][c];
        }
        __syncthreads();
    }
    if (m < M && n < N) epilogue<float>(e, m, n, floatx4{acc[0], acc[1], acc[2], acc[3]});
}

}  // namespace

hipError_t launch_gemm(int dtype, const void* X, int M, int K, int ldx, const void* W, int N,
                       const EpiArgs& e, int kernel_class, hipStream_t s) {
    TraceScope ts(kernel_class, s);
    if (dtype == DARD_DTYPE_F32) {
        dim3 grid((N + 63) / 64, (M + 15) / 16);
        hipLaunchKernelGGL(gemm_f32, grid, dim3(256), 0, s, reinterpret_cast<const float*>(X), M, K, ldx,
                           reinterpret_cast<const float*>(W), N, e);
        return hipGetLastError();
    }
    const bf16_t* x = reinterpret_cast<const bf16_t*>(X);
    const bf16_t* w = reinterpret_cast<const bf16_t*>(W);
    if (M <= 64) {
        // enough workgroups to cover 256 CUs at least twice
        if (N / 64 >= 512) {
            hipLaunchKernelGGL((gemm_skinny_bf16<4, 4>), dim3((N + 63) / 64, 1), dim3(256), 0, s, x, M, K, ldx, w, N, e);
        } else if (N / 32 >= 512) {
            hipLaunchKernelGGL((gemm_skinny_bf16<2, 4>), dim3((N + 31) / 32, 1), dim3(256), 0, s, x, M, K, ldx, w, N, e);
        } else {
            hipLaunchKernelGGL((gemm_skinny_bf16<1, 8>), dim3((N + 15) / 16, 1), dim3(512), 0, s, x, M, K, ldx, w, N, e);
        }
        return hipGetLastError();
    }
    const int tiles_m = (M + TBM - 1) / TBM, tiles_n = (N + TBN - 1) / TBN;
    hipLaunchKernelGGL(gemm_tiled_bf16, dim3(tiles_m * tiles_n), dim3(256), 0, s, x, M, K, ldx, w, N, e,
                       tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace dard
