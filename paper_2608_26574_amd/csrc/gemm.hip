// Projection GEMMs Y = X * W^T (X [M][K] activations, W [N][K] weights) with
// fused epilogues:
//   STORE_F32  plain fp32 store (LM head logits, dard_linear)
//   RESID      fp32 residual add into the residual stream (O and down proj.)
//   SWIGLU     silu(gate) * up on interleaved gate/up rows, stored as dtype
//   QKV        rotary embedding on adjacent (t, t + dh/2) pairs, Q to its
//              buffer, K and V straight into the KV cache at the rows' keys
//              (K [cap][dh], V dims-major [dh][cap] per KV head)
//   PARTIAL    fp32 split-K partial [split][M][N], reduced by the consumer
//
// bf16 weights are packed fragment-major: the 16 x 64 block (row block nb,
// k unit u) is stored contiguously at element ((nb * K/64 + u) * 1024), as two
// halves of 512 (k 8h..8h+7 of each 16-wide group) in which lane l of a wave
// finds its 8 values at 8*l.  One 16-byte load per lane then reads exactly the
// A operand of v_mfma_f32_16x16x32_bf16 and a wave load is 1 KB contiguous;
// a wave streaming a row block over K reads one contiguous region.
//
// W is the A operand (16 output columns), X the B operand (16 tokens), so each
// lane ends with 4 consecutive output columns of one token.
//   gemm_stream: M <= 64 tokens (a decoding step).  Each wave owns 16*NW
//     columns; the KSPLIT waves of a workgroup take interleaved k units and are
//     summed in LDS in a fixed order; DEPTH units per wave are in flight in a
//     register ring.  Weights are read with non-temporal loads (streamed once).
//     Optional split of K across SPLIT workgroups writes fp32 partials.
//   gemm_pipe: 64 < M < 256 with fragment-major X, 128 x 128 tiles through a
//     register ring and an LDS double buffer.
//   gemm_big: M >= 256 with fragment-major X (prefill, large batches), tiles of
//     up to 256 x 128 / 128 x 256 fed by global_load_lds slice stages.
//   gemm_tiled: row-major X (dard_linear), 128 x 128 tiles through LDS.
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

// Two adjacent values (p 2-element aligned): one 4- or 8-byte store.
template <typename T>
__device__ __forceinline__ void store2(T* p, float a, float b);
template <>
__device__ __forceinline__ void store2<float>(float* p, float a, float b) {
    *reinterpret_cast<float2*>(p) = make_float2(a, b);
}
template <>
__device__ __forceinline__ void store2<bf16_t>(bf16_t* p, float a, float b) {
    *reinterpret_cast<uint32_t*>(p) = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// x * sigmoid(x) with the hardware exp2 and reciprocal (about 1 ulp each):
// exp2 of a large argument is +inf and its reciprocal 0, so the limits hold.
__device__ __forceinline__ float silu(float x) {
    return x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x * -1.4426950408889634f));
}

// The epilogue kind is uniform over a launch; kernels branch on it once and
// run a loop specialised for it (Kind<k>), so a tile's epilogue carries no
// per-tile dispatch and no code of the other kinds.
template <int K>
struct Kind {
    static constexpr int value = K;
};

template <typename F>
__device__ __forceinline__ void with_kind(int kind, F&& f) {
    switch (kind) {
    case EPI_STORE_F32: f(Kind<EPI_STORE_F32>{}); break;
    case EPI_PARTIAL: f(Kind<EPI_PARTIAL>{}); break;
    case EPI_RESID: f(Kind<EPI_RESID>{}); break;
    case EPI_SWIGLU: f(Kind<EPI_SWIGLU>{}); break;
    case EPI_QKV: f(Kind<EPI_QKV>{}); break;
    case EPI_LMHEAD: f(Kind<EPI_LMHEAD>{}); break;
    default: break;
    }
}

// Row m of the QKV output: sequence s, rotary position and cache index.
struct QkvRow {
    int s, pos, cidx;
};
__device__ __forceinline__ QkvRow qkv_row(const EpiArgs& e, int m) {
    const int s = m / e.rows_per_seq, r = m - s * e.rows_per_seq;
    if (e.step == 2)   // full sequence: the other positions, then the block's x and s rows
        return QkvRow{s, r < e.P ? (r < e.blk ? r : r + e.B) : e.blk + (r - e.P) % e.B, r};
    if (e.step == 3)   // positions after a shared prompt of P
        return QkvRow{s, e.P + r, e.P + r};
    return QkvRow{s, e.step ? e.P + (r % e.B) : r, e.step ? e.P + r : r};
}

// Epilogue for output columns n..n+3 (n % 4 == 0) of token row m, in two
// halves: epi_fetch loads what the epilogue reads (the residual, or the two
// rotary (cos, sin) pairs), epi_store combines and writes.  A kernel that
// owns several tiles fetches for all of them before its first store, so the
// loads overlap instead of each waiting behind the stores before it.  head_dim
// is 64 or 128, so dims and heads come from shifts.
template <int EK>
__device__ __forceinline__ float4 epi_fetch(const EpiArgs& e, int m, int n) {
    if constexpr (EK == EPI_RESID) return *reinterpret_cast<const float4*>(e.y + (size_t)m * e.ldy + n);
    if constexpr (EK == EPI_QKV) {
        const int qd = e.Hq * e.dh, kd = e.Hkv * e.dh;
        if (n < qd + kd) {
            const int ein = (n < qd ? n : n - qd) & (e.dh - 1);
            const float* t = e.rope + ((size_t)qkv_row(e, m).pos * (e.dh / 2) + ein / 2) * 2;
            const float2 c0 = *reinterpret_cast<const float2*>(t);
            const float2 c1 = *reinterpret_cast<const float2*>(t + 2);
            return make_float4(c0.x, c0.y, c1.x, c1.y);
        }
    }
    return make_float4(0.f, 0.f, 0.f, 0.f);
}

template <typename T, int EK>
__device__ __forceinline__ void epi_store(const EpiArgs& e, int m, int n, floatx4 v, float4 f) {
    if constexpr (EK == EPI_STORE_F32 || EK == EPI_PARTIAL) {
        *reinterpret_cast<float4*>(e.y + (size_t)m * e.ldy + n) = make_float4(v[0], v[1], v[2], v[3]);
    } else if constexpr (EK == EPI_RESID) {
        *reinterpret_cast<float4*>(e.y + (size_t)m * e.ldy + n) =
            make_float4(f.x + v[0], f.y + v[1], f.z + v[2], f.w + v[3]);
    } else if constexpr (EK == EPI_SWIGLU) {
        // interleaved rows: (gate, up) pairs at (n, n+1) and (n+2, n+3)
        T* a = reinterpret_cast<T*>(e.act) + (e.act_frag ? frag_off(m, n / 2, e.ld_act) : (size_t)m * e.ld_act + n / 2);
        store2<T>(a, silu(v[0]) * v[1], silu(v[2]) * v[3]);
    } else if constexpr (EK == EPI_LMHEAD) {
        // a listed row of the LM head: stored at its logit row when its code says so
        const int code = e.rowmap[m];
        const size_t o = (size_t)(code & kLmRowMask) * e.ldy + n;
        const float4 val = make_float4(v[0], v[1], v[2], v[3]);
        if (code & kLmStore) *reinterpret_cast<float4*>(e.y + o) = val;
        if (e.y2) *reinterpret_cast<float4*>(e.y2 + o) = val;
    } else if constexpr (EK == EPI_QKV) {
        const QkvRow row = qkv_row(e, m);
        const int qd = e.Hq * e.dh, kd = e.Hkv * e.dh;
        const int sh = e.dh == 128 ? 7 : 6;
        if (n < qd + kd) {
            // rotary pairs (v0, v1) and (v2, v3): natural dims (t, t + dh/2)
            const float a0 = v[0] * f.x - v[1] * f.y, b0 = v[1] * f.x + v[0] * f.y;
            const float a1 = v[2] * f.z - v[3] * f.w, b1 = v[3] * f.z + v[2] * f.w;
            if (n < qd) {
                store4<T>(reinterpret_cast<T*>(e.q) + (size_t)m * e.ldq + n, a0, b0, a1, b1);
            } else {
                const int nk = n - qd, kvh = nk >> sh, ein = nk & (e.dh - 1);
                const size_t ko = (((size_t)row.s * e.Hkv + kvh) * e.cap + row.cidx) * e.dh + ein;
                if (e.kv_fp8)
                    *reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(e.kc) + ko) =
                        f2e4m3(a0) | (f2e4m3(b0) << 8) | (f2e4m3(a1) << 16) | (f2e4m3(b1) << 24);
                else
                    store4<T>(reinterpret_cast<T*>(e.kc) + ko, a0, b0, a1, b1);
            }
        } else {
            // the V cache is dims-major ([dh][cap] per KV head): four strided stores
            const int nv = n - qd - kd, kvh = nv >> sh, ein = nv & (e.dh - 1);
            const size_t vo = (((size_t)row.s * e.Hkv + kvh) * e.dh + ein) * e.cap + row.cidx;
            if (e.kv_fp8) {
                uint8_t* vc = reinterpret_cast<uint8_t*>(e.vc) + vo;
#pragma unroll
                for (int i = 0; i < 4; ++i) vc[(size_t)i * e.cap] = (uint8_t)f2e4m3(v[i]);
            } else {
                T* vc = reinterpret_cast<T*>(e.vc) + vo;
#pragma unroll
                for (int i = 0; i < 4; ++i) St<T>::st(vc + (size_t)i * e.cap, v[i]);
            }
        }
    }
}

// Rows of the launch whose results are kept: all M, or the device count of
// an LM-head launch over listed rows.
__device__ __forceinline__ int valid_rows(const EpiArgs& e, int M) {
    return e.rows_dev ? min(M, __builtin_amdgcn_readfirstlane(*e.rows_dev)) : M;
}

__device__ __forceinline__ bf16x8 ld_nt(const bf16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p));
}

// ---------------------------------------------------------------- streaming
template <int NW, int KSPLIT, int DEPTH, bool XF>
__global__ __launch_bounds__(64 * KSPLIT) void gemm_stream_bf16(const bf16_t* __restrict__ X, int M, int K, int ldx,
                                                               const bf16_t* __restrict__ W, int N, EpiArgs e) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, g = lane >> 4;
    const int nb0 = blockIdx.x * NW;
    const int KU = K / 64;
    // this workgroup's k units: [u_begin, u_end) of split blockIdx.y
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int u_begin = (int)((long)KU * split / nsplit), u_end = (int)((long)KU * (split + 1) / nsplit);

    floatx4 acc[NW][4];
#pragma unroll
    for (int j = 0; j < NW; ++j)
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) acc[j][mb] = floatx4{0.f, 0.f, 0.f, 0.f};

    const bf16_t* wp[NW];
#pragma unroll
    for (int j = 0; j < NW; ++j) wp[j] = W + (size_t)min(nb0 + j, N / 16 - 1) * KU * 1024 + 8 * lane;
    // X row-major: lane (lr, g) reads token 16mb+lr at k 64u + 16g + 8h; X
    // fragment-major: 1 KB block (mb, u), half h at +512h, lane at +8*lane.
    // Token blocks past the last one re-read it (their results are not stored).
    const bf16_t* xp[4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
        xp[mb] = XF ? X + (size_t)min(mb, (M - 1) >> 4) * KU * 1024 + 8 * lane
                    : X + (size_t)min(16 * mb + lr, M - 1) * ldx + 16 * g;
    constexpr int xu = XF ? 1024 : 64, xh = XF ? 512 : 8;   // element steps per k unit / half

    bf16x8 wb[DEPTH][NW][2], xb[DEPTH][4][2];
    auto load = [&](int s, int u) {
#pragma unroll
        for (int j = 0; j < NW; ++j) {
            wb[s][j][0] = ld_nt(wp[j] + (size_t)u * 1024);
            wb[s][j][1] = ld_nt(wp[j] + (size_t)u * 1024 + 512);
        }
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            xb[s][mb][0] = ld_bf16x8(xp[mb] + (size_t)xu * u);
            xb[s][mb][1] = ld_bf16x8(xp[mb] + (size_t)xu * u + xh);
        }
    };
#pragma unroll
    for (int s = 0; s < DEPTH; ++s) {
        const int u = u_begin + wave + s * KSPLIT;
        if (u < u_end) load(s, u);
    }
    for (int base = u_begin + wave; base < u_end; base += DEPTH * KSPLIT) {
#pragma unroll
        for (int s = 0; s < DEPTH; ++s) {
            const int u = base + s * KSPLIT;
            if (u < u_end) {
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int j = 0; j < NW; ++j)
#pragma unroll
                        for (int mb = 0; mb < 4; ++mb) acc[j][mb] = mfma16x16x32(wb[s][j][h], xb[s][mb][h], acc[j][mb]);
                const int un = u + DEPTH * KSPLIT;
                if (un < u_end) load(s, un);
            }
        }
    }

    // Sum the KSPLIT partial tiles through LDS in wave order; wave w then
    // finishes token blocks [NQ w, NQ (w + 1)) so the epilogue runs on every wave.
    static_assert(4 % KSPLIT == 0, "KSPLIT divides the 4 token blocks");
    constexpr int NQ = 4 / KSPLIT;
    const int mb0 = wave * NQ;
    floatx4 res[NW][NQ];
    if constexpr (KSPLIT > 1) {
        __shared__ floatx4 red[KSPLIT][NW * 4][64];
#pragma unroll
        for (int j = 0; j < NW; ++j)
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) red[wave][j * 4 + mb][lane] = acc[j][mb];
        __syncthreads();
#pragma unroll
        for (int j = 0; j < NW; ++j)
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                floatx4 t = red[0][j * 4 + mb0 + q][lane];
#pragma unroll
                for (int w = 1; w < KSPLIT; ++w) t += red[w][j * 4 + mb0 + q][lane];
                res[j][q] = t;
            }
    } else {
#pragma unroll
        for (int j = 0; j < NW; ++j)
#pragma unroll
            for (int q = 0; q < NQ; ++q) res[j][q] = acc[j][q];
    }
    EpiArgs ee = e;
    if (e.kind == EPI_PARTIAL) ee.y = e.y + (size_t)split * M * e.ldy;
    const int Mv = valid_rows(e, M);
    with_kind(e.kind, [&](auto kind) {
        constexpr int EK = decltype(kind)::value;
        float4 pre[NW][NQ];
#pragma unroll
        for (int j = 0; j < NW; ++j)
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int n = 16 * (nb0 + j) + 4 * g, m = 16 * (mb0 + q) + lr;
                pre[j][q] = (m < Mv && n < N) ? epi_fetch<EK>(ee, m, n) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
        for (int j = 0; j < NW; ++j)
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int n = 16 * (nb0 + j) + 4 * g, m = 16 * (mb0 + q) + lr;
                if (m < Mv && n < N) epi_store<bf16_t, EK>(ee, m, n, res[j][q], pre[j][q]);
            }
    });
}

// ---------------------------------------------------------------- pipelined tiles
// M > 64 (prefill, large batches) with fragment-major X.  A workgroup owns a
// 128-token x (32 WN)-column output tile; wave (wm, wn) computes tokens
// 64wm..64wm+63 x 16 WN columns with WN x 4 accumulator tiles.  Per 64-wide k
// unit the workgroup copies the 2 WN weight blocks and 8 activation blocks it
// needs (both fragment-major, so every 16-byte chunk is a plain copy) into one
// of two LDS stages; each thread holds its chunks of the next two units in a
// register ring, so global loads run two units ahead of the MFMAs and one
// barrier per unit separates the stages.  An optional split of K across
// workgroups writes fp32 partials (EPI_PARTIAL).
constexpr int PBM = 128;

template <int WN>
struct PipeTile {
    static constexpr int BN = 32 * WN;              // output columns per workgroup
    static constexpr int CHW = BN / 16 * 128;       // 16-byte weight chunks per stage
    static constexpr int CHX = PBM / 16 * 128;      // activation chunks per stage
    static constexpr int CH = CHW + CHX;
    static constexpr int PER = CH / 256;            // chunks per thread per unit
};

template <int WN>
__global__ __launch_bounds__(256, WN <= 4 ? 2 : 1) void gemm_pipe_bf16(const bf16_t* __restrict__ X, int M, int K,
                                                      const bf16_t* __restrict__ W, int N, EpiArgs e,
                                                      int tiles_m, int tiles_n) {
    using T = PipeTile<WN>;
    __shared__ bf16x8 lds[2][T::CH];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = lane & 15, g = lane >> 4;
    // XCD-aware order (workgroups are dealt round-robin to the 8 XCDs): each
    // XCD gets a contiguous run of tiles, m fastest, so tiles sharing a weight
    // panel share that XCD's L2
    const int total = tiles_m * tiles_n;
    int bid = blockIdx.x;
    if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
    const int tm = bid % tiles_m, tn = bid / tiles_m;
    const int Mv = valid_rows(e, M);
    if (tm * PBM >= Mv) return;   // the whole row tile is past the kept rows
    const int KU = K / 64, NB = N / 16, MB = (M + 15) / 16;
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int u_begin = (int)((long)KU * split / nsplit), u_end = (int)((long)KU * (split + 1) / nsplit);
    const int nu = u_end - u_begin;

    // this thread's chunks: c = tid + 256 i; c < CHW: weight block c / 128 of
    // the tile, else activation block (c - CHW) / 128; blocks past the matrix
    // re-read its last block (their results are never stored)
    // Loads go through buffer descriptors (base and size in scalar registers,
    // 32-bit byte offsets per lane; the hardware returns 0 past the size).
    static_assert(T::CHW % 256 == 0, "a thread's chunks are all weight or all activation");
    // (the library rejects bf16 weight matrices of 4 GiB or more, so the byte
    // counts fit the descriptors' 32-bit record field)
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void*)W, (short)0, (int)(uint32_t)((size_t)NB * KU * 2048), 0x00020000);
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        (void*)X, (short)0, (int)(uint32_t)((size_t)MB * KU * 2048), 0x00020000);
    uint32_t off[T::PER];
#pragma unroll
    for (int i = 0; i < T::PER; ++i) {
        const int c = tid + 256 * i;
        if (i < T::CHW / 256) {
            const int nb = min(tn * (T::BN / 16) + c / 128, NB - 1);
            off[i] = ((uint32_t)nb * KU * 1024 + (c & 127) * 8) * 2;
        } else {
            const int mb = min(tm * (PBM / 16) + (c - T::CHW) / 128, MB - 1);
            off[i] = ((uint32_t)mb * KU * 1024 + (c & 127) * 8) * 2;
        }
    }
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    bf16x8 ring[2][T::PER];
    auto gload = [&](int slot, int u) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < T::PER; ++i) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(i < T::CHW / 256 ? rw : rx,
                                                                  off[i] + (uint32_t)u * 2048, 0, 0);
            ring[slot][i] = __builtin_bit_cast(bf16x8, v);
        }
    };
    auto sstore = [&](int stage, int slot) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < T::PER; ++i) lds[stage][tid + 256 * i] = ring[slot][i];
    };

    floatx4 acc[WN][4];
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int stage) __attribute__((always_inline)) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            bf16x8 af[WN], bfr[4];
#pragma unroll
            for (int j = 0; j < WN; ++j) af[j] = lds[stage][(wn * WN + j) * 128 + h * 64 + lane];
#pragma unroll
            for (int i = 0; i < 4; ++i) bfr[i] = lds[stage][T::CHW + (wm * 4 + i) * 128 + h * 64 + lane];
#pragma unroll
            for (int j = 0; j < WN; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[j][i] = mfma16x16x32(af[j], bfr[i], acc[j][i]);
        }
    };

    // Unit k lives in ring slot k % 2 and LDS stage k % 2.  The loop body is
    // two straight-line steps with no data-dependent branch, so each LDS store
    // waits only for its own slot's loads while the other slot's are in
    // flight; prefetches past the last unit re-read the last unit and their
    // stages are never computed.
    const int last = u_begin + (nu > 0 ? nu - 1 : 0);
    gload(0, u_begin);
    gload(1, min(u_begin + 1, last));
    sstore(0, 0);
    gload(0, min(u_begin + 2, last));
    for (int k = 0; k < nu; k += 2) {
        __syncthreads();   // stage 0 holds unit k; stage 1 is no longer read
        sstore(1, 1);      // unit k + 1
        gload(1, min(u_begin + k + 3, last));
        compute(0);
        if (k + 1 >= nu) break;
        __syncthreads();   // stage 1 holds unit k + 1; stage 0 is no longer read
        sstore(0, 0);      // unit k + 2
        gload(0, min(u_begin + k + 4, last));
        compute(1);
    }

    EpiArgs ee = e;
    if (e.kind == EPI_PARTIAL) ee.y = e.y + (size_t)split * M * e.ldy;
    const int nb0 = tn * (T::BN / 16) + wn * WN, m0 = tm * PBM + wm * 64;
    with_kind(e.kind, [&](auto kind) {
        constexpr int EK = decltype(kind)::value;
#pragma unroll
        for (int jh = 0; jh < WN / 2; ++jh) {   // pairs of column blocks: bounds the prefetch registers
            float4 pre[2][4];
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = 16 * (nb0 + 2 * jh + j) + 4 * g, m = m0 + 16 * i + lr;
                    pre[j][i] = (m < Mv && n < N) ? epi_fetch<EK>(ee, m, n) : make_float4(0.f, 0.f, 0.f, 0.f);
                }
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = 16 * (nb0 + 2 * jh + j) + 4 * g, m = m0 + 16 * i + lr;
                    if (m < Mv && n < N) epi_store<bf16_t, EK>(ee, m, n, acc[2 * jh + j][i], pre[j][i]);
                }
        }
    });
}

// ---------------------------------------------------------------- large tiles
// M >= 256 (prefill of long prefixes, large batches) with fragment-major X.
// A workgroup of 4 waves (2 x 2) owns a (32 TI)-token x (32 TJ)-column output
// tile; wave (wm, wn) computes 16 TI tokens x 16 TJ columns with TI x TJ
// accumulator tiles, so every operand read from LDS feeds 8 or 4 MFMAs.  The
// K loop runs over 32-wide slices (one half of a 64-wide fragment-major unit,
// 1 KB per 16-row block): a slice stage is the 2 TI activation halves and the
// 2 TJ weight halves the tile needs, copied with global_load_lds straight into
// LDS in the layout the MFMA operand reads use (a wave's read is 1 KB
// contiguous, so conflict-free).  NST stages keep the copies NST - 1 slices
// ahead of the MFMAs with one barrier per slice; the barrier is the plain
// s_barrier, since __syncthreads() would also wait for the newer copies.
// OCC workgroups share a CU (the launches use 2, so one workgroup's copy
// waits and barriers overlap the other's MFMAs).
template <int LPW>
__device__ __forceinline__ void wait_copies(int newer) {   // all but the newest `newer` slices' copies
    switch (newer) {
    case 0: __builtin_amdgcn_s_waitcnt(waitcnt_vm(0)); break;
    case 1: __builtin_amdgcn_s_waitcnt(waitcnt_vm(LPW)); break;
    case 2: __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * LPW)); break;
    default: __builtin_amdgcn_s_waitcnt(waitcnt_vm(3 * LPW)); break;
    }
}

template <int TI, int TJ, int NST, int OCC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void gemm_big_bf16(const bf16_t* __restrict__ X, int M, int K, const bf16_t* __restrict__ W, int N, EpiArgs e,
                   int tiles_m, int tiles_n) {
    constexpr int XB = 2 * TI, WB = 2 * TJ;        // 16-row blocks per tile side
    constexpr int STAGE = (XB + WB) * 1024;        // bytes per slice stage
    constexpr int LPW = (XB + WB) / 4;             // 1 KB copies per wave per slice
    static_assert((XB + WB) % 4 == 0, "whole copies per wave");
    static_assert(NST >= 2 && NST <= 5 && 3 * LPW <= 63, "stage count and vmcnt range");
    static_assert(NST * STAGE >= 4 * (TJ / 2) * TI * 1024, "the epilogue's parking space fits the stages");
    typedef __attribute__((address_space(3))) void* lds_ptr;
    typedef __attribute__((address_space(1))) void* glb_ptr;
    __shared__ __attribute__((aligned(16))) char smem[NST * STAGE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = lane & 15, g = lane >> 4;
    // XCD-aware order (workgroups are dealt round-robin to the 8 XCDs): each
    // XCD gets a contiguous run of tiles, m fastest, so the tiles that share a
    // weight panel share that XCD's L2
    const int total = tiles_m * tiles_n;
    int bid = blockIdx.x;
    if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
    const int tm = bid % tiles_m, tn = bid / tiles_m;
    const int Mv = valid_rows(e, M);
    if (tm * 32 * TI >= Mv) return;   // the whole row tile is past the kept rows
    const int KU = K / 64, NB = N / 16, MB = (M + 15) / 16;
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int u_begin = (int)((long)KU * split / nsplit), u_end = (int)((long)KU * (split + 1) / nsplit);
    const int s_begin = 2 * u_begin, nsl = 2 * (u_end - u_begin);

    // this wave's copies: block q = wave * LPW + j of the stage, activation
    // blocks first; blocks past the matrix re-read its last block (their
    // results are never stored)
    const bf16_t* src[LPW];
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
        const int q = wave * LPW + j;
        if (q < XB) {
            const int mb = min(tm * XB + q, MB - 1);
            src[j] = X + (size_t)mb * KU * 1024 + 8 * lane;
        } else {
            const int nb = min(tn * WB + (q - XB), NB - 1);
            src[j] = W + (size_t)nb * KU * 1024 + 8 * lane;
        }
    }
    // slice sl of a block: unit sl / 2, half sl % 2
    auto issue = [&](int sl, int stage) __attribute__((always_inline)) {
        const size_t off = (size_t)(sl >> 1) * 1024 + (sl & 1) * 512;
        char* dst = smem + stage * STAGE + wave * LPW * 1024;
#pragma unroll
        for (int j = 0; j < LPW; ++j)
            __builtin_amdgcn_global_load_lds((glb_ptr)(src[j] + off), (lds_ptr)(dst + j * 1024), 16, 0, 0);
    };

    floatx4 acc[TJ][TI];
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int i = 0; i < TI; ++i) acc[j][i] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int stage) __attribute__((always_inline)) {
        const char* st = smem + stage * STAGE;
        bf16x8 xf[TI], wf[TJ];
#pragma unroll
        for (int i = 0; i < TI; ++i) xf[i] = *reinterpret_cast<const bf16x8*>(st + (wm * TI + i) * 1024 + 16 * lane);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
            wf[j] = *reinterpret_cast<const bf16x8*>(st + (XB + wn * TJ + j) * 1024 + 16 * lane);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int i = 0; i < TI; ++i) acc[j][i] = mfma16x16x32(wf[j], xf[i], acc[j][i]);
    };

    // Slice t lives in stage t % NST.  Step t waits for its own copies (the
    // newer ones stay in flight), and the barrier both publishes them and
    // retires every wave's reads of slice t - 1, whose stage the copy of slice
    // t + NST - 1 then overwrites.
#pragma unroll
    for (int p = 0; p < NST - 1; ++p)
        if (p < nsl) issue(s_begin + p, p);
    for (int t = 0; t < nsl; ++t) {
        wait_copies<LPW>(min(nsl - 1 - t, NST - 2));
        // (no compiler barrier around it: one keeps the accumulators out of
        // registers; the LDS reads of the step follow its copy issue, and the
        // barrier has side effects, so nothing moves across it)
        __builtin_amdgcn_s_barrier();
        if (t + NST - 1 < nsl) issue(s_begin + t + NST - 1, (t + NST - 1) % NST);
        compute(t % NST);
    }

    // Epilogue through LDS, half the column blocks at a time: each wave parks
    // its accumulators in its own LDS region (written straight from the
    // accumulator registers) and reads them back one tile at a time, which
    // keeps the epilogue's registers small.  Every wave has finished reading
    // the slice stages once it passes the barrier.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __builtin_amdgcn_s_barrier();
    EpiArgs ee = e;
    if (e.kind == EPI_PARTIAL) ee.y = e.y + (size_t)split * M * e.ldy;
    const int nb0 = tn * WB + wn * TJ, m0 = tm * 32 * TI + wm * 16 * TI;
    constexpr int kPark = (TJ / 2) * TI * 64;       // floatx4 slots of one wave's parking region
    floatx4* park = reinterpret_cast<floatx4*>(smem) + wave * kPark + lane;
    with_kind(e.kind, [&](auto kind) {
        constexpr int EK = decltype(kind)::value;
        // LM head with fused confidence partials: per row, (max, first argmax,
        // sum of exp(l - max)) over the tile's columns (Eq. 1)
        const bool parts = EK == EPI_LMHEAD && e.lpart != nullptr;
        SmPart pt[TI];
#pragma unroll
        for (int i = 0; i < TI; ++i) pt[i] = SmPart{-INFINITY, 0x7fffffff, 0.f};
        // the halves are separate instances (compile-time indices into acc,
        // which must stay in registers)
        auto half = [&](auto hjc) __attribute__((always_inline)) {
            constexpr int hj = decltype(hjc)::value;
#pragma unroll
            for (int j = 0; j < TJ / 2; ++j)
#pragma unroll
                for (int i = 0; i < TI; ++i) park[(j * TI + i) * 64] = acc[hj * (TJ / 2) + j][i];
            asm volatile("" ::: "memory");   // the tiles are read back from LDS, not forwarded
#pragma unroll
            for (int j = 0; j < TJ / 2; ++j) {
                const int n = 16 * (nb0 + hj * (TJ / 2) + j) + 4 * g;
                float4 pre[TI];
#pragma unroll
                for (int i = 0; i < TI; ++i) {
                    const int m = m0 + 16 * i + lr;
                    pre[i] = (m < Mv && n < N) ? epi_fetch<EK>(ee, m, n) : make_float4(0.f, 0.f, 0.f, 0.f);
                }
#pragma unroll
                for (int i = 0; i < TI; ++i) {
                    const int m = m0 + 16 * i + lr;
                    if (m < Mv && n < N) epi_store<bf16_t, EK>(ee, m, n, park[(j * TI + i) * 64], pre[i]);
                }
            }
            if constexpr (EK == EPI_LMHEAD) {
                if (parts) {
                    // this half's columns: the maximum and its first column, then
                    // the sum of exp2(l log2e - mb) (mb = max log2e rounded once;
                    // its rounding error, common to every term, is corrected at the end)
                    constexpr float kL2e = 1.4426950408889634f;
#pragma unroll
                    for (int i = 0; i < TI; ++i) {
                        SmPart h{-INFINITY, 0x7fffffff, 0.f};
#pragma unroll
                        for (int j = 0; j < TJ / 2; ++j) {
                            const int n = 16 * (nb0 + hj * (TJ / 2) + j) + 4 * g;
                            if (n < N) {
                                const floatx4 v = park[(j * TI + i) * 64];
#pragma unroll
                                for (int q = 0; q < 4; ++q)
                                    if (v[q] > h.m) { h.m = v[q]; h.a = n + q; }
                            }
                        }
                        const float mb = h.m * kL2e;
#pragma unroll
                        for (int j = 0; j < TJ / 2; ++j) {
                            const int n = 16 * (nb0 + hj * (TJ / 2) + j) + 4 * g;
                            if (n < N) {
                                const floatx4 v = park[(j * TI + i) * 64];
#pragma unroll
                                for (int q = 0; q < 4; ++q) h.s += __builtin_amdgcn_exp2f(fmaf(v[q], kL2e, -mb));
                            }
                        }
                        if (h.m != -INFINITY) h.s *= exp2f(-fmaf(h.m, kL2e, -mb));
                        pt[i] = smpart_merge(pt[i], h);
                    }
                }
            }
        };
        half(Kind<0>{});
        half(Kind<1>{});
        if constexpr (EK == EPI_LMHEAD) {
            if (parts) {
                // merge the four column groups of a row (lanes lr + 16 g), then the
                // two waves that share the rows (wn = 0 holds the lower columns)
#pragma unroll
                for (int i = 0; i < TI; ++i)
#pragma unroll
                    for (int o = 16; o < 64; o <<= 1) {
                        const SmPart y{__shfl_xor(pt[i].m, o, 64), __shfl_xor(pt[i].a, o, 64),
                                       __shfl_xor(pt[i].s, o, 64)};
                        pt[i] = smpart_merge(pt[i], y);
                    }
                // wave wn = 1 leaves its partials in its own (finished) parking region
                float* mine = reinterpret_cast<float*>(reinterpret_cast<floatx4*>(smem) + wave * kPark);
                if (wn == 1 && g == 0) {
#pragma unroll
                    for (int i = 0; i < TI; ++i) {
                        mine[(i * 16 + lr) * 3 + 0] = pt[i].m;
                        mine[(i * 16 + lr) * 3 + 1] = __int_as_float(pt[i].a);
                        mine[(i * 16 + lr) * 3 + 2] = pt[i].s;
                    }
                }
                __syncthreads();
                if (wn == 0 && g == 0) {
                    const float* other = reinterpret_cast<const float*>(reinterpret_cast<floatx4*>(smem) +
                                                                        (wave + 1) * kPark);
#pragma unroll
                    for (int i = 0; i < TI; ++i) {
                        const int m = m0 + 16 * i + lr;
                        const SmPart y{other[(i * 16 + lr) * 3 + 0], __float_as_int(other[(i * 16 + lr) * 3 + 1]),
                                       other[(i * 16 + lr) * 3 + 2]};
                        const SmPart r = smpart_merge(pt[i], y);
                        if (m < Mv) {
                            float* o = e.lpart + ((size_t)m * e.ntile + tn) * 3;
                            o[0] = r.m;
                            o[1] = __int_as_float(r.a);
                            o[2] = r.s;
                        }
                    }
                }
            }
        }
    });
}

// ---------------------------------------------------------------- tiled
constexpr int TBM = 128, TBN = 128, TBK = 64, TPAD = TBK + 8;

__global__ __launch_bounds__(256) void gemm_tiled_bf16(const bf16_t* __restrict__ X, int M, int K, int ldx,
                                                       const bf16_t* __restrict__ W, int N, EpiArgs e,
                                                       int tiles_m, int tiles_n) {
    __shared__ __attribute__((aligned(16))) bf16_t Ws[8 * 1024];      // 8 fragment blocks of one k unit
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
    const int nb_base = tn * (TBN / 16), m0 = tm * TBM;
    const int wn = wave & 1, wm = wave >> 1;
    const int KU = K / 64, NB = N / 16;

    floatx4 acc[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = floatx4{0.f, 0.f, 0.f, 0.f};

    bf16x8 wr[4], xr[4];
    auto gload = [&](int u) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int c = threadIdx.x + 256 * it;      // 16-byte chunk of the 16 KB tile
            const int nbl = c >> 7, off = c & 127;
            wr[it] = ld_bf16x8(W + ((size_t)min(nb_base + nbl, NB - 1) * KU + u) * 1024 + off * 8);
            const int row = c >> 3, c8 = c & 7;
            xr[it] = ld_bf16x8(X + (size_t)min(m0 + row, M - 1) * ldx + u * 64 + c8 * 8);
        }
    };
    auto sstore = [&]() {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int c = threadIdx.x + 256 * it;
            *reinterpret_cast<bf16x8*>(&Ws[c * 8]) = wr[it];
            const int row = c >> 3, c8 = c & 7;
            *reinterpret_cast<bf16x8*>(&Xs[row * TPAD + c8 * 8]) = xr[it];
        }
    };
    gload(0);
    for (int u = 0; u < KU; ++u) {
        __syncthreads();
        sstore();
        __syncthreads();
        if (u + 1 < KU) gload(u + 1);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            bf16x8 af[4], bfr[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                af[j] = *reinterpret_cast<const bf16x8*>(&Ws[(wn * 4 + j) * 1024 + hh * 512 + lane * 8]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                bfr[i] = *reinterpret_cast<const bf16x8*>(&Xs[(wm * 64 + 16 * i + lr) * TPAD + 16 * g + 8 * hh]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[j][i] = mfma16x16x32(af[j], bfr[i], acc[j][i]);
        }
    }
    with_kind(e.kind, [&](auto kind) {
        constexpr int EK = decltype(kind)::value;
        float4 pre[4][4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = 16 * (nb_base + wn * 4 + j) + 4 * g, m = m0 + wm * 64 + 16 * i + lr;
                pre[j][i] = (m < M && n < N) ? epi_fetch<EK>(e, m, n) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = 16 * (nb_base + wn * 4 + j) + 4 * g, m = m0 + wm * 64 + 16 * i + lr;
                if (m < M && n < N) epi_store<bf16_t, EK>(e, m, n, acc[j][i], pre[j][i]);
            }
    });
}

// ---------------------------------------------------------------- fp32
// One thread per (token, 4 output columns); 16 tokens x 16 column-quads per
// workgroup with the K loop staged through LDS in 32-wide slices.  Row-major W.
__global__ __launch_bounds__(256) void gemm_f32(const float* __restrict__ X, int M, int K, int ldx,
                                                const float* __restrict__ W, int N, EpiArgs e) {
    __shared__ float xs[16][33];
    __shared__ float ws[64][33];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int m = blockIdx.y * 16 + ty;
    const int n = blockIdx.x * 64 + tx * 4;
    const int Mv = valid_rows(e, M);
    if (blockIdx.y * 16 >= Mv) return;   // the whole row block is past the kept rows
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
    if (m < Mv && n < N)
        with_kind(e.kind, [&](auto kind) {
            constexpr int EK = decltype(kind)::value;
            epi_store<float, EK>(e, m, n, floatx4{acc[0], acc[1], acc[2], acc[3]}, epi_fetch<EK>(e, m, n));
        });
}

// Fragment-major packing of a bf16 weight matrix (see the file comment), with
// an optional row permutation: mode 1 puts rotary pairs (t, t + dh/2) of each
// head on adjacent rows, mode 2 interleaves the rows of src0 (gate) and src1
// (up).  One thread per 16-byte piece.
__global__ void pack_frag_kernel(const bf16_t* __restrict__ src0, const bf16_t* __restrict__ src1,
                                 bf16_t* __restrict__ dst, int N, int K, int mode, int dh) {
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)N * K / 8;
    if (t >= total) return;
    const int KU = K / 64;
    const int lane = t & 63;
    const int h = (t >> 6) & 1;
    const size_t blk = t >> 7;                // (nb, u)
    const int u = blk % KU, nb = blk / KU;
    const int row = 16 * nb + (lane & 15);
    const int k0 = 64 * u + 16 * (lane >> 4) + 8 * h;
    const bf16_t* src;
    if (mode == 1) {
        const int head = row / dh, e = row % dh, tt = e / 2;
        src = src0 + (size_t)(head * dh + ((e & 1) ? tt + dh / 2 : tt)) * K;
    } else if (mode == 2) {
        src = ((row & 1) ? src1 : src0) + (size_t)(row / 2) * K;
    } else {
        src = src0 + (size_t)row * K;
    }
    *reinterpret_cast<bf16x8*>(dst + t * 8) = *reinterpret_cast<const bf16x8*>(src + k0);
}

}  // namespace

hipError_t launch_pack_frag(const void* src0, const void* src1, void* dst, int N, int K, int mode, int dh,
                            hipStream_t s) {
    const size_t total = (size_t)N * K / 8;
    launch(pack_frag_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                       (const bf16_t*)src0, (const bf16_t*)src1, (bf16_t*)dst, N, K, mode, dh);
    return hipGetLastError();
}

// Configuration of the streaming kernel for one projection shape:
//   nw     16-column blocks per wave (wave tile 16*nw columns)
//   ks     waves per workgroup splitting K
//   depth  k units in flight per wave
//   split  workgroups splitting K (fp32 partials, reduced by the consumer)
// Chosen from measurements on MI355X at 64 tokens.  Every wave reads all 64
// token rows of its k units (8 KB per unit), so a wider wave tile amortises
// that over more weight columns: the widest of 8, 6, 4, 3 column blocks whose
// grid still covers the 256 CUs; otherwise the tile that fills the CUs most
// evenly, with 4 waves per workgroup.  The O and down projections, whose
// 4096-wide output has too few column tiles, split K 4 ways instead, with 4
// waves per workgroup splitting K again (3 k units in flight for the long K
// of the down projection).
struct StreamCfg {
    int nw, ks, depth, split;
};

StreamCfg stream_cfg(int N, int K, bool partial) {
    const int KU = K / 64;
    if (partial) {
        int S = 4;
        while (S > 1 && KU / S < 8) S /= 2;
        if (N % 64 == 0) return K > 4096 ? StreamCfg{4, 4, 3, S} : StreamCfg{4, 4, 2, S};
        return StreamCfg{1, 4, 2, S};
    }
    for (int c : {8, 6}) {
        if (N % (16 * c) == 0 && N / (16 * c) >= 256) return c == 8 ? StreamCfg{8, 2, 3, 1} : StreamCfg{6, 4, 3, 1};
    }
    int nw = 0;
    double best = -1.0;
    for (int c : {4, 3}) {
        if (N % (16 * c)) continue;
        const int grid = N / (16 * c);
        const double eff = (double)grid / (((grid + 255) / 256) * 256);
        if (eff > best + 1e-9) { best = eff; nw = c; }
    }
    if (nw == 0) nw = N % 32 == 0 ? 2 : 1;
    const int grid = N / (16 * nw);
    const int ks = grid <= 256 ? 4 : 2;
    const int depth = (nw == 3 && ks == 4) ? 3 : 2;
    return StreamCfg{nw, ks, depth, 1};
}

// K split of the pipelined kernel (O and down projections, whose residual
// epilogue can take fp32 partials): measured on MI355X at 512-736 tokens, 4
// ways while the tiles alone give fewer than 256 workgroups, 2 below 512; at
// least 8 k units per split.
int pipe_split(int M, int N, int K) {
    const int tiles = ((M + PBM - 1) / PBM) * ((N + PipeTile<4>::BN - 1) / PipeTile<4>::BN);
    int S = tiles < 256 ? 4 : (tiles < 512 ? 2 : 1);
    while (S > 1 && K / 64 / S < 8) S /= 2;
    return S;
}

// Large-tile kernel choice for M >= 256: two workgroups per CU, tiles of
// 256 x 128 (A), 128 x 256 (B), 128 x 128 (C) or 128 x 192 (D) tokens x
// columns.  The time model is rounds of 512 workgroups times the work of one
// tile over its relative throughput (a round costs about the same however
// full it is), fitted to kernel-trace sweeps on MI355X over the 7B batch-8
// and 8B batch-32 steps (1024 / 2048 rows) and prefills of 640 to 26624
// rows: A 1.0, B 0.97 (1.2 from 4096 rows, where each XCD's run of tiles
// shares a wider weight panel), C 0.72, D 0.9 (D only without a K split: as
// split-K partials it measured 12-24 % slower than A at 640 rows; with full
// sums it takes 9-17 % off the QKV and gate/up projections of 700-800-row
// prefills and 4 % off the 8B batch-32 QKV).  Partial (split-K) epilogues
// split K while there are fewer than two workgroups per CU, keeping at least
// 8 k units per split.
struct BigCfg {
    int ti, tj, split;   // ti == 0: use the pipelined kernel
};
BigCfg big_cfg(int M, int N, int K, bool partial, bool no192 = false) {
    if (M < 256) return BigCfg{0, 0, 1};
    const int cand[4][2] = {{8, 4}, {4, 8}, {4, 4}, {4, 6}};
    const double eff[4] = {1.0, M >= 4096 ? 1.2 : 0.97, 0.72, 0.9};
    BigCfg best{0, 0, 1};
    double best_t = 0.0;
    for (int v = 0; v < 4; ++v) {
        if (v == 3 && (partial || no192)) continue;
        const int ti = cand[v][0], tj = cand[v][1];
        const long tiles = (long)((M + 32 * ti - 1) / (32 * ti)) * ((N + 32 * tj - 1) / (32 * tj));
        int S = 1;
        if (partial)
            while (S < 4 && tiles * S < 512 && K / 64 / (2 * S) >= 8) S *= 2;
        const double t = (double)((tiles * S + 511) / 512) * (32.0 * ti) * (32.0 * tj) * ((double)K / S) / eff[v];
        if (best.ti == 0 || t < best_t) {
            best = BigCfg{ti, tj, S};
            best_t = t;
        }
    }
    return best;
}

void gemm_plan(int dtype, int M, int N, int K, bool partial, bool xfrag, int32_t* plan, bool fused_head) {
    plan[1] = plan[2] = 0;
    plan[3] = 1;
    if (dtype == DARD_DTYPE_F32) {
        plan[0] = DARD_GEMM_F32;
        return;
    }
    if (M <= 64) {
        const StreamCfg c = stream_cfg(N, K, partial);
        plan[0] = DARD_GEMM_STREAM;
        plan[1] = 4;
        plan[2] = c.nw;
        plan[3] = c.split;
        return;
    }
    if (!xfrag) {
        plan[0] = DARD_GEMM_TILED;
        plan[1] = TBM / 32;
        plan[2] = TBN / 32;
        return;
    }
    const BigCfg c = big_cfg(M, N, K, partial, fused_head);
    if (c.ti) {
        plan[0] = DARD_GEMM_BIG;
        plan[1] = c.ti;
        plan[2] = c.tj;
        plan[3] = c.split;
        return;
    }
    plan[0] = DARD_GEMM_PIPE;
    plan[1] = PBM / 32;
    plan[2] = PipeTile<4>::BN / 32;
    plan[3] = partial ? pipe_split(M, N, K) : 1;
}

int gemm_split(int dtype, int M, int N, int K) {
    if (dtype != DARD_DTYPE_BF16) return 1;
    if (M > 64) {
        const BigCfg c = big_cfg(M, N, K, true);
        return c.ti ? c.split : pipe_split(M, N, K);
    }
    return stream_cfg(N, K, true).split;
}

hipError_t launch_gemm(int dtype, const void* X, int M, int K, int ldx, const void* W, int N,
                       const EpiArgs& e, int kernel_class, hipStream_t s, bool xfrag) {
    TraceScope ts(kernel_class, s);
    if (e.kind == EPI_LMHEAD && (!e.rowmap || !e.rows_dev || !e.y)) return hipErrorInvalidValue;
    // fused LM-head partials: only the large-tile kernel forms them
    if (e.kind == EPI_LMHEAD && e.lpart && (dtype != DARD_DTYPE_BF16 || M <= 64 || !xfrag))
        return hipErrorInvalidValue;
    if (dtype == DARD_DTYPE_F32) {
        dim3 grid((N + 63) / 64, (M + 15) / 16);
        launch(gemm_f32, grid, dim3(256), 0, s, reinterpret_cast<const float*>(X), M, K, ldx,
                           reinterpret_cast<const float*>(W), N, e);
        return hipGetLastError();
    }
    const bf16_t* x = reinterpret_cast<const bf16_t*>(X);
    const bf16_t* w = reinterpret_cast<const bf16_t*>(W);
    if (xfrag && !frag_rows(dtype, M)) return hipErrorInvalidValue;
    if (M <= 64) {
        const StreamCfg c = stream_cfg(N, K, e.kind == EPI_PARTIAL);
        const dim3 grid(N / (16 * c.nw), c.split), block(64 * c.ks);
#define DARD_GS(NW, KS, D)                                                                               \
    do {                                                                                                 \
        if (xfrag) launch((gemm_stream_bf16<NW, KS, D, true>), grid, block, 0, s, x, M, K, ldx, w, N, e);  \
        else launch((gemm_stream_bf16<NW, KS, D, false>), grid, block, 0, s, x, M, K, ldx, w, N, e);       \
    } while (0)
        if (c.nw == 8) DARD_GS(8, 2, 3);
        else if (c.nw == 6) DARD_GS(6, 4, 3);
        else if (c.nw == 4 && c.ks == 4 && c.depth == 3) DARD_GS(4, 4, 3);
        else if (c.nw == 4 && c.ks == 4) DARD_GS(4, 4, 2);
        else if (c.nw == 4) DARD_GS(4, 2, 2);
        else if (c.nw == 3 && c.ks == 4) DARD_GS(3, 4, 3);
        else if (c.nw == 3) DARD_GS(3, 2, 2);
        else if (c.nw == 2) DARD_GS(2, 4, 2);
        else DARD_GS(1, 4, 2);
#undef DARD_GS
        return hipGetLastError();
    }
    if (xfrag) {
        // the fused LM-head partials need tile widths that divide the 8192-logit chunks
        const BigCfg c = big_cfg(M, N, K, e.kind == EPI_PARTIAL, e.kind == EPI_LMHEAD && e.lpart);
        if (c.ti && e.kind == EPI_LMHEAD && e.lpart && e.ntile != (N + 32 * c.tj - 1) / (32 * c.tj))
            return hipErrorInvalidValue;
        if (c.ti) {
            const int tiles_m = (M + 32 * c.ti - 1) / (32 * c.ti), tiles_n = (N + 32 * c.tj - 1) / (32 * c.tj);
            const dim3 grid(tiles_m * tiles_n, c.split);
            if (c.ti == 8)
                launch(gemm_big_bf16<8, 4, 3, 2>, grid, dim3(256), 0, s, x, M, K, w, N, e, tiles_m, tiles_n);
            else if (c.tj == 8)
                launch(gemm_big_bf16<4, 8, 3, 2>, grid, dim3(256), 0, s, x, M, K, w, N, e, tiles_m, tiles_n);
            else if (c.tj == 6)
                launch(gemm_big_bf16<4, 6, 4, 2>, grid, dim3(256), 0, s, x, M, K, w, N, e, tiles_m, tiles_n);
            else
                launch(gemm_big_bf16<4, 4, 5, 2>, grid, dim3(256), 0, s, x, M, K, w, N, e, tiles_m, tiles_n);
            return hipGetLastError();
        }
        if (e.kind == EPI_LMHEAD && e.lpart) return hipErrorInvalidValue;   // partials need the large tiles
        const int tiles_m = (M + PBM - 1) / PBM, tiles_n = (N + PipeTile<4>::BN - 1) / PipeTile<4>::BN;
        const int S = e.kind == EPI_PARTIAL ? pipe_split(M, N, K) : 1;
        launch(gemm_pipe_bf16<4>, dim3(tiles_m * tiles_n, S), dim3(256), 0, s, x, M, K, w, N, e, tiles_m, tiles_n);
        return hipGetLastError();
    }
    const int tiles_m = (M + TBM - 1) / TBM, tiles_n = (N + TBN - 1) / TBN;
    launch(gemm_tiled_bf16, dim3(tiles_m * tiles_n), dim3(256), 0, s, x, M, K, ldx, w, N, e,
                       tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace dard
