// State-masked attention over the augmented block (Sec. 2, Sec. 3.2).
//
// bf16 path: flash-style, one workgroup = 64 query rows of one (sequence,
// query head), 4 waves of 16 rows.  K tiles of 64 keys are staged in LDS
// row-major, V tiles transposed (key-contiguous), so that both products run on
// v_mfma_f32_16x16x32_bf16:
//   S^T = K * Q^T   (A = K rows from LDS, B = this wave's Q rows in registers)
//   O^T += V^T P^T  (A = V^T from LDS, B = probabilities straight from the
//                    S^T accumulators; the MFMA k index is permuted so that a
//                    lane's 8 probabilities are its own score values)
// The mask is built in-kernel: each row's "take x" bits (Eq. 2-3) live in LDS;
// prefix keys are always visible, block key P+j is x^j, P+B+j is s^j.
// Long key ranges are split across workgroups (flash-decoding) and merged by
// a log-sum-exp combine.
//
// fp32 path: one thread per (row, head), plain online softmax.
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr int kRows = 64;   // query rows per workgroup
constexpr int kKeys = 64;   // keys per tile
constexpr float kLog2e = 1.4426950408889634f;

struct MaskSmem {
    uint64_t sel[kRows][2];
};

// Row visibility bits for the rows [r0, r0 + 64) of sequence s.
__device__ void build_row_bits(const AttnArgs& a, int s, int r0, uint8_t* st, float* cf,
                               uint64_t (*sel)[2]) {
    for (int j = threadIdx.x; j < a.B; j += blockDim.x) {
        st[j] = a.state[(size_t)s * a.B + j];
        cf[j] = a.conf[(size_t)s * a.B + j];
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kRows * 2; t += blockDim.x) {
        const int rl = t >> 1, w = t & 1;
        const int r = r0 + rl;
        uint64_t word = 0;
        if (r < a.R) {
            const int i = r % a.B;
            const bool shadow = r >= a.B;
            const int j0 = w * 64, j1 = min(a.B, j0 + 64);
            for (int j = j0; j < j1; ++j)
                if (take_x(st[i], st[j], cf[i], cf[j], shadow, i == j, a.flags))
                    word |= 1ull << (j - j0);
        }
        sel[rl][w] = word;
    }
    __syncthreads();
}

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a, int rowtiles, int tiles_per_split) {
    constexpr int KPAD = DH + 8;      // K row stride (bf16): 16-byte bank shift per row
    constexpr int VPAD = kKeys + 4;   // V^T row stride (bf16)
    __shared__ __attribute__((aligned(16))) bf16_t Ks[kKeys * KPAD];
    __shared__ __attribute__((aligned(16))) bf16_t Vt[DH * VPAD];
    __shared__ uint64_t sel[kRows][2];
    __shared__ uint8_t st[128];
    __shared__ float cf[128];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, g = lane >> 4;
    int bid = blockIdx.x;
    const int rt = bid % rowtiles; bid /= rowtiles;
    const int h = bid % a.Hq;
    const int s = bid / a.Hq;
    const int kvh = h / (a.Hq / a.Hkv);
    const int r0 = rt * kRows;
    const int split = blockIdx.y;

    const int ntiles = (a.nkeys + kKeys - 1) / kKeys;
    const int t_begin = split * tiles_per_split;
    const int t_end = min(ntiles, t_begin + tiles_per_split);
    const int key_end = min(a.nkeys, t_end * kKeys);

    if (a.masked) build_row_bits(a, s, r0, st, cf, sel);

    const bf16_t* q = reinterpret_cast<const bf16_t*>(a.q);
    const bf16_t* kbase = reinterpret_cast<const bf16_t*>(a.k) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    const bf16_t* vbase = reinterpret_cast<const bf16_t*>(a.v) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;

    // this lane's query row and its Q fragments (B operand of S^T = K Q^T)
    const int my_row = r0 + wave * 16 + lr;
    const bool row_ok = my_row < a.R;
    bf16x8 qf[DH / 32];
    {
        const bf16_t* qp = q + (((size_t)s * a.R + (row_ok ? my_row : 0)) * a.Hq + h) * DH;
#pragma unroll
        for (int c = 0; c < DH / 32; ++c) {
            bf16x8 z = {};
            qf[c] = row_ok ? ld_bf16x8(qp + 32 * c + 8 * g) : z;
        }
    }
    const uint64_t sel0 = a.masked ? sel[wave * 16 + lr][0] : 0;
    const uint64_t sel1 = a.masked ? sel[wave * 16 + lr][1] : 0;
    const float sl2 = a.scale * kLog2e;

    floatx4 o[DH / 16];
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[d] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    // cooperative tile loads: K 4 chunks of 16 B per thread, V 4 rows x 16 B
    constexpr int KCH = kKeys * DH / 8 / 256;  // 16-byte K chunks per thread
    constexpr int VUNITS = (kKeys / 4) * (DH / 8);
    bf16x8 kreg[KCH];
    bf16x8 vreg[4];
    auto load_tile = [&](int tile) {
        const int kb0 = tile * kKeys;
#pragma unroll
        for (int it = 0; it < KCH; ++it) {
            const int qd = threadIdx.x + 256 * it;
            const int key = qd / (DH / 8), c8 = qd % (DH / 8);
            const int kabs = kb0 + key;
            bf16x8 z = {};
            kreg[it] = kabs < key_end ? ld_bf16x8(kbase + (size_t)kabs * DH + c8 * 8) : z;
        }
        if (threadIdx.x < VUNITS) {
            const int kg = threadIdx.x / (DH / 8), dg = threadIdx.x % (DH / 8);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int kabs = kb0 + 4 * kg + e;
                bf16x8 z = {};
                vreg[e] = kabs < key_end ? ld_bf16x8(vbase + (size_t)kabs * DH + dg * 8) : z;
            }
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int it = 0; it < KCH; ++it) {
            const int qd = threadIdx.x + 256 * it;
            const int key = qd / (DH / 8), c8 = qd % (DH / 8);
            *reinterpret_cast<bf16x8*>(&Ks[key * KPAD + c8 * 8]) = kreg[it];
        }
        if (threadIdx.x < VUNITS) {
            const int kg = threadIdx.x / (DH / 8), dg = threadIdx.x % (DH / 8);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                bf16x4 t4 = {vreg[0][e], vreg[1][e], vreg[2][e], vreg[3][e]};
                *reinterpret_cast<bf16x4*>(&Vt[(dg * 8 + e) * VPAD + 4 * kg]) = t4;
            }
        }
    };

    if (t_begin < t_end) load_tile(t_begin);
    for (int tile = t_begin; tile < t_end; ++tile) {
        __syncthreads();   // previous tile fully consumed
        store_tile();
        __syncthreads();
        if (tile + 1 < t_end) load_tile(tile + 1);

        // ---- S^T = K * Q^T for this wave's 16 rows: 4 blocks of 16 keys
        floatx4 sc[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < DH / 32; ++c) {
                const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[(16 * kb + lr) * KPAD + 32 * c + 8 * g]);
                acc = mfma16x16x32(kf, qf[c], acc);
            }
            sc[kb] = acc;
        }
        // ---- scale, mask, tile max
        const int kb0 = tile * kKeys;
        float mt = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = kb0 + 16 * kb + 4 * g + i;
                bool vis = key < key_end;
                if (a.masked && key >= a.P) {
                    const int j = key - a.P;
                    const int jj = j < a.B ? j : j - a.B;
                    const uint64_t word = jj < 64 ? sel0 : sel1;
                    const bool bx = (word >> (jj & 63)) & 1ull;
                    vis = vis && (j < a.B ? bx : !bx);
                }
                const float v = vis ? sc[kb][i] * sl2 : -INFINITY;
                sc[kb][i] = v;
                mt = fmaxf(mt, v);
            }
        }
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float m_new = fmaxf(m_run, mt);
        const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m_run - m_new);
        float psum = 0.f;
        bf16x8 pb[2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = (m_new == -INFINITY) ? 0.f : exp2f(sc[kb][i] - m_new);
                psum += p;
                pb[kb >> 1][(kb & 1) * 4 + i] = (__bf16)p;
            }
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) o[d] *= alpha;

        // ---- O^T += V^T * P^T
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                const bf16_t* vp = &Vt[(16 * d + lr) * VPAD + 32 * c + 4 * g];
                const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vp);
                const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vp + 16);
                const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                o[d] = mfma16x16x32(vf, pb[c], o[d]);
            }
        }
    }

    // ---- epilogue: row sum over the 4 lanes sharing a row
    float l_tot = l_run + __shfl_xor(l_run, 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);
    if (!row_ok) return;
    const size_t orow = ((size_t)s * a.R + my_row) * a.Hq + h;
    if (gridDim.y == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        bf16_t* out = reinterpret_cast<bf16_t*>(a.out) + orow * DH;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) {
            uint32_t w0 = (uint32_t)f2bf(o[d][0] * inv) | ((uint32_t)f2bf(o[d][1] * inv) << 16);
            uint32_t w1 = (uint32_t)f2bf(o[d][2] * inv) | ((uint32_t)f2bf(o[d][3] * inv) << 16);
            *reinterpret_cast<uint2*>(out + 16 * d + 4 * g) = make_uint2(w0, w1);
        }
    } else {
        const size_t nrow = (size_t)a.b * a.R * a.Hq;
        float* po = a.part + ((size_t)split * nrow + orow) * DH;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d)
            *reinterpret_cast<float4*>(po + 16 * d + 4 * g) = make_float4(o[d][0], o[d][1], o[d][2], o[d][3]);
        if (g == 0) {
            float* pm = a.part_ml + ((size_t)split * nrow + orow) * 2;
            pm[0] = m_run;
            pm[1] = l_tot;
        }
    }
}

// Merge split partials: O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M).
template <typename T>
__global__ __launch_bounds__(128) void attn_combine_kernel(const float* __restrict__ part,
                                                           const float* __restrict__ part_ml,
                                                           int nsplit, size_t nrow, int dh,
                                                           T* __restrict__ out) {
    const size_t row = blockIdx.x;
    float M = -INFINITY;
    for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, part_ml[(sp * nrow + row) * 2]);
    float L = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
        const float m = part_ml[(sp * nrow + row) * 2];
        if (m != -INFINITY) L += part_ml[(sp * nrow + row) * 2 + 1] * exp2f(m - M);
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    for (int e = threadIdx.x; e < dh; e += blockDim.x) {
        float acc = 0.f;
        for (int sp = 0; sp < nsplit; ++sp) {
            const float m = part_ml[(sp * nrow + row) * 2];
            if (m != -INFINITY) acc += part[(sp * nrow + row) * dh + e] * exp2f(m - M);
        }
        St<T>::st(out + row * dh + e, acc * inv);
    }
}

// fp32 path: one thread per (sequence, row, head).
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)a.b * a.R * a.Hq;
    if (t >= total) return;
    const int h = t % a.Hq;
    const int r = (t / a.Hq) % a.R;
    const int s = t / ((size_t)a.Hq * a.R);
    const int kvh = h / (a.Hq / a.Hkv);
    const float* q = reinterpret_cast<const float*>(a.q) + t * DH;
    const float* kb = reinterpret_cast<const float*>(a.k) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    const float* vb = reinterpret_cast<const float*>(a.v) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    float qr[DH], o[DH];
    for (int e = 0; e < DH; ++e) { qr[e] = q[e]; o[e] = 0.f; }
    float m = -INFINITY, l = 0.f;
    const int i = a.masked ? r % a.B : 0;
    const bool shadow = a.masked && r >= a.B;
    const uint8_t* st = a.masked ? a.state + (size_t)s * a.B : nullptr;
    const float* cf = a.masked ? a.conf + (size_t)s * a.B : nullptr;
    for (int key = 0; key < a.nkeys; ++key) {
        if (a.masked && key >= a.P) {
            const int j = key - a.P;
            const int jj = j < a.B ? j : j - a.B;
            const bool bx = take_x(st[i], st[jj], cf[i], cf[jj], shadow, i == jj, a.flags);
            if (bx != (j < a.B)) continue;
        }
        float sdot = 0.f;
        for (int e = 0; e < DH; ++e) sdot += qr[e] * kb[(size_t)key * DH + e];
        sdot *= a.scale;
        const float mn = fmaxf(m, sdot);
        const float alpha = expf(m - mn);
        const float p = expf(sdot - mn);
        l = l * alpha + p;
        for (int e = 0; e < DH; ++e) o[e] = o[e] * alpha + p * vb[(size_t)key * DH + e];
        m = mn;
    }
    float* out = reinterpret_cast<float*>(a.out) + t * DH;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    for (int e = 0; e < DH; ++e) out[e] = o[e] * inv;
}

}  // namespace

int attention_splits(int dtype, int b, int R, int Hq, int nkeys, size_t slots) {
    if (dtype != DARD_DTYPE_BF16) return 1;
    const int rowtiles = (R + kRows - 1) / kRows;
    const int ntiles = (nkeys + kKeys - 1) / kKeys;
    const int wgs = b * Hq * rowtiles;
    int ns = (512 + wgs - 1) / wgs;       // aim at >= 512 workgroups
    ns = ns < 1 ? 1 : (ns > ntiles ? ntiles : ns);
    if (ns > 16) ns = 16;
    // never more partial slots (split, row, head) than the workspace holds
    const size_t per_split = (size_t)b * R * Hq;
    while (ns > 1 && (size_t)ns * per_split > slots) --ns;
    if (ns <= 1 || ntiles == 0) return 1;
    const int tps = (ntiles + ns - 1) / ns;
    return (ntiles + tps - 1) / tps;      // no empty split
}

size_t attention_partial_slots(int dtype, int b, int R, int Hq, int nkeys) {
    const int ns = attention_splits(dtype, b, R, Hq, nkeys, (size_t)-1);
    return ns <= 1 ? 0 : (size_t)ns * b * R * Hq;
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
    if (dtype == DARD_DTYPE_BF16) {
        const int rowtiles = (a.R + kRows - 1) / kRows;
        const int ntiles = (a.nkeys + kKeys - 1) / kKeys;
        const int ns = (a.part && a.part_ml) ? attention_splits(dtype, a.b, a.R, a.Hq, a.nkeys, a.part_slots) : 1;
        const int tps = (ntiles + ns - 1) / ns;
        dim3 grid(a.b * a.Hq * rowtiles, ns);
        if (a.dh == 128)
            hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(256), 0, s, a, rowtiles, tps);
        else
            hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(256), 0, s, a, rowtiles, tps);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || ns == 1) return e;
        const size_t nrow = (size_t)a.b * a.R * a.Hq;
        hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, dim3(nrow), dim3(128), 0, s, a.part,
                           a.part_ml, ns, nrow, a.dh, reinterpret_cast<bf16_t*>(a.out));
        return hipGetLastError();
    }
    const size_t total = (size_t)a.b * a.R * a.Hq;
    dim3 grid((total + 63) / 64);
    if (a.dh == 128)
        hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
    else
        hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
    return hipGetLastError();
}

}  // namespace dard
