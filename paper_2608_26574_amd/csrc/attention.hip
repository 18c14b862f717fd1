// State-masked attention over the augmented block (Sec. 2, Sec. 3.2).
//
// bf16 path: flash-style.  A workgroup serves 64 query rows of one (sequence,
// query head) with G groups of 4 waves (16 rows per wave); the groups take
// interleaved 64-key tiles of the workgroup's key range and are merged
// through LDS at the end, so a short key range costs few serial steps
// without any cross-workgroup synchronisation.  Per group, K tiles are staged
// in LDS row-major and V tiles transposed (key-contiguous), so that both
// products run on v_mfma_f32_16x16x32_bf16:
//   S^T = K * Q^T   (A = K rows from LDS, B = this wave's Q rows in registers)
//   O^T += V^T P^T  (A = V^T from LDS, B = probabilities straight from the
//                    S^T accumulators; the MFMA k index is permuted so that a
//                    lane's 8 probabilities are its own score values)
// Keys are tiled in two runs: the prefix [0, P) in 64-key tiles, then the
// block [P, P + 2B) (x^j at P+j, s^j at P+B+j) in 64-key tiles of its own.  A
// row's block visibility is the "take x" word of the state mask (Eq. 2-3,
// built once per step) widened to 2B bits: x^j where the bit is set, s^j
// where it is clear; so one aligned 64-bit word per block tile says which
// keys a row sees, and full prefix tiles need no test at all.
// Very long key ranges are additionally split across workgroups and merged
// by a log-sum-exp combine kernel.
//
// fp32 path: one thread per (row, head), plain online softmax.
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr int kKeys = 64;      // keys per tile
constexpr int kMaxSplit = 16;  // key splits across workgroups
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinLog2 = -1e30f;   // running-max floor (log2 units): exp2 of anything below it is 0

// LDS of one group of TPG threads: a K tile row-major and a V tile transposed
// (or, at the end, every lane's o, m and l for the merge of the groups).
template <int DH, int TPG>
struct Lds {
    static constexpr int KPAD = DH + 8;       // K row stride (bf16): 16-byte bank shift per row
    static constexpr int VPAD = kKeys + 4;    // V^T row stride (bf16)
    static constexpr int TILE_BYTES = (kKeys * KPAD + DH * VPAD) * 2;
    static constexpr int MERGE_BYTES = (DH / 4 + 2) * TPG * 4;
    static constexpr int GROUP_BYTES = ((TILE_BYTES > MERGE_BYTES ? TILE_BYTES : MERGE_BYTES) + 15) / 16 * 16;
};

// The 2B-bit block visibility of a row from its take-x words (x1:x0), B <= 128:
// bit j (j < B) = x bit j, bit B + j = NOT x bit j; returned as 4 words.
__device__ __forceinline__ void block_vis(uint64_t x0, uint64_t x1, int B, uint64_t& v0, uint64_t& v1,
                                          uint64_t& v2, uint64_t& v3) {
    const uint64_t m0 = B >= 64 ? ~0ull : (1ull << B) - 1;
    const uint64_t m1 = B >= 128 ? ~0ull : (B > 64 ? (1ull << (B - 64)) - 1 : 0ull);
    x0 &= m0;
    x1 &= m1;
    const uint64_t s0 = ~x0 & m0, s1 = ~x1 & m1;
    // word i of the 256-bit value (0 : 0 : s1 : s0) << B
    const int q = B >> 6, r = B & 63;
    // source word j of (s1 : s0), zero outside
#define DARD_SRC(j) ((j) == 0 ? s0 : ((j) == 1 ? s1 : 0ull))
#define DARD_SHL(i) (r ? (DARD_SRC((i) - q) << r) | (DARD_SRC((i) - q - 1) >> (64 - r)) : DARD_SRC((i) - q))
    v0 = x0 | DARD_SHL(0);
    v1 = x1 | DARD_SHL(1);
    v2 = DARD_SHL(2);
    v3 = DARD_SHL(3);
#undef DARD_SHL
#undef DARD_SRC
}

// First key and key count of tile t (npre prefix tiles over [0, pre_end),
// then block tiles over [P, P + 2B)).
__device__ __forceinline__ int tile_first(int t, int npre, int P) { return t < npre ? t * kKeys : P + (t - npre) * kKeys; }
__device__ __forceinline__ int tile_count(int t, int npre, int pre_end, int B2) {
    return t < npre ? min(kKeys, pre_end - t * kKeys) : min(kKeys, B2 - (t - npre) * kKeys);
}

// G groups of WPG waves; a workgroup serves 16 WPG query rows of one
// (sequence, query head) and its groups take interleaved key tiles.
template <int DH, int G, int RING, int WPG>
__global__ __launch_bounds__(64 * WPG * G) void attn_bf16_kernel(AttnArgs a, int rowtiles, int tiles_per_split) {
    constexpr int TPG = 64 * WPG, ROWS = 16 * WPG;
    using L = Lds<DH, TPG>;
    constexpr int KPAD = L::KPAD, VPAD = L::VPAD;
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    __shared__ __attribute__((aligned(16))) char smem[G * L::GROUP_BYTES];

    // group and wave are wave-uniform: say so, so that tile bookkeeping stays scalar
    const int grp = __builtin_amdgcn_readfirstlane(threadIdx.x / TPG), tid = threadIdx.x % TPG;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 15, g = lane >> 4;
    bf16_t* Ks = reinterpret_cast<bf16_t*>(smem + grp * L::GROUP_BYTES);
    bf16_t* Vt = Ks + kKeys * KPAD;
    int bid = blockIdx.x;
    const int rt = bid % rowtiles; bid /= rowtiles;
    const int h = bid % a.Hq;
    const int s = bid / a.Hq;
    const int kvh = h / (a.Hq / a.Hkv);
    const int r0 = rt * ROWS;
    const int split = blockIdx.y, nsplit = gridDim.y;

    // prefix tiles [0, npre), then block tiles (masked mode)
    const int pre_end = a.masked ? a.P : a.nkeys;
    const int npre = (pre_end + kKeys - 1) / kKeys;
    const int ntiles = npre + (a.masked ? (2 * a.B + kKeys - 1) / kKeys : 0);
    const int t_begin = split * tiles_per_split;
    const int t_end = min(ntiles, t_begin + tiles_per_split);
    const int iters = (t_end - t_begin + G - 1) / G;   // tile steps of every group
    const int P = a.P, B2 = 2 * a.B;

    const bf16_t* q = reinterpret_cast<const bf16_t*>(a.q);
    const bf16_t* kbase = reinterpret_cast<const bf16_t*>(a.k) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    const bf16_t* vbase = reinterpret_cast<const bf16_t*>(a.v) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;

    // ---- issue the loads of this group's first RING tiles before anything else
    constexpr int KCH = kKeys * DH / 8 / TPG;  // 16-byte K chunks per thread
    constexpr int VUNITS = (kKeys / 4) * (DH / 8);           // (4 keys x 8 dims) V units per tile
    constexpr int VQ = (VUNITS + TPG - 1) / TPG;              // V units per thread
    bf16x8 kreg[RING][KCH];
    bf16x8 vreg[RING][VQ][4];
    auto load_tile = [&](int slot, int tile) __attribute__((always_inline)) {
        const int k0 = tile_first(tile, npre, P), n = tile_count(tile, npre, pre_end, B2);
        const bf16_t* kt = kbase + (size_t)k0 * DH;
        const bf16_t* vt = vbase + (size_t)k0 * DH;
        // V unit u = tid + TPG v: (kg, dg) = (u % 16, u / 16) holds keys
        // 4kg..4kg+3 at dims 8dg..8dg+7
        if (n == kKeys) {   // full tile (uniform): no per-key test
#pragma unroll
            for (int it = 0; it < KCH; ++it) kreg[slot][it] = ld_bf16x8(kt + (size_t)(tid + TPG * it) * 8);
#pragma unroll
            for (int vq = 0; vq < VQ; ++vq) {
                const int u = tid + TPG * vq, kg = u & 15, dg = u >> 4;
                if (u < VUNITS) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        vreg[slot][vq][e] = ld_bf16x8(vt + (size_t)(4 * kg + e) * DH + dg * 8);
                }
            }
        } else {
#pragma unroll
            for (int it = 0; it < KCH; ++it) {
                const int qd = tid + TPG * it;
                bf16x8 z = {};
                kreg[slot][it] = qd / (DH / 8) < n ? ld_bf16x8(kt + (size_t)qd * 8) : z;
            }
#pragma unroll
            for (int vq = 0; vq < VQ; ++vq) {
                const int u = tid + TPG * vq, kg = u & 15, dg = u >> 4;
                if (u < VUNITS) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int key = 4 * kg + e;
                        bf16x8 z = {};
                        vreg[slot][vq][e] = key < n ? ld_bf16x8(vt + (size_t)key * DH + dg * 8) : z;
                    }
                }
            }
        }
    };
    auto store_tile = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
        for (int it = 0; it < KCH; ++it) {
            const int qd = tid + TPG * it;
            const int key = qd / (DH / 8), c8 = qd % (DH / 8);
            *reinterpret_cast<bf16x8*>(&Ks[key * KPAD + c8 * 8]) = kreg[slot][it];
        }
        // 16 consecutive lanes write one contiguous 128-byte run of a V^T row
#pragma unroll
        for (int vq = 0; vq < VQ; ++vq) {
            const int u = tid + TPG * vq, kg = u & 15, dg = u >> 4;
            if (u < VUNITS) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    bf16x4 t4 = {vreg[slot][vq][0][e], vreg[slot][vq][1][e], vreg[slot][vq][2][e],
                                 vreg[slot][vq][3][e]};
                    *reinterpret_cast<bf16x4*>(&Vt[(dg * 8 + e) * VPAD + 4 * kg]) = t4;
                }
            }
        }
    };
#pragma unroll
    for (int sl = 0; sl < RING; ++sl) {
        const int tile = t_begin + grp + G * sl;
        if (sl < iters && tile < t_end) load_tile(sl, tile);
    }

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
    // this lane's row of the state mask, widened to the block's 2B keys
    uint64_t bv0 = 0, bv1 = 0, bv2 = 0, bv3 = 0;
    if (a.masked && row_ok) {
        const int W = (a.B + 63) / 64;
        const uint64_t* sp = a.sel + ((size_t)s * a.R + my_row) * W;
        block_vis(sp[0], W > 1 ? sp[1] : 0ull, a.B, bv0, bv1, bv2, bv3);
    }
    const float sl2 = a.scale * kLog2e;

    floatx4 o[DH / 16];
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[d] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run = kMinLog2, l_run = 0.f;

    auto compute_tile = [&](int tile) __attribute__((always_inline)) {
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
        // ---- visibility: only tiles with block keys or a ragged end test it
        // (tile and n are wave-uniform, so this is a scalar branch)
        const int n = tile_count(tile, npre, pre_end, B2);
        if (!(tile < npre && n == kKeys)) {
            uint64_t vis;
            if (tile < npre) {
                vis = (1ull << n) - 1;     // n < 64 here
            } else {
                // word bt of the block visibility, selected with masks (a select
                // chain here becomes a lookup table in private memory)
                const uint64_t bt = (uint64_t)(tile - npre);
                vis = (bv0 & (0ull - (uint64_t)(bt == 0))) | (bv1 & (0ull - (uint64_t)(bt == 1))) |
                      (bv2 & (0ull - (uint64_t)(bt == 2))) | (bv3 & (0ull - (uint64_t)(bt == 3)));
            }
            // this lane's keys 16kb + 4g + i: bits 16(kb%2) + i of w[kb/2]
            const uint32_t w0 = (uint32_t)vis >> (4 * g), w1 = (uint32_t)(vis >> 32) >> (4 * g);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (!(((kb < 2 ? w0 : w1) >> (16 * (kb & 1) + i)) & 1u)) sc[kb][i] = -INFINITY;
        }
        // ---- online softmax in the log2 domain; the running max starts at a
        // finite floor, so rows with no visible key yet need no special case
        float mt = sc[0][0];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sc[kb][i]);
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float m_new = fmaxf(m_run, mt * sl2);     // sl2 > 0: the max commutes with the scale
        // arguments are <= 0: the hardware exp2 (v_exp_f32) needs no range handling
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        float psum = 0.f;
        bf16x8 pb[2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = __builtin_amdgcn_exp2f(fmaf(sc[kb][i], sl2, -m_new));
                psum += p;
                pb[kb >> 1][(kb & 1) * 4 + i] = (__bf16)p;
            }
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
        if (__ballot(alpha != 1.f)) {             // some row's max moved
#pragma unroll
            for (int d = 0; d < DH / 16; ++d) o[d] *= alpha;
        }
        // ---- O^T += V^T * P^T
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const bf16_t* vp = &Vt[(16 * d + lr) * VPAD + 32 * c + 4 * g];
                const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vp);
                const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vp + 16);
                const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                o[d] = mfma16x16x32(vf, pb[c], o[d]);
            }
        }
    };

    for (int base = 0; base < iters; base += RING) {
#pragma unroll
        for (int sl = 0; sl < RING; ++sl) {
            const int it = base + sl;
            if (it < iters) {                     // uniform across the workgroup
                const int tile = t_begin + grp + G * it;
                const bool mine = tile < t_end;
                __syncthreads();                  // the previous tiles are fully consumed
                if (mine) store_tile(sl);
                __syncthreads();
                if (mine) {
                    const int next = tile + G * RING;
                    if (next < t_end) load_tile(sl, next);
                    compute_tile(tile);
                }
            }
        }
    }

    // ---- merge the groups through LDS (group 0 keeps the result)
    if constexpr (G > 1) {
        __syncthreads();
        float* mb = reinterpret_cast<float*>(smem + grp * L::GROUP_BYTES);
        if (grp > 0) {
#pragma unroll
            for (int d = 0; d < DH / 16; ++d)
#pragma unroll
                for (int i = 0; i < 4; ++i) mb[(4 * d + i) * TPG + tid] = o[d][i];
            mb[(DH / 4) * TPG + tid] = m_run;
            mb[(DH / 4 + 1) * TPG + tid] = l_run;
        }
        __syncthreads();
        if (grp > 0) return;
        float M = m_run;
#pragma unroll
        for (int gg = 1; gg < G; ++gg)
            M = fmaxf(M, reinterpret_cast<const float*>(smem + gg * L::GROUP_BYTES)[(DH / 4) * TPG + tid]);
        const float f0 = m_run == -INFINITY ? 0.f : exp2f(m_run - M);
        float lsum = l_run * f0;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) o[d] *= f0;
#pragma unroll
        for (int gg = 1; gg < G; ++gg) {
            const float* ob = reinterpret_cast<const float*>(smem + gg * L::GROUP_BYTES);
            const float mg = ob[(DH / 4) * TPG + tid];
            const float f = mg == -INFINITY ? 0.f : exp2f(mg - M);
            lsum += ob[(DH / 4 + 1) * TPG + tid] * f;
#pragma unroll
            for (int d = 0; d < DH / 16; ++d)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[d][i] += ob[(4 * d + i) * TPG + tid] * f;
        }
        m_run = M;
        l_run = lsum;
    }

    // ---- epilogue: row sum over the 4 lanes sharing a row
    float l_tot = l_run + __shfl_xor(l_run, 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);
    if (!row_ok) return;
    const size_t nrow = (size_t)a.b * a.R * a.Hq;
    const size_t orow = ((size_t)s * a.R + my_row) * a.Hq + h;
    if (nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        bf16_t* out = reinterpret_cast<bf16_t*>(a.out);
        const int tok = s * a.R + my_row, KO = a.Hq * DH;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) {
            const uint32_t w0 = (uint32_t)f2bf(o[d][0] * inv) | ((uint32_t)f2bf(o[d][1] * inv) << 16);
            const uint32_t w1 = (uint32_t)f2bf(o[d][2] * inv) | ((uint32_t)f2bf(o[d][3] * inv) << 16);
            const int k = h * DH + 16 * d + 4 * g;
            *reinterpret_cast<uint2*>(out + (a.out_frag ? frag_off(tok, k, KO) : orow * DH + 16 * d + 4 * g)) =
                make_uint2(w0, w1);
        }
        return;
    }
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

// Merge key splits: O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M).  One
// thread per (row, head, 4 dims); every load of a thread is issued up front.
template <int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part,
                                                           const float* __restrict__ part_ml, int ns,
                                                           size_t nrow, int Hq, int frag,
                                                           bf16_t* __restrict__ out) {
    const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t row = t / (DH / 4);
    const int q4 = t % (DH / 4);
    if (row >= nrow) return;
    float m[kMaxSplit], l[kMaxSplit];
    float4 ov[kMaxSplit];
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) {
        if (sp < ns) {
            m[sp] = part_ml[(sp * nrow + row) * 2];
            l[sp] = part_ml[(sp * nrow + row) * 2 + 1];
            ov[sp] = reinterpret_cast<const float4*>(part + (sp * nrow + row) * DH)[q4];
        } else {
            m[sp] = -INFINITY;
            l[sp] = 0.f;
            ov[sp] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) M = fmaxf(M, m[sp]);
    float Lsum = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) {
        if (m[sp] == -INFINITY) continue;
        const float f = exp2f(m[sp] - M);
        Lsum += l[sp] * f;
        acc.x += ov[sp].x * f; acc.y += ov[sp].y * f; acc.z += ov[sp].z * f; acc.w += ov[sp].w * f;
    }
    const float inv = Lsum > 0.f ? 1.f / Lsum : 0.f;
    const uint32_t w0 = (uint32_t)f2bf(acc.x * inv) | ((uint32_t)f2bf(acc.y * inv) << 16);
    const uint32_t w1 = (uint32_t)f2bf(acc.z * inv) | ((uint32_t)f2bf(acc.w * inv) << 16);
    const size_t o = frag ? frag_off((int)(row / Hq), (int)(row % Hq) * DH + 4 * q4, Hq * DH) : row * DH + 4 * q4;
    *reinterpret_cast<uint2*>(out + o) = make_uint2(w0, w1);
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

// Shape of a bf16 launch: WPG waves per group (16 WPG query rows per
// workgroup) and G groups taking interleaved key tiles.  While one-group
// workgroups of 64 rows would leave the chip short of 1024 waves, the key
// tiles are walked by more groups: 4 groups of 2 waves (32 rows per
// workgroup, so a head's 64 rows take two workgroups) when there are at least
// 4 tiles, else 2 groups of 4 waves.
struct AttnCfg {
    int wpg, g;
};

AttnCfg attention_cfg(int b, int R, int Hq, int ntiles) {
    const int wgs64 = b * Hq * ((R + 63) / 64);
    if (4 * wgs64 >= 1024 || ntiles < 2) return {4, 1};
    if (R > 32 && ntiles >= 4) return {2, 4};
    return {4, 2};
}

}  // namespace

int attention_tiles(int masked, int P, int B, int nkeys) {
    return masked ? (P + kKeys - 1) / kKeys + (2 * B + kKeys - 1) / kKeys : (nkeys + kKeys - 1) / kKeys;
}

int attention_splits(int dtype, int b, int R, int Hq, int ntiles, size_t slots) {
    if (dtype != DARD_DTYPE_BF16) return 1;
    const AttnCfg c = attention_cfg(b, R, Hq, ntiles);
    const int wgs = b * Hq * ((R + 16 * c.wpg - 1) / (16 * c.wpg));
    // Measured at 64 rows x 32 heads: a tile step costs about 2 us, the
    // combine kernel about 4.3 us plus its launch, so a split pays only when
    // the workgroups would otherwise walk more than 5 tile steps; then about
    // 3 tiles per split.  No split once the workgroups alone cover the chip.
    if (wgs * c.g * c.wpg >= 1024 || (ntiles + c.g - 1) / c.g <= 5) return 1;
    int ns = 1;
    while (ns < kMaxSplit && ntiles > 3 * ns) ns *= 2;
    const size_t per_split = (size_t)b * R * Hq;
    while (ns > 1 && (size_t)ns * per_split > slots) --ns;
    if (ns <= 1) return 1;
    const int tps = (ntiles + ns - 1) / ns;
    return (ntiles + tps - 1) / tps;      // no empty split
}

size_t attention_partial_slots(int dtype, int b, int R, int Hq, int ntiles) {
    const int ns = attention_splits(dtype, b, R, Hq, ntiles, (size_t)-1);
    return ns <= 1 ? 0 : (size_t)ns * b * R * Hq;
}

hipError_t launch_attention_splits(int dtype, const AttnArgs& a, int ns, hipStream_t s) {
    if (a.out_frag && !frag_rows(dtype, a.b * a.R)) return hipErrorInvalidValue;
    if (dtype == DARD_DTYPE_BF16) {
        if (a.masked && (!a.sel || a.B > 128)) return hipErrorInvalidValue;
        const int ntiles = attention_tiles(a.masked, a.P, a.B, a.nkeys);
        const bool can_split = a.part && a.part_ml;
        if (!can_split || ns < 1 || ns > kMaxSplit || (size_t)ns * a.b * a.R * a.Hq > a.part_slots) ns = 1;
        if (ns > ntiles) ns = ntiles > 0 ? ntiles : 1;
        const int tps = (ntiles + ns - 1) / ns;
        ns = ntiles > 0 ? (ntiles + tps - 1) / tps : 1;
        const AttnCfg c = attention_cfg(a.b, a.R, a.Hq, tps);
        const int rowtiles = (a.R + 16 * c.wpg - 1) / (16 * c.wpg);
        dim3 grid(a.b * a.Hq * rowtiles, ns);
#define DARD_ATT(DHV, GV, WV) \
    launch((attn_bf16_kernel<DHV, GV, WV == 2 ? 1 : 2, WV>), grid, dim3(64 * WV * GV), 0, s, a, rowtiles, tps)
        if (a.dh == 128) {
            if (c.wpg == 2) DARD_ATT(128, 4, 2); else if (c.g == 2) DARD_ATT(128, 2, 4); else DARD_ATT(128, 1, 4);
        } else {
            if (c.wpg == 2) DARD_ATT(64, 4, 2); else if (c.g == 2) DARD_ATT(64, 2, 4); else DARD_ATT(64, 1, 4);
        }
#undef DARD_ATT
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || ns == 1) return e;
        const size_t nrow = (size_t)a.b * a.R * a.Hq;
        const size_t threads = nrow * (a.dh / 4);
        if (a.dh == 128)
            launch(attn_combine_kernel<128>, dim3((threads + 255) / 256), dim3(256), 0, s, a.part,
                               a.part_ml, ns, nrow, a.Hq, a.out_frag, reinterpret_cast<bf16_t*>(a.out));
        else
            launch(attn_combine_kernel<64>, dim3((threads + 255) / 256), dim3(256), 0, s, a.part,
                               a.part_ml, ns, nrow, a.Hq, a.out_frag, reinterpret_cast<bf16_t*>(a.out));
        return hipGetLastError();
    }
    const size_t total = (size_t)a.b * a.R * a.Hq;
    dim3 grid((total + 63) / 64);
    if (a.dh == 128)
        launch(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
    else
        launch(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
    const bool can_split = a.part && a.part_ml;
    const int ns = can_split ? attention_splits(dtype, a.b, a.R, a.Hq, attention_tiles(a.masked, a.P, a.B, a.nkeys),
                                                a.part_slots)
                             : 1;
    return launch_attention_splits(dtype, a, ns, s);
}

}  // namespace dard
