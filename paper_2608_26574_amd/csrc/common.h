// Device-side helpers shared by the gfx950 kernels of libdard.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dard.h"

namespace dard {

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bfloat16, round to nearest even (finite inputs).
__device__ __forceinline__ bf16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

// Storage-type traits: activations and weights are either float or bf16.
template <typename T> struct St;
template <> struct St<float> {
    static __device__ __forceinline__ float ld(const float* p) { return *p; }
    static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
    static __device__ __forceinline__ float cvt(float v) { return v; }
};
template <> struct St<bf16_t> {
    static __device__ __forceinline__ float ld(const bf16_t* p) { return bf2f(*p); }
    static __device__ __forceinline__ void st(bf16_t* p, float v) { *p = f2bf(v); }
    static __device__ __forceinline__ float cvt(float v) { return bf2f(f2bf(v)); }
};

// ---------------------------------------------------------------- MFMA
// D(16x16) += A(16x32) * B(32x16), bf16 in, fp32 accumulate.  Lane l holds
// A[l%16][8*(l/16) .. +7], B[8*(l/16) .. +7][l%16] and D[4*(l/16) .. +3][l%16].
__device__ __forceinline__ floatx4 mfma16x16x32(bf16x8 a, bf16x8 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D(32x32) += A(32x16) * B(16x32), bf16 in, fp32 accumulate.  Lane l holds
// A[l%32][8*(l/32) .. +7], B[8*(l/32) .. +7][l%32], and D[i][l%32] in element
// v for i = 8*(v/4) + 4*(l/32) + v%4.
typedef float floatx16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ floatx16 mfma32x32x16(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 ld_bf16x8(const bf16_t* p) {
    return *reinterpret_cast<const bf16x8*>(p);
}

// Element (m, k) of a fragment-major [rows][K] activation: the 16 x 64 block
// (m/16, k/64) sits at ((m/16) * K/64 + k/64) * 1024; inside it half
// h = (k/8) % 2 at +512h, lane l = m%16 + 16 * ((k%64)/16) at +8l, then k%8.
// Lane l of a wave then finds the B operand of mfma16x16x32 (token m%16,
// k = 16 * (l/16) + 8h + 0..7) at 8l of half h, as for the packed weights.
__device__ __forceinline__ size_t frag_off(int m, int k, int K) {
    const int kk = k & 63;
    return ((size_t)(m >> 4) * (K >> 6) + (k >> 6)) * 1024 + ((kk >> 3) & 1) * 512 +
           ((m & 15) + 16 * (kk >> 4)) * 8 + (kk & 7);
}

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// ---------------------------------------------------------------- DARD mask
// Does query row (stream, position i) read the ORIGINAL key x^j (true) or the
// shadow key s^j (false)?  Sec. 3.2: U queries read U tokens from x and the
// rest from s; C queries read U and the candidates at least as confident as
// themselves (Eq. 3) from x; the shadow query of any position never reads its
// own x key.  The x query of an M token reads the whole x block (or, with
// MKEYS_SHADOW, C, U and itself from x), its shadow query only U from x.
// Sec. 5.1 variants of the candidate order: C_BIDIR (every candidate),
// ORDER_L2R (the candidates j <= i).
__device__ __forceinline__ bool take_x(int si, int sj, float ci, float cj, int i, int j, bool shadow,
                                       uint32_t flags) {
    const bool self = i == j;
    if (si == DARD_STATE_U) {
        if (self && (shadow || (flags & DARD_F_XSELF_SHADOW))) return false;
        return sj == DARD_STATE_U;
    }
    if (si == DARD_STATE_C) {
        if (self && shadow) return false;
        const bool before = (flags & DARD_F_C_BIDIR) ? true : (flags & DARD_F_ORDER_L2R) ? j <= i : ci <= cj;
        return sj == DARD_STATE_U || (sj == DARD_STATE_C && before);
    }
    if (shadow) return sj == DARD_STATE_U;
    if (flags & DARD_F_MKEYS_SHADOW) return sj == DARD_STATE_C || sj == DARD_STATE_U || self;
    return true;
}

// The same rule for whole rows, one wave at a time: lane l holds positions l
// and l + 64 of the block (B <= 128), ballots give the U and C sets as bit
// masks, and a candidate row's set {j in C : c_i <= c_j} (Eq. 3) is one more
// ballot.  Every lane of the wave must call these with the same arguments.
struct BlockView {
    int s0, s1;        // states of positions lane, lane + 64 (-1 beyond B)
    float c0, c1;      // their confidences
    uint64_t U0, U1, C0, C1;
};

__device__ __forceinline__ BlockView load_block_view(const uint8_t* state, const float* conf, int B) {
    const int lane = threadIdx.x & 63;
    BlockView v;
    v.s0 = lane < B ? (int)state[lane] : -1;
    v.s1 = lane + 64 < B ? (int)state[lane + 64] : -1;
    v.c0 = lane < B ? conf[lane] : 0.f;
    v.c1 = lane + 64 < B ? conf[lane + 64] : 0.f;
    v.U0 = __ballot(v.s0 == DARD_STATE_U);
    v.U1 = __ballot(v.s1 == DARD_STATE_U);
    v.C0 = __ballot(v.s0 == DARD_STATE_C);
    v.C1 = __ballot(v.s1 == DARD_STATE_C);
    return v;
}

// "Take x" words (positions 0..63, 64..127) of query row r (x rows r < B,
// shadow rows r >= B); r must be the same on every lane.
__device__ __forceinline__ void row_take_x(const BlockView& v, int r, int B, uint32_t flags, uint64_t& x0,
                                           uint64_t& x1) {
    const int i = r % B;
    const bool shadow = r >= B;
    const int sa = __shfl(v.s0, i & 63, 64), sb = __shfl(v.s1, i & 63, 64);
    const float ca = __shfl(v.c0, i & 63, 64), cb = __shfl(v.c1, i & 63, 64);
    const int si = i < 64 ? sa : sb;
    const float ci = i < 64 ? ca : cb;
    const uint64_t self0 = i < 64 ? 1ull << i : 0ull, self1 = i < 64 ? 0ull : 1ull << (i - 64);
    const uint64_t all0 = B >= 64 ? ~0ull : (1ull << B) - 1;
    const uint64_t all1 = B >= 128 ? ~0ull : (B > 64 ? (1ull << (B - 64)) - 1 : 0ull);
    if (si == DARD_STATE_U) {
        x0 = v.U0; x1 = v.U1;
        if (shadow || (flags & DARD_F_XSELF_SHADOW)) { x0 &= ~self0; x1 &= ~self1; }
    } else if (si == DARD_STATE_C) {
        if (flags & DARD_F_C_BIDIR) {
            x0 = v.U0 | v.C0; x1 = v.U1 | v.C1;
        } else if (flags & DARD_F_ORDER_L2R) {
            // positions 0..i: words below i's word whole, i's word up to bit i
            const uint64_t upto0 = i < 64 ? (i == 63 ? ~0ull : (2ull << i) - 1) : ~0ull;
            const uint64_t upto1 = i < 64 ? 0ull : (i == 127 ? ~0ull : (2ull << (i - 64)) - 1);
            x0 = v.U0 | (v.C0 & upto0); x1 = v.U1 | (v.C1 & upto1);
        } else {
            x0 = v.U0 | __ballot(v.s0 == DARD_STATE_C && ci <= v.c0);
            x1 = v.U1 | __ballot(v.s1 == DARD_STATE_C && ci <= v.c1);
        }
        if (shadow) { x0 &= ~self0; x1 &= ~self1; }
    } else if (shadow) {
        x0 = v.U0; x1 = v.U1;
    } else if (flags & DARD_F_MKEYS_SHADOW) {
        x0 = v.U0 | v.C0 | self0; x1 = v.U1 | v.C1 | self1;
    } else {
        x0 = all0; x1 = all1;
    }
}

}  // namespace dard
