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

// ---------------------------------------------------------------- FP8 (OCP E4M3)
// float -> E4M3 code (sign in bit 7): round to nearest, ties to the even code;
// magnitudes from 448 (the largest finite value) up, and non-finite inputs,
// give +-448.  Below 2^-6 the format steps by 2^-9 (subnormals).
__device__ __forceinline__ uint32_t f2e4m3(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7FFFFFFFu;
    uint32_t code;
    if (a >= 0x43E00000u) {                 // |f| >= 448
        code = 0x7Eu;
    } else if (a < 0x3C800000u) {           // |f| < 2^-6: multiples of 2^-9, 8 = the smallest normal
        code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
    } else {                                // keep 3 mantissa bits (ties to even on bit 20), rebias 127 -> 7
        const uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
        code = (r >> 20) - (120u << 3);
        code = code > 0x7Eu ? 0x7Eu : code;
    }
    return sign | code;
}

// Eight E4M3 codes (little-endian in w) -> eight bf16 values.  The hardware
// conversion gives the exact value in fp32; E4M3 values have at most 4
// significant bits and exponents within bf16's, so keeping the upper half of
// each fp32 is exact.
template <bool HI>   // HI: the codes in bits 16..31, else bits 0..15
__device__ __forceinline__ uint32_t e4m3x2_to_bf16x2(uint32_t x) {
    const auto f = __builtin_amdgcn_cvt_pk_f32_fp8((int)x, HI);
    return (__float_as_uint(f[0]) >> 16) | (__float_as_uint(f[1]) & 0xFFFF0000u);
}
__device__ __forceinline__ uint4 e4m3x8_to_bf16x8(uint2 w) {
    return make_uint4(e4m3x2_to_bf16x2<false>(w.x), e4m3x2_to_bf16x2<true>(w.x), e4m3x2_to_bf16x2<false>(w.y),
                      e4m3x2_to_bf16x2<true>(w.y));
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

// s_waitcnt immediate: at most n vector-memory operations outstanding, no LDS
// operation outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4 left at its maximum, lgkmcnt 11:8 zero).
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// Workgroup barrier that waits for nothing itself.  __syncthreads() also
// drains every outstanding vector-memory operation (its fence does), which
// would cancel copies issued ahead for later steps; callers of wg_barrier
// first wait (s_waitcnt) for exactly the operations it has to cover.  The
// empty asm statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void wg_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
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

// ---------------------------------------------------------------- softmax partials
// (max, first argmax, sum of exp(l - max)) of a run of logits (Eq. 1 needs the
// first two and the sum), and the merge of two runs: the larger maximum wins,
// ties go to the lower index, the sums are rescaled to the common maximum.
// Evaluated without contraction, so merge(x, y) == merge(y, x) bit for bit.
struct SmPart {
    float m;
    int a;
    float s;
};

__device__ __forceinline__ SmPart smpart_merge(SmPart x, SmPart y) {
#pragma clang fp contract(off)
    constexpr float kL2e = 1.4426950408889634f;
    SmPart r;
    const bool take_y = (y.m > x.m) || (y.m == x.m && y.a < x.a);
    r.a = take_y ? y.a : x.a;
    r.m = fmaxf(x.m, y.m);
    const float ex = x.m == -INFINITY ? 0.f : exp2f((x.m - r.m) * kL2e);
    const float ey = y.m == -INFINITY ? 0.f : exp2f((y.m - r.m) * kL2e);
    r.s = x.s * ex + y.s * ey;
    return r;
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

// The same rule for whole rows, one wave at a time: lane l holds positions
// l, l + 64, l + 128 and l + 192 of the block (B <= 256), ballots give the U
// and C sets as bit masks, and a candidate row's set {j in C : c_i <= c_j}
// (Eq. 3) is one more ballot per word.  Every lane of the wave must call
// these with the same arguments.
constexpr int kMaxBlock = 256;
constexpr int kBlockWords = kMaxBlock / 64;

struct BlockView {
    int st[kBlockWords];       // states of positions lane + 64 q (-1 beyond B)
    float c[kBlockWords];      // their confidences
    uint64_t U[kBlockWords], C[kBlockWords];
};

__device__ __forceinline__ BlockView load_block_view(const uint8_t* state, const float* conf, int B) {
    const int lane = threadIdx.x & 63;
    BlockView v;
#pragma unroll
    for (int q = 0; q < kBlockWords; ++q) {
        const int j = lane + 64 * q;
        v.st[q] = j < B ? (int)state[j] : -1;
        v.c[q] = j < B ? conf[j] : 0.f;
        v.U[q] = __ballot(v.st[q] == DARD_STATE_U);
        v.C[q] = __ballot(v.st[q] == DARD_STATE_C);
    }
    return v;
}

// Positions [0, B) as words: bit j of word q set for 64 q + j < B.
__device__ __forceinline__ uint64_t block_word_mask(int B, int q) {
    const int n = B - 64 * q;
    return n >= 64 ? ~0ull : (n > 0 ? (1ull << n) - 1 : 0ull);
}

// "Take x" words x[q] (positions 64 q .. 64 q + 63) of query row r (x rows
// r < B, shadow rows r >= B); r must be the same on every lane.
__device__ __forceinline__ void row_take_x(const BlockView& v, int r, int B, uint32_t flags,
                                           uint64_t (&x)[kBlockWords]) {
    const int i = r % B;
    const bool shadow = r >= B;
    const int qi = i >> 6, li = i & 63;
    int si = -1;
    float ci = 0.f;
#pragma unroll
    for (int q = 0; q < kBlockWords; ++q) {
        const int sq = __shfl(v.st[q], li, 64);
        const float cq = __shfl(v.c[q], li, 64);
        if (q == qi) { si = sq; ci = cq; }
    }
#pragma unroll
    for (int q = 0; q < kBlockWords; ++q) {
        const uint64_t self = q == qi ? 1ull << li : 0ull;
        uint64_t w;
        if (si == DARD_STATE_U) {
            w = v.U[q];
            if (shadow || (flags & DARD_F_XSELF_SHADOW)) w &= ~self;
        } else if (si == DARD_STATE_C) {
            uint64_t cw;
            if (flags & DARD_F_C_BIDIR) {
                cw = v.C[q];
            } else if (flags & DARD_F_ORDER_L2R) {
                // candidates at positions 0..i
                const uint64_t upto = q < qi ? ~0ull : (q == qi ? (li == 63 ? ~0ull : (2ull << li) - 1) : 0ull);
                cw = v.C[q] & upto;
            } else {
                cw = __ballot(v.st[q] == DARD_STATE_C && ci <= v.c[q]);
            }
            w = v.U[q] | cw;
            if (shadow) w &= ~self;
        } else if (shadow) {
            w = v.U[q];
        } else if (flags & DARD_F_MKEYS_SHADOW) {
            w = v.U[q] | v.C[q] | self;
        } else {
            w = block_word_mask(B, q);
        }
        x[q] = w;
    }
}

}  // namespace dard
