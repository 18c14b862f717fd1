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

__device__ __forceinline__ bf16x8 ld_bf16x8(const bf16_t* p) {
    return *reinterpret_cast<const bf16x8*>(p);
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
__device__ __forceinline__ bool take_x(int si, int sj, float ci, float cj, bool shadow,
                                       bool self, uint32_t flags) {
    if (si == DARD_STATE_U) {
        if (self && (shadow || (flags & DARD_F_XSELF_SHADOW))) return false;
        return sj == DARD_STATE_U;
    }
    if (si == DARD_STATE_C) {
        if (self && shadow) return false;
        return sj == DARD_STATE_U || (sj == DARD_STATE_C && ci <= cj);
    }
    if (shadow) return sj == DARD_STATE_U;
    if (flags & DARD_F_MKEYS_SHADOW) return sj == DARD_STATE_C || sj == DARD_STATE_U || self;
    return true;
}

}  // namespace dard
