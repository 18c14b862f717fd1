// Vocab-wide confidence reduction (Eq. 1) with optional logit mixing (Eq. 7).
//
// A row of V float32 logits is cut into chunks of 8192; one 256-thread
// workgroup reduces one chunk with 16-byte loads into a partial
// (max, first argmax, sum of exp(l - max)), so that even a single step's few
// rows fill the chip.  Partials are merged in chunk order, which keeps the
// result independent of scheduling.  Mixed rows are formed on the fly,
// (w * l_x) + ((1 - w) * l_s) with every operation rounded once in fp32.
//
// The statistics variant (entropy and margin orderings of Sec. 5.1) carries
// two more terms in the same pass: t = sum exp(l - max) (l - max), so that
// the entropy is ln(s) - t / s, and the second-largest logit m2, so that the
// margin p_(1) - p_(2) is (1 - exp(m2 - max)) / s.  Moving a partial to a
// larger maximum M scales s and t by e = exp(m - M) and adds (m - M) s e to t.
#include <mutex>

#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr int kChunk = kConfChunk;
constexpr float kLog2e = 1.4426950408889634f;

struct Acc {
    float m;
    int a;
    float s;
    float t, m2;   // statistics variant only
};

// Merge two partials; the larger maximum wins, ties go to the lower index.
template <bool STATS>
__device__ __forceinline__ Acc merge(Acc x, Acc y) {
    Acc r;
    const bool take_y = (y.m > x.m) || (y.m == x.m && y.a < x.a);
    r.a = take_y ? y.a : x.a;
    r.m = fmaxf(x.m, y.m);
    const float ex = x.m == -INFINITY ? 0.f : exp2f((x.m - r.m) * kLog2e);
    const float ey = y.m == -INFINITY ? 0.f : exp2f((y.m - r.m) * kLog2e);
    r.s = x.s * ex + y.s * ey;
    if (STATS) {
        const float tx = x.m == -INFINITY ? 0.f : ex * (x.t + (x.m - r.m) * x.s);
        const float ty = y.m == -INFINITY ? 0.f : ey * (y.t + (y.m - r.m) * y.s);
        r.t = tx + ty;
        r.m2 = fmaxf(fminf(x.m, y.m), fmaxf(x.m2, y.m2));
    } else {
        r.t = 0.f;
        r.m2 = -INFINITY;
    }
    return r;
}

// (w * x) + (omw * s) with both products and the sum rounded separately: no
// fused multiply-add may merge a product into the sum.
__device__ __forceinline__ float mixv(float x, float s, float w, float omw) {
#pragma clang fp contract(off)
    const float a = w * x;
    const float b = omw * s;
    return a + b;
}

template <bool STATS>
__global__ __launch_bounds__(256) void conf_partial_kernel(ConfArgs a, int step_B) {
    const int row = blockIdx.x, ch = blockIdx.y;
    const float* ls;
    const float* lx = nullptr;
    float w = 0.f;
    if (step_B > 0) {
        // rows are block positions; logits hold [b][2B][V] (x rows then s rows)
        const int st = a.state[row];
        if (a.phase == 0 ? st != DARD_STATE_C : st == DARD_STATE_C) return;
        if (a.phase == 1 && a.m_only && st != DARD_STATE_M) return;
        const int s = row / step_B, i = row % step_B;
        ls = a.ls + ((size_t)s * 2 * step_B + step_B + i) * a.ld_s;
        if (a.phase == 1 && st == DARD_STATE_M && !a.no_mix) {
            lx = a.ls + ((size_t)s * 2 * step_B + i) * a.ld_s;
            w = a.w[row];
        }
    } else {
        ls = a.ls + (size_t)row * a.ld_s;
        if (a.lx) {
            lx = a.lx + (size_t)row * a.ld_x;
            w = a.w[row];
        }
    }
    const float omw = __fsub_rn(1.f, w);
    const bool use_x = lx != nullptr && w != 0.f;
    const bool use_s = !(lx != nullptr && w == 1.f);

    const int begin = ch * kChunk;
    const int end = min(a.V, begin + kChunk);
    // every float4 of this thread is loaded (non-temporal: the logits are read
    // once) before any arithmetic
    constexpr int kIt = kChunk / (4 * 256);
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    f32x4 sv4[kIt], xv4[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const int i = begin + 4 * threadIdx.x + 4 * 256 * it;
        const bool full = i + 4 <= end;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        sv4[it] = (use_s && full) ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(ls + i)) : z;
        xv4[it] = (use_x && full) ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(lx + i)) : z;
    }
    // the (mixed) values, -inf past the end of the row
    float v[kIt][4];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const int i = begin + 4 * threadIdx.x + 4 * 256 * it;
        if (i + 4 <= end) {
            const f32x4 sv = sv4[it];
            if (use_x) {
                const f32x4 xv = xv4[it];
                if (use_s) {
                    v[it][0] = mixv(xv.x, sv.x, w, omw); v[it][1] = mixv(xv.y, sv.y, w, omw);
                    v[it][2] = mixv(xv.z, sv.z, w, omw); v[it][3] = mixv(xv.w, sv.w, w, omw);
                } else {
                    v[it][0] = xv.x; v[it][1] = xv.y; v[it][2] = xv.z; v[it][3] = xv.w;
                }
            } else {
                v[it][0] = sv.x; v[it][1] = sv.y; v[it][2] = sv.z; v[it][3] = sv.w;
            }
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if (i + k < end) {
                    const float svk = use_s ? ls[i + k] : 0.f;
                    v[it][k] = use_x ? (use_s ? mixv(lx[i + k], svk, w, omw) : lx[i + k]) : svk;
                } else {
                    v[it][k] = -INFINITY;
                }
            }
        }
    }
    // pass 1: the thread's maximum and its first index (indices increase with it, then k)
    Acc acc{-INFINITY, 0x7fffffff, 0.f, 0.f, -INFINITY};
#pragma unroll
    for (int it = 0; it < kIt; ++it)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (STATS) acc.m2 = fmaxf(acc.m2, fminf(acc.m, v[it][k]));
            if (v[it][k] > acc.m) { acc.m = v[it][k]; acc.a = begin + 4 * threadIdx.x + 4 * 256 * it + k; }
        }
    // pass 2: sum of exp(l - max); arguments are <= 0, so the hardware exp2
    // (v_exp_f32) needs no range handling, and exp2(-inf) = 0.  One fma per
    // element forms l log2(e) - mb with mb = max log2(e) rounded to fp32; the
    // rounding error r = max log2(e) - mb (exact through an fma) is common to
    // every term, so the sums are scaled by 2^-r once at the end.  Without that
    // step large logits (|l| ~ 100) would bias s by up to ~1e-5 relative.
    if (acc.m != -INFINITY) {
        const float mb = acc.m * kLog2e;
#pragma unroll
        for (int it = 0; it < kIt; ++it)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float e = __builtin_amdgcn_exp2f(fmaf(v[it][k], kLog2e, -mb));
                acc.s += e;
                // -inf past the end of the row: e = 0 and the clamp keeps 0 * d finite
                if (STATS) acc.t = fmaf(e, fmaxf(v[it][k] - acc.m, -3.0e38f), acc.t);
            }
        const float fix = exp2f(-fmaf(acc.m, kLog2e, -mb));
        acc.s *= fix;
        if (STATS) acc.t *= fix;
    }
    // wave reduction then across the 4 waves, fixed order
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        Acc y{__shfl_xor(acc.m, o, 64), __shfl_xor(acc.a, o, 64), __shfl_xor(acc.s, o, 64), 0.f, -INFINITY};
        if (STATS) { y.t = __shfl_xor(acc.t, o, 64); y.m2 = __shfl_xor(acc.m2, o, 64); }
        acc = merge<STATS>(acc, y);
    }
    __shared__ Acc red[4];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        Acc t = red[0];
        for (int k = 1; k < 4; ++k) t = merge<STATS>(t, red[k]);
        constexpr int kStride = STATS ? kConfStatsStride : kConfStride;
        float* p = a.part + ((size_t)row * a.nchunk + ch) * kStride;
        p[0] = t.m;
        p[1] = __int_as_float(t.a);
        p[2] = t.s;
        if (STATS) { p[3] = t.t; p[4] = t.m2; }
    }
}

template <bool STATS>
__global__ void conf_combine_kernel(const float* __restrict__ part, int rows, int nchunk, int V,
                                    const float* __restrict__ ls, int64_t ld, const int32_t* __restrict__ cur,
                                    int32_t* __restrict__ argmax, float* __restrict__ maxprob,
                                    float* __restrict__ pcur, float* __restrict__ entropy,
                                    float* __restrict__ margin) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    constexpr int K = STATS ? kConfStatsStride : kConfStride;
    const float* p = part + (size_t)r * nchunk * K;
    auto at = [&](int c) {
        const float* q = p + (size_t)c * K;
        return Acc{q[0], __float_as_int(q[1]), q[2], STATS ? q[3] : 0.f, STATS ? q[4] : -INFINITY};
    };
    Acc t = at(0);
    for (int c = 1; c < nchunk; ++c) t = merge<STATS>(t, at(c));
    argmax[r] = t.a;
    maxprob[r] = 1.f / t.s;
    if (pcur) {
        // token ids are device data: an id outside [0, V) reads the nearest
        // entry of the row instead of memory past it
        const int ct = min(max(cur[r], 0), V - 1);
        const float lc = ls[(size_t)r * ld + ct];
        pcur[r] = exp2f((lc - t.m) * kLog2e) / t.s;
    }
    if (STATS) {
        if (entropy) entropy[r] = logf(t.s) - t.t / t.s;
        if (margin) margin[r] = (1.f - expf(t.m2 - t.m)) / t.s;
    }
}

}  // namespace

// Chunk partials of dard_confidence_noalloc: a fixed array in device memory
// (each GPU holds its own copy for the life of the process).  Its device
// address comes from hipGetSymbolAddress, once per device; the host-side
// name `scratch` is not a device address and is never passed to a kernel.
constexpr size_t kScratchFloats = size_t(1) << 20;   // 4 MiB
static __device__ __align__(256) float scratch[kScratchFloats];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch[kMaxDevices];
}  // namespace

size_t conf_scratch_floats() { return kScratchFloats; }

hipError_t conf_scratch(float** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[dev] = static_cast<float*>(p);
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

int conf_chunks(int V) { return (V + kChunk - 1) / kChunk; }

hipError_t launch_conf_partial(const ConfArgs& a, bool stats, hipStream_t s) {
    TraceScope ts(DARD_K_CONFIDENCE, s);
    ConfArgs b = a;
    b.chunk = kChunk;
    b.nchunk = conf_chunks(a.V);
    const int step_B = a.step_B;
    if (stats)
        launch(conf_partial_kernel<true>, dim3(a.rows, b.nchunk), dim3(256), 0, s, b, step_B);
    else
        launch(conf_partial_kernel<false>, dim3(a.rows, b.nchunk), dim3(256), 0, s, b, step_B);
    return hipGetLastError();
}

hipError_t launch_conf_combine(const float* part, int rows, int nchunk, int V, const float* ls, int64_t ld,
                               const int32_t* cur_tok, int32_t* argmax, float* maxprob, float* pcur,
                               float* entropy, float* margin, hipStream_t s) {
    TraceScope ts(DARD_K_CONFIDENCE, s);
    const dim3 g((rows + 127) / 128), blk(128);
    if (entropy || margin)
        launch(conf_combine_kernel<true>, g, blk, 0, s, part, rows, nchunk, V, ls, ld, cur_tok, argmax, maxprob,
               pcur, entropy, margin);
    else
        launch(conf_combine_kernel<false>, g, blk, 0, s, part, rows, nchunk, V, ls, ld, cur_tok, argmax, maxprob,
               pcur, entropy, margin);
    return hipGetLastError();
}

}  // namespace dard
