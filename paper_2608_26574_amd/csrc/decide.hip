// Decision part of one DARD step (Algorithm 1): candidate verification, the
// promotion / demotion sets, the guidance weight of masked tokens (Eq. 5-6)
// and the three-state transition with token fill (Eq. 8).  One workgroup per
// sequence, one thread per block position.  Distance-weighted sums are formed
// in float64 in position order from a table of lambda^k.  In step mode the
// vocab-chunk partials of the confidence reduction are first copied to LDS
// in one coalesced pass and merged there in chunk order.
//
// Sec. 5.1 variants: with a fixed weight every M position takes w_fixed
// instead of Eq. 5-6; with the entropy or margin ordering the key carried to
// the next step's mask (conf_out) is -entropy or the margin of the row that
// gave the confidence, from the statistics partials (chunk stride 5).
#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ int transition(float c, float tau_c, float tau_u) {
    if (c <= tau_c) return DARD_STATE_M;
    if (c <= tau_u) return DARD_STATE_C;
    return DARD_STATE_U;
}

struct Red {
    float m;
    int a;
    float s;
    float t, m2;   // statistics partials only: sum e (l - max), second-largest l
};

// Merge the chunk partials of one row (stride K floats each) in chunk order.
__device__ Red combine(const float* p, int nchunk, int K) {
    const bool stats = K == kConfStatsStride;
    Red t{p[0], __float_as_int(p[1]), p[2], stats ? p[3] : 0.f, stats ? p[4] : -INFINITY};
    for (int c = 1; c < nchunk; ++c) {
        const float* q = p + (size_t)c * K;
        const float m2 = q[0], s2 = q[2];
        const int a2 = __float_as_int(q[1]);
        const float mm = fmaxf(t.m, m2);
        const bool take = (m2 > t.m) || (m2 == t.m && a2 < t.a);
        const float e1 = t.m == -INFINITY ? 0.f : exp2f((t.m - mm) * kLog2e);
        const float e2 = m2 == -INFINITY ? 0.f : exp2f((m2 - mm) * kLog2e);
        if (stats) {
            const float t1 = t.m == -INFINITY ? 0.f : e1 * (t.t + (t.m - mm) * t.s);
            const float t2 = m2 == -INFINITY ? 0.f : e2 * (q[3] + (m2 - mm) * s2);
            t.t = t1 + t2;
            t.m2 = fmaxf(fminf(t.m, m2), fmaxf(t.m2, q[4]));
        }
        t.a = take ? a2 : t.a;
        t.s = t.s * e1 + s2 * e2;
        t.m = mm;
    }
    return t;
}

__device__ __forceinline__ float red_entropy(const Red& t) { return logf(t.s) - t.t / t.s; }
__device__ __forceinline__ float red_margin(const Red& t) { return (1.f - expf(t.m2 - t.m)) / t.s; }

constexpr int kThreads = kMaxBlock;   // one thread per block position
constexpr size_t kStageBytes = 64 * 1024;   // chunk partials larger than this are read in place

// Copy n floats from global to LDS with all of a thread's loads in flight.
__device__ void stage(float* dst, const float* src, int n) {
    constexpr int U = 8;
    for (int base = 0; base < n; base += U * kThreads) {
        float v[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int t = base + k * kThreads + threadIdx.x;
            v[k] = t < n ? src[t] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int t = base + k * kThreads + threadIdx.x;
            if (t < n) dst[t] = v[k];
        }
    }
}

struct PosConf {
    float maxprob, pcur;
    int argmax;
    float entropy, margin, key;   // key: the caller's ordering key (array mode)
};

// Shadow-row confidence of position i: from staged chunk partials (step mode)
// or from the per-position arrays.
__device__ PosConf shadow_conf(const DecideArgs& a, const float* part, int s, int i, int tok) {
    PosConf r{0.f, 0.f, 0, 0.f, 0.f, 0.f};
    const int pos = s * a.B + i;
    if (part) {
        const Red t = combine(part + (size_t)i * a.nchunk * a.stride, a.nchunk, a.stride);
        r.maxprob = 1.f / t.s;
        r.argmax = t.a;
        tok = min(max(tok, 0), (int)a.ld - 1);   // stay inside the row whatever the id
        const float lc = a.logits[((size_t)s * 2 * a.B + a.B + i) * a.ld + tok];
        r.pcur = exp2f((lc - t.m) * kLog2e) / t.s;
        if (a.stride == kConfStatsStride) { r.entropy = red_entropy(t); r.margin = red_margin(t); }
    } else {
        r.maxprob = a.maxprob_s[pos];
        r.argmax = a.argmax_s ? a.argmax_s[pos] : 0;
        r.pcur = a.pcur_s ? a.pcur_s[pos] : 0.f;
        r.key = a.key_s ? a.key_s[pos] : 0.f;
    }
    return r;
}

// The key the next step's mask orders candidates by (Eq. 3 or its Sec. 5.1
// variants): the confidence, -entropy or the margin.
__device__ __forceinline__ float order_key(uint32_t flags, bool from_partials, float c, float entropy,
                                           float margin, float given) {
    if (!(flags & (DARD_F_ORDER_ENTROPY | DARD_F_ORDER_MARGIN))) return c;
    if (!from_partials) return given;
    return (flags & DARD_F_ORDER_ENTROPY) ? -entropy : margin;
}

__global__ __launch_bounds__(kThreads) void decide_kernel(DecideArgs a, int in_lds) {
    extern __shared__ float staged[];            // [2][B][nchunk][stride] in step mode (in_lds)
    __shared__ uint8_t promoted[kThreads], demoted[kThreads];
    __shared__ double lam_pow[kThreads];
    __shared__ int all_u, entered_u, bad_code;
    __shared__ float c_all[kThreads];
    __shared__ int nxt_all[kThreads], xhat_all[kThreads];
    const int s = blockIdx.x, i = threadIdx.x;
    const bool live = i < a.B;
    const int pos = s * a.B + i;
    const int st = live ? a.state_in[pos] : DARD_STATE_U;
    const bool pcur_mode = (a.flags & DARD_F_VERIFY_PCUR) != 0;
    const int per_seq = a.B * a.nchunk * a.stride;
    // the sequence's chunk partials: copied to LDS in one coalesced pass, or
    // (large blocks) read where they are
    const float* sv = a.part_v ? a.part_v + (size_t)s * per_seq : nullptr;
    const float* sm = a.part_m ? a.part_m + (size_t)s * per_seq : nullptr;
    if (in_lds) {
        if (a.part_v) stage(staged, sv, per_seq);
        if (a.part_m && a.phase == DARD_PHASE_FINAL) stage(staged + per_seq, sm, per_seq);
        sv = a.part_v ? staged : nullptr;
        sm = a.part_m ? staged + per_seq : nullptr;
    }

    if (a.phase == DARD_PHASE_VERIFY) {
        promoted[i] = 0;
        demoted[i] = 0;
        if (live) lam_pow[i] = pow(a.lambda, (double)i);
        __syncthreads();
        if (live && st == DARD_STATE_C) {
            const int tok = a.tok_in ? a.tok_in[pos] : 0;
            const PosConf pc = shadow_conf(a, a.part_v ? sv : nullptr, s, i, tok);
            const float c = pcur_mode ? pc.pcur : pc.maxprob;
            const int nxt = transition(c, a.tau_c, a.tau_u);
            promoted[i] = nxt == DARD_STATE_U;
            demoted[i] = nxt == DARD_STATE_M;
        }
        __syncthreads();
        if (!live) return;
        float w = 0.f;
        if (st == DARD_STATE_M && (a.flags & DARD_F_FIXED_W)) {
            w = a.w_fixed;
        } else if (st == DARD_STATE_M) {
            double P = 0.0, D = 0.0;
            for (int j = 0; j < a.B; ++j) {
                const double k = lam_pow[abs(i - j)];
                if (promoted[j]) P += k;
                if (demoted[j]) D += k;
            }
            w = (float)((P + a.p0) / (P + D + a.p0));
        }
        a.w_out[pos] = w;
        return;
    }

    // ---- FINAL: confidences of every position, transition, fill
    if (i == 0) { all_u = 1; entered_u = 0; bad_code = 0; }
    __syncthreads();
    if (live && st > DARD_STATE_U) atomicOr(&bad_code, 1);
    if (live) {
        const int tok = a.tok_in ? a.tok_in[pos] : 0;
        float c, key;
        int xhat;
        float mp_s = 0.f, pc_s = 0.f, mp_mix = 0.f, ent = 0.f, mrg = 0.f;
        int am_s = -1, am_mix = -1;
        const bool from_part = a.part_m != nullptr;
        if (st == DARD_STATE_M) {
            float given = 0.f;
            if (from_part) {
                const Red t = combine(sm + (size_t)i * a.nchunk * a.stride, a.nchunk, a.stride);
                mp_mix = 1.f / t.s;
                am_mix = t.a;
                if (a.stride == kConfStatsStride) { ent = red_entropy(t); mrg = red_margin(t); }
            } else {
                mp_mix = a.maxprob_mix[pos];
                am_mix = a.argmax_mix[pos];
                given = a.key_mix ? a.key_mix[pos] : 0.f;
            }
            c = mp_mix;
            xhat = am_mix;
            key = order_key(a.flags, from_part, c, ent, mrg, given);
        } else {
            const float* part = from_part ? (st == DARD_STATE_C ? sv : sm) : nullptr;
            const PosConf pc = shadow_conf(a, part, s, i, tok);
            mp_s = pc.maxprob; pc_s = pc.pcur; am_s = pc.argmax;
            ent = pc.entropy; mrg = pc.margin;
            c = pcur_mode ? pc.pcur : pc.maxprob;
            xhat = pc.argmax;
            key = order_key(a.flags, from_part, c, ent, mrg, pc.key);
        }
        const int nxt = transition(c, a.tau_c, a.tau_u);
        if (nxt != DARD_STATE_U) atomicAnd(&all_u, 0);
        if (nxt == DARD_STATE_U && st != DARD_STATE_U) atomicOr(&entered_u, 1);
        c_all[i] = c;
        nxt_all[i] = nxt;
        xhat_all[i] = xhat;
        a.state_out[pos] = (uint8_t)nxt;
        a.tok_out[pos] = nxt == DARD_STATE_M ? a.mask_id : xhat;
        a.conf_out[pos] = key;
        if (a.dbg_maxprob_s) a.dbg_maxprob_s[pos] = mp_s;
        if (a.dbg_argmax_s) a.dbg_argmax_s[pos] = am_s;
        if (a.dbg_pcur_s) a.dbg_pcur_s[pos] = pc_s;
        if (a.dbg_maxprob_mix) a.dbg_maxprob_mix[pos] = mp_mix;
        if (a.dbg_argmax_mix) a.dbg_argmax_mix[pos] = am_mix;
        if (a.dbg_entropy) a.dbg_entropy[pos] = ent;
        if (a.dbg_margin) a.dbg_margin[pos] = mrg;
    }
    __syncthreads();
    // progress rule (DARD_F_PROGRESS): no position entered U in an unfinished
    // block -> the most confident non-U position (lowest on ties) becomes U
    if (i == 0 && (a.flags & DARD_F_PROGRESS) && !entered_u && !all_u) {
        int best = -1;
        for (int j = 0; j < a.B; ++j)
            if (nxt_all[j] != DARD_STATE_U && (best < 0 || c_all[j] > c_all[best])) best = j;
        const int bp = s * a.B + best;
        a.state_out[bp] = (uint8_t)DARD_STATE_U;
        a.tok_out[bp] = xhat_all[best];
        int done = 1;
        for (int j = 0; j < a.B; ++j)
            if (j != best && nxt_all[j] != DARD_STATE_U) done = 0;
        all_u = done;
    }
    if (i == 0 && a.block_done)
        a.block_done[s] = ((a.flags & DARD_F_CHECK_STATES) && bad_code) ? DARD_BAD_STATE : all_u;
}

}  // namespace

hipError_t launch_decide(const DecideArgs& a, hipStream_t s) {
    TraceScope ts(DARD_K_DECIDE, s);
    if (a.B < 1 || a.B > kThreads) return hipErrorInvalidValue;
    size_t lds = (a.part_v || a.part_m) ? (size_t)2 * a.B * a.nchunk * a.stride * sizeof(float) : 0;
    const int in_lds = lds > 0 && lds <= kStageBytes;
    if (!in_lds) lds = 0;
    launch(decide_kernel, dim3(a.b), dim3(kThreads), lds, s, a, in_lds);
    return hipGetLastError();
}

}  // namespace dard
