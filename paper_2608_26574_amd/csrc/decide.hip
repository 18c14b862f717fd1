// Decision part of one DARD step (Algorithm 1): candidate verification, the
// promotion / demotion sets, the guidance weight of masked tokens (Eq. 5-6)
// and the three-state transition with token fill (Eq. 8).  One workgroup per
// sequence, one thread per block position.  Distance-weighted sums are formed
// in float64 in position order from a table of lambda^k.  In step mode the
// vocab-chunk partials of the confidence reduction are first copied to LDS
// in one coalesced pass and merged there in chunk order.
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
};

// Merge the chunk partials of one row in chunk order.
__device__ Red combine(const float* p, int nchunk) {
    Red t{p[0], __float_as_int(p[1]), p[2]};
    for (int c = 1; c < nchunk; ++c) {
        const float m2 = p[3 * c], s2 = p[3 * c + 2];
        const int a2 = __float_as_int(p[3 * c + 1]);
        const float mm = fmaxf(t.m, m2);
        const bool take = (m2 > t.m) || (m2 == t.m && a2 < t.a);
        const float s1 = t.m == -INFINITY ? 0.f : t.s * exp2f((t.m - mm) * kLog2e);
        const float s2s = m2 == -INFINITY ? 0.f : s2 * exp2f((m2 - mm) * kLog2e);
        t.a = take ? a2 : t.a;
        t.m = mm;
        t.s = s1 + s2s;
    }
    return t;
}

// Copy n floats from global to LDS with all of a thread's loads in flight.
__device__ void stage(float* dst, const float* src, int n) {
    constexpr int U = 8;
    for (int base = 0; base < n; base += U * 128) {
        float v[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int t = base + k * 128 + threadIdx.x;
            v[k] = t < n ? src[t] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int t = base + k * 128 + threadIdx.x;
            if (t < n) dst[t] = v[k];
        }
    }
}

struct PosConf {
    float maxprob, pcur;
    int argmax;
};

// Shadow-row confidence of position i: from staged chunk partials (step mode)
// or from the per-position arrays.
__device__ PosConf shadow_conf(const DecideArgs& a, const float* part, int s, int i, int tok) {
    PosConf r;
    const int pos = s * a.B + i;
    if (part) {
        const Red t = combine(part + (size_t)i * a.nchunk * 3, a.nchunk);
        r.maxprob = 1.f / t.s;
        r.argmax = t.a;
        tok = min(max(tok, 0), (int)a.ld - 1);   // stay inside the row whatever the id
        const float lc = a.logits[((size_t)s * 2 * a.B + a.B + i) * a.ld + tok];
        r.pcur = exp2f((lc - t.m) * kLog2e) / t.s;
    } else {
        r.maxprob = a.maxprob_s[pos];
        r.argmax = a.argmax_s ? a.argmax_s[pos] : 0;
        r.pcur = a.pcur_s ? a.pcur_s[pos] : 0.f;
    }
    return r;
}

__global__ __launch_bounds__(128) void decide_kernel(DecideArgs a) {
    extern __shared__ float staged[];            // [2][B][nchunk][3] in step mode
    __shared__ uint8_t promoted[128], demoted[128];
    __shared__ double lam_pow[128];
    __shared__ int all_u, entered_u;
    __shared__ float c_all[128];
    __shared__ int nxt_all[128], xhat_all[128];
    const int s = blockIdx.x, i = threadIdx.x;
    const bool live = i < a.B;
    const int pos = s * a.B + i;
    const int st = live ? a.state_in[pos] : DARD_STATE_U;
    const bool pcur_mode = (a.flags & DARD_F_VERIFY_PCUR) != 0;
    const int per_seq = a.B * a.nchunk * 3;
    float* sv = staged;
    float* sm = staged + per_seq;
    if (a.part_v) stage(sv, a.part_v + (size_t)s * per_seq, per_seq);
    if (a.part_m && a.phase == DARD_PHASE_FINAL) stage(sm, a.part_m + (size_t)s * per_seq, per_seq);

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
        if (st == DARD_STATE_M) {
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
    if (i == 0) { all_u = 1; entered_u = 0; }
    __syncthreads();
    if (live) {
        const int tok = a.tok_in ? a.tok_in[pos] : 0;
        float c;
        int xhat;
        float mp_s = 0.f, pc_s = 0.f, mp_mix = 0.f;
        int am_s = -1, am_mix = -1;
        if (st == DARD_STATE_M) {
            if (a.part_m) {
                const Red t = combine(sm + (size_t)i * a.nchunk * 3, a.nchunk);
                mp_mix = 1.f / t.s;
                am_mix = t.a;
            } else {
                mp_mix = a.maxprob_mix[pos];
                am_mix = a.argmax_mix[pos];
            }
            c = mp_mix;
            xhat = am_mix;
        } else {
            const float* part = a.part_m ? (st == DARD_STATE_C ? sv : sm) : nullptr;
            const PosConf pc = shadow_conf(a, part, s, i, tok);
            mp_s = pc.maxprob; pc_s = pc.pcur; am_s = pc.argmax;
            c = pcur_mode ? pc.pcur : pc.maxprob;
            xhat = pc.argmax;
        }
        const int nxt = transition(c, a.tau_c, a.tau_u);
        if (nxt != DARD_STATE_U) atomicAnd(&all_u, 0);
        if (nxt == DARD_STATE_U && st != DARD_STATE_U) atomicOr(&entered_u, 1);
        c_all[i] = c;
        nxt_all[i] = nxt;
        xhat_all[i] = xhat;
        a.state_out[pos] = (uint8_t)nxt;
        a.tok_out[pos] = nxt == DARD_STATE_M ? a.mask_id : xhat;
        a.conf_out[pos] = c;
        if (a.dbg_maxprob_s) a.dbg_maxprob_s[pos] = mp_s;
        if (a.dbg_argmax_s) a.dbg_argmax_s[pos] = am_s;
        if (a.dbg_pcur_s) a.dbg_pcur_s[pos] = pc_s;
        if (a.dbg_maxprob_mix) a.dbg_maxprob_mix[pos] = mp_mix;
        if (a.dbg_argmax_mix) a.dbg_argmax_mix[pos] = am_mix;
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
    if (i == 0 && a.block_done) a.block_done[s] = all_u;
}

}  // namespace

hipError_t launch_decide(const DecideArgs& a, hipStream_t s) {
    TraceScope ts(DARD_K_DECIDE, s);
    const size_t lds = (a.part_v || a.part_m) ? (size_t)2 * a.B * a.nchunk * 3 * sizeof(float) : 0;
    if (lds > 96 * 1024) return hipErrorInvalidValue;
    launch(decide_kernel, dim3(a.b), dim3(128), lds, s, a);
    return hipGetLastError();
}

}  // namespace dard
