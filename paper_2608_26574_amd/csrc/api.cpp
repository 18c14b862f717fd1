// C ABI of libdard (include/dard.h): argument validation, the packed weight
// image, workspace layout and the stream-ordered orchestration of a DARD step
// and of the prefix prefill.  No entry point synchronises the stream except
// dard_pack_weights (a one-off) and dard_trace_read.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dard.h"
#include "launch.h"

namespace dard {

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define HIPOK(expr)                                                                        \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess) return fail(DARD_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t esize(int dtype) { return dtype == DARD_DTYPE_BF16 ? 2 : 4; }
// bytes per value of the KV cache
size_t kv_esize(const dard_dims* d) { return d->kv_format == DARD_KV_FP8 ? 1 : esize(d->dtype); }

int check_dims(const dard_dims* d) {
    if (!d) return fail(DARD_ERR_ARG, "dims is NULL");
    if (d->dtype != DARD_DTYPE_F32 && d->dtype != DARD_DTYPE_BF16)
        return fail(DARD_ERR_ARG, "unknown dtype %d", d->dtype);
    if (d->n_layers < 0 || d->d_model <= 0 || d->n_heads <= 0 || d->n_kv_heads <= 0 || d->ffn_dim <= 0 ||
        d->vocab <= 1 || d->max_pos <= 0)
        return fail(DARD_ERR_SHAPE, "non-positive model dimension");
    if (d->head_dim != 64 && d->head_dim != 128) return fail(DARD_ERR_SHAPE, "head_dim must be 64 or 128");
    if (d->n_heads % d->n_kv_heads) return fail(DARD_ERR_SHAPE, "n_heads %% n_kv_heads != 0");
    if (d->n_heads * d->head_dim != d->d_model) return fail(DARD_ERR_SHAPE, "d_model != n_heads * head_dim");
    if (d->dtype == DARD_DTYPE_BF16 && (d->d_model % 64 || d->ffn_dim % 64 || d->vocab % 16))
        return fail(DARD_ERR_SHAPE, "bf16 needs d_model, ffn_dim %% 64 == 0 and vocab %% 16 == 0");
    if (d->d_model > 8192) return fail(DARD_ERR_SHAPE, "d_model must be <= 8192");
    if (d->dtype == DARD_DTYPE_BF16) {
        // the pipelined GEMM (65-255 rows) addresses a weight matrix through a
        // buffer descriptor: 32-bit byte offsets, so every matrix stays under 4 GiB
        const size_t D = d->d_model, F = d->ffn_dim, V = d->vocab;
        const size_t qkv = (size_t)(d->n_heads + 2 * d->n_kv_heads) * d->head_dim;
        size_t most = V * D;
        most = 2 * F * D > most ? 2 * F * D : most;
        most = qkv * D > most ? qkv * D : most;
        if (most * 2 > 0xFFFFFFFFull)
            return fail(DARD_ERR_SHAPE, "bf16 weight matrices must be under 4 GiB (largest: %zu bytes)", most * 2);
    }
    if (d->dtype == DARD_DTYPE_F32 && (d->d_model % 4 || d->ffn_dim % 4 || d->vocab % 4))
        return fail(DARD_ERR_SHAPE, "f32 needs d_model, ffn_dim, vocab %% 4 == 0");
    if (!(d->norm_eps >= 0.f) || !(d->rope_theta > 0.f)) return fail(DARD_ERR_ARG, "bad norm_eps / rope_theta");
    if (d->kv_format != DARD_KV_DTYPE && d->kv_format != DARD_KV_FP8)
        return fail(DARD_ERR_ARG, "unknown kv_format %d", d->kv_format);
    if (d->kv_format == DARD_KV_FP8 && d->dtype != DARD_DTYPE_BF16)
        return fail(DARD_ERR_UNSUPPORTED, "the FP8 KV cache is a bf16-model format");
    return DARD_OK;
}

// Byte offsets of the packed weight image.
struct Layout {
    size_t embed, lm_head, final_norm, rope, layer0, layer_stride;
    size_t attn_norm, wqkv, wo, ffn_norm, wgu, wdown;   // relative to the layer
    size_t total;
};

Layout layout_of(const dard_dims* d) {
    const size_t es = esize(d->dtype);
    const size_t D = d->d_model, F = d->ffn_dim, V = d->vocab;
    const size_t qd = (size_t)d->n_heads * d->head_dim, kd = (size_t)d->n_kv_heads * d->head_dim;
    Layout L{};
    size_t o = 0;
    L.embed = o; o = align256(o + V * D * es);
    L.lm_head = o; o = align256(o + V * D * es);
    L.final_norm = o; o = align256(o + D * es);
    L.rope = o; o = align256(o + (size_t)d->max_pos * (d->head_dim / 2) * 2 * sizeof(float));
    L.layer0 = o;
    size_t l = 0;
    L.attn_norm = l; l = align256(l + D * es);
    L.wqkv = l; l = align256(l + (qd + 2 * kd) * D * es);
    L.wo = l; l = align256(l + D * qd * es);
    L.ffn_norm = l; l = align256(l + D * es);
    L.wgu = l; l = align256(l + 2 * F * D * es);
    L.wdown = l; l = align256(l + D * F * es);
    L.layer_stride = l;
    L.total = o + l * d->n_layers;
    return L;
}

// Workspace of dard_step / dard_prefill.
struct WsLayout {
    size_t h, xn, q, attn, act, sel, part, part_ml, part_slots, gpart, logits, cpart_v, cpart_m, w, ids, tok;
    size_t hx, rowmap, lmcount, lpart;   // the LM head on listed rows (lmhead.hip)
    size_t total;
};

WsLayout ws_layout(const dard_dims* d, int b, int B, int cap) {
    const size_t es = esize(d->dtype);
    size_t rows = (size_t)b * (2 * B > cap ? 2 * B : cap);
    rows = (rows + 63) / 64 * 64;   // fragment-major activations hold whole 16-row blocks, 64 at least
    const size_t qd = (size_t)d->n_heads * d->head_dim;
    const size_t step_rows = (size_t)b * 2 * B;
    const size_t nch = conf_chunks(d->vocab);
    WsLayout W{};
    size_t o = 0;
    W.h = o; o = align256(o + rows * d->d_model * 4);
    W.xn = o; o = align256(o + rows * d->d_model * es);
    W.q = o; o = align256(o + rows * qd * es);
    W.attn = o; o = align256(o + rows * qd * es);
    W.act = o; o = align256(o + rows * d->ffn_dim * es);
    W.sel = o; o = align256(o + step_rows * ((B + 63) / 64) * 8);   // state mask of the step
    // split-key attention partials: room for the largest split a step picks at
    // any prefix length the cache holds (0 .. cap - 2B keys); a prefill splits
    // only as far as this room allows
    W.part_slots = 0;
    const int max_tiles = attention_tiles(1, cap - 2 * B > 0 ? cap - 2 * B : 0, B, cap);
    for (int t = 1; t <= max_tiles; ++t) {
        const size_t sl = attention_partial_slots(d->dtype, b, 2 * B, d->n_heads, d->n_kv_heads, t);
        W.part_slots = sl > W.part_slots ? sl : W.part_slots;
    }
    W.part = o; o = align256(o + W.part_slots * d->head_dim * 4);
    W.part_ml = o; o = align256(o + W.part_slots * 2 * 4);
    W.logits = o; o = align256(o + step_rows * d->vocab * 4);
    W.cpart_v = o; o = align256(o + (size_t)b * B * nch * kConfStatsStride * 4);
    W.cpart_m = o; o = align256(o + (size_t)b * B * nch * kConfStatsStride * 4);
    W.w = o; o = align256(o + (size_t)b * B * 4);
    W.ids = o; o = align256(o + rows * 4);          // full-sequence mode: row token ids
    W.tok = o; o = align256(o + (size_t)b * B * 4);   // and the current block's tokens
    // split-K partials of the O and down projections: up to 8 splits of 64
    // rows (streaming GEMM) or 4 splits of all rows (pipelined and large-tile GEMMs)
    const size_t prow = rows * 4 > 8 * 64 ? rows * 4 : 8 * 64;
    W.gpart = o; o = align256(o + prow * d->d_model * 4);
    // listed LM-head rows: the compact input (whole 64-row blocks), two row
    // lists, their device counts, and the fused column-tile partials (tiles of
    // 128 columns or more)
    const size_t lrows = (step_rows + 63) / 64 * 64;
    W.hx = o; o = align256(o + lrows * d->d_model * es);
    W.rowmap = o; o = align256(o + 2 * step_rows * 4);
    W.lmcount = o; o = align256(o + 4 * 4);
    W.lpart = o; o = align256(o + step_rows * (((size_t)d->vocab + 127) / 128) * 3 * 4);
    W.total = o;
    return W;
}

int check_flags(uint32_t flags) {
    if (flags & ~DARD_F_ALL) return fail(DARD_ERR_ARG, "unknown flag bits 0x%x", flags);
    const uint32_t o = flags & DARD_F_ORDERS;
    if (o & (o - 1)) return fail(DARD_ERR_ARG, "more than one candidate-ordering flag (0x%x)", o);
    return DARD_OK;
}

int check_params(const dard_params* p) {
    if (!p) return fail(DARD_ERR_ARG, "params is NULL");
    if (!(p->tau_c >= 0.f) || !(p->tau_c <= p->tau_u) || !(p->tau_u <= 1.f))
        return fail(DARD_ERR_ARG, "need 0 <= tau_c <= tau_u <= 1");
    if (!(p->lambda > 0.0) || !(p->lambda < 1.0)) return fail(DARD_ERR_ARG, "need 0 < lambda < 1");
    if (!(p->p0 > 0.0)) return fail(DARD_ERR_ARG, "need p0 > 0");
    if (int rc = check_flags(p->flags)) return rc;
    if ((p->flags & DARD_F_FIXED_W) && !(p->w_fixed >= 0.f && p->w_fixed <= 1.f))
        return fail(DARD_ERR_ARG, "need 0 <= w_fixed <= 1");
    return DARD_OK;
}

// Entropy or margin ordering: the confidence pass also forms their terms.
bool needs_stats(uint32_t flags) { return (flags & (DARD_F_ORDER_ENTROPY | DARD_F_ORDER_MARGIN)) != 0; }

// ---------------------------------------------------------------- tracing
struct TraceRec {
    hipEvent_t a, b;
};
std::mutex g_trace_mu;
uint32_t g_trace_mask = 0;
std::vector<TraceRec> g_trace[DARD_K_COUNT];
int g_trace_period = 1;               // every period-th launch of a traced class is timed
long long g_trace_seen[DARD_K_COUNT];

}  // namespace

thread_local TraceScope* g_scope = nullptr;

TraceScope::TraceScope(int kernel_class, hipStream_t)
    : cls(kernel_class), on((g_trace_mask >> kernel_class) & 1u), prev(g_scope) {
    g_scope = this;
}

TraceScope::~TraceScope() { g_scope = prev; }

bool TraceScope::next_events(hipEvent_t* a, hipEvent_t* b) {
    const TraceScope* t = g_scope;
    if (!t || !t->on) return false;
    {
        std::lock_guard<std::mutex> lk(g_trace_mu);
        if (g_trace_seen[t->cls]++ % g_trace_period != 0) return false;
    }
    if (hipEventCreate(a) != hipSuccess) return false;
    if (hipEventCreate(b) != hipSuccess) {
        hipEventDestroy(*a);
        return false;
    }
    std::lock_guard<std::mutex> lk(g_trace_mu);
    g_trace[t->cls].push_back({*a, *b});
    return true;
}

}  // namespace dard

using namespace dard;

extern "C" {

const char* dard_last_error(void) { return g_err.c_str(); }
int dard_version(void) { return 1; }

// ---------------------------------------------------------------- state codes
dard_status dard_check_states(const uint8_t* state, int n, int32_t* status, void* stream) {
    if (!state || !status) return fail(DARD_ERR_ARG, "NULL pointer");
    if (n < 1) return fail(DARD_ERR_SHAPE, "need n >= 1");
    HIPOK(launch_check_states(state, n, status, (hipStream_t)stream));
    return DARD_OK;
}

// ---------------------------------------------------------------- mask
dard_status dard_build_state_mask(const uint8_t* state, const float* conf, int b, int B, uint32_t flags,
                                  uint64_t* sel, void* stream) {
    if (!state || !conf || !sel) return fail(DARD_ERR_ARG, "NULL pointer");
    if (b < 1 || B < 1 || B > 256) return fail(DARD_ERR_SHAPE, "need b >= 1 and 1 <= B <= 256");
    if (int rc = check_flags(flags)) return rc;
    HIPOK(launch_build_state_mask(state, conf, b, B, flags, sel, (hipStream_t)stream));
    return DARD_OK;
}

// ---------------------------------------------------------------- attention
namespace {

// Workspace of dard_masked_attention: the state mask of the block, then the
// partial results of a key split (room for the largest split over every
// KV-head count that divides Hq).
struct AttnWs {
    size_t mask, part, part_ml, part_slots, total;
};

AttnWs attn_ws(int dtype, int b, int B, int Hq, int dh, int P) {
    AttnWs w{};
    size_t slots = 0;
    for (int hkv = 1; hkv <= Hq; ++hkv) {
        if (Hq % hkv) continue;
        const size_t sl = attention_partial_slots(dtype, b, 2 * B, Hq, hkv, attention_tiles(1, P, B, P + 2 * B));
        slots = sl > slots ? sl : slots;
    }
    size_t o = 0;
    w.mask = o; o = align256(o + (size_t)b * 2 * B * ((B + 63) / 64) * 8);
    w.part = o; w.part_slots = slots; o = align256(o + slots * dh * 4);
    w.part_ml = o; o = align256(o + slots * 8);
    w.total = o;
    return w;
}

}  // namespace

size_t dard_attention_workspace_bytes(int dtype, int b, int B, int Hq, int dh, int P) {
    if (b < 1 || B < 1 || B > 256 || Hq < 1 || P < 0 || (dh != 64 && dh != 128)) return 0;
    if (dtype != DARD_DTYPE_BF16 && dtype != DARD_DTYPE_BF16_KV_FP8) return 0;
    return attn_ws(DARD_DTYPE_BF16, b, B, Hq, dh, P).total;
}

dard_status dard_masked_attention(int dtype, const void* q, const void* k, const void* v, int P, int cap,
                                  const uint8_t* state, const float* conf, int b, int B, int Hq, int Hkv, int dh,
                                  float scale, uint32_t flags, void* out, void* ws, size_t ws_bytes,
                                  void* stream) {
    if (!q || !k || !v || !state || !conf || !out) return fail(DARD_ERR_ARG, "NULL pointer");
    if (dtype != DARD_DTYPE_F32 && dtype != DARD_DTYPE_BF16 && dtype != DARD_DTYPE_BF16_KV_FP8)
        return fail(DARD_ERR_ARG, "unknown dtype");
    const bool kv8 = dtype == DARD_DTYPE_BF16_KV_FP8;
    if (kv8) dtype = DARD_DTYPE_BF16;
    if (int rc = check_flags(flags)) return rc;
    if (b < 1 || B < 1 || B > 256 || P < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv || P + 2 * B > cap)
        return fail(DARD_ERR_SHAPE, "bad attention shape (b=%d B=%d P=%d cap=%d Hq=%d Hkv=%d)", b, B, P, cap, Hq, Hkv);
    if (dh != 64 && dh != 128) return fail(DARD_ERR_SHAPE, "dh must be 64 or 128");
    const size_t need = dard_attention_workspace_bytes(dtype, b, B, Hq, dh, P);
    if (need && (!ws || ws_bytes < need)) return fail(DARD_ERR_WORKSPACE, "workspace needs %zu bytes", need);
    AttnArgs a{};
    a.q = q; a.k = k; a.v = v; a.out = out; a.state = state; a.conf = conf;
    a.b = b; a.R = 2 * B; a.Hq = Hq; a.Hkv = Hkv; a.dh = dh; a.cap = cap;
    a.P = P; a.B = B; a.nkeys = P + 2 * B; a.masked = 1; a.scale = scale; a.flags = flags;
    a.kv_fp8 = kv8;
    hipStream_t s = (hipStream_t)stream;
    TraceScope ts(DARD_K_ATTENTION, s);
    if (dtype == DARD_DTYPE_BF16) {
        const AttnWs w = attn_ws(dtype, b, B, Hq, dh, P);
        char* base = (char*)ws;
        a.sel = (const uint64_t*)(base + w.mask);
        a.part = (float*)(base + w.part);
        a.part_ml = (float*)(base + w.part_ml);
        a.part_slots = w.part_slots;
        TraceScope tm(DARD_K_MASK, s);
        HIPOK(launch_build_state_mask(state, conf, b, B, flags, (uint64_t*)(base + w.mask), s));
    }
    HIPOK(launch_attention(dtype, a, s));
    return DARD_OK;
}

// ---------------------------------------------------------------- confidence
size_t dard_confidence_workspace_bytes(int rows, int V) {
    if (rows < 1 || V < 1) return 0;
    return align256((size_t)rows * conf_chunks(V) * kConfStatsStride * 4);
}

namespace {

int check_confidence_args(const float* logits_s, const float* logits_x, const float* w, const int32_t* cur_tok,
                          int rows, int V, int64_t ld, const int32_t* argmax, const float* maxprob,
                          const float* pcur) {
    if (!logits_s || !argmax || !maxprob) return fail(DARD_ERR_ARG, "NULL pointer");
    if (logits_x && !w) return fail(DARD_ERR_ARG, "mixing needs w");
    if (pcur && (!cur_tok || logits_x)) return fail(DARD_ERR_ARG, "pcur needs cur_tok and no mixing");
    if (rows < 1 || V < 1 || ld < V || ld % 4) return fail(DARD_ERR_SHAPE, "need rows, V >= 1, ld >= V, ld %% 4 == 0");
    return DARD_OK;
}

// The two kernels of the confidence reduction with chunk partials at `part`.
int run_confidence(float* part, const float* logits_s, const float* logits_x, const float* w,
                   const int32_t* cur_tok, int rows, int V, int64_t ld, int32_t* argmax, float* maxprob, float* pcur,
                   float* entropy, float* margin, hipStream_t s) {
    ConfArgs a{};
    a.ls = logits_s; a.lx = logits_x; a.w = w; a.ld_s = ld; a.ld_x = ld;
    a.rows = rows; a.V = V; a.part = part; a.state = nullptr; a.phase = 0; a.step_B = 0;
    HIPOK(launch_conf_partial(a, entropy || margin, s));
    HIPOK(launch_conf_combine(part, rows, conf_chunks(V), V, logits_s, ld, cur_tok, argmax, maxprob, pcur, entropy,
                              margin, s));
    return DARD_OK;
}

}  // namespace

dard_status dard_confidence(const float* logits_s, const float* logits_x, const float* w, const int32_t* cur_tok,
                            int rows, int V, int64_t ld, int32_t* argmax, float* maxprob, float* pcur,
                            float* entropy, float* margin, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_confidence_args(logits_s, logits_x, w, cur_tok, rows, V, ld, argmax, maxprob, pcur)) return rc;
    const size_t need = dard_confidence_workspace_bytes(rows, V);
    if (!ws || ws_bytes < need) return fail(DARD_ERR_WORKSPACE, "workspace needs %zu bytes", need);
    return run_confidence((float*)ws, logits_s, logits_x, w, cur_tok, rows, V, ld, argmax, maxprob, pcur, entropy,
                          margin, (hipStream_t)stream);
}

dard_status dard_confidence_noalloc(const float* logits_s, const float* logits_x, const float* w,
                                    const int32_t* cur_tok, int rows, int V, int64_t ld, int32_t* argmax,
                                    float* maxprob, float* pcur, float* entropy, float* margin, void* stream) {
    if (int rc = check_confidence_args(logits_s, logits_x, w, cur_tok, rows, V, ld, argmax, maxprob, pcur)) return rc;
    const size_t stride = (entropy || margin) ? kConfStatsStride : kConfStride;
    const size_t need = (size_t)rows * conf_chunks(V) * stride;
    if (need > conf_scratch_floats())
        return fail(DARD_ERR_SHAPE, "rows x ceil(V / 8192) x %zu = %zu partial floats exceed the %zu of the "
                    "preallocated scratch", stride, need, conf_scratch_floats());
    float* part = nullptr;
    HIPOK(conf_scratch(&part));
    return run_confidence(part, logits_s, logits_x, w, cur_tok, rows, V, ld, argmax, maxprob, pcur, entropy, margin,
                          (hipStream_t)stream);
}

// ---------------------------------------------------------------- decisions
dard_status dard_commit_remask(int phase, const dard_params* params, int b, int B, const uint8_t* state_in,
                               const float* maxprob_s, const float* pcur_s, const int32_t* argmax_s,
                               const float* maxprob_mix, const int32_t* argmax_mix, const float* key_s,
                               const float* key_mix, float* w_out, uint8_t* state_out, int32_t* tok_out,
                               float* conf_out, int32_t* block_done, void* stream) {
    int rc = check_params(params);
    if (rc) return rc;
    if (b < 1 || B < 1 || B > 256) return fail(DARD_ERR_SHAPE, "need b >= 1 and 1 <= B <= 256");
    const bool pcur_mode = params->flags & DARD_F_VERIFY_PCUR;
    if (!state_in) return fail(DARD_ERR_ARG, "NULL state_in");
    if (phase == DARD_PHASE_VERIFY) {
        if (!w_out || (pcur_mode ? !pcur_s : !maxprob_s)) return fail(DARD_ERR_ARG, "VERIFY needs w_out and c");
    } else if (phase == DARD_PHASE_FINAL) {
        if (!maxprob_s || !argmax_s || !maxprob_mix || !argmax_mix || !state_out || !tok_out || !conf_out ||
            (pcur_mode && !pcur_s))
            return fail(DARD_ERR_ARG, "FINAL needs confidences, predictions and outputs");
        if ((params->flags & DARD_F_CHECK_STATES) && !block_done)
            return fail(DARD_ERR_ARG, "DARD_F_CHECK_STATES reports through block_done");
        if (needs_stats(params->flags) && (!key_s || !key_mix))
            return fail(DARD_ERR_ARG, "entropy / margin ordering needs key_s and key_mix");
    } else {
        return fail(DARD_ERR_ARG, "unknown phase %d", phase);
    }
    DecideArgs a{};
    a.phase = phase; a.b = b; a.B = B;
    a.tau_c = params->tau_c; a.tau_u = params->tau_u; a.lambda = params->lambda; a.p0 = params->p0;
    a.mask_id = params->mask_id; a.flags = params->flags; a.w_fixed = params->w_fixed;
    a.state_in = state_in;
    a.maxprob_s = maxprob_s; a.pcur_s = pcur_s; a.argmax_s = argmax_s;
    a.maxprob_mix = maxprob_mix; a.argmax_mix = argmax_mix;
    a.key_s = key_s; a.key_mix = key_mix; a.stride = kConfStride;
    a.w_out = w_out; a.state_out = state_out; a.tok_out = tok_out; a.conf_out = conf_out;
    a.block_done = block_done;
    HIPOK(launch_decide(a, (hipStream_t)stream));
    return DARD_OK;
}

// ---------------------------------------------------------------- weights / KV
size_t dard_packed_weight_bytes(const dard_dims* dims) {
    if (check_dims(dims)) return 0;
    return layout_of(dims).total;
}

size_t dard_kv_bytes(const dard_dims* d, int b, int cap) {
    if (check_dims(d) || b < 1 || cap < 1) return 0;
    return (size_t)d->n_layers * 2 * b * d->n_kv_heads * cap * d->head_dim * kv_esize(d);
}

dard_status dard_pack_weights(const dard_dims* d, const void* const* src, int n_src, void* packed,
                              size_t packed_bytes, void* stream) {
    int rc = check_dims(d);
    if (rc) return rc;
    if (!src || !packed) return fail(DARD_ERR_ARG, "NULL pointer");
    if (n_src != 3 + 9 * d->n_layers) return fail(DARD_ERR_ARG, "expected %d weight pointers", 3 + 9 * d->n_layers);
    for (int i = 0; i < n_src; ++i)
        if (!src[i]) return fail(DARD_ERR_ARG, "weight pointer %d is NULL", i);
    const Layout L = layout_of(d);
    if (packed_bytes < L.total) return fail(DARD_ERR_WORKSPACE, "packed image needs %zu bytes", L.total);
    hipStream_t s = (hipStream_t)stream;
    const size_t es = esize(d->dtype);
    const int D = d->d_model, F = d->ffn_dim, V = d->vocab, dh = d->head_dim;
    const int qd = d->n_heads * dh, kd = d->n_kv_heads * dh;
    char* P = (char*)packed;
    const int rowD = (int)(D * es), rowF = (int)(F * es);
    if (rowD % 16 || rowF % 16) return fail(DARD_ERR_SHAPE, "weight rows must be multiples of 16 bytes");
    HIPOK(launch_pack_rows(src[0], nullptr, P + L.embed, V, rowD, 0, dh, s));
    const bool frag = d->dtype == DARD_DTYPE_BF16;
    // projection matrices: bf16 fragment-major, fp32 row-major (same row order)
    auto pack = [&](const void* a, const void* b2, char* dst, int N, int K, int mode) -> hipError_t {
        return frag ? launch_pack_frag(a, b2, dst, N, K, mode, dh, s)
                    : launch_pack_rows(a, b2, dst, N, (int)(K * es), mode, dh, s);
    };
    for (int l = 0; l < d->n_layers; ++l) {
        const void* const* w = src + 1 + 9 * l;
        char* base = P + L.layer0 + L.layer_stride * l;
        HIPOK(launch_copy_rows(w[0], base + L.attn_norm, D * es, s));
        HIPOK(pack(w[1], nullptr, base + L.wqkv, qd, D, 1));
        HIPOK(pack(w[2], nullptr, base + L.wqkv + (size_t)qd * rowD, kd, D, 1));
        HIPOK(pack(w[3], nullptr, base + L.wqkv + (size_t)(qd + kd) * rowD, kd, D, 0));
        HIPOK(pack(w[4], nullptr, base + L.wo, D, qd, 0));
        HIPOK(launch_copy_rows(w[5], base + L.ffn_norm, D * es, s));
        HIPOK(pack(w[6], w[7], base + L.wgu, 2 * F, D, 2));
        HIPOK(pack(w[8], nullptr, base + L.wdown, D, F, 0));
    }
    HIPOK(launch_copy_rows(src[1 + 9 * d->n_layers], P + L.final_norm, D * es, s));
    HIPOK(pack(src[2 + 9 * d->n_layers], nullptr, P + L.lm_head, V, D, 0));
    // small norm vectors may not be a multiple of 16 bytes: copy the tail
    if ((D * es) % 16) {
        const size_t tail = (D * es) % 16, off = D * es - tail;
        for (int l = 0; l < d->n_layers; ++l) {
            const void* const* w = src + 1 + 9 * l;
            char* base = P + L.layer0 + L.layer_stride * l;
            HIPOK(hipMemcpyAsync(base + L.attn_norm + off, (const char*)w[0] + off, tail, hipMemcpyDeviceToDevice, s));
            HIPOK(hipMemcpyAsync(base + L.ffn_norm + off, (const char*)w[5] + off, tail, hipMemcpyDeviceToDevice, s));
        }
        HIPOK(hipMemcpyAsync(P + L.final_norm + off, (const char*)src[1 + 9 * d->n_layers] + off, tail,
                             hipMemcpyDeviceToDevice, s));
    }
    // rotary table: cos / sin of pos * theta^(-2t/dh), built in double precision
    std::vector<float> rope((size_t)d->max_pos * (dh / 2) * 2);
    for (int pos = 0; pos < d->max_pos; ++pos)
        for (int t = 0; t < dh / 2; ++t) {
            const double ang = (double)pos * std::pow((double)d->rope_theta, -2.0 * t / dh);
            rope[((size_t)pos * (dh / 2) + t) * 2] = (float)std::cos(ang);
            rope[((size_t)pos * (dh / 2) + t) * 2 + 1] = (float)std::sin(ang);
        }
    HIPOK(hipMemcpyAsync(P + L.rope, rope.data(), rope.size() * sizeof(float), hipMemcpyHostToDevice, s));
    HIPOK(hipStreamSynchronize(s));
    return DARD_OK;
}

// ---------------------------------------------------------------- forward
size_t dard_workspace_bytes(const dard_dims* d, int b, int B, int cap) {
    if (check_dims(d) || b < 1 || B < 1 || B > 256 || cap < 2 * B) return 0;
    return ws_layout(d, b, B, cap).total;
}

namespace {

struct Fwd {
    const dard_dims* d;
    Layout L;
    WsLayout W;
    const char* pk;
    char* kv;
    char* ws;
    int b, cap;
    hipStream_t s;
    const char* kv_sh = nullptr;   // a prompt cache the batch shares (b = 1, cap_sh keys)
    int cap_sh = 0;

    const void* layer(int l, size_t off) const { return pk + L.layer0 + L.layer_stride * l + off; }
    void* kc(int l) const {
        return kv + (size_t)(2 * l) * b * d->n_kv_heads * cap * d->head_dim * kv_esize(d);
    }
    void* vc(int l) const {
        return kv + (size_t)(2 * l + 1) * b * d->n_kv_heads * cap * d->head_dim * kv_esize(d);
    }
    const void* kc_sh(int l) const {
        return kv_sh + (size_t)(2 * l) * d->n_kv_heads * cap_sh * d->head_dim * kv_esize(d);
    }
    const void* vc_sh(int l) const {
        return kv_sh + (size_t)(2 * l + 1) * d->n_kv_heads * cap_sh * d->head_dim * kv_esize(d);
    }
};

// The transformer layers over `rows` token rows (R per sequence).  step 1:
// the rows are the augmented block (x then s) of block length B after P
// cached keys, attention under the state mask; step 0: the rows are the P
// prefix tokens, attention bidirectional among them; step 2 (full sequence):
// the P = N - B positions outside the current block (which starts at blk),
// then its x and s rows, with the keys in the same order; step 3: the rows
// are the positions P..P+R-1 after a shared prompt of P keys, attention
// bidirectional over the prompt and themselves.  P_sh > 0: keys [0, P_sh)
// come from the shared prompt cache f.kv_sh.
int run_layers(const Fwd& f, int R, int P, int B, int step, const uint8_t* state, const float* conf,
               uint32_t flags, int blk = 0, int P_sh = 0) {
    const dard_dims* d = f.d;
    const int dt = d->dtype;
    const int rows = f.b * R;
    const int D = d->d_model, F = d->ffn_dim, dh = d->head_dim;
    const int qd = d->n_heads * dh, kd = d->n_kv_heads * dh;
    float* h = (float*)(f.ws + f.W.h);
    void* xn = f.ws + f.W.xn;
    void* q = f.ws + f.W.q;
    void* at = f.ws + f.W.attn;
    void* act = f.ws + f.W.act;
    const bool fr = frag_rows(dt, rows);   // activations feeding the GEMMs fragment-major
    for (int l = 0; l < d->n_layers; ++l) {
        EpiArgs e{};
        e.kind = EPI_QKV; e.q = q; e.ldq = qd; e.kc = f.kc(l); e.vc = f.vc(l);
        e.rope = (const float*)(f.pk + f.L.rope);
        e.rows_per_seq = R; e.P = P; e.B = B; e.cap = f.cap; e.Hq = d->n_heads; e.Hkv = d->n_kv_heads; e.dh = dh;
        e.step = step; e.blk = blk; e.kv_fp8 = d->kv_format == DARD_KV_FP8;
        HIPOK(launch_gemm(dt, xn, rows, D, D, f.layer(l, f.L.wqkv), qd + 2 * kd, e, DARD_K_GEMM_QKV, f.s, fr));

        AttnArgs a{};
        a.q = q; a.k = f.kc(l); a.v = f.vc(l); a.out = at; a.state = state; a.conf = conf;
        a.sel = (step == 1 || step == 2) ? (const uint64_t*)(f.ws + f.W.sel) : nullptr;
        a.b = f.b; a.R = R; a.Hq = d->n_heads; a.Hkv = d->n_kv_heads; a.dh = dh; a.cap = f.cap;
        const bool masked = step == 1 || step == 2;
        a.P = P; a.B = B; a.nkeys = masked ? P + 2 * B : (step == 3 ? P + R : P); a.masked = masked;
        a.scale = 1.f / std::sqrt((float)dh);
        a.ctx_rows = step == 2 ? P : 0;
        if (P_sh > 0) {
            a.k_sh = f.kc_sh(l); a.v_sh = f.vc_sh(l); a.cap_sh = f.cap_sh; a.P_sh = P_sh;
        }
        a.flags = flags; a.part = (float*)(f.ws + f.W.part); a.part_ml = (float*)(f.ws + f.W.part_ml);
        a.part_slots = f.W.part_slots;
        a.out_frag = fr;
        a.kv_fp8 = d->kv_format == DARD_KV_FP8;
        {
            TraceScope ts(DARD_K_ATTENTION, f.s);
            HIPOK(launch_attention(dt, a, f.s));
        }
        EpiArgs r{};
        r.kind = EPI_RESID; r.y = h; r.ldy = D;
        // O projection: residual add in the epilogue, or split-K partials that
        // the residual-norm kernel adds in a fixed order
        const int so = gemm_split(dt, rows, D, qd);
        float* gp = (float*)(f.ws + f.W.gpart);
        EpiArgs po{};
        po.kind = EPI_PARTIAL; po.y = gp; po.ldy = D;
        HIPOK(launch_gemm(dt, at, rows, qd, qd, f.layer(l, f.L.wo), D, so > 1 ? po : r, DARD_K_GEMM_O, f.s, fr));
        HIPOK(launch_resid_norm(dt, h, gp, so > 1 ? so : 0, rows, D, f.layer(l, f.L.ffn_norm), d->norm_eps, xn, fr,
                                f.s));
        EpiArgs g{};
        g.kind = EPI_SWIGLU; g.act = act; g.ld_act = F; g.act_frag = fr;
        HIPOK(launch_gemm(dt, xn, rows, D, D, f.layer(l, f.L.wgu), 2 * F, g, DARD_K_GEMM_GU, f.s, fr));
        const int sd = gemm_split(dt, rows, D, F);
        HIPOK(launch_gemm(dt, act, rows, F, F, f.layer(l, f.L.wdown), D, sd > 1 ? po : r, DARD_K_GEMM_DOWN, f.s, fr));
        const void* gain = l + 1 < d->n_layers ? f.layer(l + 1, f.L.attn_norm) : f.pk + f.L.final_norm;
        HIPOK(launch_resid_norm(dt, h, gp, sd > 1 ? sd : 0, rows, D, gain, d->norm_eps, xn, fr, f.s));
    }
    return DARD_OK;
}

int fwd_setup(Fwd& f, const dard_dims* d, const void* packed, void* kv, int cap, int b, int B, void* ws,
              size_t ws_bytes, void* stream) {
    int rc = check_dims(d);
    if (rc) return rc;
    if (!packed || !kv || !ws) return fail(DARD_ERR_ARG, "NULL pointer");
    if (b < 1 || B < 1 || B > 256 || cap < 2 * B) return fail(DARD_ERR_SHAPE, "need b >= 1, 1 <= B <= 256, cap >= 2B");
    f.d = d; f.L = layout_of(d); f.W = ws_layout(d, b, B, cap);
    if (ws_bytes < f.W.total) return fail(DARD_ERR_WORKSPACE, "workspace needs %zu bytes", f.W.total);
    f.pk = (const char*)packed; f.kv = (char*)kv; f.ws = (char*)ws; f.b = b; f.cap = cap;
    f.s = (hipStream_t)stream;
    return DARD_OK;
}

}  // namespace

dard_status dard_prefill(const dard_dims* d, const void* packed, void* kv, int cap, int b, int P, const int32_t* ids,
                         const void* embeds, void* ws, size_t ws_bytes, void* stream) {
    Fwd f;
    // the workspace is sized for (b, B, cap); prefill rows b*P fit because P <= cap
    int rc = check_dims(d);
    if (rc) return rc;
    if (!ids) return fail(DARD_ERR_ARG, "NULL ids");
    if (P < 1 || P > cap || P > d->max_pos) return fail(DARD_ERR_SHAPE, "need 1 <= P <= min(cap, max_pos)");
    rc = fwd_setup(f, d, packed, kv, cap, b, 1, ws, ws_bytes, stream);
    if (rc) return rc;
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    HIPOK(launch_embed_norm(d->dtype, ids, embeds, f.pk + f.L.embed, gain0, b * P, d->d_model, d->vocab, d->norm_eps, 0, 0,
                            (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, b * P), f.s));
    return run_layers(f, P, P, 0, 0, nullptr, nullptr, 0);
}

namespace {

// The end of a step, shared by every step mode (a4-a8): the LM head over the
// final-normalised rows xrows (x then s rows of each sequence, b * 2B rows),
// the shadow confidences of the candidates, verification and guidance
// weights, the mixed confidences of the M positions and the transitions.
//   - With at most 64 rows (the weight-streaming LM head, which reads every
//     token slot of its 64 anyway) the head runs over all 2B rows.
//   - Otherwise it runs only on the rows the decisions read (lmhead.hip):
//     B + |M| rows per sequence with logit mixing; with hidden-state mixing
//     (DARD_F_HIDDEN_MIX, Eq. 7 applied to the final hidden state) the
//     candidates' shadow rows first, then, once their verification has given
//     the guidance weights, the U shadow rows and one mixed row per M
//     position: B rows per sequence.
//   - When the large-tile GEMM runs the head (and neither the entropy /
//     margin statistics nor the current-token probability are asked for),
//     its epilogue forms the (max, argmax, sum) partials of the C and U
//     shadow rows itself and their logits are never written.
int step_tail(const Fwd& f, const dard_params* params, int b, int B, const void* xrows, const int32_t* tok_in,
              const uint8_t* state_in, int32_t* tok_out, uint8_t* state_out, float* conf_out, int32_t* block_done,
              const dard_step_debug* dbg) {
    const dard_dims* d = f.d;
    const int rows = b * 2 * B, V = d->vocab, D = d->d_model, dt = d->dtype;
    float* logits = (float*)(f.ws + f.W.logits);
    float* cpv = (float*)(f.ws + f.W.cpart_v);
    float* cpm = (float*)(f.ws + f.W.cpart_m);
    float* wbuf = (float*)(f.ws + f.W.w);
    const uint32_t flags = params->flags;
    const bool stats = needs_stats(flags);
    const bool hidden = (flags & DARD_F_HIDDEN_MIX) != 0;
    const bool frag = frag_rows(dt, rows);
    const void* head_w = f.pk + f.L.lm_head;

    ConfArgs c{};
    c.ls = logits; c.ld_s = V; c.ld_x = V; c.rows = b * B; c.V = V; c.state = state_in; c.step_B = B;
    DecideArgs a{};
    a.b = b; a.B = B; a.tau_c = params->tau_c; a.tau_u = params->tau_u; a.lambda = params->lambda;
    a.p0 = params->p0; a.mask_id = params->mask_id; a.flags = flags; a.w_fixed = params->w_fixed;
    a.state_in = state_in; a.tok_in = tok_in; a.stride = stats ? kConfStatsStride : kConfStride;
    a.part_v = cpv; a.part_m = cpm;
    a.logits = logits; a.ld = V; a.nchunk = conf_chunks(V);
    a.w_out = wbuf;
    auto verify = [&]() -> int {
        a.phase = DARD_PHASE_VERIFY;
        HIPOK(launch_decide(a, f.s));
        return DARD_OK;
    };
    auto final_phase = [&]() -> int {
        a.phase = DARD_PHASE_FINAL;
        a.state_out = state_out; a.tok_out = tok_out; a.conf_out = conf_out; a.block_done = block_done;
        if (dbg) {
            a.dbg_maxprob_s = dbg->maxprob_s; a.dbg_argmax_s = dbg->argmax_s; a.dbg_pcur_s = dbg->pcur_s;
            a.dbg_maxprob_mix = dbg->maxprob_mix; a.dbg_argmax_mix = dbg->argmax_mix;
            if (stats) { a.dbg_entropy = dbg->entropy; a.dbg_margin = dbg->margin; }
        }
        HIPOK(launch_decide(a, f.s));
        if (dbg && dbg->w) HIPOK(hipMemcpyAsync(dbg->w, wbuf, (size_t)b * B * 4, hipMemcpyDeviceToDevice, f.s));
        return DARD_OK;
    };

    const int max_rows = hidden ? b * B : rows;
    int32_t plan[4];
    gemm_plan(dt, max_rows, V, D, false, frag, plan, true);
    if (!hidden && plan[0] == DARD_GEMM_STREAM) {
        EpiArgs e{};
        e.kind = EPI_STORE_F32; e.y = logits; e.ldy = V;
        HIPOK(launch_gemm(dt, xrows, rows, D, D, head_w, V, e, DARD_K_GEMM_HEAD, f.s, frag));
        c.phase = 0; c.part = cpv;
        HIPOK(launch_conf_partial(c, stats, f.s));
        if (int rc = verify()) return rc;
        c.phase = 1; c.w = wbuf; c.part = cpm;
        HIPOK(launch_conf_partial(c, stats, f.s));
        if (int rc = final_phase()) return rc;
        if (dbg && dbg->logits)
            HIPOK(hipMemcpyAsync(dbg->logits, logits, (size_t)rows * V * 4, hipMemcpyDeviceToDevice, f.s));
        return DARD_OK;
    }

    const bool fused = dt == DARD_DTYPE_BF16 && plan[0] == DARD_GEMM_BIG && !stats &&
                       !(flags & DARD_F_VERIFY_PCUR);
    int32_t* rm0 = (int32_t*)(f.ws + f.W.rowmap);
    int32_t* rm1 = rm0 + rows;
    int32_t* cnt = (int32_t*)(f.ws + f.W.lmcount);
    void* hx = f.ws + f.W.hx;
    float* lpart = (float*)(f.ws + f.W.lpart);
    const int tile_cols = 32 * plan[2];
    {
        TraceScope ts(DARD_K_GEMM_HEAD, f.s);   // the row lists belong to the LM-head stage
        HIPOK(launch_lm_select(state_in, b, B, hidden ? 1 : 0, fused, rm0, rm1, cnt, f.s));
    }
    auto head = [&](const int32_t* rm, const int32_t* count) -> int {
        {
            TraceScope ts(DARD_K_GEMM_HEAD, f.s);
            HIPOK(launch_lm_gather(dt, xrows, D, frag, rm, count, max_rows, wbuf, B, hx, f.s));
        }
        EpiArgs e{};
        e.kind = EPI_LMHEAD; e.y = logits; e.ldy = V; e.rowmap = rm; e.rows_dev = count;
        e.y2 = dbg ? dbg->logits : nullptr;
        if (fused) { e.lpart = lpart; e.ntile = (V + tile_cols - 1) / tile_cols; }
        HIPOK(launch_gemm(dt, hx, max_rows, D, D, head_w, V, e, DARD_K_GEMM_HEAD, f.s, frag_rows(dt, max_rows)));
        if (fused) {
            TraceScope ts(DARD_K_CONFIDENCE, f.s);
            HIPOK(launch_lm_merge(lpart, e.ntile, tile_cols, rm, count, max_rows, B, V, cpv, cpm, f.s));
        }
        return DARD_OK;
    };
    // the candidates' shadow rows (and, with logit mixing, every other listed row)
    if (int rc = head(rm0, cnt)) return rc;
    if (!fused) {
        c.phase = 0; c.part = cpv;
        HIPOK(launch_conf_partial(c, stats, f.s));
    }
    if (int rc = verify()) return rc;
    if (hidden) {
        // U shadow rows and the mixed rows of the M positions (guidance weights from verify)
        if (int rc = head(rm1, cnt + 1)) return rc;
        if (!fused) {
            c.phase = 1; c.no_mix = 1; c.part = cpm;
            HIPOK(launch_conf_partial(c, stats, f.s));
        }
    } else {
        // logit mixing of the M positions (Eq. 7); with the fused head the U rows' partials are already there
        c.phase = 1; c.w = wbuf; c.part = cpm; c.m_only = fused;
        HIPOK(launch_conf_partial(c, stats, f.s));
    }
    return final_phase();
}

int check_step_args(const dard_dims* d, const dard_params* params, const void* tok, const uint8_t* state_in,
                    const float* conf_in, const int32_t* tok_out, const uint8_t* state_out, const float* conf_out,
                    const int32_t* block_done) {
    if (int rc = check_params(params)) return rc;
    if (!tok || !state_in || !conf_in || !tok_out || !state_out || !conf_out) return fail(DARD_ERR_ARG, "NULL pointer");
    if ((params->flags & DARD_F_CHECK_STATES) && !block_done)
        return fail(DARD_ERR_ARG, "DARD_F_CHECK_STATES reports through block_done");
    if (params->mask_id < 0 || params->mask_id >= d->vocab) return fail(DARD_ERR_ARG, "mask_id outside the vocab");
    return DARD_OK;
}

}  // namespace

dard_status dard_step(const dard_dims* d, const void* packed, void* kv, int cap, int P, const dard_params* params,
                      int b, int B, const int32_t* tok_in, const uint8_t* state_in, const float* conf_in,
                      int32_t* tok_out, uint8_t* state_out, float* conf_out, int32_t* block_done,
                      const dard_step_debug* dbg, void* ws, size_t ws_bytes, void* stream) {
    Fwd f;
    int rc = fwd_setup(f, d, packed, kv, cap, b, B, ws, ws_bytes, stream);
    if (rc) return rc;
    rc = check_step_args(d, params, tok_in, state_in, conf_in, tok_out, state_out, conf_out, block_done);
    if (rc) return rc;
    if (P < 0 || P + 2 * B > cap || P + B > d->max_pos)
        return fail(DARD_ERR_SHAPE, "need P >= 0, P + 2B <= cap, P + B <= max_pos");
    const int R = 2 * B, rows = b * R;
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    // the state mask (Eq. 2-3) is the same for every layer of the step: build it once
    {
        TraceScope ts(DARD_K_MASK, f.s);
        HIPOK(launch_build_state_mask(state_in, conf_in, b, B, params->flags, (uint64_t*)(f.ws + f.W.sel), f.s));
    }
    HIPOK(launch_embed_norm(d->dtype, tok_in, nullptr, f.pk + f.L.embed, gain0, rows, d->d_model, d->vocab, d->norm_eps, B,
                            params->mask_id, (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, rows), f.s));
    rc = run_layers(f, R, P, B, 1, state_in, conf_in, params->flags);
    if (rc) return rc;
    return step_tail(f, params, b, B, f.ws + f.W.xn, tok_in, state_in, tok_out, state_out, conf_out, block_done, dbg);
}

dard_status dard_step_full(const dard_dims* d, const void* packed, void* kv, int cap, int N, int blk,
                           const dard_params* params, int b, int B, const int32_t* seq, const uint8_t* state_in,
                           const float* conf_in, int32_t* tok_out, uint8_t* state_out, float* conf_out,
                           int32_t* block_done, const dard_step_debug* dbg, void* ws, size_t ws_bytes,
                           void* stream) {
    Fwd f;
    int rc = fwd_setup(f, d, packed, kv, cap, b, B, ws, ws_bytes, stream);
    if (rc) return rc;
    rc = check_step_args(d, params, seq, state_in, conf_in, tok_out, state_out, conf_out, block_done);
    if (rc) return rc;
    if (N < B || blk < 0 || blk + B > N || N + B > cap || N > d->max_pos)
        return fail(DARD_ERR_SHAPE, "need B <= N, 0 <= blk <= N - B, N + B <= cap, N <= max_pos");
    const int R = N + B, Nc = N - B, rows = b * R;
    int32_t* row_ids = (int32_t*)(f.ws + f.W.ids);
    int32_t* tok = (int32_t*)(f.ws + f.W.tok);
    HIPOK(launch_full_rows(seq, b, N, blk, B, params->mask_id, row_ids, tok, f.s));
    {
        TraceScope ts(DARD_K_MASK, f.s);
        HIPOK(launch_build_state_mask(state_in, conf_in, b, B, params->flags, (uint64_t*)(f.ws + f.W.sel), f.s));
    }
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    HIPOK(launch_embed_norm(d->dtype, row_ids, nullptr, f.pk + f.L.embed, gain0, rows, d->d_model, d->vocab,
                            d->norm_eps, 0, 0, (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, rows), f.s));
    rc = run_layers(f, R, Nc, B, 2, state_in, conf_in, params->flags, blk);
    if (rc) return rc;
    // the current block's x and s rows (the last 2B of each sequence) feed the
    // LM head; the Q buffer (rows x d_model) is free once the last layer ran
    void* xrows = f.ws + f.W.q;
    HIPOK(launch_gather_rows(d->dtype, f.ws + f.W.xn, b, R, Nc, 2 * B, d->d_model, frag_rows(d->dtype, rows), xrows,
                             f.s));
    return step_tail(f, params, b, B, xrows, tok, state_in, tok_out, state_out, conf_out, block_done, dbg);
}

namespace {

int attach_shared(Fwd& f, const void* kv_shared, int cap_shared, int Ps, int P) {
    if (!kv_shared) return fail(DARD_ERR_ARG, "NULL shared cache");
    if (Ps < 64 || Ps % 64 || Ps > cap_shared || Ps > P)
        return fail(DARD_ERR_SHAPE, "need a shared prompt of 64k keys, 64 <= Ps <= min(cap_shared, P)");
    f.kv_sh = (const char*)kv_shared;
    f.cap_sh = cap_shared;
    return DARD_OK;
}

}  // namespace

dard_status dard_prefill_suffix(const dard_dims* d, const void* packed, void* kv, int cap, const void* kv_shared,
                                int cap_shared, int Ps, int b, int Pc, const int32_t* ids, void* ws, size_t ws_bytes,
                                void* stream) {
    Fwd f;
    int rc = fwd_setup(f, d, packed, kv, cap, b, 1, ws, ws_bytes, stream);
    if (rc) return rc;
    if (!ids) return fail(DARD_ERR_ARG, "NULL ids");
    if (Pc < 1 || Ps + Pc > cap || Ps + Pc > d->max_pos) return fail(DARD_ERR_SHAPE, "need Pc >= 1, Ps + Pc <= min(cap, max_pos)");
    rc = attach_shared(f, kv_shared, cap_shared, Ps, Ps + Pc);
    if (rc) return rc;
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    HIPOK(launch_embed_norm(d->dtype, ids, nullptr, f.pk + f.L.embed, gain0, b * Pc, d->d_model, d->vocab, d->norm_eps,
                            0, 0, (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, b * Pc), f.s));
    return run_layers(f, Pc, Ps, 0, 3, nullptr, nullptr, 0, 0, Ps);
}

dard_status dard_prefill_extend(const dard_dims* d, const void* packed, void* kv, int cap, int P, int b, int Pn,
                                const int32_t* ids, void* ws, size_t ws_bytes, void* stream) {
    Fwd f;
    int rc = fwd_setup(f, d, packed, kv, cap, b, 1, ws, ws_bytes, stream);
    if (rc) return rc;
    if (!ids) return fail(DARD_ERR_ARG, "NULL ids");
    if (P < 0 || Pn < 1 || P + Pn > cap || P + Pn > d->max_pos)
        return fail(DARD_ERR_SHAPE, "need P >= 0, Pn >= 1, P + Pn <= min(cap, max_pos)");
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    HIPOK(launch_embed_norm(d->dtype, ids, nullptr, f.pk + f.L.embed, gain0, b * Pn, d->d_model, d->vocab, d->norm_eps,
                            0, 0, (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, b * Pn), f.s));
    // the new rows at positions P.., keys 0..P+Pn-1 of the sequence's own cache
    return run_layers(f, Pn, P, 0, 3, nullptr, nullptr, 0, 0, 0);
}

dard_status dard_step_shared(const dard_dims* d, const void* packed, void* kv, int cap, const void* kv_shared,
                             int cap_shared, int Ps, int P, const dard_params* params, int b, int B,
                             const int32_t* tok_in, const uint8_t* state_in, const float* conf_in, int32_t* tok_out,
                             uint8_t* state_out, float* conf_out, int32_t* block_done, const dard_step_debug* dbg,
                             void* ws, size_t ws_bytes, void* stream) {
    Fwd f;
    int rc = fwd_setup(f, d, packed, kv, cap, b, B, ws, ws_bytes, stream);
    if (rc) return rc;
    rc = check_step_args(d, params, tok_in, state_in, conf_in, tok_out, state_out, conf_out, block_done);
    if (rc) return rc;
    if (P + 2 * B > cap || P + B > d->max_pos) return fail(DARD_ERR_SHAPE, "need P + 2B <= cap, P + B <= max_pos");
    rc = attach_shared(f, kv_shared, cap_shared, Ps, P);
    if (rc) return rc;
    const int R = 2 * B, rows = b * R;
    const void* gain0 = d->n_layers > 0 ? f.layer(0, f.L.attn_norm) : f.pk + f.L.final_norm;
    {
        TraceScope ts(DARD_K_MASK, f.s);
        HIPOK(launch_build_state_mask(state_in, conf_in, b, B, params->flags, (uint64_t*)(f.ws + f.W.sel), f.s));
    }
    HIPOK(launch_embed_norm(d->dtype, tok_in, nullptr, f.pk + f.L.embed, gain0, rows, d->d_model, d->vocab, d->norm_eps, B,
                            params->mask_id, (float*)(f.ws + f.W.h), f.ws + f.W.xn, frag_rows(d->dtype, rows), f.s));
    rc = run_layers(f, R, P, B, 1, state_in, conf_in, params->flags, 0, Ps);
    if (rc) return rc;
    return step_tail(f, params, b, B, f.ws + f.W.xn, tok_in, state_in, tok_out, state_out, conf_out, block_done, dbg);
}

// ---------------------------------------------------------------- linear
dard_status dard_pack_matrix(int dtype, const void* W, int N, int K, void* Wp, void* stream) {
    if (!W || !Wp) return fail(DARD_ERR_ARG, "NULL pointer");
    if (dtype != DARD_DTYPE_F32 && dtype != DARD_DTYPE_BF16) return fail(DARD_ERR_ARG, "unknown dtype");
    if (N < 1 || K < 1) return fail(DARD_ERR_SHAPE, "need N, K >= 1");
    if (dtype == DARD_DTYPE_BF16 && (K % 64 || N % 16)) return fail(DARD_ERR_SHAPE, "bf16 needs K %% 64 == 0, N %% 16 == 0");
    if (dtype == DARD_DTYPE_F32 && K % 4) return fail(DARD_ERR_SHAPE, "f32 needs K %% 4 == 0");
    hipStream_t s = (hipStream_t)stream;
    if (dtype == DARD_DTYPE_BF16)
        HIPOK(launch_pack_frag(W, nullptr, Wp, N, K, 0, 64, s));
    else
        HIPOK(launch_copy_rows(W, Wp, (size_t)N * K * 4, s));
    return DARD_OK;
}

dard_status dard_linear(int dtype, const void* X, int M, int K, const void* Wp, int N, float* Y, void* stream) {
    if (!X || !Wp || !Y) return fail(DARD_ERR_ARG, "NULL pointer");
    if (dtype != DARD_DTYPE_F32 && dtype != DARD_DTYPE_BF16) return fail(DARD_ERR_ARG, "unknown dtype");
    if (M < 1 || N < 1 || K < 1) return fail(DARD_ERR_SHAPE, "need M, N, K >= 1");
    if (dtype == DARD_DTYPE_BF16 && (K % 64 || N % 16)) return fail(DARD_ERR_SHAPE, "bf16 needs K %% 64 == 0, N %% 16 == 0");
    if (dtype == DARD_DTYPE_F32 && (N % 4 || K % 4)) return fail(DARD_ERR_SHAPE, "f32 needs N, K %% 4 == 0");
    EpiArgs e{};
    e.kind = EPI_STORE_F32; e.y = Y; e.ldy = N;
    HIPOK(launch_gemm(dtype, X, M, K, K, Wp, N, e, DARD_K_GEMM_HEAD, (hipStream_t)stream));
    return DARD_OK;
}

dard_status dard_gemm_plan(int dtype, int M, int N, int K, int partial, int frag_x, int32_t* plan) {
    if (!plan) return fail(DARD_ERR_ARG, "NULL pointer");
    if (dtype != DARD_DTYPE_F32 && dtype != DARD_DTYPE_BF16) return fail(DARD_ERR_ARG, "unknown dtype");
    if (M < 1 || N < 1 || K < 1) return fail(DARD_ERR_SHAPE, "need M, N, K >= 1");
    if (dtype == DARD_DTYPE_BF16 && (K % 64 || N % 16)) return fail(DARD_ERR_SHAPE, "bf16 needs K %% 64 == 0, N %% 16 == 0");
    gemm_plan(dtype, M, N, K, partial != 0, frag_x != 0, plan);
    return DARD_OK;
}

// ---------------------------------------------------------------- tracing
dard_status dard_trace_enable(uint32_t class_mask) {
    g_trace_mask = class_mask;
    return DARD_OK;
}

dard_status dard_trace_read(int cls, int64_t* launches, double* total_ms) {
    if (cls < 0 || cls >= DARD_K_COUNT || !launches || !total_ms) return fail(DARD_ERR_ARG, "bad trace query");
    std::lock_guard<std::mutex> lk(g_trace_mu);
    double sum = 0.0;
    for (auto& r : g_trace[cls]) {
        HIPOK(hipEventSynchronize(r.b));
        float ms = 0.f;
        HIPOK(hipEventElapsedTime(&ms, r.a, r.b));
        sum += ms;
    }
    *launches = (int64_t)g_trace[cls].size();
    *total_ms = sum;
    return DARD_OK;
}

dard_status dard_trace_sample(int period) {
    if (period < 1) return fail(DARD_ERR_ARG, "period must be >= 1");
    std::lock_guard<std::mutex> lk(g_trace_mu);
    g_trace_period = period;
    return DARD_OK;
}

dard_status dard_trace_reset(void) {
    std::lock_guard<std::mutex> lk(g_trace_mu);
    for (auto& n : g_trace_seen) n = 0;
    for (auto& v : g_trace) {
        for (auto& r : v) {
            hipEventSynchronize(r.b);
            hipEventDestroy(r.a);
            hipEventDestroy(r.b);
        }
        v.clear();
    }
    return DARD_OK;
}

}  // extern "C"
