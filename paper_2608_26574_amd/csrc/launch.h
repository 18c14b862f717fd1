// Host-side launchers of the libdard kernels (internal interface between the
// C ABI in api.cpp and the kernel translation units).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/dard.h"

namespace dard {

// bf16 activations that feed a projection GEMM are stored fragment-major, in
// the layout of the packed weights: the 16 x 64 block (m/16, k/64) is
// contiguous, so every wave load (streaming GEMM) or tile copy (pipelined
// GEMM) of them reads whole 1 KB runs.  Producers (norms, SwiGLU epilogue,
// attention output) write that layout when frag_rows(dtype, rows) holds;
// buffers then hold whole blocks (rows rounded up to 64).
inline bool frag_rows(int dtype, int rows) { return dtype == DARD_DTYPE_BF16 && rows > 0; }

// ---- mask.hip
hipError_t launch_build_state_mask(const uint8_t* state, const float* conf, int b, int B,
                                   uint32_t flags, uint64_t* sel, hipStream_t s);
// status[0] = number of codes outside {0, 1, 2} among state[0..n), status[1] = first index or -1
hipError_t launch_check_states(const uint8_t* state, int n, int32_t* status, hipStream_t s);

// ---- attention.hip
struct AttnArgs {
    const void* q;      // [b][R][Hq][dh]
    const void* k;      // [b][Hkv][cap][dh]
    const void* v;      // [b][Hkv][dh][cap] (dims-major)
    void* out;          // [b][R][Hq][dh]
    const uint8_t* state;  // [b][B] (masked mode, fp32 path)
    const float* conf;     // [b][B]
    const uint64_t* sel;   // [b][R - ctx_rows][ceil(B/64)] take-x words of the block rows (masked mode, bf16)
    int b, R, Hq, Hkv, dh, cap;
    int P;              // prefix keys (always visible)
    int B;              // block length (masked mode); keys = P + 2B
    int nkeys;          // total keys per sequence
    int masked;         // 1: state-specific mask on keys >= P; 0: all visible
    int ctx_rows;       // masked mode: leading rows of a sequence outside the block (full-sequence
                        // mode); they see the P keys and the B x keys, no shadow key
    const void* k_sh;   // keys [0, P_sh) of every sequence come from one cache shared by the
    const void* v_sh;   // batch (K [Hkv][cap_sh][dh], V [Hkv][dh][cap_sh]); P_sh % 64 == 0
    int cap_sh, P_sh;
    float scale;
    uint32_t flags;
    float* part;        // key-split partials [nsplit][b][R][Hq][dh] fp32 (bf16 only)
    float* part_ml;     // [nsplit][b][R][Hq][2]: running max (log2 units) and sum
    size_t part_slots;  // capacity of part / part_ml in (split, row, head) slots
    int out_frag;       // 1: out is fragment-major [b*R][Hq*dh] (bf16 only)
    int kv_fp8;         // 1: k, v (and k_sh, v_sh) hold OCP FP8 E4M3 codes (bf16 q / out)
};
// 64-key tiles of a launch: the prefix (or all keys when unmasked), then the block.
int attention_tiles(int masked, int P, int B, int nkeys);
// Partial slots a launch of these sizes would use (0 = no key split).
size_t attention_partial_slots(int dtype, int b, int R, int Hq, int Hkv, int ntiles);
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s);

// ---- gemm.hip
enum EpiKind { EPI_STORE_F32 = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_PARTIAL = 4, EPI_LMHEAD = 5 };

// Code of a listed LM-head row (lmhead.hip): its logit row (sequence * 2B +
// row) and what becomes of its logits.
constexpr int kLmRowMask = (1 << 24) - 1;
constexpr int kLmStore = 1 << 24;   // stored at the logit row
constexpr int kLmToV = 1 << 25;     // merged partial of a candidate's shadow row (verification)
constexpr int kLmToM = 1 << 26;     // merged partial of a U shadow row or of a mixed M row
constexpr int kLmMix = 1 << 27;     // the row is w x + (1 - w) s of an M position (hidden-state mixing)

struct EpiArgs {
    int kind;
    // LMHEAD: the rows are listed rows (rowmap codes); rows at or past the
    // device count *rows_dev are skipped (row tiles entirely past it exit
    // before their K loop).  Stored rows go to y (ldy = V) at their logit
    // row, every row also to y2 when it is set (debug capture); with lpart
    // the large-tile kernel writes per-column-tile (max, argmax, sum)
    // partials [M][ntile][3] of every row instead of needing its logits.
    const int32_t* rowmap;
    const int32_t* rows_dev;
    float* y2;
    float* lpart;
    int ntile;
    float* y;  int ldy;             // STORE_F32 / RESID (fp32, RESID adds)
    void* act; int ld_act;          // SWIGLU output (dtype), columns N/2
    int act_frag;                   // 1: act fragment-major with K = ld_act
    // QKV
    void* q; int ldq;               // [rows][Hq*dh]
    void* kc; void* vc;             // cache base of this layer: K [b][Hkv][cap][dh], V [b][Hkv][dh][cap]
    const float* rope;              // [max_pos][dh/2][2] (cos, sin)
    int rows_per_seq;               // R
    int P, B, cap, Hq, Hkv, dh;
    int kv_fp8;                     // 1: K and V are written to the cache as OCP FP8 E4M3 codes
    int step;                       // 1: row r -> pos P + r%B, cache P + r; 0: pos = cache = r;
                                    // 2 (full sequence): cache r, pos r (r < blk), r + B (blk <= r < P),
                                    //   blk + (r - P) % B (block rows r >= P);
                                    // 3 (positions after a shared prompt of P): pos = cache = P + r
    int blk;                        // step 2: position of the current block
};
// Y = X * W^T with X [M][K] (leading dim ldx, or fragment-major when xfrag),
// W [N][K] packed (bf16: fragment-major, fp32: row-major); epilogue per `e`.
// With EPI_PARTIAL the output is gemm_split(...) fp32 partials [split][M][ldy]
// at e.y.  xfrag needs frag_rows(dtype, M).
hipError_t launch_gemm(int dtype, const void* X, int M, int K, int ldx, const void* W, int N,
                       const EpiArgs& e, int kernel_class, hipStream_t s, bool xfrag = false);
int gemm_split(int dtype, int M, int N, int K);
// The kernel and tiling launch_gemm picks for these sizes (dard_gemm_plan);
// fused_head: the LM-head epilogue with column-tile partials (tile widths
// that divide kConfChunk only).
void gemm_plan(int dtype, int M, int N, int K, bool partial, bool xfrag, int32_t* plan, bool fused_head = false);
// bf16 fragment-major packing (mode 0 plain, 1 rotary-pair rows, 2 gate/up interleave)
hipError_t launch_pack_frag(const void* src0, const void* src1, void* dst, int N, int K, int mode, int dh,
                            hipStream_t s);

// ---- elementwise.hip
// h[row] = embedding of ids[row] (or embeds[row] when ids[row] < 0), then
// xn[row] = RMSNorm(h[row]) * gain.  When step_B > 0 the rows are the
// augmented block: row r of sequence s embeds tok[s][r] for r < B and mask_id
// for r >= B.
hipError_t launch_embed_norm(int dtype, const int32_t* ids, const void* embeds,
                             const void* table, const void* gain, int rows, int d, int vocab,
                             float eps, int step_B, int mask_id, float* h, void* xn,
                             bool frag, hipStream_t s);
// h[row] += sum of the nsplit fp32 partials part[s][row] (nsplit may be 0),
// then xn[row] = RMSNorm(h[row]) * gain (fragment-major when frag).  Needs
// d % 4 == 0, d <= 8192.
hipError_t launch_resid_norm(int dtype, float* h, const float* part, int nsplit, int rows, int d,
                             const void* gain, float eps, void* xn, bool frag, hipStream_t s);
hipError_t launch_copy_rows(const void* src, void* dst, size_t bytes, hipStream_t s);
// Full-sequence mode rows: row_ids [b][N + B] = the sequence seq [b][N] with the
// current block (positions blk..blk+B-1) moved behind the other N - B
// positions, then B shadow rows of mask_id; tok [b][B] = the block's tokens.
hipError_t launch_full_rows(const int32_t* seq, int b, int N, int blk, int B, int mask_id, int32_t* row_ids,
                            int32_t* tok, hipStream_t s);
// Copy rows first..first+count-1 of every sequence of R rows ([b*R][d], dtype,
// fragment-major when frag) to a compact [b*count][d] of the same layout.
hipError_t launch_gather_rows(int dtype, const void* src, int b, int R, int first, int count, int d, bool frag,
                              void* dst, hipStream_t s);
hipError_t launch_pack_rows(const void* src0, const void* src1, void* dst, int nrows, int rowbytes, int mode,
                            int dh, hipStream_t s);

// ---- confidence.hip
struct ConfArgs {
    const float* ls;       // shadow / plain rows
    const float* lx;       // x rows or NULL
    const float* w;        // per-row weight or NULL
    int64_t ld_s, ld_x;    // row strides (elements)
    int rows, V, nchunk, chunk;
    float* part;           // [rows][nchunk][kConfStride]: max, argmax (as int bits), sum;
                           // statistics variant [rows][nchunk][kConfStatsStride]:
                           // also sum exp(l - max) (l - max) and the second-largest l
    // step mode: skip rows by state (phase 0: only C rows; phase 1: only M/U)
    const uint8_t* state;  // [rows] or NULL
    int phase;
    int step_B;            // >0: rows are block positions of [b][2B][V] logits
    int m_only;            // phase 1: only M rows (the U rows' partials come from elsewhere)
    int no_mix;            // phase 1: M rows already mixed (hidden-state mixing): plain shadow-slot rows
};
constexpr int kConfStride = 3, kConfStatsStride = 5;
constexpr int kConfChunk = 8192;   // logits per confidence partial
int conf_chunks(int V);
// The device-resident partials array of dard_confidence_noalloc on the
// current device (looked up on first use per device) and its size in floats.
hipError_t conf_scratch(float** out);
size_t conf_scratch_floats();
// stats: also form the entropy / margin terms (partials of kConfStatsStride)
hipError_t launch_conf_partial(const ConfArgs& a, bool stats, hipStream_t s);
// entropy or margin != NULL reads statistics partials
hipError_t launch_conf_combine(const float* part, int rows, int nchunk, int V, const float* ls,
                               int64_t ld, const int32_t* cur_tok, int32_t* argmax,
                               float* maxprob, float* pcur, float* entropy, float* margin,
                               hipStream_t s);

// ---- lmhead.hip (the LM head on the rows the decisions read)
// mode 0: logit mixing (one list); mode 1: hidden-state mixing (two passes).
hipError_t launch_lm_select(const uint8_t* state, int b, int B, int mode, bool fused, int32_t* rowmap0,
                            int32_t* rowmap1, int32_t* count, hipStream_t s);
// Listed rows of xn ([b*2B][d], fragment-major when frag) into out (the same
// layout, compact); mixed rows take w [b][B].
hipError_t launch_lm_gather(int dtype, const void* xn, int d, bool frag, const int32_t* rowmap, const int32_t* count,
                            int max_rows, const float* w, int B, void* out, hipStream_t s);
// Column-tile partials (tile_cols columns each) into the chunk partials
// [b*B][conf_chunks(V)][kConfStride] of part_v (candidates) / part_m.
hipError_t launch_lm_merge(const float* lpart, int ntile, int tile_cols, const int32_t* rowmap, const int32_t* count,
                           int max_rows, int B, int V, float* part_v, float* part_m, hipStream_t s);

// ---- decide.hip
struct DecideArgs {
    int phase;
    int b, B;
    float tau_c, tau_u;
    double lambda, p0;
    int32_t mask_id;
    uint32_t flags;
    float w_fixed;
    const uint8_t* state_in;
    const int32_t* tok_in;
    // combined per-position inputs
    const float* maxprob_s; const float* pcur_s; const int32_t* argmax_s;
    const float* maxprob_mix; const int32_t* argmax_mix;
    const float* key_s; const float* key_mix;   // ordering keys (entropy / margin orders)
    // chunk partials (step mode; used when the per-position arrays are NULL)
    const float* part_v;     // [b*B][nchunk][stride] shadow rows (phase VERIFY)
    const float* part_m;     // [b*B][nchunk][stride] mixed / shadow rows (phase FINAL)
    const float* logits;     // [b][2B][V] (step mode, for pcur)
    int64_t ld;
    int nchunk, stride;      // stride kConfStatsStride: partials carry entropy / margin terms
    float* w_out;
    uint8_t* state_out; int32_t* tok_out; float* conf_out; int32_t* block_done;
    // optional debug copies
    float* dbg_maxprob_s; int32_t* dbg_argmax_s; float* dbg_pcur_s;
    float* dbg_maxprob_mix; int32_t* dbg_argmax_mix;
    float* dbg_entropy; float* dbg_margin;
};
hipError_t launch_decide(const DecideArgs& a, hipStream_t s);

// ---- tracing (api.cpp)
// While a TraceScope whose class is enabled (dard_trace_enable) is alive on
// this thread, every kernel started through launch() records its own begin
// and end timestamps, so traced times are kernel execution times without the
// dispatch gaps between kernels.  Scopes nest; the innermost one decides.
struct TraceScope {
    TraceScope(int kernel_class, hipStream_t s);
    ~TraceScope();
    // A fresh pair of timing events for the next kernel; false when the
    // innermost scope is not traced.
    static bool next_events(hipEvent_t* a, hipEvent_t* b);
    int cls;
    bool on;
    TraceScope* prev;
};

// Kernel launch used by every entry point.
template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t s, Args... args) {
    hipEvent_t a = nullptr, b = nullptr;
    TraceScope::next_events(&a, &b);
    hipExtLaunchKernelGGL(kernel, grid, block, lds, s, a, b, 0u, args...);
}

}  // namespace dard
