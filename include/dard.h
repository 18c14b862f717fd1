/*
 * dard.h -- C ABI of libdard.so, the gfx950 (MI355X) hot path of
 * Dependency-Aware Revocable Decoding (DARD, arXiv 2608.26574).
 *
 * One DARD step (Algorithm 1, one iteration of its loop) runs a bidirectional
 * transformer over the augmented block (x; s): the current block x of B
 * positions and its all-[Mask] shadow copy s, both at positions P..P+B-1 after
 * a cached prefix of P tokens.  Attention uses the state-specific mask of
 * Sec. 3.2, built from every position's state (M / C / U) and its previous
 * confidence.  The logits then drive the vocab-wide confidence reduction
 * (Eq. 1), the verification of candidates, the guidance weight of masked
 * tokens (Eq. 5-6), logit mixing (Eq. 7) and the state transition (Eq. 8).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers owned by the caller, row-major,
 *     naturally aligned (16-byte aligned for bf16/f32 tensors).  The library
 *     never frees them and, on the hot calls, allocates nothing: scratch space
 *     comes from the caller's workspace `ws` of `ws_bytes` bytes, sized by the
 *     matching *_workspace_bytes() query.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *     enqueues work on it and returns at once; results are valid once the
 *     stream has run.
 *   - Every call returns a dard_status.  Arguments are validated on the host
 *     first; on any violation nothing is enqueued and the call returns
 *     DARD_ERR_ARG / DARD_ERR_SHAPE / DARD_ERR_UNSUPPORTED.  A failing HIP call
 *     returns DARD_ERR_HIP.  dard_last_error() gives a thread-local message.
 *   - Token state codes outside {0,1,2} in device arrays give unspecified
 *     (but memory-safe) results.  They are found by dard_check_states(), or,
 *     inside a step, with the DARD_F_CHECK_STATES flag (see block_done).
 *   - Token ids in device arrays are clamped into [0, vocab) wherever a
 *     kernel indexes a table or a logit row with them (memory-safe; an id
 *     outside the vocabulary reads the nearest valid entry).
 */
#ifndef DARD_H
#define DARD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
typedef int dard_status;
#define DARD_OK               0
#define DARD_ERR_ARG        (-1)  /* null pointer, bad flag, bad parameter     */
#define DARD_ERR_SHAPE      (-2)  /* sizes outside the supported ranges        */
#define DARD_ERR_UNSUPPORTED (-3) /* valid but not implemented on this path     */
#define DARD_ERR_HIP        (-4)  /* a HIP runtime call failed                 */
#define DARD_ERR_WORKSPACE  (-5)  /* ws smaller than the size query asked for  */

/* Token states (Sec. 3.2; Eq. 8): masked, candidate, unmasked. */
#define DARD_STATE_M 0
#define DARD_STATE_C 1
#define DARD_STATE_U 2

/* Storage types of weights / activations / KV cache.  Logits, confidences
 * and the residual stream are always float32.  DARD_DTYPE_BF16_KV_FP8 is an
 * operation type of dard_masked_attention only: bf16 q / out with K and V in
 * OCP FP8 E4M3. */
#define DARD_DTYPE_F32  0
#define DARD_DTYPE_BF16 1
#define DARD_DTYPE_BF16_KV_FP8 2

/* KV-cache formats (dard_dims.kv_format): the model's storage dtype, or OCP
 * FP8 E4M3 (4 exponent bits, 3 mantissa bits, largest finite 448; bf16
 * models only).  FP8 halves the cache and the attention's key/value reads;
 * K and V are rounded to nearest-even from fp32 once, when written, with
 * magnitudes beyond 448 saturating, and widened to bf16 (exactly) before the
 * matrix cores.  Prefix caching of the prompt (App. C.5) makes the cache the
 * shadow block's memory cost; this is the variant that halves it. */
#define DARD_KV_DTYPE 0
#define DARD_KV_FP8   1

/* Flags selecting alternative readings where the paper leaves a choice open
 * (the default, 0, is the reading the library documents as primary):
 *   XSELF_SHADOW  the x query of a U token does not see its own x key
 *                 (default: it does; only shadow queries are blocked from
 *                 their own position, Sec. 3.2 "Verification of U tokens");
 *   MKEYS_SHADOW  the x query of an M token reads the other M positions from
 *                 s (default: from x, i.e. the x stream is vanilla decoding);
 *   VERIFY_PCUR   C/U confidence = probability of the current token instead of
 *                 the top-1 probability of Eq. 1 (default);
 *   PROGRESS      a decoding-loop rule, not the paper's (Alg. 1 assumes the
 *                 confidences eventually pass tau_u): if no position of an
 *                 unfinished block entered U in this step, the most confident
 *                 position that is not U after the transitions (ties: lowest
 *                 position) becomes U with its prediction, so every step
 *                 of an unfinished block commits at least one position (U
 *                 positions are re-verified and may fall back, so a
 *                 decoding loop still bounds its steps per block).
 * Variants of the design-choice analysis (Sec. 5.1, mask-design and
 * logit-mixing ablations); at most one of the four ordering flags is allowed:
 *   C_BIDIR       a candidate's queries see every candidate in x (no order;
 *                 the shadow query still never sees its own x key);
 *   ORDER_L2R     candidates ordered by position: candidate i sees the
 *                 candidates j <= i in x (Eq. 3 with the key -j);
 *   ORDER_ENTROPY candidates ordered by the entropy of their prediction,
 *                 lowest first: the key carried to the next step (conf_out
 *                 of dard_step) is -H, H = -sum_v p_v ln p_v;
 *   ORDER_MARGIN  ordered by the margin p_(1) - p_(2) of the two largest
 *                 probabilities, largest first: the carried key is the margin;
 *   FIXED_W       every masked token mixes its logits with the constant
 *                 params.w_fixed instead of the weight of Eq. 5-6.
 * An evaluation order (the steps only; other entry points ignore it):
 *   HIDDEN_MIX    Eq. 7 applied to the final normalised hidden state instead
 *                 of the logits: the LM head has no bias, so
 *                 W (w x + (1 - w) s) = w W x + (1 - w) W s in exact
 *                 arithmetic; the mixed row is rounded to the storage type
 *                 before the head, so results differ from logit mixing by
 *                 that rounding.  The head then runs twice, over the
 *                 candidates' shadow rows (their verification gives w) and
 *                 over the U shadow rows plus one mixed row per M position:
 *                 B rows per sequence instead of B + |M|.
 * Validation:
 *   CHECK_STATES  the steps (dard_step, dard_step_full, dard_step_shared) and
 *                 the FINAL phase of dard_commit_remask check every state
 *                 code of state_in: a sequence holding a code outside {0,1,2}
 *                 gets block_done[s] = DARD_BAD_STATE instead of 0 / 1
 *                 (block_done must then be given).  The codes themselves are
 *                 the caller's: there is no other effect on the results. */
#define DARD_F_XSELF_SHADOW   (1u << 0)
#define DARD_F_MKEYS_SHADOW   (1u << 1)
#define DARD_F_VERIFY_PCUR    (1u << 2)
#define DARD_F_PROGRESS       (1u << 3)
#define DARD_F_C_BIDIR        (1u << 4)
#define DARD_F_ORDER_L2R      (1u << 5)
#define DARD_F_ORDER_ENTROPY  (1u << 6)
#define DARD_F_ORDER_MARGIN   (1u << 7)
#define DARD_F_FIXED_W        (1u << 8)
#define DARD_F_CHECK_STATES   (1u << 9)
#define DARD_F_HIDDEN_MIX     (1u << 10)
#define DARD_F_ORDERS (DARD_F_C_BIDIR | DARD_F_ORDER_L2R | DARD_F_ORDER_ENTROPY | DARD_F_ORDER_MARGIN)
#define DARD_F_ALL    (DARD_F_XSELF_SHADOW | DARD_F_MKEYS_SHADOW | DARD_F_VERIFY_PCUR | DARD_F_PROGRESS | \
                       DARD_F_ORDERS | DARD_F_FIXED_W | DARD_F_CHECK_STATES | DARD_F_HIDDEN_MIX)

/* block_done value of a sequence whose state_in held a code outside {0,1,2}
 * (only with DARD_F_CHECK_STATES). */
#define DARD_BAD_STATE (-1)

/* Decoding hyper-parameters (Alg. 1 inputs; App. A.2 fixes lambda = 0.5^(1/8),
 * p0 = 0.1).  Requires 0 <= tau_c <= tau_u <= 1, 0 < lambda < 1, p0 > 0,
 * and 0 <= w_fixed <= 1 when DARD_F_FIXED_W is set. */
typedef struct {
    float tau_c;      /* c <= tau_c -> M                                   */
    float tau_u;      /* tau_c < c <= tau_u -> C, tau_u < c -> U (Eq. 8)    */
    double lambda;    /* geometric kernel K(i,j) = lambda^|i-j| (Eq. 5)     */
    double p0;        /* prior constant of the guidance weight (Eq. 6)     */
    int32_t mask_id;  /* token id of [Mask]                                */
    uint32_t flags;   /* DARD_F_* bits                                     */
    float w_fixed;    /* mixing weight of every M token with FIXED_W       */
} dard_params;

/* Transformer shape.  Pre-norm blocks: RMSNorm (norm_eps), rotary position
 * embedding of the rotate-half form (rope_theta), multi-head / grouped-query
 * attention, SwiGLU feed-forward, no biases, untied LM head.
 * Supported: head_dim in {64, 128}; n_heads % n_kv_heads == 0;
 * d_model == n_heads * head_dim; d_model <= 8192; bf16 needs d_model,
 * ffn_dim % 64 == 0, vocab % 16 == 0 and every weight matrix under 4 GiB
 * (vocab * d_model, 2 * ffn_dim * d_model and (n_heads + 2 n_kv_heads) *
 * head_dim * d_model values of 2 bytes); max_pos bounds prefix + block
 * positions.  Other shapes are refused with DARD_ERR_SHAPE. */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab, max_pos;
    int32_t dtype;    /* DARD_DTYPE_F32 or DARD_DTYPE_BF16 */
    float norm_eps, rope_theta;
    int32_t kv_format; /* DARD_KV_DTYPE or DARD_KV_FP8 */
} dard_dims;

/* ------------------------------------------------------------ library */
const char* dard_last_error(void);
int dard_version(void);

/* ------------------------------------------------------------ state codes
 * Validation of n token state codes (Sec. 3.2 and Eq. 8 define exactly the
 * three states M = 0, C = 1, U = 2):
 *   status[0] = number of codes outside {0, 1, 2},
 *   status[1] = index of the first of them, or -1 if there is none.
 * state: device uint8 [n] (n >= 1); status: device int32 [2], written by one
 * kernel on `stream` (no initialisation needed). */
dard_status dard_check_states(const uint8_t* state, int n, int32_t* status, void* stream);

/* ------------------------------------------------------------ a1: mask
 * State-specific attention mask of Sec. 3.2 (Eq. 2-4) for b sequences of
 * block length B (1 <= B <= 256).  By Eq. 2 every query row sees exactly one
 * of x^j and s^j, so the block part of the mask is one bit per (row, j):
 *   sel[s][r][w] (uint64, W = ceil(B/64) words per row), bit j%64 of word j/64
 *   = 1 if row r reads x^j, 0 if it reads s^j.
 * Rows r < B are the x queries of position r, rows B..2B-1 the s queries of
 * position r-B.  The prefix is always visible and not encoded.
 *   state [b][B] uint8, conf [b][B] float32 (c_{t-1}, the ordering key of
 *   Eq. 3; not read by C_BIDIR and ORDER_L2R), sel [b][2B][W] uint64.
 * flags: the mask reads XSELF_SHADOW, MKEYS_SHADOW, C_BIDIR and ORDER_L2R;
 * the other bits are accepted and ignored. */
dard_status dard_build_state_mask(const uint8_t* state, const float* conf, int b, int B,
                                  uint32_t flags, uint64_t* sel, void* stream);

/* ------------------------------------------------------------ a3: attention
 * State-masked attention over the augmented block (Sec. 3.1 "parallelized
 * inference over distinct decoding contexts", Sec. 3.2 masks):
 *   out[s][r][h] = sum_k softmax_k(scale * q[s][r][h] . k_k) v_k
 * over the visible keys of row r: the prefix keys 0..P-1, and for every block
 * position j either x^j (cache index P+j) or s^j (cache index P+B+j) as the
 * mask of dard_build_state_mask says.
 *   q   [b][2B][Hq][dh]     dtype (bf16 for DARD_DTYPE_BF16_KV_FP8)
 *   k   [b][Hkv][cap][dh]   dtype (FP8 E4M3 codes for DARD_DTYPE_BF16_KV_FP8);
 *                           keys P..P+2B-1 hold the block (x then s)
 *   v   [b][Hkv][dh][cap]   as k, dims-major (the transpose of k's layout),
 *                           so a tile of V^T is contiguous per dim
 *   out [b][2B][Hq][dh]     dtype (bf16 for DARD_DTYPE_BF16_KV_FP8)
 * Query head h reads KV head h / (Hq/Hkv).  Any permutation of the head_dim
 * axis applied to both q and k gives the same result.  Needs P >= 0,
 * P + 2B <= cap, dh in {64, 128}.
 * Workspace (device, caller-owned, no alignment beyond 256 bytes needed):
 * bf16 needs at least dard_attention_workspace_bytes(...) bytes, which hold
 * the state mask the call builds and, when the key range is split across
 * workgroups, the partial results; more room never hurts.  fp32 needs none
 * (0 is returned and ws may be NULL). */
size_t dard_attention_workspace_bytes(int dtype, int b, int B, int Hq, int dh, int P);
dard_status dard_masked_attention(int dtype, const void* q, const void* k, const void* v,
                                  int P, int cap, const uint8_t* state, const float* conf,
                                  int b, int B, int Hq, int Hkv, int dh, float scale,
                                  uint32_t flags, void* out, void* ws, size_t ws_bytes,
                                  void* stream);

/* ------------------------------------------------------------ a5/a7: confidence
 * Vocab-wide confidence reduction (Eq. 1), with the optional logit mixing of
 * Eq. 7.  For each row r:
 *   l_v = logits_s[r][v]                                  if logits_x == NULL
 *   l_v = (w[r] * logits_x[r][v]) + ((1 - w[r]) * logits_s[r][v])   otherwise,
 *         each product, the difference 1 - w and the sum rounded once in fp32
 *   argmax[r]  = first index of the largest l_v
 *   maxprob[r] = 1 / sum_v exp(l_v - l_max)              (top-1 probability)
 *   pcur[r]    = exp(l_cur - l_max) * maxprob[r], l_cur = l at cur_tok[r]
 *                (only if pcur != NULL; needs cur_tok [rows] int32, no
 *                mixing; an id outside [0, V) is clamped into it)
 *   entropy[r] = -sum_v p_v ln p_v of p = softmax(l)   (only if != NULL)
 *   margin[r]  = p_(1) - p_(2), the two largest probabilities, 0 on a tie
 *                at the top, p_(1) when V = 1          (only if != NULL)
 *   (the scores of the entropy and margin orderings of Sec. 5.1; either
 *   output being non-NULL selects the slightly longer pass that forms both)
 * logits_* rows have leading dimension ld >= V (elements, multiple of 4).
 * Outputs: argmax int32 [rows]; maxprob, pcur, entropy, margin float32 [rows]. */
size_t dard_confidence_workspace_bytes(int rows, int V);
dard_status dard_confidence(const float* logits_s, const float* logits_x, const float* w,
                            const int32_t* cur_tok, int rows, int V, int64_t ld,
                            int32_t* argmax, float* maxprob, float* pcur,
                            float* entropy, float* margin,
                            void* ws, size_t ws_bytes, void* stream);

/* dard_confidence for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and results, with the chunk partials in
 * a scratch array the library keeps in device memory (4 MiB per GPU, held
 * until the process ends) instead of a caller workspace.  It calls no
 * hipMalloc / hipFree.  Needs rows * ceil(V / 8192) * k <= 1048576 (k = 5
 * when entropy or margin is asked for, else 3): about 11000 rows at
 * V = 152064 with k = 5; larger sizes return DARD_ERR_SHAPE and launch
 * nothing.  Every call on one GPU uses that GPU's one array, so calls that
 * overlap on one GPU (other streams, other threads) race; calls ordered on
 * one stream do not.  Each call writes every partial it reads, so nothing
 * carries over from the previous call. */
dard_status dard_confidence_noalloc(const float* logits_s, const float* logits_x, const float* w,
                                    const int32_t* cur_tok, int rows, int V, int64_t ld,
                                    int32_t* argmax, float* maxprob, float* pcur,
                                    float* entropy, float* margin, void* stream);

/* ------------------------------------------------------------ a6/a8: decisions
 * Decision part of Algorithm 1 for b sequences of block length B.
 * phase DARD_PHASE_VERIFY (after the shadow confidences of the candidates):
 *   for C positions, the transition of Eq. 8 on c (maxprob_s, or pcur_s with
 *   VERIFY_PCUR) gives the promoted set P_t (-> U) and demoted set D_t (-> M);
 *   for every M position i:  P^i = sum_{j in P_t} lambda^|i-j|,
 *   D^i likewise (Eq. 5), w_out[i] = (P^i + p0) / (P^i + D^i + p0) (Eq. 6),
 *   or params.w_fixed with FIXED_W; w_out = 0 at C and U positions.  Reads
 *   state_in, maxprob_s / pcur_s.
 * phase DARD_PHASE_FINAL (after the mixed confidences of the M positions):
 *   c_i = maxprob_s (or pcur_s) for C/U positions, maxprob_mix for M;
 *   prediction x_i = argmax_s for C/U, argmax_mix for M;
 *   state_out by Eq. 8; tok_out = mask_id for next-M, x_i otherwise;
 *   conf_out = the ordering key of the next step: c_i, or with ORDER_ENTROPY
 *   / ORDER_MARGIN key_s[i] (C/U) / key_mix[i] (M), the -entropy or margin
 *   the caller formed with dard_confidence from the same rows as c_i;
 *   block_done[s] = 1 iff every position is next-U.
 * All per-position arrays are [b][B]; block_done is [b] int32.  Arrays not
 * read or written by a phase may be NULL. */
#define DARD_PHASE_VERIFY 0
#define DARD_PHASE_FINAL  1
dard_status dard_commit_remask(int phase, const dard_params* params, int b, int B,
                               const uint8_t* state_in, const float* maxprob_s,
                               const float* pcur_s, const int32_t* argmax_s,
                               const float* maxprob_mix, const int32_t* argmax_mix,
                               const float* key_s, const float* key_mix,
                               float* w_out, uint8_t* state_out, int32_t* tok_out,
                               float* conf_out, int32_t* block_done, void* stream);

/* ------------------------------------------------------------ weights and KV cache
 * The library runs on its own packed weight image.  dard_pack_weights() copies
 * the logical weights into it once (not a hot call; synchronous on `stream`).
 * src: 3 + 9 * n_layers device pointers of the storage dtype, in this order:
 *   embed [V][d];
 *   per layer: attn_norm [d], wq [Hq*dh][d], wk [Hkv*dh][d], wv [Hkv*dh][d],
 *              wo [d][Hq*dh], ffn_norm [d], w_gate [F][d], w_up [F][d],
 *              w_down [d][F];
 *   final_norm [d], lm_head [V][d].
 * The packed image also holds the rotary cos/sin table (float32).  Inside it
 * the rows of wq/wk are reordered per head so that each rotary pair (t, t+dh/2)
 * is adjacent, and the rows of w_gate/w_up interleave; the Q and K caches
 * therefore hold each head's dims in the order (0, dh/2, 1, dh/2+1, ...),
 * which leaves every attention score unchanged.
 *
 * KV cache: per layer a K block [b][Hkv][cap][dh] then a V block
 * [b][Hkv][dh][cap] (dims-major), of the storage dtype or, with
 * kv_format = DARD_KV_FP8, one byte per value (E4M3 codes), sized by
 * dard_kv_bytes().  Keys 0..P-1 hold the prefix (dard_prefill); a step writes
 * its block keys at P..P+2B-1. */
size_t dard_packed_weight_bytes(const dard_dims* dims);
dard_status dard_pack_weights(const dard_dims* dims, const void* const* src, int n_src,
                              void* packed, size_t packed_bytes, void* stream);
size_t dard_kv_bytes(const dard_dims* dims, int b, int cap);

/* ------------------------------------------------------------ a9: prefill
 * Prefix KV cache of block decoding (App. C.5, attention overhead: prefix
 * caching of system, visual and text-prompt tokens).  Runs the model over the
 * P prefix positions of each sequence with bidirectional attention among them
 * and writes K/V[0..P-1] of every layer.
 *   ids    [b][P] int32; an id < 0 takes row [s][p] of `embeds` instead
 *   embeds [b][P][d] dtype or NULL (visual tokens of a multimodal prompt). */
size_t dard_workspace_bytes(const dard_dims* dims, int b, int B, int cap);
dard_status dard_prefill(const dard_dims* dims, const void* packed, void* kv, int cap,
                         int b, int P, const int32_t* ids, const void* embeds,
                         void* ws, size_t ws_bytes, void* stream);

/* Extend-only refresh of the prefix cache at a block boundary (an
 * approximation; the exact refresh runs dard_prefill over the prompt and the
 * committed blocks again): only the Pn new positions P..P+Pn-1 of each
 * sequence -- the block just committed -- are run through the model, each of
 * their rows seeing the P cached keys of its own sequence and the Pn new
 * positions (bidirectionally among the new ones), and their K/V are written
 * at P..P+Pn-1 of every layer.  Keys 0..P-1 are read as they are, although a
 * recompute would change them from the first layer's output on (every
 * prefix position also attends to the new block); layer-0 keys are the same
 * either way.  The cost is a forward over Pn rows instead of P + Pn.
 *   ids [b][Pn] int32 token ids (no embedding rows).
 * Needs P >= 0, Pn >= 1, P + Pn <= min(cap, max_pos); kv and ws as for
 * dard_prefill with the same b and cap (ws sized by dard_workspace_bytes). */
dard_status dard_prefill_extend(const dard_dims* dims, const void* packed, void* kv, int cap,
                                int P, int b, int Pn, const int32_t* ids, void* ws, size_t ws_bytes,
                                void* stream);

/* ------------------------------------------------------------ a1-a8: one step
 * One DARD step (one loop iteration of Algorithm 1) for b sequences whose
 * current block has B positions after a prefix of P cached keys:
 *   build the augmented block (x = tok_in, s = [Mask] at the same positions),
 *   run the model under the state-specific mask (state_in, conf_in as the
 *   ordering key), take the shadow confidences of C and U tokens, verify the
 *   candidates, mix the two logit rows of every M token with its guidance
 *   weight, apply the transitions and fill the tokens.
 *   tok_in/tok_out [b][B] int32, state_in/state_out [b][B] uint8,
 *   conf_in/conf_out [b][B] float32 (the ordering key: c_i, or -entropy /
 *   margin under ORDER_ENTROPY / ORDER_MARGIN), block_done [b] int32.
 * Outputs may alias the matching inputs.  `dbg`, when not NULL, receives
 * copies of intermediate results (any member may be NULL).
 * Rows of the LM head: for a bf16 model with at most 64 rows per step
 * (b * 2B <= 64) and logit mixing, the head runs over all of them (its
 * weight-streaming kernel reads the weights once either way); otherwise
 * (fp32 models included) only over the rows the
 * decisions read -- the shadow row of every position and the x row of every
 * M position (with HIDDEN_MIX: the shadow rows of C and U positions and the
 * mixed row of every M position, which takes the M position's shadow slot).
 * dbg->logits receives exactly the rows the head ran over; the others are
 * left as they were. */
typedef struct {
    float* logits;       /* [b][2B][V]: x rows then s rows                  */
    float* w;            /* [b][B] guidance weights (0 at C/U)              */
    float* maxprob_s;    /* [b][B] shadow top-1 prob. (C/U positions)       */
    int32_t* argmax_s;   /* [b][B]                                          */
    float* pcur_s;       /* [b][B] shadow prob. of the current token (C/U)  */
    float* maxprob_mix;  /* [b][B] mixed top-1 prob. (M positions)          */
    int32_t* argmax_mix; /* [b][B]                                          */
    float* entropy;      /* [b][B] entropy of the row that gave c_i, and    */
    float* margin;       /* [b][B] its margin (ORDER_ENTROPY/MARGIN only)   */
} dard_step_debug;

dard_status dard_step(const dard_dims* dims, const void* packed, void* kv, int cap, int P,
                      const dard_params* params, int b, int B, const int32_t* tok_in,
                      const uint8_t* state_in, const float* conf_in, int32_t* tok_out,
                      uint8_t* state_out, float* conf_out, int32_t* block_done,
                      const dard_step_debug* dbg, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------ shared prompt cache
 * Batching many sequences that share one prompt (the same image and text,
 * App. C.5, attention overhead: the system, visual and text-prompt
 * tokens are prefix-cached): the prompt's cache is computed once, by
 * dard_prefill with b = 1 over the Ps prompt positions into kv_shared (a KV
 * cache of the same layout for one sequence and cap_shared keys), and every
 * sequence reads it in place of its own first Ps keys.  Reading for the
 * positions after it (each sequence's committed blocks, recomputed at a
 * block start): their rows see the shared prompt and their own positions,
 * bidirectionally among those; the prompt is not re-encoded with them.
 *   dard_prefill_suffix: positions Ps..Ps+Pc-1 of each sequence, ids
 *     [b][Pc]; writes keys Ps..Ps+Pc-1 of every layer into kv (keys below Ps
 *     of kv are never read or written).
 *   dard_step_shared: dard_step with a prefix of P >= Ps keys whose first Ps
 *     come from kv_shared.
 * Needs Ps a multiple of 64 (whole key tiles), 64 <= Ps <= cap_shared, and
 * the sizes of dard_prefill / dard_step for the per-sequence part. */
dard_status dard_prefill_suffix(const dard_dims* dims, const void* packed, void* kv, int cap,
                                const void* kv_shared, int cap_shared, int Ps, int b, int Pc,
                                const int32_t* ids, void* ws, size_t ws_bytes, void* stream);
dard_status dard_step_shared(const dard_dims* dims, const void* packed, void* kv, int cap,
                             const void* kv_shared, int cap_shared, int Ps, int P,
                             const dard_params* params, int b, int B, const int32_t* tok_in,
                             const uint8_t* state_in, const float* conf_in, int32_t* tok_out,
                             uint8_t* state_out, float* conf_out, int32_t* block_done,
                             const dard_step_debug* dbg, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------ a1-a8: full-sequence step
 * The same step without a prefix cache, in the setting of the paper's
 * single-step latency table (App. C.5, latency and memory table; the attention
 * overhead paragraph counts the shadow block as B extra queries and keys):
 * every step runs the model over the whole sequence of N positions -- prompt,
 * committed blocks, the current block at positions blk..blk+B-1 and the
 * future blocks, which hold [Mask] -- plus the current block's shadow.
 * Mask reading (the paper states the per-state rules for the current block
 * only): a query outside the current block sees the N original positions and
 * no shadow key; a query of the current block (x or s) sees every position
 * outside the block and, for each block position, x^j or s^j by the rules
 * of dard_build_state_mask.  Decisions as in dard_step.
 *   seq [b][N] int32 (the current block's tokens at blk..blk+B-1),
 *   state_in, conf_in, tok_out, state_out, conf_out, block_done as in
 *   dard_step.  Needs 1 <= B <= 256, 0 <= blk <= N - B, N + B <= cap,
 *   N <= max_pos; kv sized by dard_kv_bytes(dims, b, cap) (all N + B keys of
 *   every layer are rewritten by each call) and ws by
 *   dard_workspace_bytes(dims, b, B, cap). */
dard_status dard_step_full(const dard_dims* dims, const void* packed, void* kv, int cap, int N, int blk,
                           const dard_params* params, int b, int B, const int32_t* seq,
                           const uint8_t* state_in, const float* conf_in, int32_t* tok_out,
                           uint8_t* state_out, float* conf_out, int32_t* block_done,
                           const dard_step_debug* dbg, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------ plain linear layer
 * Y[m][n] = sum_k X[m][k] * W[n][k] in float32 (the projection GEMM of every
 * layer and the LM head, exposed for testing and measurement).
 * dard_pack_matrix() converts a row-major W [N][K] of `dtype` into the
 * library's weight layout Wp (same size; bf16: 16 x 64 blocks stored in the
 * order the matrix cores consume them, needs K % 64 == 0 and N % 16 == 0;
 * fp32: row-major copy, needs K % 4 == 0).  dard_linear() takes X [M][K] of
 * `dtype`, the packed Wp, and writes Y [M][N] float32. */
dard_status dard_pack_matrix(int dtype, const void* W, int N, int K, void* Wp, void* stream);
dard_status dard_linear(int dtype, const void* X, int M, int K, const void* Wp, int N,
                        float* Y, void* stream);

/* The kernel and tiling the library runs for a projection of M token rows,
 * N output columns and K inputs (a host-side query; nothing is launched):
 *   plan[0] = DARD_GEMM_* kernel, plan[1] x plan[2] = the workgroup tile in
 *   units of 32 rows x 32 columns (the streaming kernel: 16-column blocks
 *   per wave in plan[2]), plan[3] = workgroups splitting K.
 * partial != 0 asks for the plan of a split-K (residual) projection; step
 * and prefill activations are fragment-major (frag_x != 0), dard_linear's
 * row-major (frag_x = 0).  plan: host int32 [4]. */
#define DARD_GEMM_STREAM 0
#define DARD_GEMM_PIPE   1
#define DARD_GEMM_BIG    2
#define DARD_GEMM_TILED  3
#define DARD_GEMM_F32    4
dard_status dard_gemm_plan(int dtype, int M, int N, int K, int partial, int frag_x, int32_t* plan);

/* ------------------------------------------------------------ tracing
 * When enabled, the library brackets each launch of the kernel classes in
 * `class_mask` with HIP events on the launch stream.  dard_trace_read()
 * synchronises with those events and returns, for one class, the number of
 * launches timed and their summed duration since the last reset.  Timing
 * events cost a few microseconds per launch; dard_trace_sample(n) times only
 * every n-th launch of each traced class (counted from the last reset;
 * 1 = every launch, the default). */
#define DARD_K_GEMM_QKV   0
#define DARD_K_GEMM_O     1
#define DARD_K_GEMM_GU    2
#define DARD_K_GEMM_DOWN  3
#define DARD_K_GEMM_HEAD  4
#define DARD_K_ATTENTION  5
#define DARD_K_CONFIDENCE 6
#define DARD_K_DECIDE     7
#define DARD_K_NORM       8
#define DARD_K_MASK       9
#define DARD_K_COUNT      10
dard_status dard_trace_enable(uint32_t class_mask);
dard_status dard_trace_read(int kernel_class, int64_t* launches, double* total_ms);
dard_status dard_trace_reset(void);
dard_status dard_trace_sample(int period);

#ifdef __cplusplus
}
#endif
#endif /* DARD_H */
