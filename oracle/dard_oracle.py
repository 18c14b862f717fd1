"""Plain CPU oracle for one Dependency-Aware Revocable Decoding (DARD) step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library; both sides receive the same seeded inputs and nothing else.

Everything here is written from the paper (arXiv 2608.26574) as plainly as
possible: loops or whole-array numpy expressions in float64, with a matrix
product (``@``) as the only library primitive.  No blocking, fusion or
reordering beyond what the definitions state.

Numeric conventions (the "storage rounding points").  The paper fixes no
precision, so values are accumulated in float64 and rounded to the storage type
(bfloat16, round-to-nearest-even, or float32 in the fp32 configuration) exactly
where a real implementation stores them: the embedding output, every RMSNorm
output, Q/K/V after RoPE (the KV cache), the attention output and the SwiGLU
output.  The FP8 KV-cache variant (the prefix-cache discussion of App. C.5
names the KV cache's size as the shadow block's memory cost) rounds K and V
to OCP FP8 E4M3 instead (``dims['kv_dtype'] = 'fp8'``); Q stays bf16.  The residual stream and the logits are float32.  Decisions that turn
floats into integers (argmax, threshold tests of Eq. 8, logit mixing feeding an
argmax) are taken on float32 values, the precision of the GPU kernels.

Parity pins (see ``tests/test_oracle_*.py``):
  * take_x / visible_keys   -- brute-force dense mask built from the per-state
                               prose rules of Sec. 3.2, invariants of Eq. 2-4.
  * masked_attention        -- dense textbook evaluation with -inf and torch's
                               CPU scaled_dot_product_attention.
  * rmsnorm, rope, swiglu   -- closed forms (unit RMS, norm preservation,
                               relative-position property, silu identities);
                               the FFN half of a layer against a closed form
                               with one-hot gate / up / down rows.
  * to_fp8                  -- the format's defining constants (448, 2^-6,
                               2^-9, spacing), ties to even, saturation, and
                               its relative error bound 2^-4 on normals.
  * confidence              -- closed forms (uniform row, single spike, shift
                               invariance), argmax tie rule.
  * guidance_weights        -- closed forms of Eq. 5-6 (lambda^8 = 1/2, a
                               hand-computed worked example, P4 of the tests).
  * transition              -- exact inequalities of Eq. 8.
  * ordering / mixing variants of Sec. 5.1 (F_C_BIDIR, F_ORDER_*, F_FIXED_W)
                            -- equivalences with the primary mask (all keys
                               tied; keys = -position), closed forms of entropy
                               and margin, scipy's entropy, exact float32
                               identities of Eq. 7 at w in {0, 1/2, 1}.
  * shared prompt cache (prefill_suffix, join_shared)
                            -- a dense block-causal forward of prompt +
                               committed positions, one-layer equality with
                               the per-sequence prefill, and the batch-shared
                               cache equal to per-sequence caches of equal
                               prompts.
  * full-sequence mode (no prefix cache; full_step_logits)
                            -- one-layer equality with the prefix-cache step,
                               a plain forward without the shadow block (rows
                               outside the block at one layer, every original
                               row without candidates, P1), and a brute-force
                               mask from the rules.
  * step_logits / prefill   -- special cases P1 (all-M block), P2 (empty C) and
                               P3 (one-layer independence from C tokens); the
                               full multi-layer logits beyond these cases are
                               "parity unpinned" (no published values exist).
"""
from __future__ import annotations

import math

import numpy as np

# Token state codes (Sec. 3.2): masked, candidate, unmasked.
STATE_M, STATE_C, STATE_U = 0, 1, 2

# Flags selecting the alternative readings of points the paper leaves open.
F_XSELF_SHADOW = 1 << 0   # x-row of a U token does not see its own x key
F_MKEYS_SHADOW = 1 << 1   # x-row of an M token sees M keys through s
F_VERIFY_PCUR = 1 << 2    # C/U confidence = prob. of the current token
F_PROGRESS = 1 << 3       # driver rule: every step of an unfinished block commits >= 1 token
# Variants of the design-choice analysis (Sec. 5.1, mask-design and mixing
# ablations).  At most one of the four ordering flags may be set.
F_C_BIDIR = 1 << 4        # candidates see every candidate (no ordering)
F_ORDER_L2R = 1 << 5      # candidates ordered by position, left first
F_ORDER_ENTROPY = 1 << 6  # ... by entropy of the prediction, lowest first
F_ORDER_MARGIN = 1 << 7   # ... by top-1 minus top-2 probability, largest first
F_FIXED_W = 1 << 8        # every M token mixes with the constant w_fixed
F_CHECK_STATES = 1 << 9   # library-side validation of state codes (no effect on the arithmetic)
F_HIDDEN_MIX = 1 << 10    # library-side evaluation order of Eq. 7 (the oracle mixes logits)
F_ORDERS = F_C_BIDIR | F_ORDER_L2R | F_ORDER_ENTROPY | F_ORDER_MARGIN

LAMBDA_DEFAULT = 0.5 ** (1.0 / 8.0)   # App. A.2: lambda = 0.917, i.e. 0.5^(1/8)
P0_DEFAULT = 0.1                      # App. A.2: prior constant p_0


# --------------------------------------------------------------------------
# storage rounding
# --------------------------------------------------------------------------
def to_f32(x):
    """Round to IEEE binary32 (round-to-nearest-even) and return float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def to_bf16(x):
    """Round to bfloat16 (round-to-nearest-even on the binary32 bit pattern).

    bfloat16 keeps the upper 16 bits of a binary32 number; ties go to the even
    upper half.  The value is first rounded to binary32, as a kernel holding a
    float32 accumulator does.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# The finite non-negative values of the OCP 8-bit floating-point format E4M3
# (4 exponent bits, bias 7, 3 mantissa bits; no infinities, the all-ones
# pattern is NaN): code c = 8 e + m is m/8 * 2^-6 for e = 0 (subnormal) and
# (1 + m/8) * 2^(e-7) otherwise, for c = 0 .. 126.  The largest is 448.
E4M3_VALUES = np.array([(m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
                        for e in range(16) for m in range(8)][:127])


def to_fp8(x):
    """Round to OCP FP8 E4M3 (round to nearest, ties to the even code, i.e. the
    one whose last mantissa bit is 0; magnitudes beyond 448 saturate to 448),
    after rounding to binary32 as a kernel holding a float32 value does.
    Returns float64 values of the format."""
    a = np.abs(np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64))
    sign = np.sign(np.asarray(x, dtype=np.float64))
    hi = np.clip(np.searchsorted(E4M3_VALUES, a), 1, 126)     # E4M3_VALUES[hi - 1] <= a <= E4M3_VALUES[hi]
    lo = hi - 1
    below, above = E4M3_VALUES[lo], E4M3_VALUES[hi]
    take_hi = (a - below > above - a) | ((a - below == above - a) & (hi % 2 == 0))
    code = np.where(take_hi, hi, lo)
    code = np.where(a >= E4M3_VALUES[126], 126, code)           # saturation at 448
    return sign * E4M3_VALUES[code]


def storage(x, dtype):
    """Round to a storage type: 'bf16', 'f32', or 'fp8' (OCP E4M3, the KV cache
    format of the fp8 variant)."""
    if dtype == "bf16":
        return to_bf16(x)
    if dtype == "f32":
        return to_f32(x)
    if dtype == "fp8":
        return to_fp8(x)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# state-specific attention mask (Sec. 3.1 "parallelized inference", Eq. 2-3,
# Sec. 3.2 paragraphs on U, C and M tokens)
# --------------------------------------------------------------------------
def take_x(state, conf, flags=0):
    """Return X[r, j] (bool, shape [2B, B]): row r sees x^j (True) or s^j.

    Rows 0..B-1 are the queries of the original block x, rows B..2B-1 those of
    the shadow block s; row r belongs to position i = r mod B.  Eq. 2 demands
    that each query sees exactly one of x^j and s^j, so one boolean per
    (row, position) describes the whole block part of the mask; the prefix is
    always visible.

    Per query state (Sec. 3.2):
      U  -- sees the U tokens in x, everything else in s; the shadow query s^i
            never sees its own x^i (leakage block).  The x query uses the same
            pattern; it keeps its own x^i unless F_XSELF_SHADOW.
      C  -- sees U in x and, by Eq. 3, the C tokens j with c_i <= c_j in x
            (itself included); the shadow query drops its own x^i (Eq. 4
            conditions the k-th candidate on the k-1 more confident ones only).
            Variants of Sec. 5.1: F_C_BIDIR takes every C token from x;
            F_ORDER_L2R takes the C tokens j <= i (position order replaces
            confidence order).  Entropy and margin orderings keep this rule
            and change the key passed as ``conf`` (see ``order_key``).
      M  -- the x query sees C and U in x; M keys are taken from x as well
            (vanilla decoding of the x stream) unless F_MKEYS_SHADOW, which
            takes them from s except its own position.  The shadow query sees
            U in x and C in s ("C regarded as masked"); M keys from s.
    """
    state = np.asarray(state)
    conf = np.asarray(conf, dtype=np.float32)
    B = state.shape[0]
    X = np.zeros((2 * B, B), dtype=bool)
    for r in range(2 * B):
        i = r % B
        shadow = r >= B
        si = state[i]
        for j in range(B):
            sj = state[j]
            if si == STATE_U:
                vis = sj == STATE_U
                if j == i and (shadow or (flags & F_XSELF_SHADOW)):
                    vis = False
            elif si == STATE_C:
                if flags & F_C_BIDIR:
                    before = True
                elif flags & F_ORDER_L2R:
                    before = j <= i
                else:
                    before = conf[i] <= conf[j]
                vis = sj == STATE_U or (sj == STATE_C and before)
                if j == i and shadow:
                    vis = False
            elif si == STATE_M:
                if shadow:
                    vis = sj == STATE_U
                elif flags & F_MKEYS_SHADOW:
                    vis = sj in (STATE_C, STATE_U) or j == i
                else:
                    vis = True
            else:
                raise ValueError("state code out of range")
            X[r, j] = vis
    return X


def visible_keys(state, conf, P, flags=0):
    """Dense mask [2B, P + 2B]: prefix keys, then x^0..x^{B-1}, then s^0..s^{B-1}."""
    X = take_x(state, conf, flags)
    R, B = X.shape
    vis = np.zeros((R, P + 2 * B), dtype=bool)
    vis[:, :P] = True
    vis[:, P:P + B] = X
    vis[:, P + B:] = ~X
    return vis


# --------------------------------------------------------------------------
# transformer pieces (the paper's models are LLaDA / MMaDA-like; the internals
# used here are the common pre-norm RMSNorm / RoPE / SwiGLU block)
# --------------------------------------------------------------------------
def rmsnorm(h, gain, eps):
    """y = h / sqrt(mean(h^2) + eps) * gain, over the last axis."""
    h = np.asarray(h, dtype=np.float64)
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps) * gain


def rope(x, pos, theta):
    """Rotate-half rotary embedding.  x: [..., rows, heads, dh], pos: [rows].

    Dimension t < dh/2 is paired with t + dh/2 and both are rotated by the angle
    pos * theta^(-2t/dh).
    """
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    t = np.arange(half, dtype=np.float64)
    inv = theta ** (-2.0 * t / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]   # [rows, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def masked_attention(q, k, v, visible, scale, n_kv_heads):
    """Softmax attention restricted to the visible keys, in float64.

    q: [R, Hq, dh]; k, v: [Nk, Hkv, dh]; visible: bool [R, Nk].
    o[r, h] = sum_k softmax_k(q.k / sqrt(dh) over visible k) v_k.
    Query head h reads KV head h // (Hq / Hkv).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    R, Hq, dh = q.shape
    group = Hq // n_kv_heads
    out = np.zeros((R, Hq, dh))
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) * scale          # [R, Nk]
        s = np.where(visible, s, -np.inf)
        m = np.max(s, axis=1, keepdims=True)
        p = np.exp(s - m)
        p = p / np.sum(p, axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


# --------------------------------------------------------------------------
# forward passes
# --------------------------------------------------------------------------
def _layer(w, dims, h, pos, kv_prefix, visible_fn, scale):
    """One pre-norm block over the rows of every sequence.

    h: [b, R, d] residual (float32 values); pos: [R] absolute positions.
    kv_prefix: (K, V) each [b, P, Hkv, dh] or None.  visible_fn(bi) -> bool
    [R, P + R] mask over (prefix keys, the rows' own keys).
    Returns the new residual and this layer's (K, V) of the rows.
    """
    dt = dims["dtype"]
    kvdt = dims.get("kv_dtype") or dt      # the KV cache's storage type (the fp8 variant: 'fp8')
    Hq, Hkv, dh = dims["n_heads"], dims["n_kv_heads"], dims["head_dim"]
    b, R, d = h.shape
    xn = storage(rmsnorm(h, w["attn_norm"], dims["norm_eps"]), dt)
    q = (xn @ w["wq"].T).reshape(b, R, Hq, dh)
    k = (xn @ w["wk"].T).reshape(b, R, Hkv, dh)
    v = (xn @ w["wv"].T).reshape(b, R, Hkv, dh)
    q = storage(rope(q, pos, dims["rope_theta"]), dt)
    k = storage(rope(k, pos, dims["rope_theta"]), kvdt)
    v = storage(v, kvdt)
    att = np.zeros((b, R, Hq, dh))
    for bi in range(b):
        if kv_prefix is not None:
            kk = np.concatenate([kv_prefix[0][bi], k[bi]], axis=0)
            vv = np.concatenate([kv_prefix[1][bi], v[bi]], axis=0)
        else:
            kk, vv = k[bi], v[bi]
        att[bi] = masked_attention(q[bi], kk, vv, visible_fn(bi), scale, Hkv)
    att = storage(att, dt).reshape(b, R, Hq * dh)
    h = to_f32(h + att @ w["wo"].T)
    xn = storage(rmsnorm(h, w["ffn_norm"], dims["norm_eps"]), dt)
    act = storage(silu(xn @ w["w_gate"].T) * (xn @ w["w_up"].T), dt)
    h = to_f32(h + act @ w["w_down"].T)
    return h, (k, v)


def embed_rows(weights, dims, ids, embeds=None):
    """Token embedding lookup; ids < 0 take the row of ``embeds`` instead
    (visual prefix positions of a multimodal prompt)."""
    ids = np.asarray(ids)
    out = np.zeros(ids.shape + (dims["d_model"],))
    tok = ids >= 0
    out[tok] = weights["embed"][ids[tok]]
    if (~tok).any():
        out[~tok] = np.asarray(embeds, dtype=np.float64)[~tok]
    return storage(out, dims["dtype"])


def prefill(weights, dims, ids, embeds=None):
    """Prefix cache of block decoding (App. C.5, attention overhead of the
    shadow sequence: prefix caching).  The prefix tokens attend
    bidirectionally to each other only.

    ids: [b, P] (negative = take ``embeds[b, p]``).  Returns a list over layers
    of (K, V), each [b, P, Hkv, dh], rounded to the storage type.
    """
    ids = np.asarray(ids)
    b, P = ids.shape
    h = to_f32(embed_rows(weights, dims, ids, embeds))
    pos = np.arange(P)
    scale = 1.0 / math.sqrt(dims["head_dim"])
    allvis = np.ones((P, P), dtype=bool)
    cache = []
    for layer in range(dims["n_layers"]):
        h, kv = _layer(weights["layers"][layer], dims, h, pos, None,
                       lambda bi: allvis, scale)
        cache.append(kv)
    return cache


def prefill_suffix(weights, dims, shared, ids, embeds=None):
    """Per-sequence part of a prefix cache whose first Ps positions are shared
    by the whole batch (the same image and prompt for every sequence).

    The paper caches the system, visual and text-prompt tokens (App. C.5, on the
    attention overhead); with one prompt for the batch that cache is computed
    once, over the prompt alone (``prefill`` with b = 1), and shared.  Reading
    for the positions after it (each sequence's committed blocks, recomputed at
    a block start): their rows see the shared prompt and their own positions,
    bidirectionally among those.

    shared: per layer (K, V) of the prompt, each [1, Ps, Hkv, dh].
    ids: [b, Pc] ids of the positions Ps..Ps+Pc-1.  Returns per layer (K, V),
    each [b, Pc, Hkv, dh].
    """
    ids = np.asarray(ids)
    b, Pc = ids.shape
    Ps = shared[0][0].shape[1] if dims["n_layers"] > 0 else 0
    h = to_f32(embed_rows(weights, dims, ids, embeds))
    pos = Ps + np.arange(Pc)
    scale = 1.0 / math.sqrt(dims["head_dim"])
    allvis = np.ones((Pc, Ps + Pc), dtype=bool)
    cache = []
    for layer in range(dims["n_layers"]):
        kv_sh = tuple(np.broadcast_to(t, (b,) + t.shape[1:]) for t in shared[layer])
        h, kv = _layer(weights["layers"][layer], dims, h, pos, kv_sh, lambda bi: allvis, scale)
        cache.append(kv)
    return cache


def prefill_extend(weights, dims, cache, ids):
    """Extend-only refresh of a per-sequence prefix cache at a block boundary
    (an approximation of the refresh at a block start, whose exact form is
    ``prefill`` over the prompt and the committed blocks; prefix caching is
    App. C.5, attention overhead): only the new positions P..P+Pn-1 of each
    sequence go through the model, each of their rows seeing the sequence's
    P cached keys and the new positions, bidirectionally among those; the
    cached keys are kept as they are.

    cache: per layer (K, V) of the prefix, each [b, P, Hkv, dh].  ids: [b, Pn].
    Returns per layer (K, V) of the extended prefix, each [b, P + Pn, Hkv, dh].
    """
    ids = np.asarray(ids)
    b, Pn = ids.shape
    P = cache[0][0].shape[1] if dims["n_layers"] > 0 else 0
    h = to_f32(embed_rows(weights, dims, ids))
    pos = P + np.arange(Pn)
    scale = 1.0 / math.sqrt(dims["head_dim"])
    allvis = np.ones((Pn, P + Pn), dtype=bool)
    out = []
    for layer in range(dims["n_layers"]):
        h, (k, v) = _layer(weights["layers"][layer], dims, h, pos, cache[layer], lambda bi: allvis, scale)
        out.append((np.concatenate([cache[layer][0], k], axis=1), np.concatenate([cache[layer][1], v], axis=1)))
    return out


def join_shared(shared, suffix):
    """Per-sequence prefix cache [b, Ps + Pc] from the shared prompt's cache
    (broadcast over the batch) followed by each sequence's suffix."""
    out = []
    for (ks, vs), (kc, vc) in zip(shared, suffix):
        b = kc.shape[0]
        out.append((np.concatenate([np.broadcast_to(ks, (b,) + ks.shape[1:]), kc], axis=1),
                    np.concatenate([np.broadcast_to(vs, (b,) + vs.shape[1:]), vc], axis=1)))
    return out


def step_logits(weights, dims, cache, tok, state, conf, mask_id, flags=0):
    """Forward over the augmented block (x; s) of one DARD step (Alg. 1:
    construct the augmented input, build the mask, run the model).

    cache: per layer (K, V) of the prefix, each [b, P, Hkv, dh].
    tok, state, conf: [b, B].  x^i embeds tok[i]; every s^i embeds [Mask].
    x^i and s^i share the position P + i (Sec. 3.1).  Returns float32-valued
    logits [b, 2B, V] (rows 0..B-1 from x, B..2B-1 from s) and the block's
    per-layer (K, V).
    """
    tok = np.asarray(tok)
    state = np.asarray(state)
    conf = np.asarray(conf, dtype=np.float32)
    b, B = tok.shape
    P = cache[0][0].shape[1] if dims["n_layers"] > 0 else 0
    ids = np.concatenate([tok, np.full((b, B), mask_id, dtype=tok.dtype)], axis=1)
    h = to_f32(embed_rows(weights, dims, ids))
    pos = P + np.concatenate([np.arange(B), np.arange(B)])
    scale = 1.0 / math.sqrt(dims["head_dim"])
    masks = [visible_keys(state[bi], conf[bi], P, flags) for bi in range(b)]
    block_kv = []
    for layer in range(dims["n_layers"]):
        h, kv = _layer(weights["layers"][layer], dims, h, pos, cache[layer],
                       lambda bi: masks[bi], scale)
        block_kv.append(kv)
    xn = storage(rmsnorm(h, weights["final_norm"], dims["norm_eps"]), dims["dtype"])
    logits = to_f32(xn @ weights["lm_head"].T)
    return logits, block_kv


def full_sequence_visible(state, conf, N, blk, flags=0):
    """Dense mask of the full-sequence mode (no prefix cache): rows and keys
    are the N positions of the whole sequence (prompt, committed blocks, the
    current block x at blk..blk+B-1, future all-[Mask] blocks) followed by the
    B shadow positions s.  Returns bool [N + B, N + B].

    The paper gives the per-state rules of Sec. 3.2 for the current block and
    its shadow only; this mode reads the rest as plain bidirectional decoding
    of the original sequence (App. C.5, on the attention overhead, counts
    the shadow block as B extra queries and keys on top of it):
      * a query outside the current block sees the N original positions and
        no shadow key (the shadow exists for verifying the current block);
      * a query of the current block (x^i or s^i) sees every position outside
        the current block, and for each block position j exactly one of x^j
        and s^j, chosen by the state rules (``take_x``).
    """
    X = take_x(state, conf, flags)
    B = X.shape[1]
    vis = np.zeros((N + B, N + B), dtype=bool)
    ctx = np.ones(N, dtype=bool)
    ctx[blk:blk + B] = False
    for r in range(N):
        if ctx[r]:
            vis[r, :N] = True
    for i in range(B):
        for row, xrow in ((blk + i, i), (N + i, B + i)):
            vis[row, :N] = ctx
            vis[row, blk:blk + B] = X[xrow]
            vis[row, N:] = ~X[xrow]
    return vis


def full_step_logits(weights, dims, seq, blk, B, state, conf, mask_id, flags=0, all_rows=False):
    """One DARD step in full-sequence mode: the model runs over the whole
    sequence plus the shadow block, every step, without a prefix cache (the
    setting of the paper's single-step latency table).

    seq: [b, N] token ids of the whole sequence, the current block's tokens
    at blk..blk+B-1 and [Mask] in future blocks.  The shadow block embeds
    [Mask] at the positions of the current block.  Returns float32-valued
    logits [b, 2B, V] (x rows of the current block, then its s rows), or with
    all_rows the logits of all N + B rows.
    """
    seq = np.asarray(seq)
    state = np.asarray(state)
    conf = np.asarray(conf, dtype=np.float32)
    b, N = seq.shape
    ids = np.concatenate([seq, np.full((b, B), mask_id, dtype=seq.dtype)], axis=1)
    h = to_f32(embed_rows(weights, dims, ids))
    pos = np.concatenate([np.arange(N), blk + np.arange(B)])
    scale = 1.0 / math.sqrt(dims["head_dim"])
    masks = [full_sequence_visible(state[bi], conf[bi], N, blk, flags) for bi in range(b)]
    for layer in range(dims["n_layers"]):
        h, _ = _layer(weights["layers"][layer], dims, h, pos, None, lambda bi: masks[bi], scale)
    xn = storage(rmsnorm(h, weights["final_norm"], dims["norm_eps"]), dims["dtype"])
    logits = to_f32(xn @ weights["lm_head"].T)
    if all_rows:
        return logits
    rows = np.concatenate([blk + np.arange(B), N + np.arange(B)])
    return logits[:, rows]


def dard_step_full(weights, dims, seq, blk, B, state, conf, params):
    """A DARD step in full-sequence mode: the forward above, then the same
    decisions (Alg. 1) on the current block's 2B logit rows."""
    tok = np.asarray(seq)[:, blk:blk + B]
    logits = full_step_logits(weights, dims, seq, blk, B, state, conf, params["mask_id"], params.get("flags", 0))
    out = decide(logits, tok, state, params)
    out["logits"] = logits
    return out


# --------------------------------------------------------------------------
# confidence, guidance weight, transitions (Eq. 1, 5-8, Alg. 1)
# --------------------------------------------------------------------------
def confidence(row, cur_tok=None):
    """Eq. 1: prediction = argmax of the distribution, confidence = its top-1
    probability.  Returns (argmax, maxprob, prob of cur_tok) with the argmax
    taken on the given (float32) logits, the lowest index winning ties, and
    the probabilities in float64."""
    row = np.asarray(row, dtype=np.float64)
    a = int(np.argmax(row))                    # first maximal index
    m = row[a]
    z = np.sum(np.exp(row - m))
    pc = math.exp(row[cur_tok] - m) / z if cur_tok is not None else float("nan")
    return a, 1.0 / z, pc


def entropy_margin(row):
    """Entropy and margin of the distribution softmax(row), the scores of the
    entropy and margin orderings of Sec. 5.1 (mask-design analysis):
    H = -sum_v p_v ln p_v (natural log, 0 ln 0 = 0) and margin = p_(1) - p_(2),
    the two largest probabilities (p_(2) = 0 for a one-entry row).  Both in
    float64 from the given (float32) logits."""
    row = np.asarray(row, dtype=np.float64)
    e = np.exp(row - np.max(row))
    p = e / np.sum(e)
    nz = p > 0
    H = -float(np.sum(p[nz] * np.log(p[nz])))
    top = np.sort(p)[::-1]
    second = top[1] if len(top) > 1 else 0.0
    return H, float(top[0] - second)


def order_key(c, H, margin, flags):
    """The per-position key that Eq. 3 compares (larger = earlier in the
    verification chain) under the ordering the flags select: the confidence c
    (the paper's), -H (lowest entropy first) or the margin (largest first).
    float32 value, the type the key is stored in."""
    if flags & F_ORDER_ENTROPY:
        return float(np.float32(-H))
    if flags & F_ORDER_MARGIN:
        return float(np.float32(margin))
    return float(np.float32(c))


def mix_logits(lx, ls, w):
    """Eq. 7: w * logit(x) + (1 - w) * logit(s), evaluated in float32 as
    (w * lx) + ((1 - w) * ls), each operation rounded once."""
    w = np.float32(w)
    lx = np.asarray(lx, dtype=np.float32)
    ls = np.asarray(ls, dtype=np.float32)
    return (w * lx) + ((np.float32(1.0) - w) * ls)


def guidance_weights(promoted, demoted, lam, p0):
    """Eq. 5-6 for every position i of the block.

    promoted, demoted: bool [B] (the sets P_t and D_t).  Returns float64
    arrays (P^i, D^i, w^i) with P^i = sum_{j in P_t} lam^|i-j|, D^i likewise,
    w^i = (P^i + p0) / (P^i + D^i + p0).
    """
    B = len(promoted)
    Pi = np.zeros(B)
    Di = np.zeros(B)
    for i in range(B):
        for j in range(B):
            kern = lam ** abs(i - j)
            if promoted[j]:
                Pi[i] += kern
            if demoted[j]:
                Di[i] += kern
    return Pi, Di, (Pi + p0) / (Pi + Di + p0)


def transition(c, tau_c, tau_u):
    """Eq. 8 on float32 values: c <= tau_c -> M, c <= tau_u -> C, else U."""
    c = np.float32(c)
    if c <= np.float32(tau_c):
        return STATE_M
    if c <= np.float32(tau_u):
        return STATE_C
    return STATE_U


def verify_candidates(state, c, params):
    """Update of the C tokens in Alg. 1 and the guidance weights of the M
    tokens (Eq. 5-6).  state, c: [B] (c = confidence of the C tokens, float32
    values).  Returns (next state of C tokens or -1, promoted, demoted, w) with
    w = 0 at C and U positions and w rounded to float32."""
    B = len(state)
    nxt = np.full(B, -1, dtype=np.int64)
    promoted = np.zeros(B, dtype=bool)
    demoted = np.zeros(B, dtype=bool)
    for i in range(B):
        if state[i] == STATE_C:
            nxt[i] = transition(c[i], params["tau_c"], params["tau_u"])
            promoted[i] = nxt[i] == STATE_U
            demoted[i] = nxt[i] == STATE_M
    _, _, w = guidance_weights(promoted, demoted, params["lam"], params["p0"])
    if params.get("flags", 0) & F_FIXED_W:
        # mixing ablation of Sec. 5.1: one constant weight replaces Eq. 5-6
        w = np.full(B, float(params["w_fixed"]))
    w = np.where(np.asarray(state) == STATE_M, w, 0.0).astype(np.float32).astype(np.float64)
    return nxt, promoted, demoted, w


def finalize(c, xhat, params, state_in=None):
    """Transition of every position by Eq. 8 and the fill rule: next-M
    positions hold [Mask], the others their prediction.  c, xhat: [B].

    With F_PROGRESS (a driver rule, not the paper's: Alg. 1 assumes that
    confidences eventually exceed tau_u), a step of an unfinished block in
    which no position entered U promotes the most confident position that
    is not U after the transitions (ties: lowest position) to U with its
    prediction, so every step commits at least one token."""
    B = len(c)
    st = np.array([transition(c[i], params["tau_c"], params["tau_u"]) for i in range(B)], dtype=np.int64)
    if params.get("flags", 0) & F_PROGRESS and state_in is not None:
        entered = (st == STATE_U) & (np.asarray(state_in) != STATE_U)
        if not entered.any() and not np.all(st == STATE_U):
            cand = [i for i in range(B) if st[i] != STATE_U]
            best = max(cand, key=lambda i: (np.float32(c[i]), -i))
            st[best] = STATE_U
    tok = np.where(st == STATE_M, params["mask_id"], np.asarray(xhat, dtype=np.int64))
    return st, tok, np.asarray(c, dtype=np.float64), int(np.all(st == STATE_U))


def decide(logits, tok, state, params):
    """The decision part of one loop iteration of Alg. 1 for every sequence.

    logits: [b, 2B, V] float32 values (x rows then s rows).
    params: dict with tau_c, tau_u, lam, p0, mask_id, flags (and w_fixed
    with F_FIXED_W).  conf_out is the key the next step's mask orders the
    candidates by: the confidence, or with F_ORDER_ENTROPY / F_ORDER_MARGIN
    the negated entropy / the margin of the same row.
    Returns a dict of per-position arrays: tok_out, state_out, conf_out,
    block_done, w, and the intermediate argmax / confidences.
    """
    logits = np.asarray(logits, dtype=np.float32)
    tok = np.asarray(tok)
    state = np.asarray(state)
    b, B = tok.shape
    flags = params.get("flags", 0)
    out = {k: np.zeros((b, B), dtype=np.float64) for k in
           ("w", "conf_out", "maxprob_s", "pcur_s", "maxprob_mix", "entropy", "margin")}
    out.update({k: np.zeros((b, B), dtype=np.int64) for k in
                ("tok_out", "state_out", "argmax_s", "argmax_mix")})
    out["block_done"] = np.zeros(b, dtype=np.int64)
    for bi in range(b):
        xhat = np.zeros(B, dtype=np.int64)
        c = np.zeros(B)
        key = np.zeros(B)
        # confidences of C and U tokens from the shadow stream
        for i in range(B):
            a, mp, pc = confidence(logits[bi, B + i], int(tok[bi, i]))
            out["argmax_s"][bi, i] = a
            out["maxprob_s"][bi, i] = np.float32(mp)
            out["pcur_s"][bi, i] = np.float32(pc)
            if state[bi, i] in (STATE_C, STATE_U):
                xhat[i] = a
                c[i] = np.float32(pc if flags & F_VERIFY_PCUR else mp)
                if flags & (F_ORDER_ENTROPY | F_ORDER_MARGIN):
                    H, mg = entropy_margin(logits[bi, B + i])
                    out["entropy"][bi, i], out["margin"][bi, i] = np.float32(H), np.float32(mg)
                    key[i] = order_key(c[i], H, mg, flags)
                else:
                    key[i] = c[i]
        # update the C tokens; promoted / demoted sets; weights of M tokens
        _, _, _, w = verify_candidates(state[bi], c, params)
        out["w"][bi] = w
        # decode the M tokens with logit mixing
        for i in range(B):
            if state[bi, i] == STATE_M:
                mixed = mix_logits(logits[bi, i], logits[bi, B + i], w[i])
                a, mp, _ = confidence(mixed)
                out["argmax_mix"][bi, i] = a
                out["maxprob_mix"][bi, i] = np.float32(mp)
                xhat[i] = a
                c[i] = np.float32(mp)
                if flags & (F_ORDER_ENTROPY | F_ORDER_MARGIN):
                    H, mg = entropy_margin(mixed)
                    out["entropy"][bi, i], out["margin"][bi, i] = np.float32(H), np.float32(mg)
                    key[i] = order_key(c[i], H, mg, flags)
                else:
                    key[i] = c[i]
        # transitions of all tokens (C ones repeat the rule above) and fill
        st, tk, cf, done = finalize(c, xhat, params, state[bi])
        out["state_out"][bi] = st
        out["tok_out"][bi] = tk
        # the key the next step's mask orders candidates by (Eq. 3): the
        # confidence itself unless an entropy or margin ordering is selected
        out["conf_out"][bi] = key
        out["block_done"][bi] = done
    return out


def dard_step(weights, dims, cache, tok, state, conf, params):
    """One DARD step (one iteration of the loop of Alg. 1)."""
    logits, _ = step_logits(weights, dims, cache, tok, state, conf,
                            params["mask_id"], params.get("flags", 0))
    out = decide(logits, tok, state, params)
    out["logits"] = logits
    return out
