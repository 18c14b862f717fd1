"""Pins of the oracle's full-sequence mode (no prefix cache): the whole
sequence, future all-[Mask] blocks included, plus the shadow block run through
the model at every step (the setting of the paper's single-step latency
table and of its attention-overhead paragraph, App. C.5).

The mode is pinned by what its reading fixes exactly: the mask against a
brute-force construction from the rules; a plain forward of the original
sequence without any shadow block, which the rows outside the current block
must reproduce for a one-layer model (no shadow key is visible to them), every
original row must reproduce without candidates at any depth, and the x and s
rows of the all-masked first step (P1) must reproduce; and, for a one-layer
model whose current block ends the sequence, equality with the prefix-cache
step (a layer-0 key depends only on its token and position).
"""
import numpy as np
import pytest

from oracle import dard_oracle as O
from paper_2608_26574_amd import synth

from test_oracle_mask import brute_force_mask


def _tiny(n_layers, dtype="f32"):
    dims = synth.Dims(n_layers, 64, 2, 2, 32, 96, 97, 512, dtype)
    return dims.as_dict(), synth.OracleWeights(dims, synth.make_weights(dims, seed=11))


def _sequence(P, blk, B, N, V, seed):
    """Prompt ids, committed ids up to blk, the current block's ids, [Mask]
    after it."""
    rng = np.random.default_rng(seed)
    seq = rng.integers(0, V - 1, (1, N)).astype(np.int32)
    seq[0, blk + B:] = V - 1
    return seq


def _states(B, seed):
    rng = np.random.default_rng(seed)
    state = rng.integers(0, 3, (1, B)).astype(np.uint8)
    conf = rng.permutation(np.linspace(0.45, 0.85, B)).astype(np.float32)[None, :]
    return state, conf


def _plain_forward(w, dims, seq):
    """The original sequence alone, every row seeing every row (vanilla
    bidirectional decoding), through the oracle's layer."""
    b, N = seq.shape
    h = O.to_f32(O.embed_rows(w, dims, seq))
    allvis = np.ones((N, N), dtype=bool)
    for layer in range(dims["n_layers"]):
        h, _ = O._layer(w["layers"][layer], dims, h, np.arange(N), None, lambda bi: allvis,
                        1.0 / np.sqrt(dims["head_dim"]))
    xn = O.storage(O.rmsnorm(h, w["final_norm"], dims["norm_eps"]), dims["dtype"])
    return O.to_f32(xn @ w["lm_head"].T)


@pytest.mark.parametrize("N,blk,B", [(20, 8, 6), (16, 10, 6), (12, 0, 4), (40, 16, 8)])
@pytest.mark.parametrize("flags", [0, O.F_MKEYS_SHADOW, O.F_ORDER_L2R])
def test_mask_matches_brute_force(N, blk, B, flags):
    state, conf = _states(B, seed=N + blk)
    vis = O.full_sequence_visible(state[0], conf[0], N, blk, flags)
    block = brute_force_mask(state[0], conf[0], 0, flags)          # [2B, 2B]: x keys, s keys
    ctx = [p for p in range(N) if not blk <= p < blk + B]
    expect = np.zeros((N + B, N + B), dtype=bool)
    for p in ctx:                                   # outside the block: the original sequence
        expect[p, :N] = True
    for i in range(B):
        for row, brow in ((blk + i, i), (N + i, B + i)):
            expect[row, ctx] = True
            expect[row, blk:blk + B] = block[brow, :B]
            expect[row, N:] = block[brow, B:]
    assert np.array_equal(vis, expect)
    # every row of the block sees exactly one of x^j, s^j (Eq. 2); no other row sees s
    assert np.all(vis[blk:blk + B, blk:blk + B] ^ vis[blk:blk + B, N:])
    assert not vis[ctx][:, N:].any()


def test_one_layer_rows_outside_the_block_are_plain_decoding():
    """No shadow key is visible to a row outside the current block, and a
    layer-0 key depends only on its token: with one layer those rows' logits
    are the plain forward's, candidates or not."""
    dims, w = _tiny(1)
    V = dims["vocab"]
    N, blk, B = 24, 8, 8
    seq = _sequence(6, blk, B, N, V, seed=1)
    state, conf = _states(B, seed=2)
    state[0, :3] = O.STATE_C
    full = O.full_step_logits(w, dims, seq, blk, B, state, conf, V - 1, all_rows=True)
    plain = _plain_forward(w, dims, seq)
    ctx = [p for p in range(N) if not blk <= p < blk + B]
    assert np.allclose(full[0, ctx], plain[0, ctx], rtol=0, atol=1e-6)
    # the block rows differ: candidates are hidden from some of them
    assert not np.allclose(full[0, blk:blk + B], plain[0, blk:blk + B], atol=1e-4)


@pytest.mark.parametrize("n_layers", [1, 2, 3])
@pytest.mark.parametrize("flags", [0, O.F_MKEYS_SHADOW])
def test_no_candidates_is_plain_decoding(n_layers, flags):
    """Without candidates every original-sequence row is the plain forward's
    at any depth: the x and s copies of an M position hold the same token and
    read the same keys, so whichever copy a row reads is the plain one (by
    induction over layers), and the shadow rows of M positions equal their x
    rows."""
    dims, w = _tiny(n_layers)
    V = dims["vocab"]
    N, blk, B = 24, 8, 8
    seq = _sequence(6, blk, B, N, V, seed=9)
    state = np.array([[0, 2, 2, 0, 0, 2, 0, 2]], dtype=np.uint8)
    seq[0, blk:blk + B][state[0] == O.STATE_M] = V - 1
    conf = np.zeros((1, B), dtype=np.float32)
    full = O.full_step_logits(w, dims, seq, blk, B, state, conf, V - 1, all_rows=True, flags=flags)
    plain = _plain_forward(w, dims, seq)
    assert np.allclose(full[0, :N], plain[0], rtol=0, atol=1e-6)
    m = [i for i in range(B) if state[0, i] == O.STATE_M]
    assert np.allclose(full[0, [N + i for i in m]], full[0, [blk + i for i in m]], rtol=0, atol=1e-6)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_p1_all_masked_block_is_plain_decoding(dtype):
    """First step of a block (every position M): x rows see the original
    sequence, so they are the plain forward's rows, and the shadow rows equal
    them (the same [Mask] tokens at the same positions, by induction)."""
    dims, w = _tiny(2, dtype)
    V = dims["vocab"]
    N, blk, B = 20, 6, 6
    seq = _sequence(6, blk, B, N, V, seed=3)
    seq[0, blk:blk + B] = V - 1
    state = np.zeros((1, B), dtype=np.uint8)
    conf = np.zeros((1, B), dtype=np.float32)
    lg = O.full_step_logits(w, dims, seq, blk, B, state, conf, V - 1)
    plain = _plain_forward(w, dims, seq)
    tol = 1e-6 if dtype == "f32" else 1e-2
    assert np.allclose(lg[0, :B], plain[0, blk:blk + B], rtol=0, atol=tol)
    assert np.allclose(lg[0, B:], lg[0, :B], rtol=0, atol=1e-6)


def test_one_layer_equals_prefix_cache_step():
    """With one layer and the current block at the end of the sequence, the
    full-sequence step and the prefix-cache step see the same keys: a layer-0
    key depends only on its token and position."""
    dims, w = _tiny(1)
    V = dims["vocab"]
    P, B = 14, 8
    seq = _sequence(P, P, B, P + B, V, seed=5)
    state, conf = _states(B, seed=6)
    tok = seq[:, P:]
    full = O.full_step_logits(w, dims, seq, P, B, state, conf, V - 1)
    cache = O.prefill(w, dims, seq[:, :P])
    cached, _ = O.step_logits(w, dims, cache, tok, state, conf, V - 1)
    assert np.allclose(full, cached, rtol=0, atol=1e-6)


def test_two_layers_differ_from_prefix_cache_step():
    """With two layers the prefix rows of the full-sequence mode also read the
    current block, so the modes differ: the one-layer equality above is not
    an accident of the construction."""
    dims, w = _tiny(2)
    V = dims["vocab"]
    P, B = 14, 8
    seq = _sequence(P, P, B, P + B, V, seed=5)
    state, conf = _states(B, seed=6)
    full = O.full_step_logits(w, dims, seq, P, B, state, conf, V - 1)
    cached, _ = O.step_logits(w, dims, O.prefill(w, dims, seq[:, :P]), seq[:, P:], state, conf, V - 1)
    assert not np.allclose(full, cached, atol=1e-5)


def test_full_step_decisions_follow_alg1():
    dims, w = _tiny(2)
    V = dims["vocab"]
    N, blk, B = 24, 8, 8
    seq = _sequence(6, blk, B, N, V, seed=7)
    state, conf = _states(B, seed=8)
    params = dict(tau_c=0.4, tau_u=0.9, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=V - 1)
    out = O.dard_step_full(w, dims, seq, blk, B, state, conf, params)
    again = O.decide(out["logits"], seq[:, blk:blk + B], state, params)
    for k in ("tok_out", "state_out", "w", "conf_out"):
        assert np.array_equal(out[k], again[k])
