"""Pins of the oracle's batch-shared prompt cache (prefill_suffix,
join_shared): the prompt's cache is computed once over the prompt alone and
shared; each sequence's committed positions see the shared prompt and their
own positions.

Checked against a single dense forward of prompt + committed positions with
the block-causal visibility that reading implies (prompt rows see the prompt,
committed rows see everything), built as one pass with a mask instead of two
passes with a broadcast cache; against the per-sequence prefill for a
one-layer model (a layer-0 key depends only on its token and position); and
shown to differ from the per-sequence prefill with two layers (where the
prompt rows of the per-sequence prefill also read the committed positions).
"""
import numpy as np
import pytest

from oracle import dard_oracle as O
from paper_2608_26574_amd import synth


def _tiny(n_layers, dtype="f32"):
    dims = synth.Dims(n_layers, 64, 2, 2, 32, 96, 97, 512, dtype)
    return dims.as_dict(), synth.OracleWeights(dims, synth.make_weights(dims, seed=12))


def _block_causal_cache(w, dims, prompt, committed):
    """One forward over prompt + committed of one sequence with the dense
    block-causal mask; per layer (K, V) of all rows."""
    Ps, Pc = prompt.shape[1], committed.shape[1]
    N = Ps + Pc
    ids = np.concatenate([prompt, committed], axis=1)
    vis = np.ones((N, N), dtype=bool)
    vis[:Ps, Ps:] = False
    h = O.to_f32(O.embed_rows(w, dims, ids))
    out = []
    for layer in range(dims["n_layers"]):
        h, kv = O._layer(w["layers"][layer], dims, h, np.arange(N), None, lambda bi: vis,
                         1.0 / np.sqrt(dims["head_dim"]))
        out.append(kv)
    return out


@pytest.mark.parametrize("n_layers", [1, 3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_suffix_matches_one_block_causal_forward(n_layers, dtype):
    dims, w = _tiny(n_layers, dtype)
    V = dims["vocab"]
    prompt = synth.prompt_ids(1, 10, V, seed=1)
    committed = synth.prompt_ids(2, 6, V, seed=2)
    shared = O.prefill(w, dims, prompt)
    suffix = O.prefill_suffix(w, dims, shared, committed)
    joined = O.join_shared(shared, suffix)
    for s in range(2):
        ref = _block_causal_cache(w, dims, prompt, committed[s:s + 1])
        for layer in range(n_layers):
            for t in range(2):
                assert np.allclose(joined[layer][t][s], ref[layer][t][0], rtol=0, atol=1e-6)


def test_one_layer_equals_per_sequence_prefill():
    dims, w = _tiny(1)
    V = dims["vocab"]
    prompt = synth.prompt_ids(1, 12, V, seed=3)
    committed = synth.prompt_ids(3, 8, V, seed=4)
    joined = O.join_shared(O.prefill(w, dims, prompt), O.prefill_suffix(w, dims, O.prefill(w, dims, prompt), committed))
    full = O.prefill(w, dims, np.concatenate([np.repeat(prompt, 3, axis=0), committed], axis=1))
    for t in range(2):
        assert np.allclose(joined[0][t], full[0][t], rtol=0, atol=1e-6)


def test_two_layers_differ_from_per_sequence_prefill():
    dims, w = _tiny(2)
    V = dims["vocab"]
    prompt = synth.prompt_ids(1, 12, V, seed=3)
    committed = synth.prompt_ids(1, 8, V, seed=4)
    shared = O.prefill(w, dims, prompt)
    joined = O.join_shared(shared, O.prefill_suffix(w, dims, shared, committed))
    full = O.prefill(w, dims, np.concatenate([prompt, committed], axis=1))
    assert not np.allclose(joined[1][0], full[1][0], atol=1e-4)


def test_empty_suffix_step_equals_duplicated_prompt_step():
    """Without committed positions (the first block) the shared cache is the
    per-sequence prefill of identical prompts, so the step is the same."""
    dims, w = _tiny(2)
    V = dims["vocab"]
    prompt = synth.prompt_ids(1, 10, V, seed=5)
    tok, state, conf = synth.tiny_block(2, 6, V, seed=6)
    shared = O.prefill(w, dims, prompt)
    joined = O.join_shared(shared, O.prefill_suffix(w, dims, shared, np.zeros((2, 0), dtype=np.int32)))
    per_seq = O.prefill(w, dims, np.repeat(prompt, 2, axis=0))
    a, _ = O.step_logits(w, dims, joined, tok, state, conf, V - 1)
    b_, _ = O.step_logits(w, dims, per_seq, tok, state, conf, V - 1)
    assert np.array_equal(a, b_)
