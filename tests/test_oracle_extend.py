"""Pins of the oracle's extend-only prefix-cache refresh (prefill_extend):
at a block boundary only the new positions run through the model, their rows
seeing the sequence's cached keys and each other, and the cached keys stay.

Checked against one dense forward over prefix + new positions with the
block-causal visibility that reading implies (prefix rows see the prefix only,
new rows see everything), built with a mask in one pass instead of a cache
and a second pass; against the full prefill for a one-layer model (a layer-0
key depends only on its token and position); shown to differ from the full
prefill with two layers (where the prefix rows also read the new positions);
and chained over several blocks, each sequence with its own prefix.
"""
import numpy as np
import pytest

from oracle import dard_oracle as O
from paper_2608_26574_amd import synth


def _tiny(n_layers, dtype="f32"):
    dims = synth.Dims(n_layers, 64, 2, 2, 32, 96, 97, 512, dtype)
    return dims.as_dict(), synth.OracleWeights(dims, synth.make_weights(dims, seed=14))


def _block_causal(w, dims, ids, cuts):
    """One forward over ids [1, N] where the rows before each cut see only the
    positions before that cut (prefix and earlier blocks) and the rows of a
    block see everything up to its end; per layer (K, V)."""
    N = ids.shape[1]
    vis = np.zeros((N, N), dtype=bool)
    starts = [0] + list(cuts)
    ends = list(cuts) + [N]
    for a, e in zip(starts, ends):
        vis[a:e, :e] = True
    h = O.to_f32(O.embed_rows(w, dims, ids))
    out = []
    for layer in range(dims["n_layers"]):
        h, kv = O._layer(w["layers"][layer], dims, h, np.arange(N), None, lambda bi: vis,
                         1.0 / np.sqrt(dims["head_dim"]))
        out.append(kv)
    return out


@pytest.mark.parametrize("n_layers", [1, 3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_extend_matches_one_block_causal_forward(n_layers, dtype):
    dims, w = _tiny(n_layers, dtype)
    V = dims["vocab"]
    prefix = synth.prompt_ids(2, 9, V, seed=1)
    blocks = [synth.prompt_ids(2, 5, V, seed=2), synth.prompt_ids(2, 4, V, seed=3)]
    cache = O.prefill(w, dims, prefix)
    for blk in blocks:
        cache = O.prefill_extend(w, dims, cache, blk)
    for s in range(2):
        ids = np.concatenate([prefix[s:s + 1]] + [blk[s:s + 1] for blk in blocks], axis=1)
        ref = _block_causal(w, dims, ids, (9, 14))
        for layer in range(n_layers):
            for t in range(2):
                assert cache[layer][t].shape[1] == 18
                assert np.allclose(cache[layer][t][s], ref[layer][t][0], rtol=0, atol=1e-6)


def test_one_layer_equals_full_prefill():
    dims, w = _tiny(1)
    V = dims["vocab"]
    prefix = synth.prompt_ids(3, 12, V, seed=4)
    blk = synth.prompt_ids(3, 8, V, seed=5)
    ext = O.prefill_extend(w, dims, O.prefill(w, dims, prefix), blk)
    full = O.prefill(w, dims, np.concatenate([prefix, blk], axis=1))
    for t in range(2):
        assert np.allclose(ext[0][t], full[0][t], rtol=0, atol=1e-6)


def test_two_layers_differ_from_full_prefill():
    dims, w = _tiny(2)
    V = dims["vocab"]
    prefix = synth.prompt_ids(1, 12, V, seed=4)
    blk = synth.prompt_ids(1, 8, V, seed=5)
    ext = O.prefill_extend(w, dims, O.prefill(w, dims, prefix), blk)
    full = O.prefill(w, dims, np.concatenate([prefix, blk], axis=1))
    # layer 1: the prefix keys are kept (the full prefill's prefix rows also read the block)
    assert np.allclose(ext[1][0][:, :12], O.prefill(w, dims, prefix)[1][0], rtol=0, atol=0)
    assert not np.allclose(ext[1][0], full[1][0], atol=1e-4)


def test_extend_from_an_empty_prefix_is_the_prefill():
    dims, w = _tiny(2)
    V = dims["vocab"]
    ids = synth.prompt_ids(2, 10, V, seed=6)
    empty = [(np.zeros((2, 0, 2, 32)), np.zeros((2, 0, 2, 32))) for _ in range(2)]
    ext = O.prefill_extend(w, dims, empty, ids)
    full = O.prefill(w, dims, ids)
    for layer in range(2):
        for t in range(2):
            assert np.allclose(ext[layer][t], full[layer][t], rtol=0, atol=1e-6)
