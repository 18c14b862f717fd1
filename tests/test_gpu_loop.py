"""The decoding loop of Alg. 1 end to end on the GPU, checked against the
oracle at every step.

Each block starts all-[Mask] (Alg. 1: every position masked, confidences 0);
every step's state, tokens and keys are the next step's inputs, and a block
ends when all its positions are unmasked (block_done) or after 2B steps; the
next block's prefix cache is then recomputed over the prompt and the tokens
the GPU committed (the prefix-cache reading of App. C.5).  The oracle runs
each step on the same inputs the GPU step received, so the comparison covers
the GPU's own trajectory through several blocks, including the re-prefill
with decoded tokens; every step goes through the decision-parity protocol
(op level exact, step level exact wherever the margins decide).  Tiny fp32
model with the LM head sharpened so that confidences pass tau_u and blocks
complete."""
import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth
from parity import P, announce, check_decisions, collect, cparams, dev, logit_err, sharpen, step_buffers

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("flags", [O.F_PROGRESS, O.F_PROGRESS | O.F_ORDER_ENTROPY, O.F_PROGRESS | O.F_HIDDEN_MIX])
def test_decoding_loop_tiny_fp32(flags):
    dims = synth.TINY
    b, B, P0, nblocks, lm_scale = 2, 16, 24, 3, 40.0
    announce("decoding loop, tiny fp32", flags)
    w = sharpen(synth.make_weights(dims, seed=31), lm_scale)
    cap = P0 + B * nblocks + 2 * B
    eng = dard.Engine(dims, {k: v.cuda() for k, v in w.items()}, b, B, cap)
    ow = synth.OracleWeights(dims, w)
    dd = dims.as_dict()
    prm = P(dims.mask_id, flags)
    seq = synth.prompt_ids(b, P0, dims.vocab, seed=32)
    steps, done_blocks, excluded, committed_u = [], 0, 0, 0
    for k in range(nblocks):
        Pk = seq.shape[1]
        eng.dard_prefill(dev(seq))
        cache = O.prefill(ow, dd, seq)
        tok = np.full((b, B), dims.mask_id, dtype=np.int32)
        state = np.zeros((b, B), dtype=np.uint8)
        conf = np.zeros((b, B), dtype=np.float32)
        n = 0
        while True:
            out, dbg = step_buffers(b, B, dims.vocab)
            eng.dard_step(Pk, cparams(dard, prm), dev(tok), dev(state), dev(conf), out["tok_out"],
                          out["state_out"], out["conf_out"], out["block_done"], debug=dbg)
            got = collect(out, dbg)
            ref = O.dard_step(ow, dd, cache, tok, state, conf, prm)
            err = logit_err(got, ref, state, prm)
            # the sharpened head multiplies every upstream rounding difference by lm_scale
            assert err < 1e-4 * lm_scale, (k, n, err)
            _, excl, _ = check_decisions(tok, state, got, ref, prm, f"loop block {k} step {n}")
            excluded += excl
            n += 1
            tok, state, conf = got["tok_out"], got["state_out"], got["conf_out"]
            if np.all(got["block_done"] == 1) or n >= 2 * B:
                break
        steps.append(n)
        done_blocks += int(np.all(state == O.STATE_U))
        committed_u += int(np.sum(state == O.STATE_U))
        # the block's tokens join the sequence: the next prefix cache covers them
        seq = np.concatenate([seq, tok.astype(seq.dtype)], axis=1)
    print(f"loop flags {flags}: steps per block {steps}, finished blocks {done_blocks} of {nblocks}, "
          f"excluded positions {excluded}", flush=True)
    # the loop really decodes: blocks finish and commit their tokens
    assert done_blocks >= 1 and committed_u >= B, (steps, done_blocks, committed_u)
    assert excluded <= 2, excluded
    if excluded == 0:
        # no decision was left to the margins: the oracle decoding on its own
        # produces the same sequence in the same number of steps
        ref_seq, ref_steps = oracle_loop(ow, dd, prm, synth.prompt_ids(b, P0, dims.vocab, seed=32), B, nblocks)
        assert ref_steps == steps, (ref_steps, steps)
        assert np.array_equal(ref_seq, seq)


def oracle_loop(ow, dd, prm, seq, B, nblocks):
    """The same loop driven by the oracle's own decisions."""
    b = seq.shape[0]
    steps = []
    for _ in range(nblocks):
        cache = O.prefill(ow, dd, seq)
        tok = np.full((b, B), prm["mask_id"], dtype=np.int32)
        state = np.zeros((b, B), dtype=np.uint8)
        conf = np.zeros((b, B), dtype=np.float32)
        n = 0
        while True:
            ref = O.dard_step(ow, dd, cache, tok, state, conf, prm)
            n += 1
            tok = ref["tok_out"].astype(np.int32)
            state = ref["state_out"].astype(np.uint8)
            conf = ref["conf_out"].astype(np.float32)
            if np.all(ref["block_done"] == 1) or n >= 2 * B:
                break
        steps.append(n)
        seq = np.concatenate([seq, tok.astype(seq.dtype)], axis=1)
    return seq, steps
