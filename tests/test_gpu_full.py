"""GPU parity of dard_step_full (the step without a prefix cache: the whole
sequence with its future masked blocks plus the shadow block) against the
oracle's full-sequence mode, with the decision-parity protocol of the
prefix-cache step tests."""
import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth

from parity import (P, announce, check_bf16_logits, check_decisions, check_workload_decisions, collect, cparams,
                    dev, Floor, logit_err, sharpen, step_buffers)

pytestmark = pytest.mark.gpu

WORKLOAD_LM_SCALE = 6.0


def full_case(dims, b, prompt, gen, B, blk_index, params, seed=1, lm_scale=None, frac=None, wdevice="cpu"):
    """Sequence = prompt ids, committed blocks (random ids) before the current
    block, the current block's tokens, [Mask] after it."""
    V = dims.vocab
    N = prompt + gen
    blk = prompt + blk_index * B
    w = sharpen(synth.make_weights(dims, seed=seed, device=wdevice), lm_scale)
    eng = dard.Engine(dims, {k: v.cuda() for k, v in w.items()}, b, B, N + B)
    seq = synth.prompt_ids(b, N, V, seed=seed + 1)
    if frac is None:
        tok, state, conf = synth.tiny_block(b, B, V, seed=seed + 2)
    else:
        tok, state, conf = synth.workload_block(b, B, frac, V, seed=seed + 2)
    seq[:, blk:blk + B] = tok
    seq[:, blk + B:] = dims.mask_id
    out, dbg = step_buffers(b, B, V)
    eng.dard_step_full(blk, cparams(dard, params), dev(seq), dev(state), dev(conf), out["tok_out"], out["state_out"],
                       out["conf_out"], out["block_done"], debug=dbg)
    got = collect(out, dbg)
    ow = synth.OracleWeights(dims, w)
    dd = dims.as_dict()
    ref = O.dard_step_full(ow, dd, seq, blk, B, state, conf, params)
    ref["state"], ref["params"] = state, params
    ref["floor"] = Floor(
        lambda: O.full_step_logits(ow, dd, seq, blk, B, state, conf, params["mask_id"], params.get("flags", 0)),
        ref["logits"])
    return tok, state, conf, got, ref


@pytest.mark.parametrize("blk_index,flags", [(0, 0), (1, 0), (2, 0), (1, O.F_MKEYS_SHADOW), (1, O.F_ORDER_L2R),
                                             (0, O.F_ORDER_ENTROPY | O.F_FIXED_W), (2, O.F_C_BIDIR | O.F_PROGRESS)])
def test_tiny_full_step_fp32(blk_index, flags):
    """Tiny fp32 model, prompt 40, generation 96 in blocks of 32: the current
    block first (two future blocks), in the middle, and last."""
    dims = synth.TINY
    announce("tiny fp32 full step", blk_index, flags)
    prm = P(dims.mask_id, flags, w_fixed=0.5)
    tok, state, conf, got, ref = full_case(dims, 1, 40, 96, 32, blk_index, prm, seed=3, lm_scale=20.0)
    err = logit_err(got, ref, state, prm)
    assert err < 1e-4 * 20, err
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, f"tiny full step {blk_index} {flags}")
    assert excl <= 1


@pytest.mark.parametrize("case", [
    dict(d=512, H=4, Hkv=2, dh=128, F=1024, V=2048, b=2, prompt=40, gen=96, B=32, k=1),   # GQA, batch 2
    dict(d=256, H=4, Hkv=4, dh=64, F=512, V=4096, b=1, prompt=17, gen=64, B=16, k=3),     # ragged, block last
])
def test_small_full_step_bf16(case):
    dims = synth.Dims(2, case["d"], case["H"], case["Hkv"], case["dh"], case["F"], case["V"], 1024, "bf16")
    announce("small bf16 full step", case)
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, case["b"], case["prompt"], case["gen"], case["B"], case["k"], prm,
                                           seed=4, lm_scale=8.0)
    err = logit_err(got, ref, state, prm)
    assert err < 2e-2 * 8, err
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "full step")
    assert excl <= state.size // 4


def test_small_full_step_bf16_fp8_kv():
    """The full-sequence step with the KV cache in OCP FP8 E4M3: every row's K
    and V are rounded to E4M3 where they are written and read back as codes."""
    dims = synth.with_fp8_kv(synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16"))
    announce("small bf16 full step, fp8 kv")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 2, 40, 96, 32, 1, prm, seed=6, lm_scale=8.0)
    check_bf16_logits(got, ref, "full step, fp8 kv", scale=8.0)
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "full step, fp8 kv")
    assert excl <= state.size // 4


def test_small_full_step_bf16_hidden_mix():
    """The full-sequence step with DARD_F_HIDDEN_MIX (Eq. 7 on the final hidden
    rows, two LM-head passes) against the oracle's logit mixing."""
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16")
    announce("small bf16 full step, hidden mix")
    prm = P(dims.mask_id, O.F_HIDDEN_MIX)
    tok, state, conf, got, ref = full_case(dims, 2, 40, 96, 32, 1, prm, seed=8, lm_scale=8.0)
    check_bf16_logits(got, ref, "full step, hidden mix", scale=8.0)
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "full step, hidden mix")
    assert excl <= state.size // 4
    assert np.all(np.isnan(got["logits"][:, :32]))   # the x rows never ran through the head


def test_block128_full_step_fp32():
    """Block 128 (the paper's default block length) as the first of two
    generation blocks after a 64-token prompt; fp32, so that the decision
    margins stay far above the logit error."""
    dims = synth.Dims(2, 512, 8, 8, 64, 1024, 2048, 1024, "f32")
    announce("block-128 fp32 full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 64, 256, 128, 0, prm, seed=4, lm_scale=8.0)
    err = logit_err(got, ref, state, prm)
    assert err < 1e-4 * 8, err
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "full step")
    assert excl <= state.size // 4


def test_block256_full_step_fp32():
    """Block 256, the longest of the paper's latency table: the whole 256-token
    generation is one block after a 64-token prompt; fp32."""
    dims = synth.Dims(2, 256, 4, 4, 64, 512, 2048, 1024, "f32")
    announce("block-256 fp32 full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 64, 256, 256, 0, prm, seed=6, lm_scale=8.0)
    err = logit_err(got, ref, state, prm)
    assert err < 1e-4 * 8, err


def test_llada8b_block256_full_step_two_layers():
    """The paper's block-256 latency setting at the 8B shape (two layers):
    prompt 128, one generation block of 256 (its partials exceed the decision
    kernel's LDS staging, so they are read in place)."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("llada8b 2-layer full step, block 256")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 128, 256, 256, 0, prm, seed=2, frac=0.25, wdevice="cuda",
                                           lm_scale=WORKLOAD_LM_SCALE)
    check_bf16_logits(got, ref, "llada8b block-256 full step", scale=WORKLOAD_LM_SCALE)
    check_workload_decisions(tok, state, got, ref, prm, "llada8b block-256 full step")


def test_llada8b_full_step_two_layers():
    """The paper's latency setting at the 8B shape (two layers): prompt 128,
    generation 256 in blocks of 128, the first block current (one future
    block), candidate fraction 0.25."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("llada8b 2-layer full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 128, 256, 128, 0, prm, seed=1, frac=0.25, wdevice="cuda",
                                           lm_scale=WORKLOAD_LM_SCALE)
    check_bf16_logits(got, ref, "llada8b full step", scale=WORKLOAD_LM_SCALE)
    check_workload_decisions(tok, state, got, ref, prm, "llada8b full step")
