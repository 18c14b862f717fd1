"""GPU parity of dard_step_full (the step without a prefix cache: the whole
sequence with its future masked blocks plus the shadow block) against the
oracle's full-sequence mode, with the decision-parity protocol of the
prefix-cache step tests."""
import sys

import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth

from test_gpu_step import P, check_decisions

pytestmark = pytest.mark.gpu


def announce(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def full_case(dims, b, prompt, gen, B, blk_index, params, seed=1, lm_scale=None, frac=None, wdevice="cpu"):
    """Sequence = prompt ids, committed blocks (random ids) before the current
    block, the current block's tokens, [Mask] after it."""
    V = dims.vocab
    N = prompt + gen
    blk = prompt + blk_index * B
    w = synth.make_weights(dims, seed=seed, device=wdevice)
    if lm_scale is not None:
        w["lm_head"] = (w["lm_head"].float() * lm_scale).to(w["lm_head"].dtype)
    eng = dard.Engine(dims, {k: v.cuda() for k, v in w.items()}, b, B, N + B)
    seq = synth.prompt_ids(b, N, V, seed=seed + 1)
    if frac is None:
        tok, state, conf = synth.tiny_block(b, B, V, seed=seed + 2)
    else:
        tok, state, conf = synth.workload_block(b, B, frac, V, seed=seed + 2)
    seq[:, blk:blk + B] = tok
    seq[:, blk + B:] = dims.mask_id
    cp = dard.make_params(params["tau_c"], params["tau_u"], params["lam"], params["p0"], params["mask_id"],
                          params.get("flags", 0), params.get("w_fixed", 0.0))
    t_out = torch.zeros(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.zeros(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.zeros(b, B, device="cuda")
    done = torch.zeros(b, dtype=torch.int32, device="cuda")
    dbg = {"logits": torch.zeros(b, 2 * B, V, device="cuda"), "w": torch.zeros(b, B, device="cuda")}
    eng.dard_step_full(blk, cp, dev(seq), dev(state), dev(conf), t_out, s_out, c_out, done, debug=dbg)
    torch.cuda.synchronize()
    ow = synth.OracleWeights(dims, w)
    dd = dims.as_dict()
    ref = O.dard_step_full(ow, dd, seq, blk, B, state, conf, params)

    def floor(amp=1e-7):
        # the oracle's own logits under one-ulp perturbations before every bf16 rounding
        rng = np.random.default_rng(0)
        orig = O.storage
        O.storage = lambda x, dt: orig(np.asarray(x, dtype=np.float64) * (1.0 + amp * rng.standard_normal(np.shape(x))), dt)
        try:
            l2 = O.full_step_logits(ow, dd, seq, blk, B, state, conf, params["mask_id"], params.get("flags", 0))
        finally:
            O.storage = orig
        return float(np.max(np.abs(l2 - ref["logits"])))

    ref["floor"] = floor
    got = dict(logits=dbg["logits"].cpu().numpy(), w=dbg["w"].cpu().numpy(), state_out=s_out.cpu().numpy(),
               tok_out=t_out.cpu().numpy(), conf_out=c_out.cpu().numpy(), block_done=done.cpu().numpy())
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
    err = np.max(np.abs(got["logits"] - ref["logits"]))
    assert err < 1e-4 * 20, err
    eps, excl = check_decisions(tok, state, got, ref, prm)
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
    err = np.max(np.abs(got["logits"] - ref["logits"]))
    assert err < 2e-2 * 8, err
    eps, excl = check_decisions(tok, state, got, ref, prm)
    print(f"max |dlogit| {eps:.3e}, rows excluded {excl} of {state.size}", file=sys.stderr)
    assert excl <= state.size // 2


def test_block128_full_step_fp32():
    """Block 128 (the paper's default block length) as the first of two
    generation blocks after a 64-token prompt; fp32, so that the decision
    margins stay far above the logit error."""
    dims = synth.Dims(2, 512, 8, 8, 64, 1024, 2048, 1024, "f32")
    announce("block-128 fp32 full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 64, 256, 128, 0, prm, seed=4, lm_scale=8.0)
    err = np.max(np.abs(got["logits"] - ref["logits"]))
    assert err < 1e-4 * 8, err
    eps, excl = check_decisions(tok, state, got, ref, prm)
    print(f"max |dlogit| {eps:.3e}, rows excluded {excl} of {state.size}", file=sys.stderr)
    assert excl <= state.size // 2


def test_block256_full_step_fp32():
    """Block 256, the longest of the paper's latency table: the whole 256-token
    generation is one block after a 64-token prompt; fp32."""
    dims = synth.Dims(2, 256, 4, 4, 64, 512, 2048, 1024, "f32")
    announce("block-256 fp32 full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 64, 256, 256, 0, prm, seed=6, lm_scale=8.0)
    err = np.max(np.abs(got["logits"] - ref["logits"]))
    assert err < 1e-4 * 8, err


def test_llada8b_block256_full_step_two_layers():
    """The paper's block-256 latency setting at the 8B shape (two layers):
    prompt 128, one generation block of 256 (its partials exceed the decision
    kernel's LDS staging, so they are read in place)."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("llada8b 2-layer full step, block 256")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 128, 256, 256, 0, prm, seed=2, frac=0.25, wdevice="cuda")
    d = got["logits"] - ref["logits"]
    err, rms = float(np.max(np.abs(d))), float(np.sqrt(np.mean(d * d)))
    floor = ref["floor"]() if err >= 2e-2 else 0.0
    print(f"llada8b block-256 full step: max {err:.3e} rms {rms:.3e} floor {floor:.3e}", file=sys.stderr)
    assert rms < 2e-2
    assert err < max(2e-2, 2.0 * floor), (err, floor)
    check_decisions(tok, state, got, ref, prm)


def test_llada8b_full_step_two_layers():
    """The paper's latency setting at the 8B shape (two layers): prompt 128,
    generation 256 in blocks of 128, the first block current (one future
    block), candidate fraction 0.25."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("llada8b 2-layer full step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = full_case(dims, 1, 128, 256, 128, 0, prm, seed=1, frac=0.25, wdevice="cuda")
    d = got["logits"] - ref["logits"]
    err, rms = float(np.max(np.abs(d))), float(np.sqrt(np.mean(d * d)))
    floor = ref["floor"]() if err >= 2e-2 else 0.0
    print(f"llada8b full step: max {err:.3e} rms {rms:.3e} floor {floor:.3e}", file=sys.stderr)
    assert rms < 2e-2
    assert err < max(2e-2, 2.0 * floor), (err, floor)
    check_decisions(tok, state, got, ref, prm)
