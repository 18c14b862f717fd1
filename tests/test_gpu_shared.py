"""GPU parity of the batch-shared prompt cache: dard_prefill (b = 1) over the
prompt, dard_prefill_suffix for each sequence's committed positions, and
dard_step_shared, against the oracle's prefill / prefill_suffix / join_shared
and its step, with the decision-parity protocol of the step tests."""
import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth

from parity import (P, announce, check_bf16_logits, check_decisions, check_fp8_cache_layers, check_workload_decisions,
                    collect, cparams, dev, e4m3_decode, Floor, logit_err, sharpen, step_buffers)

pytestmark = pytest.mark.gpu

WORKLOAD_LM_SCALE = 6.0


def shared_case(dims, b, Ps, Pc, B, params, seed=1, lm_scale=None, frac=None, wdevice="cpu", n_image=0):
    V = dims.vocab
    w = sharpen(synth.make_weights(dims, seed=seed, device=wdevice), lm_scale)
    sh = dard.Engine(dims, {k: v.cuda() for k, v in w.items()}, 1, B, Ps)
    eng = dard.Engine(dims, None, b, B, Ps + Pc + 2 * B + 3, packed=sh.packed)
    prompt = synth.prompt_ids(1, Ps, V, seed=seed + 1)
    embeds = None
    if n_image:
        prompt[:, :n_image] = -1
        g = torch.Generator().manual_seed(seed + 3)
        td = torch.float32 if dims.dtype == "f32" else torch.bfloat16
        embeds = torch.randn(1, Ps, dims.d_model, generator=g).to(td)
    committed = synth.prompt_ids(b, Pc, V, seed=seed + 4)
    if frac is None:
        tok, state, conf = synth.tiny_block(b, B, V, seed=seed + 2)
    else:
        tok, state, conf = synth.workload_block(b, B, frac, V, seed=seed + 2)
    sh.dard_prefill(dev(prompt), embeds=None if embeds is None else embeds.cuda())
    if Pc:
        eng.dard_prefill_suffix(sh, Ps, dev(committed))
    out, dbg = step_buffers(b, B, V)
    eng.dard_step_shared(sh, Ps, Ps + Pc, cparams(dard, params), dev(tok), dev(state), dev(conf), out["tok_out"],
                         out["state_out"], out["conf_out"], out["block_done"], debug=dbg)
    got = collect(out, dbg)
    ow = synth.OracleWeights(dims, w)
    dd = dims.as_dict()
    shared = O.prefill(ow, dd, prompt, None if embeds is None else embeds.double().numpy())
    suffix = O.prefill_suffix(ow, dd, shared, committed)
    cache = O.join_shared(shared, suffix)
    ref = O.dard_step(ow, dd, cache, tok, state, conf, params)
    ref["state"], ref["params"] = state, params

    def perturbed():
        shp = O.prefill(ow, dd, prompt, None if embeds is None else embeds.double().numpy())
        c2 = O.join_shared(shp, O.prefill_suffix(ow, dd, shp, committed))
        return O.step_logits(ow, dd, c2, tok, state, conf, params["mask_id"], params.get("flags", 0))[0]

    ref["floor"] = Floor(perturbed, ref["logits"])
    # the suffix keys written by dard_prefill_suffix (V of every layer; K is stored with
    # each head's rotary pairs interleaved)
    if Pc and dims.kv_dtype == "fp8":
        _, vc = eng.kv_view(torch.uint8)
        check_fp8_cache_layers([(layer, 1, e4m3_decode(vc[layer, :, :, Ps:Ps + Pc]).transpose(0, 2, 1, 3),
                                 suffix[layer][1]) for layer in range(dims.n_layers)], "suffix")
    elif Pc:
        kvd = torch.float32 if dims.dtype == "f32" else torch.bfloat16
        _, vc = eng.kv_view(kvd)
        vc = vc.float().cpu().numpy()
        tol = 1e-4 if dims.dtype == "f32" else 8e-2
        for layer in range(dims.n_layers):
            v_gpu = vc[layer, :, :, Ps:Ps + Pc].transpose(0, 2, 1, 3)
            assert np.max(np.abs(v_gpu - suffix[layer][1])) < tol, layer
    return tok, state, conf, got, ref


@pytest.mark.parametrize("b,Ps,Pc,flags", [(2, 64, 32, 0), (3, 128, 0, 0), (1, 64, 96, 0),
                                          (2, 64, 32, O.F_ORDER_MARGIN | O.F_MKEYS_SHADOW)])
def test_tiny_shared_step_fp32(b, Ps, Pc, flags):
    dims = synth.TINY
    announce("tiny fp32 shared step", b, Ps, Pc, flags)
    prm = P(dims.mask_id, flags)
    tok, state, conf, got, ref = shared_case(dims, b, Ps, Pc, 32, prm, seed=3, lm_scale=20.0)
    err = logit_err(got, ref, state, prm)
    assert err < 1e-4 * 20, err
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "tiny shared step")
    assert excl <= 1


def test_small_shared_step_bf16_gqa():
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16")
    announce("small bf16 shared step")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = shared_case(dims, 4, 128, 64, 32, prm, seed=5, lm_scale=8.0)
    err = logit_err(got, ref, state, prm)
    assert err < 2e-2 * 8, err
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "small shared step")
    assert excl <= state.size // 4


def test_small_shared_step_bf16_gqa_fp8_kv():
    """The shared prompt cache, the sequences' suffixes and the step with the
    KV caches in OCP FP8 E4M3."""
    dims = synth.with_fp8_kv(synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16"))
    announce("small bf16 shared step, fp8 kv")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = shared_case(dims, 4, 128, 64, 32, prm, seed=7, lm_scale=8.0)
    check_bf16_logits(got, ref, "small shared step, fp8 kv", scale=8.0)
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "small shared step, fp8 kv")
    assert excl <= state.size // 4


def test_small_shared_step_bf16_hidden_mix():
    """The shared-prompt step with DARD_F_HIDDEN_MIX against the oracle's
    logit mixing."""
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16")
    announce("small bf16 shared step, hidden mix")
    prm = P(dims.mask_id, O.F_HIDDEN_MIX)
    tok, state, conf, got, ref = shared_case(dims, 3, 64, 32, 32, prm, seed=9, lm_scale=8.0)
    check_bf16_logits(got, ref, "small shared step, hidden mix", scale=8.0)
    eps, excl, _ = check_decisions(tok, state, got, ref, prm, "small shared step, hidden mix")
    assert excl <= state.size // 4
    assert np.all(np.isnan(got["logits"][:, :32]))


def test_multimodal_shared_prompt_two_layers():
    """8B shape, two layers: one 576-embedding image + 256-id prompt shared by
    a batch of 4, one committed block of 32 per sequence, block 32, candidate
    fraction 0.3."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("8B shared multimodal prompt, 2 layers")
    prm = P(dims.mask_id)
    tok, state, conf, got, ref = shared_case(dims, 4, 832, 32, 32, prm, seed=4, frac=0.3, wdevice="cuda",
                                             n_image=576, lm_scale=WORKLOAD_LM_SCALE)
    check_bf16_logits(got, ref, "8B shared prompt 2 layers", scale=WORKLOAD_LM_SCALE)
    check_workload_decisions(tok, state, got, ref, prm, "8B shared prompt 2 layers")
