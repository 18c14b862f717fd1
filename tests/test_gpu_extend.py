"""GPU parity of dard_prefill_extend, the extend-only refresh of the prefix
cache at a block boundary: after a prefill, blocks are appended one at a time
(their rows see the cached keys and each other) and compared with the
oracle's prefill_extend chain, then a step runs on the extended cache and goes
through the step tests' decision-parity protocol."""
import numpy as np
import pytest
import torch

from oracle import dard_oracle as O
from paper_2608_26574_amd import dard, synth
from parity import (P, announce, check_bf16_logits, check_decisions, check_fp8_cache_layers, check_workload_decisions,
                    collect, cparams, dev, e4m3_decode, Floor, logit_err, sharpen, step_buffers)
from test_gpu_step import unpermute_k

pytestmark = pytest.mark.gpu


def extend_case(dims, b, P0, blocks, B, seed, lm_scale, frac=None):
    V = dims.vocab
    w = sharpen(synth.make_weights(dims, seed=seed, device="cpu"), lm_scale)
    P_end = P0 + sum(blocks)
    eng = dard.Engine(dims, {k: v.cuda() for k, v in w.items()}, b, B, P_end + 2 * B)
    ow = synth.OracleWeights(dims, w)
    dd = dims.as_dict()
    prefix = synth.prompt_ids(b, P0, V, seed=seed + 1)
    eng.dard_prefill(dev(prefix))
    cache = O.prefill(ow, dd, prefix)
    P_ = P0
    for k, n in enumerate(blocks):
        ids = synth.prompt_ids(b, n, V, seed=seed + 10 + k)
        eng.dard_prefill_extend(P_, dev(ids))
        cache = O.prefill_extend(ow, dd, cache, ids)
        P_ += n
    # the extended cache, every layer
    if dims.kv_dtype == "fp8":
        kc, vc = eng.kv_view(torch.uint8)
        pairs = []
        for layer in range(dims.n_layers):
            k_gpu = unpermute_k(e4m3_decode(kc[layer, :, :, :P_]), dims.head_dim).transpose(0, 2, 1, 3)
            v_gpu = e4m3_decode(vc[layer, :, :, :P_]).transpose(0, 2, 1, 3)
            pairs += [(layer, 0, k_gpu, cache[layer][0]), (layer, 1, v_gpu, cache[layer][1])]
        check_fp8_cache_layers(pairs, "extended")
    else:
        tol = 1e-4 if dims.dtype == "f32" else 8e-2
        kvd = torch.float32 if dims.dtype == "f32" else torch.bfloat16
        kc, vc = eng.kv_view(kvd)
        kc, vc = kc.float().cpu().numpy(), vc.float().cpu().numpy()
        for layer in range(dims.n_layers):
            k_gpu = unpermute_k(kc[layer, :, :, :P_], dims.head_dim).transpose(0, 2, 1, 3)
            v_gpu = vc[layer, :, :, :P_].transpose(0, 2, 1, 3)
            ek = float(np.max(np.abs(k_gpu - cache[layer][0])))
            ev = float(np.max(np.abs(v_gpu - cache[layer][1])))
            print(f"extended cache layer {layer}: max |dK| {ek:.3e} |dV| {ev:.3e}", flush=True)
            assert ek < tol and ev < tol, (layer, ek, ev)
    # a step on the extended cache
    if frac is None:
        tok, state, conf = synth.tiny_block(b, B, V, seed=seed + 2)
    else:
        tok, state, conf = synth.workload_block(b, B, frac, V, seed=seed + 2)
    params = P(dims.mask_id)
    out, dbg = step_buffers(b, B, V)
    eng.dard_step(P_, cparams(dard, params), dev(tok), dev(state), dev(conf), out["tok_out"], out["state_out"],
                  out["conf_out"], out["block_done"], debug=dbg)
    got = collect(out, dbg)
    ref = O.dard_step(ow, dd, cache, tok, state, conf, params)
    ref["state"], ref["params"] = state, params

    def perturbed():
        c2 = O.prefill(ow, dd, prefix)
        for k, n in enumerate(blocks):
            c2 = O.prefill_extend(ow, dd, c2, synth.prompt_ids(b, n, V, seed=seed + 10 + k))
        return O.step_logits(ow, dd, c2, tok, state, conf, params["mask_id"])[0]

    ref["floor"] = Floor(perturbed, ref["logits"])
    return tok, state, got, ref, params


def test_extend_tiny_fp32():
    """Tiny fp32 model, batch 2: prefill of 40, then blocks of 16, 16 and 7."""
    announce("extend tiny fp32")
    tok, state, got, ref, prm = extend_case(synth.TINY, 2, 40, (16, 16, 7), 16, seed=71, lm_scale=20.0)
    err = logit_err(got, ref, state, prm)
    assert err < 1e-4 * 20, err
    _, excl, _ = check_decisions(tok, state, got, ref, prm, "extend tiny fp32")
    assert excl <= 1


def test_extend_small_bf16_gqa():
    """bf16, 4 query heads on 2 KV heads x 128, batch 3: prefill of 64, blocks of 24 and 24."""
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 512, "bf16")
    announce("extend small bf16")
    tok, state, got, ref, prm = extend_case(dims, 3, 64, (24, 24), 24, seed=72, lm_scale=8.0)
    err = logit_err(got, ref, state, prm)
    assert err < 2e-2 * 8, err
    _, excl, _ = check_decisions(tok, state, got, ref, prm, "extend small bf16")
    assert excl <= state.size // 4


def test_extend_small_bf16_gqa_fp8_kv():
    """The same chain with the KV cache in OCP FP8 E4M3: the appended blocks'
    K and V are rounded to E4M3 where they are written, and their rows read
    the cached codes."""
    dims = synth.with_fp8_kv(synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 512, "bf16"))
    announce("extend small bf16, fp8 kv")
    tok, state, got, ref, prm = extend_case(dims, 3, 64, (24, 24), 24, seed=74, lm_scale=8.0)
    check_bf16_logits(got, ref, "extend small bf16, fp8 kv", scale=8.0)
    _, excl, _ = check_decisions(tok, state, got, ref, prm, "extend small bf16, fp8 kv")
    assert excl <= state.size // 4


def test_extend_llada8b_two_layers():
    """The 8B shape with two layers at the headline block: prefill of the 512
    prompt positions, then two committed blocks of 32 appended."""
    dims = synth.truncated(synth.LLADA8B, 2)
    announce("extend llada8b 2 layers")
    tok, state, got, ref, prm = extend_case(dims, 1, 512, (32, 32), 32, seed=73, lm_scale=6.0, frac=0.25)
    check_bf16_logits(got, ref, "extend llada8b 2 layers", scale=6.0)
    check_workload_decisions(tok, state, got, ref, prm, "extend llada8b 2 layers", require_transitions=False)
