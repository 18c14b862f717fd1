"""A DARD step captured in a HIP graph (torch.cuda.CUDAGraph over the
library's launches) and replayed: dard_step makes no host synchronisation,
allocation or memset, so the captured step must reproduce the eager step
exactly.  The replays alternate two sets of inputs written into the captured
input tensors, with eager steps, zeroed outputs and synchronisations between
them, and every replay is compared bit for bit with the eager step on the same
inputs."""
import numpy as np
import pytest
import torch

from paper_2608_26574_amd import dard, synth
from parity import P, announce, cparams, dev, sharpen

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", [
    # 8B shape, 2 layers, batch 1: weight-streaming GEMMs, split-key attention and its combine
    dict(dims=("llada8b", 2), b=1, B=32, P=544, frac=0.25, scale=6.0),
    # 7B GQA shape, 1 layer, batch 4 (256 step rows): large-tile GEMMs, the fused LM-head partials
    dict(dims=("dream7b", 1), b=4, B=64, P=160, frac=0.3, scale=6.0),
])
def test_step_graph_replay(case):
    name, layers = case["dims"]
    dims = synth.truncated(synth.LLADA8B if name == "llada8b" else synth.DREAM7B, layers)
    b, B, P_ = case["b"], case["B"], case["P"]
    announce("graph replay", name, layers, b, B, P_)
    w = sharpen(synth.make_weights(dims, seed=51, device="cuda"), case["scale"])
    eng = dard.Engine(dims, w, b, B, P_ + 2 * B)
    del w
    eng.dard_prefill(dev(synth.prompt_ids(b, P_, dims.vocab, seed=52)))
    params = cparams(dard, P(dims.mask_id))
    inputs = [tuple(dev(a) for a in synth.workload_block(b, B, case["frac"], dims.vocab, seed=53 + k))
              for k in range(2)]

    def outputs():
        return (torch.zeros(b, B, dtype=torch.int32, device="cuda"), torch.zeros(b, B, dtype=torch.uint8, device="cuda"),
                torch.zeros(b, B, device="cuda"), torch.zeros(b, dtype=torch.int32, device="cuda"))

    # eager reference of each input set
    ref = []
    for tok, st, cf in inputs:
        o = outputs()
        eng.dard_step(P_, params, tok, st, cf, *o)
        ref.append(o)
    torch.cuda.synchronize()
    # the two input sets must lead to different decisions, or the replays would prove nothing
    assert not all(torch.equal(x, y) for x, y in zip(ref[0][:3], ref[1][:3]))

    # capture one step on static tensors
    s_tok, s_st, s_cf = (t.clone() for t in inputs[0])
    s_out = outputs()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        eng.dard_step(P_, params, s_tok, s_st, s_cf, *s_out)
    torch.cuda.synchronize()

    scratch = outputs()
    for r, k in enumerate((0, 1, 1, 0, 1)):
        # eager work between replays: a step on the other inputs, the outputs zeroed
        tok, st, cf = inputs[1 - k]
        eng.dard_step(P_, params, tok, st, cf, *scratch)
        for t in s_out:
            t.zero_()
        for dst, src in zip((s_tok, s_st, s_cf), inputs[k]):
            dst.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want, what in zip(s_out, ref[k], ("tok_out", "state_out", "conf_out", "block_done")):
            assert torch.equal(got, want), (r, k, what)
        for got, want in zip(scratch, ref[1 - k]):
            assert torch.equal(got, want), (r, "eager step between replays")
    print(f"graph replay {name} x{layers}: 5 replays equal the eager steps", flush=True)


def test_steps_on_two_streams():
    """Two engines stepping on two streams at once (default priority) give the
    same results as each engine alone: a step keeps all of its state in the
    caller's workspace and KV cache, none in the library."""
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 512, "bf16")
    b, B, P_ = 2, 32, 96
    announce("two streams")
    engines, inputs = [], []
    for k in range(2):
        w = sharpen(synth.make_weights(dims, seed=61 + k, device="cuda"), 12.0)
        eng = dard.Engine(dims, w, b, B, P_ + 2 * B)
        eng.dard_prefill(dev(synth.prompt_ids(b, P_, dims.vocab, seed=63 + k)))
        engines.append(eng)
        inputs.append(tuple(dev(a) for a in synth.workload_block(b, B, 0.3, dims.vocab, seed=65 + k)))
    params = cparams(dard, P(dims.mask_id))

    def outputs():
        return (torch.zeros(b, B, dtype=torch.int32, device="cuda"), torch.zeros(b, B, dtype=torch.uint8, device="cuda"),
                torch.zeros(b, B, device="cuda"), torch.zeros(b, dtype=torch.int32, device="cuda"))

    alone = []
    for eng, inp in zip(engines, inputs):
        o = outputs()
        eng.dard_step(P_, params, *inp, *o)
        torch.cuda.synchronize()
        alone.append(o)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    together = [[outputs() for _ in range(4)] for _ in range(2)]
    torch.cuda.synchronize()
    for r in range(4):
        for k in range(2):
            with torch.cuda.stream(streams[k]):
                engines[k].dard_step(P_, params, *inputs[k], *together[k][r])
    torch.cuda.synchronize()
    for k in range(2):
        for r in range(4):
            for got, want in zip(together[k][r], alone[k]):
                assert torch.equal(got, want), (k, r)


@pytest.mark.parametrize("mode", ["full", "shared"])
def test_full_and_shared_steps_graph_replay(mode):
    """dard_step_full and dard_step_shared captured in a HIP graph and
    replayed on alternating inputs, every replay equal to the eager step."""
    dims = synth.Dims(2, 512, 4, 2, 128, 1024, 2048, 1024, "bf16")
    b, B = 2, 32
    announce("graph replay", mode)
    w = sharpen(synth.make_weights(dims, seed=71, device="cuda"), 8.0)
    params = cparams(dard, P(dims.mask_id))
    if mode == "full":
        prompt, gen = 40, 96
        N, blk = prompt + gen, prompt + B
        eng = dard.Engine(dims, w, b, B, N + B)
        inputs = []
        for k in range(2):
            tok, state, conf = synth.workload_block(b, B, 0.3, dims.vocab, seed=74 + k)
            seq = synth.prompt_ids(b, N, dims.vocab, seed=72 + k)
            seq[:, blk:blk + B] = tok
            seq[:, blk + B:] = dims.mask_id
            inputs.append((dev(seq), dev(state), dev(conf)))

        def step(inp, o):
            eng.dard_step_full(blk, params, inp[0], inp[1], inp[2], *o)
    else:
        Ps, Pc = 64, 32
        sh = dard.Engine(dims, w, 1, B, Ps)
        eng = dard.Engine(dims, None, b, B, Ps + Pc + 2 * B, packed=sh.packed)
        sh.dard_prefill(dev(synth.prompt_ids(1, Ps, dims.vocab, seed=76)))
        eng.dard_prefill_suffix(sh, Ps, dev(synth.prompt_ids(b, Pc, dims.vocab, seed=77)))
        inputs = [tuple(dev(a) for a in synth.workload_block(b, B, 0.3, dims.vocab, seed=78 + k)) for k in range(2)]

        def step(inp, o):
            eng.dard_step_shared(sh, Ps, Ps + Pc, params, *inp, *o)
    del w

    def outputs():
        return (torch.zeros(b, B, dtype=torch.int32, device="cuda"), torch.zeros(b, B, dtype=torch.uint8, device="cuda"),
                torch.zeros(b, B, device="cuda"), torch.zeros(b, dtype=torch.int32, device="cuda"))

    ref = []
    for inp in inputs:
        o = outputs()
        step(inp, o)
        ref.append(o)
    torch.cuda.synchronize()
    assert not all(torch.equal(x, y) for x, y in zip(ref[0][:3], ref[1][:3]))
    s_in = tuple(t.clone() for t in inputs[0])
    s_out = outputs()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(s_in, s_out)
    torch.cuda.synchronize()
    for r, k in enumerate((1, 0, 1)):
        for t in s_out:
            t.zero_()
        for dst, src in zip(s_in, inputs[k]):
            dst.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want, what in zip(s_out, ref[k], ("tok_out", "state_out", "conf_out", "block_done")):
            assert torch.equal(got, want), (mode, r, k, what)
    print(f"graph replay {mode}: 3 replays equal the eager steps", flush=True)
