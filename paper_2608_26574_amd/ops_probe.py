"""Workload for the counter profiles of the isolated operations.

Runs, in this order and with inputs rotated through copies larger than the
256 MB MALL (so every launch reads from HBM):
  1. state-masked attention at the 7B GQA shape (28 query heads on 4 KV
     heads x 128, batch 8, block 64, prefix 1024, candidate fraction 0.3),
     10 calls -- the compute-bound attention shape;
  2. state-masked attention at the 8B MHA shape (32 x 128 heads, batch 16,
     prefix 512, block 32, candidate fraction 0.25), 10 calls;
  3. the vocab-wide confidence reduction over 696 rows x 152064 fp32 logits
     (the 7B GQA batch-8 step's rows), 10 calls;
  4. 3 DARD steps of the 7B GQA model truncated to 2 layers (28/4 heads x
     128, d 3584, FFN 18944, vocab 152064, bf16) at batch 8, block 64,
     prefix 1024: 1024 token rows, so every projection and the LM head run
     the MFMA-bound large-tile GEMM;
  5. one 1 GiB device-to-device copy (the calibration of the byte counters).
A profiler pass (rocprofv3 --kernel-trace, or --pmc with MFMA or byte
counters) attributes each kernel to its operation by name and grid.
"""
import sys

import torch

from paper_2608_26574_amd import dard, synth

COPY_BYTES = 1 << 30


def attention(b, Hq, Hkv, B, P, frac, calls, seed):
    dh, cap = 128, P + 2 * B
    g = torch.Generator(device="cuda").manual_seed(seed)
    kv_bytes = 2 * b * Hkv * cap * dh * 2
    ncopy = max(2, -(-600 * 2**20 // kv_bytes))
    q = torch.randn(b, 2 * B, Hq, dh, generator=g, device="cuda").bfloat16()
    ks = [torch.randn(b, Hkv, cap, dh, generator=g, device="cuda").bfloat16() for _ in range(ncopy)]
    vs = [torch.randn(b, Hkv, dh, cap, generator=g, device="cuda").bfloat16() for _ in range(ncopy)]
    _, state, conf = synth.workload_block(b, B, frac, 100, seed=seed)
    state, conf = torch.from_numpy(state).cuda(), torch.from_numpy(conf).cuda()
    out = torch.empty_like(q)
    ws = torch.empty(max(dard.dard_attention_workspace_bytes(1, b, B, Hq, dh, P), 1), dtype=torch.uint8,
                     device="cuda")
    for i in range(calls):
        dard.dard_masked_attention(q, ks[i % ncopy], vs[i % ncopy], P, state, conf, dh ** -0.5, 0, out, ws)
    torch.cuda.synchronize()


def confidence(rows, V, calls):
    nbytes = rows * V * 4
    ncopy = max(2, -(-600 * 2**20 // nbytes))
    g = torch.Generator(device="cuda").manual_seed(4)
    ls = [torch.randn(rows, V, generator=g, device="cuda") for _ in range(ncopy)]
    am = torch.empty(rows, dtype=torch.int32, device="cuda")
    mp = torch.empty(rows, device="cuda")
    ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
    for i in range(calls):
        dard.dard_confidence(ls[i % ncopy], am, mp, ws=ws)
    torch.cuda.synchronize()


def gqa_steps(steps):
    dims = synth.truncated(synth.DREAM7B, 2)
    b, B, P = 8, 64, 1024
    w = synth.make_weights(dims, seed=1, device="cuda")
    eng = dard.Engine(dims, w, b, B, P + 2 * B)
    del w
    ids = torch.from_numpy(synth.prompt_ids(b, P, dims.vocab, seed=2)).cuda()
    eng.dard_prefill(ids)
    tok, state, conf = (torch.from_numpy(a).cuda() for a in synth.workload_block(b, B, 0.3, dims.vocab, seed=3))
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.empty(b, B, device="cuda")
    for _ in range(steps):
        eng.dard_step(P, params, tok, state, conf, t_out, s_out, c_out)
    torch.cuda.synchronize()


def main():
    attention(8, 28, 4, 64, 1024, 0.3, 10, seed=1)
    print("[ops] GQA attention done", flush=True)
    attention(16, 32, 32, 32, 512, 0.25, 10, seed=2)
    print("[ops] MHA attention done", flush=True)
    confidence(8 * 87, 152064, 10)
    print("[ops] confidence done", flush=True)
    gqa_steps(3)
    print("[ops] 7B GQA steps done", flush=True)
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    print(f"[ops] copied {COPY_BYTES} bytes", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
