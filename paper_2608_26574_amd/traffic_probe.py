"""Workload for the HBM-traffic counters of the decoding step.

Runs a few DARD steps at the 8B shape (32 layers, d 4096, 32 x 128 heads,
FFN 12288, vocab 126464, bf16; batch 1, block 32, prompt 512) and then one
plain device-to-device copy of exactly COPY_BYTES, so that a profiler pass
(rocprofv3 --pmc FETCH_SIZE or WRITE_SIZE) sees both the step's kernels and a
copy kernel of known size in the same process.  The copy calibrates the
counters: a copy of S bytes reads S and writes S bytes of HBM.
"""
import sys

import torch

from paper_2608_26574_amd import dard, synth

COPY_BYTES = 1 << 30


def main():
    dims = synth.LLADA8B
    b, B, P, cap = 1, 32, 512, 800
    print("[traffic] packing weights", flush=True)
    w = synth.make_weights(dims, seed=1, device="cuda")
    eng = dard.Engine(dims, w, b, B, cap)
    del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    ids = torch.from_numpy(synth.prompt_ids(b, P, dims.vocab, seed=2)).cuda()
    eng.dard_prefill(ids)
    tok, state, conf = (torch.from_numpy(a).cuda() for a in synth.workload_block(b, B, 0.25, dims.vocab, seed=1000))
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.empty(b, B, device="cuda")
    done = torch.empty(b, dtype=torch.int32, device="cuda")
    for _ in range(3):
        eng.dard_step(P, params, tok, state, conf, t_out, s_out, c_out, done)
    torch.cuda.synchronize()
    print("[traffic] 3 steps done", flush=True)
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    print(f"[traffic] copied {COPY_BYTES} bytes", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
