"""Throughput of the DARD hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

Workload: the 8B-shape DARD step -- a random-init LLaDA-8B-like model
(32 layers, d 4096, 32 x 128 MHA, SwiGLU FFN 12288, vocab 126464, bf16),
batch 1, prompt 512, generation 256 in blocks of 32, prefix KV cache, per-step
token states drawn at candidate fraction 0.25, thresholds (0.4, 0.9).

A step is one dard_step call: the augmented-block forward through all 32
layers, the LM head, both confidence passes and both decision phases.  The
timed region runs K steps with inputs resident in HBM, cycling the prefix
length over the 8 blocks of the generation, after one second of untimed
steps that brings the GPU to its steady step time (the first pass from the
start of sustained load is reported beside it).  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DARD decode steps/sec and tokens committed/sec at 8B shape; attention % MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
TRACE_PERIOD = 33             # timing events on one gate/up launch in 33 inside the timed region
TOKENS_PER_STEP = 6.0          # mean tokens decoded per DARD step on LLaDA (App. C.2)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=24)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--burn-in", type=float, default=1.0,
                    help="seconds of untimed steps before the warm-up steps (the first 0.5 s of sustained load "
                         "runs about 3%% slower; the first window of steps is reported as cold_ms_per_step)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the 7B GQA and multimodal full-step lines")
    ap.add_argument("--layers", type=int, default=32, help=argparse.SUPPRESS)
    ap.add_argument("--profile", choices=("ops", "traffic"), default=None,
                    help="run a fixed workload for a profiler pass instead of the benchmark: 'ops' (isolated "
                         "attention, confidence reduction, 7B GQA large-tile steps, a 1 GiB copy) or 'traffic' "
                         "(three 8B-shape steps and a 1 GiB copy, for the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the DARD step is data-parallel "
              f"over sequences and is measured on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_26574_amd import dard, synth

    if args.profile == "ops":
        return profile_ops()
    if args.profile == "traffic":
        return profile_traffic()

    dims = synth.LLADA8B if args.layers == 32 else synth.truncated(synth.LLADA8B, args.layers)
    b, B, prompt, gen, frac = 1, 32, 512, 256, 0.25
    nblocks = gen // B
    cap = prompt + gen + B
    V = dims.vocab
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    log(f"[bench] weights: {dims}")
    t0 = time.time()
    w = synth.make_weights(dims, seed=1, device="cuda")
    eng = dard.Engine(dims, w, b, B, cap)
    del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"[bench] packed weights in {time.time() - t0:.1f}s; workspace {eng.ws.numel() / 2**20:.0f} MiB")

    # prefix cache for the longest prefix; step t reads the prefix of its block
    P_max = prompt + gen - B
    ids = torch.from_numpy(synth.prompt_ids(b, P_max, V, seed=2)).cuda()
    eng.dard_prefill(ids)
    torch.cuda.synchronize()

    total = args.warmup + args.steps
    S_b = math.ceil(B / TOKENS_PER_STEP)
    inputs = []
    for t in range(total):
        tok, state, conf = synth.workload_block(b, B, frac, V, seed=1000 + t)
        inputs.append(tuple(torch.from_numpy(a).cuda() for a in (tok, state, conf)))
    Ps = [prompt + B * ((t // S_b) % nblocks) for t in range(total)]
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device=dev)
    s_out = torch.empty(b, B, dtype=torch.uint8, device=dev)
    c_out = torch.empty(b, B, device=dev)
    done = torch.empty(b, dtype=torch.int32, device=dev)

    def step(t):
        tok, state, conf = inputs[t]
        eng.dard_step(Ps[t], params, tok, state, conf, t_out, s_out, c_out, done)

    # ---- burn-in: from the start of sustained load the GPU takes about half a
    # second to reach its steady step time (4.26 ms per step during the first
    # 0.5 s, 4.14 ms after; idle gaps of up to 3 s do not undo it), so untimed
    # steps run for --burn-in seconds before the warm-up steps.  The first pass
    # over the K steps is timed on its own and reported as the cold-start figure.
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for t in range(args.warmup, total):
        step(t)
    ev1.record()
    torch.cuda.synchronize()
    cold_ms = ev0.elapsed_time(ev1) / args.steps
    tb = time.perf_counter()
    n_burn = 0
    while time.perf_counter() - tb < args.burn_in:
        for t in range(args.warmup, total):
            step(t)
        torch.cuda.synchronize()
        n_burn += args.steps
    log(f"[bench] cold start: {cold_ms:.3f} ms/step; burn-in of {n_burn} steps")

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()

    # ---- timed region: K steps; one gate/up launch in 33 (about one per step,
    # a different layer each step) carries HIP timing events, the begin and
    # end timestamps of the kernel itself (events on every launch would cost
    # a few microseconds each)
    dard.dard_trace_reset()
    dard.dard_trace_sample(TRACE_PERIOD)
    dard.dard_trace_enable(1 << dard.K_GEMM_GU)
    torch.cuda.synchronize()
    ev0.record()
    tw = time.perf_counter()
    for t in range(args.warmup, total):
        step(t)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - tw
    ms_total = ev0.elapsed_time(ev1)
    dard.dard_trace_enable(0)
    n_gu, ms_gu = dard.dard_trace_read(dard.K_GEMM_GU)
    dard.dard_trace_sample(1)
    ms_per_step = ms_total / args.steps
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (wall {1e3 * wall / args.steps:.3f})")

    # ---- per-kernel-class breakdown (a separate traced pass over the same steps)
    dard.dard_trace_reset()
    dard.dard_trace_enable((1 << dard.K_COUNT) - 1)
    for t in range(args.warmup, total):
        step(t)
    torch.cuda.synchronize()
    dard.dard_trace_enable(0)
    names = ["gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "gemm_lm_head", "attention", "confidence",
             "decide", "norm", "mask"]
    breakdown = {}
    for k, nm in enumerate(names):
        n, ms = dard.dard_trace_read(k)
        breakdown[nm] = {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
    dard.dard_trace_reset()

    # ---- roofline of the dominant kernel: gate/up projection with SwiGLU epilogue
    rows = b * 2 * B
    d, F = dims.d_model, dims.ffn_dim
    gu_bytes = 2 * F * d * 2 + rows * d * 2 + rows * F * 2          # weights + X + act
    gu_ms = ms_gu / max(n_gu, 1)
    gu_gbs = gu_bytes / (gu_ms * 1e-3) / 1e9
    roofline = {"kernel": "gemm_stream_bf16 (gate/up + SwiGLU), per launch", "bound": "hbm",
                "achieved": round(gu_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gu_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                "algorithmic_bytes_per_launch": gu_bytes, "avg_launch_us": round(gu_ms * 1e3, 2)}

    # all weight-streaming GEMMs of a step together
    qd, kd = dims.n_heads * dims.head_dim, dims.n_kv_heads * dims.head_dim
    per_layer = (qd + 2 * kd) * d + d * qd + 2 * F * d + d * F
    weight_bytes = 2 * (dims.n_layers * per_layer + V * d)
    gemm_ms = sum(breakdown[k]["ms_per_step"] for k in names[:5])
    kern_ms = sum(v["ms_per_step"] for v in breakdown.values())

    # attention: algorithmic flops / bytes per step (each row sees P + B keys)
    P_avg = sum(Ps[args.warmup:]) / args.steps
    att_flops = 4 * dims.head_dim * dims.n_heads * rows * (P_avg + B) * dims.n_layers
    att_bytes = dims.n_layers * b * dims.n_kv_heads * (P_avg + 2 * B) * dims.head_dim * 2 * 2
    att_ms = breakdown["attention"]["ms_per_step"]
    attention = {"tflops": round(att_flops / (att_ms * 1e-3) / 1e12, 2),
                 "mfma_frac": round(att_flops / (att_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                 "kv_gbs": round(att_bytes / (att_ms * 1e-3) / 1e9, 1),
                 "hbm_frac": round(att_bytes / (att_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                 "ms_per_step": round(att_ms, 4)}

    # ---- the ordering / mixing variants cost: the same steps under each flag
    variants = {}
    for vname, vflags in (("entropy_order", dard.F_ORDER_ENTROPY), ("margin_order", dard.F_ORDER_MARGIN),
                          ("bidirectional", dard.F_C_BIDIR), ("left_to_right", dard.F_ORDER_L2R),
                          ("fixed_w_0.5", dard.F_FIXED_W), ("hidden_mix", dard.F_HIDDEN_MIX)):
        vp = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, vflags, 0.5)

        def vstep(t):
            tok, state, conf = inputs[t]
            eng.dard_step(Ps[t], vp, tok, state, conf, t_out, s_out, c_out, done)
        vstep(args.warmup)
        torch.cuda.synchronize()
        ev0.record()
        for t in range(args.warmup, total):
            vstep(t)
        ev1.record()
        torch.cuda.synchronize()
        variants[vname + "_ms_per_step"] = round(ev0.elapsed_time(ev1) / args.steps, 4)

    # ---- the same steps with the FP8 (E4M3) KV cache (the packed weights shared)
    d8 = synth.with_fp8_kv(dims)
    eng8 = dard.Engine(d8, None, b, B, cap, packed=eng.packed)
    eng8.dard_prefill(ids)

    def step8(t):
        tok, state, conf = inputs[t]
        eng8.dard_step(Ps[t], params, tok, state, conf, t_out, s_out, c_out, done)
    step8(args.warmup)
    torch.cuda.synchronize()
    ev0.record()
    for t in range(args.warmup, total):
        step8(t)
    ev1.record()
    torch.cuda.synchronize()
    variants["fp8_kv_ms_per_step"] = round(ev0.elapsed_time(ev1) / args.steps, 4)
    dard.dard_trace_reset()
    dard.dard_trace_enable(1 << dard.K_ATTENTION)
    for t in range(args.warmup, total):
        step8(t)
    torch.cuda.synchronize()
    dard.dard_trace_enable(0)
    variants["fp8_kv_attention_ms_per_step"] = round(dard.dard_trace_read(dard.K_ATTENTION)[1] / args.steps, 4)
    dard.dard_trace_reset()
    del eng8
    torch.cuda.empty_cache()

    # ---- tokens committed / s: 8 blocks of prefill + ceil(B / 6) steps each
    def generation():
        for k in range(nblocks):
            eng.dard_prefill(ids[:, : prompt + B * k].contiguous())
            for j in range(S_b):
                step(args.warmup + (k * S_b + j) % args.steps)
    generation()
    torch.cuda.synchronize()
    g0 = time.perf_counter()
    generation()
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - g0
    tokens_per_s = b * gen / gen_s

    # the same generation with the extend-only refresh at block boundaries:
    # the prompt prefilled once, each finished block appended with
    # dard_prefill_extend (an approximation of the re-encoding above)
    def generation_extend():
        for k in range(nblocks):
            if k == 0:
                eng.dard_prefill(ids[:, :prompt].contiguous())
            else:
                P0 = prompt + B * (k - 1)
                eng.dard_prefill_extend(P0, ids[:, P0:P0 + B].contiguous())
            for j in range(S_b):
                step(args.warmup + (k * S_b + j) % args.steps)
    generation_extend()
    torch.cuda.synchronize()
    g0 = time.perf_counter()
    generation_extend()
    torch.cuda.synchronize()
    tokens_per_s_ext = b * gen / (time.perf_counter() - g0)

    out = {
        "metric": METRIC, "value": round(1e3 / ms_per_step, 2), "unit": "steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "cold_ms_per_step": round(cold_ms, 4),
        "burn_in": f"{n_burn} untimed steps ({args.burn_in:g} s) before the warm-up; cold_ms_per_step is the "
                   f"first pass over the same {args.steps} steps from the start of sustained load",
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded random-init weights N(0, 0.02), uniform prompt ids, drawn token states",
        "config": {"workload": f"llada8b-like full DARD step: {dims.n_layers} layers, d 4096, 32x128 MHA, FFN 12288, "
                               "vocab 126464, bf16; batch 1, prompt 512, generation 256, block 32, "
                               "candidate fraction 0.25, prefix KV cache",
                   "batch": b, "block": B, "prompt": prompt, "gen_len": gen, "cand_frac": frac,
                   "layers": dims.n_layers},
        "tokens_committed_per_s": round(tokens_per_s, 1),
        "tokens_committed_note": f"{nblocks} blocks x (prefill + {S_b} steps), 6.0 tokens/step as reported",
        "tokens_committed_per_s_extend_refresh": round(tokens_per_s_ext, 1),
        "tokens_committed_extend_note": "the prompt prefilled once, each finished block appended to the prefix "
                                        "cache (dard_prefill_extend: its rows see the cached keys) instead of "
                                        "re-encoding prompt + committed blocks; an approximation",
        "roofline": roofline,
        "weight_stream": {"gb_per_step": round(weight_bytes / 1e9, 3), "gemm_ms_per_step": round(gemm_ms, 4),
                          "gbs": round(weight_bytes / (gemm_ms * 1e-3) / 1e9, 1)},
        "attention": attention,
        "breakdown_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in breakdown.items()},
        "kernel_ms_per_step": round(kern_ms, 4),
        "gaps_ms_per_step": round(ms_per_step - kern_ms, 4),
        "variants": variants,
    }
    out["decision_driven"] = decision_driven(eng, dims, ids, b, B, prompt)
    out["ops"] = op_measurements()
    if not args.no_configs and args.layers == 32:
        out["configs"] = full_step_configs(eng)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(dims, b, B, prompt, frac)
    # attention against the bf16 MFMA peak per workload (kernel time): the
    # headline decode step (64 query rows per MHA head, about 55 flop per K/V
    # byte: bound by HBM and latency, not by the matrix cores) and the
    # isolated operations, of which the 7B GQA shape (7 query heads per KV
    # head, block 64) is the MFMA-bound one
    by_workload = {"8B step, batch 1 (in the step)": attention["mfma_frac"]}
    for a in out["ops"]["attention"]:
        key = f"{a['shape']}, batch {a['batch']}, prefix {a['prefix']}, cand {a.get('cand_frac')}"
        by_workload[key] = a["mfma_frac"]
    for name, cfg in out.get("configs", {}).items():
        if "attention_mfma_frac" in cfg:
            by_workload[f"{name} (in the step)"] = cfg["attention_mfma_frac"]
    out["attention_mfma_frac_by_workload"] = by_workload
    print(json.dumps(out), flush=True)


def decision_driven(eng, dims, ids, b, B, prompt, nblocks=2):
    """Diagnostic: blocks decoded by the decisions themselves.  Each block
    starts all-[Mask]; every step feeds its outputs back as the next inputs,
    with the progress rule on (DARD_F_PROGRESS: a step that commits no token
    commits the most confident one) and a cap of 2B steps per block.  With
    random-init weights no confidence passes tau_u and committed tokens fall
    back on re-verification, so blocks run to the cap: this measures the
    decoding loop's mechanics, not the paper's tokens per step."""
    import torch

    from paper_2608_26574_amd import dard
    F_PROGRESS = 1 << 3
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, F_PROGRESS)
    dev = ids.device
    bufs = [(torch.empty(b, B, dtype=torch.int32, device=dev), torch.empty(b, B, dtype=torch.uint8, device=dev),
             torch.empty(b, B, device=dev)) for _ in range(2)]
    done = torch.zeros(b, dtype=torch.int32, device=dev)
    steps, capped = [], 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(nblocks):
        P = prompt + B * k
        eng.dard_prefill(ids[:, :P].contiguous())
        tok, st, cf = bufs[0]
        tok.fill_(dims.mask_id)
        st.zero_()
        cf.zero_()
        n = 0
        while True:
            src, dst = bufs[n % 2], bufs[(n + 1) % 2]
            eng.dard_step(P, params, src[0], src[1], src[2], dst[0], dst[1], dst[2], done)
            n += 1
            if int(done.min().item()) == 1:
                break
            if n >= 2 * B:
                capped += 1
                break
        steps.append(n)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    return {"blocks": nblocks, "steps_per_block": steps, "capped_blocks": capped,
            "tokens_per_s": round(b * B * nblocks / el, 1),
            "note": "progress rule on, cap 2B steps; random-init weights, so blocks reach the cap"}


def full_step_configs(eng8b, steps=6):
    """The two other full-step workloads, measured the same way as the headline
    step (HIP events around `steps` dard_step calls with inputs resident;
    prefix lengths cycling over the generation's blocks; per-step states drawn
    at the workload's candidate fraction), plus tokens committed/s over a whole
    generation (prefill at every block start + ceil(B / r) steps per block,
    r = the paper's mean tokens decoded per step):
    - 7B GQA shape: Dream-7B-like random-init model (28 layers, d 3584, 28/4
      heads x 128, FFN 18944, vocab 152064, bf16), batch 8, prompt 1024,
      generation 512 in blocks of 64, candidate fraction 0.3, r = 6.0;
    - multimodal prefix at the 8B shape (the headline model's packed weights,
      shared): batch 32, 576 image-embedding positions N(0, 1) + 256 prompt
      ids, generation 128 in blocks of 32, candidate fraction swept 0.1 / 0.3 /
      0.5, r = 8.8 (the paper's MMaDA figure).
    At 1024 and 2048 rows per step every projection is a compute-bound MFMA
    GEMM; the report gives the GEMMs' achieved TFLOP/s (2 params rows per step
    over their traced time) and the attention's, against the bf16 MFMA peak."""
    import torch

    from paper_2608_26574_amd import dard, synth

    def run(eng, dims, b, B, prompt, gen, fracs, r_tok, ids, embeds, label):
        V = dims.vocab
        nblocks = gen // B
        S_b = math.ceil(B / r_tok)
        params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
        dev = ids.device
        t_out = torch.empty(b, B, dtype=torch.int32, device=dev)
        s_out = torch.empty(b, B, dtype=torch.uint8, device=dev)
        c_out = torch.empty(b, B, device=dev)
        done = torch.empty(b, dtype=torch.int32, device=dev)
        P_last = prompt + gen - B
        log(f"[bench] {label}: prefill of {b} x {P_last}")
        eng.dard_prefill(ids[:, :P_last].contiguous(), None if embeds is None else embeds[:, :P_last].contiguous())
        torch.cuda.synchronize()
        res = {"per_frac": []}
        for frac in fracs:
            ins = []
            for t in range(steps + 1):
                tok, state, conf = synth.workload_block(b, B, frac, V, seed=2000 + t)
                ins.append(tuple(torch.from_numpy(a_).cuda() for a_ in (tok, state, conf)))
            Ps = [prompt + B * (t % nblocks) for t in range(steps + 1)]

            def step(t):
                eng.dard_step(Ps[t], params, *ins[t], t_out, s_out, c_out, done)
            step(steps)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for t in range(steps):
                step(t)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            res["per_frac"].append({"cand_frac": frac, "ms_per_step": round(ms, 3), "steps_per_s": round(1e3 / ms, 2)})
            if frac == fracs[len(fracs) // 2]:
                dard.dard_trace_reset()
                dard.dard_trace_enable((1 << dard.K_COUNT) - 1)
                for t in range(steps):
                    step(t)
                torch.cuda.synchronize()
                dard.dard_trace_enable(0)
                names = ["gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "gemm_lm_head", "attention"]
                bd = {nm: dard.dard_trace_read(k)[1] / steps for k, nm in enumerate(names)}
                dard.dard_trace_reset()
                rows = b * 2 * B
                qd, kd = dims.n_heads * dims.head_dim, dims.n_kv_heads * dims.head_dim
                params_n = dims.n_layers * ((qd + 2 * kd) * dims.d_model + dims.d_model * qd +
                                            3 * dims.ffn_dim * dims.d_model) + V * dims.d_model
                gemm_ms = sum(bd[n] for n in names[:5])
                P_avg = sum(Ps[:steps]) / steps
                att_fl = 4 * dims.head_dim * dims.n_heads * rows * (P_avg + B) * dims.n_layers
                res["breakdown_ms_per_step"] = {k_: round(v, 3) for k_, v in bd.items()}
                res["gemm_tflops"] = round(2 * params_n * rows / (gemm_ms * 1e-3) / 1e12, 1)
                res["gemm_mfma_frac"] = round(2 * params_n * rows / (gemm_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)
                res["attention_tflops"] = round(att_fl / (bd["attention"] * 1e-3) / 1e12, 1)
                res["attention_mfma_frac"] = round(att_fl / (bd["attention"] * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)
        # the same steps with Eq. 7 applied to the hidden state (two LM-head passes, B rows per sequence)
        frac = fracs[len(fracs) // 2]
        hp = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, dard.F_HIDDEN_MIX)
        hins = [tuple(torch.from_numpy(a_).cuda() for a_ in synth.workload_block(b, B, frac, V, seed=2000 + t))
                for t in range(steps + 1)]
        Ph = [prompt + B * (t % nblocks) for t in range(steps + 1)]
        eng.dard_step(Ph[steps], hp, *hins[steps], t_out, s_out, c_out, done)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t in range(steps):
            eng.dard_step(Ph[t], hp, *hins[t], t_out, s_out, c_out, done)
        e1.record()
        torch.cuda.synchronize()
        res["hidden_mix_ms_per_step"] = round(e0.elapsed_time(e1) / steps, 3)
        dard.dard_trace_reset()
        dard.dard_trace_enable(1 << dard.K_GEMM_HEAD)
        for t in range(steps):
            eng.dard_step(Ph[t], hp, *hins[t], t_out, s_out, c_out, done)
        torch.cuda.synchronize()
        dard.dard_trace_enable(0)
        res["hidden_mix_lm_head_ms_per_step"] = round(dard.dard_trace_read(dard.K_GEMM_HEAD)[1] / steps, 3)
        dard.dard_trace_reset()
        # tokens committed / s over one generation (the middle candidate fraction's states)
        ins = [tuple(torch.from_numpy(a_).cuda() for a_ in synth.workload_block(b, B, frac, V, seed=3000 + j))
               for j in range(S_b)]
        torch.cuda.synchronize()
        g0 = time.perf_counter()
        for k in range(nblocks):
            P = prompt + B * k
            eng.dard_prefill(ids[:, :P].contiguous(), None if embeds is None else embeds[:, :P].contiguous())
            for j in range(S_b):
                eng.dard_step(P, params, *ins[j], t_out, s_out, c_out, done)
        torch.cuda.synchronize()
        el = time.perf_counter() - g0
        res["tokens_committed_per_s"] = round(b * gen / el, 1)
        res["tokens_committed_note"] = f"{nblocks} blocks x (prefill + {S_b} steps), {r_tok} tokens/step as reported"
        return res

    def library_gemm_us(M, N, K, reps=20):
        """torch.matmul (hipBLASLt) of bf16 [M, K] x [K, N], weight copies
        rotated through >= 600 MB so that no launch finds its weights cached."""
        g = torch.Generator(device="cuda").manual_seed(7)
        x = torch.randn(M, K, generator=g, device="cuda").bfloat16()
        ncopy = max(2, -(-600 * 2**20 // (N * K * 2)))
        ws = [torch.randn(K, N, generator=g, device="cuda").bfloat16() for _ in range(ncopy)]
        y = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        for i in range(3):
            torch.matmul(x, ws[i % ncopy], out=y)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            torch.matmul(x, ws[i % ncopy], out=y)
        e1.record()
        torch.cuda.synchronize()
        del ws
        return e0.elapsed_time(e1) / reps * 1e3

    def versus_library(dims, rows, bd):
        """Each projection's kernel time per launch in the step (its traced
        class time over the layers; QKV with RoPE and the cache writes, O and
        down as split-K partials, gate/up with SwiGLU) beside a plain library
        GEMM of the same shape."""
        qd, kd = dims.n_heads * dims.head_dim, dims.n_kv_heads * dims.head_dim
        shapes = {"gemm_qkv": (qd + 2 * kd, dims.d_model), "gemm_o": (dims.d_model, qd),
                  "gemm_gate_up": (2 * dims.ffn_dim, dims.d_model), "gemm_down": (dims.d_model, dims.ffn_dim)}
        res = []
        for nm, (N, K) in shapes.items():
            ours = bd[nm] / dims.n_layers * 1e3
            lib = library_gemm_us(rows, N, K)
            fl = 2.0 * rows * N * K
            res.append({"gemm": nm[5:], "M": rows, "N": N, "K": K, "ours_us": round(ours, 1),
                        "hipblaslt_us": round(lib, 1), "ours_over_hipblaslt": round(ours / lib, 3),
                        "ours_mfma_frac": round(fl / (ours * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
                        "hipblaslt_mfma_frac": round(fl / (lib * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)})
        return res

    out = {}
    # ---- 7B GQA shape
    d7 = synth.DREAM7B
    b, B, prompt, gen = 8, 64, 1024, 512
    w = synth.make_weights(d7, seed=1, device="cuda")
    eng7 = dard.Engine(d7, w, b, B, prompt + gen + B)
    del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    ids = torch.from_numpy(synth.prompt_ids(b, prompt + gen - B, d7.vocab, seed=2)).cuda()
    r7 = run(eng7, d7, b, B, prompt, gen, [0.3], 6.0, ids, None, "7B GQA")
    out["dream7b_gqa"] = {"workload": "dream7b-like full DARD step: 28 layers, d 3584, 28/4 x 128 GQA, FFN 18944, "
                                      "vocab 152064, bf16; batch 8, prompt 1024, generation 512, block 64, "
                                      "candidate fraction 0.3, prefix KV cache", **r7}
    del eng7, ids
    torch.cuda.empty_cache()
    vs_lib = {"dream7b_gqa_1024_rows": versus_library(d7, 8 * 2 * 64, r7["breakdown_ms_per_step"])}
    # ---- multimodal prefix at the 8B shape (weights shared with the headline engine)
    d8 = synth.LLADA8B
    b, B, n_img, n_txt, gen = 32, 32, 576, 256, 128
    prompt = n_img + n_txt
    engm = dard.Engine(d8, None, b, B, prompt + gen + B, packed=eng8b.packed)
    ids = torch.from_numpy(synth.prompt_ids(b, prompt + gen - B, d8.vocab, seed=5)).cuda()
    ids[:, :n_img] = -1
    g = torch.Generator(device="cuda").manual_seed(6)
    embeds = torch.randn(b, prompt + gen - B, d8.d_model, generator=g, device="cuda").bfloat16()
    rm = run(engm, d8, b, B, prompt, gen, [0.1, 0.3, 0.5], 8.8, ids, embeds, "multimodal")
    out["multimodal_8b"] = {"workload": "llada8b-like full DARD step with a multimodal prefix: 576 image-embedding "
                                        "positions N(0, 1) + 256 prompt ids; batch 32, generation 128, block 32, "
                                        "candidate fraction 0.1 / 0.3 / 0.5, prefix KV cache", **rm}
    del engm
    torch.cuda.empty_cache()
    vs_lib["multimodal_8b_2048_rows"] = versus_library(d8, 32 * 2 * 32, rm["breakdown_ms_per_step"])
    out["gemm_vs_hipblaslt"] = vs_lib
    # the same workload with the FP8 (E4M3) KV cache
    d8f = synth.with_fp8_kv(d8)
    engf = dard.Engine(d8f, None, b, B, prompt + gen + B, packed=eng8b.packed)
    rf = run(engf, d8f, b, B, prompt, gen, [0.3], 8.8, ids, embeds, "multimodal, FP8 KV")
    out["multimodal_8b_fp8_kv"] = {"workload": "as multimodal_8b with the KV cache in OCP FP8 E4M3, candidate "
                                               "fraction 0.3", **rf}
    del engf, ids, embeds
    torch.cuda.empty_cache()
    out["multimodal_8b_shared_prompt"] = shared_prompt_workload(eng8b, steps)
    out["paper_latency_8b"] = paper_latency_workload(eng8b, steps)
    return out


def shared_prompt_workload(eng8b, steps=6):
    """The multimodal workload with one prompt for the whole batch (the same
    image and text): the 576-embedding + 256-id prompt is prefilled once
    (dard_prefill, b = 1) and shared; each block start prefills only the
    sequences' committed positions (dard_prefill_suffix); steps read the
    shared keys in place (dard_step_shared).  Batch 32, generation 128 in
    blocks of 32, candidate fraction 0.3, 8.8 tokens per step as for the
    unshared line."""
    import torch

    from paper_2608_26574_amd import dard, synth

    d8 = synth.LLADA8B
    b, B, n_img, n_txt, gen, frac, r_tok = 32, 32, 576, 256, 128, 0.3, 8.8
    Ps = n_img + n_txt
    nblocks = gen // B
    S_b = math.ceil(B / r_tok)
    sh = dard.Engine(d8, None, 1, B, Ps, packed=eng8b.packed)
    eng = dard.Engine(d8, None, b, B, Ps + gen + B, packed=eng8b.packed)
    prompt = torch.from_numpy(synth.prompt_ids(1, Ps, d8.vocab, seed=5)).cuda()
    prompt[:, :n_img] = -1
    g = torch.Generator(device="cuda").manual_seed(6)
    embeds = torch.randn(1, Ps, d8.d_model, generator=g, device="cuda").bfloat16()
    committed = torch.from_numpy(synth.prompt_ids(b, gen - B, d8.vocab, seed=8)).cuda()
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, d8.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.empty(b, B, device="cuda")
    done = torch.empty(b, dtype=torch.int32, device="cuda")
    ins = [tuple(torch.from_numpy(a_).cuda() for a_ in synth.workload_block(b, B, frac, d8.vocab, seed=5000 + t))
           for t in range(steps + 1)]
    sh.dard_prefill(prompt, embeds)
    eng.dard_prefill_suffix(sh, Ps, committed.contiguous())
    torch.cuda.synchronize()
    Pt = [Ps + B * (t % nblocks) for t in range(steps + 1)]

    def step(t):
        eng.dard_step_shared(sh, Ps, Pt[t], params, *ins[t], t_out, s_out, c_out, done)
    step(steps)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for t in range(steps):
        step(t)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    dard.dard_trace_reset()
    dard.dard_trace_enable(1 << dard.K_ATTENTION)
    for t in range(steps):
        step(t)
    torch.cuda.synchronize()
    dard.dard_trace_enable(0)
    att_ms = dard.dard_trace_read(dard.K_ATTENTION)[1] / steps
    dard.dard_trace_reset()
    # a whole generation: the shared prompt once, then per block the committed
    # positions and ceil(B / r) steps
    torch.cuda.synchronize()
    g0 = time.perf_counter()
    sh.dard_prefill(prompt, embeds)
    for k in range(nblocks):
        if k:
            eng.dard_prefill_suffix(sh, Ps, committed[:, :B * k].contiguous())
        for j in range(S_b):
            eng.dard_step_shared(sh, Ps, Ps + B * k, params, *ins[j % steps], t_out, s_out, c_out, done)
    torch.cuda.synchronize()
    el = time.perf_counter() - g0
    res = {"workload": "llada8b-like DARD step, batch 32 sharing one prompt (576 image-embedding positions N(0, 1) + "
                       "256 ids, cached once), generation 128, block 32, candidate fraction 0.3",
           "ms_per_step": round(ms, 3), "steps_per_s": round(1e3 / ms, 2), "attention_ms_per_step": round(att_ms, 3),
           "tokens_committed_per_s": round(b * gen / el, 1),
           "tokens_committed_note": f"shared prompt prefill once + {nblocks} blocks x (suffix prefill + {S_b} steps)"}
    del sh, eng
    torch.cuda.empty_cache()
    return res


def paper_latency_workload(eng8b, steps=6):
    """The setting of the paper's single-step latency table (App. C.5), at the
    8B shape (the headline model's packed weights, shared): full-sequence steps
    (dard_step_full: prompt + the whole generation with future [Mask] blocks +
    the shadow block, no prefix cache), batch 1, a 256-token prompt standing in
    for a MATH-500 prompt, generation 256, candidate fraction 0.25; block 128
    (the current block first, with one future block, and last) and block 256
    (the whole generation one block).  The paper's figures (186.8 ms per step
    at block 128 and 232.0 ms at block 256 on an RTX A6000) are context from
    other hardware, not a target."""
    import torch

    from paper_2608_26574_amd import dard, synth

    d8 = synth.LLADA8B
    b, prompt, gen, frac = 1, 256, 256, 0.25
    N = prompt + gen
    seq0 = torch.from_numpy(synth.prompt_ids(b, N, d8.vocab, seed=7)).cuda()
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, d8.mask_id, 0)
    res = {"workload": "llada8b-like full-sequence DARD step (no prefix cache): batch 1, prompt 256, generation 256, "
                       "blocks of 128 and of 256, candidate fraction 0.25",
           "paper_context": "186.8 ms/step at block 128, 232.0 ms at block 256 (RTX A6000, LLaDA-8B, MATH-500)"}
    for B in (128, 256):
        eng = dard.Engine(d8, None, b, B, N + B, packed=eng8b.packed)
        t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
        s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
        c_out = torch.empty(b, B, device="cuda")
        done = torch.empty(b, dtype=torch.int32, device="cuda")
        ms_blocks = []
        for k in range(gen // B):
            blk = prompt + k * B
            ins = []
            for t in range(steps + 1):
                tok, state, conf = synth.workload_block(b, B, frac, d8.vocab, seed=4000 + t)
                sq = seq0.clone()
                sq[:, blk + B:] = d8.mask_id
                sq[:, blk:blk + B] = torch.from_numpy(tok).cuda()
                ins.append((sq, torch.from_numpy(state).cuda(), torch.from_numpy(conf).cuda()))

            def step(t):
                eng.dard_step_full(blk, params, ins[t][0], ins[t][1], ins[t][2], t_out, s_out, c_out, done)
            step(steps)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for t in range(steps):
                step(t)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            ms_blocks.append(ms)
            res[f"block{B}_{'first' if k == 0 else 'last'}_ms_per_step"] = round(ms, 3)
        # tokens committed / s over the generation at the paper's 6.0 tokens per step
        S_b = math.ceil(B / TOKENS_PER_STEP)
        res[f"block{B}_tokens_committed_per_s"] = round(b * gen / (S_b * sum(ms_blocks) * 1e-3), 1)
        del eng
        torch.cuda.empty_cache()
    res["tokens_committed_note"] = "gen / (ceil(B / 6.0) steps per block x the measured per-step times)"
    return res


def op_measurements(reps=20):
    """The two isolated operations the roofline targets name, measured cold
    (inputs rotated through copies whose total exceeds the 256 MB MALL):
    - state-masked attention, bf16 Q/K/V ~ N(0, 1), against the bf16 MFMA peak
      (algorithmic flops 4 dh Hq 2B (P+B) b: each query row reads P + B keys)
      and the HBM peak (K/V of P+2B keys, Q and O), at the 8B attention shape
      (32 x 128 MHA heads, prompt KV 512, block 32, candidate fraction 0.25;
      batch 1, 4, 16) and at the 7B GQA shape (28 query heads on 4 KV heads,
      batch 8, block 64, candidate fraction 0.3, prefix 1024 and 1472: the
      first and last block of a 512-token generation), the one where attention
      is compute-bound.  `us` is the whole call (state mask + attention
      kernels, HIP events around the calls); `kernel_us` the attention
      kernels alone (kernel timestamps), since a step builds the mask once for
      all its layers; mfma_frac uses kernel_us;
    - the vocab-wide confidence reduction (argmax, max-prob) over fp32 logits
      at the 8B step's row count (B + |M| = 44 rows x 126464) and at the 7B GQA
      batch-8 step's (8 x 87 rows x 152064), against the HBM peak."""
    import torch

    from paper_2608_26574_amd import dard, synth

    def timed(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn(0)
        torch.cuda.synchronize()
        e0.record()
        for i in range(n):
            fn(i + 1)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def traced(fn, n, cls):
        dard.dard_trace_reset()
        dard.dard_trace_enable(1 << cls)
        for i in range(n):
            fn(i + 1)
        torch.cuda.synchronize()
        dard.dard_trace_enable(0)
        _, ms = dard.dard_trace_read(cls)
        dard.dard_trace_reset()
        return ms / n

    res = {"attention": [], "confidence": []}
    # the isolated-attention workload: batch 1 / 4 / 16 x candidate fraction 0.1 / 0.25 / 0.5
    shapes = [("8B MHA", bsz, 32, 32, 32, 512, frac) for bsz in (1, 4, 16) for frac in (0.1, 0.25, 0.5)] + \
             [("7B GQA", 8, 28, 4, 64, P, 0.3) for P in (1024, 1472)] + \
             [("8B MHA, FP8 KV", bsz, 32, 32, 32, 512, 0.25) for bsz in (1, 4, 16)] + \
             [("7B GQA, FP8 KV", 8, 28, 4, 64, 1024, 0.3)]
    dh = 128
    for label, bsz, H, Hkv, B, P, frac in shapes:
        fp8 = "FP8" in label
        kvb = 1 if fp8 else 2                       # bytes per cached value
        cap = P + 2 * B
        kv_bytes = bsz * Hkv * cap * dh * kvb
        ncopy = max(4, -(-600 * 2**20 // (2 * kv_bytes)))
        g = torch.Generator(device="cuda").manual_seed(2)
        q = torch.randn(bsz, 2 * B, H, dh, generator=g, device="cuda").bfloat16()

        def kvt(shape):
            x = torch.randn(shape, generator=g, device="cuda").bfloat16()
            # FP8: random E4M3 codes of magnitude below 16 (exponent field < 11), either sign
            return torch.randint(0, 88, shape, generator=g, device="cuda", dtype=torch.int32).to(torch.uint8) | \
                (torch.randint(0, 2, shape, generator=g, device="cuda", dtype=torch.int32) * 128).to(torch.uint8) \
                if fp8 else x
        ks = [kvt((bsz, Hkv, cap, dh)) for _ in range(ncopy)]
        vs = [kvt((bsz, Hkv, dh, cap)) for _ in range(ncopy)]
        _, state, conf = synth.workload_block(bsz, B, frac, 100, seed=3)
        state, conf = torch.from_numpy(state).cuda(), torch.from_numpy(conf).cuda()
        out = torch.empty_like(q)
        ws = torch.empty(max(dard.dard_attention_workspace_bytes(2 if fp8 else 1, bsz, B, H, dh, P), 1),
                         dtype=torch.uint8, device="cuda")

        def att(i):
            dard.dard_masked_attention(q, ks[i % ncopy], vs[i % ncopy], P, state, conf, dh ** -0.5, 0, out, ws)
        ms = timed(att, reps)
        kms = traced(att, reps, dard.K_ATTENTION)
        flops = 4 * dh * H * 2 * B * (P + B) * bsz
        nbytes = 2 * bsz * Hkv * (P + 2 * B) * dh * kvb + 2 * q.numel() * 2
        res["attention"].append({"shape": label, "batch": bsz, "heads": [H, Hkv], "block": B, "prefix": P,
                                 "cand_frac": frac,
                                 "us": round(ms * 1e3, 2), "kernel_us": round(kms * 1e3, 2),
                                 "tflops": round(flops / (kms * 1e-3) / 1e12, 2),
                                 "mfma_frac": round(flops / (kms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                                 "gbs": round(nbytes / (kms * 1e-3) / 1e9, 1),
                                 "hbm_frac": round(nbytes / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)})
        del ks, vs
    for rows, V, label in ((44, 126464, "8B step, 44 rows"), (8 * 87, 152064, "7B GQA batch-8 step, 696 rows")):
        nbytes = rows * V * 4
        ncopy = max(2, -(-600 * 2**20 // nbytes))
        g = torch.Generator(device="cuda").manual_seed(4)
        ls = [torch.randn(rows, V, generator=g, device="cuda") for _ in range(ncopy)]
        am = torch.empty(rows, dtype=torch.int32, device="cuda")
        mp = torch.empty(rows, device="cuda")
        ws = torch.empty(max(dard.dard_confidence_workspace_bytes(rows, V), 1), dtype=torch.uint8, device="cuda")

        ent = torch.empty(rows, device="cuda")
        mrg = torch.empty(rows, device="cuda")

        def cf(i):
            dard.dard_confidence(ls[i % ncopy], am, mp, ws=ws)

        def cf_stats(i):   # with the entropy / margin scores of the ordering variants
            dard.dard_confidence(ls[i % ncopy], am, mp, ws=ws, entropy=ent, margin=mrg)
        ms = timed(cf, reps)
        ms_st = timed(cf_stats, reps)
        res["confidence"].append({"shape": label, "us": round(ms * 1e3, 2),
                                  "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                                  "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                  "entropy_margin_us": round(ms_st * 1e3, 2),
                                  "entropy_margin_hbm_frac": round(nbytes / (ms_st * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                                                   4)})
        del ls
    torch.cuda.empty_cache()
    return res


def measured_traffic():
    """HBM bytes per gate/up launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), or None when the GEMM
    sources changed since the counters were taken."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    try:
        text = open(os.path.join(root, "profiles", "gate_up_gemm_hbm_traffic.md")).read()
        h = hashlib.sha256()
        for f in ("gemm.hip", "common.h", "launch.h"):
            h.update(open(os.path.join(root, "paper_2608_26574_amd", "csrc", f), "rb").read())
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if line.count(": ") == 1 and " " not in line.split(": ")[0])
    if fields.get("source_sha256", "").strip() != h.hexdigest():
        return None
    return int(fields["traffic_bytes_per_launch"])


def cpu_baseline(dims, b, B, P, frac, layers_made=2, min_s=10.0):
    """The CPU oracle on a bounded sample of the same workload: whole DARD
    steps at full depth (embedding, all layers, final norm, LM head,
    decisions), repeated for at least min_s seconds.  Only two layers' weights
    are generated and converted to float64, and the full depth cycles through
    them: a layer's cost does not depend on its values, and 32 distinct
    float64 layers of the 8B shape would need about 56 GB of host memory.
    Inputs are seeded and synthetic (the prefix KV cache is random of the
    right shape, one per generated layer, cycled the same way)."""
    import torch
    from threadpoolctl import threadpool_info

    from oracle import dard_oracle as O
    from paper_2608_26574_amd import synth

    sub = synth.truncated(dims, layers_made)
    w = synth.make_weights(sub, seed=1, device="cuda")
    ow = synth.OracleWeights(sub, w)
    g = torch.Generator(device="cuda").manual_seed(7)
    made = []
    for _ in range(layers_made):
        k = torch.randn(b, P, sub.n_kv_heads, sub.head_dim, generator=g, device="cuda").bfloat16()
        v = torch.randn(b, P, sub.n_kv_heads, sub.head_dim, generator=g, device="cuda").bfloat16()
        made.append((k.double().cpu().numpy(), v.double().cpu().numpy()))
    tok, state, conf = synth.workload_block(b, B, frac, sub.vocab, seed=1000)
    params = dict(tau_c=0.4, tau_u=0.9, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=sub.mask_id)
    # weights are converted to float64 once, outside the timed sample
    converted = [ow.layers[i] for i in range(layers_made)]
    layers = [converted[i % layers_made] for i in range(dims.n_layers)]
    cache = [made[i % layers_made] for i in range(dims.n_layers)]
    wd = {"embed": ow["embed"], "final_norm": ow["final_norm"], "lm_head": ow["lm_head"], "layers": layers}
    dd = dims.as_dict()

    n, t0 = 0, time.perf_counter()
    while True:
        O.dard_step(wd, dd, cache, tok, state, conf, params)
        n += 1
        el = time.perf_counter() - t0
        if el >= min_s:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(n / el, 5), "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "cpu_model": cpu_model,
            "sample": f"{n} whole oracle DARD steps at full depth ({dims.n_layers} layers, LM head and decisions) "
                      f"in {el:.1f} s; the layers cycle through {layers_made} generated layers' weights",
            "host_cpus": os.cpu_count()}


# ---------------------------------------------------------------- profiler workloads
COPY_BYTES = 1 << 30


def _copy_calibration(tag):
    """One plain device-to-device copy of COPY_BYTES: its kernel calibrates the
    byte counters (a copy of S bytes reads S and writes S bytes of HBM)."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[{tag}] copied {COPY_BYTES} bytes")


def profile_traffic():
    """Three DARD steps at the 8B shape (32 layers, batch 1, block 32, prompt
    512) and one 1 GiB copy, for rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE."""
    import torch

    from paper_2608_26574_amd import dard, synth
    dims = synth.LLADA8B
    b, B, P, cap = 1, 32, 512, 800
    log("[traffic] packing weights")
    w = synth.make_weights(dims, seed=1, device="cuda")
    eng = dard.Engine(dims, w, b, B, cap)
    del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    eng.dard_prefill(torch.from_numpy(synth.prompt_ids(b, P, dims.vocab, seed=2)).cuda())
    tok, state, conf = (torch.from_numpy(a).cuda() for a in synth.workload_block(b, B, 0.25, dims.vocab, seed=1000))
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.empty(b, B, device="cuda")
    done = torch.empty(b, dtype=torch.int32, device="cuda")
    for _ in range(3):
        eng.dard_step(P, params, tok, state, conf, t_out, s_out, c_out, done)
    torch.cuda.synchronize()
    log("[traffic] 3 steps done")
    _copy_calibration("traffic")
    return 0


def profile_ops():
    """The isolated operations for counter passes, inputs rotated through
    copies larger than the 256 MB MALL: 10 attention calls at the 7B GQA
    shape (28/4 heads x 128, batch 8, block 64, prefix 1024, candidate
    fraction 0.3), 10 at the 8B MHA shape (32 x 128, batch 16, prefix 512,
    block 32, fraction 0.25), 10 confidence reductions over 696 x 152064
    fp32 logits, 3 steps of the 7B GQA model truncated to 2 layers at batch 8
    (1024 token rows: the large-tile GEMMs), 3 library GEMMs (torch.matmul) of
    each of its four projection shapes at 1024 rows, then a 1 GiB copy."""
    import torch

    from paper_2608_26574_amd import dard, synth

    def attention(b, Hq, Hkv, B, P, frac, calls, seed):
        dh, cap = 128, P + 2 * B
        g = torch.Generator(device="cuda").manual_seed(seed)
        ncopy = max(2, -(-600 * 2**20 // (2 * b * Hkv * cap * dh * 2)))
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
        ncopy = max(2, -(-600 * 2**20 // (rows * V * 4)))
        g = torch.Generator(device="cuda").manual_seed(4)
        ls = [torch.randn(rows, V, generator=g, device="cuda") for _ in range(ncopy)]
        am = torch.empty(rows, dtype=torch.int32, device="cuda")
        mp = torch.empty(rows, device="cuda")
        ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
        for i in range(calls):
            dard.dard_confidence(ls[i % ncopy], am, mp, ws=ws)
        torch.cuda.synchronize()

    attention(8, 28, 4, 64, 1024, 0.3, 10, seed=1)
    log("[ops] GQA attention done")
    attention(16, 32, 32, 32, 512, 0.25, 10, seed=2)
    log("[ops] MHA attention done")
    confidence(8 * 87, 152064, 10)
    log("[ops] confidence done")
    dims = synth.truncated(synth.DREAM7B, 2)
    b, B, P = 8, 64, 1024
    w = synth.make_weights(dims, seed=1, device="cuda")
    eng = dard.Engine(dims, w, b, B, P + 2 * B)
    del w
    eng.dard_prefill(torch.from_numpy(synth.prompt_ids(b, P, dims.vocab, seed=2)).cuda())
    tok, state, conf = (torch.from_numpy(a).cuda() for a in synth.workload_block(b, B, 0.3, dims.vocab, seed=3))
    params = dard.make_params(0.4, 0.9, 0.5 ** 0.125, 0.1, dims.mask_id, 0)
    t_out = torch.empty(b, B, dtype=torch.int32, device="cuda")
    s_out = torch.empty(b, B, dtype=torch.uint8, device="cuda")
    c_out = torch.empty(b, B, device="cuda")
    for _ in range(3):
        eng.dard_step(P, params, tok, state, conf, t_out, s_out, c_out)
    torch.cuda.synchronize()
    log("[ops] 7B GQA steps done")
    del eng
    torch.cuda.empty_cache()
    # the library's GEMMs (torch.matmul, hipBLASLt) on the same step shapes
    # (1024 rows), weight copies rotated through >= 600 MB, 3 calls each
    g = torch.Generator(device="cuda").manual_seed(7)
    for N, K in ((4608, 3584), (3584, 3584), (37888, 3584), (3584, 18944)):
        x = torch.randn(1024, K, generator=g, device="cuda").bfloat16()
        ncopy = max(2, -(-600 * 2**20 // (N * K * 2)))
        ws = [torch.randn(K, N, generator=g, device="cuda").bfloat16() for _ in range(ncopy)]
        y = torch.empty(1024, N, device="cuda", dtype=torch.bfloat16)
        for i in range(3):
            torch.matmul(x, ws[i % ncopy], out=y)
        torch.cuda.synchronize()
        del ws
    log("[ops] library GEMMs done")
    _copy_calibration("ops")
    return 0


if __name__ == "__main__":
    sys.exit(main() or 0)
