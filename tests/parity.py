"""Decision-parity protocol shared by the GPU step tests (not a test module).

Two levels, as the decision part of Alg. 1 (Eq. 1, 5-8) demands:

op level (bit-exact, no exclusions)
    The GPU's own step intermediates -- the shadow-row argmax / top-1
    probability of every C and U position, the guidance weight w of every M
    position, the mixed-row argmax / top-1 probability -- are fed to the
    oracle's decision functions (verify_candidates for Eq. 5-6, mix_logits for
    Eq. 7, finalize for Eq. 8 and the fill).  The GPU's w, states, tokens,
    block flags and carried keys must equal the oracle's exactly.  The GPU's
    argmaxes must equal the first maximal index of its own (mixed) logit rows
    exactly; its probabilities must agree with the oracle's evaluation of the
    same rows within 1e-5 relative.

step level (against the independent oracle, measured margins)
    A row's argmax is compared when the oracle's top-1 / top-2 gap exceeds
    twice the largest logit error among the row's contenders (the entries
    within twice the run's maximal logit error of the top: no other entry can
    overtake the top); a state decision when the oracle's confidence is
    further from both thresholds than twice the position's confidence error;
    M positions whose guidance weight differs because an excluded candidate
    decided differently are excluded as well.  Excluded positions are counted
    and reported.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import dard_oracle as O


def announce(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def P(mask_id, flags=0, tc=0.4, tu=0.9, w_fixed=0.0):
    return dict(tau_c=tc, tau_u=tu, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=mask_id, flags=flags, w_fixed=w_fixed)


def cparams(dard, params):
    return dard.make_params(params["tau_c"], params["tau_u"], params["lam"], params["p0"], params["mask_id"],
                            params.get("flags", 0), params.get("w_fixed", 0.0))


def sharpen(w, lm_scale):
    """Scale the LM head so that top-1 probabilities spread over (0, 1)."""
    if lm_scale is not None:
        w["lm_head"] = (w["lm_head"].float() * lm_scale).to(w["lm_head"].dtype)
    return w


def step_buffers(b, B, V):
    """Output tensors of one step and the debug captures (dard_step_debug)."""
    z = lambda dt=torch.float32: torch.zeros(b, B, dtype=dt, device="cuda")
    out = dict(tok_out=z(torch.int32), state_out=z(torch.uint8), conf_out=z(),
               block_done=torch.zeros(b, dtype=torch.int32, device="cuda"))
    dbg = dict(logits=torch.zeros(b, 2 * B, V, device="cuda"), w=z(), maxprob_s=z(), argmax_s=z(torch.int32),
               pcur_s=z(), maxprob_mix=z(), argmax_mix=z(torch.int32), entropy=z(), margin=z())
    return out, dbg


def collect(out, dbg):
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    got.update({k: v.cpu().numpy() for k, v in dbg.items()})
    return got


def noise_floor(run_perturbed, ref_logits, seeds=(0, 1, 2), amp=1e-7):
    """How far the oracle's own logits move when every value is perturbed by
    one float32 ulp (relative `amp`) just before each storage rounding; the
    maximum over several perturbation seeds.  run_perturbed() recomputes the
    logits with O.storage replaced."""
    orig = O.storage
    worst = 0.0
    for sd in seeds:
        rng = np.random.default_rng(sd)

        def noisy(x, dt, rng=rng):
            x = np.asarray(x, dtype=np.float64)
            return orig(x * (1.0 + amp * rng.standard_normal(x.shape)), dt)

        O.storage = noisy
        try:
            l2 = run_perturbed()
        finally:
            O.storage = orig
        worst = max(worst, float(np.max(np.abs(l2 - ref_logits))))
    return worst


def check_bf16_logits(got, ref, label, scale=1.0):
    """bf16 multi-layer logits: the root-mean-square error within 2e-2 and the
    maximum error within 2e-2 or twice the oracle's own noise floor (maximum
    over three perturbation seeds).  The 2e-2 bound is stated for the
    random-init model; an LM head sharpened by `scale` multiplies every logit,
    and the effect of every upstream rounding difference, by that factor."""
    d = got["logits"] - ref["logits"]
    err, rms = float(np.max(np.abs(d))), float(np.sqrt(np.mean(d * d)))
    tol = 2e-2 * scale
    floor = ref["floor"]() if err >= tol else 0.0
    print(f"{label}: max |dlogit| {err:.3e} rms {rms:.3e} oracle noise floor {floor:.3e} (bound {tol:.3e})",
          file=sys.stderr, flush=True)
    assert rms < tol, rms
    assert err < max(tol, 2.0 * floor), (err, floor)
    return err, rms, floor


def confidences(dec, state, flags):
    """c_i of Eq. 8 from a decision record (conf_out carries the ordering key,
    which is c_i only under the primary ordering)."""
    shadow = dec["pcur_s"] if flags & O.F_VERIFY_PCUR else dec["maxprob_s"]
    return np.where(state == O.STATE_M, dec["maxprob_mix"], shadow)


def check_op_level(tok, state, got, params):
    """The oracle's decision functions on the GPU's own intermediates must
    reproduce the GPU's decisions exactly."""
    flags = params.get("flags", 0)
    stats = bool(flags & (O.F_ORDER_ENTROPY | O.F_ORDER_MARGIN))
    pcur_mode = bool(flags & O.F_VERIFY_PCUR)
    L = np.asarray(got["logits"], dtype=np.float32)
    b, B = state.shape
    f32 = np.float32
    for s in range(b):
        # shadow rows of C and U positions: argmax exact, probabilities 1e-5 relative
        for i in range(B):
            if state[s, i] == O.STATE_M:
                continue
            a, mp, pc = O.confidence(L[s, B + i], int(tok[s, i]))
            assert got["argmax_s"][s, i] == a, ("argmax_s", s, i)
            assert abs(got["maxprob_s"][s, i] - mp) <= 1e-5 * mp, ("maxprob_s", s, i, got["maxprob_s"][s, i], mp)
            if pcur_mode:
                assert abs(got["pcur_s"][s, i] - pc) <= 1e-5 * pc + 1e-30, ("pcur_s", s, i)
        c_s = (got["pcur_s"] if pcur_mode else got["maxprob_s"])[s].astype(np.float64)
        # Eq. 5-6 on the GPU's candidate confidences: w bit-exact
        _, _, _, w = O.verify_candidates(state[s], c_s, params)
        assert np.array_equal(w.astype(f32), got["w"][s]), ("w", s, w, got["w"][s])
        # Eq. 7 with the GPU's w, on the GPU's rows: argmax exact
        for i in range(B):
            if state[s, i] != O.STATE_M:
                continue
            mixed = O.mix_logits(L[s, i], L[s, B + i], got["w"][s, i])
            a, mp, _ = O.confidence(mixed)
            assert got["argmax_mix"][s, i] == a, ("argmax_mix", s, i)
            assert abs(got["maxprob_mix"][s, i] - mp) <= 1e-5 * mp, ("maxprob_mix", s, i)
            if stats:
                H, mg = O.entropy_margin(mixed)
                assert abs(got["entropy"][s, i] - H) <= 1e-4 + 1e-5 * H, ("entropy", s, i)
                assert abs(got["margin"][s, i] - mg) <= 1e-6 + 1e-5 * mg, ("margin", s, i)
        if stats:
            for i in range(B):
                if state[s, i] != O.STATE_M:
                    H, mg = O.entropy_margin(L[s, B + i])
                    assert abs(got["entropy"][s, i] - H) <= 1e-4 + 1e-5 * H, ("entropy", s, i)
                    assert abs(got["margin"][s, i] - mg) <= 1e-6 + 1e-5 * mg, ("margin", s, i)
        # Eq. 8 and the fill on the GPU's confidences and predictions: exact
        m = state[s] == O.STATE_M
        c = np.where(m, got["maxprob_mix"][s], c_s).astype(np.float64)
        xhat = np.where(m, got["argmax_mix"][s], got["argmax_s"][s])
        st, tk, _, done = O.finalize(c, xhat, params, state[s])
        assert np.array_equal(st, got["state_out"][s]), ("state_out", s, st, got["state_out"][s])
        assert np.array_equal(tk, got["tok_out"][s]), ("tok_out", s)
        assert done == got["block_done"][s], ("block_done", s)
        if flags & O.F_ORDER_ENTROPY:
            key = (-got["entropy"][s]).astype(f32)
        elif flags & O.F_ORDER_MARGIN:
            key = got["margin"][s].astype(f32)
        else:
            key = c.astype(f32)
        assert np.array_equal(key, got["conf_out"][s].astype(f32)), ("conf_out", s)


def check_step_level(tok, state, got, ref, params, label=""):
    """GPU decisions against the independent oracle's, where the measured
    margins make them unambiguous.  Returns (max |dlogit|, excluded count,
    transition counts of the candidates)."""
    flags = params.get("flags", 0)
    Lg = np.asarray(got["logits"], dtype=np.float64)
    Lr = np.asarray(ref["logits"], dtype=np.float64)
    diff = np.abs(Lg - Lr)
    eps = float(np.max(diff))
    c_ref = confidences(ref, state, flags)
    c_gpu = np.where(state == O.STATE_M, got["maxprob_mix"],
                     got["pcur_s"] if flags & O.F_VERIFY_PCUR else got["maxprob_s"])
    b, B = state.shape
    excluded = 0
    for s in range(b):
        for i in range(B):
            rows = [B + i] if state[s, i] != O.STATE_M else [i, B + i]
            ambiguous = False
            for r in rows:
                row = Lr[s, r]
                a = int(np.argmax(row))
                top2 = np.partition(row, -2)[-2:]
                gap = float(top2[1] - top2[0])
                contenders = row >= row[a] - 2 * eps
                eps_r = float(np.max(diff[s, r][contenders]))
                ambiguous |= gap <= 2 * eps_r
            c = float(c_ref[s, i])
            dc = abs(float(c_gpu[s, i]) - c)
            ambiguous |= min(abs(c - params["tau_c"]), abs(c - params["tau_u"])) <= 2 * dc + 1e-7
            if state[s, i] == O.STATE_M:
                ambiguous |= abs(float(got["w"][s, i]) - float(ref["w"][s, i])) > 1e-6
            if ambiguous:
                excluded += 1
                continue
            assert got["state_out"][s, i] == ref["state_out"][s, i], (label, "state", s, i)
            assert got["tok_out"][s, i] == ref["tok_out"][s, i], (label, "token", s, i)
    C = state == O.STATE_C
    trans = {"C->U": int(np.sum(C & (got["state_out"] == O.STATE_U))),
             "C->M": int(np.sum(C & (got["state_out"] == O.STATE_M))),
             "C->C": int(np.sum(C & (got["state_out"] == O.STATE_C))),
             "M->U": int(np.sum((state == O.STATE_M) & (got["state_out"] == O.STATE_U))),
             "U->M": int(np.sum((state == O.STATE_U) & (got["state_out"] == O.STATE_M)))}
    print(f"{label}: max |dlogit| {eps:.3e}; positions excluded by the margin rule {excluded} of {state.size}; "
          f"transitions {trans}", file=sys.stderr, flush=True)
    return eps, excluded, trans


def check_decisions(tok, state, got, ref, params, label=""):
    check_op_level(tok, state, got, params)
    eps, excl, trans = check_step_level(tok, state, got, ref, params, label)
    return eps, excl, trans


def check_workload_decisions(tok, state, got, ref, params, label):
    """The workload-shape protocol: op level exact, at most 10 % of positions
    excluded at step level, and both candidate promotions and demotions
    among the GPU's decisions (so that the comparison is not vacuous)."""
    eps, excl, trans = check_decisions(tok, state, got, ref, params, label)
    assert excl <= state.size // 10, (excl, state.size)
    assert trans["C->U"] >= 1 and trans["C->M"] >= 1, trans
    return eps, excl, trans
