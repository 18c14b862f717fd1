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

import math
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
    # rows the LM head does not run over stay NaN (the head skips the x rows of C and U positions)
    dbg = dict(logits=torch.full((b, 2 * B, V), float("nan"), device="cuda"), w=z(), maxprob_s=z(),
               argmax_s=z(torch.int32),
               pcur_s=z(), maxprob_mix=z(), argmax_mix=z(torch.int32), entropy=z(), margin=z())
    return out, dbg


def collect(out, dbg):
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    got.update({k: v.cpu().numpy() for k, v in dbg.items()})
    return got


def under_perturbation(run, seed, amp=1e-7):
    """run() with every value the oracle computes perturbed by about one
    float32 ulp (relative `amp`) just before each storage rounding (O.storage
    is replaced meanwhile).  Any implementation whose accumulation order
    differs from the oracle's flips some of those roundings, so such runs
    measure the noise floor of a comparison."""
    orig = O.storage
    rng = np.random.default_rng(seed)

    def noisy(x, dt):
        x = np.asarray(x, dtype=np.float64)
        return orig(x * (1.0 + amp * rng.standard_normal(x.shape)), dt)

    O.storage = noisy
    try:
        return run()
    finally:
        O.storage = orig


def perturbed_logits(run_perturbed, seeds=(0, 1, 2), amp=1e-7):
    """The oracle's logits recomputed by run_perturbed() under the one-ulp
    perturbation, once per seed."""
    return [np.asarray(under_perturbation(run_perturbed, sd, amp), dtype=np.float32) for sd in seeds]


def noise_floor(run_perturbed, ref_logits, seeds=(0, 1, 2), amp=1e-7):
    """Largest maximum and root-mean-square difference of the perturbed runs
    from the oracle's logits."""
    worst, worst_rms = 0.0, 0.0
    for l2 in perturbed_logits(run_perturbed, seeds, amp):
        d = l2.astype(np.float64) - ref_logits
        worst = max(worst, float(np.max(np.abs(d))))
        worst_rms = max(worst_rms, float(np.sqrt(np.mean(d * d))))
    return worst, worst_rms


class Floor:
    """Lazily computed perturbed runs of the oracle (three seeds), shared by
    the logit floor and the decision floor."""

    def __init__(self, run_perturbed, ref_logits):
        self.run, self.ref, self.runs = run_perturbed, ref_logits, None

    def logits(self):
        if self.runs is None:
            self.runs = perturbed_logits(self.run)
        return self.runs

    def __call__(self):
        worst, worst_rms = 0.0, 0.0
        for l2 in self.logits():
            d = l2.astype(np.float64) - self.ref
            worst = max(worst, float(np.max(np.abs(d))))
            worst_rms = max(worst_rms, float(np.sqrt(np.mean(d * d))))
        return worst, worst_rms


def e4m3_decode(codes):
    """Values of OCP FP8 E4M3 codes (a uint8 tensor or array), from the
    oracle's table of the format's magnitudes."""
    c = (codes.cpu().numpy() if hasattr(codes, "cpu") else np.asarray(codes)).astype(np.int64)
    mag = O.E4M3_VALUES[np.minimum(c & 0x7F, 126)]
    return np.where(c & 0x80, -mag, mag)


def e4m3_steps(a, b):
    """Distance in code steps between two arrays of E4M3 values (signed code
    ordinals)."""
    def ordinal(v):
        m = np.searchsorted(O.E4M3_VALUES, np.abs(v))
        return np.where(v < 0, -m, m)
    return np.abs(ordinal(a) - ordinal(b))


def check_fp8_cache_layers(pairs, label):
    """Per layer (GPU values, oracle values) of K or V held as E4M3: in the
    first layer, whose inputs agree with the oracle's up to fp32 rounding
    order, nearly every code is equal and none more than one step away;
    deeper layers inherit the first layer's flipped roundings (each a whole
    code step) through attention, so there the bound only rules out gross
    errors (a layer offset, a scale or a sign change 98 % of the codes or
    more)."""
    for layer, j, g, r in pairs:
        dg = e4m3_steps(g, r)
        print(f"{label} fp8 cache layer {layer} {'KV'[j]}: codes differing {np.mean(dg > 0):.4f}, "
              f"by more than one step {np.mean(dg > 1):.4f}", file=sys.stderr, flush=True)
        if layer == 0:
            assert np.mean(dg == 0) > 0.97 and dg.max() <= 1, (label, layer, j, np.mean(dg == 0), dg.max())
        else:
            assert np.mean(dg > 0) < 0.35 and np.mean(dg > 1) < 0.08, (label, layer, j)


def hidden_mix(params):
    return bool(params.get("flags", 0) & O.F_HIDDEN_MIX)


def reference_logits(got, ref, state, params):
    """The oracle's values for the logit rows the GPU step computed: every
    row as the oracle has it, except that with hidden-state mixing the shadow
    slot of an M position holds the mixed row, compared with the oracle's
    logit mixing (Eq. 7) under the GPU's guidance weight, and the x rows are
    not computed."""
    R = np.array(ref["logits"], dtype=np.float64)
    if hidden_mix(params):
        b, B = state.shape
        for s_ in range(b):
            for i in range(B):
                if state[s_, i] == O.STATE_M:
                    R[s_, B + i] = O.mix_logits(ref["logits"][s_, i], ref["logits"][s_, B + i], got["w"][s_, i])
        R[:, :B] = np.nan
    return R


def needed_rows(state, params):
    """[b][2B] bool: the logit rows the decisions read."""
    b, B = state.shape
    need = np.zeros((b, 2 * B), dtype=bool)
    need[:, B:] = True
    if not hidden_mix(params):
        need[:, :B] = state == O.STATE_M
    return need


def logit_diff(got, ref, state, params):
    """GPU minus oracle over the rows the GPU computed (flattened); every row
    the decisions read must be among them."""
    G = np.asarray(got["logits"], dtype=np.float64)
    R = reference_logits(got, ref, state, params)
    computed = np.all(np.isfinite(G), axis=-1)
    need = needed_rows(state, params)
    assert np.all(computed[need]), "a logit row the decisions read was not computed"
    rows = computed & np.all(np.isfinite(R), axis=-1)
    return (G - R)[rows]


def logit_err(got, ref, state, params):
    return float(np.max(np.abs(logit_diff(got, ref, state, params))))


def check_bf16_logits(got, ref, label, scale=1.0):
    """bf16 multi-layer logits: the maximum error within 2e-2 or twice the
    oracle's own noise floor, and the root-mean-square error within 2e-2 or
    twice the floor's root-mean-square (the floors: the largest over three
    perturbation seeds; computed only when an error exceeds 2e-2).  The 2e-2
    bound is stated for the random-init model; an LM head sharpened by
    `scale` multiplies every logit, and the effect of every upstream rounding
    difference, by that factor."""
    d = logit_diff(got, ref, ref["state"], ref["params"])
    err, rms = float(np.max(np.abs(d))), float(np.sqrt(np.mean(d * d)))
    tol = 2e-2 * scale
    floor, floor_rms = ref["floor"]() if (err >= tol or rms >= tol) else (0.0, 0.0)
    print(f"{label}: max |dlogit| {err:.3e} rms {rms:.3e}; oracle noise floor max {floor:.3e} rms {floor_rms:.3e} "
          f"(bound {tol:.3e})", file=sys.stderr, flush=True)
    assert rms < max(tol, 2.0 * floor_rms), (rms, floor_rms)
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
        # Eq. 7 with the GPU's w, on the GPU's rows: argmax exact (with hidden-state
        # mixing the GPU's mixed row sits in the shadow slot)
        for i in range(B):
            if state[s, i] != O.STATE_M:
                continue
            if hidden_mix(params):
                mixed = L[s, B + i]
            else:
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
    margins make them unambiguous.

    The decision row of a position is its shadow row (C, U) or its mixed row
    (M, Eq. 7).  M rows are mixed with the GPU's weight on both sides: the
    weights themselves are checked at op level, and they differ from the
    oracle's only after a candidate decided differently, which is counted
    there.  A position is excluded when its argmax is ambiguous (the oracle's
    top-1 / top-2 gap within twice the largest error among the row's
    contenders, the entries within twice the run's maximal logit error of the
    top) or its state is (the oracle's confidence within twice the
    position's confidence error of a threshold).  A confidence error must
    itself stay within what the run's logit error allows, c (e^(2 eps) - 1):
    a gross error cannot pass as an exclusion.  Returns (max |dlogit|,
    excluded count, transition counts of the GPU's decisions)."""
    flags = params.get("flags", 0)
    pcur_mode = bool(flags & O.F_VERIFY_PCUR)
    Lg = np.asarray(got["logits"], dtype=np.float32)
    Lr = np.asarray(ref["logits"], dtype=np.float32)
    b, B = state.shape
    rows_g, rows_r = np.empty((b, B, Lg.shape[-1])), np.empty((b, B, Lr.shape[-1]))
    for s in range(b):
        for i in range(B):
            if state[s, i] == O.STATE_M:
                wg = got["w"][s, i]
                rows_g[s, i] = Lg[s, B + i] if hidden_mix(params) else O.mix_logits(Lg[s, i], Lg[s, B + i], wg)
                rows_r[s, i] = O.mix_logits(Lr[s, i], Lr[s, B + i], wg)
            else:
                rows_g[s, i], rows_r[s, i] = Lg[s, B + i], Lr[s, B + i]
    diff = np.abs(rows_g - rows_r)
    eps = float(np.max(np.abs(logit_diff(got, ref, state, params))))
    eps_rows = float(np.max(diff))
    c_gpu = np.where(state == O.STATE_M, got["maxprob_mix"], got["pcur_s"] if pcur_mode else got["maxprob_s"])
    excluded = 0
    for s in range(b):
        for i in range(B):
            row = rows_r[s, i]
            a, c, pc = O.confidence(row, int(tok[s, i]) if state[s, i] != O.STATE_M else None)
            if pcur_mode and state[s, i] != O.STATE_M:
                c = pc
            c = float(np.float32(c))
            top2 = np.partition(row, -2)[-2:]
            gap = float(top2[1] - top2[0])
            contenders = row >= row[a] - 2 * eps_rows
            eps_r = float(np.max(diff[s, i][contenders]))
            dc = abs(float(c_gpu[s, i]) - c)
            assert dc <= c * (math.exp(2 * eps_rows) - 1.0) + 1e-6, (label, "confidence error", s, i, dc, eps_rows)
            st = O.transition(c, params["tau_c"], params["tau_u"])
            state_ambiguous = min(abs(c - params["tau_c"]), abs(c - params["tau_u"])) <= 2 * dc + 1e-7
            # the prediction matters only where the position does not fall back to [Mask]
            if state_ambiguous or (st != O.STATE_M and gap <= 2 * eps_r):
                excluded += 1
                continue
            assert got["state_out"][s, i] == st or flags & O.F_PROGRESS, (label, "state", s, i)
            if got["state_out"][s, i] != O.STATE_M:
                assert got["tok_out"][s, i] == a, (label, "token", s, i)
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


def decision_floor(tok, state, ref, params):
    """Positions the same step-level protocol excludes when the oracle is
    compared with its own perturbed runs (the largest count over the seeds):
    the part of the bf16 exclusions that the rounding noise alone causes."""
    worst = 0
    prm = dict(params, flags=params.get("flags", 0) & ~O.F_HIDDEN_MIX)
    for l2 in ref["floor"].logits():
        pseudo = O.decide(l2, tok, state, prm)
        pseudo["logits"] = l2
        pseudo["w"] = pseudo["w"].astype(np.float32)
        for k in ("maxprob_s", "pcur_s", "maxprob_mix"):
            pseudo[k] = pseudo[k].astype(np.float32)
        _, excl, _ = check_step_level(tok, state, pseudo, ref, prm, "oracle vs its perturbed run")
        worst = max(worst, excl)
    return worst


def check_workload_decisions(tok, state, got, ref, params, label, require_transitions=True):
    """The workload-shape protocol: op level exact; at step level at most 10 %
    of the positions excluded, or twice what the oracle's own one-ulp
    perturbation excludes (the same rule as for the logits); and both
    candidate promotions and demotions among the GPU's decisions, so that the
    comparison is not vacuous."""
    eps, excl, trans = check_decisions(tok, state, got, ref, params, label)
    bound = state.size // 10
    if excl > bound:
        floor = decision_floor(tok, state, ref, params)
        print(f"{label}: decision floor (oracle vs its perturbed runs) {floor} of {state.size}", file=sys.stderr,
              flush=True)
        bound = max(bound, 2 * floor)
    assert excl <= bound, (excl, bound, state.size)
    if require_transitions:
        assert trans["C->U"] >= 1 and trans["C->M"] >= 1, trans
    return eps, excl, trans
