"""Pins of the oracle's confidence, guidance weight, transitions and the
decision part of Alg. 1, all against closed forms worked out by hand."""
import math

import numpy as np
import pytest

from oracle import dard_oracle as O

LAM = O.LAMBDA_DEFAULT


# ---------------------------------------------------------------- Eq. 1
def test_confidence_uniform_row():
    a, c, pc = O.confidence(np.zeros(1000, dtype=np.float32), 5)
    assert a == 0 and abs(c - 1e-3) < 1e-15 and abs(pc - 1e-3) < 1e-15


@pytest.mark.parametrize("h", [0.5, 3.0, 9.0])
def test_confidence_single_spike(h):
    V = 2048
    row = np.zeros(V, dtype=np.float32)
    row[77] = h
    a, c, pc = O.confidence(row, 3)
    expect = math.exp(h) / (math.exp(h) + V - 1)
    assert a == 77 and abs(c - expect) < 1e-12
    assert abs(pc - 1.0 / (math.exp(h) + V - 1)) < 1e-12


def test_confidence_shift_invariance_and_ties():
    rng = np.random.default_rng(0)
    # logits on a 2^-10 grid so that adding 64 is exact in float32
    row = (np.round(rng.standard_normal(500) * 1024) / 1024).astype(np.float32)
    a1, c1, _ = O.confidence(row)
    a2, c2, _ = O.confidence(row + np.float32(64.0))
    assert a1 == a2 and abs(c1 - c2) < 1e-9
    tie = np.zeros(10, dtype=np.float32)
    tie[[7, 3, 8]] = 2.0
    assert O.confidence(tie)[0] == 3          # lowest index wins a tie


# ---------------------------------------------------------------- Eq. 5-6
def test_lambda_halves_every_eight_positions():
    assert abs(LAM ** 8 - 0.5) < 1e-15
    assert abs(LAM - 0.917) < 5e-4            # the paper rounds it to 0.917


def test_guidance_weight_worked_example():
    """Position 6, demoted candidates at 2 and 7, nothing promoted:
    D = lam^4 + lam^1, P = 0, w = p0 / (p0 + D)."""
    B = 11
    prom = np.zeros(B, dtype=bool)
    dem = np.zeros(B, dtype=bool)
    dem[[2, 7]] = True
    Pi, Di, w = O.guidance_weights(prom, dem, LAM, 0.1)
    assert Pi[6] == 0.0
    assert abs(Di[6] - (LAM ** 4 + LAM)) < 1e-15
    assert abs(w[6] - 0.1 / (0.1 + LAM ** 4 + LAM)) < 1e-15
    assert abs(w[6] - 0.0580010) < 1e-6


def test_guidance_weight_cases():
    B = 20
    none = np.zeros(B, dtype=bool)
    # P4: w = 1 whenever nothing was demoted
    prom = none.copy(); prom[[0, 19]] = True
    _, _, w = O.guidance_weights(prom, none, LAM, 0.1)
    assert np.all(w == 1.0)
    _, _, w = O.guidance_weights(none, none, LAM, 0.1)
    assert np.all(w == 1.0)
    # one promotion and one demotion at the same distance d: (l^d+p0)/(2l^d+p0)
    prom = none.copy(); prom[4] = True
    dem = none.copy(); dem[12] = True
    _, _, w = O.guidance_weights(prom, dem, LAM, 0.1)
    assert abs(w[8] - (LAM ** 4 + 0.1) / (2 * LAM ** 4 + 0.1)) < 1e-15
    # closer promotion pulls w above 1/2, closer demotion below
    assert w[5] > 0.5 > w[11]


# ---------------------------------------------------------------- Eq. 8
def test_transition_thresholds():
    tc, tu = np.float32(0.4), np.float32(0.9)
    assert O.transition(tc, tc, tu) == O.STATE_M                      # c = tau_c -> M
    assert O.transition(np.nextafter(tc, np.float32(1)), tc, tu) == O.STATE_C
    assert O.transition(tu, tc, tu) == O.STATE_C                      # c = tau_u -> C
    assert O.transition(np.nextafter(tu, np.float32(1)), tc, tu) == O.STATE_U
    assert O.transition(np.float32(0.0), tc, tu) == O.STATE_M
    # tau_c = tau_u leaves no room for C
    assert O.transition(np.float32(0.9), 0.9, 0.9) == O.STATE_M
    assert O.transition(np.float32(0.95), 0.9, 0.9) == O.STATE_U


def test_mix_endpoints_exact():
    rng = np.random.default_rng(1)
    lx = rng.standard_normal(100).astype(np.float32)
    ls = rng.standard_normal(100).astype(np.float32)
    assert np.array_equal(O.mix_logits(lx, ls, 1.0), lx)
    assert np.array_equal(O.mix_logits(lx, ls, 0.0), ls)


# ---------------------------------------------------------------- Alg. 1
def _spike_logits(V, idx, h):
    row = np.zeros(V, dtype=np.float32)
    row[idx] = h
    return row


def _h_for(p, V):
    """spike height whose top-1 probability is p: e^h / (e^h + V - 1) = p."""
    return math.log(p * (V - 1) / (1 - p))


def test_decide_all_nine_transitions():
    """Planted spikes drive every (from-state, to-state) pair; expected
    tokens, states and confidences come from the closed form of a single
    spike (e^h / (e^h + V - 1)) and Eq. 6-8, not from the oracle."""
    V, B = 64, 9
    mask_id = V - 1
    tc, tu = 0.4, 0.9
    froms = [0, 0, 0, 1, 1, 1, 2, 2, 2]
    targ_p = [0.2, 0.6, 0.97, 0.2, 0.6, 0.97, 0.2, 0.6, 0.97]
    tok = np.array([[mask_id, mask_id, mask_id, 10, 11, 12, 13, 14, 15]], dtype=np.int32)
    state = np.array([froms], dtype=np.uint8)
    logits = np.zeros((1, 2 * B, V), dtype=np.float32)
    for i in range(B):
        h = np.float32(_h_for(targ_p[i], V))
        # the shadow row carries the spike; M rows get the same spike in x so
        # that the mixture keeps it whatever the weight
        logits[0, B + i] = _spike_logits(V, 20 + i, h)
        logits[0, i] = _spike_logits(V, 20 + i, h)
    params = dict(tau_c=tc, tau_u=tu, lam=LAM, p0=0.1, mask_id=mask_id)
    out = O.decide(logits, tok, state, params)
    to = [0, 1, 2] * 3
    assert list(out["state_out"][0]) == to
    for i in range(B):
        expect_tok = mask_id if to[i] == 0 else 20 + i
        assert out["tok_out"][0, i] == expect_tok
        assert abs(out["conf_out"][0, i] - targ_p[i]) < 1e-6
    # candidates: pos 3 demoted, pos 5 promoted -> weights of the M tokens
    dem = np.zeros(B, dtype=bool); dem[3] = True
    prom = np.zeros(B, dtype=bool); prom[5] = True
    for i in (0, 1, 2):
        P_ = LAM ** abs(i - 5)
        D_ = LAM ** abs(i - 3)
        assert abs(out["w"][0, i] - np.float32((P_ + 0.1) / (P_ + D_ + 0.1))) < 1e-7
    assert out["block_done"][0] == 0


def test_decide_mixing_selects_by_weight():
    """An M token whose x and s rows disagree: with a nearby demotion w is
    small and the shadow prediction wins; with a nearby promotion the x
    prediction wins."""
    V, B = 32, 3
    mask_id = V - 1
    tok = np.array([[mask_id, 5, 6]], dtype=np.int32)
    for cand_p, winner in ((0.1, "s"), (0.99, "x")):
        state = np.array([[0, 1, 2]], dtype=np.uint8)
        logits = np.zeros((1, 2 * B, V), dtype=np.float32)
        logits[0, 0] = _spike_logits(V, 3, 5.0)          # x row of the M token
        logits[0, B + 0] = _spike_logits(V, 9, 4.0)      # s row of the M token
        logits[0, B + 1] = _spike_logits(V, 5, np.float32(_h_for(cand_p, V)))
        logits[0, B + 2] = _spike_logits(V, 6, 20.0)
        out = O.decide(logits, tok, state, dict(tau_c=0.4, tau_u=0.9, lam=LAM, p0=0.1,
                                                mask_id=mask_id))
        if winner == "s":
            w = 0.1 / (0.1 + LAM)
            assert abs(out["w"][0, 0] - w) < 1e-7
            assert out["argmax_mix"][0, 0] == 9
        else:
            assert out["w"][0, 0] == 1.0
            assert out["argmax_mix"][0, 0] == 3


def test_decide_verify_pcur_flag():
    V, B = 16, 1
    logits = np.zeros((1, 2, V), dtype=np.float32)
    logits[0, 1] = _spike_logits(V, 4, 6.0)
    tok = np.array([[2]], dtype=np.int32)
    state = np.array([[O.STATE_U]], dtype=np.uint8)
    base = dict(tau_c=0.4, tau_u=0.9, lam=LAM, p0=0.1, mask_id=V - 1)
    top = O.decide(logits, tok, state, base)
    assert top["state_out"][0, 0] == O.STATE_U and top["tok_out"][0, 0] == 4
    cur = O.decide(logits, tok, state, dict(base, flags=O.F_VERIFY_PCUR))
    assert cur["state_out"][0, 0] == O.STATE_M and cur["tok_out"][0, 0] == V - 1
    assert abs(cur["conf_out"][0, 0] - 1 / (math.exp(6) + V - 1)) < 1e-9


def test_block_done_when_all_unmasked():
    V, B = 8, 2
    logits = np.zeros((1, 4, V), dtype=np.float32)
    logits[0, 2] = _spike_logits(V, 1, 20.0)
    logits[0, 3] = _spike_logits(V, 2, 20.0)
    out = O.decide(logits, np.array([[1, 2]]), np.array([[2, 2]], dtype=np.uint8),
                   dict(tau_c=0.4, tau_u=0.9, lam=LAM, p0=0.1, mask_id=V - 1))
    assert out["block_done"][0] == 1


def test_progress_rule():
    """F_PROGRESS: a step of an unfinished block in which no position entered
    U promotes the most confident non-U position (lowest on ties) to U."""
    p = dict(tau_c=0.4, tau_u=0.9, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=99, flags=O.F_PROGRESS)
    c = np.array([0.1, 0.3, 0.3, 0.05, 0.95, 0.2], dtype=np.float32)
    xhat = np.array([10, 11, 12, 13, 14, 15])
    state_in = np.array([O.STATE_M, O.STATE_M, O.STATE_C, O.STATE_M, O.STATE_U, O.STATE_M])
    # position 4 stays U (not a new U); nothing else passes tau_u: position 1
    # (0.3, the lower of the tied positions 1 and 2) is promoted
    st, tok, cf, done = O.finalize(c, xhat, p, state_in)
    assert list(st) == [O.STATE_M, O.STATE_U, O.STATE_M, O.STATE_M, O.STATE_U, O.STATE_M]
    assert list(tok) == [99, 11, 99, 99, 14, 99]
    assert done == 0
    # without the flag the same step commits nothing new
    st0, _, _, _ = O.finalize(c, xhat, dict(p, flags=0), state_in)
    assert list(st0) == [O.STATE_M] * 4 + [O.STATE_U, O.STATE_M]
    # a position that enters U by Eq. 8 suppresses the rule
    c2 = c.copy(); c2[3] = 0.91
    st2, _, _, _ = O.finalize(c2, xhat, p, state_in)
    assert list(st2) == [O.STATE_M, O.STATE_M, O.STATE_M, O.STATE_U, O.STATE_U, O.STATE_M]
    # the last non-U position promoted finishes the block
    c3 = np.array([0.95, 0.5], dtype=np.float32)
    st3, _, _, done3 = O.finalize(c3, np.array([1, 2]), p, np.array([O.STATE_U, O.STATE_C]))
    assert list(st3) == [O.STATE_U, O.STATE_U] and done3 == 1


def test_progress_bounds_block_length():
    """With F_PROGRESS, and committed tokens that stay confident (U tokens are
    re-verified every step and may fall back, so this needs their confidence
    above tau_u), a block finishes within B steps although no other position
    ever passes tau_u."""
    rng = np.random.default_rng(3)
    B = 16
    p = dict(tau_c=0.4, tau_u=0.9, lam=O.LAMBDA_DEFAULT, p0=0.1, mask_id=99, flags=O.F_PROGRESS)
    state = np.zeros(B, dtype=np.int64)
    for step in range(B):
        c = rng.uniform(0.0, 0.9, B).astype(np.float32)
        c[state == O.STATE_U] = 0.95
        state, _, _, done = O.finalize(c, np.arange(B), p, state)
        assert (state == O.STATE_U).sum() == step + 1
        if done:
            break
    assert done == 1 and step == B - 1
