"""Pins of the oracle's ordering and mixing variants (Sec. 5.1, the
mask-design and logit-mixing analyses).

The variants replace one ingredient of the method each: the order in which
candidates see each other (bidirectional, left-to-right, entropy, margin
instead of confidence, Eq. 3) or the guidance weight (a constant instead of
Eq. 5-6).  They are pinned by equivalences with the primary rule that follow
from the definitions (a bidirectional mask is the confidence mask with every
key tied; left-to-right is the confidence mask keyed by -position), closed
forms of entropy and margin, an independent library entropy, and exact
float32 identities of the mixing formula at w in {0, 1/2, 1}.
"""
import math

import numpy as np
import pytest
import scipy.stats

from oracle import dard_oracle as O

LAM = 0.5 ** 0.125


def _block(seed, B):
    rng = np.random.default_rng(seed)
    state = rng.integers(0, 3, size=B).astype(np.uint8)
    conf = rng.permutation(np.linspace(0.05, 0.95, B)).astype(np.float32)
    return state, conf


# ---------------------------------------------------------------- mask orderings
@pytest.mark.parametrize("B", [1, 5, 33, 64, 128])
@pytest.mark.parametrize("extra", [0, O.F_XSELF_SHADOW, O.F_MKEYS_SHADOW])
def test_bidir_is_confidence_mask_with_all_keys_tied(B, extra):
    """Eq. 3 with c_i = c_j for every pair makes every candidate visible to
    every other: the bidirectional variant."""
    state, conf = _block(B, B)
    tied = np.full(B, 0.5, dtype=np.float32)
    assert np.array_equal(O.visible_keys(state, conf, 4, O.F_C_BIDIR | extra),
                          O.visible_keys(state, tied, 4, extra))


@pytest.mark.parametrize("B", [1, 5, 33, 64, 128])
@pytest.mark.parametrize("extra", [0, O.F_XSELF_SHADOW, O.F_MKEYS_SHADOW])
def test_l2r_is_confidence_mask_keyed_by_minus_position(B, extra):
    """Left-to-right order is the confidence order of keys that decrease
    strictly with the position; the confidences passed in are ignored."""
    state, conf = _block(B + 1, B)
    key = -np.arange(B, dtype=np.float32)
    assert np.array_equal(O.visible_keys(state, conf, 3, O.F_ORDER_L2R | extra),
                          O.visible_keys(state, key, 3, extra))


def test_l2r_shadow_rows_form_a_causal_chain():
    """Under l2r the shadow query of the k-th candidate from the left sees
    exactly the k-1 candidates to its left (and the U tokens) in x: the
    autoregressive factorisation of Eq. 4 in position order."""
    state = np.array([1, 2, 1, 0, 1, 1, 2, 1], dtype=np.uint8)
    conf = np.array([0.9, 0.1, 0.2, 0.3, 0.8, 0.5, 0.6, 0.7], dtype=np.float32)
    B = len(state)
    X = O.take_x(state, conf, O.F_ORDER_L2R)
    C = [j for j in range(B) if state[j] == O.STATE_C]
    U = [j for j in range(B) if state[j] == O.STATE_U]
    for k, i in enumerate(C):
        assert sorted(np.nonzero(X[B + i])[0]) == sorted(C[:k] + U)


def test_entropy_and_margin_orderings_leave_the_mask_rule_alone():
    state, conf = _block(9, 40)
    for f in (O.F_ORDER_ENTROPY, O.F_ORDER_MARGIN):
        assert np.array_equal(O.take_x(state, conf, f), O.take_x(state, conf, 0))


def test_bidir_catches_planted_mistake():
    """Keeping the shadow query's own x key under the bidirectional mask (a
    plausible slip: 'no constraint' read as 'no leakage block') breaks Eq. 2's
    per-position choice against the tied-key equivalent."""
    state = np.array([1, 1, 2, 0], dtype=np.uint8)
    conf = np.array([0.3, 0.6, 0.9, 0.1], dtype=np.float32)
    X = O.take_x(state, conf, O.F_C_BIDIR)
    assert not X[4 + 0, 0] and not X[4 + 1, 1]
    assert X[0, 1] and X[1, 0]               # the two candidates see each other


# ---------------------------------------------------------------- entropy, margin
def test_entropy_margin_uniform_row():
    for V in (1, 2, 7, 1000):
        H, m = O.entropy_margin(np.full(V, 3.25, dtype=np.float32))
        assert abs(H - math.log(V)) < 1e-12
        assert m == (1.0 if V == 1 else 0.0)


@pytest.mark.parametrize("h", [0.5, 3.0, 12.0])
def test_entropy_margin_single_spike(h):
    """One logit h above V-1 zeros: p1 = e^h/Z, q = 1/Z, Z = e^h + V - 1."""
    V = 50
    row = np.zeros(V, dtype=np.float32)
    row[17] = h
    Z = math.exp(h) + V - 1
    p1, q = math.exp(h) / Z, 1.0 / Z
    H, m = O.entropy_margin(row)
    assert abs(H - (-(p1 * math.log(p1)) - (V - 1) * q * math.log(q))) < 1e-12
    assert abs(m - (p1 - q)) < 1e-12


def test_entropy_matches_scipy_and_margin_matches_sorted_logits():
    rng = np.random.default_rng(3)
    for V in (2, 9, 4096):
        row = (rng.standard_normal(V) * 3).astype(np.float32)
        H, m = O.entropy_margin(row)
        p = scipy.special.softmax(row.astype(np.float64))
        assert abs(H - scipy.stats.entropy(p)) < 1e-10
        l1, l2 = np.sort(row.astype(np.float64))[::-1][:2]
        Z = np.sum(np.exp(row.astype(np.float64) - l1))
        assert abs(m - (1.0 - math.exp(l2 - l1)) / Z) < 1e-12
        # shift invariance
        H2, m2 = O.entropy_margin(row.astype(np.float64) + 100.0)
        assert abs(H2 - H) < 1e-9 and abs(m2 - m) < 1e-12


def test_margin_of_a_tie_at_the_top_is_zero():
    row = np.array([1.0, 4.0, -2.0, 4.0], dtype=np.float32)
    assert O.entropy_margin(row)[1] == 0.0


def test_order_key_direction():
    """Larger key = earlier in the chain: low entropy, large margin, high
    confidence come first."""
    sharp, flat = (0.01, 0.98), (2.0, 0.05)     # (entropy, margin)
    for f in (O.F_ORDER_ENTROPY, O.F_ORDER_MARGIN):
        assert O.order_key(0.5, *sharp, f) > O.order_key(0.5, *flat, f)
    assert O.order_key(0.7, *flat, 0) > O.order_key(0.6, *sharp, 0)


# ---------------------------------------------------------------- decisions
def _logits(seed, B, V):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((1, 2 * B, V)) * 2.5).astype(np.float32)


def _params(**kw):
    p = dict(tau_c=0.2, tau_u=0.5, lam=LAM, p0=0.1, mask_id=0, flags=0, w_fixed=0.0)
    p.update(kw)
    return p


@pytest.mark.parametrize("flag", [O.F_ORDER_ENTROPY, O.F_ORDER_MARGIN])
def test_ordering_changes_only_the_carried_key(flag):
    """The entropy / margin orderings act on the next step's mask only: this
    step's tokens, states and weights are those of the primary method, and the
    carried key is -H (entropy) or the margin of the row that gave c_i (the
    shadow row of a C/U position, the mixed row of an M position)."""
    B, V = 12, 64
    logits = _logits(1, B, V)
    state = np.array([[0, 1, 2] * 4], dtype=np.uint8)
    tok = np.where(state == 0, 0, 7).astype(np.int32)
    base = O.decide(logits, tok, state, _params())
    var = O.decide(logits, tok, state, _params(flags=flag))
    for k in ("tok_out", "state_out", "w", "argmax_mix", "block_done"):
        assert np.array_equal(base[k], var[k])
    for i in range(B):
        if state[0, i] == O.STATE_M:
            row = O.mix_logits(logits[0, i], logits[0, B + i], base["w"][0, i])
        else:
            row = logits[0, B + i]
        H, m = O.entropy_margin(row)
        expect = -H if flag == O.F_ORDER_ENTROPY else m
        assert var["conf_out"][0, i] == np.float32(expect)
    # the primary ordering carries the confidence itself
    assert np.array_equal(base["conf_out"], np.maximum(
        np.where(state == 0, base["maxprob_mix"], 0), np.where(state == 0, 0, base["maxprob_s"])))


@pytest.mark.parametrize("wf", [0.0, 1.0])
def test_fixed_weight_endpoints(wf):
    """w = 1 decodes every M token from its x row, w = 0 from its shadow row
    (Eq. 7 at the endpoints is exact in float32)."""
    B, V = 10, 40
    logits = _logits(2, B, V)
    state = np.array([[0, 1, 0, 2, 1, 0, 0, 2, 1, 0]], dtype=np.uint8)
    tok = np.where(state == 0, 0, 3).astype(np.int32)
    out = O.decide(logits, tok, state, _params(flags=O.F_FIXED_W, w_fixed=wf))
    for i in range(B):
        if state[0, i] == O.STATE_M:
            assert out["w"][0, i] == wf
            src = logits[0, i] if wf == 1.0 else logits[0, B + i]
            a, mp, _ = O.confidence(src)
            assert out["argmax_mix"][0, i] == a
            assert out["maxprob_mix"][0, i] == np.float32(mp)
        else:
            assert out["w"][0, i] == 0.0


def test_fixed_half_weight_is_the_rounded_sum():
    """w = 1/2: (0.5 l_x) + (0.5 l_s) in float32 is the float32 sum of the two
    rows halved exactly, so the prediction is the argmax of l_x + l_s."""
    B, V = 6, 300
    logits = _logits(4, B, V)
    state = np.zeros((1, B), dtype=np.uint8)
    tok = np.zeros((1, B), dtype=np.int32)
    out = O.decide(logits, tok, state, _params(flags=O.F_FIXED_W, w_fixed=0.5))
    for i in range(B):
        s = (logits[0, i] + logits[0, B + i]).astype(np.float32)
        assert out["argmax_mix"][0, i] == int(np.argmax(s))
        assert np.array_equal(O.mix_logits(logits[0, i], logits[0, B + i], 0.5), s * np.float32(0.5))


def test_fixed_weight_ignores_verification_outcome():
    """Eq. 5-6 move w with the promoted / demoted candidates; the fixed
    variant does not."""
    B, V = 5, 16
    logits = np.zeros((1, 2 * B, V), dtype=np.float32)
    logits[0, B + 1, 3] = 30.0                  # candidate 1 promoted
    state = np.array([[0, 1, 0, 0, 0]], dtype=np.uint8)
    tok = np.array([[0, 3, 0, 0, 0]], dtype=np.int32)
    adaptive = O.decide(logits, tok, state, _params())
    fixed = O.decide(logits, tok, state, _params(flags=O.F_FIXED_W, w_fixed=0.25))
    assert adaptive["w"][0, 0] > 0.9
    assert np.all(fixed["w"][0, [0, 2, 3, 4]] == np.float32(0.25))
