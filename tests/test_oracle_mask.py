"""Pins of the oracle's state-specific attention mask (Sec. 3.2, Eq. 2-4).

The oracle's rule table is checked against (a) masks worked out by hand in
tests/golden/, (b) a brute-force dense mask written block by block from the
prose, listing the x keys and the s keys of every query block separately (so
that Eq. 2 is a real check, not a consequence of the construction), and
(c) the structural invariants the paper states.
"""
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import dard_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    state = conf = None
    rows = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#")[0].strip()
        if not line:
            continue
        parts = line.split()
        if parts[0] == "state":
            state = np.array([int(x) for x in parts[1:]], dtype=np.uint8)
        elif parts[0] == "conf":
            conf = np.array([float(x) for x in parts[1:]], dtype=np.float32)
        else:
            rows[parts[0]] = [int(c) for c in parts[1] + parts[2]]
    B = len(state)
    order = [f"x{i}" for i in range(B)] + [f"s{i}" for i in range(B)]
    return state, conf, np.array([rows[k] for k in order], dtype=bool)


@pytest.mark.parametrize("name", ["mask_b5.txt", "mask_b6_tie.txt"])
def test_golden_hand_worked_masks(name):
    state, conf, expect = _read_golden(name)
    got = O.visible_keys(state, conf, P=0)
    assert np.array_equal(got, expect)


def brute_force_mask(state, conf, P, flags=0):
    """Dense [2B, P+2B] mask written from the prose, per query block.

    For each (stream, state) block the visible x keys and the visible s keys
    are listed independently, straight from the sentences of Sec. 3.2.
    """
    B = len(state)
    U = {j for j in range(B) if state[j] == O.STATE_U}
    C = {j for j in range(B) if state[j] == O.STATE_C}
    M = {j for j in range(B) if state[j] == O.STATE_M}
    dense = np.zeros((2 * B, P + 2 * B), dtype=bool)
    for stream in ("x", "s"):
        for i in range(B):
            r = i if stream == "x" else B + i
            if state[i] == O.STATE_U:
                # U queries: U keys in x, M and C keys in s; s^i never sees x^i.
                xs, ss = set(U), M | C
                if stream == "s" or flags & O.F_XSELF_SHADOW:
                    xs, ss = xs - {i}, ss | {i}
            elif state[i] == O.STATE_C:
                # C queries: U keys and more confident C keys in x (Eq. 3);
                # everything else (M and less confident C) from s.
                if flags & O.F_C_BIDIR:
                    # Sec. 5.1 bidirectional variant: every candidate in x
                    higher = set(C)
                elif flags & O.F_ORDER_L2R:
                    # Sec. 5.1 left-to-right variant: candidates to the left
                    higher = {j for j in C if j <= i}
                else:
                    higher = {j for j in C if conf[i] <= conf[j]}
                xs = U | higher
                ss = M | (C - higher)
                if stream == "s":
                    xs, ss = xs - {i}, ss | {i}
            else:
                if stream == "x":
                    if flags & O.F_MKEYS_SHADOW:
                        xs, ss = C | U | {i}, M - {i}
                    else:
                        # x queries of M tokens: C and U keys in x (M keys in x too).
                        xs, ss = C | U | M, set()
                else:
                    # s queries of M tokens: U keys in x, C keys in s ("as masked").
                    xs, ss = set(U), C | M
            dense[r, :P] = True
            for j in xs:
                dense[r, P + j] = True
            for j in ss:
                dense[r, P + B + j] = True
    return dense


def _random_block(rng, B, ties=False):
    state = rng.integers(0, 3, size=B).astype(np.uint8)
    if ties:
        conf = rng.choice(np.array([0.5, 0.6, 0.7], dtype=np.float32), size=B)
    else:
        conf = rng.permutation(np.linspace(0.05, 0.95, B)).astype(np.float32)
    return state, conf


@settings(max_examples=60, deadline=None)
@given(B=st.integers(1, 40), P=st.integers(0, 5), seed=st.integers(0, 10**6),
       flags=st.sampled_from([0, O.F_XSELF_SHADOW, O.F_MKEYS_SHADOW,
                              O.F_XSELF_SHADOW | O.F_MKEYS_SHADOW,
                              O.F_C_BIDIR, O.F_ORDER_L2R,
                              O.F_C_BIDIR | O.F_MKEYS_SHADOW,
                              O.F_ORDER_L2R | O.F_XSELF_SHADOW,
                              O.F_ORDER_ENTROPY, O.F_ORDER_MARGIN]),
       ties=st.booleans())
def test_rule_table_equals_brute_force(B, P, seed, flags, ties):
    rng = np.random.default_rng(seed)
    state, conf = _random_block(rng, B, ties)
    assert np.array_equal(O.visible_keys(state, conf, P, flags),
                          brute_force_mask(state, conf, P, flags))


@pytest.mark.parametrize("B", [1, 7, 32, 64, 128])
def test_invariants(B):
    rng = np.random.default_rng(B)
    for trial in range(3):
        state, conf = _random_block(rng, B)
        P = 3
        vis = O.visible_keys(state, conf, P)
        X = O.take_x(state, conf)
        U = np.nonzero(state == O.STATE_U)[0]
        C = np.nonzero(state == O.STATE_C)[0]
        # I1 (Eq. 2): every query sees exactly one of x^j, s^j -> P + B keys.
        assert np.all(vis.sum(axis=1) == P + B)
        assert np.all(vis[:, P:P + B] ^ vis[:, P + B:])
        # I2: no U query (x or s) sees the x key of a candidate.
        for i in U:
            for r in (i, B + i):
                assert not X[r, C].any()
        # I4: no shadow query sees its own original key.
        for i in range(B):
            assert not X[B + i, i]
        # I3 (Eq. 4): with distinct confidences sorted descending (pi), the
        # shadow query of the k-th candidate sees exactly x of pi(1..k-1) and U.
        pi = C[np.argsort(-conf[C], kind="stable")]
        for k, i in enumerate(pi):
            expect = np.zeros(B, dtype=bool)
            expect[pi[:k]] = True
            expect[U] = True
            assert np.array_equal(X[B + i], expect)
        # I5: the C x C block of the x queries, permuted by pi, is lower
        # triangular including the diagonal.
        sub = X[np.ix_(pi, pi)]
        assert np.array_equal(sub, np.tril(np.ones_like(sub)))


def test_all_masked_block_is_vanilla():
    """All-M block: x queries see the whole x block, s queries the whole s
    block (first step of a block)."""
    B = 9
    state = np.zeros(B, dtype=np.uint8)
    conf = np.zeros(B, dtype=np.float32)
    X = O.take_x(state, conf)
    assert X[:B].all() and not X[B:].any()


def test_state_code_out_of_range_rejected():
    with pytest.raises(ValueError):
        O.take_x(np.array([3], dtype=np.uint8), np.zeros(1, dtype=np.float32))


def test_brute_force_catches_planted_mistake():
    """A plausible mistake in the rule table (shadow C query keeping its own x
    key) is caught by the brute-force comparison."""
    rng = np.random.default_rng(5)
    state, conf = _random_block(rng, 12)
    state[3] = O.STATE_C
    good = O.visible_keys(state, conf, 2)
    bad = good.copy()
    bad[12 + 3, 2 + 3] = True
    bad[12 + 3, 2 + 12 + 3] = False
    assert not np.array_equal(bad, brute_force_mask(state, conf, 2))
