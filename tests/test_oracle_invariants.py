"""Pins the oracle's update by invariants that the paper's rule implies.

* Hidden weights start at ±1 and move by ±2, so they stay odd, and the clip
  keeps |h| <= B; the visible weights are sign(H) (Section 3.1).
* The local classifiers P are fixed random matrices that never change.
* At most G = K_l / gamma perceptrons are selected per pattern, none for a
  pattern outside M, and each selected one is the largest negative stability
  of its group (Algorithm 2, Section 3.3).
* Reinforcement moves h away from zero, never across it (Algorithm 3).
* One Clipped-Perceptron increment on perceptron k for pattern mu raises
  rho * (a^mu . h^k) by exactly 2 K_{l-1} (the Hebbian direction that fixes
  the error).
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1


def _run(cfg, steps, n, seed, p_r=0.5):
    rng = np.random.default_rng(seed)
    s = ob.init(cfg)
    P0 = [p.copy() for p in s.P]
    hist = []
    for t in range(steps):
        x = random_pm1((n, cfg.widths[0]), rng)
        y = rng.integers(0, cfg.n_classes, size=n)
        before = s.copy()
        tr = ob.train_step(s, x, y, t, p_r)
        hist.append((before, s.copy(), tr, x, y))
    return s, P0, hist


@settings(max_examples=12, deadline=None)
@given(kin=st.integers(1, 90), gamma=st.integers(1, 6), groups=st.integers(1, 5),
       c=st.integers(2, 6), n=st.integers(1, 12), bound=st.sampled_from([1, 3, 5, 15]),
       seed=st.integers(0, 2**32 - 1), depth=st.integers(1, 3))
def test_state_invariants(kin, gamma, groups, c, n, bound, seed, depth):
    widths = (kin,) + (gamma * groups,) * depth
    cfg = ob.Config(widths, c, bound, gamma, 0.25, seed)
    s, P0, hist = _run(cfg, 3, n, seed & 0xFFFF, p_r=2.0)
    for l in range(cfg.n_layers):
        H = s.H[l].astype(np.int64)
        assert np.all(np.abs(H) % 2 == 1)
        assert np.abs(H).max() <= bound
        np.testing.assert_array_equal(s.W(l + 1), np.sign(H))
        np.testing.assert_array_equal(s.P[l], P0[l])
        if bound == 1:
            np.testing.assert_array_equal(H, s.W(l + 1))
    for before, after, tr, x, y in hist:
        for l, lt in enumerate(tr):
            G = widths[l + 1] // gamma
            sel = (lt.kstar >= 0).sum(axis=1)
            assert np.all(sel <= G)
            assert np.all(sel[~lt.upd] == 0)
            assert lt.stats[2] == sel.sum()
            # each selection is the largest negative stability of its group
            rho = before.P[l][y].astype(np.int64)
            delta = (lt.z * rho).reshape(len(y), G, gamma)
            for m, g in zip(*np.nonzero(lt.kstar >= 0)):
                d = delta[m, g]
                k = lt.kstar[m, g]
                assert d[k] < 0
                assert not np.any((d < 0) & (d > d[k]))
                assert not np.any(d[:k] == d[k])
            for m, g in zip(*np.nonzero((lt.kstar < 0) & lt.upd[:, None])):
                assert not np.any(delta[m, g] < 0)


def test_reinforcement_never_flips_sign():
    """With no pattern to fix except through reinforcement, |h| grows, never
    shrinks, and no sign changes."""
    cfg = ob.Config((50, 20), 3, 9, 5, 0.25, 11)
    rng = np.random.default_rng(0)
    H = random_pm1((20, 50), rng) * rng.choice([1, 3, 5, 7, 9], size=(20, 50)).astype(np.int8)
    mask = rng.random(H.size) < 0.5
    H2 = ob.reinforce(H.astype(np.int64), mask, cfg.bound)
    assert np.all(np.sign(H2) == np.sign(H))
    assert np.all(np.abs(H2) >= np.abs(H))
    assert np.all(np.abs(H2) <= cfg.bound)
    moved = np.abs(H2) != np.abs(H)
    np.testing.assert_array_equal(moved, mask.reshape(H.shape) & (np.abs(H) < cfg.bound))


def test_hebbian_increment_is_2k():
    """A single selected pair (mu, k*) raises rho * (a^mu . h^k*) by 2 K_{l-1}."""
    kin, kout, gamma, c = 45, 12, 4, 3
    cfg = ob.Config((kin, kout), c, 127, gamma, 0.25, 5)
    s = ob.init(cfg)
    rng = np.random.default_rng(1)
    for trial in range(20):
        x = random_pm1((1, kin), rng)
        y = rng.integers(0, c, size=1)
        W = s.W(1)
        z = ob.preactivation(x, W)
        ks = ob.select_easiest(z, s.P[0], y, np.array([True]), gamma)
        S = ob.selection_matrix(ks, s.P[0], y, gamma)
        dH = ob.cp_increment(S, x)
        for g in range(kout // gamma):
            if ks[0, g] < 0:
                assert not dH[g * gamma:(g + 1) * gamma].any()
                continue
            k = g * gamma + ks[0, g]
            rho = int(s.P[0][y[0], k])
            gain = rho * int(x[0].astype(np.int64) @ dH[k])
            assert gain == 2 * kin
            others = [r for r in range(g * gamma, (g + 1) * gamma) if r != k]
            assert not dH[others].any()


def test_cp_increment_even_and_bounded():
    """Every entry of the batch increment is even and |dH| <= 2 * n."""
    cfg = ob.Config((60, 24), 4, 127, 6, 0.25, 9)
    s = ob.init(cfg)
    rng = np.random.default_rng(2)
    n = 17
    x = random_pm1((n, 60), rng)
    y = rng.integers(0, 4, size=n)
    W = s.W(1)
    z = ob.preactivation(x, W)
    a = ob.activation(z)
    _, _, _, upd = ob.local_error(ob.local_output(a, s.P[0]), y, ob.robustness_threshold(0.25, 24))
    ks = ob.select_easiest(z, s.P[0], y, upd, 6)
    dH = ob.cp_increment(ob.selection_matrix(ks, s.P[0], y, 6), x)
    assert np.all(dH % 2 == 0)
    assert np.abs(dH).max() <= 2 * n
    # per row, |dH| is at most twice the number of patterns selecting it
    cnt = np.zeros(24, dtype=np.int64)
    for m, g in zip(*np.nonzero(ks >= 0)):
        cnt[g * 6 + ks[m, g]] += 1
    assert np.all(np.abs(dH).max(axis=1) <= 2 * cnt)
