"""Pins the oracle on special cases where the paper's rule reduces to
something simpler, and on the paper's worked examples of the gamma* rule."""
import os

import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_gamma():
    rows = []
    with open(os.path.join(GOLDEN, "gamma_star.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(int(v) for v in line.split()))
    return rows


@pytest.mark.parametrize("k,gamma,groups", _golden_gamma())
def test_gamma_star_paper_examples(k, gamma, groups):
    assert ob.gamma_star(k) == gamma
    assert k // gamma == groups


@pytest.mark.parametrize("k,expect", [(4096, 64), (8192, 64), (2048, 64), (1024, 64), (256, 64),
                                      (90, 90), (100, 100), (97, 97), (210, 105), (7, 7)])
def test_gamma_star_closed_cases(k, expect):
    # a divisor inside [75, 105] has distance 0; powers of two pick 64 (11
    # away) over 128 (23 away); a prime below the range can only use itself
    assert ob.gamma_star(k) == expect


def test_thresholds_closed_form():
    assert ob.robustness_threshold(0.25, 4096) == 1024
    assert ob.robustness_threshold(0.25, 35) == 9          # 8.75 -> 9
    assert ob.robustness_threshold(0.0, 100) == 0
    # q = p_r sqrt(2/(pi K)); at K = 2/pi * 4 the probability is p_r / 2
    assert ob.reinforce_threshold(0.0, 4096) == 0
    assert ob.reinforce_threshold(1e9, 4096) == 1 << 32
    q = ob.reinforce_probability(0.5, 4096)
    assert abs(q - 0.5 * (2 / (np.pi * 4096)) ** 0.5) < 1e-15
    T = ob.reinforce_threshold(0.5, 4096)
    assert (T - 1) < q * 2**32 <= T


def _batch(cfg, n, seed):
    rng = np.random.default_rng(seed)
    return random_pm1((n, cfg.widths[0]), rng), rng.integers(0, cfg.n_classes, size=n)


def test_bound_one_is_pure_binary():
    """B = 1 leaves only the visible weights (the 1-bit case of Appendix A.5)."""
    cfg = ob.Config((40, 30, 30), 4, 1, 5, 0.25, 3)
    s = ob.init(cfg)
    for t in range(4):
        x, y = _batch(cfg, 16, t)
        ob.train_step(s, x, y, t, 1.0)
        for l in range(2):
            np.testing.assert_array_equal(s.H[l], s.W(l + 1))


def test_zero_reinforcement_is_pure_cp():
    """p_r = 0: the step is exactly the clipped batch CP increment."""
    cfg = ob.Config((50, 24), 3, 5, 6, 0.25, 4)
    s = ob.init(cfg)
    x, y = _batch(cfg, 20, 0)
    H0 = s.H[0].astype(np.int64)
    tr = ob.train_step(s, x, y, 0, 0.0)
    assert tr[0].stats[3] == 0
    S = ob.selection_matrix(tr[0].kstar, s.P[0], y, 6)
    np.testing.assert_array_equal(s.H[0], np.clip(H0 + ob.cp_increment(S, x), -5, 5))


def test_zero_robustness_updates_only_errors():
    cfg = ob.Config((50, 24), 3, 5, 6, 0.0, 4)
    s = ob.init(cfg)
    x, y = _batch(cfg, 30, 1)
    tr = ob.train_step(s, x, y, 0, 0.5)
    np.testing.assert_array_equal(tr[0].upd, tr[0].err)


def test_single_group_selects_at_most_one():
    cfg = ob.Config((50, 24), 3, 5, 24, 0.25, 4)
    s = ob.init(cfg)
    x, y = _batch(cfg, 30, 2)
    tr = ob.train_step(s, x, y, 0, 0.5)
    assert tr[0].kstar.shape == (30, 1)
    assert tr[0].stats[2] <= 30


def test_empty_update_set_changes_nothing():
    """With M empty (huge margin cannot be beaten with r = 0 and all correct)
    the layer is left untouched, reinforcement included."""
    cfg = ob.Config((20, 8), 2, 15, 4, 0.0, 8)
    s = ob.init(cfg)
    # construct inputs whose local prediction equals the label
    rng = np.random.default_rng(3)
    x = random_pm1((12, 20), rng)
    a = ob.activation(ob.preactivation(x, s.W(1)))
    y = np.argmax(ob.local_output(a, s.P[0]), axis=1)
    H0 = s.H[0].copy()
    tr = ob.train_step(s, x, y, 0, 5.0)
    assert not tr[0].upd.any()
    assert tr[0].stats.tolist() == [0, 0, 0, 0]
    np.testing.assert_array_equal(s.H[0], H0)


def test_layers_use_pre_step_weights():
    """R13: the forward of every layer in a step sees the weights from before
    the step, so the activations equal a pure forward on the old state."""
    cfg = ob.Config((30, 16, 16, 16), 3, 7, 4, 0.25, 12)
    s = ob.init(cfg)
    x, y = _batch(cfg, 10, 4)
    old = s.copy()
    tr = ob.train_step(s, x, y, 0, 1.0)
    a = x
    for l in range(3):
        a = ob.activation(ob.preactivation(a, old.W(l + 1)))
        np.testing.assert_array_equal(tr[l].a, a)
    yh = ob.forward(old, x)
    for l in range(3):
        np.testing.assert_array_equal(tr[l].yhat, yh[l])


def test_evaluate_counts_correct():
    cfg = ob.Config((30, 16, 16), 4, 7, 4, 0.25, 12)
    s = ob.init(cfg)
    x, y = _batch(cfg, 25, 5)
    cor = ob.evaluate(s, x, y)
    yh = ob.forward(s, x)
    for l in range(2):
        assert cor[l] == sum(int(np.argmax(yh[l][m]) == y[m]) for m in range(25))
