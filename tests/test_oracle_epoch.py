"""Pins the oracle's epoch loop and p_r rescale (Algorithm 1, Section 3.4;
reading R16) and its early-exit evaluation (Section 3.1; reading R17)."""
import math

import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1


def _data(cfg, n, seed):
    rng = np.random.default_rng(seed)
    return random_pm1((n, cfg.widths[0]), rng), rng.integers(0, cfg.n_classes, n), rng


def test_epoch_is_its_batches_in_order():
    # brute force: the same batches trained one by one, gathered here
    cfg = ob.Config((37, 24, 12), 3, 5, 4, 0.25, seed=11)
    x, y, rng = _data(cfg, 45, 1)
    order = rng.permutation(45)
    a, b = ob.init(cfg), ob.init(cfg)
    res = ob.train_epoch(a, x, y, order, 8, 100, 0.7)
    assert res.steps == 5                          # 45 // 8 full batches; 5 samples left out
    wrong = 0
    for k in range(5):
        rows = [int(i) for i in order[8 * k:8 * k + 8]]
        tr = ob.train_step(b, x[rows], y[rows], 100 + k, 0.7)
        wrong += int(tr[-1].err.sum())
        np.testing.assert_array_equal(res.stats[k], np.stack([t.stats for t in tr]))
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(a.H[l], b.H[l])
    assert res.error_fraction == wrong / 40
    assert 0.0 <= res.p_r <= 0.7


def _constant_classifier(cfg, seed):
    # every row of the last classifier equal: every y_hat row is a tie, so
    # the prediction is class 0 (R2) whatever the network does
    st = ob.init(cfg)
    st.P[-1][:] = st.P[-1][0]
    return st


@pytest.mark.parametrize("label,e", [(1, 1.0), (0, 0.0)])
def test_rescale_when_the_error_fraction_is_known(label, e):
    cfg = ob.Config((20, 8, 8), 2, 7, 4, 0.25, seed=5)
    x, _, rng = _data(cfg, 24, 2)
    y = np.full(24, label)
    res = ob.train_epoch(_constant_classifier(cfg, 5), x, y, rng.permutation(24), 8, 0, 0.5)
    assert res.error_fraction == e
    assert res.p_r == (0.5 if e == 1.0 else 0.0)   # p_r sqrt(1) and p_r sqrt(0)


def test_epoch_without_a_full_batch_keeps_p_r():
    cfg = ob.Config((20, 8), 2, 7, 4, 0.25, seed=5)
    x, y, _ = _data(cfg, 6, 3)
    st = ob.init(cfg)
    h0 = [h.copy() for h in st.H]
    res = ob.train_epoch(st, x, y, np.arange(6), 8, 0, 0.3)
    assert res.steps == 0 and res.p_r == 0.3
    for h, g in zip(h0, st.H):
        np.testing.assert_array_equal(h, g)


def test_two_epochs_compound_the_rescale():
    cfg = ob.Config((30, 16, 16), 3, 7, 4, 0.25, seed=9)
    x, y, rng = _data(cfg, 32, 4)
    st = ob.init(cfg)
    r1 = ob.train_epoch(st, x, y, rng.permutation(32), 8, 0, 0.5)
    r2 = ob.train_epoch(st, x, y, rng.permutation(32), 8, r1.steps, r1.p_r)
    assert r2.p_r == pytest.approx(0.5 * math.sqrt(r1.error_fraction) * math.sqrt(r2.error_fraction), rel=1e-15)


def _exit_brute(state, x, y):
    # per pattern: walk the layers, exit at the first whose two largest
    # local outputs differ by at least ceil(r K_l)
    cfg = state.cfg
    yh = ob.forward(state, x)
    out = np.zeros((cfg.n_layers, 3), dtype=np.int64)
    for mu in range(len(y)):
        done = False
        for l in range(cfg.n_layers):
            row = [int(v) for v in yh[l][mu]]
            best = max(range(len(row)), key=lambda c: (row[c], -c))
            rest = sorted(row, reverse=True)
            ok = best == int(y[mu])
            out[l, 0] += ok
            thr = math.ceil(cfg.robustness * cfg.widths[l + 1])
            if not done and (rest[0] - rest[1] >= thr or l == cfg.n_layers - 1):
                out[l, 1] += 1
                out[l, 2] += ok
                done = True
    return out


@pytest.mark.parametrize("r", [0.0, 0.1, 0.25, 1e9])
def test_early_exit_brute_force(r):
    cfg = ob.Config((30, 16, 16, 16), 3, 7, 4, r, seed=13)
    x, y, rng = _data(cfg, 50, 5)
    st = ob.init(cfg)
    ob.train_epoch(st, x, y, rng.permutation(50), 10, 0, 0.5)
    got = ob.early_exit(st, x, y)
    np.testing.assert_array_equal(got, _exit_brute(st, x, y))
    assert got[:, 1].sum() == 50
    np.testing.assert_array_equal(got[:, 0], ob.evaluate(st, x, y))
    if r == 0.0:      # margin >= 0 always: everyone leaves at layer 1
        assert got[0, 1] == 50 and got[0, 2] == got[0, 0]
    if r == 1e9:      # never confident: everyone reaches the last layer
        assert got[-1, 1] == 50 and got[-1, 2] == got[-1, 0]
