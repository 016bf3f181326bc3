"""Pins the oracle's method variants: K_{l-1} in the reinforcement
probability (R11's alternative), one classifier shared by every layer
(Section 3.1) and z held in min(8, ceil(log2(2 K_{l-1}))) bits
(Section 3.5)."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1


@pytest.mark.parametrize("fan_in", [False, True])
def test_fan_in_reinforcement(fan_in):
    # q(K=4) at p_r = 3 is above 1, so T saturates at 2^32 and every weight
    # of the layer reinforces; q(K=40) is 0.38
    assert ob.reinforce_threshold(3.0, 4) == 1 << 32
    assert ob.reinforce_threshold(3.0, 40) < 1 << 31
    cfg = ob.Config((4, 40), 2, 7, 8, 0.25, seed=3, fan_in_reinforce=fan_in)
    st = ob.init(cfg)
    rng = np.random.default_rng(1)
    tr = ob.train_step(st, random_pm1((16, 4), rng), rng.integers(0, 2, 16), 0, 3.0)
    assert tr[0].upd.any()
    if fan_in:
        assert tr[0].stats[3] == 4 * 40
    else:
        assert 0 < tr[0].stats[3] < 4 * 40


def test_shared_classifier():
    base = ob.init(ob.Config((20, 16, 16, 16), 3, 7, 4, 0.25, seed=5))
    st = ob.init(ob.Config((20, 16, 16, 16), 3, 7, 4, 0.25, seed=5, shared_classifier=True))
    for l in range(3):
        np.testing.assert_array_equal(st.P[l], base.P[0])
    with pytest.raises(ValueError):
        ob.Config((20, 16, 8), 3, 7, 4, 0.25, shared_classifier=True)


@pytest.mark.parametrize("k,bits", [(1, 1), (2, 2), (32, 6), (33, 7), (64, 7), (65, 8), (100, 8), (4096, 8)])
def test_z_bits_closed_form(k, bits):
    # ceil(log2(2K)) bits hold every z in [-K, K] but +K when 2K is a power
    # of two; 8 is the cap
    assert ob.z_bits(k) == bits


def _brute_select(z, rho_rows, upd, gamma):
    n, k = z.shape
    out = -np.ones((n, k // gamma), dtype=np.int64)
    for mu in range(n):
        if not upd[mu]:
            continue
        for g in range(k // gamma):
            best, babs = -1, None
            for e in range(gamma):
                kk = g * gamma + e
                d = int(z[mu, kk]) * int(rho_rows[mu][kk])
                if d < 0 and (babs is None or abs(int(z[mu, kk])) < babs):
                    best, babs = e, abs(int(z[mu, kk]))
            out[mu, g] = best
    return out


def test_saturated_selection_brute_force():
    # W rows are +x0 and -x0 alternately, so z = +-300 on pattern x0: all
    # saturate, to 127 and -128, and ties move
    k_in, k_out = 300, 16
    # r = 100 puts every pattern in M; for label 0 the classifier row makes
    # perceptrons 1 (z = -300 -> -128) and 2 (z = +300 -> 127) the wrong
    # ones: exact z picks 1, saturated z picks 2
    cfg = ob.Config((k_in, k_out), 2, 7, 16, 100.0, seed=7, saturate_z=True)
    exact = ob.Config((k_in, k_out), 2, 7, 16, 100.0, seed=7)
    rng = np.random.default_rng(2)
    x0 = random_pm1((1, k_in), rng)[0]
    x = np.stack([x0] * 3 + list(random_pm1((5, k_in), rng)))
    y = np.array([0, 1, 0, 1, 0, 1, 0, 1])
    picks = []
    for c in (cfg, exact):
        st = ob.init(c)
        st.H[0][:] = np.where(np.arange(k_out)[:, None] % 2 == 0, 1, -1) * x0[None, :]
        st.P[0][0] = np.where(np.arange(k_out) % 2 == 0, 1, -1)
        st.P[0][0, 1], st.P[0][0, 2] = 1, -1
        tr = ob.train_step(st.copy(), x, y, 0, 0.0)[0]
        z_exact = ob.preactivation(x, st.W(1))
        zs = ob.saturate(z_exact, k_in) if c.saturate_z else z_exact
        np.testing.assert_array_equal(tr.z, zs)
        np.testing.assert_array_equal(tr.a, ob.activation(z_exact))
        np.testing.assert_array_equal(tr.kstar, _brute_select(zs, st.P[0][y], tr.upd, 16))
        picks.append(tr.kstar)
    assert not np.array_equal(picks[0], picks[1])   # saturation changed a choice


def test_group_permutation_layout():
    # the key of perceptron k is word k & 3 of Philox block k >> 2 of stream
    # 6 at counter (block, l-1, t, 6); the order sorts keys, ties by index
    from oracle.philox import philox4x32_10
    seed, layer, t, k = 11, 2, 5, 37
    k0, k1 = ob.philox_key(seed)
    keys = []
    for kk in range(k):
        w = philox4x32_10(np.array([kk >> 2], np.uint64), layer - 1, t, 6, k0, k1)
        keys.append(int(w[kk & 3][0]))
    want = sorted(range(k), key=lambda i: (keys[i], i))
    got = ob.group_permutation(seed, layer, t, k)
    assert sorted(got.tolist()) == list(range(k))
    assert got.tolist() == want
    assert ob.group_permutation(seed, layer, t + 1, k).tolist() != want


def _brute_select_perm(z, rho_rows, upd, gamma, perm):
    n, k = z.shape
    out = -np.ones((n, k // gamma), dtype=np.int64)
    for mu in range(n):
        if not upd[mu]:
            continue
        for g in range(k // gamma):
            best, bkey = -1, None
            for e in range(gamma):
                kk = int(perm[g * gamma + e])
                d = int(z[mu, kk]) * int(rho_rows[mu][kk])
                key = (abs(int(z[mu, kk])), kk)
                if d < 0 and (bkey is None or key < bkey):
                    best, bkey = e, key
            out[mu, g] = best
    return out


def test_reshuffled_selection_brute_force():
    # small K_{l-1} makes many |z| ties, so the lowest-index rule is exercised
    cfg = ob.Config((6, 32, 16), 3, 7, 4, 100.0, seed=9, reshuffle_groups=True)
    st = ob.init(cfg)
    rng = np.random.default_rng(4)
    x, y = random_pm1((40, 6), rng), rng.integers(0, 3, 40)
    for t in range(3):
        before = st.copy()
        tr = ob.train_step(st, x, y, t, 0.0)
        for l, lt in enumerate(tr, start=1):
            perm = ob.group_permutation(cfg.seed, l, t, cfg.widths[l])
            np.testing.assert_array_equal(lt.perm, perm)
            np.testing.assert_array_equal(
                lt.kstar, _brute_select_perm(lt.z, before.P[l - 1][y], lt.upd, 4, perm))
            # the clipped-perceptron step moves exactly the selected rows
            S = ob.selection_matrix(lt.kstar, before.P[l - 1], y, 4, perm)
            moved = np.nonzero((st.H[l - 1] != before.H[l - 1]).any(axis=1))[0]
            assert set(moved.tolist()) <= set(np.nonzero(S.any(axis=0))[0].tolist())


def test_reshuffle_one_group_is_fixed_groups():
    # with gamma = K_l there is one group whatever the order, so training
    # is the same as with fixed groups
    runs = []
    for rs in (False, True):
        cfg = ob.Config((24, 16, 16), 2, 7, 16, 0.5, seed=13, reshuffle_groups=rs)
        st = ob.init(cfg)
        rng = np.random.default_rng(6)
        for t in range(4):
            ob.train_step(st, random_pm1((32, 24), rng), rng.integers(0, 2, 32), t, 0.3)
        runs.append(st)
    for a, b in zip(runs[0].H, runs[1].H):
        np.testing.assert_array_equal(a, b)


def test_reshuffle_changes_groups():
    cfg = ob.Config((24, 32), 2, 7, 4, 100.0, seed=13, reshuffle_groups=True)
    fixed = ob.Config((24, 32), 2, 7, 4, 100.0, seed=13)
    rng = np.random.default_rng(8)
    x, y = random_pm1((32, 24), rng), rng.integers(0, 2, 32)
    S = []
    for c in (cfg, fixed):
        st = ob.init(c)
        tr = ob.train_step(st.copy(), x, y, 0, 0.0)[0]
        S.append(ob.selection_matrix(tr.kstar, st.P[0], y, 4, tr.perm))
    assert not np.array_equal(S[0], S[1])


def test_sequential_clip_order_matters():
    # h = B, then +2 and -2 from two patterns: one at a time gives B - 2,
    # the batch sum gives B
    B = 7
    H = np.array([[B, -B, 1]], dtype=np.int8)
    a = np.array([[1, -1, 1], [1, -1, -1]], dtype=np.int8)
    S = np.array([[1], [-1]], dtype=np.int8)       # rho of the selected row per pattern
    # column 2 never reaches the bound: 1 + 2 + 2 = 5 either way
    np.testing.assert_array_equal(ob.cp_sequential(H, S, a, B), [[B - 2, -B + 2, 5]])
    np.testing.assert_array_equal(ob.clip(H.astype(np.int64) + ob.cp_increment(S, a), B), [[B, -B, 5]])


def _brute_sequential(H, S, a, B):
    h = H.astype(np.int64).tolist()
    n, k = S.shape
    for mu in range(n):
        for kk in range(k):
            if S[mu, kk]:
                for i in range(len(h[kk])):
                    h[kk][i] = max(-B, min(B, h[kk][i] + 2 * int(S[mu, kk]) * int(a[mu, i])))
    return np.array(h)


def test_sequential_clip_brute_force():
    rng = np.random.default_rng(12)
    B = 3
    H = rng.integers(-1, 2, (10, 9)) * 2 + 1
    H = np.clip(H, -B, B).astype(np.int8)
    a = random_pm1((30, 9), rng)
    S = (rng.integers(0, 3, (30, 10)) - 1).astype(np.int8)
    np.testing.assert_array_equal(ob.cp_sequential(H, S, a, B), _brute_sequential(H, S, a, B))


def test_sequential_clip_without_saturation_is_the_sum():
    # a bound no sum reaches: clipping never acts, both readings agree
    runs = []
    for seq in (False, True):
        cfg = ob.Config((24, 32, 16), 3, 127, 8, 0.5, seed=21, sequential_clip=seq)
        st = ob.init(cfg)
        rng = np.random.default_rng(3)
        for t in range(3):
            ob.train_step(st, random_pm1((16, 24), rng), rng.integers(0, 3, 16), t, 0.0)
        runs.append(st)
    for a_, b_ in zip(runs[0].H, runs[1].H):
        np.testing.assert_array_equal(a_, b_)


def test_sequential_clip_train_step():
    # B = 1: every increment saturates at once, so the order shows
    cfg = ob.Config((24, 32), 2, 1, 8, 100.0, seed=5, sequential_clip=True)
    st = ob.init(cfg)
    rng = np.random.default_rng(9)
    x, y = random_pm1((48, 24), rng), rng.integers(0, 2, 48)
    before = st.copy()
    tr = ob.train_step(st, x, y, 0, 0.0)[0]
    S = ob.selection_matrix(tr.kstar, before.P[0], y, 8)
    np.testing.assert_array_equal(st.H[0], _brute_sequential(before.H[0], S, x, 1))
    batch = ob.clip(before.H[0].astype(np.int64) + ob.cp_increment(S, x), 1)
    assert not np.array_equal(st.H[0], batch)
