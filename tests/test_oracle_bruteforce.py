"""Pins the oracle's per-layer arithmetic against brute force on tiny layers.

Every expected value here is computed by plain Python loops over ±1 entries,
written from the paper's definitions (Algorithm 1 lines for z, a, y_hat, the
01-loss of Eq. 1 and the margin tau; Algorithm 2 for the stabilities and the
easiest perceptron; Algorithm 3 for the Clipped-Perceptron increment), or by
an independent route (bit packing with numpy and Python's popcount).
"""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1


def py_dot(u, v):
    s = 0
    for a, b in zip(u, v):
        s += int(a) * int(b)
    return s


def brute_layer(a_prev, W, P, y, thr, gamma):
    """Plain loops for one layer: z, a, y_hat, pred, tau, err, M, k*."""
    n, kin = a_prev.shape
    kout = W.shape[0]
    c = P.shape[0]
    z = [[py_dot(a_prev[m], W[k]) for k in range(kout)] for m in range(n)]
    a = [[1 if z[m][k] >= 0 else -1 for k in range(kout)] for m in range(n)]
    yhat = [[py_dot(a[m], P[cl]) for cl in range(c)] for m in range(n)]
    pred, tau, err, upd = [], [], [], []
    for m in range(n):
        best = 0
        for cl in range(1, c):
            if yhat[m][cl] > yhat[m][best]:
                best = cl
        vals = sorted(yhat[m], reverse=True)
        pred.append(best)
        tau.append(vals[0] - vals[1])
        e = best != int(y[m])
        err.append(e)
        upd.append(e or (vals[0] - vals[1]) < thr)
    G = kout // gamma
    kstar = [[-1] * G for _ in range(n)]
    for m in range(n):
        if not upd[m]:
            continue
        for g in range(G):
            sel = -1
            for off in range(gamma):
                k = g * gamma + off
                d = z[m][k] * int(P[int(y[m])][k])
                if d < 0 and (sel < 0 or d > z[m][g * gamma + sel] * int(P[int(y[m])][g * gamma + sel])):
                    sel = off
            kstar[m][g] = sel
    return (np.array(z), np.array(a), np.array(yhat), np.array(pred), np.array(tau),
            np.array(err), np.array(upd), np.array(kstar))


def brute_cp(H, a_prev, P, y, kstar, gamma, bound):
    """Algorithm 3's clipped-perceptron increment applied one selected pair at a time, no clipping
    inside the loop, clip once at the end."""
    h = [[int(v) for v in row] for row in H]
    n, G = kstar.shape
    for m in range(n):
        for g in range(G):
            if kstar[m][g] < 0:
                continue
            k = g * gamma + int(kstar[m][g])
            rho = int(P[int(y[m])][k])
            for i in range(a_prev.shape[1]):
                h[k][i] += 2 * int(a_prev[m][i]) * rho
    return np.clip(np.array(h), -bound, bound)


@pytest.mark.parametrize("kin,kout,gamma,c,n,seed", [
    (37, 12, 4, 3, 9, 0),     # odd fan-in: z is never 0
    (64, 16, 8, 5, 7, 1),
    (70, 18, 6, 4, 11, 2),    # widths not multiples of 64
    (33, 10, 10, 2, 6, 3),    # one group spanning the layer
    (16, 9, 3, 7, 13, 4),
])
def test_layer_matches_brute_force(kin, kout, gamma, c, n, seed):
    rng = np.random.default_rng(seed)
    a_prev = random_pm1((n, kin), rng)
    H = random_pm1((kout, kin), rng) * rng.choice([1, 3, 5], size=(kout, kin)).astype(np.int8)
    P = random_pm1((c, kout), rng)
    y = rng.integers(0, c, size=n)
    W = np.where(H > 0, 1, -1).astype(np.int8)
    thr = ob.robustness_threshold(0.25, kout)
    bz, ba, byh, bpred, btau, berr, bupd, bks = brute_layer(a_prev, W, P, y, thr, gamma)

    z = ob.preactivation(a_prev, W)
    a = ob.activation(z)
    yhat = ob.local_output(a, P)
    pred, tau, err, upd = ob.local_error(yhat, y, thr)
    ks = ob.select_easiest(z, P, y, upd, gamma)
    np.testing.assert_array_equal(z, bz)
    np.testing.assert_array_equal(a, ba)
    np.testing.assert_array_equal(yhat, byh)
    np.testing.assert_array_equal(pred, bpred)
    np.testing.assert_array_equal(tau, btau)
    np.testing.assert_array_equal(err, berr)
    np.testing.assert_array_equal(upd, bupd)
    np.testing.assert_array_equal(ks, bks)

    bound = 7
    S = ob.selection_matrix(ks, P, y, gamma)
    h1 = ob.clip(H.astype(np.int64) + ob.cp_increment(S, a_prev), bound)
    np.testing.assert_array_equal(h1, brute_cp(H, a_prev, P, y, ks, gamma, bound))


@pytest.mark.parametrize("kin", [1, 31, 32, 33, 63, 64, 65, 784, 1000])
def test_popcount_identity(kin):
    """z = K - 2 popc(a XOR w) = 2 popc(XNOR(a, w)) - K, on bit-packed rows."""
    rng = np.random.default_rng(kin)
    a = random_pm1((6, kin), rng)
    W = random_pm1((5, kin), rng)
    z = ob.preactivation(a, W)
    pa = np.packbits(a > 0, axis=1, bitorder="little")
    pw = np.packbits(W > 0, axis=1, bitorder="little")
    for m in range(6):
        ia = int.from_bytes(pa[m].tobytes(), "little")
        for k in range(5):
            iw = int.from_bytes(pw[k].tobytes(), "little")
            x = ia ^ iw
            assert z[m, k] == kin - 2 * bin(x).count("1")
            xnor = (~x) & ((1 << kin) - 1)
            assert z[m, k] == 2 * bin(xnor).count("1") - kin
            assert (z[m, k] - kin) % 2 == 0   # z has the parity of K_{l-1}


def test_float32_matmul_agrees():
    """An independent library route: float32 BLAS is exact here (sums < 2^24)."""
    rng = np.random.default_rng(7)
    a = random_pm1((40, 300), rng)
    W = random_pm1((50, 300), rng)
    ref = (a.astype(np.float32) @ W.T.astype(np.float32)).astype(np.int64)
    np.testing.assert_array_equal(ob.preactivation(a, W), ref)


def test_tie_rules():
    """R2/R3: argmax takes the lowest class on a tie, and a tie at the top
    gives tau = 0 (so the robustness test always fires on a tie)."""
    yhat = np.array([[3, 7, 7, -1], [5, 5, 5, 5], [9, 1, 9, 0], [-4, -2, -8, -2]])
    y = np.array([2, 0, 0, 3])
    pred, tau, err, upd = ob.local_error(yhat, y, 1)
    np.testing.assert_array_equal(pred, [1, 0, 0, 1])
    np.testing.assert_array_equal(tau, [0, 0, 0, 0])
    np.testing.assert_array_equal(err, [True, False, False, True])
    np.testing.assert_array_equal(upd, [True, True, True, True])
    # with threshold 0, a tie is not "below" it
    _, _, _, upd0 = ob.local_error(yhat, y, 0)
    np.testing.assert_array_equal(upd0, err)


def test_kstar_ties_and_zero_stability():
    """R5: equal negative stabilities pick the lowest index; delta = 0 is not
    eligible; a group without a negative stability selects nothing."""
    z = np.array([[-3, -1, -1, 2, 0, 0, 5, 1]])
    P = np.ones((2, 8), dtype=np.int8)
    y = np.array([0])
    ks = ob.select_easiest(z, P, y, np.array([True]), 4)
    np.testing.assert_array_equal(ks, [[1, -1]])
    # flipping rho turns positive z into negative stabilities
    P2 = -P
    ks2 = ob.select_easiest(z, P2, y, np.array([True]), 4)
    np.testing.assert_array_equal(ks2, [[3, 3]])   # delta = [3,1,1,-2 | 0,0,-5,-1]
    # not in M: nothing selected
    ks3 = ob.select_easiest(z, P, y, np.array([False]), 4)
    np.testing.assert_array_equal(ks3, [[-1, -1]])


def test_sign_of_zero_preactivation():
    """R1: a pre-activation of exactly 0 (even fan-in) gives a = +1."""
    a_prev = np.array([[1, -1, 1, -1]], dtype=np.int8)
    W = np.array([[1, 1, 1, 1], [1, -1, 1, -1], [-1, 1, -1, 1]], dtype=np.int8)
    z = ob.preactivation(a_prev, W)
    np.testing.assert_array_equal(z, [[0, 4, -4]])
    np.testing.assert_array_equal(ob.activation(z), [[1, 1, -1]])
