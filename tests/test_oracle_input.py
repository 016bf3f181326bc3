"""Pins the oracle's input side: median binarisation (Algorithm 1's input step,
reading R18) and the fixed random ±1 expansion layer for integer inputs
(Section 3.2, footnote 1; reading R19)."""
import numpy as np
import pytest

import oracle.bmlp as ob
from oracle.philox import philox4x32_10


@pytest.mark.parametrize("n,k,seed", [(1, 5, 0), (2, 3, 1), (7, 4, 2), (50, 9, 3), (64, 1, 4)])
def test_median_brute_force(n, k, seed):
    x = np.random.default_rng(seed).integers(-128, 128, (n, k)).astype(np.int8)
    m = ob.feature_median(x)
    for f in range(k):
        col = sorted(int(v) for v in x[:, f])
        assert m[f] == col[(n - 1) // 2]
        # at least half the column is <= m, fewer than half is < m
        assert sum(v <= m[f] for v in col) >= (n - 1) // 2 + 1
        assert sum(v < m[f] for v in col) <= (n - 1) // 2


def test_binarize_special_cases():
    x = np.array([[5, -3, 0], [5, 7, 0], [5, 1, 0]], dtype=np.int8)
    m = ob.feature_median(x)
    np.testing.assert_array_equal(m, [5, 1, 0])
    # a constant column is all +1 (x >= its median); the median itself is +1
    np.testing.assert_array_equal(ob.median_binarize(x, m), [[1, -1, 1], [1, 1, 1], [1, 1, 1]])


def test_expansion_matrix_layout_and_balance():
    seed, k_raw, k0 = 0x1234_5678_9ABC_DEF0, 37, 300
    R = ob.expansion_matrix(seed, k_raw, k0)
    assert R.shape == (k0, k_raw) and set(np.unique(R)) <= {-1, 1}
    # element e = j*K_raw + i is bit (e & 127) of block e >> 7 of stream 5,
    # counter layer word 2^32 - 1, t = 0
    for e in (0, 1, 31, 32, 127, 128, 5000, k_raw * k0 - 1):
        w = philox4x32_10(e >> 7, 0xFFFFFFFF, 0, 5, seed & 0xFFFFFFFF, seed >> 32)
        bit = (int(w[(e & 127) >> 5]) >> (e & 31)) & 1
        assert R.reshape(-1)[e] == (1 if bit else -1)
    # a fair coin: 11100 draws within 4 sigma of half
    assert abs(int((R > 0).sum()) - k_raw * k0 / 2) < 4 * (k_raw * k0) ** 0.5 / 2


def test_expand_closed_form_single_input():
    # K_raw = 1: sign(x r) = sign(x) r for x != 0, and +1 for x = 0
    R = ob.expansion_matrix(7, 1, 64)
    x = np.array([[3], [-2], [0], [127], [-128]], dtype=np.int8)
    a = ob.expand(x, R)
    for mu, v in enumerate(x[:, 0]):
        want = np.ones(64, np.int8) if v == 0 else (np.sign(v) * R[:, 0]).astype(np.int8)
        np.testing.assert_array_equal(a[mu], want)


def test_expand_brute_force():
    rng = np.random.default_rng(5)
    x = rng.integers(-128, 128, (6, 11)).astype(np.int8)
    R = ob.expansion_matrix(9, 11, 13)
    a = ob.expand(x, R)
    for mu in range(6):
        for j in range(13):
            z = sum(int(x[mu, i]) * int(R[j, i]) for i in range(11))
            assert a[mu, j] == (1 if z >= 0 else -1)
