"""Pins the oracle's Philox4x32-10 and its use for the method's random draws.

* The generator is checked against rocRAND's Philox4x32-10 (a separate
  library implementation of the same published generator), compiled here for
  the host from its headers.
* The two key increments are checked against the closed forms they come from
  (the fractional parts of the golden ratio and of sqrt(3), times 2^32).
* The reinforcement draws are checked for what Algorithm 3 needs: a hidden
  weight is reinforced with probability p_r * sqrt(2 / (pi K_l)), independently
  of the others (binomial interval on the count, uniform byte histogram).
"""
import ctypes
import math
import os
import shutil
import subprocess
from decimal import Decimal, getcontext

import numpy as np
import pytest

import oracle.bmlp as ob
from oracle.philox import PHILOX_W0, PHILOX_W1, philox4x32_10

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_kernel.h"):
        pytest.skip("hipcc / rocRAND headers not available")
    out = tmp_path_factory.mktemp("rr") / "rr.so"
    subprocess.run([hipcc, "-O1", "-fPIC", "-shared", os.path.join(HERE, "rocrand_philox_shim.cpp"),
                    "-o", str(out)], check=True, capture_output=True)
    lib = ctypes.CDLL(str(out))
    lib.ref_philox4x32_10.argtypes = [ctypes.c_uint32] * 6 + [ctypes.POINTER(ctypes.c_uint32)]

    def ref(c0, c1, c2, c3, k0, k1):
        o = (ctypes.c_uint32 * 4)()
        lib.ref_philox4x32_10(c0, c1, c2, c3, k0, k1, o)
        return list(o)
    return ref


def test_against_rocrand(rocrand_ref):
    rng = np.random.default_rng(123)
    cases = [(0, 0, 0, 0, 0, 0), (1, 0, 0, 0, 0, 0), (0, 3, 7, 4, 0xDEADBEEF, 0x12345678)]
    for _ in range(200):
        c = [int(v) for v in rng.integers(0, 2**32, size=4)]
        c[1] &= (1 << 30) - 1        # keep offset * 4 inside 64 bits for the wrapper
        k = [int(v) for v in rng.integers(0, 2**32, size=2)]
        cases.append((*c, *k))
    for c0, c1, c2, c3, k0, k1 in cases:
        got = [int(w) for w in philox4x32_10(c0, c1, c2, c3, k0, k1)]
        assert got == rocrand_ref(c0, c1, c2, c3, k0, k1), (c0, c1, c2, c3, k0, k1)


def test_vectorised_matches_scalar(rocrand_ref):
    """The array form used by the oracle gives the scalar result per element."""
    blocks = np.arange(1000, 1064, dtype=np.uint64)
    w = np.stack(philox4x32_10(blocks, 2, 77, ob.STREAM_R_COARSE, 99, 5), axis=-1)
    for i, b in enumerate(blocks):
        assert [int(v) for v in w[i]] == rocrand_ref(int(b), 2, 77, ob.STREAM_R_COARSE, 99, 5)


def test_weyl_constants_closed_form():
    getcontext().prec = 60
    phi = (1 + Decimal(5).sqrt()) / 2
    assert PHILOX_W0 == int((phi - 1) * (1 << 32))
    assert PHILOX_W1 == int((Decimal(3).sqrt() - 1) * (1 << 32))


def test_init_bits_layout():
    """Bit j of stream s is bit (j & 127) of block j >> 7, word-major, LSB first."""
    j = np.arange(0, 1024, dtype=np.uint64)
    bits = ob.stream_bits(42, 3, ob.STREAM_H_INIT, j)
    w = np.stack(philox4x32_10(np.arange(8, dtype=np.uint64), 2, 0, ob.STREAM_H_INIT, 42, 0), axis=-1)
    expect = np.unpackbits(w.astype("<u4").view(np.uint8), bitorder="little")
    np.testing.assert_array_equal(bits, expect)
    # a scattered sample gives the same bits
    idx = np.array([5, 900, 128, 127, 77], dtype=np.uint64)
    np.testing.assert_array_equal(ob.stream_bits(42, 3, ob.STREAM_H_INIT, idx), expect[idx.astype(int)])


@pytest.mark.parametrize("n", [1, 127, 128, 129, 1000, 4096 + 5])
def test_prefix_bits_match_gathered_bits(n):
    """The whole-range form used at init equals the per-index form."""
    for stream in (ob.STREAM_H_INIT, ob.STREAM_P_INIT):
        np.testing.assert_array_equal(ob.stream_bits_prefix(0x1234_5678_9ABC, 2, stream, n),
                                      ob.stream_bits(0x1234_5678_9ABC, 2, stream, np.arange(n, dtype=np.uint64)))


@pytest.mark.parametrize("k_in", [40, 64, 100])
def test_reinforce_draws_layout(k_in):
    """u8 of weight (k, i): bit p is bit (i & 31) of word p of the two stream-3
    blocks of the row's 32-column group; u24 comes from stream 4 by flat index."""
    j = np.arange(3 * k_in, dtype=np.uint64)
    u = ob.reinforce_draws(7, 2, 5, j, k_in)
    groups = (k_in + 31) // 32
    expect = []
    for jj in range(3 * k_in):
        k, i = divmod(jj, k_in)
        q = k * groups + (i >> 5)
        planes = [int(w) for w in philox4x32_10(2 * q, 1, 5, ob.STREAM_R_COARSE, 7, 0)]
        planes += [int(w) for w in philox4x32_10(2 * q + 1, 1, 5, ob.STREAM_R_COARSE, 7, 0)]
        u8 = sum(((planes[p] >> (i & 31)) & 1) << p for p in range(8))
        u24 = int(philox4x32_10(jj >> 2, 1, 5, ob.STREAM_R_FINE, 7, 0)[jj & 3]) & 0xFFFFFF
        expect.append((u8 << 24) | u24)
    np.testing.assert_array_equal(u, np.array(expect, dtype=np.uint64))


def test_reinforcement_rate_binomial():
    """Count of reinforced weights within 5 sigma of n q, for several q."""
    n = 1 << 20
    for p_r, k in [(0.5, 4096), (0.5, 256), (0.05, 1024), (2.0, 64)]:
        T = ob.reinforce_threshold(p_r, k)
        q = T / 2**32
        m = ob.reinforce_mask(1234, 1, 17, T, n, 4096)
        sd = math.sqrt(n * q * (1 - q))
        assert abs(m.sum() - n * q) < 5 * sd + 1, (p_r, k, m.sum(), n * q)


def test_draws_are_uniform_bytes():
    """Chi-square of the top byte of the 32-bit draws over 2^20 samples."""
    u = ob.reinforce_draws(99, 1, 3, np.arange(1 << 20, dtype=np.uint64), 1000)
    top = (u >> np.uint64(24)).astype(np.int64)
    hist = np.bincount(top, minlength=256)
    e = len(top) / 256
    chi2 = ((hist - e) ** 2 / e).sum()
    assert chi2 < 255 + 6 * math.sqrt(2 * 255)
    low = (u & np.uint64(0xFF)).astype(np.int64)
    hist = np.bincount(low, minlength=256)
    chi2 = ((hist - e) ** 2 / e).sum()
    assert chi2 < 255 + 6 * math.sqrt(2 * 255)


def test_streams_and_steps_differ():
    j = np.arange(4096, dtype=np.uint64)
    a = ob.reinforce_draws(1, 1, 0, j, 512)
    b = ob.reinforce_draws(1, 1, 1, j, 512)
    c = ob.reinforce_draws(1, 2, 0, j, 512)
    d = ob.reinforce_draws(2, 1, 0, j, 512)
    for other in (b, c, d):
        assert (a == other).mean() < 0.01


def test_hierarchical_threshold_equivalence():
    """u < T holds exactly when the top byte is below T >> 24, or equal to it
    with the low 24 bits below T & 0xFFFFFF: the GPU may read the low bits
    only in the equal case."""
    rng = np.random.default_rng(5)
    u = rng.integers(0, 2**32, size=200000, dtype=np.uint64)
    for T in [0, 1, 255, 1 << 24, (1 << 24) + 5, 26772564, 107090253, (1 << 32) - 1, 1 << 32]:
        hi, lo = T >> 24, T & 0xFFFFFF
        u8, u24 = u >> np.uint64(24), u & np.uint64(0xFFFFFF)
        alt = (u8 < hi) | ((u8 == hi) & (u24 < lo))
        np.testing.assert_array_equal(alt, u < np.uint64(T))
