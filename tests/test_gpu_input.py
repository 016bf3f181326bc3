"""GPU parity of the input side with the oracle, bit for bit: per-feature
medians, median binarisation, and the fixed random ±1 expansion layer
(single and multiple input passes, ragged column and pattern tails), and a
few training steps on expanded inputs."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import bmlp as B

from gpu_common import Pair, note, pack_np, torch_cuda

pytestmark = pytest.mark.gpu


def _int8(rng, shape):
    return rng.integers(-128, 128, shape).astype(np.int8)


@pytest.mark.parametrize("n,k", [(1, 5), (2, 70), (999, 300), (1000, 129)])
def test_median_and_binarize(n, k):
    torch = torch_cuda()
    rng = np.random.default_rng(n + k)
    x = _int8(rng, (n, k))
    x[:, 3 % k] = 7                                  # a constant column
    xd = torch.from_numpy(x).cuda()
    note(f"median n={n} k={k}")
    med = B.feature_median(xd)
    bits = B.binarize(xd, med)
    torch.cuda.synchronize()
    m = ob.feature_median(x)
    np.testing.assert_array_equal(med.cpu().numpy(), m)
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64),
                                  pack_np(ob.median_binarize(x, m), bits.shape[1]))


@pytest.mark.parametrize("n,k_raw,k0", [(5, 1, 64), (300, 37, 100), (70, 300, 257), (257, 5000, 64),
                                        (64, 4096, 128)])
def test_expand(n, k_raw, k0):
    torch = torch_cuda()
    rng = np.random.default_rng(k_raw + k0)
    x = _int8(rng, (n, k_raw))
    seed = 0xFEEDFACE12345
    note(f"expand n={n} k_raw={k_raw} k0={k0}")
    bits = B.expand(torch.from_numpy(x).cuda(), k0, seed)
    torch.cuda.synchronize()
    want = ob.expand(x, ob.expansion_matrix(seed, k_raw, k0))
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), pack_np(want, bits.shape[1]))


def test_training_on_expanded_inputs():
    torch = torch_cuda()
    p = Pair((256, 128), 5, 15, 64, 64, 0.25, seed=3)
    rng = np.random.default_rng(8)
    seed = 77
    R = ob.expansion_matrix(seed, 40, 256)
    for t in range(3):
        x = _int8(rng, (64, 40))
        y = rng.integers(0, 5, 64).astype(np.int32)
        a0 = ob.expand(x, R)
        xb = B.expand(torch.from_numpy(x).cuda(), 256, seed)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(xb.cpu().numpy().view(np.uint64), pack_np(a0, xb.shape[1]))
        note(f"expanded step {t}")
        p.step(a0, y, t, 0.5, tag=f"step {t}")
