"""Bit-exact parity at depth: networks of more layers than one classifier or
update launch takes (eight), so that every layer slot of those launches and
the launches after the first are compared with the oracle in full (a_l,
01-loss, M_l, the selected perceptrons, the step counts, H_l, W_l and P_l
after every step); and a step in which layer 1 has nothing to update while
deeper layers do (Alg. 2 runs the layer update only for a non-empty M_l)."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1

from gpu_common import Pair, note

pytestmark = pytest.mark.gpu

IMPLS = {"popcount": 1, "mfma_fp4": 2}

DEEP = [
    # widths, c, B, gamma (0: gamma*), n, steps, p_r
    ((70,) + (64,) * 9, 10, 63, 0, 100, 4, 0.5),
    # gamma*(192) = 96 (the generic selection) among layers of gamma 64;
    # eleven layers: launches of eight and three
    ((100, 128, 64, 192, 64, 128, 64, 64, 128, 64, 64, 128), 7, 15, 0, 65, 3, 0.9),
    # sixteen layers: two full launches of eight
    ((64,) * 17, 4, 7, 0, 33, 2, 2.0),
]


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("case", DEEP, ids=[f"L{len(c[0]) - 1}-c{c[1]}-B{c[2]}-n{c[4]}" for c in DEEP])
def test_deep_networks(case, impl):
    widths, c, bound, gamma, n, steps, p_r = case
    rng = np.random.default_rng(len(widths) * 1000 + n)
    p = Pair(widths, c, bound, n, gamma, 0.25, seed=int(rng.integers(1 << 62)), fwd_impl=IMPLS[impl])
    for t in range(steps):
        note(f"deep {len(widths) - 1} layers, {impl}, step {t}")
        x = random_pm1((n, widths[0]), rng)
        y = rng.integers(0, c, size=n).astype(np.int32)
        st = p.step(x, y, 7 + t, p_r, tag=f"step {t}")
        # the deep layers really update: later layers have patterns in M
        assert st[len(widths) - 2][1] > 0


@pytest.mark.parametrize("impl", list(IMPLS))
def test_layer_with_empty_update_set(impl):
    # r = 0 puts only the misclassified patterns in M (R4: tau < ceil(0) never
    # holds); labels equal to layer 1's own prediction leave M_1 empty, so
    # layer 1 takes no Clipped-Perceptron step and no reinforcement, while
    # layer 2, with its own classifier, still updates.
    widths, c = (96, 64, 64), 5
    rng = np.random.default_rng(17)
    p = Pair(widths, c, 7, 80, 16, 0.0, seed=99, fwd_impl=IMPLS[impl])
    for t in range(2):
        x = random_pm1((80, widths[0]), rng)
        a1 = ob.activation(ob.preactivation(x, p.ora.W(1)))
        pred1, _, _, _ = ob.local_error(ob.local_output(a1, p.ora.P[0]), np.zeros(80, np.int64), 0)
        y = pred1.astype(np.int32)
        H1_before = p.gpu.H(1).cpu().numpy().copy()
        W1_before = p.gpu.W(1).cpu().numpy().copy()
        note(f"empty M_1, {impl}, step {t}")
        st = p.step(x, y, t, 1.0, tag=f"empty M_1 step {t}")
        np.testing.assert_array_equal(st[0], np.zeros(4, np.int64))
        assert st[1][1] > 0 and st[1][3] > 0, "layer 2 should update and reinforce"
        np.testing.assert_array_equal(p.gpu.H(1).cpu().numpy(), H1_before)
        np.testing.assert_array_equal(p.gpu.W(1).cpu().numpy(), W1_before)
