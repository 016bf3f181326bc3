"""Layers with more classes than the classifier kernel stages at once (above
128): y_hat = a_l P_l^T then comes from the forward kernel with P_l in
place of W_l, up to eight layers per launch (int16 rows inside a step or an
evaluation, int32 rows as bmlp_forward's output), and the error signal of Eq. 1 and the robustness
test from a separate kernel.  Bit-exact against the oracle: a_l, 01-loss,
M_l, the selected perceptrons, the counts, H_l and W_l after every step;
y_hat, correct counts and early-exit counts.  Narrow layers give y_hat few
distinct values, so many classes tie at the top (tau = 0)."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1

from gpu_common import Pair, note

pytestmark = pytest.mark.gpu

IMPLS = {"popcount": 1, "mfma_fp4": 2}

CASES = [
    # widths, c, B, gamma, n, steps, p_r
    # three class tiles (the last ragged) and two pattern tiles; layer 2's
    # rows are 3 words (4-byte loads)
    ((300, 256, 192), 300, 15, 64, 200, 2, 0.5),
    # the fewest classes that take this path; eight pattern tiles, which the
    # launch spreads over the XCDs by patterns
    ((64, 128), 129, 7, 64, 1024, 2, 0.5),
    # y_hat of an 8-perceptron layer takes 9 values over 200 classes: ties
    ((64, 8, 16), 200, 7, 8, 150, 2, 1.0),
    # a thousand classes, as in the 8192-wide stress network
    ((512, 640), 1000, 31, 64, 96, 2, 0.5),
    # nine layers: the products of eight layers in one launch, then one more
    ((100,) + (64,) * 9, 150, 7, 64, 70, 2, 0.5),
]


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-c{c[1]}-n{c[4]}" for c in CASES])
def test_train_steps(case, impl):
    widths, c, bound, gamma, n, steps, p_r = case
    rng = np.random.default_rng(c * 7 + n)
    p = Pair(widths, c, bound, n, gamma, 0.25, seed=int(rng.integers(1 << 62)), fwd_impl=IMPLS[impl])
    for t in range(steps):
        note(f"many classes {widths} c={c} n={n} {impl} step {t}")
        x = random_pm1((n, widths[0]), rng)
        y = rng.integers(0, c, size=n).astype(np.int32)
        if widths[1] <= 16:   # the tie case really ties at the top of y_hat (tau = 0)
            yh = ob.local_output(ob.activation(ob.preactivation(x, p.ora.W(1))), p.ora.P[0])
            assert (ob.local_error(yh, y, 0)[1] == 0).mean() > 0.25
        p.step(x, y, 3 + t, p_r, tag=f"step {t}")


@pytest.mark.parametrize("impl", list(IMPLS))
def test_forward_eval_and_exits(impl):
    widths, c = (300, 256, 192), 300
    rng = np.random.default_rng(41)
    p = Pair(widths, c, 15, 400, 64, 0.25, seed=4242, fwd_impl=IMPLS[impl])
    x = random_pm1((256, widths[0]), rng)
    y = rng.integers(0, c, size=256).astype(np.int32)
    p.step(x, y, 0, 0.5, check_state=False)
    xt = random_pm1((333, widths[0]), rng)
    # labels from layer 2's own prediction for part of the batch, so the
    # correct counts are not all near zero
    yt = rng.integers(0, c, size=333).astype(np.int32)
    ref = ob.forward(p.ora, xt)
    yt[:150] = ref[1][:150].argmax(axis=1)
    xb, ytd = p.to_dev(xt, yt)
    note(f"many classes forward/eval {impl}")
    yh = p.gpu.forward(xb)
    cor = p.gpu.eval(xb, ytd)
    ex = p.gpu.eval_exit(xb[:200], ytd[:200])
    ex = p.gpu.eval_exit(xb[200:], ytd[200:], ex)
    p.torch.cuda.synchronize()
    for l in range(2):
        np.testing.assert_array_equal(yh[l].cpu().numpy(), ref[l], err_msg=f"y_hat layer {l + 1}")
    got = cor.cpu().numpy()
    np.testing.assert_array_equal(got, ob.evaluate(p.ora, xt, yt))
    assert got[1] >= 150
    np.testing.assert_array_equal(ex.cpu().numpy(), ob.early_exit(p.ora, xt, yt))
