"""The local classifier kernel (at most 128 classes, matrix-core path):
y_hat = a_l P_l^T, the 01-loss of Eq. 1 and the robustness test of
Algorithm 1, bit-exact against the oracle for every class-block count (1 to
8 blocks of 16 classes), for layer widths whose 512-element super-blocks
end in a partial one or not at all, for rows of an odd number of 64-bit
words (8-byte loads) and of an even number (16-byte loads), and for pattern
counts that leave the last work-group partly empty.  Each case trains two
steps in full parity (a_l, 01-loss, M_l, the selections, the counts, H_l and
W_l), then compares y_hat of bmlp_forward (the kernel's y_hat output, which
takes back the per-pattern offset of its encoding), the correct counts of
bmlp_eval and the early-exit counts of bmlp_eval_exit."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1

from gpu_common import Pair, note

pytestmark = pytest.mark.gpu

CASES = [
    # widths, c, n: the comment names what the classifier's layer exercises
    ((130, 37), 3, 37),            # one block; K = 37: a single 1-word row, only a partial super-block
    ((200, 1100), 20, 50),         # two blocks; K = 1100: two whole super-blocks and a partial one
    ((64, 512), 2, 17),            # the fewest classes; K = 512: exactly one super-block
    ((96, 2560), 33, 64),          # three blocks (the last holds one class); five whole super-blocks
    ((64, 8704), 49, 40),          # four blocks; 17 whole super-blocks: load rounds of four and of one
    ((96, 4160), 100, 70),         # seven blocks, as in the 4096-wide benchmark network; 65-word rows
    ((64, 2560, 640), 128, 33),    # eight blocks, all full; two layers (K = 2560 and 640)
    ((72, 640, 1090), 90, 129),    # six blocks; K = 640 and 1090 (17-word rows); nine pattern groups
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-c{c[1]}-n{c[2]}" for c in CASES])
def test_classifier_case(case):
    widths, c, n = case
    rng = np.random.default_rng(c * 131 + n)
    gamma = 0   # gamma* for widths that 64 does not divide
    p = Pair(widths, c, 15, 2 * n, gamma, 0.25, seed=int(rng.integers(1 << 62)), fwd_impl=2)
    for t in range(2):
        note(f"classifier {widths} c={c} n={n} step {t}")
        x = random_pm1((n, widths[0]), rng)
        y = rng.integers(0, c, size=n).astype(np.int32)
        p.step(x, y, t, 0.5, tag=f"step {t}")
    xt = random_pm1((2 * n, widths[0]), rng)
    ref = ob.forward(p.ora, xt)
    # half of the labels from the last layer's own prediction, so that the
    # correct counts are not all near chance
    yt = rng.integers(0, c, size=2 * n).astype(np.int32)
    yt[:n] = ref[-1][:n].argmax(axis=1)
    xb, ytd = p.to_dev(xt, yt)
    note(f"classifier {widths} c={c} forward/eval/exit")
    yh = p.gpu.forward(xb)
    cor = p.gpu.eval(xb, ytd)
    ex = p.gpu.eval_exit(xb, ytd)
    p.torch.cuda.synchronize()
    for l in range(len(widths) - 1):
        np.testing.assert_array_equal(yh[l].cpu().numpy(), ref[l], err_msg=f"y_hat layer {l + 1}")
    got = cor.cpu().numpy()
    np.testing.assert_array_equal(got, ob.evaluate(p.ora, xt, yt))
    assert got[-1] >= n
    np.testing.assert_array_equal(ex.cpu().numpy(), ob.early_exit(p.ora, xt, yt))
