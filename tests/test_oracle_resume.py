"""Checkpoint/resume of the oracle is exact: the random draws depend only on
(seed, layer, step, index), so the state after t1 + t2 steps does not depend
on whether the run was stopped and restored in between."""
import numpy as np

import oracle.bmlp as ob
from paper_2412_00119_amd.synth import random_pm1


def test_resume_bit_exact(tmp_path):
    cfg = ob.Config((60, 32, 32), 5, 15, 8, 0.25, 77)
    rng = np.random.default_rng(0)
    batches = [(random_pm1((24, 60), rng), rng.integers(0, 5, size=24)) for _ in range(6)]
    a = ob.init(cfg)
    for t, (x, y) in enumerate(batches):
        ob.train_step(a, x, y, t, 0.7)
    b = ob.init(cfg)
    for t, (x, y) in enumerate(batches[:3]):
        ob.train_step(b, x, y, t, 0.7)
    np.savez(tmp_path / "ck.npz", *b.H)
    with np.load(tmp_path / "ck.npz") as f:
        H = [f[f"arr_{i}"] for i in range(2)]
    c = ob.State(cfg, H, ob.init(cfg).P)        # P is re-derived from the seed
    for t, (x, y) in enumerate(batches[3:], start=3):
        ob.train_step(c, x, y, t, 0.7)
    for l in range(2):
        np.testing.assert_array_equal(a.H[l], c.H[l])
        np.testing.assert_array_equal(a.P[l], c.P[l])
