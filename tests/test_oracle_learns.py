"""Sanity, not parity: one epoch of the tiny workload learns far above chance
(the paper's method is a working learning rule, Section 4)."""
import numpy as np

import oracle.bmlp as ob
from paper_2412_00119_amd import synth


def test_tiny_learns_one_epoch():
    w = synth.TINY
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    s = ob.init(cfg)
    before = ob.evaluate(s, *(lambda d: (d.x, d.y))(synth.make_split(w, "test")))
    d = synth.make_split(w)
    errs = []
    for t, (x, y) in enumerate(d.batches(w.batch)):
        tr = ob.train_step(s, x, y, t, w.p_r)
        errs.append(int(tr[-1].stats[0]))
    te = synth.make_split(w, "test")
    acc = ob.evaluate(s, te.x, te.y)[-1] / len(te.y)
    assert acc > 0.8, acc
    assert before[-1] / len(te.y) < 0.5
    assert errs[-1] < errs[0]
