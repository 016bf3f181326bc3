"""Parity at the largest workload (8192 -> 8192 x 8, 1000 classes, batch 4096,
B = 63) in the launch configuration the benchmark uses, through all eight
layers:

* for every layer and all 4096 patterns: a_l, 01-loss, M_l, the selected
  perceptrons of every group, and the step counts |errors|, |M_l|, |U_l|;
* the fourth count (reinforcement draws that fired over all 67 M hidden
  weights of the layer) against the oracle's value stored in
  tests/golden/stress_step0_reinforced.txt (too slow to recompute here);
* H_l and W_l after the step on sampled rows of every layer (the first and
  last rows of the first and last groups, and random rows), the oracle's
  Clipped-Perceptron sum, clip and reinforcement applied to those rows;
* P_l of every layer.

The oracle's functions are applied exactly as its train_step applies them
(Algorithms 1-3), with every layer's forward from the pre-step weights."""
import os

import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import synth

from gpu_common import note, pack_np, torch_cuda, unpack

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "stress_step0_reinforced.txt")


def _stored_reinforced():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        l, kin, kout, T, n = (int(v) for v in line.split())
        out[l] = (kin, kout, T, n)
    return out


def test_stress_workload_every_layer():
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    w = synth.STRESS
    t, p_r = 0, w.p_r
    stored = _stored_reinforced()
    note(f"stress {w.widths} c={w.n_classes} B={w.bound} bs={w.batch}: GPU step")
    net = BMLP(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness, w.seed_model)
    x, y = synth.stream_batch(w, 0)
    y = np.asarray(y, dtype=np.int64)
    xb = net.pack(torch.from_numpy(np.ascontiguousarray(x)).cuda())
    stats = net.train_step(xb, torch.from_numpy(y.astype(np.int32)).cuda(), t, p_r)
    torch.cuda.synchronize()
    st = stats.cpu().numpy()
    n, L = w.batch, w.n_layers
    rng = np.random.default_rng(5)

    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    a_prev = np.asarray(x, dtype=np.int8)
    for l in range(1, L + 1):
        note(f"oracle layer {l}")
        kin, kout = w.widths[l - 1], w.widths[l]
        gamma = cfg.gamma(kout)
        H, P = ob.init_layer(cfg, l)
        W = np.where(H > 0, 1, -1).astype(np.int8)
        z = ob.preactivation(a_prev, W)
        a = ob.activation(z)
        _, _, err, upd = ob.local_error(ob.local_output(a, P), y, ob.robustness_threshold(w.robustness, kout))
        raw = ob.select_easiest(z, P, y, np.ones(n, bool), gamma)
        del z
        kstar = np.where(upd[:, None], raw, -1).astype(np.int16)
        g = net.trace(l, n)
        Pg = net.P(l).cpu().numpy().view(np.uint64)
        np.testing.assert_array_equal(Pg, pack_np(P, Pg.shape[1]), err_msg=f"P_{l}")
        np.testing.assert_array_equal(unpack(g["a"], kout), a, err_msg=f"a_{l}")
        np.testing.assert_array_equal(g["err"].cpu().numpy(), err.astype(np.uint8), err_msg=f"err_{l}")
        np.testing.assert_array_equal(g["upd"].cpu().numpy(), upd.astype(np.uint8), err_msg=f"upd_{l}")
        np.testing.assert_array_equal(g["kstar"].cpu().numpy(), raw, err_msg=f"kstar_{l}")
        # sampled rows of H_l: first and last of the first and last groups, and random
        rows = np.unique(np.concatenate([[0, gamma - 1, gamma, kout - gamma, kout - 1],
                                         rng.choice(kout, 11, replace=False)]))
        S = ob.selection_matrix(kstar, P, y, gamma)
        h = ob.clip(H[rows].astype(np.int64) + ob.cp_increment(S[:, rows], a_prev), cfg.bound)
        del S
        T = ob.reinforce_threshold(p_r, kout)
        nreinf = 0
        if upd.any():
            j = (rows[:, None].astype(np.uint64) * np.uint64(kin) + np.arange(kin, dtype=np.uint64)).ravel()
            mask = ob.reinforce_draws(cfg.seed, l, t, j, kin) < np.uint64(T)
            h = ob.reinforce(h, mask, cfg.bound)
            assert stored[l][:3] == (kin, kout, T), f"stored counts are for another layer shape or T ({l})"
            nreinf = stored[l][3]
        want_stats = np.array([err.sum(), upd.sum(), (kstar >= 0).sum(), nreinf], dtype=np.int64)
        np.testing.assert_array_equal(st[l - 1], want_stats, err_msg=f"stats_{l}")
        Hg = net.H(l)[torch.from_numpy(rows).cuda()].cpu().numpy()
        np.testing.assert_array_equal(Hg, h.astype(np.int8), err_msg=f"H_{l} rows {rows.tolist()}")
        Wg = net.W(l)[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint64)
        np.testing.assert_array_equal(Wg, pack_np(np.where(h > 0, 1, -1).astype(np.int8), Wg.shape[1]),
                                      err_msg=f"W_{l} rows")
        note(f"layer {l}: |M| = {int(upd.sum())}, |U| = {int((kstar >= 0).sum())}, reinforced {nreinf}")
        a_prev = a
