"""GPU parity of the epoch driver (bmlp_train_epoch + bmlp_epoch_rescale)
and of early-exit evaluation (bmlp_eval_exit) against the oracle, bit for
bit: every step's counts, the error fraction, the rescaled p_r and the
state after each epoch; per-layer correct, exit and correct-exit counts."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import synth

from gpu_common import Pair, note, pack_np, torch_cuda

pytestmark = pytest.mark.gpu

IMPLS = {"popcount": 1, "mfma_fp4": 2}


def _epochs(p, x, y, batch, epochs, p_r, seed, n_order=None):
    torch = p.torch
    xb, yt = p.to_dev(x, y)
    n = len(y)
    t = 0
    for e in range(epochs):
        order = np.random.default_rng([seed, e]).permutation(n).astype(np.int32)
        if n_order is not None:
            order = order[:n_order]
        note(f"epoch {e}: {len(order)} indices, batch {batch}, p_r {p_r!r}")
        p_gpu, e_gpu, counts = p.gpu.train_epoch(xb, yt, torch.from_numpy(order).cuda(), t, p_r, batch=batch)
        res = ob.train_epoch(p.ora, x, y, order, batch, t, p_r)
        assert res.steps == counts.shape[0]
        np.testing.assert_array_equal(counts.numpy(), res.stats, err_msg=f"epoch {e} step counts")
        if res.steps:
            assert e_gpu == res.error_fraction
        assert p_gpu == res.p_r, (p_gpu, res.p_r)
        p.check_state(f"after epoch {e}")
        t += res.steps
        p_r = p_gpu
    return p_r


@pytest.mark.parametrize("impl", list(IMPLS))
def test_tiny_workload_two_epochs(impl):
    w = synth.TINY
    p = Pair(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness, w.seed_model,
             fwd_impl=IMPLS[impl])
    d = synth.make_split(w, "train", n=1000)   # 7 full batches of 128, 104 left out
    _epochs(p, d.x, d.y, w.batch, 2, w.p_r, seed=3)


def test_epochs_with_every_variant():
    # the epoch driver runs the variant step: reshuffled groups, sequential
    # clipping, saturated z, fan-in reinforcement and one shared classifier
    from paper_2412_00119_amd import bmlp as B
    v = (B.BMLP_VARIANT_FAN_IN_REINFORCE | B.BMLP_VARIANT_SHARED_CLASSIFIER | B.BMLP_VARIANT_SATURATE_Z
         | B.BMLP_VARIANT_RESHUFFLE_GROUPS | B.BMLP_VARIANT_SEQUENTIAL_CLIP)
    w = synth.TINY
    p = Pair((784, 256, 256), w.n_classes, 7, w.batch, 32, w.robustness, w.seed_model, variants=v)
    d = synth.make_split(w, "train", n=600)
    _epochs(p, d.x, d.y, w.batch, 2, w.p_r, seed=9)


def test_ragged_shapes_epochs():
    # odd word counts (37, 130 inputs), gamma* = 105, batch below max_batch
    p = Pair((130, 525, 37), 7, 9, 64, 0, 0.25, seed=21)
    rng = np.random.default_rng(4)
    x = np.where(rng.random((150, 130)) < 0.5, 1, -1).astype(np.int8)
    y = rng.integers(0, 7, 150).astype(np.int32)
    _epochs(p, x, y, 48, 2, 0.9, seed=5)


def test_epoch_without_a_full_batch():
    p = Pair((64, 64), 4, 7, 32, 64, 0.25, seed=2)
    rng = np.random.default_rng(6)
    x = np.where(rng.random((40, 64)) < 0.5, 1, -1).astype(np.int8)
    y = rng.integers(0, 4, 40).astype(np.int32)
    assert _epochs(p, x, y, 32, 1, 0.4, seed=7, n_order=20) == 0.4


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("r", [0.0, 0.25, 100.0])
def test_early_exit_matches(impl, r):
    w = synth.SMALL
    p = Pair(w.widths, w.n_classes, w.bound, 300, w.group_size, r, w.seed_model, fwd_impl=IMPLS[impl])
    d = synth.make_split(w, "train", n=512)
    for t, (x, y) in enumerate(d.batches(256)):
        p.step(x, y, t, w.p_r, check_state=False)
    te = synth.make_split(w, "test", n=300)
    xb, yt = p.to_dev(te.x, te.y)
    note(f"eval_exit r={r}")
    got = p.gpu.eval_exit(xb[:200], yt[:200])
    got = p.gpu.eval_exit(xb[200:], yt[200:], got)    # counts add up over batches
    p.torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), ob.early_exit(p.ora, te.x, te.y))


def test_small_workload_five_epochs():
    # The 784 -> 1024 -> 1024 workload over its whole schedule: five epochs of
    # 234 full batches of 256 through bmlp_train_epoch, the p_r rescale after
    # each (Alg. 1's epoch loop, Sec. 3.4), against the oracle's run stored by
    # tests/golden/make_oracle_golden.py: every step's counts, E^e, the next
    # p_r, H_l after each epoch, and held-out early-exit counts (Sec. 3.1).
    import hashlib
    import json
    import os
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "small_five_epochs.json")))
    w = synth.SMALL
    assert (tuple(gold["widths"]), gold["batch"], gold["bound"]) == (w.widths, w.batch, w.bound)
    net = BMLP(w.widths, w.n_classes, w.bound, 1000, w.group_size, w.robustness, w.seed_model)
    tr = synth.make_split(w, "train")
    te = synth.make_split(w, "test")
    xb = net.pack(torch.from_numpy(tr.x).cuda())
    yt = torch.from_numpy(tr.y.astype(np.int32)).cuda()
    xe = net.pack(torch.from_numpy(te.x).cuda())
    ye = torch.from_numpy(te.y.astype(np.int32)).cuda()
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    P0 = [ob.init_layer(cfg, l)[1] for l in range(1, w.n_layers + 1)]
    p_r, t = w.p_r, 0
    for ep in gold["epochs"]:
        e = ep["epoch"]
        assert ep["step0"] == t and float.fromhex(ep["p_r"]) == p_r
        order = torch.from_numpy(synth.epoch_order(w, e, len(tr.y)).astype(np.int32)).cuda()
        p_next, err_frac, counts = net.train_epoch(xb, yt, order, t, p_r, batch=w.batch)
        np.testing.assert_array_equal(counts.numpy(), np.asarray(ep["stats"]), err_msg=f"epoch {e} step counts")
        assert err_frac == float.fromhex(ep["error_fraction"]), (e, err_frac)
        assert p_next == float.fromhex(ep["p_r_next"]), (e, p_next)
        for l in range(1, w.n_layers + 1):
            h = net.H(l).cpu().numpy()
            assert hashlib.sha256(h.tobytes()).hexdigest() == ep["h_sha256"][l - 1], f"epoch {e} H_{l}"
            Wg = net.W(l).cpu().numpy().view(np.uint64)
            np.testing.assert_array_equal(Wg, pack_np(np.where(h > 0, 1, -1).astype(np.int8), Wg.shape[1]),
                                          err_msg=f"epoch {e} W_{l} = sign(H_{l})")
            Pg = net.P(l).cpu().numpy().view(np.uint64)
            np.testing.assert_array_equal(Pg, pack_np(P0[l - 1], Pg.shape[1]), err_msg=f"epoch {e} P_{l}")
        exits = None
        for s in range(0, len(te.y), 1000):
            exits = net.eval_exit(xe[s:s + 1000], ye[s:s + 1000], exits)
        exits = exits.cpu().numpy()
        np.testing.assert_array_equal(exits, np.asarray(ep["heldout_exit_counts"]), err_msg=f"epoch {e} exits")
        note(f"epoch {e}: E = {err_frac:.5f}, p_r -> {p_next:.6f}, held-out correct per layer "
             f"{exits[:, 0].tolist()} of {len(te.y)}, exits {exits[:, 1].tolist()}")
        t += counts.shape[0]
        p_r = p_next
