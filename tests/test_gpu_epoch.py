"""GPU parity of the epoch driver (bmlp_train_epoch + bmlp_epoch_rescale)
and of early-exit evaluation (bmlp_eval_exit) against the oracle, bit for
bit: every step's counts, the error fraction, the rescaled p_r and the
state after each epoch; per-layer correct, exit and correct-exit counts."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import synth

from gpu_common import Pair, note, torch_cuda

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
