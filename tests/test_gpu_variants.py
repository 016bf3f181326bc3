"""GPU parity of the method variants (bmlp_config.variants) with the
oracle, bit for bit, every step: K_{l-1} in the reinforcement probability,
one classifier shared by every layer, the selection on z held in
min(8, ceil(log2(2 K_{l-1}))) bits, group membership drawn again every
step, and the increments clipped pattern by pattern."""
import dataclasses

import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import bmlp as B
from paper_2412_00119_amd import synth

from gpu_common import Pair, note

pytestmark = pytest.mark.gpu

IMPLS = {"popcount": 1, "mfma_fp4": 2}
VARIANTS = {
    "fan_in": B.BMLP_VARIANT_FAN_IN_REINFORCE,
    "shared": B.BMLP_VARIANT_SHARED_CLASSIFIER,
    "saturate": B.BMLP_VARIANT_SATURATE_Z,
    "reshuffle": B.BMLP_VARIANT_RESHUFFLE_GROUPS,
    "sequential": B.BMLP_VARIANT_SEQUENTIAL_CLIP,
    "all": B.BMLP_VARIANT_FAN_IN_REINFORCE | B.BMLP_VARIANT_SHARED_CLASSIFIER | B.BMLP_VARIANT_SATURATE_Z
    | B.BMLP_VARIANT_RESHUFFLE_GROUPS | B.BMLP_VARIANT_SEQUENTIAL_CLIP,
}


def _run(widths, gamma, variants, impl, steps=6, p_r=0.5, r=0.25):
    w = synth.TINY    # prototype data: rows align with prototypes, so |z| grows past 127
    p = Pair(widths, w.n_classes, 15, w.batch, gamma, r, seed=17, fwd_impl=IMPLS[impl], variants=variants)
    d = synth.make_split(w, "train", n=steps * w.batch)
    zmax = 0
    for t, (x, y) in enumerate(d.batches(w.batch)):
        note(f"variants {variants} impl {impl} widths {widths} step {t}")
        p.step(x, y, t, p_r, tag=f"step {t}")
        zmax = max(zmax, max(int(np.abs(ob.preactivation(x, p.ora.W(1))).max()), 0))
    return p, zmax


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("name", list(VARIANTS))
def test_variant_matches_oracle(name, impl):
    p, zmax = _run((784, 256, 256), 64, VARIANTS[name], impl)
    if name in ("saturate", "all"):
        assert zmax > 128      # the clip to [-128, 127] was in play
    if name in ("shared", "all"):
        np.testing.assert_array_equal(p.gpu.P(1).cpu().numpy(), p.gpu.P(2).cpu().numpy())


@pytest.mark.parametrize("impl", list(IMPLS))
def test_saturated_selection_with_gamma_star(impl):
    # gamma* = 105 for 525: the generic selection kernel reads z back
    _run((784, 525), 0, B.BMLP_VARIANT_SATURATE_Z, impl, steps=4)


@pytest.mark.parametrize("impl", list(IMPLS))
def test_reshuffle_large_layer(impl):
    # K = 2304 spans two key chunks of the order kernel and 9 work-groups;
    # gamma* = 96 for 2304: 24 groups whose rows come from all over the layer
    _run((784, 2304), 0, B.BMLP_VARIANT_RESHUFFLE_GROUPS, impl, steps=3)


@pytest.mark.parametrize("impl", list(IMPLS))
def test_sequential_clip_saturating(impl):
    # B = 3 with prototype data: rows saturate within a step, so the order of
    # the increments shows; gamma = 16 gives 64 selections per pattern
    w = synth.TINY
    p = Pair((784, 1024), w.n_classes, 3, w.batch, 16, 0.25, seed=23, fwd_impl=IMPLS[impl],
             variants=B.BMLP_VARIANT_SEQUENTIAL_CLIP)
    d = synth.make_split(w, "train", n=3 * w.batch)
    order_showed = False
    for t, (x, y) in enumerate(d.batches(w.batch)):
        note(f"sequential clip impl {impl} step {t}")
        # the batch reading from the same state, on the CPU
        alt = p.ora.copy()
        alt.cfg = dataclasses.replace(p.ora.cfg, sequential_clip=False)
        ob.train_step(alt, x, y, t, 0.5)
        p.step(x, y, t, 0.5, tag=f"step {t}")
        order_showed |= not np.array_equal(alt.H[0], p.ora.H[0])
    assert order_showed


RAGGED = [
    # widths, c, B, gamma, n, steps, p_r, r
    ((37, 24, 12), 3, 5, 4, 9, 4, 2.0, 0.25),          # K_l not a multiple of 4 or 64
    ((70, 60, 60), 5, 1, 6, 33, 3, 0.5, 0.25),          # B = 1
    ((1000, 525), 10, 15, 0, 100, 3, 0.5, 0.25),        # gamma* = 105
    ((200, 135, 135), 10, 3, 0, 64, 3, 0.5, 0.25),      # gamma* = 135, B = 3
]


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("case", RAGGED, ids=[f"{c[0]}-B{c[2]}-g{c[3]}-n{c[4]}" for c in RAGGED])
def test_all_variants_ragged(case, impl):
    widths, c, bound, gamma, n, steps, p_r, r = case
    v = (B.BMLP_VARIANT_FAN_IN_REINFORCE | B.BMLP_VARIANT_SATURATE_Z | B.BMLP_VARIANT_RESHUFFLE_GROUPS
         | B.BMLP_VARIANT_SEQUENTIAL_CLIP)
    if len(set(widths[1:])) == 1:
        v |= B.BMLP_VARIANT_SHARED_CLASSIFIER
    rng = np.random.default_rng(sum(widths) + n + 7)
    p = Pair(widths, c, bound, n + 3, gamma, r, seed=int(rng.integers(1 << 62)), fwd_impl=IMPLS[impl],
             variants=v)
    for t in range(steps):
        note(f"variants {v} shape {widths} step {t}")
        x = synth.random_pm1((n, widths[0]), rng)
        y = rng.integers(0, c, size=n).astype(np.int32)
        p.step(x, y, 500 + t, p_r, tag=f"step {t}")
