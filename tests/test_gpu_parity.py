"""Bit-exact parity of the HIP library with the CPU oracle: activations,
01-loss, update mask, selected perceptrons, statistics, hidden weights,
visible weights and classifiers, after every step."""
import numpy as np
import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import synth
from paper_2412_00119_amd.synth import random_pm1

from gpu_common import Pair, note, pack_np, torch_cuda, unpack

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,K", [(1, 1), (3, 63), (5, 64), (7, 65), (130, 784), (64, 3072), (9, 200)])
def test_pack(n, K):
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    note(f"pack n={n} K={K}")
    net = BMLP((K, 64), 2, 1, 8)
    rng = np.random.default_rng(K)
    x = random_pm1((n, K), rng)
    bits = net.pack(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), pack_np(x, bits.shape[1]))


@pytest.mark.parametrize("widths,c,gamma", [((37, 24, 12), 3, 4), ((784, 256), 10, 64),
                                            ((1000, 525, 525), 10, 0), ((64, 130), 7, 13)])
def test_init_matches_oracle(widths, c, gamma):
    note(f"init {widths} c={c} gamma={gamma}")
    p = Pair(widths, c, 15, 16, gamma, seed=0xDEADBEEF12345)
    p.check_state("init")


CASES = [
    # widths, c, B, gamma, n, steps, p_r, r
    ((37, 24, 12), 3, 5, 4, 9, 4, 2.0, 0.25),
    ((130, 192), 7, 9, 64, 130, 3, 0.5, 0.25),
    ((64, 96, 64), 2, 3, 32, 257, 3, 1.0, 0.25),
    ((1000, 525), 10, 15, 0, 100, 3, 0.5, 0.25),      # gamma* = 105
    ((200, 135, 135), 10, 15, 0, 64, 3, 0.5, 0.25),   # gamma* = 135
    ((70, 64), 5, 1, 8, 33, 3, 0.5, 0.25),            # B = 1: pure binary
    ((70, 64), 5, 7, 8, 33, 2, 0.0, 0.0),             # no reinforcement, r = 0
    ((3000, 128, 128), 100, 31, 64, 200, 2, 0.5, 0.25),
    ((48, 64), 4, 127, 64, 16, 3, 50.0, 0.25),       # one group per layer, T saturates
]


IMPLS = {"popcount": 1, "mfma_fp4": 2}


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-c{c[1]}-B{c[2]}-g{c[3]}-n{c[4]}" for c in CASES])
def test_random_shapes(case, impl):
    widths, c, bound, gamma, n, steps, p_r, r = case
    rng = np.random.default_rng(sum(widths) + n)
    p = Pair(widths, c, bound, n + 3, gamma, r, seed=int(rng.integers(1 << 62)), fwd_impl=IMPLS[impl])
    for t in range(steps):
        note(f"shape {widths} step {t}")
        x = random_pm1((n, widths[0]), rng)
        y = rng.integers(0, c, size=n).astype(np.int32)
        p.step(x, y, 1000 + t, p_r, tag=f"step {t}")


def _workload_run(w, steps, n=None, check_every=1, fwd_impl=0):
    n = w.batch if n is None else n
    p = Pair(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness, w.seed_model,
             fwd_impl=fwd_impl)
    d = synth.make_split(w, "train", n=steps * n)
    for t, (x, y) in enumerate(d.batches(n)):
        if t >= steps:
            break
        note(f"{w.name} step {t}")
        p.step(x, y, t, w.p_r, check_state=(t % check_every == 0 or t == steps - 1), tag=f"{w.name} t={t}")
    return p


@pytest.mark.parametrize("impl", list(IMPLS))
def test_tiny_workload_full_epoch(impl):
    w = synth.TINY
    _workload_run(w, w.steps_per_epoch, fwd_impl=IMPLS[impl])


@pytest.mark.parametrize("impl", list(IMPLS))
def test_small_workload(impl):
    _workload_run(synth.SMALL, 4, fwd_impl=IMPLS[impl])


def test_field_workload():
    _workload_run(synth.FIELD, 2)


def test_headline_workload_two_steps():
    _workload_run(synth.HEADLINE, 2)


@pytest.mark.parametrize("impl", list(IMPLS))
def test_forward_and_eval_match(impl):
    torch = torch_cuda()
    w = synth.SMALL
    p = Pair(w.widths, w.n_classes, w.bound, 300, w.group_size, w.robustness, w.seed_model,
             fwd_impl=IMPLS[impl])
    d = synth.make_split(w, "train", n=512)
    for t, (x, y) in enumerate(d.batches(256)):
        p.step(x, y, t, w.p_r, check_state=False)
    te = synth.make_split(w, "test", n=300)
    xb, yt = p.to_dev(te.x, te.y)
    note("forward/eval")
    yh = p.gpu.forward(xb)
    cor = p.gpu.eval(xb, yt)
    torch.cuda.synchronize()
    ref = ob.forward(p.ora, te.x)
    for l in range(2):
        np.testing.assert_array_equal(yh[l].cpu().numpy(), ref[l])
    np.testing.assert_array_equal(cor.cpu().numpy(), ob.evaluate(p.ora, te.x, te.y))


def test_step_is_deterministic():
    """The same step from the same state gives the same bytes."""
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    w = synth.SMALL
    d = synth.make_split(w, "train", n=256)
    outs = []
    for rep in range(2):
        net = BMLP(w.widths, w.n_classes, w.bound, 256, w.group_size, w.robustness, 5)
        xb = net.pack(torch.from_numpy(d.x).cuda())
        yt = torch.from_numpy(d.y).cuda()
        for t in range(3):
            net.train_step(xb, yt, t, 0.5)
        torch.cuda.synchronize()
        outs.append(net.state.cpu().numpy().copy())
    np.testing.assert_array_equal(outs[0], outs[1])


def test_resume_from_state_is_exact():
    """Continuing from a copy of the state (H and P only; W is re-derived)
    equals an uninterrupted run."""
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    w = synth.SMALL
    d = synth.make_split(w, "train", n=256 * 4)
    batches = list(d.batches(256))
    a = BMLP(w.widths, w.n_classes, w.bound, 256, w.group_size, w.robustness, 9)
    for t, (x, y) in enumerate(batches):
        xb, yt = a.pack(torch.from_numpy(x).cuda()), torch.from_numpy(y).cuda()
        a.train_step(xb, yt, t, 0.5)
    b = BMLP(w.widths, w.n_classes, w.bound, 256, w.group_size, w.robustness, 9)
    for t, (x, y) in enumerate(batches[:2]):
        xb, yt = b.pack(torch.from_numpy(x).cuda()), torch.from_numpy(y).cuda()
        b.train_step(xb, yt, t, 0.5)
    snap = b.state.clone()
    for l in (1, 2):   # scramble W in the snapshot: attach must rebuild it from H
        i = b.info[l - 1]
        snap[i.off_w:i.off_w + i.k_out * i.words_in * 8] = 0
    c = BMLP(w.widths, w.n_classes, w.bound, 256, w.group_size, w.robustness, 9, state=snap)
    for t, (x, y) in enumerate(batches[2:], start=2):
        xb, yt = c.pack(torch.from_numpy(x).cuda()), torch.from_numpy(y).cuda()
        c.train_step(xb, yt, t, 0.5)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(a.state.cpu().numpy(), c.state.cpu().numpy())


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("variants", [0, 16], ids=["batch_clip", "sequential_clip"])
def test_maximum_batch(impl, variants):
    # 16384 patterns, the most the library takes (the update's selector
    # entries keep a pattern index in 15 bits, the sign of rho in the 16th)
    n = 16384
    rng = np.random.default_rng(77)
    p = Pair((64, 128, 64), 10, 7, n, 16, 0.25, seed=99, fwd_impl=IMPLS[impl], variants=variants)
    for t in range(2):
        note(f"maximum batch {n} variants {variants} step {t}")
        x = random_pm1((n, 64), rng)
        y = rng.integers(0, 10, size=n).astype(np.int32)
        p.step(x, y, t, 0.5, tag=f"step {t}")


@pytest.mark.parametrize("impl", list(IMPLS))
def test_maximum_width(impl):
    # K_1 = 32767, the widest layer the library takes (|z| of layer 2 is
    # bounded by 32767, int16's range): gamma* = 31, 1057 groups, and
    # layer 2 reads 1024-word rows
    rng = np.random.default_rng(78)
    p = Pair((64, 32767, 48), 5, 7, 256, 0, 0.25, seed=98, fwd_impl=IMPLS[impl])
    for t in range(2):
        note(f"maximum width step {t}")
        x = random_pm1((256, 64), rng)
        y = rng.integers(0, 5, size=256).astype(np.int32)
        p.step(x, y, t, 0.5, tag=f"step {t}")
