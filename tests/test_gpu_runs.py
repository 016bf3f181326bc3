"""The 3072 -> 4096 x 4 and 3072 -> 2048 x 3 workloads over their first 24
steps, bit-exact against the oracle's run stored in tests/golden/ (written
by tests/golden/make_oracle_golden.py from oracle/ and the input generator
only; an oracle step of the 4096-wide network takes about 45 s on the host,
too slow to run beside the GPU).  The first steps have every pattern in
M_l; the later ones have a few, where the update is mostly the reinforcement
pass over every hidden weight: the regime the benchmark times.  Per step and
layer: the counts (01-loss, |M_l|, |U_l|, reinforced draws), a_l and H_l by
SHA-256, and W_l = sign(H_l); on both forward paths."""
import hashlib
import json
import os

import numpy as np
import pytest

from paper_2412_00119_amd import synth

from gpu_common import note, pack_np, torch_cuda, unpack

pytestmark = pytest.mark.gpu

IMPLS = {"popcount": 1, "mfma_fp4": 2}
RUNS = {"headline": ("headline_24_steps.json", synth.HEADLINE),
        "field": ("field_24_steps.json", synth.FIELD)}


def _sha(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=np.int8).tobytes()).hexdigest()


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("run", list(RUNS))
def test_stored_run(run, impl):
    torch = torch_cuda()
    from paper_2412_00119_amd.bmlp import BMLP
    fname, w = RUNS[run]
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", fname)))
    assert (tuple(gold["widths"]), gold["batch"], gold["bound"], gold["classes"]) == \
        (w.widths, w.batch, w.bound, w.n_classes)
    p_r = float.fromhex(gold["p_r"])
    net = BMLP(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness, w.seed_model,
               IMPLS[impl])
    d = synth.make_split(w, "train", n=len(gold["steps"]) * w.batch)
    for (x, y), g in zip(d.batches(w.batch), gold["steps"]):
        t = g["t"]
        note(f"{w.name} {impl} step {t}")
        xb = net.pack(torch.from_numpy(x).cuda())
        yt = torch.from_numpy(y.astype(np.int32)).cuda()
        stats = net.train_step(xb, yt, t, p_r)
        torch.cuda.synchronize()
        st = stats.cpu().numpy()
        for l in range(1, w.n_layers + 1):
            tag = f"{w.name} {impl} t={t} layer {l}"
            np.testing.assert_array_equal(st[l - 1][:4], np.asarray(g["stats"][l - 1]), err_msg=f"{tag} counts")
            a = unpack(net.trace(l, w.batch)["a"], w.widths[l])
            assert _sha(a) == g["a_sha256"][l - 1], f"{tag} a_l"
            h = net.H(l).cpu().numpy()
            assert _sha(h) == g["h_sha256"][l - 1], f"{tag} H_l"
            Wg = net.W(l).cpu().numpy().view(np.uint64)
            np.testing.assert_array_equal(Wg, pack_np(np.where(h > 0, 1, -1).astype(np.int8), Wg.shape[1]),
                                          err_msg=f"{tag} W_l = sign(H_l)")
