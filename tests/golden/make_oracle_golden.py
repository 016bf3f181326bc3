"""Writes the stored expected values that the GPU tests compare against.

Every value here comes from the CPU oracle (oracle/) on inputs from the seeded
input generator (paper_2412_00119_amd/synth.py, which holds none of the
method's arithmetic).  Nothing is read from the HIP library.  Both files are
too slow to recompute inside a GPU test run, which is why they are stored.

    python tests/golden/make_oracle_golden.py small    # small_five_epochs.json
    python tests/golden/make_oracle_golden.py stress   # stress_step0_reinforced.txt
    python tests/golden/make_oracle_golden.py headline # headline_24_steps.json
    python tests/golden/make_oracle_golden.py field    # field_24_steps.json

small: the 784 -> 1024 -> 1024 workload (10 classes, B = 127, batch 256,
60 000 training and 10 000 held-out samples) over its five-epoch schedule:
Algorithm 1's epoch loop with the p_r <- p_r sqrt(E^e) rescale after each
epoch (Section 3.4), epoch e visiting the training set in the order
synth.epoch_order(w, e, N) and stepping t = 234 e, ..., 234 e + 233.  After
each epoch it records every step's layer counts, E^e, the next p_r (as a
hexadecimal double, so it round-trips exactly), the SHA-256 of each H_l
(int8, [K_l][K_{l-1}], C order), and on the held-out split each layer's
correct, exit and correct-exit counts (early exit, Section 3.1).

stress: the 8192 -> 8192 x 8 workload's first step (t = 0, p_r = 0.5): the
number of reinforcement draws u < T_l over every hidden weight of each layer
(Algorithm 3), the one step statistic a GPU test cannot afford to recompute.

headline, field: the 3072 -> 4096 x 4 workload (100 classes, B = 31, batch
1024) and the 3072 -> 2048 x 3 workload (10 classes, B = 127, batch 512) over
their first 24 steps (t = 0 .. 23, p_r = 0.5, batch b of the training split's
first 24 batches at step b): the steps where every pattern is in M_l and the
ones after them where M_l has a few patterns and the update is mostly the
reinforcement pass.  Per step and layer: the counts (01-loss, |M_l|, |U_l|,
reinforced draws) and the SHA-256 of a_l (int8 ±1, [n][K_l], C order) and of
H_l after the step (int8, [K_l][K_{l-1}], C order).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle.bmlp as ob  # noqa: E402
from paper_2412_00119_amd import synth  # noqa: E402

SMALL_FILE = os.path.join(HERE, "small_five_epochs.json")
RUN_FILES = {"headline": os.path.join(HERE, "headline_24_steps.json"),
             "field": os.path.join(HERE, "field_24_steps.json")}
RUN_STEPS = 24
STRESS_FILE = os.path.join(HERE, "stress_step0_reinforced.txt")


def h_digest(h: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(h, dtype=np.int8).tobytes()).hexdigest()


def small() -> None:
    w = synth.SMALL
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    st = ob.init(cfg)
    tr = synth.make_split(w, "train")
    te = synth.make_split(w, "test")
    p_r, t = w.p_r, 0
    epochs = []
    for e in range(w.epochs):
        t0 = time.time()
        order = synth.epoch_order(w, e, len(tr.y))
        res = ob.train_epoch(st, tr.x, tr.y, order, w.batch, t, p_r)
        exits = ob.early_exit(st, te.x, te.y)
        epochs.append({
            "epoch": e,
            "step0": t,
            "p_r": p_r.hex(),
            "steps": res.steps,
            "error_fraction": res.error_fraction.hex(),
            "p_r_next": res.p_r.hex(),
            "stats": res.stats.astype(int).tolist(),
            "h_sha256": [h_digest(st.H[l]) for l in range(cfg.n_layers)],
            "heldout_exit_counts": exits.astype(int).tolist(),
        })
        print(f"epoch {e}: E = {res.error_fraction:.5f}, p_r -> {res.p_r:.6f}, "
              f"held-out correct {exits[:, 0].tolist()} ({time.time() - t0:.0f} s)", flush=True)
        t += res.steps
        p_r = res.p_r
    out = {"workload": w.name, "widths": list(w.widths), "classes": w.n_classes, "bound": w.bound,
           "batch": w.batch, "n_train": len(tr.y), "n_test": len(te.y), "seed_model": w.seed_model,
           "robustness": w.robustness, "group_size": w.group_size, "epochs": epochs,
           "made_by": "python tests/golden/make_oracle_golden.py small"}
    with open(SMALL_FILE, "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")


def stress() -> None:
    w = synth.STRESS
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    lines = ["# Reinforcement draws u < T_l over all hidden weights of each layer of the",
             "# 8192 -> 8192 x 8 workload at its first step (t = 0, p_r = 0.5), from the",
             "# oracle: python tests/golden/make_oracle_golden.py stress",
             "# columns: layer  K_{l-1}  K_l  T_l  reinforced"]
    for l in range(1, cfg.n_layers + 1):
        kin, kout = w.widths[l - 1], w.widths[l]
        T = ob.reinforce_threshold(w.p_r, kout)
        n = int(ob.reinforce_mask(cfg.seed, l, 0, T, kin * kout, kin).sum())
        lines.append(f"{l} {kin} {kout} {T} {n}")
        print(lines[-1], flush=True)
    with open(STRESS_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")


def steps_run(name: str) -> None:
    w = {"headline": synth.HEADLINE, "field": synth.FIELD}[name]
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    st = ob.init(cfg)
    d = synth.make_split(w, "train", n=RUN_STEPS * w.batch)
    steps = []
    for t, (x, y) in enumerate(d.batches(w.batch)):
        t0 = time.time()
        tr = ob.train_step(st, x, y, t, w.p_r)
        steps.append({
            "t": t,
            "stats": [lt.stats.astype(int).tolist() for lt in tr],
            "a_sha256": [h_digest(lt.a) for lt in tr],
            "h_sha256": [h_digest(st.H[l]) for l in range(cfg.n_layers)],
        })
        print(f"{name} step {t}: |M| {[int(lt.stats[1]) for lt in tr]} ({time.time() - t0:.0f} s)", flush=True)
    out = {"workload": w.name, "widths": list(w.widths), "classes": w.n_classes, "bound": w.bound,
           "batch": w.batch, "seed_model": w.seed_model, "robustness": w.robustness,
           "group_size": w.group_size, "p_r": w.p_r.hex(), "steps": steps,
           "made_by": f"python tests/golden/make_oracle_golden.py {name}"}
    with open(RUN_FILES[name], "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")


if __name__ == "__main__":
    which = sys.argv[1:] or ["small", "stress", "headline", "field"]
    for name in which:
        {"small": small, "stress": stress, "headline": lambda: steps_run("headline"),
         "field": lambda: steps_run("field")}[name]()
