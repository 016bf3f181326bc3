"""CPU oracle of the fully binary BMLP training step (arXiv 2412.00119).

TEST INFRASTRUCTURE ONLY: the plain, slow, dense ±1 reference that the GPU
library is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it.  It shares no code, headers,
tables or helpers with the GPU path, and the GPU path never imports it.

Every function is pinned by the CPU tests (brute force on tiny layers, the
popcount identity, invariants of the update, the paper's worked examples of
the group-size rule, and an independent library Philox).
"""
from .bmlp import (Config, State, init, train_step, forward, evaluate, gamma_star,
                   robustness_threshold, reinforce_probability, reinforce_threshold,
                   reinforce_draws, reinforce_mask, stream_bits, LayerTrace)
from .philox import philox4x32_10

__all__ = ["Config", "State", "init", "train_step", "forward", "evaluate", "gamma_star",
           "robustness_threshold", "reinforce_probability", "reinforce_threshold",
           "reinforce_draws", "reinforce_mask", "stream_bits", "LayerTrace", "philox4x32_10"]
