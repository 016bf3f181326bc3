"""MI355X-native train step for fully binary multi-layer perceptrons trained
with random local binary error signals (Colombo, Pittorino, Roveri,
arXiv 2412.00119).

The method runs in the HIP library ``libbmlp.so`` (C ABI in include/bmlp.h);
``paper_2412_00119_amd.bmlp`` is its thin Python binding and
``paper_2412_00119_amd.synth`` generates the seeded synthetic workloads.
Importing the package loads nothing; the library is loaded on first use.
"""
from .bmlp import BMLP, BmlpError  # noqa: F401

__all__ = ["BMLP", "BmlpError"]
