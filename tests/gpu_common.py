"""Helpers shared by the GPU parity tests: run the HIP library and the oracle
on the same seeded inputs and compare every observable bit for bit."""
import sys

import numpy as np
import pytest

import oracle.bmlp as ob


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    return torch


def note(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def unpack(bits_t, K: int) -> np.ndarray:
    """int64 bit rows [n][w] (tensor) -> int8 ±1 [n][K]."""
    a = bits_t.detach().cpu().numpy()
    n = a.shape[0]
    b = np.unpackbits(a.view(np.uint8).reshape(n, -1), axis=1, bitorder="little")
    return np.where(b[:, :K] == 1, 1, -1).astype(np.int8)


def pack_np(pm1: np.ndarray, words: int) -> np.ndarray:
    """int8 ±1 [n][K] -> uint64 [n][words] with zero tail bits (numpy route)."""
    n, K = pm1.shape
    b = np.packbits(pm1 > 0, axis=1, bitorder="little")
    out = np.zeros((n, words * 8), dtype=np.uint8)
    out[:, :b.shape[1]] = b
    return out.view(np.uint64)


class Pair:
    """A GPU network and an oracle network from the same configuration."""

    def __init__(self, widths, c, bound, max_batch, gamma=64, r=0.25, seed=1, fwd_impl=0, variants=0):
        torch = torch_cuda()
        from paper_2412_00119_amd import bmlp as B
        self.torch = torch
        self.gpu = B.BMLP(widths, c, bound, max_batch, gamma, r, seed, fwd_impl, variants=variants)
        self.ora = ob.init(ob.Config(
            widths, c, bound, gamma, r, seed,
            fan_in_reinforce=bool(variants & B.BMLP_VARIANT_FAN_IN_REINFORCE),
            shared_classifier=bool(variants & B.BMLP_VARIANT_SHARED_CLASSIFIER),
            saturate_z=bool(variants & B.BMLP_VARIANT_SATURATE_Z),
            reshuffle_groups=bool(variants & B.BMLP_VARIANT_RESHUFFLE_GROUPS),
            sequential_clip=bool(variants & B.BMLP_VARIANT_SEQUENTIAL_CLIP)))
        self.widths = tuple(widths)
        self.c = c

    def to_dev(self, x, y=None):
        t = self.torch
        xb = self.gpu.pack(t.from_numpy(np.ascontiguousarray(x)).cuda())
        yt = None if y is None else t.from_numpy(np.asarray(y, dtype=np.int32)).cuda()
        return xb, yt

    def check_state(self, tag=""):
        t = self.torch
        t.cuda.synchronize()
        for l in range(1, len(self.widths)):
            H = self.gpu.H(l).cpu().numpy()
            np.testing.assert_array_equal(H, self.ora.H[l - 1], err_msg=f"{tag} H layer {l}")
            Wg = self.gpu.W(l).cpu().numpy().view(np.uint64)
            np.testing.assert_array_equal(Wg, pack_np(self.ora.W(l), Wg.shape[1]),
                                          err_msg=f"{tag} W layer {l}")
            Pg = self.gpu.P(l).cpu().numpy().view(np.uint64)
            np.testing.assert_array_equal(Pg, pack_np(self.ora.P[l - 1], Pg.shape[1]),
                                          err_msg=f"{tag} P layer {l}")

    def step(self, x, y, t, p_r, check_state=True, tag=""):
        torch = self.torch
        xb, yt = self.to_dev(x, y)
        stats = self.gpu.train_step(xb, yt, t, p_r)
        torch.cuda.synchronize()
        tr = ob.train_step(self.ora, x, y, t, p_r)
        n = len(y)
        st = stats.cpu().numpy()
        for l, lt in enumerate(tr, start=1):
            g = self.gpu.trace(l, n)
            np.testing.assert_array_equal(unpack(g["a"], self.widths[l]), lt.a, err_msg=f"{tag} a_{l}")
            np.testing.assert_array_equal(g["err"].cpu().numpy(), lt.err.astype(np.uint8),
                                          err_msg=f"{tag} err_{l}")
            np.testing.assert_array_equal(g["upd"].cpu().numpy(), lt.upd.astype(np.uint8),
                                          err_msg=f"{tag} upd_{l}")
            # the library keeps the selection of every pattern; U_l is its
            # restriction to the patterns in M_l (checked through H and stats)
            cfg = self.ora.cfg
            raw = ob.select_easiest(lt.z, self.ora.P[l - 1], np.asarray(y), np.ones(len(y), bool),
                                    cfg.gamma(self.widths[l]), lt.perm)
            ks = g["kstar"].cpu().numpy()
            np.testing.assert_array_equal(ks, raw, err_msg=f"{tag} kstar_{l}")
            np.testing.assert_array_equal(np.where(lt.upd[:, None], ks, -1), lt.kstar,
                                          err_msg=f"{tag} U_{l}")
            np.testing.assert_array_equal(st[l - 1], lt.stats, err_msg=f"{tag} stats_{l}")
        if check_state:
            self.check_state(tag)
        return st
