"""Python binding of the HIP train-step library (include/bmlp.h).

Argument marshalling only: every step of the method runs in the library's HIP
kernels.  PyTorch supplies device memory (torch.empty on the GPU) and the
stream (the current torch stream); it computes nothing here.

The functions with the C names (bmlp_init, bmlp_train_step, ...) take raw
integers for pointers and streams; the BMLP class wraps them around torch
buffers.  If the library has not been built, every entry point raises: there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

from .build import LIB_PATH

BMLP_OK = 0
BMLP_EINVAL = -1
BMLP_ESHAPE = -2
BMLP_EHIP = -3
BMLP_ESTATE = -4

BMLP_FWD_AUTO = 0
BMLP_FWD_POPCOUNT = 1
BMLP_FWD_MFMA_FP4 = 2

# method variants (bmlp_config.variants)
BMLP_VARIANT_FAN_IN_REINFORCE = 1
BMLP_VARIANT_SHARED_CLASSIFIER = 2
BMLP_VARIANT_SATURATE_Z = 4
BMLP_VARIANT_RESHUFFLE_GROUPS = 8
BMLP_VARIANT_SEQUENTIAL_CLIP = 16

MAX_BATCH = 16384


class BmlpError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = f"{where}: {status_string(status)} ({status})"
        if status == BMLP_EHIP:
            msg += f": {last_error()}"
        super().__init__(msg)
        self.status = status


class bmlp_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("h_widths", ctypes.POINTER(ctypes.c_int32)),
        ("n_classes", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("bound", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("robustness", ctypes.c_double),
        ("seed", ctypes.c_uint64),
        ("fwd_impl", ctypes.c_int32),
        ("variants", ctypes.c_int32),
    ]


class bmlp_layer_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("k_in", "k_out", "gamma", "groups", "words_in", "words_out", "ld_h", "robust_thr")] + \
               [(n, ctypes.c_uint64) for n in
                ("off_h", "off_w", "off_p", "off_a", "off_err", "off_upd", "off_kstar")] + \
               [(n, ctypes.c_int32) for n in ("h_planes", "h_ps")]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libbmlp.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is missing; build it with "
                               "paper_2412_00119_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double
        cfgp = ctypes.POINTER(bmlp_config)
        sig = {
            "bmlp_state_bytes": (ctypes.c_size_t, [cfgp]),
            "bmlp_workspace_bytes": (ctypes.c_size_t, [cfgp]),
            "bmlp_describe": (ctypes.c_int, [cfgp, i32, ctypes.POINTER(bmlp_layer_info)]),
            "bmlp_reinforce_threshold": (u64, [dbl, i32]),
            "bmlp_init": (ctypes.c_int, [cfgp, vp, vp, vp, ctypes.POINTER(vp)]),
            "bmlp_attach": (ctypes.c_int, [cfgp, vp, vp, vp, ctypes.POINTER(vp)]),
            "bmlp_pack": (ctypes.c_int, [vp, i32, i32, vp, vp]),
            "bmlp_forward": (ctypes.c_int, [vp, vp, i32, vp, vp]),
            "bmlp_forward_noalloc": (ctypes.c_int, [vp, vp, i32, vp, vp]),
            "bmlp_train_step": (ctypes.c_int, [vp, vp, vp, i32, u64, dbl, vp, vp]),
            "bmlp_eval": (ctypes.c_int, [vp, vp, vp, i32, vp, vp]),
            "bmlp_eval_exit": (ctypes.c_int, [vp, vp, vp, i32, vp, vp]),
            "bmlp_feature_median": (ctypes.c_int, [vp, i32, i32, vp, vp]),
            "bmlp_binarize": (ctypes.c_int, [vp, i32, i32, vp, vp, vp]),
            "bmlp_expand": (ctypes.c_int, [vp, i32, i32, i32, u64, vp, vp]),
            "bmlp_train_epoch": (ctypes.c_int, [vp, vp, vp, i32, vp, i32, i32, u64, dbl, vp, vp]),
            "bmlp_epoch_rescale": (dbl, [dbl, ctypes.c_int64, ctypes.c_int64]),
            "bmlp_epoch_summary": (ctypes.c_int, [vp, i32, i32, i32, dbl, ctypes.POINTER(dbl),
                                                  ctypes.POINTER(dbl)]),
            "bmlp_layer_views": (ctypes.c_int, [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                                ctypes.POINTER(vp)]),
            "bmlp_step_trace": (ctypes.c_int, [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                               ctypes.POINTER(vp), ctypes.POINTER(vp)]),
            "bmlp_read_h": (ctypes.c_int, [vp, i32, vp, vp]),
            "bmlp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "bmlp_last_error": (ctypes.c_char_p, []),
            "bmlp_destroy": (None, [vp]),
            "bmlp_profile_start": (ctypes.c_int, [vp, i32]),
            "bmlp_profile_stop": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(ctypes.c_int64)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


# ---------------------------------------------------------------------------
# C-named entry points
# ---------------------------------------------------------------------------

def make_config(widths: Sequence[int], n_classes: int, bound: int, max_batch: int,
                group_size: int = 64, robustness: float = 0.25, seed: int = 0,
                fwd_impl: int = BMLP_FWD_AUTO, variants: int = 0):
    """A bmlp_config plus the widths array it points to (keep both alive)."""
    arr = (ctypes.c_int32 * len(widths))(*[int(w) for w in widths])
    cfg = bmlp_config(len(widths) - 1, arr, n_classes, max_batch, bound, group_size,
                      float(robustness), int(seed) & (2**64 - 1), fwd_impl, int(variants))
    cfg._widths_keepalive = arr
    return cfg


def _check(st: int, where: str):
    if st != BMLP_OK:
        raise BmlpError(st, where)


def status_string(st: int) -> str:
    return lib().bmlp_status_string(st).decode()


def last_error() -> str:
    return lib().bmlp_last_error().decode()


def bmlp_state_bytes(cfg) -> int:
    return lib().bmlp_state_bytes(ctypes.byref(cfg))


def bmlp_workspace_bytes(cfg) -> int:
    return lib().bmlp_workspace_bytes(ctypes.byref(cfg))


def bmlp_describe(cfg, layer: int) -> bmlp_layer_info:
    info = bmlp_layer_info()
    _check(lib().bmlp_describe(ctypes.byref(cfg), layer, ctypes.byref(info)), "bmlp_describe")
    return info


def bmlp_reinforce_threshold(p_r: float, k: int) -> int:
    return lib().bmlp_reinforce_threshold(p_r, k)


def bmlp_init(cfg, d_state: int, d_ws: int, stream: int) -> int:
    ctx = ctypes.c_void_p()
    _check(lib().bmlp_init(ctypes.byref(cfg), d_state, d_ws, stream, ctypes.byref(ctx)), "bmlp_init")
    return ctx.value


def bmlp_attach(cfg, d_state: int, d_ws: int, stream: int) -> int:
    ctx = ctypes.c_void_p()
    _check(lib().bmlp_attach(ctypes.byref(cfg), d_state, d_ws, stream, ctypes.byref(ctx)),
           "bmlp_attach")
    return ctx.value


def bmlp_pack(d_pm1: int, n: int, K: int, d_bits: int, stream: int):
    _check(lib().bmlp_pack(d_pm1, n, K, d_bits, stream), "bmlp_pack")


def bmlp_forward(ctx: int, d_x: int, n: int, d_yhat: int, stream: int):
    _check(lib().bmlp_forward(ctx, d_x, n, d_yhat, stream), "bmlp_forward")


def bmlp_forward_noalloc(ctx: int, d_x: int, n: int, d_yhat: int, stream: int):
    _check(lib().bmlp_forward_noalloc(ctx, d_x, n, d_yhat, stream), "bmlp_forward_noalloc")


def bmlp_train_step(ctx: int, d_x: int, d_y: int, n: int, step: int, p_r: float, d_stats: int,
                    stream: int):
    _check(lib().bmlp_train_step(ctx, d_x, d_y, n, step, p_r, d_stats, stream), "bmlp_train_step")


def bmlp_eval(ctx: int, d_x: int, d_y: int, n: int, d_correct: int, stream: int):
    _check(lib().bmlp_eval(ctx, d_x, d_y, n, d_correct, stream), "bmlp_eval")


def bmlp_feature_median(d_x: int, n: int, K: int, d_median: int, stream: int):
    _check(lib().bmlp_feature_median(d_x, n, K, d_median, stream), "bmlp_feature_median")


def bmlp_binarize(d_x: int, n: int, K: int, d_median: int, d_bits: int, stream: int):
    _check(lib().bmlp_binarize(d_x, n, K, d_median, d_bits, stream), "bmlp_binarize")


def bmlp_expand(d_x: int, n: int, k_raw: int, k0: int, seed: int, d_bits: int, stream: int):
    _check(lib().bmlp_expand(d_x, n, k_raw, k0, seed & (2**64 - 1), d_bits, stream), "bmlp_expand")


def feature_median(x_int8):
    """Per-feature lower median of int8 rows [n][K] (a CUDA tensor), int8 [K]."""
    import torch
    n, K = x_int8.shape
    out = torch.empty(K, dtype=torch.int8, device=x_int8.device)
    bmlp_feature_median(x_int8.data_ptr(), n, K, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    return out


def binarize(x_int8, median):
    """Median binarisation of int8 rows [n][K] to bit rows int64 [n][ceil(K/64)]."""
    import torch
    n, K = x_int8.shape
    out = torch.empty((n, words64(K)), dtype=torch.int64, device=x_int8.device)
    bmlp_binarize(x_int8.data_ptr(), n, K, median.data_ptr(), out.data_ptr(),
                  torch.cuda.current_stream().cuda_stream)
    return out


def expand(x_int8, k0: int, seed: int):
    """The fixed random ±1 expansion layer: int8 rows [n][K_raw] to bit rows
    int64 [n][ceil(k0/64)]."""
    import torch
    n, k_raw = x_int8.shape
    out = torch.empty((n, words64(k0)), dtype=torch.int64, device=x_int8.device)
    bmlp_expand(x_int8.data_ptr(), n, k_raw, k0, int(seed), out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    return out


def bmlp_eval_exit(ctx: int, d_x: int, d_y: int, n: int, d_counts: int, stream: int):
    _check(lib().bmlp_eval_exit(ctx, d_x, d_y, n, d_counts, stream), "bmlp_eval_exit")


def bmlp_train_epoch(ctx: int, d_x_all: int, d_y_all: int, n_all: int, d_order: int, n_order: int,
                     batch: int, step0: int, p_r: float, d_stats: int, stream: int):
    _check(lib().bmlp_train_epoch(ctx, d_x_all, d_y_all, n_all, d_order, n_order, batch, step0, p_r,
                                  d_stats, stream), "bmlp_train_epoch")


def bmlp_epoch_rescale(p_r: float, wrong: int, samples: int) -> float:
    return lib().bmlp_epoch_rescale(p_r, wrong, samples)


def bmlp_epoch_summary(h_stats: int, steps: int, n_layers: int, batch: int, p_r: float):
    """(E^e, p_r for the next epoch) from a host copy of an epoch's stats."""
    e, nxt = ctypes.c_double(), ctypes.c_double()
    _check(lib().bmlp_epoch_summary(h_stats, steps, n_layers, batch, p_r, ctypes.byref(e), ctypes.byref(nxt)),
           "bmlp_epoch_summary")
    return e.value, nxt.value


def bmlp_read_h(ctx: int, layer: int, d_out: int, stream: int):
    _check(lib().bmlp_read_h(ctx, layer, d_out, stream), "bmlp_read_h")


def bmlp_destroy(ctx: int):
    lib().bmlp_destroy(ctx)


STATS_STRIDE = 32   # BMLP_STATS_STRIDE: int32 entries per layer row of the step statistics
KERNEL_KINDS = ("fwd", "cls", "select", "update", "other")


def bmlp_profile_start(ctx: int, max_launches: int):
    _check(lib().bmlp_profile_start(ctx, max_launches), "bmlp_profile_start")


def bmlp_profile_stop(ctx: int):
    """{kind: (total_ms, launches)} of the launches timed since start."""
    ms = (ctypes.c_double * len(KERNEL_KINDS))()
    cnt = (ctypes.c_int64 * len(KERNEL_KINDS))()
    _check(lib().bmlp_profile_stop(ctx, ms, cnt), "bmlp_profile_stop")
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNEL_KINDS)}


# ---------------------------------------------------------------------------
# torch-facing wrapper
# ---------------------------------------------------------------------------

def words64(k: int) -> int:
    return (k + 63) // 64


class BMLP:
    """A network whose state and workspace live in torch-owned GPU buffers.

    Inputs are bit rows (int64 tensors [n][ceil(K_0/64)], see ``pack``) and
    int32 labels; all calls run on the current torch stream.
    """

    def __init__(self, widths: Sequence[int], n_classes: int, bound: int, max_batch: int,
                 group_size: int = 64, robustness: float = 0.25, seed: int = 0,
                 fwd_impl: int = BMLP_FWD_AUTO, device="cuda", state=None, variants: int = 0):
        import torch
        self.torch = torch
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.widths = tuple(int(w) for w in widths)
        self.n_layers = len(self.widths) - 1
        self.n_classes = int(n_classes)
        self.max_batch = int(max_batch)
        self.cfg = make_config(self.widths, n_classes, bound, max_batch, group_size, robustness,
                               seed, fwd_impl, variants)
        sb, wb = bmlp_state_bytes(self.cfg), bmlp_workspace_bytes(self.cfg)
        if sb == 0 or wb == 0:
            raise BmlpError(BMLP_ESHAPE, "configuration")
        self.info = [bmlp_describe(self.cfg, l) for l in range(1, self.n_layers + 1)]
        if state is None:
            self.state = torch.empty(sb, dtype=torch.uint8, device=self.device)
        else:
            if state.numel() != sb or state.dtype != torch.uint8:
                raise ValueError("state buffer does not match the configuration")
            self.state = state.to(self.device).contiguous().clone()
        self.ws = torch.empty(wb, dtype=torch.uint8, device=self.device)
        fn = bmlp_attach if state is not None else bmlp_init
        self.ctx = fn(self.cfg, self.state.data_ptr(), self.ws.data_ptr(), self._stream())

    def __del__(self):
        ctx = getattr(self, "ctx", None)
        if ctx:
            bmlp_destroy(ctx)
            self.ctx = None

    def _stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    # ---- inputs -------------------------------------------------------------
    def pack(self, x_pm1):
        """int8 ±1 tensor [n][K] (on the GPU) -> int64 bit rows [n][ceil(K/64)]."""
        torch = self.torch
        x = x_pm1.to(self.device, torch.int8).contiguous()
        n, K = x.shape
        out = torch.empty((n, words64(K)), dtype=torch.int64, device=self.device)
        bmlp_pack(x.data_ptr(), n, K, out.data_ptr(), self._stream())
        return out

    def _batch(self, x_bits, y=None):
        torch = self.torch
        if x_bits.dtype != torch.int64 or x_bits.device != self.device or not x_bits.is_contiguous():
            raise ValueError("x must be a contiguous int64 bit-row tensor on the library's device")
        if x_bits.dim() != 2 or x_bits.shape[1] != words64(self.widths[0]):
            raise ValueError("x has the wrong number of words per row")
        if y is not None and (y.dtype != torch.int32 or y.device != self.device
                              or not y.is_contiguous() or y.shape[0] != x_bits.shape[0]):
            raise ValueError("y must be a contiguous int32 tensor of n labels on the device")
        return x_bits.shape[0]

    # ---- the method -----------------------------------------------------------
    def train_step(self, x_bits, y, step: int, p_r: float, stats=None):
        """One mini-batch; returns int32 stats [L][4] (err, |M|, |U|, reinforced).

        ``stats``, if given, is an int32 tensor [L][BMLP_STATS_STRIDE] that the
        library fills (each layer's counts in a 128-byte row of their own)."""
        n = self._batch(x_bits, y)
        if stats is None:
            stats = self.torch.empty((self.n_layers, STATS_STRIDE), dtype=self.torch.int32, device=self.device)
        if tuple(stats.shape) != (self.n_layers, STATS_STRIDE) or stats.dtype != self.torch.int32 \
                or not stats.is_contiguous():
            raise ValueError(f"stats must be a contiguous int32 tensor [{self.n_layers}][{STATS_STRIDE}]")
        bmlp_train_step(self.ctx, x_bits.data_ptr(), y.data_ptr(), n, int(step), float(p_r),
                        stats.data_ptr(), self._stream())
        return stats[:, :4]

    def train_epoch(self, x_bits_all, y_all, order, step0: int, p_r: float, batch: Optional[int] = None):
        """One epoch (Algorithm 1's epoch loop) over the full batches of ``order``
        (int32 training-set indices) taken from the device-resident training set
        ``x_bits_all`` (int64 bit rows [N][ceil(K_0/64)]), ``y_all`` (int32 [N]),
        with steps step0, step0 + 1, ....  Returns (p_r for the next epoch,
        E^e, int32 stats [batches][L][4]); E^e and the rescale need the
        epoch's counts, so this waits for the stream."""
        batch = self.max_batch if batch is None else int(batch)
        t = self.torch
        if x_bits_all.dim() != 2 or x_bits_all.shape[1] != words64(self.widths[0]) \
                or x_bits_all.dtype != t.int64 or not x_bits_all.is_contiguous():
            raise ValueError("x_bits_all must be contiguous int64 [N][ceil(K_0/64)]")
        if y_all.dtype != t.int32 or y_all.shape != (x_bits_all.shape[0],) or not y_all.is_contiguous():
            raise ValueError("y_all must be contiguous int32 [N]")
        if order.dtype != t.int32 or order.dim() != 1 or not order.is_contiguous():
            raise ValueError("order must be contiguous int32 [n_order]")
        nb = order.shape[0] // batch
        stats = t.zeros((max(nb, 1), self.n_layers, STATS_STRIDE), dtype=t.int32, device=self.device)
        bmlp_train_epoch(self.ctx, x_bits_all.data_ptr(), y_all.data_ptr(), x_bits_all.shape[0],
                         order.data_ptr(), order.shape[0], batch, int(step0), float(p_r), stats.data_ptr(),
                         self._stream())
        host = stats.cpu()   # waits for the stream
        e, p_next = bmlp_epoch_summary(host.data_ptr(), nb, self.n_layers, batch, float(p_r))
        return p_next, e, host[:nb, :, :4]

    def eval_exit(self, x_bits, y, counts=None):
        """Adds per layer [correct, exits, correct exits] of this batch to
        ``counts`` (int32 [L][3]); see bmlp_eval_exit for the exit rule."""
        n = self._batch(x_bits, y)
        if counts is None:
            counts = self.torch.zeros((self.n_layers, 3), dtype=self.torch.int32, device=self.device)
        bmlp_eval_exit(self.ctx, x_bits.data_ptr(), y.data_ptr(), n, counts.data_ptr(), self._stream())
        return counts

    def forward(self, x_bits):
        """Local outputs y_hat of every layer, int32 [L][n][c]."""
        n = self._batch(x_bits)
        out = self.torch.empty((self.n_layers, n, self.n_classes), dtype=self.torch.int32,
                               device=self.device)
        bmlp_forward(self.ctx, x_bits.data_ptr(), n, out.data_ptr(), self._stream())
        return out

    def eval(self, x_bits, y, correct=None):
        """Adds per-layer correct counts of this batch to ``correct`` (int32 [L])."""
        n = self._batch(x_bits, y)
        if correct is None:
            correct = self.torch.zeros(self.n_layers, dtype=self.torch.int32, device=self.device)
        bmlp_eval(self.ctx, x_bits.data_ptr(), y.data_ptr(), n, correct.data_ptr(), self._stream())
        return correct

    # ---- views ----------------------------------------------------------------
    def _view(self, buf, off: int, nbytes: int, dtype, shape):
        return buf[off:off + nbytes].view(dtype).view(*shape)

    def H(self, l: int):
        """Hidden weights of layer l unpacked to int8 [K_l][K_{l-1}] (a new tensor;
        the state keeps them bit-sliced, see H_planes)."""
        i = self.info[l - 1]
        out = self.torch.empty((i.k_out, i.k_in), dtype=self.torch.int8, device=self.device)
        bmlp_read_h(self.ctx, l, out.data_ptr(), self._stream())
        return out

    def H_planes(self, l: int):
        """The state's bit-sliced hidden weights of layer l, uint8 [K_l][ld_h]."""
        i = self.info[l - 1]
        return self._view(self.state, i.off_h, i.k_out * i.ld_h, self.torch.uint8, (i.k_out, i.ld_h))

    def W(self, l: int):
        i = self.info[l - 1]
        return self._view(self.state, i.off_w, i.k_out * i.words_in * 8, self.torch.int64,
                          (i.k_out, i.words_in))

    def P(self, l: int):
        i = self.info[l - 1]
        return self._view(self.state, i.off_p, self.n_classes * i.words_out * 8, self.torch.int64,
                          (self.n_classes, i.words_out))

    def trace(self, l: int, n: int):
        """Last train step's a_l bits, err, upd and kstar of layer l (first n patterns)."""
        i = self.info[l - 1]
        t = self.torch
        return {
            "a": self._view(self.ws, i.off_a, n * i.words_out * 8, t.int64, (n, i.words_out)),
            "err": self._view(self.ws, i.off_err, n, t.uint8, (n,)),
            "upd": self._view(self.ws, i.off_upd, n, t.uint8, (n,)),
            # stored group-major [groups][max_batch]; returned as [n][groups]
            "kstar": self._view(self.ws, i.off_kstar, self.max_batch * i.groups * 2, t.int16,
                                (i.groups, self.max_batch))[:, :n].t(),
        }
