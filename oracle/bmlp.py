"""Plain CPU oracle of the fully binary BMLP training step.

TEST INFRASTRUCTURE ONLY.  The oracle exists to check the GPU library.  Only
the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never does.  It shares no code with the GPU path.

It follows the paper (Colombo, Pittorino, Roveri, "Training multi-layer binary
neural networks with random local binary error signals", arXiv 2412.00119)
step by step, on dense ±1 integer arrays, with no bit packing:

* Algorithm 1 (network level, Section 3.2): forward z = a W^T, a = sign(z),
  local output y_hat = a P^T, 01-loss (Eq. 1), top-two margin tau and the set
  M of patterns to update.
* Algorithm 2 (layer level, Section 3.3): stabilities delta = z * rho^y, and in
  each group of gamma perceptrons the "easiest" wrong one, the largest
  negative delta.
* Algorithm 3 (perceptron level, Section 3.4): Clipped-Perceptron increments
  h += 2 a rho, then reinforcement h += 2 sign(h) with probability
  p_r * sqrt(2 / (pi K_l)).

Readings where the paper is silent (each is listed with its reason in the
project's design notes):
  R1  sign(0) = +1 for activations (z >= 0 gives +1).
  R2  argmax ties resolve to the lowest class index.
  R3  tau is the difference of the two largest values of y_hat, so a tie
      at the top gives tau = 0.
  R4  tau < r*K_l is evaluated as tau < ceil(r*K_l) (tau is an integer).
  R5  k* ties resolve to the lowest index; delta = 0 is not eligible.
  R6  groups are contiguous blocks of gamma perceptrons, fixed for the run.
  R7  gamma*: the divisor of K_l closest to [75, 105]; ties take the largest.
  R8  the Clipped-Perceptron increments of a batch are summed, then clipped
      once to [-B, B]; reinforcement follows, then a second clip.
  R9  H and P start uniform on {-1, +1}; B is odd, so h stays odd.
  R10 reinforcement runs once per step on every hidden weight of a layer,
      only when M_l is not empty, after the CP increments.
  R11 the K in the reinforcement probability is K_l, as printed (the
      fan_in_reinforce variant uses K_{l-1}).
  R12 Uniform(0,1) is a 32-bit draw u, and "p < q" is u < ceil(q * 2^32).
  R13 all layers use the weights from before the step (the forward of layer
      l+1 reads a_l, which the update of layer l does not change).
  R14 labels are 0-based.
  R15 (the bound B = 127 of workloads that give none belongs to the
      workload definitions, not to this module.)
  R16 the epoch loop (Algorithm 1) runs over the full mini-batches of a
      given order of the training set; E^e is the fraction of those
      samples whose last-layer local classifier was wrong during the epoch
      (its 01-loss, counted as each batch is trained on), and p_r becomes
      p_r * sqrt(E^e) after the epoch; an epoch with no full batch leaves
      p_r unchanged.
  R17 early exit (Section 3.1 names the strategy, not a rule): a pattern
      exits at the first layer whose local classifier has a margin tau of
      at least ceil(r * K_l), the training-time robustness test, and at the
      last layer otherwise; its prediction is that layer's.
  R18 median binarisation (Algorithm 1, its input step): each input feature is
      compared with its median over a reference set of integer samples,
      the lower middle order statistic (index floor((N-1)/2) of the sorted
      column); +1 where x >= median.
  R19 the expansion layer for integer inputs (Section 3.2, footnote 1):
      a_0 = sign(x R^T) with R = ±1 [K_0][K_raw] fixed, exact integer sums,
      sign(0) = +1; R from Philox stream 5 with layer word 2^32 - 1 and
      t = 0, element j*K_raw + i at bit (e & 127) of block e >> 7.
  R20 group reshuffle (Section 4.3 varies group membership without giving
      the draw): at step t layer l orders its perceptrons by the 32-bit
      key word (k & 3) of Philox block k >> 2, stream 6, ties by index, and
      group g is positions g*gamma .. g*gamma + gamma - 1 of that order;
      k* is stored as the position within the group, and equal deltas go
      to the lowest perceptron index, as with fixed groups.
  R21 sequential clipping (the alternative to R8): the selected pairs of
      the batch are applied in pattern order, each increment clipped to
      [-B, B] at once; reinforcement and its clip follow as in R8.

Parity unpinned: the paper does not fix readings R1, R2, R5 (its tie
rule), R11, R17, R18, R19, R20, R21 or the Philox stream layout below, so
nothing outside this code decides them; the arithmetic of each is still
pinned by the tests (brute force, hand-computed cases, direct Philox calls).

Random numbers come from Philox4x32-10 (``oracle.philox``) keyed by the
64-bit seed (k0 = low word, k1 = high word), with counter
(block, l-1, t mod 2^32, stream):
  stream 1  H init: bit (j & 127) of the 128 output bits of block j >> 7,
            j = k*K_{l-1} + i (word b >> 5, bit b & 31 with b = j & 127).
  stream 2  P init: same, j = class*K_l + k.
  stream 3  reinforcement, coarse byte of hidden weight (k, i): with
            q = k * ceil(K_{l-1} / 32) + (i >> 5) (the row's 32-column group),
            bit p of u8 is bit (i & 31) of word p & 3 of block 2q + (p >> 2).
  stream 4  reinforcement, fine bits: u24 = low 24 bits of word (j & 3) of
            block j >> 2, j = k * K_{l-1} + i.
  stream 5  expansion layer (R19).
  stream 6  group order (R20): key of perceptron k is word (k & 3) of
            block k >> 2.
  The 32-bit draw of hidden weight (k, i) is u = u8 * 2^24 + u24; it
  reinforces when u < T_l.  Init uses t = 0.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from .philox import MASK32, philox4x32_10

STREAM_H_INIT = 1
STREAM_P_INIT = 2
STREAM_R_COARSE = 3
STREAM_R_FINE = 4
STREAM_EXPAND = 5     # the fixed random input expansion layer (counter layer word 2^32 - 1)
STREAM_GROUPS = 6     # per-step group membership (reshuffle variant)

GAMMA_RANGE = (75, 105)   # the paper's empirical optimum range (Section 4.3)
TWO32 = 1 << 32


# ---------------------------------------------------------------------------
# Host scalars
# ---------------------------------------------------------------------------

def gamma_star(k: int, lo: int = GAMMA_RANGE[0], hi: int = GAMMA_RANGE[1]) -> int:
    """Group size rule of Section 4.3: the divisor of k closest to any value
    of [lo, hi]; among equally close divisors take the largest (R7)."""
    best, best_d = None, None
    for g in range(1, k + 1):
        if k % g:
            continue
        d = 0 if lo <= g <= hi else min(abs(g - lo), abs(g - hi))
        if best is None or d < best_d or (d == best_d and g > best):
            best, best_d = g, d
    return best


def robustness_threshold(r: float, k: int) -> int:
    """Integer form of the robustness test tau < r*K_l (R4): ceil(r*K_l)."""
    return int(math.ceil(float(r) * float(k)))


def reinforce_probability(p_r: float, k: int) -> float:
    """p_r * sqrt(2 / (pi * K_l)) (Algorithm 3), in IEEE double in this order."""
    return float(p_r) * math.sqrt(2.0 / (math.pi * float(k)))


def reinforce_threshold(p_r: float, k: int) -> int:
    """T_l = ceil(q * 2^32), at most 2^32 (R12)."""
    q = reinforce_probability(p_r, k)
    t = math.ceil(q * 4294967296.0)
    return int(min(max(t, 0), TWO32))


# ---------------------------------------------------------------------------
# Random streams
# ---------------------------------------------------------------------------

def philox_key(seed: int):
    return seed & MASK32, (seed >> 32) & MASK32


def _blocks(seed: int, layer: int, t: int, stream: int, blocks: np.ndarray):
    """Philox words [m][4] for the distinct blocks, and each block's row."""
    k0, k1 = philox_key(seed)
    if blocks.size == 0:
        return np.zeros((0, 4), np.uint32), np.zeros(0, np.int64)
    lo, hi = int(blocks.min()), int(blocks.max())
    if hi - lo + 1 <= 4 * blocks.size:
        ub = np.arange(lo, hi + 1, dtype=np.uint64)
        inv = (blocks - np.uint64(lo)).astype(np.int64)
    else:
        ub, inv = np.unique(blocks, return_inverse=True)
    words = np.stack(philox4x32_10(ub, layer - 1, t & MASK32, stream, k0, k1), axis=-1)
    return words, inv


def stream_bits(seed: int, layer: int, stream: int, j: np.ndarray, t: int = 0) -> np.ndarray:
    """Bit (j & 127) of the 128-bit Philox block j >> 7 (streams 1 and 2)."""
    j = np.asarray(j, dtype=np.uint64)
    words, inv = _blocks(seed, layer, t, stream, j >> np.uint64(7))
    b = (j & np.uint64(127)).astype(np.int64)
    w = words[inv, b >> 5]
    return ((w >> (b & 31).astype(np.uint32)) & np.uint32(1)).astype(np.uint8)


def stream_bits_prefix(seed: int, layer: int, stream: int, n: int, t: int = 0) -> np.ndarray:
    """stream_bits for j = 0..n-1, written as the layout itself: the 128
    output bits of block q (four words, each LSB first) are elements
    128q .. 128q+127."""
    k0, k1 = philox_key(seed)
    nb = (int(n) + 127) // 128
    words = np.stack(philox4x32_10(np.arange(nb, dtype=np.uint64), layer - 1, t & MASK32, stream, k0, k1),
                     axis=-1).astype("<u4")
    return np.unpackbits(words.view(np.uint8).reshape(-1), bitorder="little")[:n]


def reinforce_draws(seed: int, layer: int, t: int, j: np.ndarray, k_in: int) -> np.ndarray:
    """The 32-bit uniform draw u = u8 * 2^24 + u24 of each flat index
    j = k * K_{l-1} + i of a layer with K_{l-1} = k_in inputs."""
    j = np.asarray(j, dtype=np.uint64)
    kin = np.uint64(k_in)
    k, i = j // kin, j % kin
    # coarse byte: stream 3, eight words (two blocks) per 32-column group,
    # word p giving bit p of the 32 bytes
    q = k * np.uint64((k_in + 31) // 32) + (i >> np.uint64(5))
    b2 = q * np.uint64(2)
    words, inv = _blocks(seed, layer, t, STREAM_R_COARSE, np.concatenate([b2, b2 + np.uint64(1)]))
    m = j.size
    planes = np.concatenate([words[inv[:m]], words[inv[m:]]], axis=1)   # [len(j)][8]
    bit = (i & np.uint64(31)).astype(np.uint32)
    u8 = np.zeros(j.shape, dtype=np.uint32)
    for p in range(8):
        u8 |= ((planes[:, p] >> bit) & np.uint32(1)) << np.uint32(p)
    # fine bits: stream 4, four 24-bit values per block
    fw, inv = _blocks(seed, layer, t, STREAM_R_FINE, j >> np.uint64(2))
    u24 = fw[inv, (j & np.uint64(3)).astype(np.int64)] & np.uint32(0xFFFFFF)
    return (u8.astype(np.uint64) << np.uint64(24)) | u24.astype(np.uint64)


def reinforce_mask(seed: int, layer: int, t: int, thresh: int, n: int, k_in: int,
                   chunk: int = 1 << 22) -> np.ndarray:
    """Bernoulli(T / 2^32) draws for flat indices 0..n-1 of a layer with
    K_{l-1} = k_in: u < T (R12)."""
    out = np.empty(n, dtype=bool)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        u = reinforce_draws(seed, layer, t, np.arange(s, e, dtype=np.uint64), k_in)
        out[s:e] = u < np.uint64(thresh)
    return out


# ---------------------------------------------------------------------------
# Model state
# ---------------------------------------------------------------------------

@dataclass
class Config:
    widths: Sequence[int]          # K_0..K_L
    n_classes: int
    bound: int                      # B, odd
    group_size: int = 64            # gamma; 0 = gamma* per layer
    robustness: float = 0.25
    seed: int = 0
    # method variants (each off by default)
    fan_in_reinforce: bool = False   # K_{l-1} instead of K_l in the reinforcement probability
    shared_classifier: bool = False  # one P for every layer (all K_l equal, Section 3.1)
    saturate_z: bool = False         # z held in min(8, ceil(log2(2 K_{l-1}))) bits (Section 3.5)
    reshuffle_groups: bool = False   # random group membership every step (Section 4.3)
    sequential_clip: bool = False    # the increments applied pattern by pattern, each clipped (R21)

    def __post_init__(self):
        self.widths = tuple(int(v) for v in self.widths)
        if len(self.widths) < 2 or min(self.widths) < 1:
            raise ValueError("need K_0..K_L with L >= 1 and every K >= 1")
        if self.n_classes < 2:
            raise ValueError("need at least two classes")
        if self.bound < 1 or self.bound % 2 == 0 or self.bound > 127:
            raise ValueError("B must be odd, 1..127")
        for k in self.widths[1:]:
            if self.gamma(k) < 1 or k % self.gamma(k):
                raise ValueError(f"group size must divide K_l={k}")
        if self.shared_classifier and len(set(self.widths[1:])) != 1:
            raise ValueError("a shared classifier needs every K_l equal")

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    def gamma(self, k: int) -> int:
        return self.group_size if self.group_size > 0 else gamma_star(k)


@dataclass
class State:
    cfg: Config
    H: List[np.ndarray]             # int8 [K_l][K_{l-1}] per layer
    P: List[np.ndarray]             # int8 ±1 [c][K_l] per layer

    def W(self, l: int) -> np.ndarray:
        """Visible weights W_l = sign(H_l); h is odd, so never 0."""
        return np.where(self.H[l - 1] > 0, 1, -1).astype(np.int8)

    def copy(self) -> "State":
        return State(self.cfg, [h.copy() for h in self.H], [p.copy() for p in self.P])


def init_layer(cfg: Config, l: int):
    """H_l and P_l uniform on {-1, +1} (Algorithm 1, initialisation; R9)."""
    kin, kout, c = cfg.widths[l - 1], cfg.widths[l], cfg.n_classes
    hb = stream_bits_prefix(cfg.seed, l, STREAM_H_INIT, kin * kout)
    pb = stream_bits_prefix(cfg.seed, l, STREAM_P_INIT, c * kout)
    H = np.where(hb == 1, 1, -1).astype(np.int8).reshape(kout, kin)
    P = np.where(pb == 1, 1, -1).astype(np.int8).reshape(c, kout)
    return H, P


def init(cfg: Config) -> State:
    """Every layer's H_l and P_l; with a shared classifier every layer uses
    layer 1's P (Section 3.1)."""
    Hs, Ps = [], []
    for l in range(1, cfg.n_layers + 1):
        H, P = init_layer(cfg, l)
        Hs.append(H)
        Ps.append(Ps[0] if cfg.shared_classifier and l > 1 else P)
    return State(cfg, Hs, Ps)


# ---------------------------------------------------------------------------
# The step, one paper operation per function
# ---------------------------------------------------------------------------

def int_matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Integer matrix product a @ b via float64 BLAS.  Exact here: every
    operand is in {-1, 0, +1} (or a small integer) and every partial sum is
    far below 2^53."""
    return np.rint(np.asarray(a, np.float64) @ np.asarray(b, np.float64)).astype(np.int64)


def preactivation(a_prev: np.ndarray, W: np.ndarray) -> np.ndarray:
    """z_l = a_{l-1} sign(H_l) (Algorithm 1); W stored [K_l][K_{l-1}]."""
    return int_matmul(a_prev, W.T)


def activation(z: np.ndarray) -> np.ndarray:
    """a_l = sign(z_l), with sign(0) = +1 (R1)."""
    return np.where(z >= 0, 1, -1).astype(np.int8)


def local_output(a: np.ndarray, P: np.ndarray) -> np.ndarray:
    """y_hat_l = a_l P_l (Algorithm 1); P stored [c][K_l]."""
    return int_matmul(a, P.T)


def local_error(yhat: np.ndarray, y: np.ndarray, thr: int):
    """01-loss (Eq. 1), margin tau and the update mask M (Algorithm 1).

    pred is the first index of the maximum (R2); tau is the largest minus the
    second largest value (R3); M = (loss = 1) or (tau < thr) (R4).
    """
    pred = np.argmax(yhat, axis=1)
    srt = -np.sort(-yhat, axis=1)
    tau = srt[:, 0] - srt[:, 1]
    err = pred != y
    upd = err | (tau < thr)
    return pred, tau, err, upd


def feature_median(x: np.ndarray) -> np.ndarray:
    """Per-feature median of integer samples x [N][K] (R18): the order
    statistic floor((N-1)/2) of each column."""
    x = np.asarray(x)
    return np.sort(x, axis=0)[(len(x) - 1) // 2]


def median_binarize(x: np.ndarray, median: np.ndarray) -> np.ndarray:
    """Algorithm 1's input binarisation (R18): +1 where a feature is at or above its median."""
    return np.where(np.asarray(x) >= np.asarray(median)[None, :], 1, -1).astype(np.int8)


def expansion_matrix(seed: int, k_raw: int, k0: int) -> np.ndarray:
    """The fixed ±1 expansion weights R [K_0][K_raw] (R19)."""
    k0s, k1s = philox_key(seed)
    n = k_raw * k0
    nb = (n + 127) // 128
    words = np.stack(philox4x32_10(np.arange(nb, dtype=np.uint64), MASK32, 0, STREAM_EXPAND, k0s, k1s),
                     axis=-1).astype("<u4")
    bits = np.unpackbits(words.view(np.uint8).reshape(-1), bitorder="little")[:n]
    return np.where(bits == 1, 1, -1).astype(np.int8).reshape(k0, k_raw)


def expand(x: np.ndarray, R: np.ndarray) -> np.ndarray:
    """Input layer for integer inputs (R19): a_0 = sign(x R^T), sign(0) = +1."""
    return activation(int_matmul(np.asarray(x, dtype=np.int64), R.T))


def z_bits(k_in: int) -> int:
    """min(8, ceil(log2(2 K_{l-1}))) bits for z (Section 3.5)."""
    return min(8, (2 * k_in - 1).bit_length())


def saturate(z: np.ndarray, k_in: int) -> np.ndarray:
    """z held in z_bits(K_{l-1}) two's-complement bits: clipped to
    [-2^(b-1), 2^(b-1) - 1].  Its sign is that of z, so a_l is unchanged;
    only the selection of Algorithm 2 sees the clipped magnitudes."""
    b = z_bits(k_in)
    return np.clip(z, -(1 << (b - 1)), (1 << (b - 1)) - 1)


def group_permutation(seed: int, layer: int, t: int, k: int) -> np.ndarray:
    """The reshuffle variant's group order at step t: perceptrons sorted by
    a 32-bit Philox key (word k & 3 of block k >> 2 of stream 6, counter
    (block, l-1, t, 6)), ties by index; group g holds positions
    g*gamma .. g*gamma + gamma - 1 of this order."""
    idx = np.arange(k)
    words, _ = _blocks(seed, layer, t, STREAM_GROUPS, np.arange((k + 3) // 4, dtype=np.uint64))
    return np.lexsort((idx, words[idx >> 2, idx & 3]))


def select_easiest(z: np.ndarray, P: np.ndarray, y: np.ndarray, upd: np.ndarray, gamma: int,
                   perm: Optional[np.ndarray] = None) -> np.ndarray:
    """Algorithm 2: for each pattern in M and each group of gamma perceptrons
    (contiguous, or positions of ``perm`` in the reshuffle variant), the
    offset within the group of the largest negative stability
    delta = z * rho^{y}; -1 where the pattern is not in M or the group has
    no negative stability.  Ties take the lowest perceptron index (R5, R6)."""
    n, k = z.shape
    g = k // gamma
    rho = P[y].astype(np.int64)                     # [n][K_l], rho^{y^mu}
    order = np.arange(k) if perm is None else np.asarray(perm, dtype=np.int64)
    delta = (z * rho)[:, order].reshape(n, g, gamma)
    neg = delta < 0
    # the largest delta, then the lowest perceptron index (0 <= index < K_l)
    comp = delta * k - order.reshape(1, g, gamma)
    key = np.where(neg, comp, np.iinfo(np.int64).min)
    kstar = np.argmax(key, axis=2)
    ok = neg.any(axis=2) & upd[:, None]
    return np.where(ok, kstar, -1).astype(np.int16)


def selection_matrix(kstar: np.ndarray, P: np.ndarray, y: np.ndarray, gamma: int,
                     perm: Optional[np.ndarray] = None) -> np.ndarray:
    """S[mu][k] = rho^{y^mu, k} for every selected pair (mu, k) of U_l, else 0."""
    n, g = kstar.shape
    S = np.zeros((n, g * gamma), dtype=np.int8)
    mu, grp = np.nonzero(kstar >= 0)
    pos = grp * gamma + kstar[mu, grp].astype(np.int64)
    k = pos if perm is None else np.asarray(perm, dtype=np.int64)[pos]
    S[mu, k] = P[y[mu], k]
    return S


def cp_increment(S: np.ndarray, a_prev: np.ndarray) -> np.ndarray:
    """Sum over U_l of the Clipped-Perceptron increments 2 a^mu rho (Algorithm 3):
    dH = 2 S^T a_{l-1}, shape [K_l][K_{l-1}]."""
    return 2 * int_matmul(S.T, a_prev)


def clip(h: np.ndarray, bound: int) -> np.ndarray:
    return np.clip(h, -bound, bound)


def cp_sequential(H: np.ndarray, S: np.ndarray, a_prev: np.ndarray, bound: int) -> np.ndarray:
    """The sequential reading of Algorithm 3's increment (R21): pattern by
    pattern in index order, each selected row gets 2 a^mu rho and is
    clipped to [-B, B] at once.  Rows selected by one pattern are distinct."""
    h = H.astype(np.int64).copy()
    for mu in range(S.shape[0]):
        ks = np.nonzero(S[mu])[0]
        if ks.size:
            inc = 2 * S[mu, ks].astype(np.int64)[:, None] * a_prev[mu].astype(np.int64)[None, :]
            h[ks] = clip(h[ks] + inc, bound)
    return h


def reinforce(h: np.ndarray, mask: np.ndarray, bound: int) -> np.ndarray:
    """h += 2 sign(h) where the draw fired (Algorithm 3), then clip (R8)."""
    return clip(h + 2 * np.sign(h) * mask.reshape(h.shape), bound)


@dataclass
class LayerTrace:
    a: np.ndarray         # int8 ±1 [n][K_l]
    z: np.ndarray         # int64 [n][K_l], as Algorithm 2 sees it (saturated with saturate_z)
    yhat: np.ndarray      # int64 [n][c]
    pred: np.ndarray
    tau: np.ndarray
    err: np.ndarray       # bool [n]
    upd: np.ndarray       # bool [n]
    kstar: np.ndarray     # int16 [n][G]
    stats: np.ndarray     # int64 [4]: sum(err), |M|, |U|, reinforced draws
    perm: Optional[np.ndarray] = None   # the step's group order (reshuffle variant)


def train_step(state: State, x: np.ndarray, y: np.ndarray, t: int, p_r: float,
               layers: Optional[Sequence[int]] = None) -> List[LayerTrace]:
    """One mini-batch of Algorithm 1, updating ``state`` in place.

    x is int8 ±1 [n][K_0] (already binarised), y int [n] in [0, c).
    ``layers`` restricts the update to some layers (all by default); the
    forward always runs through every layer up to the last requested one.
    Returns one trace per layer that ran.
    """
    cfg = state.cfg
    y = np.asarray(y, dtype=np.int64)
    a_prev = np.asarray(x, dtype=np.int8)
    last = cfg.n_layers if layers is None else max(layers)
    want = set(range(1, cfg.n_layers + 1)) if layers is None else set(layers)
    traces = []
    for l in range(1, last + 1):
        kin, kout = cfg.widths[l - 1], cfg.widths[l]
        gamma = cfg.gamma(kout)
        H, P = state.H[l - 1], state.P[l - 1]
        W = state.W(l)
        z = preactivation(a_prev, W)
        a = activation(z)
        if cfg.saturate_z:
            z = saturate(z, kin)
        yhat = local_output(a, P)
        pred, tau, err, upd = local_error(yhat, y, robustness_threshold(cfg.robustness, kout))
        perm = group_permutation(cfg.seed, l, t, kout) if cfg.reshuffle_groups else None
        kstar = select_easiest(z, P, y, upd, gamma, perm)
        nsel = int((kstar >= 0).sum())
        nreinf = 0
        if l in want and upd.any():
            # LayerUpdate / PerceptronUpdate run only when M_l is not empty.
            S = selection_matrix(kstar, P, y, gamma, perm)
            if cfg.sequential_clip:
                h1 = cp_sequential(H, S, a_prev, cfg.bound)
            else:
                h1 = clip(H.astype(np.int64) + cp_increment(S, a_prev), cfg.bound)
            kq = kin if cfg.fan_in_reinforce else kout     # R11, or the fan-in variant
            mask = reinforce_mask(cfg.seed, l, t, reinforce_threshold(p_r, kq), kin * kout, kin)
            nreinf = int(mask.sum())
            state.H[l - 1] = reinforce(h1, mask, cfg.bound).astype(np.int8)
        traces.append(LayerTrace(a, z, yhat, pred, tau, err, upd, kstar,
                                 np.array([err.sum(), upd.sum(), nsel, nreinf], dtype=np.int64), perm))
        a_prev = a
    return traces


def forward(state: State, x: np.ndarray) -> List[np.ndarray]:
    """Local outputs y_hat_l of every layer (inference)."""
    a = np.asarray(x, dtype=np.int8)
    out = []
    for l in range(1, state.cfg.n_layers + 1):
        a = activation(preactivation(a, state.W(l)))
        out.append(local_output(a, state.P[l - 1]))
    return out


def rescale(p_r: float, wrong: int, samples: int) -> float:
    """p_r * sqrt(E^e) with E^e = wrong / samples (the end of Algorithm 1's epoch loop,
    Section 3.4); unchanged when no sample was trained on (R16)."""
    if samples <= 0:
        return p_r
    return p_r * math.sqrt(wrong / samples)


@dataclass
class EpochResult:
    p_r: float            # p_r * sqrt(E^e): the probability for the next epoch
    error_fraction: float  # E^e
    stats: np.ndarray      # int64 [batches][L][4], each step's layer counts
    steps: int             # full batches trained


def train_epoch(state: State, x: np.ndarray, y: np.ndarray, order: np.ndarray, batch: int,
                t0: int, p_r: float) -> EpochResult:
    """One pass of Algorithm 1's loop over mini-batches and the rescale that
    ends the epoch (Section 3.4), R16: the full batches order[b*batch:(b+1)*batch]
    of the training set x (int8 ±1 [N][K_0]), y, trained with steps t0 + b,
    all at the given p_r."""
    order = np.asarray(order, dtype=np.int64)
    nb = len(order) // batch
    wrong = 0
    stats = []
    for b in range(nb):
        idx = order[b * batch:(b + 1) * batch]
        traces = train_step(state, x[idx], np.asarray(y)[idx], t0 + b, p_r)
        wrong += int(traces[-1].err.sum())
        stats.append(np.stack([tr.stats for tr in traces]))
    if nb == 0:
        return EpochResult(p_r, float("nan"), np.zeros((0, state.cfg.n_layers, 4), np.int64), 0)
    return EpochResult(rescale(p_r, wrong, nb * batch), wrong / (nb * batch), np.stack(stats), nb)


def early_exit(state: State, x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Per layer l (rows): correct predictions of its local classifier, the
    patterns that exit at l, and how many of those exits are correct (R17).
    int64 [L][3]."""
    cfg = state.cfg
    y = np.asarray(y)
    n = len(y)
    out = np.zeros((cfg.n_layers, 3), dtype=np.int64)
    left = np.ones(n, dtype=bool)           # not exited yet
    for l, yhat in enumerate(forward(state, x), start=1):
        pred, tau, err, _ = local_error(yhat, y, robustness_threshold(cfg.robustness, cfg.widths[l]))
        out[l - 1, 0] = int((~err).sum())
        here = left & ((tau >= robustness_threshold(cfg.robustness, cfg.widths[l])) | (l == cfg.n_layers))
        out[l - 1, 1] = int(here.sum())
        out[l - 1, 2] = int((here & ~err).sum())
        left &= ~here
    return out


def evaluate(state: State, x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Correct predictions of each layer's local classifier; the last layer's
    classifier is the network output, earlier ones are early exits."""
    y = np.asarray(y)
    return np.array([int((np.argmax(yh, axis=1) == y).sum()) for yh in forward(state, x)],
                    dtype=np.int64)
