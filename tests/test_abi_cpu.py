"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/bmlp.h declares, and its host logic (configuration
checks, group-size rule, thresholds, layout) behaves as documented.  The
group-size rule and thresholds are compared with the oracle and the paper's
worked examples."""
import ctypes
import os
import re

import pytest

import oracle.bmlp as ob
from paper_2412_00119_amd import bmlp as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "bmlp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(bmlp_[a-z_]+)\s*\(", src)
    return sorted(set(names))


def test_every_declared_symbol_is_exported():
    L = B.lib()
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for st in (B.BMLP_OK, B.BMLP_EINVAL, B.BMLP_ESHAPE, B.BMLP_EHIP, B.BMLP_ESTATE):
        assert B.status_string(st) != "unknown status"
    assert B.status_string(99) == "unknown status"


@pytest.mark.parametrize("k", [525, 2025, 4096, 8192, 1024, 256, 97, 210, 35, 135])
def test_gamma_star_matches_oracle(k):
    cfg = B.make_config((100, k), 10, 15, 8, group_size=0)
    assert B.bmlp_describe(cfg, 1).gamma == ob.gamma_star(k)


def test_gamma_star_paper_examples():
    for k, g in [(525, 105), (2025, 81)]:
        info = B.bmlp_describe(B.make_config((64, k), 10, 15, 8, group_size=0), 1)
        assert (info.gamma, info.groups) == (g, k // g)


@pytest.mark.parametrize("p_r,k", [(0.5, 4096), (0.5, 256), (0.5, 784), (1e-9, 100), (0.0, 10),
                                   (1e6, 64), (0.37, 2048), (0.5 * 0.81 ** 0.5, 1024)])
def test_reinforce_threshold_matches_oracle(p_r, k):
    assert B.bmlp_reinforce_threshold(p_r, k) == ob.reinforce_threshold(p_r, k)


@pytest.mark.parametrize("r,k", [(0.25, 4096), (0.25, 35), (0.0, 100), (0.3, 1000), (1.0 / 3, 999)])
def test_robust_threshold_matches_oracle(r, k):
    info = B.bmlp_describe(B.make_config((50, k), 10, 15, 8, group_size=1, robustness=r), 1)
    assert info.robust_thr == ob.robustness_threshold(r, k)


def test_layout_is_aligned_and_disjoint():
    cfg = B.make_config((784, 1024, 1024), 10, 127, 256)
    sb = B.bmlp_state_bytes(cfg)
    wb = B.bmlp_workspace_bytes(cfg)
    spans = []
    for l in (1, 2):
        i = B.bmlp_describe(cfg, l)
        assert i.h_planes == 7 and i.h_ps % 16 == 0 and 32 * i.h_ps >= i.k_in
        assert i.ld_h == 4 * i.h_planes * i.h_ps and i.ld_h % 64 == 0
        for off in (i.off_h, i.off_w, i.off_p, i.off_a, i.off_err, i.off_upd, i.off_kstar):
            assert off % 256 == 0
        spans += [(i.off_h, i.off_h + i.k_out * i.ld_h), (i.off_w, i.off_w + i.k_out * i.words_in * 8),
                  (i.off_p, i.off_p + 10 * i.words_out * 8)]
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= sb and wb > 0


@pytest.mark.parametrize("kw", [
    dict(widths=(784,), n_classes=10, bound=15, max_batch=8),             # no layer
    dict(widths=(784, 256), n_classes=1, bound=15, max_batch=8),          # one class
    dict(widths=(784, 256), n_classes=10, bound=14, max_batch=8),         # even bound
    dict(widths=(784, 256), n_classes=10, bound=129, max_batch=8),        # bound > 127
    dict(widths=(784, 250), n_classes=10, bound=15, max_batch=8),         # 64 does not divide 250
    dict(widths=(784, 256), n_classes=10, bound=15, max_batch=0),
    dict(widths=(784, 256), n_classes=10, bound=15, max_batch=B.MAX_BATCH + 1),
    dict(widths=(0, 256), n_classes=10, bound=15, max_batch=8),
    dict(widths=(784, 40000), n_classes=10, bound=15, max_batch=8, group_size=100),
    dict(widths=(784, 256), n_classes=10, bound=15, max_batch=8, robustness=-1.0),
    dict(widths=(784, 256), n_classes=10, bound=15, max_batch=8, fwd_impl=7),
])
def test_invalid_configs_rejected(kw):
    cfg = B.make_config(**kw)
    assert B.bmlp_state_bytes(cfg) == 0
    assert B.bmlp_workspace_bytes(cfg) == 0
    ctx = ctypes.c_void_p()
    # valid-looking aligned device pointers: rejection happens before any launch
    st = B.lib().bmlp_init(ctypes.byref(cfg), 1 << 20, 1 << 21, None, ctypes.byref(ctx))
    assert st in (B.BMLP_EINVAL, B.BMLP_ESHAPE)
    assert ctx.value is None


def test_null_and_misaligned_buffers_rejected():
    cfg = B.make_config((784, 256), 10, 15, 8)
    ctx = ctypes.c_void_p()
    L = B.lib()
    assert L.bmlp_init(ctypes.byref(cfg), None, 1 << 20, None, ctypes.byref(ctx)) == B.BMLP_EINVAL
    assert L.bmlp_init(ctypes.byref(cfg), (1 << 20) + 8, 1 << 21, None, ctypes.byref(ctx)) == B.BMLP_ESTATE
    assert L.bmlp_init(ctypes.byref(cfg), 1 << 20, (1 << 21) + 128, None, ctypes.byref(ctx)) == B.BMLP_ESTATE
    assert L.bmlp_init(None, 1 << 20, 1 << 21, None, ctypes.byref(ctx)) == B.BMLP_EINVAL
    assert L.bmlp_train_step(None, 1 << 20, 1 << 21, 4, 0, 0.5, 1 << 22, None) == B.BMLP_EINVAL
    assert L.bmlp_pack(None, 4, 10, None, None) == B.BMLP_EINVAL
    assert L.bmlp_pack(None, 0, 0, None, None) == B.BMLP_ESHAPE


def test_stats_stride_matches_binding():
    """The binding allocates step statistics with the header's row stride."""
    hdr = open(os.path.join(ROOT, "include", "bmlp.h")).read()
    m = re.search(r"#define\s+BMLP_STATS_STRIDE\s+(\d+)", hdr)
    assert m and int(m.group(1)) == B.STATS_STRIDE
    assert B.STATS_STRIDE * 4 % 128 == 0    # a 128-byte line per layer


@pytest.mark.parametrize("bound,planes", [(1, 1), (3, 2), (5, 3), (15, 4), (31, 5), (33, 6), (63, 6), (127, 7)])
def test_h_planes_hold_offset_values(bound, planes):
    """H stores u = (h + B) / 2 in [0, B]: bits(B) planes, the fewest that hold B."""
    i = B.bmlp_describe(B.make_config((100, 64), 10, bound, 64), 1)
    assert i.h_planes == planes
    assert (1 << planes) > bound >= (1 << (planes - 1))
    assert i.ld_h == 4 * planes * i.h_ps and i.h_ps == 16


@pytest.mark.parametrize("p_r,wrong,samples", [(0.5, 317, 1024), (0.5, 0, 48 * 1024), (0.5, 1024, 1024),
                                                (0.123456789, 12345, 49152), (2.0, 7, 9), (0.5, 3, 0)])
def test_epoch_rescale_matches_oracle(p_r, wrong, samples):
    # host arithmetic in IEEE double on both sides: equal to the last bit
    assert B.bmlp_epoch_rescale(p_r, wrong, samples) == ob.rescale(p_r, wrong, samples)


def test_variants_validated_and_shared_classifier_held_once():
    cfg = B.make_config((20, 16, 16, 16), 3, 7, 8, group_size=4)
    shared = B.make_config((20, 16, 16, 16), 3, 7, 8, group_size=4, variants=B.BMLP_VARIANT_SHARED_CLASSIFIER)
    assert 0 < B.bmlp_state_bytes(shared) < B.bmlp_state_bytes(cfg)
    offs = {B.bmlp_describe(shared, l).off_p for l in (1, 2, 3)}
    assert len(offs) == 1
    # unequal widths cannot share a classifier; unknown variant bits are refused
    assert B.bmlp_state_bytes(B.make_config((20, 16, 8), 3, 7, 8, group_size=4,
                                            variants=B.BMLP_VARIANT_SHARED_CLASSIFIER)) == 0
    assert B.bmlp_state_bytes(B.make_config((20, 16), 3, 7, 8, group_size=4, variants=32)) == 0


def test_input_side_shapes_rejected_before_any_launch():
    assert B.lib().bmlp_expand(None, 4, 0, 64, 1, None, None) == B.BMLP_ESHAPE
    assert B.lib().bmlp_expand(None, 4, 10, 0, 1, None, None) == B.BMLP_ESHAPE
    assert B.lib().bmlp_expand(None, 4, 10, 64, 1, None, None) == B.BMLP_EINVAL
    assert B.lib().bmlp_feature_median(None, 0, 8, None, None) == B.BMLP_ESHAPE
    assert B.lib().bmlp_binarize(None, 3, 8, None, None, None) == B.BMLP_EINVAL


def test_epoch_summary_from_counts():
    # E^e = last-layer errors / samples and p_r sqrt(E^e) (Alg. 1's epoch
    # loop, Sec. 3.4), from a host copy of the epoch's stats rows
    import ctypes
    import math
    import numpy as np
    from paper_2412_00119_amd import bmlp as B
    steps, L, batch = 3, 2, 10
    st = np.zeros((steps, L, B.STATS_STRIDE), dtype=np.int32)
    st[:, 1, 0] = [2, 0, 5]     # last layer's 01-loss counts
    st[:, 0, 0] = [9, 9, 9]     # other layers do not count
    e, nxt = B.bmlp_epoch_summary(st.ctypes.data, steps, L, batch, 0.5)
    assert e == 7 / 30 and nxt == 0.5 * math.sqrt(7 / 30)
    e, nxt = B.bmlp_epoch_summary(0, 0, L, batch, 0.5)
    assert math.isnan(e) and nxt == 0.5
    with pytest.raises(B.BmlpError):
        B.bmlp_epoch_summary(0, 2, L, batch, 0.5)
    with pytest.raises(B.BmlpError):
        B.bmlp_epoch_summary(st.ctypes.data, steps, 0, batch, 0.5)
