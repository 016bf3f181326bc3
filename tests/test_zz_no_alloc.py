"""bmlp_forward_noalloc (the entry point for callers that cannot allocate)
against bmlp_forward, through the C ABI: identical local outputs on two
calls in a row, the second with a smaller batch, and a batch whose
activation rows exceed the static scratch rejected before any launch."""
import ctypes

import numpy as np
import pytest

from paper_2412_00119_amd.synth import random_pm1

from gpu_common import note, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fwd_impl", [1, 2])
@pytest.mark.parametrize("c", [11, 300])   # 300: y_hat from the forward kernel, into the output
def test_forward_noalloc_matches_forward(fwd_impl, c):
    torch = torch_cuda()
    from paper_2412_00119_amd import bmlp as B
    widths = (200, 192, 130, 64)
    net = B.BMLP(widths, c, 15, 300, 0, 0.25, 11, fwd_impl)
    rng = np.random.default_rng(3)
    for n in (300, 77):
        note(f"forward_noalloc impl {fwd_impl} c={c} n={n}")
        xb = net.pack(torch.from_numpy(random_pm1((n, widths[0]), rng)).cuda())
        ref = torch.empty((net.n_layers, n, c), dtype=torch.int32, device="cuda")
        got = torch.full((net.n_layers, n, c), -7, dtype=torch.int32, device="cuda")
        B.bmlp_forward(net.ctx, xb.data_ptr(), n, ref.data_ptr(), net._stream())
        B.bmlp_forward_noalloc(net.ctx, xb.data_ptr(), n, got.data_ptr(), net._stream())
        torch.cuda.synchronize()
        np.testing.assert_array_equal(got.cpu().numpy(), ref.cpu().numpy(), err_msg=f"n={n}")


def test_forward_noalloc_leaves_the_workspace_alone():
    torch = torch_cuda()
    from paper_2412_00119_amd import bmlp as B
    widths, c, n = (128, 128), 5, 64
    net = B.BMLP(widths, c, 7, n, 64, 0.25, 5)
    rng = np.random.default_rng(8)
    xb = net.pack(torch.from_numpy(random_pm1((n, widths[0]), rng)).cuda())
    yt = torch.from_numpy(rng.integers(0, c, n).astype(np.int32)).cuda()
    net.train_step(xb, yt, 0, 0.5)
    torch.cuda.synchronize()
    before = net.trace(1, n)["a"].cpu().numpy().copy()
    x2 = net.pack(torch.from_numpy(random_pm1((n, widths[0]), rng)).cuda())
    out = torch.empty((1, n, c), dtype=torch.int32, device="cuda")
    B.bmlp_forward_noalloc(net.ctx, x2.data_ptr(), n, out.data_ptr(), net._stream())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(net.trace(1, n)["a"].cpu().numpy(), before)


def test_forward_noalloc_rejects_more_than_the_scratch():
    torch = torch_cuda()
    from paper_2412_00119_amd import bmlp as B
    # 6 layers x 16384 patterns x 128 words x 8 bytes = 96 MiB of a_l rows
    widths, n = (8192,) * 7, 16384
    net = B.BMLP(widths, 2, 1, n, 64, 0.25, 1)
    x = torch.zeros((n, 128), dtype=torch.int64, device="cuda")
    out = torch.empty((6, n, 2), dtype=torch.int32, device="cuda")
    st = B.lib().bmlp_forward_noalloc(ctypes.c_void_p(net.ctx), ctypes.c_void_p(x.data_ptr()), n,
                                      ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(net._stream()))
    assert st == B.BMLP_ESHAPE
    assert "scratch" in B.last_error()
