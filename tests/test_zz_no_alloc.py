"""The allocation-free weight-gradient entry point (split-K partials in the
library's static device scratch) against the workspace entry point on the
same inputs: two calls in a row, the second with a smaller input, each equal
to the workspace call bit for bit (same kernels, same split counts, same
fixed-order reduction) and within tolerance of the oracle; and a shape whose
partials exceed the static scratch is refused on the host."""
import numpy as np
import pytest

from oracle import ops
from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import inputs
from gpu_util import PREC, assert_close, rounded, to_dev_nhwc

pytestmark = pytest.mark.gpu


def _wgrad_both(prec, N, C, H, W, O, k, s, p, seed):
    import torch
    x = inputs.tensor(seed, (N, C, H, W))
    Ho, Wo = ops.conv_out_size(H, k, s, p), ops.conv_out_size(W, k, s, p)
    dy = inputs.tensor(seed + 1, (N, O, Ho, Wo))
    xd, dyd = to_dev_nhwc(x, prec), to_dev_nhwc(dy, prec)
    nws = B.rn18op_conv2d_wgrad_workspace(PREC[prec], N, H, W, C, O, k, s, p)
    assert 0 < nws <= B.rn18op_conv2d_wgrad_noalloc_limit()
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    dw_ws = torch.full((O, C, k, k), float("nan"), dtype=torch.float32, device="cuda")
    dw_na = torch.full((O, C, k, k), float("nan"), dtype=torch.float32, device="cuda")
    B.rn18op_conv2d_wgrad(PREC[prec], dyd, xd, dw_ws, N, H, W, C, C, O, k, s, p, ws)
    B.rn18op_conv2d_wgrad_noalloc(PREC[prec], dyd, xd, dw_na, N, H, W, C, C, O, k, s, p)
    torch.cuda.synchronize()
    ref = ops.conv2d_backward_weight(rounded(dy, prec), rounded(x, prec), (O, C, k, k), s, p)
    return dw_ws.cpu().numpy(), dw_na.cpu().numpy(), ref, nws


@pytest.mark.parametrize("prec", ["bf16", "fp32"])
def test_noalloc_wgrad_matches_workspace_entry_point(prec):
    # first call: many split-K partials (for bf16 the 64-channel halo kernel,
    # one partial per block of the whole grid); second call: a smaller input
    calls = [(16, 64, 56, 56, 64, 3, 1, 1), (3, 128, 9, 11, 256, 3, 2, 1)]
    sizes = []
    for i, (N, C, H, W, O, k, s, p) in enumerate(calls):
        a, b, ref, nws = _wgrad_both(prec, N, C, H, W, O, k, s, p, 40 + i)
        sizes.append(N * C * H * W)
        print("%s call %d: %d-byte split-K scratch" % (prec, i, nws))
        assert np.all(np.isfinite(b))
        assert np.array_equal(a, b), "no-alloc result differs from the workspace entry point"
        assert_close(b, ref, 1e-5, "no-alloc wgrad vs oracle")
    assert sizes[1] < sizes[0]


def test_noalloc_wgrad_refuses_shapes_beyond_the_scratch():
    """1024 x (3x3 x 2048) fp32 partials of one split are 75.5 MB, beyond the
    48 MiB scratch: refused before any launch (the buffers are real and sized
    for the shape all the same)."""
    import torch
    N, C, H, W, O, k, s, p = 1, 2048, 3, 3, 1024, 3, 1, 1
    assert B.rn18op_conv2d_wgrad_noalloc_limit() == 48 << 20
    x = torch.zeros((N, H, W, C), dtype=torch.bfloat16, device="cuda")
    dy = torch.zeros((N, H, W, O), dtype=torch.bfloat16, device="cuda")
    dw = torch.zeros((O, C, k, k), dtype=torch.float32, device="cuda")
    with pytest.raises(B.Rn18Error) as e:
        B.rn18op_conv2d_wgrad_noalloc(B.RN18_BF16, dy, x, dw, N, H, W, C, C, O, k, s, p)
    assert e.value.code == B.RN18_EINVAL and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert float(dw.abs().sum()) == 0.0
