"""Pins for the oracle's convolution: an explicit dense matrix built from the
definition with scalar loops (independent of the oracle's tap/contraction
code), the adjoint relation for the data gradient, and the bilinear form for
the weight gradient. 1x1 stride-1 is also checked against a plain matmul."""
import numpy as np
import pytest

from oracle import ops

CASES = [
    # (N, C, H, W, O, k, s, p)
    (2, 3, 5, 5, 4, 3, 1, 1),
    (2, 3, 6, 7, 4, 3, 2, 1),
    (1, 2, 9, 8, 3, 7, 2, 3),
    (2, 4, 6, 5, 3, 1, 2, 0),
    (1, 3, 7, 7, 2, 3, 2, 1),   # odd size, stride 2
    (2, 2, 4, 4, 3, 3, 1, 0),   # no padding
]


def dense_conv_matrix(N, C, H, W, O, k, s, p):
    """A[(n,o,i,j), (n,c,h,w)] = w-coefficient; returned as a function of w
    through a 3-index table so both dy/dx and dy/dw matrices follow."""
    Ho = (H + 2 * p - k) // s + 1
    Wo = (W + 2 * p - k) // s + 1
    entries = []   # (out_index, in_index, w_index)
    for n in range(N):
        for o in range(O):
            for i in range(Ho):
                for j in range(Wo):
                    oi = ((n * O + o) * Ho + i) * Wo + j
                    for c in range(C):
                        for kh in range(k):
                            for kw in range(k):
                                h = i * s - p + kh
                                w = j * s - p + kw
                                if 0 <= h < H and 0 <= w < W:
                                    ii = ((n * C + c) * H + h) * W + w
                                    wi = ((o * C + c) * k + kh) * k + kw
                                    entries.append((oi, ii, wi))
    return entries, Ho, Wo


@pytest.mark.parametrize("case", CASES)
def test_conv_matches_dense_matrix(case):
    N, C, H, W, O, k, s, p = case
    rng = np.random.default_rng(7)
    x = rng.standard_normal((N, C, H, W))
    w = rng.standard_normal((O, C, k, k))
    entries, Ho, Wo = dense_conv_matrix(*case)
    A = np.zeros((N * O * Ho * Wo, N * C * H * W))
    Bw = np.zeros((N * O * Ho * Wo, O * C * k * k))
    xf, wf = x.reshape(-1), w.reshape(-1)
    for oi, ii, wi in entries:
        A[oi, ii] += wf[wi]
        Bw[oi, wi] += xf[ii]
    y = ops.conv2d_forward(x, w, s, p)
    assert y.shape == (N, O, Ho, Wo)
    np.testing.assert_allclose(y.reshape(-1), A @ xf, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y.reshape(-1), Bw @ wf, rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal(y.shape)
    dx = ops.conv2d_backward_data(dy, w, x.shape, s, p)
    np.testing.assert_allclose(dx.reshape(-1), A.T @ dy.reshape(-1), rtol=1e-12, atol=1e-12)
    dw = ops.conv2d_backward_weight(dy, x, w.shape, s, p)
    np.testing.assert_allclose(dw.reshape(-1), Bw.T @ dy.reshape(-1), rtol=1e-12, atol=1e-12)


def test_conv1x1_is_matmul():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 5, 4, 6))
    w = rng.standard_normal((7, 5, 1, 1))
    y = ops.conv2d_forward(x, w, 1, 0)
    ref = np.einsum("oc,nchw->nohw", w[:, :, 0, 0], x)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_output_size_rule():
    assert ops.conv_out_size(224, 7, 2, 3) == 112
    assert ops.conv_out_size(112, 3, 2, 1) == 56
    assert ops.conv_out_size(7, 3, 2, 1) == 4
    assert ops.conv_out_size(5, 1, 2, 0) == 3
    assert ops.conv_out_size(1, 3, 2, 1) == 1
