"""Pins for the oracle's BN, ReLU, pools, FC, softmax cross-entropy, SGD and
bf16 rounding: invariants, closed forms, scalar brute force and finite
differences."""
import math

import numpy as np
import pytest
import torch

from oracle import ops


def fd_grad(f, x, h=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        idx = it.multi_index
        old = x[idx]
        x[idx] = old + h
        fp = f(x)
        x[idx] = old - h
        fm = f(x)
        x[idx] = old
        g[idx] = (fp - fm) / (2 * h)
    return g


# ---------------------------------------------------------------- BN
def test_bn_forward_invariants():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((4, 3, 5, 5)) * np.array([0.5, 2.0, 10.0])[None, :, None, None] + 3.0
    eps = 1e-5
    y, c = ops.bn_train_forward(x, np.ones(3), np.zeros(3), eps)
    np.testing.assert_allclose(y.mean(axis=(0, 2, 3)), 0.0, atol=1e-12)
    var = x.var(axis=(0, 2, 3))          # biased, library routine
    np.testing.assert_allclose((y ** 2).mean(axis=(0, 2, 3)), var / (var + eps), rtol=1e-12)
    np.testing.assert_allclose(c["var"], var, rtol=1e-12)
    g, b = np.array([2.0, -1.0, 0.5]), np.array([1.0, 0.0, -3.0])
    y2, _ = ops.bn_train_forward(x, g, b, eps)
    np.testing.assert_allclose(y2.mean(axis=(0, 2, 3)), b, atol=1e-12)


def test_bn_backward_invariants_and_fd():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 2, 3, 4)) + 1.5
    g, b = np.array([1.3, -0.7]), np.array([0.2, 0.1])
    dy = rng.standard_normal(x.shape)
    for eps in (0.0, 1e-2):
        y, c = ops.bn_train_forward(x, g, b, eps)
        dx, dg, db = ops.bn_train_backward(dy, c, g)
        np.testing.assert_allclose(dx.sum(axis=(0, 2, 3)), 0.0, atol=1e-10)
        # sum dx*xhat = gamma*rstd*sum(dy*xhat)*eps/(var+eps)  (zero iff eps=0)
        lhs = (dx * c["xhat"]).sum(axis=(0, 2, 3))
        rhs = g * c["rstd"] * dg * eps / (c["var"] + eps)
        np.testing.assert_allclose(lhs, rhs, atol=1e-10)
    eps = 1e-2
    f = lambda xx: float((ops.bn_train_forward(xx, g, b, eps)[0] * dy).sum())
    _, c = ops.bn_train_forward(x, g, b, eps)
    dx, dg, db = ops.bn_train_backward(dy, c, g)
    np.testing.assert_allclose(dx, fd_grad(f, x.copy()), rtol=1e-6, atol=1e-7)
    fg = lambda gg: float((ops.bn_train_forward(x, gg, b, eps)[0] * dy).sum())
    fb = lambda bb: float((ops.bn_train_forward(x, g, bb, eps)[0] * dy).sum())
    np.testing.assert_allclose(dg, fd_grad(fg, g.copy()), rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(db, fd_grad(fb, b.copy()), rtol=1e-6, atol=1e-7)


def test_bn_running_update_closed_form():
    rm, rv = np.array([0.0, 1.0]), np.array([1.0, 2.0])
    mean, var = np.array([2.0, -1.0]), np.array([4.0, 0.5])
    rm2, rv2 = ops.bn_running_update(rm, rv, mean, var, 5, 0.1)
    np.testing.assert_allclose(rm2, [0.2, 0.9 * 1.0 + 0.1 * -1.0])
    np.testing.assert_allclose(rv2, [0.9 + 0.1 * 4.0 * 5 / 4, 1.8 + 0.1 * 0.5 * 5 / 4])


def test_bn_eval_matches_train_when_stats_equal():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 3, 4, 4))
    g, b = rng.standard_normal(3), rng.standard_normal(3)
    y, c = ops.bn_train_forward(x, g, b, 1e-5)
    ye = ops.bn_eval_forward(x, g, b, c["mean"], c["var"], 1e-5)
    np.testing.assert_allclose(ye, y, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- ReLU
def test_relu_backward_mask():
    z = np.array([-1.0, 0.0, 0.5])
    np.testing.assert_array_equal(ops.relu_backward(np.ones(3), ops.relu(z)), [0.0, 0.0, 1.0])


# ---------------------------------------------------------------- pools
def maxpool_scalar(x, k=3, s=2, p=1):
    n, c, h, w = x.shape
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    out = np.zeros((n, c, ho, wo))
    arg = np.zeros((n, c, ho, wo), dtype=np.int64)
    for a in range(n):
        for b in range(c):
            for i in range(ho):
                for j in range(wo):
                    best, bi = -math.inf, -1
                    for kh in range(k):
                        for kw in range(k):
                            hh, ww = i * s - p + kh, j * s - p + kw
                            if 0 <= hh < h and 0 <= ww < w and x[a, b, hh, ww] > best:
                                best, bi = x[a, b, hh, ww], kh * k + kw
                    out[a, b, i, j], arg[a, b, i, j] = best, bi
    return out, arg


@pytest.mark.parametrize("shape", [(2, 3, 8, 8), (1, 2, 7, 9), (1, 1, 1, 1), (2, 2, 2, 3)])
def test_maxpool_scalar_bruteforce(shape):
    rng = np.random.default_rng(4)
    x = rng.standard_normal(shape)
    x[..., ::2] = np.round(x[..., ::2])   # plant ties
    y, arg = ops.maxpool_forward(x)
    yr, ar = maxpool_scalar(x)
    np.testing.assert_array_equal(y, yr)
    np.testing.assert_array_equal(arg, ar)
    dy = rng.standard_normal(y.shape)
    dx = ops.maxpool_backward(dy, arg, x.shape)
    dref = np.zeros(shape)
    ho, wo = y.shape[2:]
    for a in range(shape[0]):
        for b in range(shape[1]):
            for i in range(ho):
                for j in range(wo):
                    t = ar[a, b, i, j]
                    dref[a, b, i * 2 - 1 + t // 3, j * 2 - 1 + t % 3] += dy[a, b, i, j]
    np.testing.assert_allclose(dx, dref, rtol=0, atol=1e-14)


def test_maxpool_first_max_on_ties():
    x = np.zeros((1, 1, 4, 4))
    _, arg = ops.maxpool_forward(x)
    # window of output (0,0) covers rows -1..1, cols -1..1; first in-bounds
    # tap in row-major order is (kh=1, kw=1) -> 4
    assert arg[0, 0, 0, 0] == 4
    assert arg[0, 0, 1, 1] == 0


def test_avgpool_and_fc_fd():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 3, 3, 4))
    w, b = rng.standard_normal((5, 3)), rng.standard_normal(5)
    dz = rng.standard_normal((2, 5))
    f = ops.avgpool_forward(x)
    np.testing.assert_allclose(f, x.reshape(2, 3, -1).sum(-1) / 12.0)
    z = ops.fc_forward(f, w, b)
    np.testing.assert_allclose(z, np.array([[sum(f[n, k] * w[c, k] for k in range(3)) + b[c]
                                              for c in range(5)] for n in range(2)]))
    df, dw, db = ops.fc_backward(dz, f, w)
    np.testing.assert_allclose(dw, fd_grad(lambda ww: float((ops.fc_forward(f, ww, b) * dz).sum()), w.copy()), rtol=1e-6)
    np.testing.assert_allclose(db, dz.sum(0))
    np.testing.assert_allclose(df, fd_grad(lambda ff: float((ops.fc_forward(ff, w, b) * dz).sum()), f.copy()), rtol=1e-6)
    dx = ops.avgpool_backward(df, x.shape)
    np.testing.assert_allclose(dx, fd_grad(lambda xx: float((ops.avgpool_forward(xx) * df).sum()), x.copy()), rtol=1e-6, atol=1e-9)


# ---------------------------------------------------------------- CE
@pytest.mark.parametrize("c,lnc", [(10, 2.302585092994046), (100, 4.605170185988092), (1000, 6.907755278982137)])
def test_ce_zero_logits(c, lnc):
    loss, dz = ops.softmax_ce(np.zeros((4, c)), np.array([0, 1, c - 1, 3]))
    assert abs(loss - lnc) < 1e-12
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-15)


def test_ce_against_library_and_fd():
    from scipy.special import logsumexp
    rng = np.random.default_rng(6)
    z = rng.standard_normal((5, 7)) * 4
    y = rng.integers(0, 7, 5)
    loss, dz = ops.softmax_ce(z, y)
    ref = np.mean(logsumexp(z, axis=1) - z[np.arange(5), y])
    assert abs(loss - ref) < 1e-12
    np.testing.assert_allclose(dz, fd_grad(lambda zz: ops.softmax_ce(zz, y)[0], z.copy()), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-15)


def test_ce_large_logits_stable():
    loss, dz = ops.softmax_ce(np.array([[1000.0, 0.0]]), np.array([1]))
    assert abs(loss - 1000.0) < 1e-9
    assert np.all(np.isfinite(dz))


def test_ce_rejects_bad_labels():
    with pytest.raises(ValueError):
        ops.softmax_ce(np.zeros((2, 3)), np.array([0, 3]))
    with pytest.raises(ValueError):
        ops.softmax_ce(np.zeros((2, 3)), np.array([-1, 0]))


# ---------------------------------------------------------------- SGD
def test_sgd_momentum_closed_forms():
    w0, g1, g2 = np.array([1.0, -2.0]), np.array([0.5, 0.25]), np.array([-1.0, 2.0])
    lr, mu, wd = 0.1, 0.9, 5e-4
    w1, v1 = ops.sgd_momentum(w0, g1, np.zeros(2), lr, mu, wd)
    np.testing.assert_allclose(w1, w0 - lr * (g1 + wd * w0))
    w2, v2 = ops.sgd_momentum(w1, g2, v1, lr, mu, wd)
    np.testing.assert_allclose(w2, w1 - lr * (mu * (g1 + wd * w0) + g2 + wd * w1))
    w3, _ = ops.sgd_momentum(w0, g1, np.zeros(2), 0.0, mu, wd)
    np.testing.assert_array_equal(w3, w0)


def test_plain_sgd_special_case():
    """mu = wd = 0 reduces to the paper's w - eta*g (Eq. 1)."""
    w0, g = np.array([3.0, 1.0]), np.array([1.0, -4.0])
    w1, _ = ops.sgd_momentum(w0, g, np.zeros(2), 0.5, 0.0, 0.0)
    np.testing.assert_allclose(w1, [2.5, 3.0])


# ---------------------------------------------------------------- bf16
def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(8)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 3.0e38, -3.0e38, 1e-40],
                                 dtype=np.float32)]).astype(np.float32)
    # exact ties: 1 + 2^-8 (round down to even), 1 + 3*2^-8 (round up to even)
    ours = ops.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    assert ops.round_bf16(np.float32(1.00390625)) == 1.0
    assert ops.round_bf16(np.float32(1.01171875)) == 1.015625
