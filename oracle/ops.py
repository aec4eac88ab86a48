"""Single operators of the ResNet-18 training step, fp64, NCHW.

Test infrastructure only (see the package docstring). The paper names the
network (ResNet-18, Sec. 5.1.1) and plain SGD (Sec. 2.2, Eq. 1) but none of the
operator formulas; every function below is the textbook definition written
out, with each convention the paper leaves open stated where it is used.
"""
import numpy as np


# ----------------------------------------------------------------------------
# Convolution (no bias). Output size floor((H + 2p - k)/s) + 1, zero padding.
# ----------------------------------------------------------------------------
def conv_out_size(h, k, s, p):
    return (h + 2 * p - k) // s + 1


def _tap_view(xp, kh, kw, s, ho, wo):
    """Input samples seen by kernel tap (kh, kw) for every output pixel."""
    return xp[:, :, kh:kh + s * (ho - 1) + 1:s, kw:kw + s * (wo - 1) + 1:s]


def conv2d_forward(x, w, stride, pad):
    """y[n,o,i,j] = sum_{c,kh,kw} w[o,c,kh,kw] * xpad[n,c,i*s+kh,j*s+kw].

    Direct sum over the kernel taps; each tap contracts the channel axis
    (a library dot product, no reordering of the sum beyond that)."""
    n, c, h, wd = x.shape
    o, c2, kh_, kw_ = w.shape
    assert c == c2
    ho, wo = conv_out_size(h, kh_, stride, pad), conv_out_size(wd, kw_, stride, pad)
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    y = np.zeros((n, o, ho, wo))
    for kh in range(kh_):
        for kw in range(kw_):
            t = _tap_view(xp, kh, kw, stride, ho, wo)            # [N,C,Ho,Wo]
            y += np.tensordot(w[:, :, kh, kw], t, axes=([1], [1])).transpose(1, 0, 2, 3)
    return y


def conv2d_backward_data(dy, w, x_shape, stride, pad):
    """Adjoint of conv2d_forward in x: scatter each tap's contribution back
    onto the padded input grid, then drop the padding."""
    n, c, h, wd = x_shape
    o, _, kh_, kw_ = w.shape
    _, _, ho, wo = dy.shape
    dxp = np.zeros((n, c, h + 2 * pad, wd + 2 * pad))
    for kh in range(kh_):
        for kw in range(kw_):
            contrib = np.tensordot(w[:, :, kh, kw], dy, axes=([0], [1])).transpose(1, 0, 2, 3)
            dxp[:, :, kh:kh + stride * (ho - 1) + 1:stride, kw:kw + stride * (wo - 1) + 1:stride] += contrib
    return dxp[:, :, pad:pad + h, pad:pad + wd]


def conv2d_backward_weight(dy, x, w_shape, stride, pad):
    """dW[o,c,kh,kw] = sum_{n,i,j} dy[n,o,i,j] * xpad[n,c,i*s+kh,j*s+kw]."""
    o, c, kh_, kw_ = w_shape
    _, _, ho, wo = dy.shape
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    dw = np.zeros(w_shape)
    for kh in range(kh_):
        for kw in range(kw_):
            t = _tap_view(xp, kh, kw, stride, ho, wo)
            dw[:, :, kh, kw] = np.tensordot(dy, t, axes=([0, 2, 3], [0, 2, 3]))
    return dw


# ----------------------------------------------------------------------------
# Batch normalisation, training mode. Statistics per channel over (N, H, W).
# Variance is the biased one (divide by M); the running variance uses the
# unbiased estimate M/(M-1). eps and momentum are not in the paper: the
# defaults follow the common PyTorch convention (eps 1e-5, momentum 0.1).
# ----------------------------------------------------------------------------
def bn_train_forward(x, gamma, beta, eps):
    m = x.shape[0] * x.shape[2] * x.shape[3]
    mean = x.sum(axis=(0, 2, 3)) / m
    xc = x - mean[None, :, None, None]
    var = (xc * xc).sum(axis=(0, 2, 3)) / m
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = xc * rstd[None, :, None, None]
    y = gamma[None, :, None, None] * xhat + beta[None, :, None, None]
    return y, {"mean": mean, "var": var, "rstd": rstd, "xhat": xhat, "m": m}


def bn_running_update(rm, rv, mean, var, m, momentum):
    """rm <- (1-mom) rm + mom*mean ; rv <- (1-mom) rv + mom*var*M/(M-1)."""
    rm_new = (1.0 - momentum) * rm + momentum * mean
    rv_new = (1.0 - momentum) * rv + momentum * var * (m / (m - 1.0))
    return rm_new, rv_new


def bn_eval_forward(x, gamma, beta, rm, rv, eps):
    rstd = 1.0 / np.sqrt(rv + eps)
    return gamma[None, :, None, None] * (x - rm[None, :, None, None]) * rstd[None, :, None, None] \
        + beta[None, :, None, None]


def bn_train_backward(dy, cache, gamma):
    """Gradient of y = gamma*xhat + beta with batch statistics:
    dgamma = sum dy*xhat ; dbeta = sum dy ;
    dx = gamma*rstd/M * (M*dy - dbeta - xhat*dgamma)."""
    xhat, rstd, m = cache["xhat"], cache["rstd"], cache["m"]
    dbeta = dy.sum(axis=(0, 2, 3))
    dgamma = (dy * xhat).sum(axis=(0, 2, 3))
    k = (gamma * rstd / m)[None, :, None, None]
    dx = k * (m * dy - dbeta[None, :, None, None] - xhat * dgamma[None, :, None, None])
    return dx, dgamma, dbeta


# ----------------------------------------------------------------------------
# ReLU. The subgradient at exactly 0 is taken as 0.
# ----------------------------------------------------------------------------
def relu(x):
    return np.maximum(x, 0.0)


def relu_backward(dz, z):
    """z is the ReLU output; gradient passes where z > 0."""
    return dz * (z > 0)


# ----------------------------------------------------------------------------
# Max pool k x k, stride s, padding p with -inf padding. The argmax is the
# FIRST maximum in the row-major (kh, kw) scan of the window; it is returned
# as that tap index kh*k + kw. Backward adds each output gradient to its
# argmax input (overlapping windows accumulate).
# ----------------------------------------------------------------------------
def maxpool_forward(x, k=3, s=2, p=1):
    n, c, h, w = x.shape
    ho, wo = conv_out_size(h, k, s, p), conv_out_size(w, k, s, p)
    xp = np.pad(x, ((0, 0), (0, 0), (p, p), (p, p)), constant_values=-np.inf)
    best = np.full((n, c, ho, wo), -np.inf)
    arg = np.zeros((n, c, ho, wo), dtype=np.int64)
    for kh in range(k):
        for kw in range(k):
            t = xp[:, :, kh:kh + s * (ho - 1) + 1:s, kw:kw + s * (wo - 1) + 1:s]
            better = t > best                  # strict: earlier tap wins ties
            best = np.where(better, t, best)
            arg = np.where(better, kh * k + kw, arg)
    return best, arg


def maxpool_backward(dy, arg, x_shape, k=3, s=2, p=1):
    n, c, h, w = x_shape
    _, _, ho, wo = dy.shape
    dxp = np.zeros((n, c, h + 2 * p, w + 2 * p))
    ii = np.arange(ho)[:, None]
    jj = np.arange(wo)[None, :]
    for kh in range(k):
        for kw in range(k):
            sel = (arg == kh * k + kw)
            contrib = np.where(sel, dy, 0.0)
            dxp[:, :, kh + s * ii, kw + s * jj] += contrib
    return dxp[:, :, p:p + h, p:p + w]


# ----------------------------------------------------------------------------
# Global average pool and fully connected layer (with bias).
# ----------------------------------------------------------------------------
def avgpool_forward(x):
    return x.mean(axis=(2, 3))


def avgpool_backward(df, x_shape):
    n, c, h, w = x_shape
    return np.broadcast_to(df[:, :, None, None] / (h * w), x_shape).copy()


def fc_forward(f, w, b):
    """z = f W^T + b ; f [N,K], w [C,K], b [C]."""
    return f @ w.T + b[None, :]


def fc_backward(dz, f, w):
    """dW = dz^T f ; db = sum_n dz ; df = dz W."""
    return dz @ w, dz.T @ f, dz.sum(axis=0)


# ----------------------------------------------------------------------------
# Softmax cross-entropy, mean over the batch, no label smoothing.
# loss = mean_n (logsumexp(z_n) - z_n[y_n]);  dz = (softmax(z) - onehot(y))/N
# ----------------------------------------------------------------------------
def softmax_ce(z, labels):
    n, c = z.shape
    labels = np.asarray(labels)
    if labels.min() < 0 or labels.max() >= c:
        raise ValueError("label outside [0, C)")
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(s[:, 0])
    picked = z[np.arange(n), labels]
    loss = float(np.mean(lse - picked))
    dz = e / s
    dz[np.arange(n), labels] -= 1.0
    dz /= n
    return loss, dz


# ----------------------------------------------------------------------------
# SGD with momentum and weight decay (PyTorch form, no dampening/Nesterov).
# The paper's update is plain SGD, w <- w - eta*g (Sec. 2.2, Eq. 1); momentum
# and weight decay are the training configuration's additions.
#   g' = g + wd*w ; v <- mu*v + g' ; w <- w - lr*v
# ----------------------------------------------------------------------------
def sgd_momentum(w, g, v, lr, momentum, weight_decay):
    g2 = g + weight_decay * w
    v_new = momentum * v + g2
    w_new = w - lr * v_new
    return w_new, v_new


# ----------------------------------------------------------------------------
# bf16 round-to-nearest-even of float32 values (result widened back to f64).
# Defined on the IEEE-754 binary32 bit pattern: keep the top 16 bits, adding
# half an ulp of bf16 with ties to the even (low bit of the kept part) result.
# ----------------------------------------------------------------------------
def round_bf16(x):
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    if nan.any():
        out = np.where(nan, np.nan, out)
    return out


# ----------------------------------------------------------------------------
# fp16 (IEEE-754 binary16) round-to-nearest-even of float32 values (result
# widened back to f64). binary16 has an 11-bit significand (10 stored bits),
# normal exponents -14..15 and subnormals in steps of 2^-24 below 2^-14. A
# value is rounded to the nearest multiple of its binade's quantum (ties to
# the even multiple); a result beyond the largest finite value 65504 is an
# infinity of the value's sign. NaN stays NaN, infinities stay infinite.
# ----------------------------------------------------------------------------
def round_fp16(x):
    f = np.asarray(x, dtype=np.float32).astype(np.float64)
    a = np.abs(f)
    finite = np.isfinite(a) & (a > 0)
    safe = np.where(finite, a, 1.0)
    _, e = np.frexp(safe)                      # safe = m * 2^e, m in [0.5, 1)
    e = np.maximum(e - 1, -14)                 # binade exponent; subnormals share 2^-14's quantum
    q = np.ldexp(1.0, e - 10)                  # quantum of the binade
    r = np.rint(safe / q) * q                  # exact quotient; rint rounds half to even
    r = np.where(r > 65504.0, np.inf, r)
    out = np.where(finite, np.copysign(r, f), f)
    return out

