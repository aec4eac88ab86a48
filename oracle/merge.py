"""Parameter-server merge with the model-update factor, and the dual-batch
planner arithmetic.

Test infrastructure only (see the package docstring).

Sec. 2.3: a worker pulls the global model, trains and updates its local copy,
and pushes the result; the server then updates the global model. Sec. 3.4:
large-batch workers contribute with factor 1, small-batch workers with
d_S/d_L (the scheme kept in Sec. 5.1.2) or sqrt(d_S/d_L).

The paper does not write the server's update formula. Reading R1 (used by the
library): each worker pushes its update vector Delta_X = p_pulled - p_X after
its local step, and the server applies the factor-weighted sum
    p <- p - (Delta_L + f * Delta_S).
R2 and R3 are the two other readings, kept so the difference is visible:
    R2  workers push gradients, the server combines g = g_L + f*g_S and takes
        one SGD-momentum step with its own state;
    R3  weighted model average p <- (p_L + f*p_S)/(1 + f).
"""
import math

import numpy as np

from . import ops


def worker_delta(p_pulled, p_local):
    """Update vector a worker pushes: pulled parameters minus local result."""
    return np.asarray(p_pulled, dtype=np.float64) - np.asarray(p_local, dtype=np.float64)


def dual_merge_r1(p, delta_small, delta_large, factor):
    """p <- p - (Delta_L + f * Delta_S), element-wise over the whole state."""
    if not math.isfinite(factor):
        raise ValueError("factor must be finite")
    return np.asarray(p, np.float64) - (np.asarray(delta_large, np.float64) + factor * np.asarray(delta_small, np.float64))


def dual_merge_r2(p, v, g_small, g_large, factor, lr, momentum, weight_decay):
    """Reading R2: server-side SGD-momentum step on g_L + f*g_S."""
    g = np.asarray(g_large, np.float64) + factor * np.asarray(g_small, np.float64)
    return ops.sgd_momentum(np.asarray(p, np.float64), g, v, lr, momentum, weight_decay)


def dual_merge_r3(p_small, p_large, factor):
    """Reading R3: data-weighted average of the two pushed models."""
    return (np.asarray(p_large, np.float64) + factor * np.asarray(p_small, np.float64)) / (1.0 + factor)


# ----------------------------------------------------------------------------
# Model-update factor (Sec. 3.4) and the load-balanced data split (Sec. 3.3).
# ----------------------------------------------------------------------------
def update_factor(d_small, d_large, scheme="ratio"):
    """'ratio': d_S/d_L ; 'sqrt': sqrt(d_S/d_L) ; 'none': 1."""
    r = d_small / d_large
    if scheme == "ratio":
        return r
    if scheme == "sqrt":
        return math.sqrt(r)
    if scheme == "none":
        return 1.0
    raise ValueError(scheme)


def data_split(k, d, n_small, n_large, whole_images=False):
    """Eqs. 4-6: d_L = k*d/n with n = n_S + n_L; d = n_L*d_L + n_S*d_S.

    whole_images=False returns the exact real-valued solution. With
    whole_images=True, d_L is first rounded to a whole number of images and
    d_S is solved from that rounded d_L (still unrounded itself): this is
    the reading under which Table 6's ImageNet row is reproduced exactly
    (d_L = 336306, d_S = 1281167 - 3*336306 = 272249)."""
    n = n_small + n_large
    d_large = k * d / n
    if whole_images:
        d_large = float(round(d_large))
    if n_small == 0:
        return d_large, None
    d_small = (d - n_large * d_large) / n_small
    return d_large, d_small


def small_batch_size(a, b, b_large, d_large, d_small):
    """Eq. 8: B_S = b / ((a + b/B_L) * d_L/d_S - a) (unrounded)."""
    return b / ((a + b / b_large) * d_large / d_small - a)


def epoch_time(a, b, batch, d):
    """Eq. 2: t = (a*x + b) * ceil(d/x)."""
    return (a * batch + b) * math.ceil(d / batch)
