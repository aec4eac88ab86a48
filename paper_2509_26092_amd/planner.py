"""Dual-batch planner (host side): training-time model, load-balanced data
split, small batch size and model-update factor, fitted to step times
measured on this GPU.

Sec. 3.2 models the time of one batch of x images as a*x + b (linear
regression over measured batches), so an epoch over d images takes
(a*x + b) * ceil(d/x) (Eq. 2), approximately (a + b/x) * d (Eq. 3).
Sec. 3.3 balances n_L large-batch and n_S small-batch workers: every worker
gets the time k * (a + b/B_L) * d/n of an all-large run (k > 1, the extra
training-time ratio), which gives d_L = k*d/n (Eq. 4), d_S from
d = n_L*d_L + n_S*d_S (Eq. 6) and the small batch size
B_S = b / ((a + b/B_L) * d_L/d_S - a) (Eq. 8). With no large workers the
small workers share d equally and B_S solves (a + b/B_S) * d/n =
k * (a + b/B_L) * d/n. Sec. 3.4: the small workers' updates are scaled by
d_S/d_L, or by its square root (the large workers' by 1).

The hybrid scheme (Sec. 4) re-plans per resolution: a and b are fitted per
resolution and B_L is the large batch of that stage.
"""
import math

import numpy as np


def fit_linear(batches, times):
    """Least-squares a, b of time = a*batch + b (Sec. 3.2)."""
    x = np.asarray(batches, dtype=np.float64)
    t = np.asarray(times, dtype=np.float64)
    if x.size < 2 or np.ptp(x) == 0:
        raise ValueError("need at least two different batch sizes")
    A = np.stack([x, np.ones_like(x)], axis=1)
    (a, b), *_ = np.linalg.lstsq(A, t, rcond=None)
    return float(a), float(b)


def epoch_time(a, b, batch, d):
    """Eq. 2: (a*x + b) * ceil(d/x)."""
    return (a * batch + b) * math.ceil(d / batch)


def epoch_time_approx(a, b, batch, d):
    """Eq. 3: (a + b/x) * d."""
    return (a + b / batch) * d


def data_split(k, d, n_small, n_large, whole_images=False):
    """Eqs. 4 and 6: d_L = k*d/n, d_S = (d - n_L*d_L)/n_S. With whole_images,
    d_L is rounded to whole images before d_S is solved."""
    n = n_small + n_large
    if n < 1 or k <= 0 or d <= 0:
        raise ValueError("bad split")
    if n_large == 0:
        return None, d / n
    d_large = k * d / n
    if whole_images:
        d_large = float(round(d_large))
    d_small = (d - n_large * d_large) / n_small if n_small else None
    return d_large, d_small


def small_batch_size(a, b, b_large, d_large, d_small, k=None, n_large=None):
    """Eq. 8 (unrounded). With no large workers (n_large == 0), B_S solves
    (a + b/B_S) = k * (a + b/B_L)."""
    if n_large == 0:
        den = k * (a + b / b_large) - a
    else:
        den = (a + b / b_large) * d_large / d_small - a
    if np.any(np.asarray(den) <= 0):
        raise ValueError("no small batch size balances this split (k too small for the fitted a, b)")
    return b / den


def update_factor(d_small, d_large, scheme="ratio"):
    """Sec. 3.4: 'ratio' d_S/d_L, 'sqrt' its square root, 'none' 1."""
    if scheme == "none":
        return 1.0
    r = d_small / d_large
    if scheme == "ratio":
        return r
    if scheme == "sqrt":
        return math.sqrt(r)
    raise ValueError(scheme)


def plan(a, b, b_large, k, d, n_small, n_large, scheme="ratio", whole_images=False):
    """The dual-batch configuration for fitted a, b and a given B_L."""
    d_large, d_small = data_split(k, d, n_small, n_large, whole_images)
    out = {"a": a, "b": b, "B_L": b_large, "k": k, "d": d, "n_S": n_small, "n_L": n_large,
           "d_L": d_large, "d_S": d_small}
    if n_small:
        bs = small_batch_size(a, b, b_large, d_large, d_small, k, n_large)
        out["B_S_exact"] = bs
        out["B_S"] = max(1, int(round(bs)))
        out["factor"] = update_factor(d_small, d_large, scheme) if n_large else None
        # Eq. 7: both kinds of worker take the same time (exact for the unrounded B_S)
        out["t_small"] = epoch_time_approx(a, b, bs, d_small)
    if n_large:
        out["t_large"] = epoch_time_approx(a, b, b_large, d_large)
    out["t_all_large"] = epoch_time_approx(a, b, b_large, d / (n_small + n_large))
    return out


def steps_per_round(p):
    """Small-worker steps per large-worker step that keep both on the same
    epoch pace: (d_S/B_S) / (d_L/B_L)."""
    return (p["d_S"] / p["B_S"]) / (p["d_L"] / p["B_L"])
