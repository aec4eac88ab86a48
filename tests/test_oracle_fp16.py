"""Pins for the oracle's fp16 precision with loss scaling (the reading of the
16-bit mixed-precision training of Sec. 5.2.3: IEEE fp16 at the storage
points, the backward pass started from a power-of-two multiple of the loss,
the gradient divided by it before the update, and the update skipped when
the gradient is not finite).

  * fp16 rounding against numpy's binary16 conversion, and by hand at the
    binade edges, ties, subnormals and the overflow threshold;
  * loss scaling is exact algebra: with the stored tensors not rounded, any
    power-of-two scale gives the unscaled gradient bit for bit;
  * with the stored tensors rounded, the scale acts before the rounding:
    a large scale keeps small gradients out of fp16's subnormal range and
    brings the step closer to the exact one than scale 1 does;
  * an overflowing scale makes the gradient non-finite and the update is
    skipped (parameters and momentum unchanged, running statistics kept).
"""
import numpy as np
import pytest

from oracle import net, ops


def test_round_fp16_matches_numpy_binary16():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200_000) * 10.0 ** rng.integers(-9, 6, 200_000)
    x = np.concatenate([x, -x]).astype(np.float32)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(ops.round_fp16(x), ref)


@pytest.mark.parametrize("v,want", [
    (1.0, 1.0),
    (1.0 + 2.0 ** -11, 1.0),                      # tie -> even
    (1.0 + 3 * 2.0 ** -11, 1.0 + 2.0 ** -9),      # tie -> even (up)
    (1.0 + 2.0 ** -11 + 2.0 ** -20, 1.0 + 2.0 ** -10),
    (65504.0, 65504.0),                           # largest finite
    (65519.0, 65504.0),                           # below the overflow threshold
    (65520.0, np.inf),                            # tie at the threshold rounds to the even (overflowed) value
    (1e6, np.inf),
    (2.0 ** -14, 2.0 ** -14),                     # smallest normal
    (2.0 ** -24, 2.0 ** -24),                     # smallest subnormal
    (2.0 ** -25, 0.0),                            # tie between 0 and 2^-24 -> 0 (even)
    (3 * 2.0 ** -25, 2.0 ** -23),                 # tie between 2^-24 and 2^-23 -> even
    (2.0 ** -14 - 2.0 ** -25, 2.0 ** -14),        # top of the subnormal range: tie -> even (the normal)
    (-3.0e-8, -2.0 ** -25 * 2),                   # 3e-8 / 2^-24 = 0.50 -> 1 quantum, sign kept
])
def test_round_fp16_by_hand(v, want):
    got = float(ops.round_fp16(np.float32(v)))
    assert got == want or (np.isinf(want) and got == want), (v, got, want)


def test_round_fp16_specials():
    out = ops.round_fp16(np.array([np.inf, -np.inf, np.nan, 0.0, -0.0], np.float32))
    assert out[0] == np.inf and out[1] == -np.inf and np.isnan(out[2])
    assert out[3] == 0.0 and np.signbit(out[4])


def _setup(seed, N=4, H=12):
    rng = np.random.default_rng(seed)
    L = net.Layout("tiny", 10)
    st = net.init_state(L, seed)
    st[:L.n_trainable] += 0.03 * rng.standard_normal(L.n_trainable)
    x = rng.standard_normal((N, 3, H, H))
    y = rng.integers(0, 10, N)
    return L, st, x, y


@pytest.mark.parametrize("scale", [2.0 ** 4, 2.0 ** 12, 2.0 ** 24])
def test_scaling_is_exact_without_storage_rounding(scale):
    """Images and weights in fp16, stored tensors exact: the gradient of the
    scaled backward pass divided by a power-of-two scale is the unscaled
    gradient bit for bit (every operation is linear in the scale, and
    multiplying by a power of two commutes with float64 rounding)."""
    L, st, x, y = _setup(1)
    g1 = net.forward_backward(net.Config("tiny", 10, fp16=True), L, st, x, y)[2]
    gs = net.forward_backward(net.Config("tiny", 10, fp16=True, loss_scale=scale), L, st, x, y)[2]
    assert np.array_equal(g1, gs)


def test_scale_acts_before_rounding():
    """Stored tensors rounded to fp16: with scale 1 a share of the gradients
    fall into fp16's subnormal range and lose precision; a scale of 2^12
    moves them up before the rounding, so the step's parameter gradient is
    closer to the exact (unrounded) one. A scale applied after the rounding
    would leave the error unchanged."""
    L, st, x, y = _setup(2)
    # shrink the classifier so that the backward pass carries small values
    L.put(st, "fc.w", L.get(st, "fc.w") * 1e-3)
    exact = net.forward_backward(net.Config("tiny", 10, fp16=True), L, st, x, y)[2]
    errs = {}
    for s in (1.0, 2.0 ** 12):
        cfg = net.Config("tiny", 10, fp16=True, round_acts=True, loss_scale=s)
        g = net.forward_backward(cfg, L, st, x, y)[2]
        o, shp = L.off["stem.w"]
        n = int(np.prod(shp))
        errs[s] = np.linalg.norm(g[o:o + n] - exact[o:o + n]) / np.linalg.norm(exact[o:o + n])
    assert errs[2.0 ** 12] < 2e-2
    assert errs[1.0] > 5 * errs[2.0 ** 12], errs


def test_overflow_skips_the_update():
    """A scale so large that a stored gradient exceeds fp16's largest finite
    value: the gradient is not finite, and the step leaves every parameter
    and the momentum unchanged while the BN running statistics move."""
    L, st, x, y = _setup(3)
    v0 = 0.01 * np.random.default_rng(4).standard_normal(L.n_trainable)
    cfg = net.Config("tiny", 10, fp16=True, round_acts=True, loss_scale=2.0 ** 40)
    new, v1, loss, grad = net.train_step(cfg, L, st, v0, x, y, 0.1)
    assert not np.all(np.isfinite(grad))
    P = L.n_trainable
    assert np.array_equal(new[:P], st[:P]) and np.array_equal(v1, v0)
    assert not np.array_equal(L.get(new, "stem.rm"), L.get(st, "stem.rm"))
    assert np.isfinite(loss)
    # the same step at a moderate scale updates every tensor kind
    new2, _, _, grad2 = net.train_step(net.Config("tiny", 10, fp16=True, round_acts=True, loss_scale=2.0 ** 8),
                                       L, st, v0, x, y, 0.1)
    assert np.all(np.isfinite(grad2)) and not np.array_equal(new2[:P], st[:P])


def test_fp16_rounding_points_are_the_bf16_points():
    """The fp16 mode rounds at exactly the points the bf16 mode does, each
    once, with the fp16 rounding."""
    L, st, x, y = _setup(5)
    seen = {}

    def rec(kind, site, pre, default):
        if kind == "round":
            seen.setdefault(site, []).append(np.array_equal(default, ops.round_fp16(pre)))
        return default
    net.forward_backward(net.Config("tiny", 10, fp16=True, round_acts=True, loss_scale=2.0 ** 10), L, st, x, y,
                         decide=rec)
    seen_b = {}

    def rec_b(kind, site, pre, default):
        if kind == "round":
            seen_b.setdefault(site, []).append(True)
        return default
    net.forward_backward(net.Config("tiny", 10, bf16=True, round_acts=True), L, st, x, y, decide=rec_b)
    assert set(map(repr, seen)) == set(map(repr, seen_b))
    assert all(v == [True] for v in seen.values())
