"""The memory model of Sec. 5.3 (Eq. 9): fit, prediction and the largest
batch that fits, on the host. The GPU side (measured steps and the
library's addressing bound) is in test_gpu_memory.py."""
import pytest

from paper_2509_26092_amd import memory as Mm


def test_fit_recovers_an_exact_line():
    p, a = 3.0e9, 2.5e7
    bs = [64, 128, 192, 256, 320, 384, 448, 512]
    p2, a2 = Mm.fit(bs, [p + a * b for b in bs])
    assert abs(p2 - p) <= 1e-6 * p and abs(a2 - a) <= 1e-9 * a


def test_fit_is_least_squares():
    # residuals of the fitted line sum to zero and are orthogonal to B
    bs = [64, 128, 192, 256, 320, 384, 448, 512]
    ms = [1e9 + 3e6 * b + (7e5 if i % 3 == 0 else -4e5) for i, b in enumerate(bs)]
    p, a = Mm.fit(bs, ms)
    r = [m - Mm.predict(p, a, b) for b, m in zip(bs, ms)]
    assert abs(sum(r)) < 1e-3 * max(ms)
    assert abs(sum(ri * b for ri, b in zip(r, bs))) < 1e-3 * max(ms) * 512


@pytest.mark.parametrize("p,a,m", [(3.0e9, 2.5e7, 288e9), (1e9, 1e6, 1e9 + 5e6), (0.0, 7.0, 49.0), (5.0, 2.0, 4.0)])
def test_max_batch_is_the_largest_that_fits(p, a, m):
    b = Mm.max_batch(p, a, m)
    if b > 0:
        assert Mm.predict(p, a, b) <= m
    assert Mm.predict(p, a, b + 1) > m


def test_max_batch_rejects_nonpositive_slope():
    with pytest.raises(ValueError):
        Mm.max_batch(1.0, 0.0, 10.0)
