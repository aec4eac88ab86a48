"""The merge oracle's factor and the dual-batch data split against the
values the paper prints (Tables 2, 3 and 6), and the merge rule's algebra."""
import json
import math
import os

import numpy as np
import pytest

from oracle import merge

G = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(G, name)) as f:
        return json.load(f)


def test_table2_data_split_and_factor():
    t = load("table2_merge_setting.json")
    for r in t["rows"]:
        dl, ds = merge.data_split(r["k"], t["d"], r["n_S"], r["n_L"])
        if r["n_L"] == 0:
            # all workers small: each gets d/n (Eq. 6 with n_L = 0)
            assert abs(t["d"] / t["n"] - r["d_S"]) < 1e-9
            continue
        assert abs(dl - r["d_L"]) < 1e-9
        assert abs(ds - r["d_S"]) < 1.0          # printed value is truncated or rounded
        # the printed factor is d_S/d_L of the printed (whole-image) d_S:
        # (50000 - 13125)/3 = 12291.67 is printed 12291, and 12291/13125 -> 0.936
        f = merge.update_factor(r["d_S"], dl, "ratio")
        assert round(f, 3) == pytest.approx(r["ratio"], abs=1e-12)


def test_table3_sqrt_factor():
    t = load("table3_update_factor.json")
    for r in t["rows"]:
        assert round(math.sqrt(r["ratio"]), 3) == pytest.approx(r["sqrt"], abs=1e-12)
        assert merge.update_factor(1.0, 1.0, "none") == 1.0


def test_table6_data_amounts():
    t = load("table6_batch_data.json")
    for key in ("cifar", "imagenet"):
        r = t[key]
        dl, _ = merge.data_split(r["k"], r["d"], 1, 3)
        assert abs(dl - r["d_L"]) < 1.0
        assert abs(r["d"] / r["n"] - r["d_all_large"]) < 1.0
        for ns, dsp in r["d_S"].items():
            dl, ds = merge.data_split(r["k"], r["d"], int(ns), 4 - int(ns), whole_images=True)
            assert dl == r["d_L"]
            assert round(ds) == dsp            # Table 6 rounds to nearest


def test_small_batch_size_balances_time():
    """Eq. 8 makes (a + b/B_L) d_L equal (a + b/B_S) d_S (Eq. 7)."""
    a, b, bl, dl, ds = 1e-3, 0.0246, 500.0, 13125.0, 10625.0
    bs = merge.small_batch_size(a, b, bl, dl, ds)
    assert abs((a + b / bl) * dl - (a + b / bs) * ds) < 1e-9
    # with b/a in the range that reproduces Table 2, B_S rounds to the printed 83
    assert round(merge.small_batch_size(1.0, 24.65, 500.0, 13125.0, 10625.0)) == 83


def test_epoch_time_eq2():
    assert merge.epoch_time(2.0, 3.0, 10, 95) == (2.0 * 10 + 3.0) * 10


def test_merge_r1_algebra():
    rng = np.random.default_rng(0)
    p, ds, dl = rng.standard_normal((3, 50))
    np.testing.assert_allclose(merge.dual_merge_r1(p, ds, dl, 0.0), p - dl)
    np.testing.assert_allclose(merge.dual_merge_r1(p, dl, dl, 1.0), p - 2 * dl)
    # linear in f
    m0, m1, m2 = (merge.dual_merge_r1(p, ds, dl, f) for f in (0.0, 0.5, 1.0))
    np.testing.assert_allclose(m1, 0.5 * (m0 + m2), atol=1e-14)
    with pytest.raises(ValueError):
        merge.dual_merge_r1(p, ds, dl, float("nan"))


def test_merge_r1_equals_r2_without_momentum():
    """Deltas of plain SGD steps from the same pulled p are lr*g, so the
    delta merge equals one server SGD step on g_L + f g_S."""
    rng = np.random.default_rng(1)
    p, gs, gl = rng.standard_normal((3, 40))
    lr, f = 0.05, 0.81
    ds, dl = lr * gs, lr * gl
    r1 = merge.dual_merge_r1(p, ds, dl, f)
    r2, _ = merge.dual_merge_r2(p, np.zeros(40), gs, gl, f, lr, 0.0, 0.0)
    np.testing.assert_allclose(r1, r2, rtol=1e-13, atol=1e-15)


def test_merge_r3_fixed_point():
    rng = np.random.default_rng(2)
    q = rng.standard_normal(10)
    np.testing.assert_allclose(merge.dual_merge_r3(q, q, 0.636), q)
