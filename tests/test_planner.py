"""The dual-batch planner (Secs. 3.1-3.4) against the oracle's planner
arithmetic and against the batch sizes the paper prints: all eight small
batch sizes of Table 2 and every hybrid-stage row of Table 6 follow from one
b/a per configuration (b/a is the only hardware quantity Eq. 8 depends on)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import merge
from paper_2509_26092_amd import planner as P

G = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(G, name)) as f:
        return json.load(f)


def test_fit_linear_recovers_the_model():
    a, b = 2.1e-5, 1.7e-3
    x = np.array([32, 64, 128, 256, 512])
    assert P.fit_linear(x, a * x + b) == pytest.approx((a, b), rel=1e-12)
    rng = np.random.default_rng(3)
    t = a * x + b + rng.normal(0, 1e-6, x.size)
    fa, fb = P.fit_linear(x, t)
    A = np.stack([x, np.ones(x.size)], 1)
    ref = np.linalg.solve(A.T @ A, A.T @ t)                  # normal equations
    assert (fa, fb) == pytest.approx(tuple(ref), rel=1e-9)
    with pytest.raises(ValueError):
        P.fit_linear([64, 64], [1.0, 1.0])


def test_epoch_time_eq2_eq3():
    a, b = 0.5, 7.0
    assert P.epoch_time(a, b, 100, 1000) == (a * 100 + b) * 10
    assert P.epoch_time(a, b, 100, 1001) == (a * 100 + b) * 11
    assert P.epoch_time_approx(a, b, 100, 1000) == pytest.approx((a + b / 100) * 1000)
    for x, d in ((7, 95), (500, 50000), (33, 1000)):
        assert P.epoch_time(a, b, x, d) == pytest.approx(merge.epoch_time(a, b, x, d))


@pytest.mark.parametrize("k,d,ns,nl,whole", [(1.05, 50000, 1, 3, False), (1.1, 50000, 2, 2, False),
                                             (1.05, 1281167, 1, 3, True), (1.05, 1281167, 3, 1, True)])
def test_data_split_matches_oracle(k, d, ns, nl, whole):
    dl, ds = P.data_split(k, d, ns, nl, whole)
    odl, ods = merge.data_split(k, d, ns, nl, whole)
    assert dl == pytest.approx(odl) and ds == pytest.approx(ods)
    assert nl * dl + ns * ds == pytest.approx(d)              # Eq. 6


def test_small_batch_size_matches_oracle_and_balances():
    a, b, bl = 1.3e-4, 4.1e-3, 640
    dl, ds = P.data_split(1.05, 1281167, 1, 3, True)
    bs = P.small_batch_size(a, b, bl, dl, ds)
    assert bs == pytest.approx(merge.small_batch_size(a, b, bl, dl, ds), rel=1e-14)
    assert (a + b / bl) * dl == pytest.approx((a + b / bs) * ds, rel=1e-12)   # Eq. 7
    p = P.plan(a, b, bl, 1.05, 1281167, 1, 3, whole_images=True)
    assert p["t_small"] == pytest.approx(p["t_large"], rel=1e-12)
    assert p["t_large"] == pytest.approx(1.05 * p["t_all_large"], rel=1e-5)   # d_L rounded to whole images
    assert p["factor"] == pytest.approx(ds / dl)
    assert P.steps_per_round(p) == pytest.approx((ds / p["B_S"]) / (dl / bl))


def _feasible_ratio(d, bl, rows, k, whole):
    """The interval of b/a for which Eq. 8 (or its all-small form) rounds to
    every printed B_S."""
    r = np.geomspace(1.0, 1e4, 2000001)
    ok = np.ones(r.size, bool)
    for ns, bs in rows:
        nl = 4 - ns
        dl, ds = P.data_split(k, d, ns, nl, whole)
        ok &= np.round(P.small_batch_size(1.0, r, bl, dl, ds, k, nl)) == bs
    return r[ok]


def test_table2_small_batch_sizes():
    t = load("table2_merge_setting.json")
    for k in (1.05, 1.1):
        rows = [(r["n_S"], r["B_S"]) for r in t["rows"] if r["k"] == k]
        feas = _feasible_ratio(t["d"], t["B_L"], rows, k, False)
        assert feas.size, "no single b/a reproduces Table 2 at k=%g" % k
    # one b/a for both k: 24.65 reproduces all eight rows
    for r in t["rows"]:
        p = P.plan(1.0, 24.65, t["B_L"], r["k"], t["d"], r["n_S"], r["n_L"])
        assert p["B_S"] == r["B_S"], r
        if r["n_L"]:
            # the printed factor is d_S/d_L of the printed whole-image d_S
            assert round(P.update_factor(r["d_S"], r["d_L"]), 3) == pytest.approx(r["ratio"], abs=1e-12)
            assert abs(p["factor"] - r["ratio"]) < 1e-3


@pytest.mark.parametrize("dataset", ["cifar", "imagenet"])
def test_table6_hybrid_small_batch_sizes(dataset):
    t = load("table6_hybrid_batch_sizes.json")
    c = t[dataset]
    whole = dataset == "imagenet"
    for i, bl in enumerate(c["B_L"]):
        rows = [(int(ns), v[i]) for ns, v in c["B_S"].items()]
        feas = _feasible_ratio(c["d"], bl, rows, t["k"], whole)
        assert feas.size, "%s resolution %d: no single b/a reproduces the row" % (dataset, c["resolutions"][i])
        ratio = float(np.median(feas))
        for ns, bs in rows:
            p = P.plan(1.0, ratio, bl, t["k"], c["d"], ns, 4 - ns, whole_images=whole)
            assert p["B_S"] == bs


def test_update_factor_schemes():
    assert P.update_factor(10625, 13125) == pytest.approx(merge.update_factor(10625, 13125, "ratio"))
    assert P.update_factor(10625, 13125, "sqrt") == pytest.approx(math.sqrt(10625 / 13125))
    assert P.update_factor(1, 2, "none") == 1.0
    with pytest.raises(ValueError):
        P.update_factor(1, 2, "bogus")


def test_plan_rejects_unbalanceable_split():
    # k < 1 with only small workers: they would have to beat the all-large time
    with pytest.raises(ValueError):
        P.small_batch_size(1.0, 1.0, 500, None, 12500.0, 0.9, 0)
    with pytest.raises(ValueError):
        P.data_split(1.05, 50000, 0, 0)
