"""Pins for the oracle's bf16 rounding-point mode (the reading of the
paper's 16-bit mixed-precision training, Sec. 5.2.3: every activation and
activation gradient a bf16 step stores is rounded to bf16 once).

The mode is a convention, so it is pinned by what the definition implies
rather than by agreement with the GPU:
  * with an identity rounder it is the plain fp64 step, bit for bit;
  * every stored tensor passes through exactly one rounding point, once,
    from its exact value;
  * every forward rounding point is consumed downstream, and the backward
    rounding point paired with it carries the exact loss gradient with
    respect to it (central finite differences through the rounding hook),
    so a rounding placed before a term is added (e.g. a block-input
    gradient rounded before the shortcut's share) is caught;
  * with the real rounder every operand of every convolution and of every
    batch-norm is on the bf16 grid.
"""
import numpy as np
import pytest

from oracle import net, ops


def _setup(arch, classes, N, H, seed):
    rng = np.random.default_rng(seed)
    L = net.Layout(arch, classes)
    st = net.init_state(L, seed)
    st[:L.n_trainable] += 0.03 * rng.standard_normal(L.n_trainable)   # beta, bias non-zero
    x = rng.standard_normal((N, 3, H, H))
    y = rng.integers(0, classes, N)
    return L, st, x, y


CASES = [("tiny", 10, 4, 12, 21), ("imagenet", 7, 3, 20, 22)]


def _points(L):
    """Every tensor a bf16 step stores, by rounding point, from the
    architecture alone."""
    pts = []
    for name, *_ in L.convs:
        pts += [("y", name), ("dy", name)]
    pts.append(("z", "stem"))
    for bi, _ in enumerate(L.blocks):
        pts += [("z", ("z1", bi)), ("z", ("out", bi)), ("dz1", bi), ("dx", bi)]
    pts.append(("da_avg", 0))
    if L.arch == "imagenet":
        pts.append(("da_pool", 0))
    return pts


def _pairs(L):
    """(stored forward tensor, backward point holding the loss gradient wrt it)."""
    pairs = [(("y", name), ("dy", name)) for name, *_ in L.convs]
    nb = len(L.blocks)
    pairs.append((("z", "stem"), ("da_pool", 0) if L.arch == "imagenet" else ("dx", 0)))
    for bi in range(nb):
        pairs.append((("z", ("z1", bi)), ("dz1", bi)))
        pairs.append((("z", ("out", bi)), ("dx", bi + 1) if bi + 1 < nb else ("da_avg", 0)))
    return pairs


class Recorder:
    """decide() hook: identity rounding (the exact value is used) unless a
    perturbation is planted at one point; records what every rounding point
    received."""

    def __init__(self, plant=None):
        self.seen = {}
        self.calls = {}
        self.plant = plant

    def __call__(self, kind, site, pre, default):
        if kind != "round":
            return default
        self.calls[site] = self.calls.get(site, 0) + 1
        self.seen[site] = np.array(pre, copy=True)
        out = pre
        if self.plant is not None and self.plant[0] == site:
            out = pre + self.plant[1]
        return out


@pytest.mark.parametrize("arch,classes,N,H,seed", CASES)
def test_identity_rounder_is_the_plain_step(arch, classes, N, H, seed):
    L, st, x, y = _setup(arch, classes, N, H, seed)
    plain = net.forward_backward(net.Config(arch, classes, bf16=True), L, st, x, y)
    ident = net.forward_backward(net.Config(arch, classes, bf16=True, round_acts=True), L, st, x, y,
                                 decide=Recorder())
    assert plain[0] == ident[0]
    assert np.array_equal(plain[1], ident[1]) and np.array_equal(plain[2], ident[2])
    for (n1, m1, v1), (n2, m2, v2) in zip(plain[3], ident[3]):
        assert n1 == n2 and np.array_equal(m1, m2) and np.array_equal(v1, v2)


@pytest.mark.parametrize("arch,classes,N,H,seed", CASES)
def test_each_stored_tensor_rounded_once(arch, classes, N, H, seed):
    """Each point of the architecture's stored tensors is hit exactly once,
    with the shape of that tensor, and receives an exact (not yet rounded)
    value; with the real rounder the point's output is that value rounded to
    nearest even."""
    L, st, x, y = _setup(arch, classes, N, H, seed)
    cfg = net.Config(arch, classes, bf16=True, round_acts=True)
    rec = Recorder()
    net.forward_backward(cfg, L, st, x, y, decide=rec)
    expected = _points(L)
    assert sorted(map(repr, rec.calls)) == sorted(map(repr, expected))
    assert all(rec.calls[p] == 1 for p in expected)
    kinds = set(net.ROUNDING_POINTS) - (set() if arch == "imagenet" else {"da_pool"})
    assert kinds == {p[0] for p in expected}
    for p in expected:
        # an exact value, not one rounded before: off the bf16 grid wherever
        # it is not zero (ReLU and pool gradients hold exact zeros)
        v = rec.seen[p]
        nz = v[v != 0]
        assert nz.size > 0.1 * v.size, p
        off_grid = np.mean(ops.round_bf16(nz) != nz)
        assert off_grid > 0.9, (p, off_grid)
    # shapes follow the architecture
    h = ops.conv_out_size(H, L.spec["stem"][3], L.spec["stem"][4], L.spec["stem"][5])
    assert rec.seen[("y", "stem")].shape == (N, L.spec["stem"][2], h, h)
    assert rec.seen[("z", "stem")].shape == rec.seen[("y", "stem")].shape
    for bi, blk in enumerate(L.blocks):
        cin = L.spec[blk["c1"]][1]
        assert rec.seen[("dx", bi)].shape[:2] == (N, cin)
        assert rec.seen[("dz1", bi)].shape == rec.seen[("z", ("z1", bi))].shape
    # real rounder: what a point hands on is the RNE rounding of what it got
    got = {}

    def rounding(kind, site, pre, default):
        if kind == "round":
            assert np.array_equal(default, ops.round_bf16(pre))
            got[site] = default
        return default
    net.forward_backward(cfg, L, st, x, y, decide=rounding)
    assert set(map(repr, got)) == set(map(repr, expected))


@pytest.mark.parametrize("arch,classes,N,H,seed", CASES)
def test_backward_points_carry_the_loss_gradient(arch, classes, N, H, seed):
    """For every stored forward tensor T, the value at its paired backward
    point equals dLoss/dT: central differences of the loss with T perturbed
    through the rounding hook (identity rounding elsewhere) along a random
    direction v agree with <gradient point, v>."""
    L, st, x, y = _setup(arch, classes, N, H, seed)
    cfg = net.Config(arch, classes, bf16=True, round_acts=True)
    rec = Recorder()
    loss0 = net.forward_backward(cfg, L, st, x, y, decide=rec)[0]
    rng = np.random.default_rng(seed + 1)
    h = 1e-6
    for fwd, bwd in _pairs(L):
        T = rec.seen[fwd]
        v = rng.standard_normal(T.shape)
        if fwd == ("z", "stem") and arch == "imagenet":
            # the max pool is not differentiable at tied window maxima, and
            # windows of ReLU zeros tie: move only the positive entries
            v *= T > 0
        v /= np.linalg.norm(v)
        lp = net.forward_backward(cfg, L, st, x, y, need_grad=False, decide=Recorder((fwd, h * v)))[1]
        lm = net.forward_backward(cfg, L, st, x, y, need_grad=False, decide=Recorder((fwd, -h * v)))[1]
        fd = (ops.softmax_ce(lp, y)[0] - ops.softmax_ce(lm, y)[0]) / (2 * h)
        an = float(np.sum(rec.seen[bwd] * v))
        assert abs(fd - an) <= 2e-6 * max(abs(an), 1e-3), (fwd, bwd, fd, an, loss0)


def test_planted_block_input_misrounding_is_caught():
    """The finite-difference pin above detects a rounding point moved before
    a term is added: a copy of the oracle whose block-input gradient point
    receives only the first conv's data gradient (the shortcut's share added
    after the rounding) fails the pairing test."""
    L, st, x, y = _setup("tiny", 10, 4, 12, 23)
    cfg = net.Config("tiny", 10, bf16=True, round_acts=True)
    rec = Recorder()
    net.forward_backward(cfg, L, st, x, y, decide=rec)
    g_true = rec.seen[("dx", 0)]
    # what the misplaced point would see: the total minus the identity
    # shortcut's share (the masked output gradient of the block)
    mask = rec.seen[("z", ("out", 0))] > 0
    g2 = rec.seen[("da_avg", 0)] * mask
    g_bad = g_true - g2
    rng = np.random.default_rng(5)
    v = rng.standard_normal(g_true.shape)
    v /= np.linalg.norm(v)
    h = 1e-6
    lp = net.forward_backward(cfg, L, st, x, y, need_grad=False, decide=Recorder((("z", "stem"), h * v)))[1]
    lm = net.forward_backward(cfg, L, st, x, y, need_grad=False, decide=Recorder((("z", "stem"), -h * v)))[1]
    fd = (ops.softmax_ce(lp, y)[0] - ops.softmax_ce(lm, y)[0]) / (2 * h)
    assert abs(fd - np.sum(g_true * v)) <= 2e-6 * abs(fd) + 1e-9
    assert abs(fd - np.sum(g_bad * v)) > 1e-3 * abs(fd)


@pytest.mark.parametrize("arch,classes,N,H,seed", CASES)
def test_conv_and_bn_operands_on_the_bf16_grid(arch, classes, N, H, seed, monkeypatch):
    """With the real rounder, every convolution (all three passes) and every
    batch norm computes from bf16 values only: the rounding points cover
    every operand the bf16 step reads."""
    L, st, x, y = _setup(arch, classes, N, H, seed)
    cfg = net.Config(arch, classes, bf16=True, round_acts=True)
    seen = {"fwd": 0, "dgrad": 0, "wgrad": 0, "bn": 0}

    def on_grid(a):
        return np.array_equal(ops.round_bf16(a), a)

    orig = {k: getattr(ops, k) for k in ("conv2d_forward", "conv2d_backward_data", "conv2d_backward_weight",
                                        "bn_train_forward", "bn_train_backward")}

    def fwd(xx, w, s, p):
        assert on_grid(xx) and on_grid(w)
        seen["fwd"] += 1
        return orig["conv2d_forward"](xx, w, s, p)

    def dgrad(dy, w, shape, s, p):
        assert on_grid(dy) and on_grid(w)
        seen["dgrad"] += 1
        return orig["conv2d_backward_data"](dy, w, shape, s, p)

    def wgrad(dy, xx, shape, s, p):
        assert on_grid(dy) and on_grid(xx)
        seen["wgrad"] += 1
        return orig["conv2d_backward_weight"](dy, xx, shape, s, p)

    def bnf(yy, g, b, eps):
        assert on_grid(yy)
        seen["bn"] += 1
        return orig["bn_train_forward"](yy, g, b, eps)

    monkeypatch.setattr(ops, "conv2d_forward", fwd)
    monkeypatch.setattr(ops, "conv2d_backward_data", dgrad)
    monkeypatch.setattr(ops, "conv2d_backward_weight", wgrad)
    monkeypatch.setattr(ops, "bn_train_forward", bnf)
    net.forward_backward(cfg, L, st, x, y)
    nconv = len(L.convs)
    assert seen == {"fwd": nconv, "dgrad": nconv - 1, "wgrad": nconv, "bn": nconv}
