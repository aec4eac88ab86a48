"""Pins for the oracle's whole network: parameter counts of the standard
ResNet-18 variants, central finite differences of the training-mode loss on
the tiny configuration and on a small ImageNet-shaped net (every op type:
7x7 s2 stem, max pool, stride-2 blocks with projection), the BN running
statistics and the SGD update of a train step."""
import numpy as np
import pytest

from oracle import net, ops


def test_param_counts():
    # torchvision's resnet18 has 11,689,512 parameters (ImageNet, 1000 classes)
    assert net.Layout("imagenet", 1000).n_trainable == 11_689_512
    assert net.Layout("cifar", 100).n_trainable == 11_220_132
    assert net.Layout("tiny", 10).n_trainable == 5_306
    assert net.Layout("imagenet", 1000).n_state - 11_689_512 == 9_600
    assert net.Layout("tiny", 10).n_state - 5_306 == 96


def test_layer_count():
    convs, blocks, feat = net.conv_specs("imagenet")
    assert len(convs) == 20 and len(blocks) == 8 and feat == 512
    main_path = [c for c in convs if not c[0].endswith("ds")]
    assert len(main_path) == 17        # + FC = 18 weighted layers on the main path


def _directional_check(cfg, layout, state, x, y, keys, rng, n_coords=6, h=1e-6):
    loss, logits, grad, _ = net.forward_backward(cfg, layout, state, x, y)
    assert abs(loss - net.loss_only(cfg, layout, state, x, y)) < 1e-12
    # random direction over all trainable params
    v = rng.standard_normal(layout.n_trainable)
    v /= np.linalg.norm(v)        # unit step: few ReLU kinks are crossed
    sp, sm = state.copy(), state.copy()
    sp[:layout.n_trainable] += h * v
    sm[:layout.n_trainable] -= h * v
    fd = (net.loss_only(cfg, layout, sp, x, y) - net.loss_only(cfg, layout, sm, x, y)) / (2 * h)
    assert abs(fd - grad @ v) <= 1e-6 * max(1.0, abs(fd)), (fd, grad @ v)
    # individual coordinates of every tensor kind
    for key in keys:
        o, shp = layout.off[key]
        size = int(np.prod(shp))
        for idx in rng.choice(size, size=min(n_coords, size), replace=False):
            sp, sm = state.copy(), state.copy()
            sp[o + idx] += h
            sm[o + idx] -= h
            fd = (net.loss_only(cfg, layout, sp, x, y) - net.loss_only(cfg, layout, sm, x, y)) / (2 * h)
            an = grad[o + idx]
            assert abs(fd - an) <= 2e-6 * abs(an) + 5e-8, (key, idx, fd, an)


def test_fd_tiny_config():
    rng = np.random.default_rng(11)
    layout = net.Layout("tiny", 10)
    cfg = net.Config("tiny", 10)
    state = net.init_state(layout, 1)
    state[:layout.n_trainable] += 0.05 * rng.standard_normal(layout.n_trainable)  # beta/bias non-zero
    x = rng.standard_normal((8, 3, 16, 16))
    y = rng.integers(0, 10, 8)
    keys = ["stem.w", "stem.g", "stem.b", "s1b1c1.w", "s1b1c1.g", "s1b1c2.w", "s1b1c2.b", "fc.w", "fc.b"]
    _directional_check(cfg, layout, state, x, y, keys, rng)


def test_fd_tiny_config_with_dropout():
    """Dropout before the classifier (a fixed mask for the given step): the
    gradient still matches finite differences of the training loss, the mask
    changes the loss, and evaluation ignores it."""
    rng = np.random.default_rng(12)
    layout = net.Layout("tiny", 10)
    cfg = net.Config("tiny", 10, dropout=0.3, dropout_seed=99, dropout_step=4)
    state = net.init_state(layout, 2)
    state[:layout.n_trainable] += 0.05 * rng.standard_normal(layout.n_trainable)
    x = rng.standard_normal((8, 3, 16, 16))
    y = rng.integers(0, 10, 8)
    _directional_check(cfg, layout, state, x, y, ["s1b1c2.w", "s1b1c2.g", "fc.w", "fc.b"], rng)
    plain = net.Config("tiny", 10)
    assert abs(net.loss_only(cfg, layout, state, x, y) - net.loss_only(plain, layout, state, x, y)) > 1e-6
    np.testing.assert_array_equal(net.eval_logits(cfg, layout, state, x), net.eval_logits(plain, layout, state, x))
    # the FC input gradient is zero exactly where the mask drops a feature
    _, _, g, _ = net.forward_backward(cfg, layout, state, x, y)
    keep = net.philox.dropout_keep(99, 4, 8, layout.feat, 0.3)
    assert 0 < keep.sum() < keep.size


def test_fd_imagenet_shaped_small():
    rng = np.random.default_rng(12)
    layout = net.Layout("imagenet", 7)
    cfg = net.Config("imagenet", 7)
    state = net.init_state(layout, 2)
    state[:layout.n_trainable] += 0.02 * rng.standard_normal(layout.n_trainable)
    x = rng.standard_normal((4, 3, 20, 20))   # 20 -> 10 (stem) -> 5 (pool) -> 5,3,2,1
    y = rng.integers(0, 7, 4)
    keys = ["stem.w", "stem.g", "s1b1c1.w", "s2b1c1.w", "s2b1ds.w", "s2b1ds.g", "s2b1ds.b",
            "s3b2c2.w", "s4b1c1.w", "s4b2c2.g", "fc.w", "fc.b"]
    _directional_check(cfg, layout, state, x, y, keys, rng, n_coords=3)


def test_fd_cifar_shaped_small():
    rng = np.random.default_rng(13)
    layout = net.Layout("cifar", 5)
    cfg = net.Config("cifar", 5)
    state = net.init_state(layout, 3)
    x = rng.standard_normal((4, 3, 12, 12))   # stages 12,6,3,2
    y = rng.integers(0, 5, 4)
    _directional_check(cfg, layout, state, x, y, ["stem.w", "s2b1ds.w", "s4b2c1.w", "fc.w"], rng, n_coords=3)


def test_train_step_update_and_running_stats():
    rng = np.random.default_rng(14)
    layout = net.Layout("tiny", 10)
    cfg = net.Config("tiny", 10)
    state = net.init_state(layout, 4)
    x = rng.standard_normal((8, 3, 16, 16))
    y = rng.integers(0, 10, 8)
    v0 = np.zeros(layout.n_trainable)
    new, v1, loss, grad = net.train_step(cfg, layout, state, v0, x, y, 0.1)
    P = layout.n_trainable
    np.testing.assert_allclose(v1, grad + 5e-4 * state[:P], rtol=1e-14)
    np.testing.assert_allclose(new[:P], state[:P] - 0.1 * v1, rtol=1e-14)
    # stem running stats from the stem conv output's batch statistics
    y0 = ops.conv2d_forward(x, layout.get(state, "stem.w"), 1, 1)
    m = y0.shape[0] * y0.shape[2] * y0.shape[3]
    np.testing.assert_allclose(layout.get(new, "stem.rm"), 0.1 * y0.mean(axis=(0, 2, 3)), rtol=1e-12)
    np.testing.assert_allclose(layout.get(new, "stem.rv"),
                               0.9 + 0.1 * y0.var(axis=(0, 2, 3)) * m / (m - 1), rtol=1e-12)


def test_eval_logits_uses_running_stats():
    """With running stats equal to the batch's own statistics, eval-mode
    logits equal train-mode logits (single-block net)."""
    rng = np.random.default_rng(15)
    layout = net.Layout("tiny", 10)
    cfg = net.Config("tiny", 10, bn_momentum=1.0)
    state = net.init_state(layout, 5)
    x = rng.standard_normal((4, 3, 16, 16))
    y = rng.integers(0, 10, 4)
    _, logits_train, _, run = net.forward_backward(cfg, layout, state, x, y)
    st = state.copy()
    for name, rm, rv in run:
        m = 4 * 16 * 16
        layout.put(st, name + ".rm", rm)
        layout.put(st, name + ".rv", rv * (m - 1) / m)     # back to the biased variance
    np.testing.assert_allclose(net.eval_logits(cfg, layout, st, x), logits_train, rtol=1e-10, atol=1e-12)


def test_zero_fc_gives_ln_c_loss():
    rng = np.random.default_rng(16)
    layout = net.Layout("tiny", 10)
    cfg = net.Config("tiny", 10)
    state = net.init_state(layout, 6)
    layout.put(state, "fc.w", np.zeros((10, 16)))
    x = rng.standard_normal((2, 3, 16, 16))
    loss = net.loss_only(cfg, layout, state, x, np.array([3, 9]))
    assert abs(loss - np.log(10.0)) < 1e-12


def test_bf16_config_rounds_inputs_and_weights():
    rng = np.random.default_rng(17)
    layout = net.Layout("tiny", 10)
    st = net.init_state(layout, 7)
    x = rng.standard_normal((2, 3, 16, 16)).astype(np.float32)
    y = np.array([1, 2])
    c32 = net.Config("tiny", 10)
    c16 = net.Config("tiny", 10, bf16=True)
    st_r = st.copy()
    for name, *_ in layout.convs:
        layout.put(st_r, name + ".w", ops.round_bf16(layout.get(st, name + ".w")))
    l16 = net.loss_only(c16, layout, st, x, y)
    l32r = net.loss_only(c32, layout, st_r, ops.round_bf16(x), y)
    assert abs(l16 - l32r) < 1e-12
