"""ResNet-18 variants, the flat parameter state and the fp64 training step.

Test infrastructure only (see the package docstring).

The paper evaluates ResNet-18 (Sec. 5.1.1: eighteen conv layers plus one
fully connected layer) on CIFAR-100 32x32 and on ImageNet (Sec. 5.2.1). It
fixes neither the CIFAR stem nor the block details; the three variants here
are the training configurations' definitions:

  tiny      3x3 s1 stem 3->16, one BasicBlock 16->16 (identity skip), FC 16->C
  cifar     3x3 s1 stem 3->64, no max pool, stages 64/128/256/512 x 2 blocks
  imagenet  7x7 s2 p3 stem 3->64, 3x3 s2 p1 max pool, same stages

BasicBlock: conv3x3(s)-BN-ReLU-conv3x3(1)-BN, plus shortcut, then ReLU. The
stride sits in the first conv of stages 2-4; the shortcut is a 1x1 stride-s
conv + BN when the stride or the width changes, else identity. Convs have no
bias, the FC has one. The stem is conv-BN-ReLU.

Flat state (float32 on the device, float64 here), in this order:
  for every conv in forward order (stem, then per block c1, c2, [ds]):
      W [Cout, Cin, KH, KW] (OIHW), gamma [Cout], beta [Cout]
  FC weight [C, F], FC bias [C]                        -> P trainable floats
  for every BN in the same order: running_mean [Cout], running_var [Cout]
                                                       -> R floats
"""
import numpy as np

from . import ops, philox

ARCHS = ("tiny", "cifar", "imagenet")


def conv_specs(arch):
    """List of conv layers (name, cin, cout, k, stride, pad) in forward order,
    and the block structure."""
    if arch == "tiny":
        stem = ("stem", 3, 16, 3, 1, 1)
        widths, nblocks, first_stride = [16], [1], [1]
    elif arch == "cifar":
        stem = ("stem", 3, 64, 3, 1, 1)
        widths, nblocks, first_stride = [64, 128, 256, 512], [2] * 4, [1, 2, 2, 2]
    elif arch == "imagenet":
        stem = ("stem", 3, 64, 7, 2, 3)
        widths, nblocks, first_stride = [64, 128, 256, 512], [2] * 4, [1, 2, 2, 2]
    else:
        raise ValueError(arch)
    convs = [stem]
    blocks = []
    cin = stem[2]
    for si, (wd, nb, fs) in enumerate(zip(widths, nblocks, first_stride)):
        for bi in range(nb):
            s = fs if bi == 0 else 1
            pre = "s%db%d" % (si + 1, bi + 1)
            c1 = (pre + "c1", cin, wd, 3, s, 1)
            c2 = (pre + "c2", wd, wd, 3, 1, 1)
            convs += [c1, c2]
            ds = None
            if s != 1 or cin != wd:
                ds = (pre + "ds", cin, wd, 1, s, 0)
                convs.append(ds)
            blocks.append({"c1": c1[0], "c2": c2[0], "ds": ds[0] if ds else None})
            cin = wd
    return convs, blocks, cin


class Layout:
    """Offsets of every tensor in the flat state."""

    def __init__(self, arch, num_classes):
        self.arch = arch
        self.num_classes = num_classes
        self.convs, self.blocks, self.feat = conv_specs(arch)
        self.spec = {c[0]: c for c in self.convs}
        self.off = {}
        o = 0
        for name, cin, cout, k, s, p in self.convs:
            self.off[name + ".w"] = (o, (cout, cin, k, k)); o += cout * cin * k * k
            self.off[name + ".g"] = (o, (cout,)); o += cout
            self.off[name + ".b"] = (o, (cout,)); o += cout
        self.off["fc.w"] = (o, (num_classes, self.feat)); o += num_classes * self.feat
        self.off["fc.b"] = (o, (num_classes,)); o += num_classes
        self.n_trainable = o
        for name, cin, cout, k, s, p in self.convs:
            self.off[name + ".rm"] = (o, (cout,)); o += cout
            self.off[name + ".rv"] = (o, (cout,)); o += cout
        self.n_state = o

    def get(self, state, key):
        o, shp = self.off[key]
        return state[o:o + int(np.prod(shp))].reshape(shp)

    def put(self, flat, key, val):
        o, shp = self.off[key]
        flat[o:o + int(np.prod(shp))] = np.asarray(val).reshape(-1)


def init_state(layout, seed):
    """He-normal (fan_in) conv and FC weights, gamma=1, beta=0, FC bias 0,
    running mean 0, running var 1. Used only by oracle-side tests; parity
    tests hand the same state to both implementations."""
    rng = np.random.default_rng(seed)
    st = np.zeros(layout.n_state)
    for name, cin, cout, k, s, p in layout.convs:
        layout.put(st, name + ".w", rng.standard_normal((cout, cin, k, k)) * np.sqrt(2.0 / (cin * k * k)))
        layout.put(st, name + ".g", np.ones(cout))
        layout.put(st, name + ".rv", np.ones(cout))
    layout.put(st, "fc.w", rng.standard_normal((layout.num_classes, layout.feat)) * np.sqrt(2.0 / layout.feat))
    return st


class Config:
    def __init__(self, arch, num_classes, bf16=False, momentum=0.9, weight_decay=5e-4,
                 bn_eps=1e-5, bn_momentum=0.1, round_acts=False, dropout=0.0, dropout_seed=0, dropout_step=0,
                 fp16=False, loss_scale=1.0):
        assert not (bf16 and fp16)
        self.arch = arch
        self.num_classes = num_classes
        self.bf16 = bf16
        # fp16 configurations: IEEE binary16 in place of bf16 at every
        # rounding point, with loss scaling: the backward pass starts from
        # loss_scale x dLoss/dlogits, so every stored gradient is scaled,
        # and the parameter gradient is divided by loss_scale at the end (a
        # power of two: exact in float64). A step whose gradient is not
        # finite (an fp16 overflow) updates no parameter (train_step).
        self.fp16 = fp16
        self.loss_scale = float(loss_scale)
        self.half = bf16 or fp16
        self.round16 = ops.round_bf16 if bf16 else ops.round_fp16 if fp16 else None
        self.momentum = momentum
        self.weight_decay = weight_decay
        self.bn_eps = bn_eps
        self.bn_momentum = bn_momentum
        # round_acts: additionally round every stored activation and
        # activation gradient to the 16-bit type at the points where a
        # 16-bit training step stores them (see ROUNDING_POINTS). Off by
        # default.
        self.round_acts = round_acts
        # dropout before the classifier in training-mode passes (the paper's
        # adaptive regularisation, Sec. 4.1): rate, generator key and the
        # training step whose mask is used (see philox.py); 0 = off
        self.dropout = dropout
        self.dropout_seed = dropout_seed
        self.dropout_step = dropout_step


# Where a 16-bit (bf16 or fp16) training step stores a tensor in the 16-bit
# type (rounded once, RNE):
#   ("y", conv)     conv output, before BN (BN statistics are taken of it)
#   ("z", site)     ReLU output: stem, block z1, block output
#   ("da_avg", 0)   gradient entering the last block (avg-pool backward)
#   ("dy", conv)    BN backward output, the gradient entering the conv
#   ("dz1", block)  data gradient of the block's second conv
#   ("dx", block)   gradient wrt the block input: the first conv's data
#                   gradient plus the shortcut's (the masked output gradient
#                   of an identity block, the projection conv's data gradient
#                   otherwise), summed exactly and rounded once
#   ("da_pool", 0)  max-pool backward output
# Every stored tensor is rounded once, from its exact value, and is consumed
# only in its rounded form.
ROUNDING_POINTS = ("y", "z", "da_avg", "dy", "dz1", "dx", "da_pool")


def forward_backward(cfg, layout, state, images, labels, train=True, need_grad=True, decide=None):
    """One forward (batch statistics) and backward pass.

    Returns loss, logits, the flat gradient (length P), and the new running
    statistics (list of (name, rm, rv)).

    The derivative of ReLU at an input of exactly 0, the argmax of a max pool
    window with tied maxima, and the bf16 rounding of a value on a rounding
    midpoint are not fixed by the arithmetic; inputs within rounding
    distance of those points make the choice depend on the precision the
    value was computed in. `decide`, if given, is called as
    decide("relu", site, pre, mask), decide("pool", site, x, arg) and
    decide("round", point, exact, rounded) and returns the mask / argmax /
    rounded tensor to use (relu sites: "stem", ("z1", block), ("out",
    block); rounding points: ROUNDING_POINTS); the default is mask = pre > 0,
    the first maximum and round-to-nearest-even.

    16-bit configurations (the mixed precision of Sec. 5.2.3, bf16 or fp16):
    the images and the conv weights are rounded to the 16-bit type
    (round-to-nearest-even) and then used in float64; BN statistics, the FC
    layer, the loss, the master weights and the momentum stay in full
    precision. fp16 configurations scale the backward pass by
    cfg.loss_scale and divide the gradient by it at the end."""
    x = np.asarray(images, dtype=np.float64)
    if cfg.half:
        x = cfg.round16(x)
    eps = cfg.bn_eps

    def W(name):
        w = layout.get(state, name + ".w")
        return cfg.round16(w) if cfg.half else w

    caches = {}
    run_stats = []
    masks = {}
    rounding = cfg.half and cfg.round_acts

    def rb(point, v):
        if not rounding:
            return v
        r = cfg.round16(v)
        if decide is not None:
            r = decide("round", point, v, r)
        return r

    def relu_site(site, pre):
        mask = pre > 0
        if decide is not None:
            mask = decide("relu", site, pre, mask)
        masks[site] = mask
        return rb(("z", site), ops.relu(pre))

    def conv_bn(name, inp, act):
        _, cin, cout, k, s, p = layout.spec[name]
        y = rb(("y", name), ops.conv2d_forward(inp, W(name), s, p))
        g = layout.get(state, name + ".g")
        b = layout.get(state, name + ".b")
        if train:
            out, c = ops.bn_train_forward(y, g, b, eps)
            rm, rv = ops.bn_running_update(layout.get(state, name + ".rm"), layout.get(state, name + ".rv"),
                                           c["mean"], c["var"], c["m"], cfg.bn_momentum)
            run_stats.append((name, rm, rv))
        else:
            out = ops.bn_eval_forward(y, g, b, layout.get(state, name + ".rm"), layout.get(state, name + ".rv"), eps)
            c = None
        caches[name] = {"inp": inp, "bn": c}
        return out

    a = relu_site("stem", conv_bn("stem", x, True))
    stem_out = a
    pool_arg = None
    if cfg.arch == "imagenet":
        a, pool_arg = ops.maxpool_forward(a)
        if decide is not None:
            pool_arg = decide("pool", "stem", stem_out, pool_arg)
    block_io = []
    for bi, blk in enumerate(layout.blocks):
        inp = a
        z1 = relu_site(("z1", bi), conv_bn(blk["c1"], inp, True))
        b2 = conv_bn(blk["c2"], z1, False)
        sc = conv_bn(blk["ds"], inp, False) if blk["ds"] else inp
        a = relu_site(("out", bi), b2 + sc)
        block_io.append((inp, z1, a))
    f = ops.avgpool_forward(a)
    drop = None
    if train and cfg.dropout > 0.0:
        # inverted dropout on the classifier input: kept features scaled by
        # 1 / (1 - p), so the expected input is unchanged
        _, scale = philox.dropout_params(cfg.dropout)
        drop = philox.dropout_keep(cfg.dropout_seed, cfg.dropout_step, f.shape[0], f.shape[1], cfg.dropout) * scale
        f = f * drop
    wfc = layout.get(state, "fc.w")
    bfc = layout.get(state, "fc.b")
    logits = ops.fc_forward(f, wfc, bfc)
    if not need_grad:
        return None, logits, None, run_stats
    loss, dz = ops.softmax_ce(logits, labels)
    if cfg.fp16:
        dz = dz * cfg.loss_scale

    grad = np.zeros(layout.n_trainable)
    df, dwfc, dbfc = ops.fc_backward(dz, f, wfc)
    if drop is not None:
        df = df * drop
    layout.put(grad, "fc.w", dwfc)
    layout.put(grad, "fc.b", dbfc)
    da = rb(("da_avg", 0), ops.avgpool_backward(df, a.shape))

    def bn_conv_back(name, dout):
        """dout: gradient wrt this BN's output. Writes dW, dgamma, dbeta and
        returns the gradient wrt the conv input (None for the stem)."""
        _, cin, cout, k, s, p = layout.spec[name]
        c = caches[name]
        dy, dg, dbeta = ops.bn_train_backward(dout, c["bn"], layout.get(state, name + ".g"))
        dy = rb(("dy", name), dy)
        layout.put(grad, name + ".g", dg)
        layout.put(grad, name + ".b", dbeta)
        inp = c["inp"]
        layout.put(grad, name + ".w", ops.conv2d_backward_weight(dy, inp, (cout, cin, k, k), s, p))
        if name == "stem":
            return None
        return ops.conv2d_backward_data(dy, W(name), inp.shape, s, p)

    for bi in reversed(range(len(layout.blocks))):
        blk = layout.blocks[bi]
        g2 = da * masks[("out", bi)]
        dz1 = rb(("dz1", bi), bn_conv_back(blk["c2"], g2))
        g1 = dz1 * masks[("z1", bi)]
        dx = bn_conv_back(blk["c1"], g1)
        dx = dx + (bn_conv_back(blk["ds"], g2) if blk["ds"] else g2)
        da = rb(("dx", bi), dx)
    if cfg.arch == "imagenet":
        da = rb(("da_pool", 0), ops.maxpool_backward(da, pool_arg, stem_out.shape))
    g0 = da * masks["stem"]
    bn_conv_back("stem", g0)
    if cfg.fp16:
        with np.errstate(invalid="ignore", over="ignore"):
            grad = grad / cfg.loss_scale
    return loss, logits, grad, run_stats


def train_step(cfg, layout, state, momentum_buf, images, labels, lr, decide=None):
    """Forward, backward, BN running-stat update and SGD-momentum update of
    every trainable parameter (conv W, gamma, beta, FC W and b; weight decay
    on all of them). Returns (new_state, new_momentum, loss, grad).

    fp16 configurations skip the parameter and momentum update when the
    gradient is not finite (the loss-scaled backward pass overflowed fp16);
    the BN running statistics of the forward pass are kept either way."""
    loss, logits, grad, run_stats = forward_backward(cfg, layout, state, images, labels, decide=decide)
    new_state = np.array(state, dtype=np.float64, copy=True)
    P = layout.n_trainable
    if cfg.fp16 and not np.all(np.isfinite(grad)):
        w_new, v_new = new_state[:P].copy(), np.array(momentum_buf, dtype=np.float64, copy=True)
    else:
        w_new, v_new = ops.sgd_momentum(new_state[:P], grad, momentum_buf, lr, cfg.momentum, cfg.weight_decay)
    new_state[:P] = w_new
    for name, rm, rv in run_stats:
        layout.put(new_state, name + ".rm", rm)
        layout.put(new_state, name + ".rv", rv)
    return new_state, v_new, loss, grad


def eval_logits(cfg, layout, state, images):
    """Forward pass with BN in running-statistics mode; returns [N, C] logits."""
    _, logits, _, _ = forward_backward(cfg, layout, state, images, None, train=False, need_grad=False)
    return logits


def loss_only(cfg, layout, state, images, labels):
    """Training-mode loss as a function of the state (for finite differences)."""
    _, logits, _, _ = forward_backward(cfg, layout, state, images, labels, need_grad=False)
    loss, _ = ops.softmax_ce(logits, labels)
    return loss
