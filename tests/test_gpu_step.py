"""GPU parity of the whole training step (rn18_train_step through the C ABI)
against the fp64 oracle on the same seeded inputs and the same initial
state: loss, every parameter's gradient (read back as the momentum buffer
v = g + wd*w after one step from v = 0), every update and the BN running
statistics, per tensor at the training configurations' tolerance.

Full configuration sizes where the oracle finishes in seconds (the tiny
configuration, CIFAR batch 128 at 32x32); reduced batches (with ragged
tails) at every resolution the cyclic and hybrid schedules visit; and, at
the ImageNet batch-256 224x224 launch configuration itself, properties that
hold at any size (duplicated-batch invariance, lr = 0) plus per-sample
eval-mode logits checked against the oracle one image at a time."""
import resource
import time

import numpy as np
import pytest

from oracle import net
from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import inputs
from gpu_util import HALF, TAU, TOL, Decider, Mirror, compare_step, gpu_train_step, make_state

pytestmark = pytest.mark.gpu

LR = 0.1


def _run_parity(arch, classes, prec, N, H, seed, lr=LR, dropout=None, chunk=0, loss_scale=1024.0):
    """One step on both sides. The oracle takes the kernel's choice only at
    non-unique points inside the rounding band (ReLU kinks, pool ties and,
    for bf16, rounding midpoints of the stored tensors; see gpu_util), and
    every kernel decision outside the band must agree with the oracle's.
    dropout: (rate, seed, step) of the classifier-input dropout on both.
    chunk: launch every convolution over batch chunks of this many images.
    loss_scale: the loss scale of fp16 steps (a power of two), on both sides."""
    L, st = make_state(arch, classes, seed)
    x = inputs.images(seed, N, H, H)
    y = inputs.labels(seed, N, classes)
    w = B.Worker(arch, classes, prec)
    if chunk:
        B.rn18_debug_set(w.ctx, B.RN18_DBG_CONV_CHUNK, chunk)
    drop = {}
    if dropout is not None:
        B.rn18_set_dropout(w.ctx, *dropout)
        drop = dict(dropout=dropout[0], dropout_seed=dropout[1], dropout_step=dropout[2])
    bf = prec in HALF
    if prec == "fp16":
        B.rn18_set_loss_scale(w.ctx, loss_scale, 1 << 30)
        drop.update(fp16=True, loss_scale=loss_scale)
    dec = Mirror(w, L, N, H, prec, TAU) if bf else Decider(w, N, H, prec, TAU)
    gs, gv, losses, status = gpu_train_step(arch, classes, prec, st, x, y, lr, worker=w)
    assert status == B.RN18_OK
    cfg = net.Config(arch, classes, bf16=(prec == "bf16"), round_acts=bf, **drop)
    t0 = time.time()
    try:
        report, loss = compare_step(L, cfg, st, x, y, lr, gs, gv, losses[0], TOL[prec], decide=dec)
    finally:
        print("oracle step and comparison %.1f s, host peak RSS %.1f GB" %
              (time.time() - t0, resource.getrusage(resource.RUSAGE_SELF).ru_maxrss / 2 ** 20), flush=True)
        if bf:
            print("16-bit rounding band %d, kernel choices taken %d, invalid %d, outside %d %s" %
                  (dec.round_band, dec.round_taken, dec.round_invalid, dec.round_outside, dec.round_log[:4]))
        print("relu/pool band %d, taken %d, invalid %d, outside %d" % (dec.ambiguous, dec.taken, dec.invalid,
                                                                       dec.outside))
        w.close()
    worst = max(report.items(), key=lambda kv: kv[1][0])
    print("%s %s N=%d H=%d loss %.6f (oracle %.6f) worst %s norm-rel %.2e" %
          (arch, prec, N, H, losses[0], loss, worst[0], worst[1][0]))
    assert dec.outside == 0 and dec.invalid == 0
    if bf:
        assert dec.round_outside == 0 and dec.round_invalid == 0
    return report


def test_tiny_fp32_full_config():
    _run_parity("tiny", 10, "fp32", 8, 16, seed=100)


def test_tiny_fp32_ragged_batch():
    _run_parity("tiny", 10, "fp32", 5, 13, seed=101)


def test_cifar_fp32_b128_32_full_config():
    _run_parity("cifar", 100, "fp32", 128, 32, seed=102)


@pytest.mark.parametrize("N,H", [(8, 16), (6, 24), (5, 32)])
def test_cifar_fp32_cyclic_resolutions(N, H):
    _run_parity("cifar", 100, "fp32", N, H, seed=103 + H)


@pytest.mark.parametrize("N,H", [(4, 224), (3, 128), (2, 160), (2, 192), (8, 64)])
def test_imagenet_bf16_resolutions(N, H):
    _run_parity("imagenet", 1000, "bf16", N, H, seed=110 + H)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("N,H", [(512, 16), (256, 24)])
def test_cifar_fp32_cyclic_full_batch(N, H):
    """The cyclic schedule's first two stages at their full batch sizes
    (512 at 16x16, 256 at 24x24; the 128 at 32x32 stage is the full
    CIFAR configuration above)."""
    _run_parity("cifar", 100, "fp32", N, H, seed=160 + H)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("H", [128, 160, 192, 224])
def test_imagenet_bf16_small_worker_b64(H):
    """The hybrid schedule's small-batch worker (batch 64) at every
    resolution it visits. At batch 64 every persistent grid walks several
    tiles per block (the stage-1 halo conv needs 37 images at 224x224 for
    more than one row strip per block, the stem halo conv 10) and the
    weight-gradient split counts reach their caps."""
    _run_parity("imagenet", 1000, "bf16", 64, H, seed=170 + H)


@pytest.mark.timeout(900)
def test_imagenet_bf16_b256_224_full_step(capsys):
    """The headline configuration itself, batch 256 at 224x224 in bf16:
    the whole training step against the oracle, element by element, in the
    launch configuration the benchmark times. The oracle side takes about
    three minutes, so the comparison's progress lines (one per stored tensor)
    are printed as they come rather than captured."""
    with capsys.disabled():
        _run_parity("imagenet", 1000, "bf16", 256, 224, seed=175)


@pytest.mark.parametrize("arch,classes,prec,N,H,split", [("imagenet", 1000, "bf16", 3, 64, 3),
                                                         ("imagenet", 1000, "fp16", 2, 96, 5),
                                                         ("imagenet", 1000, "fp32", 3, 64, 7),
                                                         ("cifar", 100, "fp32", 6, 24, 2)])
def test_split_k_forced(arch, classes, prec, N, H, split):
    """Every forward and stride-1 data-gradient gather launch of the step
    with its K stages cut into `split` ranges (3, 5 and 7 leave ranges of
    unequal length), the partial tiles summed by the reduce pass, which also
    writes the forward launches' BN partials and applies the data
    gradients' masked-residual epilogue."""
    try:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_SPLIT, split)
        _run_parity(arch, classes, prec, N, H, seed=140 + split)
    finally:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_SPLIT, 0)


def test_imagenet_fp32_small():
    """All op types (7x7 s2 stem, max pool, projections) in fp32 at 1e-3."""
    _run_parity("imagenet", 1000, "fp32", 3, 64, seed=120)


@pytest.mark.parametrize("prec,N,H", [("fp32", 2, 65), ("bf16", 3, 63)])
def test_imagenet_odd_resolution(prec, N, H):
    """Odd image sizes: the stem runs as the plain 7x7 stride-2 conv (even
    sizes use its space-to-depth form)."""
    _run_parity("imagenet", 1000, prec, N, H, seed=121 + H)


@pytest.mark.parametrize("arch,classes,prec,N,H,chunk", [("tiny", 10, "fp32", 8, 16, 5), ("cifar", 100, "fp32", 8, 16, 3),
                                                         ("imagenet", 1000, "bf16", 5, 64, 2),
                                                         ("imagenet", 1000, "fp32", 3, 33, 1)])
def test_chunked_convolutions(arch, classes, prec, N, H, chunk):
    """Convolutions launched over batch chunks (as a step does when a tensor
    would pass the kernels' 32-bit byte offsets), forced small here: BN
    statistics entries, weight-gradient partials, residual and mask operands
    are cut at the chunk boundaries, including a shorter last chunk."""
    _run_parity(arch, classes, prec, N, H, seed=180 + N, chunk=chunk)


@pytest.mark.parametrize("arch,classes,prec,N,H", [("imagenet", 1000, "bf16", 16, 64), ("imagenet", 1000, "bf16", 64, 128),
                                                 ("cifar", 100, "fp32", 16, 32)])
def test_weight_gradients_on_side_stream_match_serial(arch, classes, prec, N, H):
    """The weight gradients run on a second stream beside the data-gradient
    chain; with profiling on, every launch stays on the caller's stream. Two
    steps from the same state, one each way, agree bit for bit. The batch-64
    128x128 case has BN applies long enough (10-20 us) that a weight
    gradient started before its dY buffer was complete would change bits."""
    L, st = make_state(arch, classes, 190)
    x = inputs.images(190, N, H, H)
    y = inputs.labels(190, N, classes)
    z = np.zeros(L.n_trainable)
    out = []
    for serial in (False, True):
        w = B.Worker(arch, classes, prec)
        try:
            B.rn18_profile_enable(w.ctx, serial)
            s1, v1, l1, status = gpu_train_step(arch, classes, prec, st, x, y, LR, steps=2, worker=w, momentum_in=z)
            assert status == B.RN18_OK
            out.append((s1, v1, l1))
        finally:
            w.close()
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])
    assert out[0][2] == out[1][2]


def test_two_steps_with_momentum():
    arch, classes, prec, N, H, seed = "tiny", 10, "fp32", 8, 16, 130
    L, st = make_state(arch, classes, seed)
    x = inputs.images(seed, N, H, H)
    y = inputs.labels(seed, N, classes)
    gs, gv, losses, _ = gpu_train_step(arch, classes, prec, st, x, y, LR, steps=2)
    cfg = net.Config(arch, classes)
    s1, v1, l1, _ = net.train_step(cfg, L, st, np.zeros(L.n_trainable), x, y, LR)
    s2, v2, l2, _ = net.train_step(cfg, L, s1, v1, x, y, LR)
    from gpu_util import assert_close
    assert abs(losses[1] - l2) <= 1e-3 * abs(l2)
    assert_close(gs, s2, 1e-3, "state after 2 steps")
    assert_close(gv, v2, 1e-3, "momentum after 2 steps")


@pytest.mark.parametrize("arch,classes,prec,N,H,p", [("tiny", 10, "fp32", 8, 16, 0.3), ("cifar", 100, "fp32", 4, 32, 0.1),
                                                     ("imagenet", 1000, "bf16", 3, 64, 0.2)])
def test_dropout_step(arch, classes, prec, N, H, p):
    """Classifier-input dropout (the paper's adaptive regularisation rates):
    the step against the oracle drawing the same Philox4x32-10 mask, with a
    64-bit key and a step counter above 2^32."""
    _run_parity(arch, classes, prec, N, H, seed=140 + H, dropout=(p, 0x0123456789ABCDEF, 2 ** 32 + 7))


def test_dropout_counter_advances_per_step():
    """Two steps draw the masks of steps t and t + 1; rate 0 leaves the step
    unchanged."""
    arch, classes, prec, N, H, seed = "tiny", 10, "fp32", 8, 16, 150
    L, st = make_state(arch, classes, seed)
    x = inputs.images(seed, N, H, H)
    y = inputs.labels(seed, N, classes)
    w = B.Worker(arch, classes, prec)
    try:
        B.rn18_set_dropout(w.ctx, 0.3, 77, 10)
        gs, gv, losses, _ = gpu_train_step(arch, classes, prec, st, x, y, LR, steps=2, worker=w)
    finally:
        w.close()
    v0 = np.zeros(L.n_trainable)
    s1, v1, _, _ = net.train_step(net.Config(arch, classes, dropout=0.3, dropout_seed=77, dropout_step=10),
                                  L, st, v0, x, y, LR)
    s2, v2, l2, _ = net.train_step(net.Config(arch, classes, dropout=0.3, dropout_seed=77, dropout_step=11),
                                   L, s1, v1, x, y, LR)
    from gpu_util import assert_close
    assert abs(losses[1] - l2) <= 1e-3 * abs(l2)
    assert_close(gs, s2, 1e-3, "state after 2 dropout steps")
    assert_close(gv, v2, 1e-3, "momentum after 2 dropout steps")
    w = B.Worker(arch, classes, prec)
    try:
        B.rn18_set_dropout(w.ctx, 0.0, 77, 10)
        g0, _, l0, _ = gpu_train_step(arch, classes, prec, st, x, y, LR, worker=w)
    finally:
        w.close()
    s_ref, _, l_ref, _ = net.train_step(net.Config(arch, classes), L, st, v0, x, y, LR)
    assert abs(l0[0] - l_ref) <= 1e-3 * abs(l_ref)
    assert_close(g0, s_ref, 1e-3, "state, dropout rate 0")


def test_dropout_rejects_bad_rates():
    w = B.Worker("tiny", 10, "fp32")
    try:
        for bad in (-0.1, 1.0, float("nan")):
            with pytest.raises(B.Rn18Error):
                B.rn18_set_dropout(w.ctx, bad, 1, 0)
    finally:
        w.close()


def test_eval_logits_parity():
    import torch
    for arch, classes, prec, N, H, seed in [("tiny", 10, "fp32", 8, 16, 140), ("cifar", 100, "fp32", 4, 32, 141),
                                            ("imagenet", 1000, "bf16", 2, 96, 142)]:
        L, st = make_state(arch, classes, seed)
        x = inputs.images(seed, N, H, H)
        w = B.Worker(arch, classes, prec)
        logits = torch.empty((N, classes), dtype=torch.float32, device="cuda")
        w.eval_logits(torch.from_numpy(st.astype(np.float32)).cuda(), torch.from_numpy(x).cuda(), logits)
        ref = net.eval_logits(net.Config(arch, classes, bf16=(prec == "bf16")), L, st, x)
        from gpu_util import assert_close
        assert_close(logits.cpu().numpy(), ref, 1e-3 if prec == "fp32" else 2e-2, arch + " eval logits")
        w.close()


def test_imagenet_bf16_b256_224_launch_config_properties():
    """At the ImageNet batch-256 224x224 launch configuration itself:
    (a) the step is bitwise deterministic; (b) sampled stem-conv outputs
    equal the oracle's conv of those images alone, rounded to bf16 (exact
    except inside the rounding band); (c) a batch of two copies of 128
    images has the same loss and the same stem BN statistics as the 128
    images alone; (d) eval-mode logits of sampled images match the oracle
    run on each image alone. (Full-step gradients at this size are checked
    against the oracle at reduced batch with the same kernels; bf16
    rounding differences are chaotic across two batch sizes, so no
    GPU-vs-GPU gradient comparison is made.)"""
    import torch
    from gpu_util import Mirror, assert_close, from_dev_nhwc
    from oracle import ops
    arch, classes, prec = "imagenet", 1000, "bf16"
    L, st = make_state(arch, classes, 150)
    x = inputs.images(150, 128, 224, 224)
    y = inputs.labels(150, 128, classes)
    xx = np.concatenate([x, x])
    yy = np.concatenate([y, y])
    z = np.zeros(L.n_trainable)
    w = B.Worker(arch, classes, prec)
    s256, v256, l256, st256 = gpu_train_step(arch, classes, prec, st, xx, yy, LR, worker=w, momentum_in=z)
    ystem = torch.empty((256, 112, 112, 64), dtype=torch.bfloat16, device="cuda")
    B.rn18_debug_copy(w.ctx, 256, 224, 224, "y", 0, ystem)
    mean256 = torch.empty(64, device="cuda")
    B.rn18_debug_copy(w.ctx, 256, 224, 224, "mean", 0, mean256)
    s256b, v256b, _, _ = gpu_train_step(arch, classes, prec, st, xx, yy, LR, worker=w, momentum_in=z)
    assert st256 == B.RN18_OK
    assert np.array_equal(v256, v256b) and np.array_equal(s256, s256b), "train step is not deterministic"
    # (b) sampled stem outputs, mirrored rounding check
    wst = ops.round_bf16(L.get(st, "stem.w"))
    for i in (0, 93, 255):
        exact = ops.conv2d_forward(ops.round_bf16(xx[i:i + 1]), wst, 2, 3)
        got = from_dev_nhwc(ystem[i:i + 1])
        b = ops.round_bf16(exact)
        mism = got != b
        assert mism.mean() < 1e-3, mism.mean()            # 1-ulp differences at rounding midpoints only
        assert_close(got, exact, 8e-3, "stem conv output of image %d" % i)
    # (c) duplicated batch
    s128, v128, l128, _ = gpu_train_step(arch, classes, prec, st, x, y, LR, worker=w, momentum_in=z)
    mean128 = torch.empty(64, device="cuda")
    B.rn18_debug_copy(w.ctx, 128, 224, 224, "mean", 0, mean128)
    assert abs(l256[0] - l128[0]) <= 1e-2 * abs(l128[0])
    assert_close(mean256.cpu().numpy(), mean128.cpu().numpy(), 1e-4, "stem BN mean, duplicated batch")
    # (d) eval-mode logits of sampled images, one by one against the oracle
    logits = torch.empty((256, classes), dtype=torch.float32, device="cuda")
    w.eval_logits(torch.from_numpy(st.astype(np.float32)).cuda(), torch.from_numpy(xx).cuda(), logits)
    lg = logits.cpu().numpy()
    cfg = net.Config(arch, classes, bf16=True)
    for i in (0, 77, 200):
        ref = net.eval_logits(cfg, L, st, xx[i:i + 1])
        assert_close(lg[i:i + 1], ref, 2e-2, "eval logits of image %d" % i)
    assert np.all(np.isfinite(v256))
    w.close()


def test_imagenet_bf16_first_chunked_batch_224():
    """Two copies of 664 images at 224x224: 1,328 stem outputs (1.6 MB each)
    pass the kernels' per-launch limit by one image, so the stem conv runs
    as a chunk of 1,327 images and one of 1; later layers still run whole.
    The step succeeds; stem-conv outputs of images at the start, middle and
    end of the batch (the last one alone in its chunk) equal the oracle's
    conv of those images; the loss and the stem BN mean equal those of the
    664 images alone; eval logits of the last image match the oracle run on
    it alone."""
    import torch
    from gpu_util import assert_close, from_dev_nhwc
    from oracle import ops
    arch, classes, prec, half = "imagenet", 1000, "bf16", 664
    N = 2 * half
    limit = (1 << 31) - (1 << 24)
    assert (N - 1) * 112 * 112 * 64 * 2 <= limit < N * 112 * 112 * 64 * 2
    L, st = make_state(arch, classes, 151)
    x = inputs.images(151, half, 224, 224)
    y = inputs.labels(151, half, classes)
    xx = np.concatenate([x, x])
    yy = np.concatenate([y, y])
    z = np.zeros(L.n_trainable)
    w = B.Worker(arch, classes, prec)
    try:
        print("chunked stem: N=%d at 224" % N, flush=True)
        sN, vN, lN, stN = gpu_train_step(arch, classes, prec, st, xx, yy, LR, worker=w, momentum_in=z)
        assert stN == B.RN18_OK and np.all(np.isfinite(vN))
        wst = ops.round_bf16(L.get(st, "stem.w"))
        yall = torch.empty((N, 112, 112, 64), dtype=torch.bfloat16, device="cuda")
        B.rn18_debug_copy(w.ctx, N, 224, 224, "y", 0, yall)
        for i in (0, half + 17, N - 1):
            exact = ops.conv2d_forward(ops.round_bf16(xx[i:i + 1]), wst, 2, 3)
            got = from_dev_nhwc(yall[i:i + 1])
            assert (got != ops.round_bf16(exact)).mean() < 1e-3
            assert_close(got, exact, 8e-3, "stem conv output of image %d" % i)
        del yall
        meanN = torch.empty(64, device="cuda")
        B.rn18_debug_copy(w.ctx, N, 224, 224, "mean", 0, meanN)
        sh, vh, lh, _ = gpu_train_step(arch, classes, prec, st, x, y, LR, worker=w, momentum_in=z)
        meanh = torch.empty(64, device="cuda")
        B.rn18_debug_copy(w.ctx, half, 224, 224, "mean", 0, meanh)
        assert abs(lN[0] - lh[0]) <= 1e-2 * abs(lh[0])
        assert_close(meanN.cpu().numpy(), meanh.cpu().numpy(), 1e-4, "stem BN mean, duplicated batch")
        logits = torch.empty((N, classes), dtype=torch.float32, device="cuda")
        w.eval_logits(torch.from_numpy(st.astype(np.float32)).cuda(), torch.from_numpy(xx).cuda(), logits)
        ref = net.eval_logits(net.Config(arch, classes, bf16=True), L, st, xx[N - 1:N])
        assert_close(logits[N - 1:N].cpu().numpy(), ref, 2e-2, "eval logits of the last image")
    finally:
        w.close()


def test_lr_zero_keeps_weights():
    arch, classes, prec, N, H, seed = "cifar", 100, "fp32", 4, 16, 160
    L, st = make_state(arch, classes, seed)
    x = inputs.images(seed, N, H, H)
    y = inputs.labels(seed, N, classes)
    gs, gv, _, _ = gpu_train_step(arch, classes, prec, st, x, y, 0.0)
    P = L.n_trainable
    assert np.array_equal(gs[:P], st[:P].astype(np.float32).astype(np.float64))


def test_bad_label_sets_sticky_error():
    arch, classes, prec, N, H, seed = "tiny", 10, "fp32", 4, 16, 170
    L, st = make_state(arch, classes, seed)
    x = inputs.images(seed, N, H, H)
    y = np.array([1, 2, 10, 3], np.int32)
    _, _, _, status = gpu_train_step(arch, classes, prec, st, x, y, LR)
    assert status == B.RN18_ELABEL


def test_host_side_errors():
    import torch
    w = B.Worker("tiny", 10, "fp32")
    st = torch.zeros(w.n_state, device="cuda")
    x = torch.zeros((1, 3, 1, 1), device="cuda")
    y = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.Rn18Error) as e:
        B.rn18_train_step(w.ctx, st, x, y, 1, 1, 1, 0.1)      # BN over a single value
    assert e.value.code == B.RN18_EINVAL
    with pytest.raises(B.Rn18Error):
        B.rn18_train_step(w.ctx, st, x, y, 0, 16, 16, 0.1)
    w.close()


def test_init_statistics():
    """rn18_init: He-normal fan-in weights (sample std within CLT bounds),
    gamma 1, beta 0, running var 1."""
    import torch
    cfg = B.make_config("cifar", 100)
    n, P = B.rn18_state_floats(cfg)
    st = torch.zeros(n, device="cuda")
    ctx = B.rn18_init(cfg, 5, st)
    B.rn18_destroy(ctx)
    s = st.cpu().numpy().astype(np.float64)
    L = net.Layout("cifar", 100)
    for name, cin, cout, k, _, _ in L.convs:
        w = L.get(s, name + ".w")
        sd = np.sqrt(2.0 / (cin * k * k))
        assert abs(w.mean()) < 5 * sd / np.sqrt(w.size)
        assert abs(w.std() / sd - 1) < 5 * np.sqrt(0.5 / w.size) + 1e-3
        assert np.all(L.get(s, name + ".g") == 1) and np.all(L.get(s, name + ".b") == 0)
        assert np.all(L.get(s, name + ".rv") == 1) and np.all(L.get(s, name + ".rm") == 0)
