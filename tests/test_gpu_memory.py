"""Sec. 5.3 on the device: the memory of training steps at the paper's eight
fitting batches (64..512) is linear in B (Eq. 9), the fitted model predicts
the measured memory of larger steps, and the library plans exactly the
shapes whose tensors stay inside the kernels' 32-bit byte offsets."""
import pytest

from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import memory as Mm

pytestmark = pytest.mark.gpu

LIMIT = 16 * ((1 << 31) - (1 << 24))   # whole-tensor bytes the kernels index (16-byte chunks, 32-bit)


def test_memory_model_predicts_larger_steps():
    import torch
    arch, classes, prec, H = "cifar", 100, "fp32", 32
    bs = [64, 128, 192, 256, 320, 384, 448, 512]
    ms = Mm.profile(B, torch, arch, classes, prec, H, bs)
    print("measured MB:", [round(m / 1e6, 1) for m in ms], flush=True)
    p, a = Mm.fit(bs, ms)
    assert a > 0 and p > 0
    # linear up to the split-K scratch, which the planner sizes per shape;
    # within the paper's 3.5% (CIFAR-100) at every fitting batch
    for b, m in zip(bs, ms):
        assert abs(m - Mm.predict(p, a, b)) <= 0.035 * m, (b, m)
    for b in (1024, 2048, 9000):                   # 9000: stage-1 convs in two launches
        used, status = Mm.measure_step(B, torch, arch, classes, prec, b, H)
        assert status == B.RN18_OK
        pred = Mm.predict(p, a, b)
        print("B=%d measured %.1f MB predicted %.1f MB" % (b, used / 1e6, pred / 1e6), flush=True)
        assert abs(pred - used) <= 0.035 * used     # the paper's 3.5% (CIFAR-100)


@pytest.mark.parametrize("arch,classes,prec,H,per_image", [
    ("imagenet", 1000, "bf16", 224, 112 * 112 * 64 * 2),    # stem conv output
    ("imagenet", 1000, "bf16", 128, 64 * 64 * 64 * 2),
    ("cifar", 100, "fp32", 32, 32 * 32 * 64 * 4),           # stem / stage-1 activations
    ("cifar", 100, "fp32", 16, 16 * 16 * 64 * 4),
])
def test_addressing_bound(arch, classes, prec, H, per_image):
    """The planner accepts a batch while its largest tensor stays inside the
    whole-tensor bound (convolutions are launched over batch chunks below
    the per-launch bound), and rejects the next one."""
    w = B.Worker(arch, classes, prec)
    try:
        nmax = LIMIT // per_image
        assert B.rn18_workspace_bytes(w.ctx, nmax, H, H) > 0
        assert B.rn18_workspace_bytes(w.ctx, nmax + 1, H, H) == 0
        assert "per-tensor limit" in B.rn18_last_error()
        assert Mm.addressing_max_batch(B, w.ctx, H, H) == nmax
    finally:
        w.close()
