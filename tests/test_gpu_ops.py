"""GPU parity of the single operators (through the C ABI of rn18_ops.h)
against the fp64 oracle on identical seeded inputs: every conv shape class
of the three networks in all three passes, fp32 and bf16, with ragged tile
tails; max pool bit-exact."""
import numpy as np
import pytest

from oracle import ops
from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import inputs
from gpu_util import PREC, assert_close, from_dev_nhwc, rounded, to_dev_nhwc

pytestmark = pytest.mark.gpu

# (N, Cin, Cin_padded, H, W, Cout, k, s, p)
CONV_CASES = [
    (3, 64, 64, 13, 11, 64, 3, 1, 1),      # 3x3 s1, M = 429 (ragged)
    (2, 64, 64, 15, 15, 128, 3, 2, 1),     # 3x3 s2 (first conv of a stage), odd input
    (2, 64, 64, 14, 14, 128, 1, 2, 0),     # 1x1 s2 projection
    (2, 128, 128, 9, 7, 128, 3, 1, 1),
    (1, 256, 256, 7, 7, 512, 3, 2, 1),     # stage 4 entry at 224/32
    (2, 512, 512, 4, 4, 512, 3, 1, 1),
    (3, 16, 16, 16, 16, 16, 3, 1, 1),      # tiny block
    (2, 3, 0, 23, 21, 64, 7, 2, 3),        # ImageNet stem, channels padded
    (4, 3, 0, 16, 16, 64, 3, 1, 1),        # CIFAR stem, channels padded
    (2, 3, 0, 10, 9, 16, 3, 1, 1),         # tiny stem
]


def case_id(c):
    return "N%d_C%d_%dx%d_O%d_k%ds%dp%d" % (c[0], c[1], c[3], c[4], c[5], c[6], c[7], c[8])


def _cp(c, prec):
    if c[2]:
        return c[2]
    return 8 if prec == "bf16" else 4


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("case", CONV_CASES, ids=case_id)
def test_conv_fwd(prec, case):
    import torch
    N, C, _, H, W, O, k, s, p = case
    cp = _cp(case, prec)
    x = inputs.tensor(11, (N, C, H, W))
    w = inputs.tensor(12, (O, C, k, k), scale=np.sqrt(2.0 / (C * k * k)))
    ref = ops.conv2d_forward(rounded(x, prec), rounded(w, prec), s, p)
    xd = to_dev_nhwc(x, prec, cp)
    wd = to_dev_nhwc(w, prec, cp)                       # [O][k][k][cp] = OHWI
    Ho, Wo = ref.shape[2:]
    y = torch.empty((N, Ho, Wo, O), dtype=xd.dtype, device="cuda")
    B.rn18op_conv2d_fwd(PREC[prec], xd, wd, y, N, H, W, cp, O, k, s, p)
    torch.cuda.synchronize()
    tol = 1e-5 if prec == "fp32" else 8e-3              # bf16: output rounded to 8 mantissa bits
    assert_close(from_dev_nhwc(y), ref, tol, "conv fwd")


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("case", [c for c in CONV_CASES if c[2]], ids=case_id)
def test_conv_dgrad(prec, case):
    import torch
    N, C, cp, H, W, O, k, s, p = case
    w = inputs.tensor(13, (O, C, k, k), scale=np.sqrt(2.0 / (C * k * k)))
    Ho, Wo = ops.conv_out_size(H, k, s, p), ops.conv_out_size(W, k, s, p)
    dy = inputs.tensor(14, (N, O, Ho, Wo))
    ref = ops.conv2d_backward_data(rounded(dy, prec), rounded(w, prec), (N, C, H, W), s, p)
    dyd = to_dev_nhwc(dy, prec)
    wt = to_dev_nhwc(np.ascontiguousarray(w.transpose(1, 0, 2, 3)), prec)   # [C][k][k][O] = IHWO
    dx = torch.empty((N, H, W, C), dtype=dyd.dtype, device="cuda")
    B.rn18op_conv2d_dgrad(PREC[prec], dyd, wt, dx, N, H, W, C, O, k, s, p)
    torch.cuda.synchronize()
    tol = 1e-5 if prec == "fp32" else 8e-3
    assert_close(from_dev_nhwc(dx), ref, tol, "conv dgrad")


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("case", CONV_CASES, ids=case_id)
def test_conv_wgrad(prec, case):
    import torch
    N, C, _, H, W, O, k, s, p = case
    cp = _cp(case, prec)
    x = inputs.tensor(15, (N, C, H, W))
    Ho, Wo = ops.conv_out_size(H, k, s, p), ops.conv_out_size(W, k, s, p)
    dy = inputs.tensor(16, (N, O, Ho, Wo))
    ref = ops.conv2d_backward_weight(rounded(dy, prec), rounded(x, prec), (O, C, k, k), s, p)
    xd = to_dev_nhwc(x, prec, cp)
    dyd = to_dev_nhwc(dy, prec)
    dw = torch.full((O, C, k, k), float("nan"), dtype=torch.float32, device="cuda")
    nws = B.rn18op_conv2d_wgrad_workspace(PREC[prec], N, H, W, cp, O, k, s, p)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    B.rn18op_conv2d_wgrad(PREC[prec], dyd, xd, dw, N, H, W, cp, C, O, k, s, p, ws)
    torch.cuda.synchronize()
    tol = 1e-5 if prec == "fp32" else 1e-5             # fp32 output, exact bf16 products
    assert_close(dw.cpu().numpy(), ref, tol, "conv wgrad")


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("case", [(6, 64, 64, 24, 24, 64, 3, 1, 1), (4, 64, 64, 17, 19, 128, 3, 2, 1),
                                  (5, 3, 0, 40, 40, 64, 7, 2, 3), (3, 128, 128, 9, 9, 256, 1, 2, 0)], ids=case_id)
def test_conv_wgrad_split_k(prec, case):
    """Pixel ranges long enough for several split-K partials."""
    test_conv_wgrad(prec, case)


@pytest.mark.parametrize("case", [(2, 64, 64, 56, 56, 64, 3, 1, 1), (3, 64, 64, 13, 11, 64, 3, 1, 1),
                                  (1, 64, 64, 40, 40, 64, 3, 1, 1), (4, 64, 64, 7, 7, 64, 3, 1, 1),
                                  (2, 64, 64, 9, 50, 64, 3, 1, 1)], ids=case_id)
def test_conv_wgrad_halo(case):
    """The halo weight-gradient kernel (64 -> 64 channel 3x3 stride-1 bf16
    shapes, picked automatically): row strips with a partial last strip,
    single-strip images and strips spread over many blocks."""
    test_conv_wgrad("bf16", case)


def test_conv_wgrad_deterministic():
    import torch
    N, C, H, W, O, k, s, p = 8, 64, 28, 28, 64, 3, 1, 1
    x = to_dev_nhwc(inputs.tensor(17, (N, C, H, W)), "bf16")
    dy = to_dev_nhwc(inputs.tensor(18, (N, O, H, W)), "bf16")
    nws = B.rn18op_conv2d_wgrad_workspace(B.RN18_BF16, N, H, W, C, O, k, s, p)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(2):
        dw = torch.empty((O, C, k, k), dtype=torch.float32, device="cuda")
        B.rn18op_conv2d_wgrad(B.RN18_BF16, dy, x, dw, N, H, W, C, C, O, k, s, p, ws)
        outs.append(dw.cpu())
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", [(2, 64, 14, 14), (3, 64, 9, 11), (1, 64, 112, 112), (2, 16, 2, 3)])
def test_maxpool_bit_exact(prec, shape):
    import torch
    N, C, H, W = shape
    x = inputs.tensor(19, shape)
    x[:, :, ::3, :] = np.round(x[:, :, ::3, :])         # plant ties
    x = np.maximum(x, 0.0)                              # post-ReLU input: many zero ties
    xr = rounded(x, prec)
    yref, aref = ops.maxpool_forward(xr)
    xd = to_dev_nhwc(x, prec)
    Ho, Wo = yref.shape[2:]
    y = torch.empty((N, Ho, Wo, C), dtype=xd.dtype, device="cuda")
    arg = torch.empty((N, Ho, Wo, C), dtype=torch.uint8, device="cuda")
    B.rn18op_maxpool_fwd(PREC[prec], xd, y, arg, N, H, W, C)
    dy = inputs.tensor(20, (N, C, Ho, Wo))
    dyd = to_dev_nhwc(dy, prec)
    dx = torch.empty((N, H, W, C), dtype=xd.dtype, device="cuda")
    B.rn18op_maxpool_bwd(PREC[prec], dyd, arg, dx, N, H, W, C)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev_nhwc(y), yref)
    np.testing.assert_array_equal(arg.cpu().numpy().transpose(0, 3, 1, 2), aref)
    dref = ops.maxpool_backward(rounded(dy, prec), aref, shape)
    tol = 1e-6 if prec == "fp32" else 8e-3
    assert_close(from_dev_nhwc(dx), dref, tol, "maxpool bwd")


def test_op_argument_errors():
    import torch
    x = torch.zeros(64, device="cuda")
    with pytest.raises(B.Rn18Error) as e:
        B.rn18op_conv2d_fwd(B.RN18_FP32, x, x, x, 1, 4, 4, 6, 4, 3, 1, 1)   # Cin not a multiple of 4
    assert e.value.code == B.RN18_EINVAL
    with pytest.raises(B.Rn18Error):
        B.rn18op_conv2d_fwd(B.RN18_FP32, x, x, x, 1, 2, 2, 4, 4, 7, 1, 0)   # empty output


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_conv_every_kernel_configuration(prec):
    """Every gather (forward / data-gradient) and weight-gradient kernel
    configuration, forced in turn, on a ragged stride-1 and a stride-2 shape."""
    cases = [(3, 64, 64, 13, 11, 128, 3, 1, 1), (2, 64, 64, 15, 15, 128, 3, 2, 1)]
    try:
        for cfg in range(1, 46):
            B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, cfg)
            for case in cases:
                test_conv_fwd(prec, case)
                test_conv_dgrad(prec, case)
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 0)
        for cfg in range(1, 11):
            B.rn18_debug_set(None, B.RN18_DBG_WGRAD_CONFIG, cfg)
            for case in cases:
                test_conv_wgrad(prec, case)
    finally:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 0)
        B.rn18_debug_set(None, B.RN18_DBG_WGRAD_CONFIG, 0)


@pytest.mark.parametrize("case", [(2, 64, 64, 56, 56, 64, 3, 1, 1), (3, 64, 64, 13, 11, 64, 3, 1, 1),
                                  (2, 64, 64, 28, 28, 64, 3, 1, 1), (1, 64, 64, 40, 40, 64, 3, 1, 1),
                                  (2, 64, 64, 9, 50, 64, 3, 1, 1)], ids=case_id)
def test_conv_halo(case):
    """The halo kernel (64 -> 64 channel 3x3 stride-1 convs in bf16, weights
    resident in LDS, one input patch per tile of whole output rows): forward
    and data gradient against the oracle, with one and several tiles per
    image and ragged widths."""
    try:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 45)
        test_conv_fwd("bf16", case)
        test_conv_dgrad("bf16", case)
    finally:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 0)


@pytest.mark.parametrize("case", [(2, 128, 128, 28, 28, 128, 3, 1, 1), (2, 256, 256, 14, 14, 256, 3, 1, 1),
                                  (3, 128, 128, 13, 11, 256, 3, 1, 1), (1, 192, 192, 20, 30, 128, 3, 1, 1),
                                  (2, 128, 128, 9, 50, 128, 3, 1, 1), (1, 512, 512, 12, 12, 128, 3, 1, 1)],
                         ids=case_id)
def test_conv_halo_wide(case):
    """The streamed-weight halo kernel (3x3 stride-1 bf16 convs with 128..512
    input channels and 128-column output tiles):
    forward and data gradient against the oracle, with one and two tiles per
    image, both pixel-wave depths, ragged widths, three and sixteen channel
    halves per block, and shapes whose data gradient falls back to the gather
    kernel (selected with the halo configuration)."""
    try:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 45)
        test_conv_fwd("bf16", case)
        test_conv_dgrad("bf16", case)
    finally:
        B.rn18_debug_set(None, B.RN18_DBG_GATHER_CONFIG, 0)


def test_bf16_storage_rounding_matches_oracle():
    """The kernels' fp32 -> bf16 storage rounding (hardware conversion) is
    bit-identical to the oracle's round-to-nearest-even on the binary32
    pattern: random values over the whole exponent range, exact ties (odd and
    even), values just around ties, signed zeros, subnormals, the bf16 overflow
    boundary and infinities."""
    import torch
    from oracle.ops import round_bf16
    rng = np.random.default_rng(7)
    bits = [rng.integers(0, 2 ** 32, 200000, dtype=np.uint64).astype(np.uint32)]
    hi = rng.integers(0, 2 ** 16, 20000, dtype=np.uint64).astype(np.uint32) << 16
    for low in (0x8000, 0x7FFF, 0x8001, 0x0000, 0xFFFF):
        bits.append(hi | low)
    bits.append(np.array([0, 0x80000000, 1, 0x807FFFFF, 0x7F7FFFFF, 0x7F7F8000, 0x7F7F7FFF, 0x7F800000, 0xFF800000,
                          0x00800000, 0x3F808000, 0x3F818000], dtype=np.uint32))
    u = np.concatenate(bits)
    u = u[(u & 0x7FFFFFFF) <= 0x7F800000]              # NaN payloads are not compared
    u = u[: len(u) // 8 * 8]
    x = u.view(np.float32)
    xd = torch.from_numpy(x.copy()).cuda()
    yd = torch.empty(len(x), dtype=torch.int16, device="cuda")
    B.rn18op_round_bf16(xd, yd, len(x))
    torch.cuda.synchronize()
    got = yd.cpu().numpy().view(np.uint16)
    ref = (round_bf16(x.astype(np.float64)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, "first mismatches: %s" % [(hex(int(u[i])), hex(int(got[i])), hex(int(ref[i])))
                                                    for i in bad[:5]]
