"""The C-ABI library loads and exports every function the headers declare;
the flat-state size the library reports agrees with the oracle's own
layout. No GPU compute calls."""
import ctypes
import os
import re

import pytest

from oracle import net
from paper_2509_26092_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("rn18.h", "rn18_ops.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\**\s+\**([a-z_][a-z0-9_]*)\s*\(", src, re.M):
            names.add(m.group(1))
    return names


def test_headers_match_binding():
    assert declared_functions() == set(B.EXPORTED)


def test_library_exports_every_symbol():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("library not built")
    lib = ctypes.CDLL(B.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


@pytest.mark.parametrize("arch,classes", [("tiny", 10), ("cifar", 100), ("imagenet", 1000), ("cifar", 7)])
def test_state_size_matches_oracle_layout(arch, classes):
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("library not built")
    total, P = B.rn18_state_floats(B.make_config(arch, classes))
    L = net.Layout(arch, classes)
    assert (total, P) == (L.n_state, L.n_trainable)


def test_invalid_config_rejected():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("library not built")
    with pytest.raises(B.Rn18Error):
        B.rn18_state_floats(B.make_config(3, 10))


def test_operator_tensor_limit_is_checked_on_the_host():
    """4096 x 64 x 64 x 64 fp32 activations are 4 GiB: beyond the kernels'
    32-bit byte offsets, so the operator returns RN18_EINVAL before it
    touches a pointer or the device (fake, aligned pointers here)."""
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("library not built")
    f = B.lib().rn18op_conv2d_fwd
    fake = ctypes.c_void_p(1 << 20)
    r = f(B.RN18_FP32, fake, fake, fake, 4096, 64, 64, 64, 64, 3, 1, 1, None)
    assert r == B.RN18_EINVAL
    assert "per-tensor limit" in B.rn18_last_error()
    r = f(B.RN18_BF16, fake, fake, fake, 4096, 64, 64, 64, 64, 3, 1, 1, None)   # 2 GiB in bf16
    assert r == B.RN18_EINVAL


def test_process_wide_debug_keys_validate_on_the_host():
    """The process-wide tuning keys take no context and touch no device:
    out-of-range gather configurations, weight-gradient configurations and
    split-K counts are refused, in-range ones accepted, and 0 restores the
    automatic choice."""
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("library not built")
    for key, good, bad in ((B.RN18_DBG_GATHER_CONFIG, (1, 44, 45), (-1, 46)),
                           (B.RN18_DBG_WGRAD_CONFIG, (1, 10), (-1, 11)),
                           (B.RN18_DBG_GATHER_SPLIT, (1, 2, 7, 64), (-1, 65))):
        try:
            for v in good:
                B.rn18_debug_set(None, key, v)
            for v in bad:
                with pytest.raises(B.Rn18Error):
                    B.rn18_debug_set(None, key, v)
        finally:
            B.rn18_debug_set(None, key, 0)
    with pytest.raises(B.Rn18Error):              # per-context keys need a context
        B.rn18_debug_set(None, B.RN18_DBG_SERIAL, 1)
