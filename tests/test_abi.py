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
