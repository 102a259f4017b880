"""The C-ABI library loads and exports every entry point that the public
header declares, and its host-only helpers answer without a GPU.

Runs on the CPU: no kernel is launched.  If the library has not been built
yet it is built first (hipcc cross-compiles for gfx950 without a GPU).
"""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))
DECL = re.compile(r"^\s*(?:const\s+char\s*\*|sp_status)\s*(sp_\w+)\s*\(", re.M)


def declared():
    names = []
    for h in HEADERS:
        names += DECL.findall(open(h).read())
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    from paper_2302_04852_amd import build as b
    if not os.path.exists(b.LIB):
        b.build()
    return ctypes.CDLL(b.LIB)


def test_header_declares_the_six_passes():
    names = declared()
    for op in ("sp_linear_fwd", "sp_linear_bwd_input", "sp_linear_bwd_weight",
               "sp_conv_fwd", "sp_conv_bwd_input", "sp_conv_bwd_weight"):
        assert op in names
    assert len(names) >= 25


def test_every_declared_symbol_is_exported(lib):
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, "declared but not exported: %s" % missing


def test_binding_names_match_header():
    import paper_2302_04852_amd as sp
    names = set(declared())
    assert set(sp.EXPORTED) == names
    for n in names:
        assert callable(getattr(sp, n)), n


def test_host_helpers_without_gpu(lib):
    lib.sp_status_string.restype = ctypes.c_char_p
    assert lib.sp_status_string(0) == b"ok"
    assert lib.sp_status_string(4) == b"workspace missing or too small"
    import paper_2302_04852_amd as sp
    s = sp.conv_shape(2, 3, 224, 224, 64, 7, 7, (2, 2), (3, 3))
    assert sp.sp_conv_out_hw(s) == (112, 112)
    s = sp.conv_shape(2, 64, 56, 56, 128, 1, 1, (2, 2), (0, 0))
    assert sp.sp_conv_out_hw(s) == (28, 28)
    with pytest.raises(sp.SparsePropError):
        sp.sp_conv_out_hw(sp.conv_shape(1, 1, 2, 2, 1, 3, 3, (1, 1), (0, 0)))
    assert sp.sp_linear_plan_bytes(768, 3072, 117965) > 0
    assert sp.sp_linear_bwd_weight_ws(8192, 768, 3072, 117965) > 0
    rp = np.array([0, 2, 3], np.int32)
    ci = np.array([0, 3, 1], np.int32)
    sp.sp_linear_validate(4, 2, rp, ci, 3)
    with pytest.raises(sp.SparsePropError):
        sp.sp_linear_validate(4, 2, rp, np.array([3, 0, 1], np.int32), 3)
