"""The oracle's pins have teeth: plant plausible mistakes in a copy of the
oracle's C source (on the CPU), rebuild it, and check that at least one pin
fails for every planted mistake."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
from tests import test_oracle_conv as tc
from tests import test_oracle_linear as tl

SRC = os.path.join(os.path.dirname(oracle.__file__), "sparseprop_oracle.c")

# (function, old text, new text, what the mistake is)
MUTATIONS = [
    ("orc_linear_fwd", "X[t * in_f + col_idx[j]]", "X[t * in_f + (col_idx[j] + 1) % in_f]", "wrong column index"),
    ("orc_linear_fwd", "a += fabs(term);", "a += term;", "abssum without abs"),
    ("orc_linear_bwd_input", "dx[col_idx[j]] += term;", "dx[col_idx[j]] -= term;", "sign flip"),
    ("orc_linear_bwd_weight", "dY[t * out_f + i]", "dY[t * out_f + (out_f - 1 - i)]", "wrong gradient row"),
    ("orc_linear_bwd_weight", "for (int64_t t = 0; t < B; ++t)", "for (int64_t t = 1; t < B; ++t)", "dropped term"),
    ("orc_linear_transpose", "for (int64_t i = 0; i < out_f; ++i)", "for (int64_t i = out_f - 1; i >= 0; --i)", "unstable transpose"),
    ("orc_linear_encode", "col_idx[k] = (int32_t)c;", "col_idx[k] = (int32_t)(in_f - 1 - c);", "mirrored columns"),
    ("orc_conv_fwd", "q * s->stride_w + w_y[si] - s->pad_w", "q * s->stride_h + w_y[si] - s->pad_w", "stride h/w swapped"),
    ("orc_conv_fwd", "p * s->stride_h + w_x[si] - s->pad_h", "p * s->stride_h + w_x[si] + s->pad_h", "padding sign"),
    ("orc_conv_bwd_input", "p * s->stride_h + w_x[si] - s->pad_h", "p * s->stride_h + w_y[si] - s->pad_h", "tap x/y swapped"),
    ("orc_conv_bwd_weight", "for (int64_t b = 0; b < s->B; ++b)", "for (int64_t b = 1; b < s->B; ++b)", "dropped image"),
    ("orc_conv_bwd_weight", "(double)g[p * OW + q] * (double)xc[m * W + n]", "(double)g[p * OW + q] * (double)xc[m * W + (W - 1 - n)]", "mirrored input column"),
    ("orc_conv_encode", "w_x[k] = (uint8_t)x;", "w_x[k] = (uint8_t)(KH - 1 - x);", "flipped kernel rows"),
    ("orc_conv_transpose", "for (int64_t oc = 0; oc < OC; ++oc)", "for (int64_t oc = OC - 1; oc >= 0; --oc)", "unstable ic-major view"),
]


def _mutate(src, func, old, new):
    start = src.index(func + "(")
    end = src.index("\n}\n", start)
    body = src[start:end]
    assert old in body, (func, old)
    return src[:start] + body.replace(old, new, 1) + src[end:]


def _pins():
    o = oracle
    checks = [
        lambda: tl.test_encode_matches_row_major_nonzeros(o),
        lambda: tl.test_transpose_matches_scipy_csc(o, 7, 11, 0.3),
        lambda: tl.test_bruteforce_dense_fp64(o, 3, 5, 33, 0.5),
        lambda: tl.test_bruteforce_dense_fp64(o, 17, 33, 33, 0.1),
        lambda: tc.test_worked_example_encoding(o),
        lambda: tc.test_transpose_is_ic_major_stable(o),
        lambda: tc.test_against_torch_conv2d_fp64(o, 7, 6, 2, 3, 2, 1),
        lambda: tc.test_against_torch_conv2d_anisotropic(o, 2, 1, 1, 2),
    ]
    return checks


@pytest.mark.parametrize("func,old,new,what", MUTATIONS, ids=[m[3] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, func, old, new, what):
    src = open(SRC).read()
    mutated = _mutate(src, func, old, new)
    c_path = tmp_path / "mut.c"
    so_path = tmp_path / "libmut.so"
    c_path.write_text(mutated)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC",
                    str(c_path), "-o", str(so_path), "-lm"], check=True)
    lib = ctypes.CDLL(str(so_path))
    lib.orc_linear_encode.restype = ctypes.c_int64
    lib.orc_conv_encode.restype = ctypes.c_int64
    lib.orc_conv_out_hw.restype = ctypes.c_int
    lib.orc_num_threads.restype = ctypes.c_int
    saved = oracle._lib
    oracle._lib = lib
    failed = 0
    try:
        for check in _pins():
            try:
                check()
            except AssertionError:
                failed += 1
    finally:
        oracle._lib = saved
    assert failed > 0, "planted mistake not caught: " + what


def test_unmutated_oracle_passes_all_pins():
    for check in _pins():
        check()
