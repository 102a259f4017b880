"""CPU checks of bench.py's host logic: the one-GPU contract, the algorithmic
byte counts behind the HBM roofline, the roofline record and the rule that
decides which layers the dense/sparse choice times.  Nothing here touches a
GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120)


def test_more_than_one_gpu_exits_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_linear_alg_bytes_closed_form():
    B, i, o, nnz = 8192, 768, 3072, 117965
    # forward: X read, Y written, values and column indices, row pointers
    assert bench.linear_alg_bytes("fwd", B, i, o, nnz) == 4 * B * i + 4 * B * o + 8 * nnz + 4 * (o + 1)
    # both gradients in one pass: dY read once, X read, dX written, values read,
    # dW written, column indices, both pointer arrays
    assert bench.linear_alg_bytes("bwd", B, i, o, nnz) == (4 * B * o + 4 * B * i + 4 * B * i + 4 * nnz + 4 * nnz
                                                          + 4 * nnz + 4 * (i + 1) + 4 * (o + 1))
    # the FFN layer's forward moves the 126,785,132 bytes quoted for it
    assert bench.linear_alg_bytes("fwd", B, i, o, nnz) == 126_785_132


def test_conv_alg_bytes_closed_form():
    B, IC, H, W, OC, OH, OW, nnz = 32, 64, 56, 56, 64, 56, 56, 3686
    act = 4 * B * IC * H * W + 4 * B * OC * OH * OW
    assert bench.conv_alg_bytes(B, IC, H, W, OC, OH, OW, nnz) == act + 6 * nnz + 2 * OC * (IC + 1) + 4 * (OC + 1)
    assert bench.conv_bwd_alg_bytes(B, IC, H, W, OC, OH, OW, nnz) == (
        8 * B * IC * H * W + 4 * B * OC * OH * OW + 10 * nnz + 2 * OC * (IC + 1) + 4 * (OC + 1))


def test_bound_follows_the_ridge_point():
    ridge = bench.VALU_FP32_PEAK_TFLOPS * 1e12 / (bench.HBM_PEAK_GBS * 1e9)  # flop per byte
    assert bench.bound_of(ridge * 0.9 * 1e6, 1e6) == "hbm"
    assert bench.bound_of(ridge * 1.1 * 1e6, 1e6) == "alu"
    assert abs(bench.VALU_FP32_PEAK_TFLOPS - 78.6432) < 1e-3


@pytest.mark.parametrize("fl,by,ms,mfma,bound,unit", [
    (1.932738560e9, 126785132, 0.12, None, "alu", "TFLOP/s"),
    (1e6, 1e9, 0.5, None, "hbm", "GB/s"),
    (1.932738560e9, 126785132, 0.35, 3.865470566e10, "mfma", "TFLOP/s"),
])
def test_roofline_record(fl, by, ms, mfma, bound, unit):
    r = bench.roofline("k", "fwd", fl, by, ms, None, None, mfma)
    assert r["bound"] == bound and r["unit"] == unit
    if bound == "alu":
        assert r["achieved"] == pytest.approx(fl / (ms * 1e-3) / 1e12, rel=1e-3)
        assert r["peak"] == pytest.approx(bench.VALU_FP32_PEAK_TFLOPS, abs=0.05)
    elif bound == "hbm":
        assert r["achieved"] == pytest.approx(by / (ms * 1e-3) / 1e9, rel=1e-3)
        assert r["peak"] == bench.HBM_PEAK_GBS
    else:
        assert r["achieved"] == pytest.approx(mfma / (ms * 1e-3) / 1e12, rel=1e-3)
        assert r["peak"] == bench.MFMA_FP32_PEAK_TFLOPS
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], rel=1e-3)
    assert r["ms_per_launch"] == pytest.approx(ms)


def test_select_flags_time_layers_pruned_to_80_percent_or_more():
    class Lib:
        SP_SELECT_ALWAYS_TIME = 1
    assert bench.select_flags(Lib, 0.80) == 1
    assert bench.select_flags(Lib, 0.95) == 1
    assert bench.select_flags(Lib, 0.79) == 0
    assert bench.select_flags(Lib, 0.5) == 0
