"""GPU parity of the dense linear variant (matrix-core GEMMs over the
densified weight) and of the dense/sparse choice, against the CPU oracle.

The dense variant computes the same sums as the sparse passes (pruned
positions contribute exact zeros), so it is held to the same bar:
|gpu - oracle| <= 1e-5 * abssum elementwise, exact zeros where abssum == 0.
The densified weight itself is a copy and must be bit-exact.
"""
import sys

import numpy as np
import pytest

from synth import linear_layer
from tests.test_gpu_linear import GpuLayer, assert_parity

pytestmark = pytest.mark.gpu


def _say(msg):
    print("[gpu-dense] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2302_04852_amd as m
    return m


def _dense_all(sp, L, Xd, dYd):
    """Densify, then the three dense products; NaN-filled outputs so that an
    unwritten element fails."""
    import torch
    B = Xd.shape[0]
    Wd = torch.full((L.out_f, L.in_f), float("nan"), device="cuda")
    sp.sp_linear_densify(L.out_f, L.in_f, L.row_ptr, L.col_idx, L.vals, L.nnz, Wd)
    ws = torch.empty(max(sp.sp_linear_dense_ws(B, L.in_f, L.out_f), 1), dtype=torch.uint8, device="cuda")
    Y = torch.full((B, L.out_f), float("nan"), device="cuda")
    sp.sp_linear_dense_fwd(Xd, B, L.in_f, L.out_f, Wd, Y, ws)
    dX = torch.full((B, L.in_f), float("nan"), device="cuda")
    sp.sp_linear_dense_bwd_input(dYd, B, L.in_f, L.out_f, Wd, dX, ws)
    dW = torch.full((max(L.nnz, 1),), float("nan"), device="cuda")
    sp.sp_linear_dense_bwd_weight(dYd, Xd, B, L.in_f, L.out_f, L.row_ptr, L.col_idx, L.nnz, dW, ws)
    return Wd, Y, dX, dW[:L.nnz]


def _check(sp, orc, mask, W, X, dY, name):
    import torch
    _say("case %s: out=%d in=%d B=%d nnz=%d" % (name, mask.shape[0], mask.shape[1], X.shape[0], int(mask.sum())))
    L = GpuLayer(sp, orc, mask, W)
    Xd = torch.from_numpy(X).cuda()
    dYd = torch.from_numpy(dY).cuda()
    Wd, Y, dX, dW = _dense_all(sp, L, Xd, dYd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(Wd.cpu().numpy(), np.where(mask != 0, W, 0).astype(np.float32),
                                  err_msg=name + " densified weight")
    Yr, Ya = orc.linear_fwd(X, L.o_rp, L.o_ci, L.o_v, mask.shape[0])
    assert_parity(Y.cpu().numpy(), Yr, Ya, name + " dense fwd")
    dXr, dXa = orc.linear_bwd_input(dY, L.o_rp, L.o_ci, L.o_v, mask.shape[1])
    assert_parity(dX.cpu().numpy(), dXr, dXa, name + " dense bwd_input")
    dWr, dWa = orc.linear_bwd_weight(dY, X, L.o_rp, L.o_ci)
    assert_parity(dW.cpu().numpy(), dWr, dWa, name + " dense bwd_weight")
    return L, Xd, dYd, (Wd, Y, dX, dW)


def _layer(seed, out_f, in_f, B, density):
    rng = np.random.default_rng(seed)
    mask = (rng.random((out_f, in_f)) < density).astype(np.uint8)
    W = ((rng.standard_normal((out_f, in_f)) * 0.05).astype(np.float32) * mask).astype(np.float32)
    X = rng.standard_normal((B, in_f)).astype(np.float32)
    dY = rng.standard_normal((B, out_f)).astype(np.float32)
    return mask, W, X, dY


def test_dense_small_layer_seed0(sp, orc):
    d = linear_layer(0, 256, 256, 16, 0.90)
    _check(sp, orc, d["mask"], d["W"], d["X"], d["dY"], "256x256@90 B16")


@pytest.mark.parametrize("out_f,in_f,B,density", [
    (200, 300, 300, 0.1),     # ragged in every dimension, several tiles
    (129, 65, 257, 0.3),      # one row/column/token past a 128 tile
    (64, 33, 9, 0.5),         # in_f not a multiple of 4 (scalar loads)
    (5, 7, 3, 1.0),           # fully dense, tiny
    (1, 1, 1, 1.0),
    (300, 150, 100, 1.0),
    (70, 130, 513, 0.05),
    (384, 256, 1000, 0.5),    # half dense: the regime the dense variant is for
    (256, 130, 4099, 0.3),    # odd k for the weight gradient's token splits
    (1024, 2048, 16, 0.3),    # few output tiles: forward and input gradient split k and reduce
    (3000, 70, 40, 0.5),      # in_f not a multiple of 4, split input gradient
])
def test_dense_ragged_shapes(sp, orc, out_f, in_f, B, density):
    mask, W, X, dY = _layer(out_f * 7 + in_f * 3 + B, out_f, in_f, B, density)
    _check(sp, orc, mask, W, X, dY, "dense ragged %dx%d B%d d%.2f" % (out_f, in_f, B, density))


def test_dense_edge_patterns(sp, orc):
    rng = np.random.default_rng(5)
    out_f, in_f, B = 260, 190, 70
    mask = (rng.random((out_f, in_f)) < 0.3).astype(np.uint8)
    mask[7, :] = 1                 # all-dense row
    mask[9, :] = 0                 # empty row: exact zeros in Y
    mask[:, 11] = 0                # empty column: exact zeros in dX
    W = (rng.standard_normal((out_f, in_f)) * 0.05).astype(np.float32) * mask
    W[7, 3] = 0.0                  # stored zero
    X = rng.standard_normal((B, in_f)).astype(np.float32)
    dY = rng.standard_normal((B, out_f)).astype(np.float32)
    _, _, _, (_, Y, dX, _) = _check(sp, orc, mask, W.astype(np.float32), X, dY, "dense edge patterns")
    assert bool((Y[:, 9] == 0).all()) and bool((dX[:, 11] == 0).all())


@pytest.mark.parametrize("layer", [0, 1])
def test_dense_ffn_layer_full_size(sp, orc, layer):
    """The FFN layers at full size (8192 tokens, 768<->3072) at 80% sparsity,
    the threshold below which the dense variant is taken; every output is
    compared with the oracle."""
    out_f, in_f = (3072, 768) if layer == 0 else (768, 3072)
    d = linear_layer(2000 + layer, out_f, in_f, 8192, 0.80)
    _check(sp, orc, d["mask"], d["W"], d["X"], d["dY"], "ffn W%d @80 full" % (layer + 1))


def test_dense_empty_and_degenerate(sp, orc):
    import torch
    mask = np.zeros((40, 30), np.uint8)
    L = GpuLayer(sp, orc, mask, np.zeros((40, 30), np.float32))
    X = torch.randn(20, 30, device="cuda")
    dY = torch.randn(20, 40, device="cuda")
    Wd, Y, dX, dW = _dense_all(sp, L, X, dY)
    assert torch.all(Wd == 0) and torch.all(Y == 0) and torch.all(dX == 0) and dW.numel() == 0
    # no tokens: nothing to write; stored entries of dW become zeros
    d = linear_layer(4, 64, 48, 8, 0.5)
    L = GpuLayer(sp, orc, d["mask"], d["W"])
    e = torch.empty(0, 48, device="cuda")
    dW = torch.full((L.nnz,), float("nan"), device="cuda")
    sp.sp_linear_dense_bwd_weight(torch.empty(0, 64, device="cuda"), e, 0, 48, 64, L.row_ptr, L.col_idx, L.nnz,
                                  dW, None)
    Y = torch.empty(0, 64, device="cuda")
    Wd = torch.empty(64, 48, device="cuda")
    sp.sp_linear_densify(64, 48, L.row_ptr, L.col_idx, L.vals, L.nnz, Wd)
    sp.sp_linear_dense_fwd(e, 0, 48, 64, Wd, Y, None)
    torch.cuda.synchronize()
    assert torch.all(dW == 0)


def test_dense_deterministic(sp, orc):
    import torch
    mask, W, X, dY = _layer(9, 384, 256, 700, 0.4)
    L = GpuLayer(sp, orc, mask, W)
    Xd, dYd = torch.from_numpy(X).cuda(), torch.from_numpy(dY).cuda()
    a = _dense_all(sp, L, Xd, dYd)
    b = _dense_all(sp, L, Xd, dYd)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_dense_error_paths(sp, orc):
    import torch
    d = linear_layer(1, 32, 16, 8, 0.5)
    L = GpuLayer(sp, orc, d["mask"], d["W"])
    X = torch.from_numpy(d["X"]).cuda()
    dY = torch.from_numpy(d["dY"]).cuda()
    dW = torch.empty(L.nnz, device="cuda")
    small = torch.empty(4, dtype=torch.uint8, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_linear_dense_bwd_weight(dY, X, 8, 16, 32, L.row_ptr, L.col_idx, L.nnz, dW, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_linear_dense_fwd(X, 8, 16, 32, None, torch.empty(8, 32, device="cuda"), None)
    assert e.value.status == sp.SP_ERR_INVALID_ARG
    # a shape whose forward splits k needs the workspace
    assert sp.sp_linear_dense_ws(16, 2048, 1024) > 0
    Wd = torch.zeros(1024, 2048, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_linear_dense_fwd(torch.zeros(16, 2048, device="cuda"), 16, 2048, 1024, Wd,
                               torch.empty(16, 1024, device="cuda"), None)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_linear_densify(32, 16, L.row_ptr, L.col_idx, L.vals, 16 * 32 + 1, torch.empty(32, 16, device="cuda"))
    assert e.value.status == sp.SP_ERR_INVALID_ARG


def _select(sp, L, Xd, dYd, reps=2, flags=0):
    import torch
    B = Xd.shape[0]
    ws = torch.empty(max(sp.sp_linear_select_ws(B, L.in_f, L.out_f, L.nnz), 1), dtype=torch.uint8, device="cuda")
    Y = torch.full((B, L.out_f), float("nan"), device="cuda")
    dX = torch.full((B, L.in_f), float("nan"), device="cuda")
    dW = torch.full((max(L.nnz, 1),), float("nan"), device="cuda")
    v, ms = sp.sp_linear_select(Xd, dYd, B, L.in_f, L.out_f, L.row_ptr, L.col_idx, L.vals, L.nnz, L.plan, Y, dX,
                                dW, ws, reps, flags)
    return v, ms, Y, dX, dW[:L.nnz]


def test_select_below_80_percent_is_dense_untimed(sp, orc):
    import torch
    mask, W, X, dY = _layer(12, 256, 192, 300, 0.5)
    L = GpuLayer(sp, orc, mask, W)
    v, ms, Y, _, _ = _select(sp, L, torch.from_numpy(X).cuda(), torch.from_numpy(dY).cuda())
    assert v == sp.SP_VARIANT_DENSE and ms == [-1.0, -1.0]
    assert bool(torch.isnan(Y).all()), "nothing runs below 80% sparsity"
    # asked to time, it times both below 80% too, and the outputs are the layer's
    v, ms, Y, dX, dW = _select(sp, L, torch.from_numpy(X).cuda(), torch.from_numpy(dY).cuda(),
                               flags=sp.SP_SELECT_ALWAYS_TIME)
    assert ms[0] > 0 and ms[1] > 0 and v == (sp.SP_VARIANT_DENSE if ms[1] < ms[0] else sp.SP_VARIANT_SPARSE)
    torch.cuda.synchronize()
    Yr, Ya = orc.linear_fwd(X, L.o_rp, L.o_ci, L.o_v, 256)
    assert_parity(Y.cpu().numpy(), Yr, Ya, "always-time select fwd")


@pytest.mark.parametrize("out_f,in_f,B,density", [
    (3072, 768, 8192, 0.05),   # the FFN's first layer at 95%
    (512, 512, 256, 0.19),     # just above 80% sparsity: timed
])
def test_select_times_both_and_outputs_match(sp, orc, out_f, in_f, B, density):
    import torch
    d = linear_layer(3000 + out_f, out_f, in_f, B, 1.0 - density)
    L = GpuLayer(sp, orc, d["mask"], d["W"])
    v, ms, Y, dX, dW = _select(sp, L, torch.from_numpy(d["X"]).cuda(), torch.from_numpy(d["dY"]).cuda())
    _say("select %dx%d B%d density %.2f: variant %d, sparse %.3f ms, dense %.3f ms" % (out_f, in_f, B, density, v,
                                                                                       ms[0], ms[1]))
    assert ms[0] > 0 and ms[1] > 0
    assert v == (sp.SP_VARIANT_DENSE if ms[1] < ms[0] else sp.SP_VARIANT_SPARSE)
    torch.cuda.synchronize()
    Yr, Ya = orc.linear_fwd(d["X"], L.o_rp, L.o_ci, L.o_v, out_f)
    assert_parity(Y.cpu().numpy(), Yr, Ya, "select fwd")
    dXr, dXa = orc.linear_bwd_input(d["dY"], L.o_rp, L.o_ci, L.o_v, in_f)
    assert_parity(dX.cpu().numpy(), dXr, dXa, "select bwd_input")
    dWr, dWa = orc.linear_bwd_weight(d["dY"], d["X"], L.o_rp, L.o_ci)
    assert_parity(dW.cpu().numpy(), dWr, dWa, "select bwd_weight")
