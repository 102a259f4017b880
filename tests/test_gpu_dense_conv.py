"""GPU parity of the dense convolution variant (implicit-im2col GEMMs on the
matrix cores over the densified weight) and of the conv dense/sparse choice,
against the CPU oracle.

Same bar as the sparse passes: |gpu - oracle| <= 1e-5 * abssum elementwise,
exact zeros where abssum == 0 (pruned taps add exact zeros); the densified
weight is a copy and must be bit-exact.  At full size the forward and input
gradient are compared on sampled images, the weight gradient on every
stored entry over the whole batch.
"""
import sys

import numpy as np
import pytest

from synth import conv_layer
from tests.test_gpu_conv import SMALL, GpuConv, _layer, _oracle_shape, assert_parity

pytestmark = pytest.mark.gpu


def _say(msg):
    print("[gpu-dense-conv] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2302_04852_amd as m
    return m


def _dense_all(sp, L, Xd, dYd):
    import torch
    B, IC, H, Wd_, OC, KH, KW = L.dims[:7]
    Wd = torch.full((OC, IC, KH, KW), float("nan"), device="cuda")
    sp.sp_conv_densify(L.shape, L.w_oc, L.w_ic, L.w_x, L.w_y, L.w_vals, L.nnz, Wd)
    ws = torch.empty(sp.sp_conv_dense_ws(L.shape), dtype=torch.uint8, device="cuda")
    Y = torch.full((B, OC, L.OH, L.OW), float("nan"), device="cuda")
    sp.sp_conv_dense_fwd(Xd, L.shape, Wd, Y, ws)
    dX = torch.full((B, IC, H, Wd_), float("nan"), device="cuda")
    sp.sp_conv_dense_bwd_input(dYd, L.shape, Wd, dX, ws)
    dW = torch.full((max(L.nnz, 1),), float("nan"), device="cuda")
    sp.sp_conv_dense_bwd_weight(dYd, Xd, L.shape, L.w_oc, L.w_ic, L.w_x, L.w_y, L.nnz, dW, ws)
    return Wd, Y, dX, dW[:L.nnz]


def _check(sp, orc, d, dims, name, sample_images=None):
    import torch
    B, IC, H, Wd_, OC, KH, KW, stride, pad = dims
    _say("case %s: B=%d IC=%d %dx%d OC=%d k%dx%d s%s p%s nnz=%d" % (
        name, B, IC, H, Wd_, OC, KH, KW, stride, pad, int(d["mask"].sum())))
    L = GpuConv(sp, orc, d["mask"], d["W"], B, H, Wd_, stride, pad)
    Xd = torch.from_numpy(d["X"]).cuda()
    dYd = torch.from_numpy(d["dY"]).cuda()
    Wd, Y, dX, dW = _dense_all(sp, L, Xd, dYd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(Wd.cpu().numpy(), np.where(d["mask"] != 0, d["W"], 0).astype(np.float32),
                                  err_msg=name + " densified weight")
    o_oc, o_ic, o_x, o_y, o_v = L.o
    imgs = list(range(B)) if sample_images is None else sorted(set(i % B for i in sample_images))
    so = _oracle_shape(orc, dims, B=len(imgs))
    Xs = np.ascontiguousarray(d["X"][imgs])
    dYs = np.ascontiguousarray(d["dY"][imgs])
    Yr, Ya = orc.conv_fwd(Xs, so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(Y.cpu().numpy()[imgs], Yr, Ya, name + " dense fwd")
    dXr, dXa = orc.conv_bwd_input(dYs, so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(dX.cpu().numpy()[imgs], dXr, dXa, name + " dense bwd_input")
    dWr, dWa = orc.conv_bwd_weight(d["dY"], d["X"], L.oshape, o_oc, o_ic, o_x, o_y)
    assert_parity(dW.cpu().numpy(), dWr, dWa, name + " dense bwd_weight")
    return L, Xd, dYd, (Wd, Y, dX, dW)


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_dense_conv_small_shapes(sp, orc, case):
    """Every small shape of the sparse tests: strides 1-3, anisotropic kernels,
    strides and padding, 1x1 and 7x7, dense and near-empty patterns."""
    B, IC, H, Wd, OC, KH, KW, stride, pad, s = SMALL[case]
    d, dims = _layer(orc, 9000 + case, B, IC, H, Wd, OC, KH, KW, stride, pad, s)
    _check(sp, orc, d, dims, "dense small%d" % case)


def test_dense_conv_many_tiles_ragged(sp, orc):
    """Token tiles spanning image boundaries, a ragged last tile, 100 output
    channels (one 128-row tile, partly empty)."""
    d, dims = _layer(orc, 9100, 5, 21, 31, 29, 100, 3, 3, (1, 1), (1, 1), 0.5)
    _check(sp, orc, d, dims, "dense ragged 5x21x31x29->100")


@pytest.mark.parametrize("spec", [
    # B, IC, H, W, OC, KH, KW, stride, pad, sparsity, sampled images
    (32, 64, 56, 56, 64, 3, 3, (1, 1), (1, 1), 0.8, [0, 13, 31]),     # the 3x3 64@56 layer at 80%
    (32, 256, 14, 14, 256, 3, 3, (1, 1), (1, 1), 0.8, [0, 17, 31]),   # sweep 256@14 at 80%
    (64, 128, 28, 28, 256, 3, 3, (2, 2), (1, 1), 0.5, [0, 29, 63]),   # ResNet-18 layer3.0.conv1 shape, 50%
    (64, 3, 224, 224, 64, 7, 7, (2, 2), (3, 3), 0.5, [0, 63]),        # the stem at 50%
    (64, 512, 7, 7, 512, 3, 3, (1, 1), (1, 1), 0.5, [0, 63]),         # 7x7 planes: split k, reduce to planes
    (32, 256, 14, 14, 1024, 1, 1, (1, 1), (0, 0), 0.8, [0, 31]),      # the sweep's 1x1 at 80%
])
def test_dense_conv_full_size(sp, orc, spec):
    B, IC, H, Wd, OC, KH, KW, stride, pad, s, imgs = spec
    d, dims = _layer(orc, 9200 + IC + OC, B, IC, H, Wd, OC, KH, KW, stride, pad, s)
    _check(sp, orc, d, dims, "dense full %dx%d@%d k%d s%d @%g" % (IC, OC, H, KH, stride[0], s),
           sample_images=imgs)


def test_dense_conv_empty_and_degenerate(sp, orc):
    import torch
    mask = np.zeros((6, 4, 3, 3), np.uint8)
    L = GpuConv(sp, orc, mask, np.zeros(mask.shape, np.float32), 2, 7, 7, (1, 1), (1, 1))
    X = torch.randn(2, 4, 7, 7, device="cuda")
    dY = torch.randn(2, 6, L.OH, L.OW, device="cuda")
    Wd, Y, dX, dW = _dense_all(sp, L, X, dY)
    assert torch.all(Wd == 0) and torch.all(Y == 0) and torch.all(dX == 0) and dW.numel() == 0
    # no images: nothing to write; stored entries of dW become zeros
    d, dims = _layer(orc, 9300, 2, 5, 6, 6, 7, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], 2, 6, 6, (1, 1), (1, 1))
    s0 = sp.conv_shape(0, 5, 6, 6, 7, 3, 3, (1, 1), (1, 1))
    dW = torch.full((L.nnz,), float("nan"), device="cuda")
    sp.sp_conv_dense_bwd_weight(None, None, s0, L.w_oc, L.w_ic, L.w_x, L.w_y, L.nnz, dW, None)
    Wd = torch.empty(7, 5, 3, 3, device="cuda")
    sp.sp_conv_densify(s0, L.w_oc, L.w_ic, L.w_x, L.w_y, L.w_vals, L.nnz, Wd)
    sp.sp_conv_dense_fwd(None, s0, Wd, None, None)
    torch.cuda.synchronize()
    assert torch.all(dW == 0)


def test_dense_conv_deterministic(sp, orc):
    import torch
    d, dims = _layer(orc, 9400, 4, 24, 17, 15, 40, 3, 3, (2, 2), (1, 1), 0.4)
    L = GpuConv(sp, orc, d["mask"], d["W"], 4, 17, 15, (2, 2), (1, 1))
    Xd, dYd = torch.from_numpy(d["X"]).cuda(), torch.from_numpy(d["dY"]).cuda()
    a = _dense_all(sp, L, Xd, dYd)
    b = _dense_all(sp, L, Xd, dYd)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_dense_conv_error_paths(sp, orc):
    import torch
    d, dims = _layer(orc, 9500, 2, 4, 6, 6, 5, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], 2, 6, 6, (1, 1), (1, 1))
    X = torch.from_numpy(d["X"]).cuda()
    dY = torch.from_numpy(d["dY"]).cuda()
    Wd = torch.zeros(5, 4, 3, 3, device="cuda")
    small = torch.empty(4, dtype=torch.uint8, device="cuda")
    dX = torch.empty(2, 4, 6, 6, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_dense_bwd_input(dY, L.shape, Wd, dX, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    dW = torch.empty(L.nnz, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_dense_bwd_weight(dY, X, L.shape, L.w_oc, L.w_ic, L.w_x, L.w_y, L.nnz, dW, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_dense_fwd(X, L.shape, None, torch.empty(2, 5, 6, 6, device="cuda"), None)
    assert e.value.status == sp.SP_ERR_INVALID_ARG


def _select(sp, L, Xd, dYd, reps=2):
    import torch
    B, IC, H, Wd_, OC = L.dims[:5]
    ws = torch.empty(max(sp.sp_conv_select_ws(L.shape, L.nnz), 1), dtype=torch.uint8, device="cuda")
    Y = torch.full((B, OC, L.OH, L.OW), float("nan"), device="cuda")
    dX = torch.full((B, IC, H, Wd_), float("nan"), device="cuda")
    dW = torch.full((max(L.nnz, 1),), float("nan"), device="cuda")
    v, ms = sp.sp_conv_select(Xd, dYd, L.shape, L.w_oc, L.w_ic, L.w_x, L.w_y, L.w_vals, L.nnz, L.plan, Y, dX, dW,
                              ws, reps)
    return v, ms, Y, dX, dW[:L.nnz]


def test_conv_select_below_80_percent_is_dense_untimed(sp, orc):
    import torch
    d, dims = _layer(orc, 9600, 2, 16, 10, 10, 24, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], 2, 10, 10, (1, 1), (1, 1))
    v, ms, Y, _, _ = _select(sp, L, torch.from_numpy(d["X"]).cuda(), torch.from_numpy(d["dY"]).cuda())
    assert v == sp.SP_VARIANT_SPARSE or v == sp.SP_VARIANT_DENSE
    assert ms[0] > 0 and ms[1] > 0, "fewer than 32 input channels: timed at every sparsity"
    d, dims = _layer(orc, 9601, 2, 40, 10, 10, 24, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], 2, 10, 10, (1, 1), (1, 1))
    v, ms, Y, _, _ = _select(sp, L, torch.from_numpy(d["X"]).cuda(), torch.from_numpy(d["dY"]).cuda())
    assert v == sp.SP_VARIANT_DENSE and ms == [-1.0, -1.0]
    assert bool(torch.isnan(Y).all()), "nothing runs below 80% sparsity"


@pytest.mark.parametrize("spec", [
    (32, 256, 14, 14, 256, 3, 3, (1, 1), (1, 1), 0.81),
    (32, 64, 56, 56, 64, 3, 3, (1, 1), (1, 1), 0.95),
])
def test_conv_select_times_both_and_outputs_match(sp, orc, spec):
    import torch
    B, IC, H, Wd, OC, KH, KW, stride, pad, s = spec
    d, dims = _layer(orc, 9700 + IC, B, IC, H, Wd, OC, KH, KW, stride, pad, s)
    L = GpuConv(sp, orc, d["mask"], d["W"], B, H, Wd, stride, pad)
    v, ms, Y, dX, dW = _select(sp, L, torch.from_numpy(d["X"]).cuda(), torch.from_numpy(d["dY"]).cuda())
    _say("select %d->%d @%dx%d sparsity %.2f: variant %d, sparse %.3f ms, dense %.3f ms" % (IC, OC, H, Wd, s, v,
                                                                                         ms[0], ms[1]))
    assert ms[0] > 0 and ms[1] > 0
    assert v == (sp.SP_VARIANT_DENSE if ms[1] < ms[0] else sp.SP_VARIANT_SPARSE)
    torch.cuda.synchronize()
    o_oc, o_ic, o_x, o_y, o_v = L.o
    imgs = [0, B - 1]
    so = _oracle_shape(orc, dims, B=len(imgs))
    Yr, Ya = orc.conv_fwd(np.ascontiguousarray(d["X"][imgs]), so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(Y.cpu().numpy()[imgs], Yr, Ya, "select fwd")
    dXr, dXa = orc.conv_bwd_input(np.ascontiguousarray(d["dY"][imgs]), so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(dX.cpu().numpy()[imgs], dXr, dXa, "select bwd_input")
    dWr, dWa = orc.conv_bwd_weight(d["dY"], d["X"], L.oshape, o_oc, o_ic, o_x, o_y)
    assert_parity(dW.cpu().numpy(), dWr, dWa, "select bwd_weight")
