"""GPU parity of the sparse convolution passes against the CPU oracle.

Structure outputs (the five-array encoding, the input-channel-major view)
must be bit-exact; values must satisfy |gpu - oracle| <= 1e-5 * abssum
elementwise, with exact zeros where no stored weight contributes
(abssum == 0, e.g. dX pixels that no tap reaches under a stride).
At full size the forward and input-gradient outputs are compared on sampled
images (each image's outputs depend on that image alone), the weight
gradient on every stored entry over the whole batch.
"""
import json
import os
import sys

import numpy as np
import pytest

from synth import CONV_3X3_56, conv_layer, conv_sweep, resnet18_convs, seed_for

pytestmark = pytest.mark.gpu

TOL = 1e-5
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "conv_format_example.json")


def _say(msg):
    print("[gpu-conv] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2302_04852_amd as m
    return m


def assert_parity(gpu, ref, abssum, what):
    gpu = np.asarray(gpu, np.float64)
    assert gpu.shape == ref.shape, what
    err = np.abs(gpu - ref)
    bound = TOL * abssum
    zero = abssum == 0
    assert np.all(gpu[zero] == 0), what + ": nonzero output where no term contributes"
    bad = err > bound
    assert not bad.any(), "%s: %d violations, worst excess %g" % (what, int(bad.sum()), float((err - bound).max()))


class GpuConv:
    """Product-side structure of one sparse convolution: encode the dense
    pattern on the GPU, check the encoding against the oracle's, plan."""

    def __init__(self, sp, orc, mask, W, B, H, Wd, stride, pad):
        import torch
        self.sp = sp
        OC, IC, KH, KW = mask.shape
        self.dims = (B, IC, H, Wd, OC, KH, KW, stride, pad)
        self.shape = sp.conv_shape(B, IC, H, Wd, OC, KH, KW, stride, pad)
        self.oshape = orc.conv_shape(B, IC, H, Wd, OC, KH, KW, stride, pad)
        self.OH, self.OW = sp.sp_conv_out_hw(self.shape)
        assert (self.OH, self.OW) == orc.conv_out_hw(self.oshape)
        dev = torch.device("cuda")
        m = torch.from_numpy(np.ascontiguousarray(mask)).to(dev)
        w = torch.from_numpy(np.ascontiguousarray(W)).to(dev)
        self.w_oc = torch.empty(OC + 1, dtype=torch.int32, device=dev)
        self.w_ic = torch.empty(OC * (IC + 1), dtype=torch.int16, device=dev)
        sp.sp_conv_encode_rows(OC, IC, KH, KW, m, self.w_oc, self.w_ic)
        nnz = int(self.w_oc[-1].item())
        self.nnz = nnz
        n1 = max(nnz, 1)
        self.w_x = torch.empty(n1, dtype=torch.uint8, device=dev)
        self.w_y = torch.empty(n1, dtype=torch.uint8, device=dev)
        self.w_vals = torch.empty(n1, dtype=torch.float32, device=dev)
        sp.sp_conv_encode_fill(OC, IC, KH, KW, m, w, self.w_oc, self.w_ic, self.w_x, self.w_y, self.w_vals)
        self.o = orc.conv_encode(mask, W)
        o_oc, o_ic, o_x, o_y, o_v = self.o
        np.testing.assert_array_equal(self.w_oc.cpu().numpy(), o_oc)
        np.testing.assert_array_equal(self.w_ic.cpu().numpy(), o_ic)
        np.testing.assert_array_equal(self.w_x.cpu().numpy()[:nnz], o_x)
        np.testing.assert_array_equal(self.w_y.cpu().numpy()[:nnz], o_y)
        np.testing.assert_array_equal(self.w_vals.cpu().numpy()[:nnz], o_v)
        self.plan = torch.empty(sp.sp_conv_plan_bytes(self.shape, nnz), dtype=torch.uint8, device=dev)
        sp.sp_conv_plan(self.shape, self.w_oc, self.w_ic, self.w_x, self.w_y, nnz, self.plan)

    def fwd(self, X):
        import torch
        B, IC, H, Wd, OC = self.dims[:5]
        Y = torch.full((B, OC, self.OH, self.OW), float("nan"), device="cuda")
        self.sp.sp_conv_fwd(X, self.shape, self.w_vals, self.nnz, self.plan, Y)
        return Y

    def bwd_input(self, dY):
        import torch
        B, IC, H, Wd = self.dims[:4]
        dX = torch.full((B, IC, H, Wd), float("nan"), device="cuda")
        self.sp.sp_conv_bwd_input(dY, self.shape, self.w_vals, self.nnz, self.plan, dX)
        return dX

    def bwd_weight(self, dY, X):
        import torch
        ws = torch.empty(max(self.sp.sp_conv_bwd_weight_ws(self.shape, self.nnz), 1), dtype=torch.uint8,
                         device="cuda")
        dW = torch.full((max(self.nnz, 1),), float("nan"), device="cuda")
        self.sp.sp_conv_bwd_weight(dY, X, self.shape, self.nnz, self.plan, dW, ws)
        return dW[:self.nnz]


    def bwd(self, dY, X):
        """Both gradients from sp_conv_bwd."""
        import torch
        B, IC, H, Wd = self.dims[:4]
        ws = torch.empty(max(self.sp.sp_conv_bwd_weight_ws(self.shape, self.nnz), 1), dtype=torch.uint8,
                         device="cuda")
        dX = torch.full((B, IC, H, Wd), float("nan"), device="cuda")
        dW = torch.full((max(self.nnz, 1),), float("nan"), device="cuda")
        self.sp.sp_conv_bwd(dY, X, self.shape, self.w_vals, self.nnz, self.plan, dX, dW, ws)
        return dX, dW[:self.nnz]


def _oracle_shape(orc, dims, B=None):
    b, IC, H, Wd, OC, KH, KW, stride, pad = dims
    return orc.conv_shape(b if B is None else B, IC, H, Wd, OC, KH, KW, stride, pad)


def _run_all(sp, orc, d, dims, name, sample_images=None):
    """All three passes on the GPU over the full batch; the oracle over the
    whole batch, or over the listed images for the per-image passes."""
    import torch
    B, IC, H, Wd, OC, KH, KW, stride, pad = dims
    _say("case %s: B=%d IC=%d %dx%d OC=%d k%dx%d s%s p%s nnz=%d" % (
        name, B, IC, H, Wd, OC, KH, KW, stride, pad, int(d["mask"].sum())))
    L = GpuConv(sp, orc, d["mask"], d["W"], B, H, Wd, stride, pad)
    Xd = torch.from_numpy(d["X"]).cuda()
    dYd = torch.from_numpy(d["dY"]).cuda()
    Y = L.fwd(Xd)
    dX = L.bwd_input(dYd)
    dW = L.bwd_weight(dYd, Xd)
    torch.cuda.synchronize()
    o_oc, o_ic, o_x, o_y, o_v = L.o
    imgs = list(range(B)) if sample_images is None else sorted(set(i % B for i in sample_images))
    so = _oracle_shape(orc, dims, B=len(imgs))
    Xs = np.ascontiguousarray(d["X"][imgs])
    dYs = np.ascontiguousarray(d["dY"][imgs])
    Yr, Ya = orc.conv_fwd(Xs, so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(Y.cpu().numpy()[imgs], Yr, Ya, name + " fwd")
    dXr, dXa = orc.conv_bwd_input(dYs, so, o_oc, o_ic, o_x, o_y, o_v)
    assert_parity(dX.cpu().numpy()[imgs], dXr, dXa, name + " bwd_input")
    dWr, dWa = orc.conv_bwd_weight(d["dY"], d["X"], L.oshape, o_oc, o_ic, o_x, o_y)
    assert_parity(dW.cpu().numpy(), dWr, dWa, name + " bwd_weight")
    # both gradients in one call: the same kernels and splits, so the same bits
    dXf, dWf = L.bwd(dYd, Xd)
    torch.cuda.synchronize()
    assert torch.equal(dXf, dX), name + " sp_conv_bwd dX differs from sp_conv_bwd_input"
    assert torch.equal(dWf, dW), name + " sp_conv_bwd dW differs from sp_conv_bwd_weight"
    return L, Y, dX, dW


def _layer(orc, seed, B, IC, H, Wd, OC, KH, KW, stride, pad, sparsity):
    dims = (B, IC, H, Wd, OC, KH, KW, stride, pad)
    oh, ow = orc.conv_out_hw(_oracle_shape(orc, dims))
    return conv_layer(seed, B, IC, H, Wd, OC, KH, KW, (oh, ow), sparsity), dims


def test_worked_example_encoding(sp, orc):
    """The format's worked example (Sec. 3.3): the GPU encoder reproduces the
    printed index arrays and the storage-order values."""
    import torch
    g = json.load(open(GOLDEN))
    OC, IC, KH, KW = g["shape"]
    mask = np.zeros((OC, IC, KH, KW), np.uint8)
    W = np.zeros((OC, IC, KH, KW), np.float32)
    for oc, ic, x, y, lab in g["entries_oc_ic_x_y_label"]:
        mask[oc, ic, x, y] = 1
        W[oc, ic, x, y] = g["labels_to_values"][lab]
    L = GpuConv(sp, orc, mask, W, 1, 4, 4, (1, 1), (0, 0))
    e = g["expected_printed"]
    assert L.w_oc.cpu().tolist() == e["W_oc"]
    assert L.w_ic.cpu().tolist() == e["W_ic"]
    assert L.w_x.cpu().tolist() == e["W_x"]
    assert L.w_y.cpu().tolist() == e["W_y"]
    want = [g["labels_to_values"][k] for k in g["expected_value_labels_storage_order"]]
    assert L.w_vals.cpu().tolist() == want
    t = [torch.empty(n, dtype=torch.int32, device="cuda") for n in (IC + 1, L.nnz, L.nnz)]
    sp.sp_conv_transpose(OC, IC, L.w_oc, L.w_ic, L.nnz, *t)
    r = orc.conv_transpose(OC, IC, *L.o[:2])
    for a, b in zip(t, r):
        np.testing.assert_array_equal(a.cpu().numpy(), b)


@pytest.mark.parametrize("OC,IC,KH,KW,density", [
    (37, 19, 3, 3, 0.1), (5, 3, 7, 7, 0.3), (130, 70, 1, 1, 0.2), (9, 40, 2, 3, 0.5), (16, 8, 3, 3, 0.0),
    (64, 300, 3, 3, 1.0),
])
def test_encode_and_transpose_bit_exact(sp, orc, OC, IC, KH, KW, density):
    import torch
    rng = np.random.default_rng(OC * 31 + IC)
    mask = (rng.random((OC, IC, KH, KW)) < density).astype(np.uint8)
    W = (rng.standard_normal(mask.shape) * 0.05).astype(np.float32) * mask
    L = GpuConv(sp, orc, mask, W.astype(np.float32), 1, 8, 8, (1, 1), (1, 1))
    n1 = max(L.nnz, 1)
    t = [torch.full((n,), -7, dtype=torch.int32, device="cuda") for n in (IC + 1, n1, n1)]
    sp.sp_conv_transpose(OC, IC, L.w_oc, L.w_ic, L.nnz, *t)
    r = orc.conv_transpose(OC, IC, *L.o[:2])
    np.testing.assert_array_equal(t[0].cpu().numpy(), r[0])
    np.testing.assert_array_equal(t[1].cpu().numpy()[:L.nnz], r[1])
    np.testing.assert_array_equal(t[2].cpu().numpy()[:L.nnz], r[2])


SMALL = [
    # B, IC, H, W, OC, KH, KW, stride, pad, sparsity
    (3, 5, 9, 11, 7, 3, 3, (1, 1), (1, 1), 0.7),
    (2, 17, 13, 10, 70, 3, 3, (2, 2), (1, 1), 0.8),      # two row panels, stride 2
    (4, 8, 15, 15, 16, 5, 5, (1, 1), (2, 2), 0.6),
    (2, 3, 23, 23, 16, 7, 7, (2, 2), (3, 3), 0.5),       # stem-like 7x7 s2 p3
    (5, 33, 7, 7, 40, 1, 1, (1, 1), (0, 0), 0.7),
    (3, 24, 14, 14, 48, 1, 1, (2, 2), (0, 0), 0.7),      # 1x1 s2 downsample
    (2, 6, 12, 9, 10, 3, 5, (2, 1), (1, 2), 0.5),        # anisotropic kernel, stride, pad
    (2, 4, 17, 16, 9, 3, 3, (3, 3), (0, 0), 0.5),        # stride 3: pixels no tap reaches
    (1, 3, 5, 5, 4, 3, 3, (1, 1), (2, 2), 0.3),          # pad larger than half the kernel
    (2, 40, 10, 10, 20, 3, 3, (1, 1), (1, 1), 0.6),      # 360 columns: several slabs
    (2, 6, 9, 9, 5, 3, 3, (1, 1), (1, 1), 0.0),          # dense
    (1, 2, 3, 3, 3, 3, 3, (1, 1), (0, 0), 0.0),          # 1x1 output
    (7, 9, 6, 5, 130, 2, 2, (1, 2), (0, 1), 0.6),        # 130 output channels, even kernel
    (2, 12, 9, 11, 20, 3, 3, (2, 2), (0, 0), 0.6),       # stride 2, odd sizes, no padding: phase classes
    (3, 20, 10, 7, 9, 2, 4, (2, 2), (1, 2), 0.5),        # stride 2, even kernel sizes
    (2, 1, 15, 15, 8, 5, 5, (2, 2), (2, 2), 0.4),        # one input channel (direct kernel), stride 2
    (2, 8, 6, 6, 300, 3, 3, (1, 1), (1, 1), 0.9),        # 8 input channels, 2700 columns (entry rounds)
    (1, 300, 9, 8, 24, 3, 3, (2, 2), (1, 1), 0.8),       # stride 2 with two input-channel panels
    (2, 16, 20, 20, 40, 7, 7, (1, 1), (3, 3), 0.9),      # 49 taps over full waves (wide tap masks)
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_shapes(sp, orc, case):
    B, IC, H, Wd, OC, KH, KW, stride, pad, s = SMALL[case]
    d, dims = _layer(orc, 7000 + case, B, IC, H, Wd, OC, KH, KW, stride, pad, s)
    _run_all(sp, orc, d, dims, "small%d" % case)


def test_many_tiles_ragged(sp, orc):
    """Several hundred token tiles with a ragged last tile and 2 panels."""
    d, dims = _layer(orc, 7100, 5, 21, 31, 29, 100, 3, 3, (1, 1), (1, 1), 0.9)
    _run_all(sp, orc, d, dims, "ragged 5x21x31x29->100")


def test_edge_patterns(sp, orc):
    rng = np.random.default_rng(17)
    B, IC, H, Wd, OC, KH, KW = 3, 12, 11, 13, 20, 3, 3
    mask = (rng.random((OC, IC, KH, KW)) < 0.1).astype(np.uint8)
    mask[3] = 1                    # a dense output channel
    mask[5] = 0                    # an empty output channel
    mask[:, 7] = 0                 # an empty input channel
    mask[:, 9, 1, 1] = 1           # centre tap of one input channel everywhere
    W = (rng.standard_normal(mask.shape) * 0.05).astype(np.float32) * mask
    W[3, 0, 0, 0] = 0.0            # a stored zero
    dims = (B, IC, H, Wd, OC, KH, KW, (1, 1), (1, 1))
    X = rng.standard_normal((B, IC, H, Wd)).astype(np.float32)
    dY = rng.standard_normal((B, OC, H, Wd)).astype(np.float32)
    d = {"mask": mask, "W": W.astype(np.float32), "X": X, "dY": dY}
    _run_all(sp, orc, d, dims, "edge patterns")


def test_empty_pattern_and_empty_batch(sp, orc):
    import torch
    mask = np.zeros((6, 4, 3, 3), np.uint8)
    W = np.zeros(mask.shape, np.float32)
    L = GpuConv(sp, orc, mask, W, 2, 7, 7, (1, 1), (1, 1))
    assert L.nnz == 0
    X = torch.randn(2, 4, 7, 7, device="cuda")
    dY = torch.randn(2, 6, 7, 7, device="cuda")
    assert torch.all(L.fwd(X) == 0)
    assert torch.all(L.bwd_input(dY) == 0)
    assert L.bwd_weight(dY, X).numel() == 0
    dXf, dWf = L.bwd(dY, X)
    assert torch.all(dXf == 0) and dWf.numel() == 0
    # an empty batch is a no-op for every pass
    d, dims = _layer(orc, 7200, 2, 4, 7, 7, 6, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], 0, 7, 7, (1, 1), (1, 1))
    e = torch.empty(0, device="cuda")
    sp.sp_conv_fwd(e, L.shape, L.w_vals, L.nnz, L.plan, e)
    sp.sp_conv_bwd_input(e, L.shape, L.w_vals, L.nnz, L.plan, e)
    dW = torch.full((L.nnz,), 5.0, device="cuda")
    sp.sp_conv_bwd_weight(e, e, L.shape, L.nnz, L.plan, dW, None)
    assert torch.all(dW == 0)
    dW.fill_(5.0)
    sp.sp_conv_bwd(e, e, L.shape, L.w_vals, L.nnz, L.plan, e, dW, None)
    assert torch.all(dW == 0)


@pytest.mark.parametrize("IC", [10, 3])
def test_plan_is_shape_independent(sp, orc, IC):
    """A plan depends on the pattern only: one plan serves other spatial
    sizes, strides, paddings and batches, for all three passes (stride 2 in
    both directions picks the tap class of each phase from the padding; with
    IC <= 8 the direct input-gradient kernel serves)."""
    import torch
    d, dims = _layer(orc, 7300 + IC, 2, IC, 12, 12, 14, 3, 3, (1, 1), (1, 1), 0.7)
    L = GpuConv(sp, orc, d["mask"], d["W"], dims[0], dims[2], dims[3], dims[7], dims[8])
    rng = np.random.default_rng(3)
    for dims2 in [(3, IC, 9, 11, 14, 3, 3, (2, 1), (0, 1)), (2, IC, 13, 10, 14, 3, 3, (2, 2), (0, 1)),
                  (2, IC, 11, 12, 14, 3, 3, (2, 2), (1, 0)), (1, IC, 8, 9, 14, 3, 3, (1, 1), (2, 0))]:
        s2 = sp.conv_shape(*dims2)
        os2 = orc.conv_shape(*dims2)
        oh, ow = sp.sp_conv_out_hw(s2)
        B2 = dims2[0]
        X = rng.standard_normal(dims2[:4]).astype(np.float32)
        dY = rng.standard_normal((B2, 14, oh, ow)).astype(np.float32)
        Y = torch.full((B2, 14, oh, ow), float("nan"), device="cuda")
        dX = torch.full(dims2[:4], float("nan"), device="cuda")
        dW = torch.full((max(L.nnz, 1),), float("nan"), device="cuda")
        ws = torch.empty(max(sp.sp_conv_bwd_weight_ws(s2, L.nnz), 1), dtype=torch.uint8, device="cuda")
        Xd, dYd = torch.from_numpy(X).cuda(), torch.from_numpy(dY).cuda()
        sp.sp_conv_fwd(Xd, s2, L.w_vals, L.nnz, L.plan, Y)
        sp.sp_conv_bwd_input(dYd, s2, L.w_vals, L.nnz, L.plan, dX)
        sp.sp_conv_bwd_weight(dYd, Xd, s2, L.nnz, L.plan, dW, ws)
        torch.cuda.synchronize()
        what = "shape %s" % (dims2,)
        Yr, Ya = orc.conv_fwd(X, os2, *L.o)
        assert_parity(Y.cpu().numpy(), Yr, Ya, what + " fwd")
        dXr, dXa = orc.conv_bwd_input(dY, os2, *L.o)
        assert_parity(dX.cpu().numpy(), dXr, dXa, what + " bwd_input")
        dWr, dWa = orc.conv_bwd_weight(dY, X, os2, *L.o[:4])
        assert_parity(dW.cpu().numpy()[:L.nnz], dWr, dWa, what + " bwd_weight")


def test_deterministic(sp, orc):
    import torch
    d, dims = _layer(orc, 7400, 4, 16, 20, 20, 32, 3, 3, (1, 1), (1, 1), 0.9)
    L = GpuConv(sp, orc, d["mask"], d["W"], dims[0], dims[2], dims[3], dims[7], dims[8])
    X = torch.from_numpy(d["X"]).cuda()
    dY = torch.from_numpy(d["dY"]).cuda()
    a = (L.fwd(X), L.bwd_input(dY), L.bwd_weight(dY, X)) + L.bwd(dY, X)
    b = (L.fwd(X), L.bwd_input(dY), L.bwd_weight(dY, X)) + L.bwd(dY, X)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_error_paths(sp, orc):
    import torch
    bad = sp.conv_shape(1, 4, 2, 2, 4, 3, 3, (1, 1), (0, 0))   # kernel larger than the padded input
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_out_hw(bad)
    assert e.value.status == sp.SP_ERR_INVALID_ARG
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_plan_bytes(sp.conv_shape(1, 4, 8, 8, 4, 3, 3, (0, 1), (0, 0)), 0)
    assert e.value.status == sp.SP_ERR_INVALID_ARG
    with pytest.raises(sp.SparsePropError) as e:   # per-channel offsets would overflow int16
        sp.sp_conv_plan_bytes(sp.conv_shape(1, 4000, 8, 8, 4, 3, 3, (1, 1), (1, 1)), 0)
    assert e.value.status == sp.SP_ERR_UNSUPPORTED
    d, dims = _layer(orc, 7500, 2, 4, 8, 8, 6, 3, 3, (1, 1), (1, 1), 0.5)
    L = GpuConv(sp, orc, d["mask"], d["W"], dims[0], dims[2], dims[3], dims[7], dims[8])
    X = torch.from_numpy(d["X"]).cuda()
    dY = torch.from_numpy(d["dY"]).cuda()
    small = torch.empty(4, dtype=torch.uint8, device="cuda")
    dW = torch.empty(L.nnz, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_bwd_weight(dY, X, L.shape, L.nnz, L.plan, dW, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_plan(L.shape, L.w_oc, L.w_ic, L.w_x, L.w_y, L.nnz, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    dX = torch.empty(2, 4, 8, 8, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_bwd(dY, X, L.shape, L.w_vals, L.nnz, L.plan, dX, dW, small)
    assert e.value.status == sp.SP_ERR_WORKSPACE
    ws = torch.empty(sp.sp_conv_bwd_weight_ws(L.shape, L.nnz), dtype=torch.uint8, device="cuda")
    with pytest.raises(sp.SparsePropError) as e:
        sp.sp_conv_bwd(dY, X, L.shape, L.w_vals, L.nnz, L.plan, None, dW, ws)
    assert e.value.status == sp.SP_ERR_INVALID_ARG


def test_validate_host(sp, orc):
    d, dims = _layer(orc, 7600, 1, 6, 5, 5, 7, 3, 3, (1, 1), (1, 1), 0.6)
    w_oc, w_ic, w_x, w_y, _ = orc.conv_encode(d["mask"], d["W"])
    sp.sp_conv_validate(7, 6, 3, 3, w_oc, w_ic, w_x, w_y, int(w_oc[-1]))
    w_x2 = w_x.copy()
    w_x2[0] = 3
    with pytest.raises(sp.SparsePropError):
        sp.sp_conv_validate(7, 6, 3, 3, w_oc, w_ic, w_x2, w_y, int(w_oc[-1]))


# ---------------------------------------------------------------- full size

def test_conv3x3_56_full_size(sp, orc):
    """64->64 3x3 s1 p1 on 32x64x56x56 at 90%: images 0, 13, 31 compared for
    the per-image passes, every stored weight for the gradient."""
    name, B, IC, H, Wd, OC, KH, KW, s, p, sparsity = CONV_3X3_56[0]
    d, dims = _layer(orc, seed_for(3, 0), B, IC, H, Wd, OC, KH, KW, (s, s), (p, p), sparsity)
    _run_all(sp, orc, d, dims, name, sample_images=[0, 13, 31])


@pytest.mark.parametrize("idx", range(12))
def test_conv_sweep_full_size(sp, orc, idx):
    name, B, IC, H, Wd, OC, KH, KW, s, p, sparsity = conv_sweep()[idx]
    d, dims = _layer(orc, seed_for(4, idx), B, IC, H, Wd, OC, KH, KW, (s, s), (p, p), sparsity)
    _run_all(sp, orc, d, dims, name, sample_images=[0, 17, 31])


@pytest.mark.parametrize("idx", range(20))
def test_resnet18_conv_full_size(sp, orc, idx):
    """The 20 convolutions of the ResNet-18 stack at batch 64, 95% sparse."""
    name, B, IC, H, Wd, OC, KH, KW, s, p, sparsity = resnet18_convs()[idx]
    d, dims = _layer(orc, seed_for(5, idx), B, IC, H, Wd, OC, KH, KW, (s, s), (p, p), sparsity)
    _run_all(sp, orc, d, dims, name, sample_images=[0, 29, 63])
