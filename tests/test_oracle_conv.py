"""Pins of the CPU oracle's convolution functions (no GPU).

Sources (SparseProp, Sec. 3.3): Eq. 3 (forward), Eq. 4 (input gradient),
Eq. 5 (weight gradient) with pruned weights skipped, the five-array format
and its worked example, and Algorithm 2's padded bounds.  Pins: PyTorch's CPU
conv2d and its autograd in float64 (a library routine computing the same
cross-correlation, with stride and padding), a brute-force 7-loop
definition, the paper's worked encoding example, identities and closed forms.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from synth import conv_layer

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "conv_format_example.json")


def _rand(rng, B, IC, H, W, OC, KH, KW, density):
    mask = (rng.random((OC, IC, KH, KW)) < density).astype(np.uint8)
    Wt = (rng.standard_normal((OC, IC, KH, KW)) * 0.3).astype(np.float32) * mask
    X = rng.standard_normal((B, IC, H, W)).astype(np.float32)
    return mask, Wt.astype(np.float32), X


def _torch_ref(X, Wd, dY, stride, pad):
    stride = tuple(stride) if isinstance(stride, (tuple, list)) else (stride, stride)
    pad = tuple(pad) if isinstance(pad, (tuple, list)) else (pad, pad)
    Xt = torch.tensor(X, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(Wd, dtype=torch.float64, requires_grad=True)
    Y = F.conv2d(Xt, Wt, stride=stride, padding=pad)
    Y.backward(torch.tensor(dY, dtype=torch.float64))
    return Y.detach().numpy(), Xt.grad.numpy(), Wt.grad.numpy()


def _close(val, ref, abssum, tol=1e-12):
    bound = tol * np.asarray(abssum) + 1e-300
    assert np.all(np.abs(np.asarray(val) - np.asarray(ref)) <= bound)


def test_worked_example_encoding(orc):
    g = json.load(open(GOLDEN))
    OC, IC, KH, KW = g["shape"]
    mask = np.zeros((OC, IC, KH, KW), np.uint8)
    W = np.zeros((OC, IC, KH, KW), np.float32)
    for oc, ic, x, y, lab in g["entries_oc_ic_x_y_label"]:
        mask[oc, ic, x, y] = 1
        W[oc, ic, x, y] = g["labels_to_values"][lab]
    w_oc, w_ic, w_x, w_y, w_vals = orc.conv_encode(mask, W)
    e = g["expected_printed"]
    np.testing.assert_array_equal(w_oc, e["W_oc"])
    np.testing.assert_array_equal(w_ic, e["W_ic"])
    np.testing.assert_array_equal(w_x, e["W_x"])
    np.testing.assert_array_equal(w_y, e["W_y"])
    expect_vals = [g["labels_to_values"][lab] for lab in g["expected_value_labels_storage_order"]]
    np.testing.assert_array_equal(w_vals, expect_vals)


def test_encode_order_is_row_major_nonzeros(orc):
    rng = np.random.default_rng(2)
    mask, W, _ = _rand(rng, 1, 5, 3, 3, 4, 3, 2, 0.4)
    mask[1] = 0  # empty output channel
    W = W * mask
    w_oc, w_ic, w_x, w_y, w_vals = orc.conv_encode(mask, W)
    oc, ic, x, y = np.nonzero(mask)
    np.testing.assert_array_equal(w_x, x)
    np.testing.assert_array_equal(w_y, y)
    np.testing.assert_array_equal(w_vals, W[oc, ic, x, y])
    np.testing.assert_array_equal(np.diff(w_oc), np.bincount(oc, minlength=4))
    counts = mask.reshape(4, 5, -1).sum(-1)
    for o in range(4):
        np.testing.assert_array_equal(w_ic[o * 6:(o + 1) * 6], np.concatenate([[0], np.cumsum(counts[o])]))


def test_transpose_is_ic_major_stable(orc):
    rng = np.random.default_rng(9)
    OC, IC = 7, 6
    mask, W, _ = _rand(rng, 1, IC, 3, 3, OC, 3, 3, 0.3)
    w_oc, w_ic, w_x, w_y, w_vals = orc.conv_encode(mask, W)
    t_ic_ptr, t_oc, t_perm = orc.conv_transpose(OC, IC, w_oc, w_ic)
    oc, ic, x, y = np.nonzero(mask)   # storage order = (oc, ic, x, y)
    order = np.lexsort((y, x, oc, ic))  # sort by (ic, oc, x, y)
    np.testing.assert_array_equal(t_perm, order)
    np.testing.assert_array_equal(t_oc, oc[order])
    np.testing.assert_array_equal(t_ic_ptr, np.concatenate([[0], np.cumsum(np.bincount(ic, minlength=IC))]))


CASES = [(H, W, KH, KW, s, p) for H, W in [(5, 5), (7, 6)] for KH, KW in [(1, 1), (2, 3), (3, 3)]
         for s in (1, 2) for p in (0, 1, 2) if H + 2 * p >= KH and W + 2 * p >= KW]


@pytest.mark.parametrize("H,W,KH,KW,s,p", CASES)
def test_against_torch_conv2d_fp64(orc, H, W, KH, KW, s, p):
    B, IC, OC = 2, 3, 4
    rng = np.random.default_rng(H * 997 + W * 89 + KH * 31 + KW * 7 + s * 3 + p)
    mask, Wd, X = _rand(rng, B, IC, H, W, OC, KH, KW, 0.5)
    sh = orc.conv_shape(B, IC, H, W, OC, KH, KW, (s, s), (p, p))
    OH, OW = orc.conv_out_hw(sh)
    assert (OH, OW) == ((H + 2 * p - KH) // s + 1, (W + 2 * p - KW) // s + 1)
    dY = rng.standard_normal((B, OC, OH, OW)).astype(np.float32)
    Yr, dXr, dWr = _torch_ref(X, Wd, dY, s, p)
    enc = orc.conv_encode(mask, Wd)
    w_oc, w_ic, w_x, w_y, w_vals = enc
    Y, Ya = orc.conv_fwd(X, sh, *enc)
    _close(Y, Yr, Ya)
    dX, dXa = orc.conv_bwd_input(dY, sh, *enc)
    _close(dX, dXr, dXa)
    dW, dWa = orc.conv_bwd_weight(dY, X, sh, w_oc, w_ic, w_x, w_y)
    oc, ic, x, y = np.nonzero(mask)
    _close(dW, dWr[oc, ic, x, y], dWa)


@pytest.mark.parametrize("sh_,sw_,ph_,pw_", [(2, 1, 1, 2), (1, 3, 0, 1)])
def test_against_torch_conv2d_anisotropic(orc, sh_, sw_, ph_, pw_):
    """Different strides/pads along H and W catch swapped dimensions."""
    B, IC, H, W, OC, KH, KW = 2, 3, 7, 8, 4, 3, 2
    rng = np.random.default_rng(sh_ * 10 + sw_)
    mask, Wd, X = _rand(rng, B, IC, H, W, OC, KH, KW, 0.5)
    sh = orc.conv_shape(B, IC, H, W, OC, KH, KW, (sh_, sw_), (ph_, pw_))
    OH, OW = orc.conv_out_hw(sh)
    dY = rng.standard_normal((B, OC, OH, OW)).astype(np.float32)
    Yr, dXr, dWr = _torch_ref(X, Wd, dY, (sh_, sw_), (ph_, pw_))
    enc = orc.conv_encode(mask, Wd)
    Y, Ya = orc.conv_fwd(X, sh, *enc)
    _close(Y, Yr, Ya)
    dX, dXa = orc.conv_bwd_input(dY, sh, *enc)
    _close(dX, dXr, dXa)
    dW, dWa = orc.conv_bwd_weight(dY, X, sh, *enc[:4])
    oc, ic, x, y = np.nonzero(mask)
    _close(dW, dWr[oc, ic, x, y], dWa)


def _brute_fwd(X, Wd, s, p):
    """Seven nested loops of the definition with explicit zero padding."""
    B, IC, H, W = X.shape
    OC, _, KH, KW = Wd.shape
    OH, OW = (H + 2 * p - KH) // s + 1, (W + 2 * p - KW) // s + 1
    Xp = np.zeros((B, IC, H + 2 * p, W + 2 * p))
    Xp[:, :, p:p + H, p:p + W] = X
    Y = np.zeros((B, OC, OH, OW))
    for b in range(B):
        for o in range(OC):
            for i in range(IC):
                for a in range(KH):
                    for c in range(KW):
                        if Wd[o, i, a, c] == 0:
                            continue
                        for u in range(OH):
                            for v in range(OW):
                                Y[b, o, u, v] += Wd[o, i, a, c] * Xp[b, i, u * s + a, v * s + c]
    return Y


def test_against_seven_loop_definition(orc):
    rng = np.random.default_rng(77)
    B, IC, H, W, OC, KH, KW, s, p = 2, 2, 6, 5, 3, 3, 2, 2, 1
    mask, Wd, X = _rand(rng, B, IC, H, W, OC, KH, KW, 0.6)
    sh = orc.conv_shape(B, IC, H, W, OC, KH, KW, (s, s), (p, p))
    Y, Ya = orc.conv_fwd(X, sh, *orc.conv_encode(mask, Wd))
    _close(Y, _brute_fwd(X.astype(np.float64), Wd.astype(np.float64), s, p), Ya)


def test_algorithm2_pad_bounds_reading():
    """Algorithm 2 bounds p in [max(0, pad - x), min(pad - x + M, OM)) at
    stride 1; the stride-s generalisation used by the kernels must select
    exactly the p with 0 <= p*s + x - pad < M."""
    for M in range(1, 9):
        for K in range(1, 6):
            for pad in range(0, 4):
                for s in (1, 2, 3):
                    if M + 2 * pad < K:
                        continue
                    OM = (M + 2 * pad - K) // s + 1
                    for x in range(K):
                        want = [u for u in range(OM) if 0 <= u * s + x - pad < M]
                        lo = max(0, -((x - pad) // s))            # ceil((pad - x)/s)
                        hi = min(OM, (M - 1 + pad - x) // s + 1)  # floor((M-1+pad-x)/s)+1
                        got = list(range(lo, hi))
                        assert got == want, (M, K, pad, s, x)
                        if s == 1:
                            assert (lo, hi) == (max(0, pad - x), min(pad - x + M, OM))


def test_identities_and_special_cases(orc):
    B, IC, H, W, OC = 3, 8, 9, 9, 6
    sh = orc.conv_shape(B, IC, H, W, OC, 3, 3, (2, 2), (1, 1))
    OH, OW = orc.conv_out_hw(sh)
    d = conv_layer(5, B, IC, H, W, OC, 3, 3, (OH, OW), 0.8)
    enc = orc.conv_encode(d["mask"], d["W"])
    w_oc, w_ic, w_x, w_y, w_vals = enc
    Y, Ya = orc.conv_fwd(d["X"], sh, *enc)
    dX, _ = orc.conv_bwd_input(d["dY"], sh, *enc)
    dW, _ = orc.conv_bwd_weight(d["dY"], d["X"], sh, w_oc, w_ic, w_x, w_y)
    lhs = float(np.sum(Y * d["dY"]))
    scale = float(np.sum(Ya * np.abs(d["dY"])))
    assert abs(lhs - float(np.sum(d["X"].astype(np.float64) * dX))) <= 1e-12 * scale   # adjoint
    assert abs(lhs - float(np.dot(w_vals.astype(np.float64), dW))) <= 1e-12 * scale    # Euler


def test_single_entry_is_shifted_scaled_channel(orc):
    B, IC, H, W, OC = 2, 3, 6, 7, 2
    mask = np.zeros((OC, IC, 3, 3), np.uint8)
    Wd = np.zeros((OC, IC, 3, 3), np.float32)
    mask[1, 2, 0, 2] = 1
    Wd[1, 2, 0, 2] = -1.5
    X = np.random.default_rng(4).standard_normal((B, IC, H, W)).astype(np.float32)
    sh = orc.conv_shape(B, IC, H, W, OC, 3, 3, (1, 1), (1, 1))
    Y, _ = orc.conv_fwd(X, sh, *orc.conv_encode(mask, Wd))
    expect = np.zeros((B, OC, H, W))
    # Y[b,1,p,q] = -1.5 * X[b,2,p-1,q+1]
    expect[:, 1, 1:, :W - 1] = -1.5 * X[:, 2, :H - 1, 1:].astype(np.float64)
    np.testing.assert_array_equal(Y, expect)


def test_pointwise_conv_equals_linear(orc):
    B, IC, H, W, OC = 2, 16, 5, 4, 12
    sh = orc.conv_shape(B, IC, H, W, OC, 1, 1, (1, 1), (0, 0))
    d = conv_layer(8, B, IC, H, W, OC, 1, 1, (H, W), 0.7)
    enc = orc.conv_encode(d["mask"], d["W"])
    Y, _ = orc.conv_fwd(d["X"], sh, *enc)
    tokens = d["X"].transpose(0, 2, 3, 1).reshape(-1, IC)
    row_ptr, col_idx, vals = orc.linear_encode(d["mask"][:, :, 0, 0], d["W"][:, :, 0, 0])
    Yl, _ = orc.linear_fwd(tokens, row_ptr, col_idx, vals, OC)
    np.testing.assert_allclose(Y.transpose(0, 2, 3, 1).reshape(-1, OC), Yl, rtol=1e-13, atol=1e-13)
    w_oc, w_ic, w_x, w_y, w_vals = enc
    dW, _ = orc.conv_bwd_weight(d["dY"], d["X"], sh, w_oc, w_ic, w_x, w_y)
    gtok = d["dY"].transpose(0, 2, 3, 1).reshape(-1, OC)
    dWl, _ = orc.linear_bwd_weight(gtok, tokens, row_ptr, col_idx)
    np.testing.assert_allclose(dW, dWl, rtol=1e-12, atol=1e-12)


def test_empty_output_channel_gives_exact_zero(orc):
    B, IC, H, W, OC = 2, 4, 5, 5, 3
    rng = np.random.default_rng(12)
    mask, Wd, X = _rand(rng, B, IC, H, W, OC, 3, 3, 0.5)
    mask[1] = 0
    Wd = Wd * mask
    sh = orc.conv_shape(B, IC, H, W, OC, 3, 3, (1, 1), (1, 1))
    Y, Ya = orc.conv_fwd(X, sh, *orc.conv_encode(mask, Wd))
    assert np.all(Y[:, 1] == 0) and np.all(Ya[:, 1] == 0)
