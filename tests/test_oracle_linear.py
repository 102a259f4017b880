"""Pins of the CPU oracle's linear-layer functions against what the paper and
the mathematics fix (no GPU).

Sources (SparseProp, Sec. 3.2): the forward product O = X W, Eq. 1
(dL/dX = dL/dO W^T), Eq. 2 (dL/dW = X^T dL/dO) evaluated only at stored
entries, the CSR layout and the CSR->CSC remark.  Each pin is independent of
the oracle's code: numpy fp64 dense products on the masked matrix, scipy's
CSR/CSC conversion, closed forms and identities.
"""
import numpy as np
import pytest
import scipy.sparse as sps

from synth import linear_layer


def _rand(rng, out_f, in_f, B, density):
    mask = (rng.random((out_f, in_f)) < density).astype(np.uint8)
    W = (rng.standard_normal((out_f, in_f)) * 0.3).astype(np.float32) * mask
    X = rng.standard_normal((B, in_f)).astype(np.float32)
    dY = rng.standard_normal((B, out_f)).astype(np.float32)
    return mask, W.astype(np.float32), X, dY


def _close(val, ref, abssum, tol=1e-12):
    val = np.asarray(val, np.float64)
    ref = np.asarray(ref, np.float64)
    assert val.shape == ref.shape
    bound = tol * np.asarray(abssum) + 1e-300
    assert np.all(np.abs(val - ref) <= bound), np.max(np.abs(val - ref) - bound)


def test_encode_matches_row_major_nonzeros(orc):
    rng = np.random.default_rng(1)
    mask, W, _, _ = _rand(rng, 13, 29, 1, 0.3)
    mask[3, :] = 0          # empty row
    mask[5, :] = 1          # full row
    W[5, 7] = 0.0           # stored zero stays stored
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    rows, cols = np.nonzero(mask)  # row-major order
    assert row_ptr[0] == 0 and row_ptr[-1] == len(rows)
    np.testing.assert_array_equal(np.diff(row_ptr), np.bincount(rows, minlength=13))
    np.testing.assert_array_equal(col_idx, cols)
    np.testing.assert_array_equal(vals, W[rows, cols])


@pytest.mark.parametrize("out_f,in_f,density", [(7, 11, 0.3), (33, 5, 0.5), (1, 40, 1.0), (20, 20, 0.0), (64, 48, 0.05)])
def test_transpose_matches_scipy_csc(orc, out_f, in_f, density):
    rng = np.random.default_rng(out_f * 100 + in_f)
    mask, W, _, _ = _rand(rng, out_f, in_f, 1, density)
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    nnz = int(row_ptr[-1])
    t_col_ptr, t_row_idx, t_perm = orc.linear_transpose(in_f, out_f, row_ptr, col_idx)
    # scipy: CSR with data = CSR position + 1, converted to CSC
    csr = sps.csr_matrix((np.arange(1, nnz + 1, dtype=np.float64), col_idx, row_ptr), shape=(out_f, in_f))
    csc = csr.tocsc()
    csc.sort_indices()
    np.testing.assert_array_equal(t_col_ptr, csc.indptr)
    np.testing.assert_array_equal(t_row_idx, csc.indices)
    np.testing.assert_array_equal(t_perm, csc.data.astype(np.int64) - 1)


@pytest.mark.parametrize("B", [1, 3, 17])
@pytest.mark.parametrize("in_f,out_f", [(1, 1), (5, 33), (33, 5), (33, 33)])
@pytest.mark.parametrize("density", [0.0, 0.1, 0.5, 1.0])
def test_bruteforce_dense_fp64(orc, B, in_f, out_f, density):
    """Eq. 1, Eq. 2 and the forward product against dense fp64 matmuls of the
    masked matrix; dW against the dense gradient sampled at the mask."""
    rng = np.random.default_rng(B * 1000 + in_f * 10 + out_f + int(density * 7))
    mask, W, X, dY = _rand(rng, out_f, in_f, B, density)
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    Wd = W.astype(np.float64) * mask
    X64, dY64 = X.astype(np.float64), dY.astype(np.float64)

    Y, Ya = orc.linear_fwd(X, row_ptr, col_idx, vals, out_f)
    _close(Y, X64 @ Wd.T, Ya)
    np.testing.assert_allclose(Ya, np.abs(X64) @ np.abs(Wd).T, rtol=1e-12, atol=0)

    dX, dXa = orc.linear_bwd_input(dY, row_ptr, col_idx, vals, in_f)
    _close(dX, dY64 @ Wd, dXa)
    np.testing.assert_allclose(dXa, np.abs(dY64) @ np.abs(Wd), rtol=1e-12, atol=0)

    dW, dWa = orc.linear_bwd_weight(dY, X, row_ptr, col_idx)
    dense_grad = dY64.T @ X64  # out x in
    rows, cols = np.nonzero(mask)
    _close(dW, dense_grad[rows, cols], dWa)
    np.testing.assert_allclose(dWa, (np.abs(dY64).T @ np.abs(X64))[rows, cols], rtol=1e-12, atol=0)


def test_adjoint_and_euler_identities(orc):
    """<fwd(X), dY> = <X, bwd_input(dY)> (adjoint) and
    <vals, bwd_weight(dY, X)> = <fwd(X), dY> (bilinearity) at a mid size."""
    d = linear_layer(7, 96, 80, 40, 0.9)
    row_ptr, col_idx, vals = orc.linear_encode(d["mask"], d["W"])
    Y, Ya = orc.linear_fwd(d["X"], row_ptr, col_idx, vals, 96)
    dX, _ = orc.linear_bwd_input(d["dY"], row_ptr, col_idx, vals, 80)
    dW, _ = orc.linear_bwd_weight(d["dY"], d["X"], row_ptr, col_idx)
    lhs = float(np.sum(Y * d["dY"].astype(np.float64)))
    rhs = float(np.sum(d["X"].astype(np.float64) * dX))
    euler = float(np.dot(vals.astype(np.float64), dW))
    scale = float(np.sum(Ya * np.abs(d["dY"])))
    assert abs(lhs - rhs) <= 1e-12 * scale
    assert abs(lhs - euler) <= 1e-12 * scale


def test_single_entry_closed_form(orc):
    out_f, in_f, B = 6, 9, 5
    mask = np.zeros((out_f, in_f), np.uint8)
    mask[4, 2] = 1
    W = np.zeros((out_f, in_f), np.float32)
    W[4, 2] = 0.75
    rng = np.random.default_rng(3)
    X = rng.standard_normal((B, in_f)).astype(np.float32)
    dY = rng.standard_normal((B, out_f)).astype(np.float32)
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    Y, _ = orc.linear_fwd(X, row_ptr, col_idx, vals, out_f)
    expect = np.zeros((B, out_f))
    expect[:, 4] = 0.75 * X[:, 2].astype(np.float64)
    np.testing.assert_array_equal(Y, expect)
    dX, _ = orc.linear_bwd_input(dY, row_ptr, col_idx, vals, in_f)
    expect = np.zeros((B, in_f))
    expect[:, 2] = 0.75 * dY[:, 4].astype(np.float64)
    np.testing.assert_array_equal(dX, expect)
    dW, _ = orc.linear_bwd_weight(dY, X, row_ptr, col_idx)
    assert dW.shape == (1,)
    assert dW[0] == pytest.approx(float(np.dot(dY[:, 4].astype(np.float64), X[:, 2].astype(np.float64))), rel=1e-14)


def test_stored_zero_weight_still_gets_gradient(orc):
    mask = np.ones((2, 3), np.uint8)
    W = np.zeros((2, 3), np.float32)
    X = np.array([[1.0, 2.0, 3.0]], np.float32)
    dY = np.array([[4.0, 5.0]], np.float32)
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    assert row_ptr[-1] == 6
    dW, _ = orc.linear_bwd_weight(dY, X, row_ptr, col_idx)
    np.testing.assert_array_equal(dW, [4, 8, 12, 5, 10, 15])


def test_empty_rows_and_columns_give_exact_zero(orc):
    rng = np.random.default_rng(11)
    mask, W, X, dY = _rand(rng, 10, 12, 4, 0.4)
    mask[2, :] = 0
    mask[:, 7] = 0
    W = W * mask
    row_ptr, col_idx, vals = orc.linear_encode(mask, W)
    Y, Ya = orc.linear_fwd(X, row_ptr, col_idx, vals, 10)
    assert np.all(Y[:, 2] == 0) and np.all(Ya[:, 2] == 0)
    dX, dXa = orc.linear_bwd_input(dY, row_ptr, col_idx, vals, 12)
    assert np.all(dX[:, 7] == 0) and np.all(dXa[:, 7] == 0)


def test_linearity_in_x_and_vals(orc):
    d = linear_layer(21, 40, 30, 9, 0.8)
    row_ptr, col_idx, vals = orc.linear_encode(d["mask"], d["W"])
    X2 = np.random.default_rng(5).standard_normal(d["X"].shape).astype(np.float32)
    Y1, A1 = orc.linear_fwd(d["X"], row_ptr, col_idx, vals, 40)
    Y2, A2 = orc.linear_fwd(X2, row_ptr, col_idx, vals, 40)
    Ys, _ = orc.linear_fwd((d["X"].astype(np.float64) + X2).astype(np.float32), row_ptr, col_idx, vals, 40)
    # float32 rounding of X1+X2 is the only difference
    assert np.all(np.abs(Ys - (Y1 + Y2)) <= 1e-6 * (A1 + A2) + 1e-12)
    Yh, _ = orc.linear_fwd(d["X"], row_ptr, col_idx, (vals * 2).astype(np.float32), 40)
    np.testing.assert_array_equal(Yh, 2 * Y1)


def test_zero_sparsity_is_dense_backprop(orc):
    d = linear_layer(4, 24, 16, 8, 0.0)
    assert d["mask"].all()
    row_ptr, col_idx, vals = orc.linear_encode(d["mask"], d["W"])
    W64 = d["W"].astype(np.float64)
    Y, Ya = orc.linear_fwd(d["X"], row_ptr, col_idx, vals, 24)
    _close(Y, d["X"].astype(np.float64) @ W64.T, Ya)
    dW, dWa = orc.linear_bwd_weight(d["dY"], d["X"], row_ptr, col_idx)
    _close(dW.reshape(24, 16), d["dY"].astype(np.float64).T @ d["X"].astype(np.float64), dWa.reshape(24, 16))


def test_synth_exact_count_mask():
    d = linear_layer(0, 256, 256, 16, 0.9)
    assert int(d["mask"].sum()) == 6554
    d2 = linear_layer(0, 256, 256, 16, 0.9)
    np.testing.assert_array_equal(d["mask"], d2["mask"])
    np.testing.assert_array_equal(d["X"], d2["X"])
    assert np.all(d["W"][d["mask"] == 0] == 0)
