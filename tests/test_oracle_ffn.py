"""Pins for the oracle's FFN definitions, sparse formulations and gradients."""
import json
import os

import numpy as np
import pytest

from oracle import ffn, sizing, twell

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_nongated_example():
    # x = [1, 2]; z = x W_up + b + s = [1, 2-1, -2, 0] + [0, 0, 0, 0] -> with b=[0,0,0,0], s=0
    X = np.array([[1.0, 2.0]])
    W_up = np.array([[1.0, -1.0, 0.0, 2.0],
                     [0.0, 1.0, -1.0, -1.0]])
    W_down = np.array([[1.0, 0.0, 3.0],
                       [0.0, 1.0, 0.0],
                       [5.0, 5.0, 5.0],
                       [7.0, 7.0, 7.0]])
    # z = [1, 1, -2, 0] -> h = [1, 1, 0, 0] (z = 0 is inactive) -> y = [1, 1, 3]
    Y, Z, H = ffn.ffn_dense(X, W_up, W_down)
    np.testing.assert_array_equal(Z, [[1.0, 1.0, -2.0, 0.0]])
    np.testing.assert_array_equal(H, [[1.0, 1.0, 0.0, 0.0]])
    np.testing.assert_array_equal(Y, [[1.0, 1.0, 3.0]])
    # bias b = [0, 0, 3, 1] and shift s = -0.5: z = [0.5, 0.5, 0.5, 0.5] -> y = 0.5*(sum of rows)
    Y2, Z2, _ = ffn.ffn_dense(X, W_up, W_down, bias_f=np.array([0.0, 0.0, 3.0, 1.0]),
                              shift_t=np.array([-0.5]))
    np.testing.assert_array_equal(Z2, [[0.5, 0.5, 0.5, 0.5]])
    np.testing.assert_array_equal(Y2, [[6.5, 6.5, 7.5]])


def test_hand_worked_gated_example():
    X = np.array([[1.0, -1.0]])
    W_gate = np.array([[1.0, 0.0, 2.0], [0.0, 1.0, 1.0]])   # g = [1, -1, 1]
    W_up = np.array([[3.0, 1.0, 1.0], [1.0, 0.0, 4.0]])     # u = [2, 1, -3]
    W_down = np.array([[1.0, 0.0], [9.0, 9.0], [0.0, 1.0]])
    Y, G, U, H = ffn.ffn_gated_dense(X, W_gate, W_up, W_down)
    np.testing.assert_array_equal(H, [[2.0, 0.0, -3.0]])
    np.testing.assert_array_equal(Y, [[2.0, -3.0]])


def rand_problem(T=9, d=6, f=11, seed=0):
    r = np.random.default_rng(seed)
    return (r.standard_normal((T, d)), r.standard_normal((d, f)) * 0.5,
            r.standard_normal((f, d)) * 0.5, r.standard_normal(f) * 0.3, r.standard_normal(T) * 0.3)


def test_relu_identity_and_homogeneity():
    """relu(z) - relu(-z) = z gives Y(X,b,s) - Y(-X,-b,-s) = (X W_up + b + s) W_down; the
    FFN without bias/shift is positively homogeneous of degree 1."""
    X, Wu, Wd, b, s = rand_problem()
    Yp, _, _ = ffn.ffn_dense(X, Wu, Wd, b, s)
    Ym, _, _ = ffn.ffn_dense(-X, Wu, Wd, -b, -s)
    lin = np.einsum("tk,kn,nd->td", X, Wu, Wd) + np.outer(s, Wd.sum(0)) + (b @ Wd)[None, :]
    np.testing.assert_allclose(Yp - Ym, lin, rtol=1e-12, atol=1e-12)
    Y1, _, _ = ffn.ffn_dense(X, Wu, Wd)
    Y3, _, _ = ffn.ffn_dense(2.5 * X, Wu, Wd)
    np.testing.assert_allclose(Y3, 2.5 * Y1, rtol=1e-12, atol=1e-13)


def test_zero_sparsity_is_linear():
    X, Wu, Wd, _, _ = rand_problem(seed=1)
    big = np.full(Wu.shape[1], 1e3)
    Y, Z, _ = ffn.ffn_dense(X, Wu, Wd, bias_f=big)
    assert (Z > 0).all()
    np.testing.assert_allclose(Y, X @ (Wu @ Wd) + big @ Wd, rtol=1e-12)


@pytest.mark.parametrize("val_dtype", ["f32", "bf16"])
def test_sparse_formulations_equal_dense(val_dtype):
    X, Wu, Wd, b, s = rand_problem(T=40, d=8, f=70, seed=2)
    b = b - 1.2
    Y, Z, H = ffn.ffn_dense(X, Wu, Wd, b, s)
    tw = twell.extract_twell(Z, 16, 16, val_dtype)      # S = T_n: nothing dropped
    Ys = ffn.ffn_from_twell(tw, Wd, *Y.shape)
    Yh, _, hy, _ = ffn.ffn_hybrid_forward(X, Wu, Wd, b, s, tile_cols=16, tile_slots=3,
                                          ell_width=8, val_dtype=val_dtype)
    assert hy.is_ovf.any() and (~hy.is_ovf).any()
    if val_dtype == "f32":
        rtol = 1e-6   # storage cast to float32
    else:
        rtol = 2e-2
    np.testing.assert_allclose(Ys, Y, rtol=rtol, atol=rtol * np.abs(Y).max())
    np.testing.assert_allclose(Yh, Y, rtol=rtol, atol=rtol * np.abs(Y).max())
    # with an exact (fp64) cast the sparse formulation is the dense one to rounding
    Yexact = np.zeros_like(Y)
    for t in range(Y.shape[0]):
        cols = np.nonzero(Z[t] > 0)[0]
        Yexact[t] = Z[t, cols] @ Wd[cols]
    np.testing.assert_allclose(Yexact, Y, rtol=1e-12, atol=1e-12)


def test_hybrid_capacity_leaves_excess_rows_unspecified():
    X, Wu, Wd, b, s = rand_problem(T=20, d=8, f=70, seed=3)
    Y, _, _ = ffn.ffn_dense(X, Wu, Wd, b, s)
    Yh, _, hy, _ = ffn.ffn_hybrid_forward(X, Wu, Wd, b, s, tile_cols=16, tile_slots=2,
                                          ell_width=3, ovf_capacity=2)
    assert len(hy.ovf_rows) > 2
    np.testing.assert_allclose(Yh[hy.ovf_rows[:2]], Y[hy.ovf_rows[:2]], rtol=1e-12)
    assert np.isnan(Yh[hy.ovf_rows[2:]]).all()


def test_gated_fused_formulation():
    X, Wu, Wd, b, s = rand_problem(T=12, d=7, f=40, seed=4)
    Wg = np.random.default_rng(5).standard_normal(Wu.shape) * 0.5
    Y, G, U, H = ffn.ffn_gated_dense(X, Wg, Wu, Wd, b, s)
    tw = twell.extract_twell(G, 8, 8, "f32")
    Yf = ffn.ffn_gated_from_twell(tw, X, Wu, Wd)
    np.testing.assert_allclose(Yf, Y, rtol=1e-6, atol=1e-6 * np.abs(Y).max())


def loss_nongated(X, Wu, Wd, dY, lam, b, s):
    Y, Z, H = ffn.ffn_dense(X, Wu, Wd, b, s)
    return (dY * Y).sum() + ffn.l1_penalty(H, lam)


def fd_grad(fun, A, eps=1e-6):
    g = np.zeros_like(A)
    it = np.nditer(A, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = A[i]
        A[i] = old + eps
        fp = fun()
        A[i] = old - eps
        fm = fun()
        A[i] = old
        g[i] = (fp - fm) / (2 * eps)
    return g


def away_from_kinks(seed, T, d, f, gated=False):
    """Random problem whose pre-activations all satisfy |z| >= 0.1 (no kink within FD reach)."""
    r = np.random.default_rng(seed)
    while True:
        X = r.standard_normal((T, d))
        Wu = r.standard_normal((d, f)) * 0.7
        Wd = r.standard_normal((f, d)) * 0.7
        Wg = r.standard_normal((d, f)) * 0.7
        Z = X @ (Wg if gated else Wu)
        if (np.abs(Z) >= 0.1).all() and 0 < (Z > 0).mean() < 1:
            return X, Wu, Wd, Wg, r.standard_normal((T, d))


@pytest.mark.parametrize("lam", [0.0, 3.0])
def test_backward_matches_finite_differences(lam):
    T, d, f = 3, 4, 5
    X, Wu, Wd, _, dY = away_from_kinks(10, T, d, f)
    b = np.zeros(f)
    s = np.zeros(T)
    Y, Z, H = ffn.ffn_dense(X, Wu, Wd)
    dX, dWu, dWd, _ = ffn.ffn_backward(X, Wu, Wd, dY, H, Z > 0, lam)
    fun = lambda: loss_nongated(X, Wu, Wd, dY, lam, b, s)
    np.testing.assert_allclose(dX, fd_grad(fun, X), atol=1e-7)
    np.testing.assert_allclose(dWu, fd_grad(fun, Wu), atol=1e-7)
    np.testing.assert_allclose(dWd, fd_grad(fun, Wd), atol=1e-7)


@pytest.mark.parametrize("lam", [0.0, 3.0])
def test_gated_backward_matches_finite_differences(lam):
    T, d, f = 3, 4, 5
    X, Wu, Wd, Wg, dY = away_from_kinks(11, T, d, f, gated=True)
    U = X @ Wu
    assert (np.abs(U) > 1e-3).all()

    def fun():
        Y, G, U_, H = ffn.ffn_gated_dense(X, Wg, Wu, Wd)
        return (dY * Y).sum() + ffn.l1_penalty(H, lam)

    Y, G, U, H = ffn.ffn_gated_dense(X, Wg, Wu, Wd)
    dX, dWg, dWu, dWd = ffn.ffn_gated_backward(X, Wg, Wu, Wd, dY, G, U, lam)
    np.testing.assert_allclose(dX, fd_grad(fun, X), atol=1e-7)
    np.testing.assert_allclose(dWg, fd_grad(fun, Wg), atol=1e-7)
    np.testing.assert_allclose(dWu, fd_grad(fun, Wu), atol=1e-7)
    np.testing.assert_allclose(dWd, fd_grad(fun, Wd), atol=1e-7)


def test_l1_penalty_scale():
    H = np.zeros((4, 5))
    H[1, 2] = 2.0
    H[3, 0] = 0.5
    assert ffn.l1_penalty(H, 10.0) == pytest.approx(10.0 * 2.5 / 20)


def test_paper_tile_overflow_claim():
    """The paper's ~1e-34 overflow chance at C = 8 holds at the 24-29 nnz end of its range."""
    claim = json.load(open(os.path.join(GOLDEN, "paper_sizing_claim.json")))
    lo, hi = claim["nnz_range"]
    p_lo = sizing.tile_overflow_probability(lo, claim["hidden"], claim["tile_cols"], claim["compression"])
    p_29 = sizing.tile_overflow_probability(29, claim["hidden"], claim["tile_cols"], claim["compression"])
    p_hi = sizing.tile_overflow_probability(hi, claim["hidden"], claim["tile_cols"], claim["compression"])
    order = claim["claimed_order_log10"]
    assert 10.0 ** (order - 2) < p_lo < 10.0 ** order < p_29 < 10.0 ** (order + 2)
    assert p_hi < 1e-28   # still negligible at the 39-nnz end


@pytest.mark.parametrize("lam", [0.0, 5.0])
def test_per_unit_and_per_row_gradients_equal_the_full_backward(lam):
    """The subset helpers (chosen hidden units, chosen tokens) return exactly the columns /
    rows of the full backward, which the finite-difference tests above pin; non-square
    shapes, a bias and a row shift, on the fp64 pattern z > 0 and on a pattern with flipped
    entries (the GPU's pattern may differ from fp64's within rounding of 0)."""
    r = np.random.default_rng(3)
    T, d, f = 13, 7, 19
    X, Wu, Wd = r.standard_normal((T, d)), r.standard_normal((d, f)) * 0.5, r.standard_normal((f, d)) * 0.5
    bias, shift, dY = r.standard_normal(f) * 0.3, r.standard_normal(T) * 0.3, r.standard_normal((T, d))
    Z = ffn.preactivation(X, Wu, bias, shift)
    units, rows = np.array([17, 0, 4, 11]), np.array([12, 3, 5])
    flip = r.random((T, f)) < 0.1
    for act in (Z > 0, (Z > 0) ^ flip):
        dX, dWu, dWd, _ = ffn.ffn_backward(X, Wu, Wd, dY, np.where(act, Z, 0.0), act, lam)
        gWu, gWd = ffn.ffn_backward_units(X, Wu, Wd, dY, units, act[:, units], lam, bias, shift)
        np.testing.assert_allclose(gWu, dWu[:, units], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(gWd, dWd[units], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(ffn.ffn_backward_rows(X, Wu, Wd, dY, rows, act[rows], lam), dX[rows],
                                   rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("lam", [0.0, 5.0])
def test_gated_per_unit_and_per_row_gradients_equal_the_full_backward(lam):
    """The gated subset helpers on the pattern G > 0 return the columns / rows of
    ffn_gated_backward (pinned by finite differences above), with a gate bias and shift."""
    r = np.random.default_rng(4)
    T, d, f = 11, 6, 17
    X = r.standard_normal((T, d))
    Wg, Wu, Wd = (r.standard_normal(s) * 0.5 for s in ((d, f), (d, f), (f, d)))
    bias, shift, dY = r.standard_normal(f) * 0.3, r.standard_normal(T) * 0.3, r.standard_normal((T, d))
    _, G, U, _ = ffn.ffn_gated_dense(X, Wg, Wu, Wd, bias, shift)
    dX, dWg, dWu, dWd = ffn.ffn_gated_backward(X, Wg, Wu, Wd, dY, G, U, lam)
    units, rows = np.array([16, 2, 9]), np.array([0, 10, 4, 7])
    act = G > 0
    gWg, gWu, gWd = ffn.ffn_gated_backward_units(X, Wg, Wu, Wd, dY, units, act[:, units], lam, bias, shift)
    np.testing.assert_allclose(gWg, dWg[:, units], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(gWu, dWu[:, units], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(gWd, dWd[units], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(ffn.ffn_gated_backward_rows(X, Wg, Wu, Wd, dY, rows, act[rows], lam, bias, shift),
                               dX[rows], rtol=1e-13, atol=1e-13)
