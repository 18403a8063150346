"""fp64 FFN definitions, sparse formulations and gradients (oracle side).

Notation follows the paper (Sec. 2.1) with the build's names: tokens T (the
paper's M), model width d (the paper's K), hidden width f (the paper's N).
X [T,d], W_up and W_gate [d,f], W_down [f,d]. All arithmetic is float64 on
the stored inputs.

Pre-activations may carry two optional additive terms that the paper's
bias-free FFN does not have (its MLP bias is off, Appendix B table): a
per-hidden-unit bias b[n] and a per-token shift s[t]. The synthetic workloads
use them to place the ReLU threshold; with both absent the functions are the
paper's equations exactly.
"""
from __future__ import annotations

import numpy as np

from . import twell as _tw


def preactivation(X, W, bias_f=None, shift_t=None):
    """z[t,n] = sum_k X[t,k] W[k,n] + b[n] + s[t]."""
    Z = np.asarray(X, dtype=np.float64) @ np.asarray(W, dtype=np.float64)
    if bias_f is not None:
        Z = Z + np.asarray(bias_f, dtype=np.float64)[None, :]
    if shift_t is not None:
        Z = Z + np.asarray(shift_t, dtype=np.float64)[:, None]
    return Z


def relu(Z):
    """ReLU with activity iff z > 0 (strict, Alg. 1's test)."""
    return np.where(Z > 0, Z, 0.0)


def ffn_dense(X, W_up, W_down, bias_f=None, shift_t=None):
    """Non-gated FFN, eq. secC:eq:non-gated-mlp: h = ReLU(x W_u), y = h W_d. Returns (Y, Z, H)."""
    Z = preactivation(X, W_up, bias_f, shift_t)
    H = relu(Z)
    return H @ np.asarray(W_down, dtype=np.float64), Z, H


def ffn_gated_dense(X, W_gate, W_up, W_down, bias_f=None, shift_t=None):
    """Gated FFN, eq. sec2:eq:gated-mlp with sigma = ReLU; the bias/shift go to the gate only.

    Returns (Y, G, U, H) with G the gate pre-activation, U = X W_up, H = ReLU(G) * U.
    """
    G = preactivation(X, W_gate, bias_f, shift_t)
    U = np.asarray(X, dtype=np.float64) @ np.asarray(W_up, dtype=np.float64)
    H = relu(G) * U
    return H @ np.asarray(W_down, dtype=np.float64), G, U, H


def ffn_from_twell(tw: _tw.TwELL, W_down, T, d):
    """Non-gated down projection read from TwELL: y[t] = sum over stored slots of v * W_down[n].

    Rows whose tiles overflowed lose entries here; the hybrid path below covers them.
    """
    Wd = np.asarray(W_down, dtype=np.float64)
    Y = np.zeros((T, d), dtype=np.float64)
    S = tw.tile_slots
    for t in range(T):
        for j in range(tw.n_tiles):
            for s in range(min(int(tw.cnt[t, j]), S)):
                n = int(tw.idx[t, j * S + s])
                v = _tw.stored_to_f64(tw.val[t, j * S + s], tw.val_dtype)
                Y[t] += v * Wd[n]
    return Y


def ffn_gated_from_twell(tw: _tw.TwELL, X, W_up, W_down):
    """Alg. 2 / eq. sec3:eq:twell_to_dense_fused_matmul: per stored gate value g at column n,
    u = x[t] . W_up[:, n] and y[t] += (g * u) W_down[n]."""
    Xd = np.asarray(X, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    T, d = Xd.shape
    Y = np.zeros((T, d), dtype=np.float64)
    S = tw.tile_slots
    for t in range(T):
        for j in range(tw.n_tiles):
            for s in range(min(int(tw.cnt[t, j]), S)):
                n = int(tw.idx[t, j * S + s])
                g = _tw.stored_to_f64(tw.val[t, j * S + s], tw.val_dtype)
                u = Xd[t] @ Wu[:, n]
                Y[t] += (g * u) * Wd[n]
    return Y


def ffn_hybrid_forward(X, W_up, W_down, bias_f, shift_t, *, tile_cols, tile_slots, ell_width,
                       val_dtype="f32", ovf_capacity=None):
    """The whole non-gated hot path as the oracle computes it.

    Steps: pre-activation (fp64), TwELL extraction (Alg. 1) with the storage cast,
    hybrid classification (Sec. 3.4), Alg. 3 - ELL rows by a gather of W_down rows,
    dense-backup rows by the dense product of their fp64 ReLU rows. When more rows
    overflow than `ovf_capacity`, only the first `ovf_capacity` dense-backup rows
    are computed and the rest of Y stays NaN (their output is unspecified).
    Returns (Y, twell, hybrid, Z).
    """
    Wd = np.asarray(W_down, dtype=np.float64)
    Z = preactivation(X, W_up, bias_f, shift_t)
    tw = _tw.extract_twell(Z, tile_cols, tile_slots, val_dtype)
    hy = _tw.classify(tw, ell_width)
    T, d = Z.shape[0], Wd.shape[1]
    Y = np.zeros((T, d), dtype=np.float64)
    for t in np.nonzero(~hy.is_ovf)[0]:
        c = int(hy.ell_cnt[t])
        if c:
            v = _tw.stored_to_f64(hy.ell_val[t, :c], val_dtype)
            Y[t] = v @ Wd[hy.ell_idx[t, :c].astype(np.int64)]
    cap = len(hy.ovf_rows) if ovf_capacity is None else min(ovf_capacity, len(hy.ovf_rows))
    dense_rows = hy.ovf_rows[:cap]
    if len(dense_rows):
        Y[dense_rows] = relu(Z[dense_rows]) @ Wd
    Y[hy.ovf_rows[cap:]] = np.nan
    return Y, tw, hy, Z


def l1_penalty(H, lam, n_layers=1):
    """eq. l1 for one layer: lam * (1/L) * (1/(T f)) * sum |h|."""
    T, f = H.shape
    return lam / n_layers * np.abs(H).sum() / (T * f)


def ffn_backward(X, W_up, W_down, dY, H, active, lam):
    """Gradients of  sum(dY * Y) + l1_penalty(H, lam)  for the non-gated ReLU FFN.

    Chain rule through h = ReLU(z) on the given activity pattern `active`
    (bool [T,f]); H holds the activation values (0 off the pattern):
      dH = dY W_down^T + lam/(T f) on active entries, dZ = dH on the pattern,
      dW_down = H^T dY, dW_up = X^T dZ, dX = dZ W_up^T
    (the non-gated case of eq. sec3:eq:all_other_gradients).
    Returns (dX, dW_up, dW_down, dZ).
    """
    X = np.asarray(X, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    T, f = H.shape
    dH = dY @ Wd.T + lam / (T * f)
    dZ = np.where(active, dH, 0.0)
    return dZ @ Wu.T, X.T @ dZ, H.T @ dY, dZ


def ffn_gated_backward(X, W_gate, W_up, W_down, dY, G, U, lam):
    """Gradients for the gated FFN (eq. sec3:eq:all_other_gradients) with the L1 term on h.

    h_g = ReLU(G), h_u = U, h = h_g * h_u. dh = dY W_down^T + lam/(T f) sign(h);
    dh_u = dh * h_g; dh_g = dh * h_u, passed through the ReLU to dG = dh_g [G > 0];
    dW_up = X^T dh_u, dW_gate = X^T dG, dW_down = h^T dY, dX = dh_u W_up^T + dG W_gate^T.
    Returns (dX, dW_gate, dW_up, dW_down).
    """
    X = np.asarray(X, dtype=np.float64)
    Wg = np.asarray(W_gate, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    hg = relu(G)
    h = hg * U
    T, f = h.shape
    dh = dY @ Wd.T + lam / (T * f) * np.sign(h)
    dhu = dh * hg
    dG = np.where(G > 0, dh * U, 0.0)
    return dhu @ Wu.T + dG @ Wg.T, X.T @ dG, X.T @ dhu, h.T @ dY


# ---- the same gradients for chosen hidden units or tokens ---------------------------------
# Each hidden unit's weight gradients (column n of dW_up and dW_gate, row n of dW_down) need
# only that unit's column of the pre-activations, and each token's dX row only that token's
# row; the helpers below evaluate eq. sec3:eq:all_other_gradients on such a subset, so that
# a layer too large for the full fp64 products can still be checked unit by unit and row by
# row. `active` is the activity pattern of the subset (the unit passes exactly there);
# lam/(T f) uses the layer's full T (rows of X) and f (columns of W_up).

def ffn_backward_units(X, W_up, W_down, dY, units, active, lam, bias_f=None, shift_t=None):
    """Non-gated: (dW_up[:, units], dW_down[units, :]) on the pattern `active` [T, len(units)].

    z = X W_up[:, n] + b[n] + s, h = z on the pattern (0 elsewhere),
    dh = dY W_down[n]^T + lam/(T f), dz = dh on the pattern; dW_up[:, n] = X^T dz,
    dW_down[n] = h^T dY.
    """
    X = np.asarray(X, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    units = np.asarray(units, dtype=np.int64)
    T, f = X.shape[0], Wu.shape[1]
    Z = preactivation(X, Wu[:, units], None if bias_f is None else np.asarray(bias_f)[units], shift_t)
    H = np.where(active, Z, 0.0)
    dZ = np.where(active, dY @ Wd[units].T + lam / (T * f), 0.0)
    return X.T @ dZ, H.T @ dY


def ffn_backward_rows(X, W_up, W_down, dY, rows, active, lam):
    """Non-gated: dX[rows] on the pattern `active` [len(rows), f]: dz = (dY W_down^T + lam/(T f))
    on the pattern, dX = dz W_up^T."""
    X = np.asarray(X, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    T, f = X.shape[0], Wu.shape[1]
    dZ = np.where(active, dY[rows] @ Wd.T + lam / (T * f), 0.0)
    return dZ @ Wu.T


def ffn_gated_backward_units(X, W_gate, W_up, W_down, dY, units, active, lam, bias_f=None, shift_t=None):
    """Gated: (dW_gate[:, units], dW_up[:, units], dW_down[units, :]) on the gate pattern
    `active` [T, len(units)].

    g = X W_gate[:, n] + b[n] + s, h_g = g on the pattern (0 elsewhere), h_u = X W_up[:, n],
    h = h_g h_u; dh = dY W_down[n]^T + lam/(T f) sign(h); dh_u = dh h_g, dg = dh h_u on the
    pattern; dW_gate[:, n] = X^T dg, dW_up[:, n] = X^T dh_u, dW_down[n] = h^T dY.
    """
    X = np.asarray(X, dtype=np.float64)
    Wg = np.asarray(W_gate, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    units = np.asarray(units, dtype=np.int64)
    T, f = X.shape[0], Wu.shape[1]
    G = preactivation(X, Wg[:, units], None if bias_f is None else np.asarray(bias_f)[units], shift_t)
    U = X @ Wu[:, units]
    hg = np.where(active, G, 0.0)
    h = hg * U
    dh = dY @ Wd[units].T + lam / (T * f) * np.sign(h)
    dG = np.where(active, dh * U, 0.0)
    return X.T @ dG, X.T @ (dh * hg), h.T @ dY


def ffn_gated_backward_rows(X, W_gate, W_up, W_down, dY, rows, active, lam, bias_f=None, shift_t=None):
    """Gated: dX[rows] on the gate pattern `active` [len(rows), f]:
    dX = dh_u W_up^T + dg W_gate^T with dh_u, dg as in ffn_gated_backward_units."""
    X = np.asarray(X, dtype=np.float64)
    Wg = np.asarray(W_gate, dtype=np.float64)
    Wu = np.asarray(W_up, dtype=np.float64)
    Wd = np.asarray(W_down, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    T, f = X.shape[0], Wu.shape[1]
    G = preactivation(X[rows], Wg, bias_f, None if shift_t is None else np.asarray(shift_t)[rows])
    U = X[rows] @ Wu
    hg = np.where(active, G, 0.0)
    h = hg * U
    dh = dY[rows] @ Wd.T + lam / (T * f) * np.sign(h)
    dG = np.where(active, dh * U, 0.0)
    return (dh * hg) @ Wu.T + dG @ Wg.T
