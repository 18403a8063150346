"""Dead hidden units and their targeted re-initialisation, for the oracle.
TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper records, for every hidden unit of every layer, the last training step in
which the unit was non-zero, and calls a unit dead for a step when it was never active
during that step (extended results, sparsity and dead neurons during training). Its
mitigation (appendix on training modifications) pulls the gate-projection column of
every dead unit toward a fresh draw of the initial distribution:
W[:, j] <- (1 - lam) W[:, j] + lam N(0, sigma^2), with sigma the initialisation
standard deviation (0.02) and lam = 0.1 in its experiments.

* `active_units(Z)`          unit n is active in a batch iff some row has Z[t, n] > 0
                             (the strict test of the ReLU pattern; NaN is never > 0).
* `update_last_active(...)`  last[n] = step for the active units, unchanged otherwise.
* `dead_units(last, step)`   units with last[n] < step.
* `reinit_dead(...)`         the interpolation above for the dead units' columns (or
                             rows, for a transposed copy), in float64, with the
                             standard-normal draws passed in; bf16 results rounded to
                             nearest even by `oracle.bf16`.
"""
from __future__ import annotations

import numpy as np

from . import bf16 as _bf16


def active_units(Z) -> np.ndarray:
    """Boolean [f]: column n has a strictly positive entry in some row."""
    Z = np.asarray(Z, dtype=np.float64)
    if Z.shape[0] == 0:
        return np.zeros(Z.shape[1], dtype=bool)
    return (Z > 0).any(axis=0)


def update_last_active(last, active, step) -> np.ndarray:
    last = np.asarray(last, dtype=np.int64)
    return np.where(np.asarray(active, dtype=bool), np.int64(step), last)


def dead_units(last, step) -> np.ndarray:
    return np.asarray(last, dtype=np.int64) < np.int64(step)


def reinit_dead(W, dead, lam, sigma, noise, units_on_rows=False, bf16_out=False) -> np.ndarray:
    """Float64 result of W with every dead unit's column (row when units_on_rows)
    replaced by (1 - lam) W + lam * sigma * noise. `dead` is a boolean per unit, `noise`
    has W's shape. With bf16_out the result is rounded to bf16 values."""
    W = np.asarray(W, dtype=np.float64)
    noise = np.asarray(noise, dtype=np.float64)
    dead = np.asarray(dead, dtype=bool)
    mask = dead[:, None] if units_on_rows else dead[None, :]
    out = np.where(mask, (1.0 - lam) * W + lam * sigma * noise, W)
    return _bf16.round_to_bf16_value(out) if bf16_out else out
