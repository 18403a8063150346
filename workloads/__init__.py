"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module only draws random numbers and rounds them to the storage dtype;
it holds none of the FFN method's arithmetic. Every array it returns is in
its *stored* form: float32 arrays for fp32 configs, and uint16 bf16 bit
patterns for bf16 configs (`bf16_bits_from_f32` rounds to nearest-even).

The paper trains on a text corpus that is not available here, so its hidden
activation statistics are stood in for by per-row pre-activation shifts on
Gaussian weights (see `row_shift_for_sparsity`): with iid N(0, sigma_w^2)
weight columns, Z[t, n] given X_t is N(0, sigma_w^2 |X_t|^2), so a shift of
-sigma_w |X_t| Phi^-1(s) makes every hidden unit of row t independently
active with probability 1 - s.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
from scipy.stats import norm

SIGMA_W = 0.02  # weight std (the paper's initializer range, Appendix B table)


def rng(seed: int, stream: int = 0) -> np.random.Generator:
    """NumPy PCG64 generator; `stream` separates independent tensors."""
    return np.random.Generator(np.random.PCG64([seed, stream]))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns uint16 bits.

    NaN inputs become a quiet NaN. Used only to store generated inputs.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal(shape, std, seed, stream) -> np.ndarray:
    return (rng(seed, stream).standard_normal(size=shape, dtype=np.float32) * np.float32(std))


def row_shift_for_sparsity(x_stored_f32: np.ndarray, sparsity) -> np.ndarray:
    """Per-row pre-activation shift giving each hidden unit P(active) = 1 - sparsity.

    `sparsity` is a scalar or a per-row array. Returns float32 [T].
    """
    norms = np.sqrt((x_stored_f32.astype(np.float64) ** 2).sum(axis=1))
    q = norm.ppf(np.asarray(sparsity, dtype=np.float64))
    return (-SIGMA_W * norms * q).astype(np.float32)


@dataclass
class Workload:
    """One synthetic FFN problem in stored form (see module docstring)."""

    name: str
    dtype: str  # "f32" or "bf16"
    T: int
    d: int
    f: int
    gated: bool
    X: np.ndarray
    W_up: np.ndarray
    W_down: np.ndarray
    W_gate: np.ndarray | None = None
    bias_f: np.ndarray | None = None  # float32 [f] or None
    shift_t: np.ndarray | None = None  # float32 [T] or None
    dY: np.ndarray | None = None  # stored like X, training configs only
    cfg: dict = field(default_factory=dict)  # tile_rows, tile_cols, tile_slots, ell_width, ovf_capacity
    notes: str = ""

    def as_f32(self, a):
        """Stored array -> float32 values (exact)."""
        if a is None:
            return None
        return f32_from_bf16_bits(a) if self.dtype == "bf16" else a

    def as_f64(self, a):
        if a is None:
            return None
        return self.as_f32(a).astype(np.float64)


def _store(x, dtype):
    return bf16_bits_from_f32(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_ffn(name, dtype, T, d, f, *, seed=0, gated=False, sparsity=None, sparsity_rows=None,
             bias_value=None, tile_rows=32, tile_cols=256, tile_slots=32, ell_width=128,
             ovf_capacity=0, with_dy=False, notes="") -> Workload:
    """Generic generator: X ~ N(0,1), weights ~ N(0, 0.02^2), optional uniform bias or row shifts.

    `sparsity` (scalar) or `sparsity_rows` (per-row array) set the row shift of the
    pattern-deciding projection (W_up, or W_gate when gated).
    """
    X = _store(normal((T, d), 1.0, seed, 1), dtype)
    W_up = _store(normal((d, f), SIGMA_W, seed, 2), dtype)
    W_down = _store(normal((f, d), SIGMA_W, seed, 3), dtype)
    W_gate = _store(normal((d, f), SIGMA_W, seed, 4), dtype) if gated else None
    Xf = f32_from_bf16_bits(X) if dtype == "bf16" else X
    shift = None
    if sparsity_rows is not None:
        shift = row_shift_for_sparsity(Xf, sparsity_rows)
    elif sparsity is not None:
        shift = row_shift_for_sparsity(Xf, sparsity)
    bias = None if bias_value is None else np.full((f,), bias_value, dtype=np.float32)
    dY = _store(normal((T, d), 1.0, seed, 5), dtype) if with_dy else None
    cfg = dict(tile_rows=tile_rows, tile_cols=tile_cols, tile_slots=tile_slots,
               ell_width=ell_width, ovf_capacity=ovf_capacity)
    return Workload(name, dtype, T, d, f, gated, X, W_up, W_down, W_gate, bias, shift, dY, cfg, notes)


# ---- the five named workloads -------------------------------------------------------------

def c1_small_fp32(seed=0):
    """fp32 T=64 d=256 f=1024; bias -2.5 sigma_Z = -2.5*0.02*sqrt(256) = -0.8 (~0.6% active)."""
    return make_ffn("fp32 T=64 d=256 f=1024 bias=-0.8", "f32", 64, 256, 1024, seed=seed,
                    bias_value=-2.5 * SIGMA_W * math.sqrt(256), tile_rows=16, ell_width=32)


def lognormal_row_counts(T, f, seed, mean=80.0, sigma=0.8, lo=1, hi=1000):
    mu = math.log(mean) - sigma * sigma / 2
    n = rng(seed, 6).lognormal(mean=mu, sigma=sigma, size=T)
    n = np.clip(n, lo, hi)
    return 1.0 - n / f


def c2_lognormal(seed=0, T=4096, d=2048, f=8192):
    """bf16 T=4096 d=2048 f=8192; per-row active counts ~ lognormal(mean 80), clipped to [1,1000]."""
    return make_ffn(f"bf16 T={T} d={d} f={f} lognormal-rows", "bf16", T, d, f, seed=seed,
                    sparsity_rows=lognormal_row_counts(T, f, seed), tile_rows=32, ell_width=128)


def gated_training(seed=0, T=8192, d=4096, f=14336, sparsity=0.995):
    """Training step of the gated block at the gated forward's shape: dY ~ N(0, 1), dense
    backup sized to T/8 rows (the paper's choice for its training runs)."""
    return make_ffn(f"gated train bf16 T={T} d={d} f={f} s={sparsity}", "bf16", T, d, f, seed=seed,
                    gated=True, sparsity=sparsity, tile_rows=32, ell_width=128, ovf_capacity=T // 8,
                    with_dy=True)


def c3_gated(seed=0, T=8192, d=4096, f=14336, sparsity=0.995):
    return make_ffn(f"gated bf16 T={T} d={d} f={f} s={sparsity}", "bf16", T, d, f, seed=seed,
                    gated=True, sparsity=sparsity, tile_rows=32, ell_width=128)


# ELL width K and tile slots S per sparsity level for the d=4096/f=16384 sweep:
# K = ceil((mean + 6 sd)/64)*64 of Binomial(16384, 1-s); S keeps tile overflow negligible.
SWEEP_PARAMS = {0.90: (1920, 64), 0.95: (1024, 48), 0.99: (256, 32), 0.999: (64, 32)}


def c4_sweep(sparsity=0.99, seed=0, T=8192, d=4096, f=16384, ell_width=None, tile_slots=None):
    K, S = SWEEP_PARAMS.get(sparsity, (256, 32))
    return make_ffn(f"bf16 T={T} d={d} f={f} s={sparsity}", "bf16", T, d, f, seed=seed,
                    sparsity=sparsity, tile_rows=32, tile_slots=tile_slots or S,
                    ell_width=ell_width or K)


def c4_shard(kind, T=8192, d=4096, f=16384, sparsity=0.99):
    """One GPU's share of the 99 % layer when it runs on eight GPUs: hidden units split
    eight ways (kind "tp8": f/8 units, K = ceil((mean + 6 sd)/64)*64 of Binomial(f/8, 1-s))
    or tokens split eight ways (kind "dp8": T/8 tokens, the full layer's K)."""
    if kind == "tp8":
        fs = f // 8
        mean, sd = fs * (1 - sparsity), math.sqrt(fs * sparsity * (1 - sparsity))
        K = int(math.ceil((mean + 6 * sd) / 64) * 64)
        w = c4_sweep(sparsity, T=T, d=d, f=fs, ell_width=K)
    elif kind == "dp8":
        w = c4_sweep(sparsity, T=T // 8, d=d, f=f)
    else:
        raise ValueError(kind)
    w.name = f"{kind} shard of the {int(round(sparsity * 100))} % layer: " + w.name
    return w


def c5_training(seed=0, T=16384, d=4096, f=16384, sparsity=0.99):
    return make_ffn(f"train bf16 T={T} d={d} f={f} s={sparsity}", "bf16", T, d, f, seed=seed,
                    sparsity=sparsity, tile_rows=32, tile_slots=32, ell_width=256, with_dy=True)
