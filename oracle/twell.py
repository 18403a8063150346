"""TwELL extraction, hybrid row classification and row-ELL (oracle side).

Format (Sec. 3.2 and Alg. 1): the f hidden columns are cut into N_T =
ceil(f / T_n) horizontal tiles of width T_n (the last may be partial). For
every row t and tile j the non-zeros of h = ReLU(z) are left-aligned in S =
T_n / C slots: `val[t, j*S + s]`, `idx[t, j*S + s]` (global column index) and
the count `cnt[t, j]`. These are the paper's h_v, h_I in R^{M x N/C} and h_nz
in R^{M x N_T}, row-major.

Readings taken where the paper leaves a choice:
* a column is active iff z > 0 strictly (Alg. 1's test); +0, -0 and NaN are
  inactive, +inf and positive subnormals are active;
* slots are filled in ascending column order (Alg. 1's scan order), which makes
  the output unique;
* `cnt` holds the true count even when it exceeds S; only the first S active
  columns are stored (nothing is wrapped);
* slots s >= min(cnt, S) are unspecified (this oracle leaves them 0);
* the stored value is the activation dtype: float32 unchanged, or bf16 rounded
  to nearest even from the float32/float64 pre-activation.

Hybrid classification (Sec. 3.4, "Hybrid Conversion for Efficient Storage"):
row t goes to the dense backup iff its true count row_nnz[t] exceeds the ELL
width K, or one of its tiles overflowed (cnt > S, so the TwELL lost entries).
The dense-backup rows are listed in ascending order. All other rows get a
compact ELL row: their tile slots concatenated in tile order, which is the
row's active columns in ascending order.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import bf16 as _bf16


@dataclass
class TwELL:
    val: np.ndarray   # [T, N_T*S]: uint16 bf16 bits, or float32
    idx: np.ndarray   # [T, N_T*S] uint16 global column
    cnt: np.ndarray   # [T, N_T] int32 true counts
    tile_cols: int
    tile_slots: int
    val_dtype: str    # "bf16" or "f32"

    @property
    def n_tiles(self):
        return self.cnt.shape[1]


def cast_value(z, val_dtype):
    """Storage cast of an activation value (exact widening of the result returned as float64)."""
    if val_dtype == "f32":
        return np.asarray(z, dtype=np.float32)
    return _bf16.to_bf16_bits(np.asarray(z, dtype=np.float64))


def stored_to_f64(val, val_dtype):
    if val_dtype == "f32":
        return np.asarray(val, dtype=np.float32).astype(np.float64)
    return _bf16.from_bf16_bits(val)


def n_tiles(f, tile_cols):
    return (f + tile_cols - 1) // tile_cols


def extract_twell_loops(Z, tile_cols, tile_slots, val_dtype="f32") -> TwELL:
    """Alg. 1 written as the plain scan: per row, per tile, per column ascending.

    Pure Python; meant for small inputs. `Z` holds pre-activations (float32 or float64).
    """
    Z = np.asarray(Z)
    T, f = Z.shape
    NT = n_tiles(f, tile_cols)
    S = tile_slots
    cnt = np.zeros((T, NT), dtype=np.int32)
    idx = np.zeros((T, NT * S), dtype=np.uint16)
    vals = np.zeros((T, NT * S), dtype=np.float64)
    present = np.zeros((T, NT * S), dtype=bool)
    for t in range(T):
        for j in range(NT):
            z_count = 0
            for c in range(j * tile_cols, min((j + 1) * tile_cols, f)):
                if Z[t, c] > 0:
                    if z_count < S:
                        idx[t, j * S + z_count] = c
                        vals[t, j * S + z_count] = Z[t, c]
                        present[t, j * S + z_count] = True
                    z_count += 1
            cnt[t, j] = z_count
    val = _cast_slots(vals, present, val_dtype)
    return TwELL(val, idx, cnt, tile_cols, tile_slots, val_dtype)


def _cast_slots(vals, present, val_dtype):
    if val_dtype == "f32":
        out = np.zeros(vals.shape, dtype=np.float32)
        out[present] = vals[present].astype(np.float32)
        return out
    out = np.zeros(vals.shape, dtype=np.uint16)
    out[present] = cast_value(vals[present], "bf16")
    return out


def extract_twell(Z, tile_cols, tile_slots, val_dtype="f32", row_chunk=256) -> TwELL:
    """Same result as `extract_twell_loops`, vectorised over rows for large inputs.

    Within a tile, the rank of an active column is the number of active columns
    before it in that tile; it is stored iff rank < S.
    """
    Z = np.asarray(Z)
    T, f = Z.shape
    NT = n_tiles(f, tile_cols)
    S = tile_slots
    cnt = np.zeros((T, NT), dtype=np.int32)
    idx = np.zeros((T, NT * S), dtype=np.uint16)
    val = np.zeros((T, NT * S), dtype=np.float32 if val_dtype == "f32" else np.uint16)
    pad = NT * tile_cols - f
    for r0 in range(0, T, row_chunk):
        zc = Z[r0:r0 + row_chunk]
        act = zc > 0
        if pad:
            act = np.concatenate([act, np.zeros((act.shape[0], pad), dtype=bool)], axis=1)
        act = act.reshape(act.shape[0], NT, tile_cols)
        rank = np.cumsum(act, axis=2, dtype=np.int32) - 1
        cnt[r0:r0 + row_chunk] = act.sum(axis=2, dtype=np.int32)
        keep = act & (rank < S)
        ti, tj, tc = np.nonzero(keep)
        slot = rank[ti, tj, tc]
        col = tj * tile_cols + tc
        idx[r0 + ti, tj * S + slot] = col.astype(np.uint16)
        val[r0 + ti, tj * S + slot] = cast_value(zc[ti, col], val_dtype)
    return TwELL(val, idx, cnt, tile_cols, tile_slots, val_dtype)


def unpack_twell(tw: TwELL, f) -> np.ndarray:
    """Dense float64 H rebuilt from the stored slots (entries beyond S are lost)."""
    T = tw.cnt.shape[0]
    S = tw.tile_slots
    H = np.zeros((T, f), dtype=np.float64)
    for j in range(tw.n_tiles):
        n_valid = np.minimum(tw.cnt[:, j], S)
        for s in range(S):
            rows = np.nonzero(n_valid > s)[0]
            cols = tw.idx[rows, j * S + s].astype(np.int64)
            H[rows, cols] = stored_to_f64(tw.val[rows, j * S + s], tw.val_dtype)
    return H


@dataclass
class Hybrid:
    row_nnz: np.ndarray    # [T] int32 true counts
    is_ovf: np.ndarray     # [T] bool: dense-backup row (h_b)
    ovf_rows: np.ndarray   # ascending int32 list of dense-backup rows (pi_d)
    n_tile_ovf: int        # number of (row, tile) pairs with cnt > S
    ell_cnt: np.ndarray    # [T] int32: ELL row length (0 for dense-backup rows)
    ell_idx: np.ndarray    # [T, K] uint16
    ell_val: np.ndarray    # [T, K] stored dtype


def classify(tw: TwELL, ell_width) -> Hybrid:
    """Route rows to the compact ELL or the dense backup from the TwELL counts."""
    S = tw.tile_slots
    K = ell_width
    T = tw.cnt.shape[0]
    row_nnz = tw.cnt.sum(axis=1, dtype=np.int64).astype(np.int32)
    tile_over = tw.cnt > S
    is_ovf = (row_nnz > K) | tile_over.any(axis=1)
    ovf_rows = np.nonzero(is_ovf)[0].astype(np.int32)
    ell_cnt = np.where(is_ovf, 0, row_nnz).astype(np.int32)
    ell_idx = np.zeros((T, K), dtype=np.uint16)
    ell_val = np.zeros((T, K), dtype=tw.val.dtype)
    for t in np.nonzero(~is_ovf)[0]:
        pos = 0
        for j in range(tw.n_tiles):
            c = int(tw.cnt[t, j])
            ell_idx[t, pos:pos + c] = tw.idx[t, j * S:j * S + c]
            ell_val[t, pos:pos + c] = tw.val[t, j * S:j * S + c]
            pos += c
    return Hybrid(row_nnz, is_ovf, ovf_rows, int(tile_over.sum()), ell_cnt, ell_idx, ell_val)


# ---- packed 32-bit TwELL (the paper's single-load inference format) ----------------------
# Appendix A's inference kernels keep each (row, tile) as one run of 32-bit words: the count
# in word 0, then one word per stored entry holding the column index and the value, so a
# tile's slots are one contiguous 128-byte load and 31 slots are usable. Here: 32 words per
# (row, tile); word 0 = the true count (may exceed 31); word 1 + s (s < min(count, 31)) =
# global column index in the low 16 bits | bf16 value bits in the high 16 bits. Words past
# the stored entries are unspecified (this oracle leaves them 0).
PACK32_WORDS = 32
PACK32_SLOTS = PACK32_WORDS - 1


def pack32(tw: TwELL) -> np.ndarray:
    """uint32 [T, N_T * 32] from a bf16 TwELL extracted with tile_slots = 31."""
    if tw.tile_slots != PACK32_SLOTS or tw.val_dtype != "bf16":
        raise ValueError("packed-32 TwELL holds 31 bf16 slots per tile")
    T, NT = tw.cnt.shape
    words = np.zeros((T, NT * PACK32_WORDS), dtype=np.uint32)
    for j in range(NT):
        base = j * PACK32_WORDS
        words[:, base] = tw.cnt[:, j].astype(np.int64).astype(np.uint32)
        n_valid = np.minimum(tw.cnt[:, j], PACK32_SLOTS)
        for s in range(PACK32_SLOTS):
            rows = np.nonzero(n_valid > s)[0]
            col = tw.idx[rows, j * PACK32_SLOTS + s].astype(np.uint32)
            val = tw.val[rows, j * PACK32_SLOTS + s].astype(np.uint32)
            words[rows, base + 1 + s] = col | (val << np.uint32(16))
    return words


def unpack32(words, tile_cols) -> TwELL:
    """The TwELL (31 bf16 slots per tile) that a packed-32 array encodes."""
    words = np.asarray(words, dtype=np.uint32)
    T = words.shape[0]
    NT = words.shape[1] // PACK32_WORDS
    S = PACK32_SLOTS
    cnt = words[:, ::PACK32_WORDS].astype(np.int64).astype(np.int32)
    idx = np.zeros((T, NT * S), dtype=np.uint16)
    val = np.zeros((T, NT * S), dtype=np.uint16)
    for j in range(NT):
        n_valid = np.minimum(cnt[:, j], S)
        for s in range(S):
            rows = np.nonzero(n_valid > s)[0]
            w = words[rows, j * PACK32_WORDS + 1 + s]
            idx[rows, j * S + s] = (w & np.uint32(0xFFFF)).astype(np.uint16)
            val[rows, j * S + s] = (w >> np.uint32(16)).astype(np.uint16)
    return TwELL(val, idx, cnt, tile_cols, S, "bf16")
