"""Pins for the oracle's TwELL extractor and hybrid classifier.

(i) brute force over every sign pattern of tiny rows, with expectations built from
integer bit operations (not from the scan the oracle uses); (ii) pack -> unpack
invariants; (iii) the T_n = f special case is ELLPACK-R, i.e. CSR with sorted
columns, checked against scipy.sparse."""
import numpy as np
import pytest
import scipy.sparse as sp

from oracle import twell


def pattern_rows(f, seed=0):
    """All 2^f sign patterns; active entries get distinct positive values, inactive
    entries cycle through -x, +0.0, -0.0 and NaN so that strictness is exercised."""
    rows = np.arange(2 ** f, dtype=np.int64)
    bits = (rows[:, None] >> np.arange(f)[None, :]) & 1
    mag = (np.arange(f, dtype=np.float64) + 1.0)[None, :] * (1.0 + rows[:, None] % 7 / 8.0)
    inactive_choices = np.stack([-mag, np.zeros_like(mag), -np.zeros_like(mag),
                                 np.full_like(mag, np.nan)], axis=0)
    pick = (rows[:, None] + np.arange(f)[None, :]) % 4
    inactive = np.take_along_axis(inactive_choices, pick[None], axis=0)[0]
    return np.where(bits == 1, mag, inactive), rows


def expected_from_bits(p, f, tile_cols, tile_slots):
    """Per tile: count = popcount of the tile's bits; slots = lowest set bits in order."""
    NT = -(-f // tile_cols)
    cnt, slots = [], []
    for j in range(NT):
        w = min(tile_cols, f - j * tile_cols)
        b = (p >> (j * tile_cols)) & ((1 << w) - 1)
        cnt.append(bin(b).count("1"))
        cols = []
        while b and len(cols) < tile_slots:
            low = b & -b
            cols.append(j * tile_cols + low.bit_length() - 1)
            b ^= low
        slots.append(cols)
    return cnt, slots


@pytest.mark.parametrize("f", [1, 2, 5, 8, 11])
@pytest.mark.parametrize("tile_cols,tile_slots", [(3, 1), (3, 2), (4, 2), (4, 3), (5, 3), (5, 1)])
def test_brute_force_sign_patterns(f, tile_cols, tile_slots):
    Z, rows = pattern_rows(f)
    tw_loop = twell.extract_twell_loops(Z, tile_cols, tile_slots, "f32")
    tw_vec = twell.extract_twell(Z, tile_cols, tile_slots, "f32", row_chunk=97)
    for tw in (tw_loop, tw_vec):
        for r, p in enumerate(rows):
            cnt, slots = expected_from_bits(int(p), f, tile_cols, tile_slots)
            assert list(tw.cnt[r]) == cnt
            for j, cols in enumerate(slots):
                got = tw.idx[r, j * tile_slots:j * tile_slots + len(cols)].tolist()
                assert got == cols
                np.testing.assert_array_equal(
                    tw.val[r, j * tile_slots:j * tile_slots + len(cols)],
                    Z[r, cols].astype(np.float32))
    # classification: row overflows iff popcount > K or some tile count > S
    for K in range(0, f + 1):
        hy = twell.classify(tw_vec, K)
        for r, p in enumerate(rows):
            cnt, _ = expected_from_bits(int(p), f, tile_cols, tile_slots)
            want = bin(int(p)).count("1") > K or max(cnt) > tile_slots
            assert bool(hy.is_ovf[r]) == want
            assert hy.row_nnz[r] == bin(int(p)).count("1")
        np.testing.assert_array_equal(hy.ovf_rows, np.nonzero(hy.is_ovf)[0])


def test_unpack_invariant_and_counts():
    r = np.random.default_rng(1)
    Z = r.standard_normal((37, 300)).astype(np.float32) - 1.5
    Z[3] = 5.0          # all-active row
    Z[4] = -1.0         # all-inactive row
    for dt in ("f32", "bf16"):
        tw = twell.extract_twell(Z, 300, 300, dt)  # S = T_n = f: nothing can be dropped
        H = twell.unpack_twell(tw, 300)
        want = np.where(Z > 0, Z, 0).astype(np.float64)
        if dt == "bf16":
            from oracle import bf16
            want = bf16.round_to_bf16_value(want)
        np.testing.assert_array_equal(H, want)
        assert tw.cnt.sum() == (Z > 0).sum()
    # multi-tile, S large enough: unpack is still exact; sum of counts still #active
    tw = twell.extract_twell(Z, 64, 64, "f32")
    np.testing.assert_array_equal(twell.unpack_twell(tw, 300), np.where(Z > 0, Z, 0))
    assert tw.cnt.sum() == (Z > 0).sum()


def test_ellpack_r_special_case_matches_csr():
    """T_n = f turns TwELL into ELLPACK-R; the hybrid row-ELL then equals CSR rows."""
    r = np.random.default_rng(2)
    Z = r.standard_normal((50, 97)) - 1.0
    tw = twell.extract_twell(Z, 97, 97, "f32")
    hy = twell.classify(tw, 97)
    csr = sp.csr_matrix(np.where(Z > 0, Z, 0.0).astype(np.float32))
    csr.sort_indices()
    for t in range(50):
        a, b = csr.indptr[t], csr.indptr[t + 1]
        assert tw.cnt[t, 0] == b - a == hy.ell_cnt[t]
        np.testing.assert_array_equal(tw.idx[t, :b - a], csr.indices[a:b])
        np.testing.assert_array_equal(hy.ell_idx[t, :b - a], csr.indices[a:b])
        np.testing.assert_array_equal(hy.ell_val[t, :b - a], csr.data[a:b])


def test_row_ell_is_tiles_concatenated_in_order():
    r = np.random.default_rng(3)
    Z = r.standard_normal((64, 1000)) - 2.0
    tw = twell.extract_twell(Z, 256, 32, "bf16")
    hy = twell.classify(tw, 64)
    for t in np.nonzero(~hy.is_ovf)[0]:
        cols = np.nonzero(Z[t] > 0)[0]
        np.testing.assert_array_equal(hy.ell_idx[t, :len(cols)], cols)
        assert hy.ell_cnt[t] == len(cols)


def test_pack32_hand_worked_words():
    """One tile of 40 columns: columns 1 (1.0 -> bf16 0x3F80) and 38 (-0.5 inactive) and
    39 (0.5 -> 0x3F00) give count 2, then 0x3F80_0001 and 0x3F00_0027; a second row with
    33 active columns keeps its true count 33 and only its first 31 entries."""
    Z = np.zeros((2, 40), dtype=np.float32)
    Z[0, 1], Z[0, 38], Z[0, 39] = 1.0, -0.5, 0.5
    Z[1, :33] = 2.0  # bf16 0x4000
    tw = twell.extract_twell_loops(Z, 40, 31, "bf16")
    w = twell.pack32(tw)
    assert w.shape == (2, 32)
    assert w[0, 0] == 2 and w[0, 1] == 0x3F800001 and w[0, 2] == 0x3F000027
    assert w[1, 0] == 33
    np.testing.assert_array_equal(w[1, 1:32], [0x40000000 | c for c in range(31)])


def test_pack32_round_trip_and_multi_tile():
    """unpack32(pack32(tw)) gives back the counts and every stored slot, over ragged tiles
    and rows whose tiles overflow."""
    r = np.random.default_rng(12)
    Z = r.standard_normal((9, 700)).astype(np.float32)
    Z[2, :300] = 1.0  # tiles over 31 slots
    tw = twell.extract_twell(Z, 256, 31, "bf16")
    back = twell.unpack32(twell.pack32(tw), 256)
    np.testing.assert_array_equal(back.cnt, tw.cnt)
    S = 31
    for j in range(tw.n_tiles):
        nv = np.minimum(tw.cnt[:, j], S)
        for s in range(S):
            rows = np.nonzero(nv > s)[0]
            np.testing.assert_array_equal(back.idx[rows, j * S + s], tw.idx[rows, j * S + s])
            np.testing.assert_array_equal(back.val[rows, j * S + s], tw.val[rows, j * S + s])
    with pytest.raises(ValueError):
        twell.pack32(twell.extract_twell(Z, 256, 32, "bf16"))
