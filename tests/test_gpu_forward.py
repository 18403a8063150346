"""sfl_ffn_forward / sfl_dense_ffn_baseline on the GPU against the fp64 oracle.

Bars: relative L2 <= 2e-2 for bf16 and <= 1e-5 for fp32 (against the oracle's dense
definition on the same stored inputs); the fused TwELL output is bit-identical to
sfl_pack_twell applied to the float32 pre-activations of the same GEMM main loop; the
pattern matches the oracle's except where |z| is within rounding of 0."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import bf16, ffn, twell
from tests.gpu_util import assert_twell_equal, dev, host_bits, rel_l2, to_f64, twell_views

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")


def transposed(W):
    out = torch.empty((W.shape[1], W.shape[0]), dtype=W.dtype, device="cuda")
    b.sfl_transpose(W, out)
    return out


def run_forward(w, rows_check=None, use_wupt=False, dense=False, packed_down=False, use_wgatet=False,
                use_wdownt=False, packed_up=False):
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    Wg = dev(w.W_gate) if w.gated else None
    cfg = b.make_cfg(**w.cfg)
    dt = "bf16" if w.dtype == "bf16" else "f32"
    bufs = b.alloc_twell(w.T, w.f, dt, cfg)
    Y = torch.full((w.T, w.d), float("nan"), dtype=X.dtype, device="cuda")
    stats = b.alloc_stats()
    WupT = transposed(Wu) if use_wupt else None
    WgT = transposed(Wg) if use_wgatet else None
    WdT = transposed(Wd) if use_wdownt else None
    WdP = None
    if packed_down:
        WdP = torch.empty_like(Wd)
        b.sfl_pack_down_weights(Wd, WdP)
    WuP = None
    if packed_up:
        WuP = torch.empty_like(Wu)
        b.sfl_pack_down_weights(transposed(Wu), WuP)
    kw = dict(Y=Y, bufs=bufs, W_gate=Wg, W_upT=WupT, W_gateT=WgT, W_downT=WdT, W_down_packed=WdP, W_up_packed=WuP,
              bias_f=dev(w.bias_f), shift_t=dev(w.shift_t), stats=stats)
    args = b.ffn_args(X, Wu, Wd, cfg, **kw)
    ws_bytes = b.sfl_workspace_size(args, 2 if dense else 0)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws)
    (b.sfl_dense_ffn_baseline if dense else b.sfl_ffn_forward)(args)
    torch.cuda.synchronize()
    return Y, bufs, stats, cfg


def oracle_rows(w, rows):
    X = w.as_f64(w.X)[rows]
    sh = None if w.shift_t is None else w.shift_t[rows]
    if w.gated:
        Y, G, U, H = ffn.ffn_gated_dense(X, w.as_f64(w.W_gate), w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, sh)
        return Y, G
    Y, Z, H = ffn.ffn_dense(X, w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, sh)
    return Y, Z


def check_pattern(got, Zref, rows, f, Tn, S):
    """GPU pattern vs the oracle's z > 0, allowing flips only where |z| <= 1e-4 * rms(z)."""
    tol = 1e-4 * np.sqrt(np.mean(Zref ** 2))
    NT = -(-f // Tn)
    for i, t in enumerate(rows):
        want = Zref[i] > 0
        ambiguous = np.abs(Zref[i]) <= tol
        cnt = got["cnt"][t]
        gpu = np.zeros(f, dtype=bool)
        for j in range(NT):
            c = min(int(cnt[j]), S)
            gpu[got["idx"][t, j * S:j * S + c].astype(np.int64)] = True
        full = cnt <= S
        for j in np.nonzero(full)[0]:
            sl = slice(j * Tn, min((j + 1) * Tn, f))
            bad = (gpu[sl] != want[sl]) & ~ambiguous[sl]
            assert not bad.any(), (t, j, np.nonzero(bad)[0])


def sample_rows(T, n, seed, extra=()):
    r = np.random.default_rng(seed)
    rows = r.choice(T, size=min(n, T), replace=False)
    return np.unique(np.concatenate([rows, np.asarray(extra, dtype=np.int64)])).astype(np.int64)


def test_c1_fp32_full():
    w = wl.c1_small_fp32()
    Y, bufs, stats, cfg = run_forward(w)
    Yref, Z = oracle_rows(w, np.arange(w.T))
    assert rel_l2(to_f64(Y), Yref) <= 1e-5
    got = twell_views(bufs, w.T, w.f, cfg)
    check_pattern(got, Z, np.arange(w.T), w.f, cfg.tile_cols, cfg.tile_slots)
    # all rows computed exactly once: rows with no active unit are exactly zero
    zero_rows = (Z > 0).sum(1) == 0
    assert (to_f64(Y)[zero_rows] == 0).all()


def test_c2_lognormal_overflow_full():
    w = wl.c2_lognormal()
    Y, bufs, stats, cfg = run_forward(w)
    got = twell_views(bufs, w.T, w.f, cfg)
    st = b.read_stats(stats)
    n_ovf = got["n_ovf"]
    assert 0.08 * w.T < n_ovf < 0.3 * w.T, n_ovf   # the dense-backup path is exercised
    assert st["n_ovf_rows"] == n_ovf and st["capacity_exceeded"] == 0
    # both ways of forming dense-backup rows are exercised: rebuilt from the TwELL slabs
    # (every tile kept its values) and recomputed (some tile overflowed)
    tile_ovf_rows = (got["cnt"] > cfg.tile_slots).any(axis=1)
    assert 0 < tile_ovf_rows.sum() < n_ovf, tile_ovf_rows.sum()
    rows = np.arange(w.T)
    Yref, Z = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    ovf = np.nonzero(got["row_ovf"])[0]
    assert rel_l2(to_f64(Y)[ovf], Yref[ovf]) <= 2e-2
    np.testing.assert_array_equal(got["ovf_rows"][:n_ovf], ovf)
    prow = sample_rows(w.T, 64, 1)
    check_pattern(got, Z[prow], prow, w.f, cfg.tile_cols, cfg.tile_slots)


@pytest.mark.parametrize("sparsity,fallback", [(0.9, None), (0.95, None), (0.95, "off"), (0.99, None),
                                               (0.999, None)])
def test_c4_sweep_sampled(sparsity, fallback, monkeypatch):
    """The sparsity sweep at full size (90 % and 95 % take the dense fallback by default; 95 %
    is also run with it disabled, through the long-row gather)."""
    if fallback:
        monkeypatch.setenv("SFL_DENSE_FALLBACK", fallback)
    w = wl.c4_sweep(sparsity)
    Y, bufs, stats, cfg = run_forward(w)
    got = twell_views(bufs, w.T, w.f, cfg)
    ovf = np.nonzero(got["row_ovf"])[0]
    rows = sample_rows(w.T, 192, 2, extra=ovf[:64])
    Yref, Z = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y)[rows], Yref) <= 2e-2
    for i, t in enumerate(rows):
        assert rel_l2(to_f64(Y)[t], Yref[i]) <= 2e-2
    check_pattern(got, Z, rows[:48], w.f, cfg.tile_cols, cfg.tile_slots)
    realised = 1 - got["row_nnz"].sum() / (w.T * w.f)
    assert abs(realised - sparsity) < 0.1 * (1 - sparsity) + 1e-4


@pytest.mark.parametrize("use_wupt", [False, True])
@pytest.mark.parametrize("T,f,Tn,S", [(777, 2048, 256, 32), (300, 1984, 128, 16), (129, 1088, 64, 16),
                                       (32, 4096, 256, 32)])
def test_fused_twell_equals_pack_of_same_mainloop(T, f, Tn, S, use_wupt):
    """The TwELL the GEMM epilogue writes equals the oracle's extraction from the float32
    pre-activations of the same GEMM main loop (sfl_up_projection), bit for bit; with W_up
    (row-contiguous B) and with W_up^T (K-contiguous B, the direct-to-LDS GEMM), for TwELL
    tiles narrower than, equal to and wider than one wave's columns, and ragged T and f.
    Small batches with W_up^T (T <= 256) take the split-K GEMM + standalone pack instead."""
    w = wl.make_ffn("fused-vs-pack", "bf16", T, 512, f, seed=7 + T, sparsity=0.97, tile_cols=Tn, tile_slots=S,
                    ell_width=128)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=use_wupt)
    X, Wu = dev(w.X), dev(w.W_up)
    WupT = None
    if use_wupt:
        WupT = torch.empty((w.f, w.d), dtype=X.dtype, device="cuda")
        b.sfl_transpose(Wu, WupT)
    Z = torch.empty((w.T, w.f), dtype=torch.float32, device="cuda")
    args = b.ffn_args(X, Wu, dev(w.W_down), cfg, shift_t=dev(w.shift_t), W_upT=WupT)
    ws = torch.empty(max(1, b.sfl_workspace_size(args, 0)), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, dev(w.W_down), cfg, shift_t=dev(w.shift_t), W_upT=WupT, workspace=ws)
    b.sfl_up_projection(args, Z)
    bufs2 = b.alloc_twell(w.T, w.f, "bf16", cfg)
    b.sfl_pack_twell(Z, "bf16", cfg, bufs2)
    torch.cuda.synchronize()
    g1 = twell_views(bufs, w.T, w.f, cfg)
    tw = twell.extract_twell(Z.cpu().numpy(), cfg.tile_cols, cfg.tile_slots, "bf16")
    hy = twell.classify(tw, cfg.ell_width)
    assert_twell_equal(g1, tw, hy)                       # fused epilogue == oracle on the same z
    assert_twell_equal(twell_views(bufs2, w.T, w.f, cfg), tw, hy)
    # the float32 pre-activations themselves match the fp64 oracle closely
    Zref = ffn.preactivation(w.as_f64(w.X), w.as_f64(w.W_up), None, w.shift_t)
    assert rel_l2(Z.cpu().numpy(), Zref) < 1e-5
    rows = sample_rows(T, 64, 3)
    Yref, _ = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y)[rows], Yref) <= 2e-2


@pytest.mark.parametrize("Tn,S,packed", [(256, 32, False), (128, 16, False), (64, 8, False), (256, 31, True)])
def test_rebuilt_dense_backup_rows_bit_exact(Tn, S, packed):
    """Above 256 tokens the dense-backup rows whose tiles all kept their values are rebuilt
    from the TwELL slabs: each equals the oracle's bf16 ReLU of the float32 pre-activations
    of the same main loop (sfl_up_projection), bit for bit, for three TwELL tile widths and
    the packed 32-bit layout. The rows with an overflowing tile are recomputed by the
    split-K GEMM (another summation order): within 1e-2 per row of the same values."""
    T, f = 600, 2048
    sr = np.full(T, 0.99)
    sr[::7] = 0.5    # overflowing tiles
    sr[3::7] = 0.95  # more than K active units, no tile over S
    w = wl.make_ffn("rebuild", "bf16", T, 512, f, seed=Tn + S, sparsity_rows=sr, tile_cols=Tn, tile_slots=S,
                    ell_width=64)
    if packed:
        w.cfg["layout"] = b.SFL_TWELL_PACKED32
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True)
    X, Wu = dev(w.X), dev(w.W_up)
    Z = torch.empty((T, f), dtype=torch.float32, device="cuda")
    kw = dict(shift_t=dev(w.shift_t), W_upT=transposed(Wu))
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, dev(w.W_down), cfg, **kw), 0)), dtype=torch.uint8,
                     device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, dev(w.W_down), cfg, **kw, workspace=ws), Z)
    torch.cuda.synchronize()
    Zn = Z.cpu().numpy()
    tw = twell.extract_twell(Zn, Tn, S, "bf16")
    hy = twell.classify(tw, cfg.ell_width)
    n = int(host_bits(bufs["n_ovf"])[0])
    rows = host_bits(bufs["ovf_rows"])[:n]
    np.testing.assert_array_equal(rows, hy.ovf_rows)
    tile_over = (tw.cnt > S).any(axis=1)
    assert 0 < tile_over[rows].sum() < n  # both kinds of dense-backup row
    got = host_bits(bufs["ovf_dense"])[:n * f].reshape(n, f)
    zr = Zn[rows].astype(np.float64)
    want = np.where(zr > 0, bf16.to_bf16_bits(zr), np.uint16(0))
    rebuilt = ~tile_over[rows]
    np.testing.assert_array_equal(got[rebuilt], want[rebuilt])
    for i in np.nonzero(~rebuilt)[0]:
        assert rel_l2(bf16.from_bf16_bits(got[i]), bf16.from_bf16_bits(want[i])) <= 1e-2, rows[i]
    Yref, _ = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y)[rows], Yref[rows]) <= 2e-2


@pytest.mark.parametrize("order", ["grouped", "hilbert"])
@pytest.mark.parametrize("use_wupt", [False, True])
@pytest.mark.parametrize("T,f,Tn", [(2048, 16384, 256), (1800, 16320, 128)])
def test_fused_twell_bit_exact_over_several_tiles_per_block(T, f, Tn, use_wupt, order, monkeypatch):
    """The up projection's blocks are persistent (one per CU) and walk several 256 x 256
    output tiles each: 512 tiles at T = 2048, f = 16384 (two or more per block), 7 x 64
    ragged ones at T = 1800, f = 16320. While a tile's epilogue runs, the next tile's first
    stage, bias and shift are already loading into the other buffer. Every tile, second and
    later ones included, with a non-zero per-column bias and per-row shift: the fused TwELL
    is bit-identical to the oracle's extraction from the float32 pre-activations of the same
    main loop (sfl_up_projection), for W_up and for W_up^T, with the tiles dealt in the
    XCD-grouped order and along a Hilbert curve (32 x 64 tiles: two 32 x 32 squares; the
    ragged grid falls back to the grouped order)."""
    monkeypatch.setenv("SFL_GEMM_TILE_ORDER", order)
    w = wl.make_ffn("multi-tile", "bf16", T, 512, f, seed=T + Tn, sparsity=0.99, tile_cols=Tn, tile_slots=32,
                    ell_width=256)
    r = np.random.default_rng(T)
    w.bias_f = (r.standard_normal(f) * 0.02).astype(np.float32)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    WupT = transposed(Wu) if use_wupt else None
    cfg = b.make_cfg(**w.cfg)
    kw = dict(bias_f=dev(w.bias_f), shift_t=dev(w.shift_t), W_upT=WupT)
    Z = torch.empty((T, f), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw), 0)), dtype=torch.uint8,
                     device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws), Z)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=use_wupt)
    Zn = Z.cpu().numpy()
    tw = twell.extract_twell(Zn, Tn, cfg.tile_slots, "bf16")
    hy = twell.classify(tw, cfg.ell_width)
    assert tw.cnt.sum() > 0.005 * T * f
    assert_twell_equal(twell_views(bufs, T, f, cfg), tw, hy)
    rows = sample_rows(T, 32, 4, extra=[0, T - 1])
    Zref = ffn.preactivation(w.as_f64(w.X)[rows], w.as_f64(w.W_up), w.bias_f, w.shift_t[rows])
    assert rel_l2(Zn[rows], Zref) < 1e-5


@pytest.mark.parametrize("use_wupt", [False, True])
@pytest.mark.parametrize("T,f,Tn,S", [(600, 1088, 256, 32), (300, 704, 128, 16), (40, 960, 256, 32)])
def test_bias_and_shift_in_the_fused_epilogue(T, f, Tn, S, use_wupt):
    """A per-column bias and a per-row shift, with f not a multiple of the GEMM tile: the
    epilogue adds both to the accumulators (columns past f never active), bit-identical
    TwELL to the oracle's extraction from the same main loop's Z, Z and Y against fp64."""
    w = wl.make_ffn("bias", "bf16", T, 512, f, seed=T + f, sparsity=0.97, tile_cols=Tn, tile_slots=S,
                    ell_width=128)
    r = np.random.default_rng(T * 3 + f)
    w.bias_f = (r.standard_normal(f) * 0.05).astype(np.float32)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    WupT = transposed(Wu) if use_wupt else None
    cfg = b.make_cfg(**w.cfg)
    kw = dict(bias_f=dev(w.bias_f), shift_t=dev(w.shift_t), W_upT=WupT)
    Z = torch.empty((T, f), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw), 0)), dtype=torch.uint8,
                     device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws), Z)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=use_wupt)
    Zn = Z.cpu().numpy()
    Zref = ffn.preactivation(w.as_f64(w.X), w.as_f64(w.W_up), w.bias_f, w.shift_t)
    assert rel_l2(Zn, Zref) < 1e-5
    tw = twell.extract_twell(Zn, Tn, S, "bf16")
    assert_twell_equal(twell_views(bufs, T, f, cfg), tw, twell.classify(tw, cfg.ell_width))
    Yref, _ = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2


@pytest.mark.parametrize("copies", [False, True])
@pytest.mark.parametrize("gated", [False, True])
@pytest.mark.parametrize("T", [5, 48])
def test_small_batch_dense_backup_rows(T, gated, copies):
    """Batches of at most 64 rows with dense-backup rows (half the rows all active): with
    K-contiguous weight copies their GEMMs split K without a reduction kernel (the last
    block of each tile adds the partial sums, counted with per-tile counters); the gated
    layer's two products then run as one launch whose last blocks form h = ReLU(g) * u.
    Each dense-backup row of h against the oracle's (two bf16 roundings, fp32 sums: 1e-2
    per row), and Y. Two calls in a row, so the second starts from the counters the first
    left behind."""
    w = wl.make_ffn("small-ovf", "bf16", T, 1024, 2048, seed=T + 2 * gated, gated=gated, sparsity=0.97,
                    ell_width=128)
    w.shift_t[::2] = 100.0
    X = w.as_f64(w.X)
    if gated:
        _, _, _, H = ffn.ffn_gated_dense(X, w.as_f64(w.W_gate), w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f,
                                         w.shift_t)
    else:
        _, _, H = ffn.ffn_dense(X, w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, w.shift_t)
    Yref, _ = oracle_rows(w, np.arange(T))
    for _ in range(2):
        Y, bufs, stats, cfg = run_forward(w, use_wupt=copies, use_wgatet=copies and gated, use_wdownt=copies)
        got = twell_views(bufs, T, w.f, cfg)
        assert got["row_ovf"][::2].all() and not got["row_ovf"][1::2].any() and got["n_ovf"] == (T + 1) // 2
        assert rel_l2(to_f64(Y), Yref) <= 2e-2
        ovf = np.nonzero(got["row_ovf"])[0]
        assert rel_l2(to_f64(Y)[ovf], Yref[ovf]) <= 2e-2
        np.testing.assert_array_equal(got["ovf_rows"][:len(ovf)], ovf)
        dense_rows = to_f64(bufs["ovf_dense"])[:len(ovf) * w.f].reshape(len(ovf), w.f)
        for i, t in enumerate(ovf):
            assert rel_l2(dense_rows[i], H[t]) <= 1e-2, (i, t)


@pytest.mark.parametrize("copies", [False, True])
@pytest.mark.parametrize("gated", [False, True])
@pytest.mark.parametrize("T,every", [(100, 2), (100, 3), (600, 12), (600, 6)])
def test_counted_dense_backup_rows_above_64_tokens(T, every, gated, copies):
    """Batches above 64 tokens (dense-backup capacity T; the GEMMs' row count comes from
    the device) with a few dozen to a hundred dense-backup rows: every `every`-th row is
    all active, so 50, 34, 50 and 100 rows overflow (above 256 tokens the non-gated layer
    recomputes them through the need list). Y, each dense-backup row of h against the
    oracle's, and the L1 statistic; two calls in a row."""
    w = wl.make_ffn("counted-ovf", "bf16", T, 1024, 2048, seed=T + every + 2 * gated, gated=gated, sparsity=0.97,
                    ell_width=128)
    w.shift_t[::every] = 100.0
    X = w.as_f64(w.X)
    if gated:
        _, _, _, H = ffn.ffn_gated_dense(X, w.as_f64(w.W_gate), w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f,
                                         w.shift_t)
    else:
        _, _, H = ffn.ffn_dense(X, w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, w.shift_t)
    Yref, _ = oracle_rows(w, np.arange(T))
    n_ovf = -(-T // every)
    for _ in range(2):
        Y, bufs, stats, cfg = run_forward(w, use_wupt=copies, use_wgatet=copies and gated, use_wdownt=copies)
        got = twell_views(bufs, T, w.f, cfg)
        assert got["row_ovf"][::every].all() and got["n_ovf"] == n_ovf == int(got["row_ovf"].sum())
        assert rel_l2(to_f64(Y), Yref) <= 2e-2
        ovf = np.nonzero(got["row_ovf"])[0]
        assert rel_l2(to_f64(Y)[ovf], Yref[ovf]) <= 2e-2
        np.testing.assert_array_equal(got["ovf_rows"][:len(ovf)], ovf)
        dense_rows = to_f64(bufs["ovf_dense"])[:len(ovf) * w.f].reshape(len(ovf), w.f)
        for i, t in enumerate(ovf):
            assert rel_l2(dense_rows[i], H[t]) <= 1e-2, (i, t)
        # eq. l1 with lambda = 1, times T f: the sum of |h| (the bar of the L1 statistic tests)
        want = ffn.l1_penalty(H, 1.0) * T * w.f
        assert abs(b.read_stats(stats)["l1_sum"] - want) <= 5e-3 * want


@pytest.mark.parametrize("T,Tn,f", [(1, 256, 2048), (17, 256, 2048), (48, 256, 2048), (64, 256, 2048),
                                    (17, 64, 2048), (64, 128, 2048), (40, 64, 2048), (33, 128, 1984)])
def test_small_batch_split_gemm(T, Tn, f):
    """Batches of at most 64 rows with K-contiguous weights take the split-K GEMMs (K
    ranges over blocks, partial sums reduced in split order, by the TwELL pack in the
    forward): Z against the fp64 oracle, the forward's TwELL bit-identical to the oracle's
    extraction from that Z
    (TwELL tiles of 64, 128 and 256 columns; f = 1984 ends in a partial 256-column GEMM tile
    and a partial TwELL tile), Y of the sparse forward and of the dense baseline against
    the oracle."""
    w = wl.make_ffn("skinny", "bf16", T, 1024, f, seed=T + Tn, sparsity=0.97, tile_cols=Tn,
                    tile_slots=min(32, Tn), ell_width=128)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    WupT = transposed(Wu)
    cfg = b.make_cfg(**w.cfg)
    Z = torch.empty((T, w.f), dtype=torch.float32, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, shift_t=dev(w.shift_t), W_upT=WupT)
    ws = torch.empty(max(1, b.sfl_workspace_size(args, 0)), dtype=torch.uint8, device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, Wd, cfg, shift_t=dev(w.shift_t), W_upT=WupT, workspace=ws), Z)
    torch.cuda.synchronize()
    Zref = ffn.preactivation(w.as_f64(w.X), w.as_f64(w.W_up), None, w.shift_t)
    assert rel_l2(Z.cpu().numpy(), Zref) < 1e-5
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wdownt=True)
    tw = twell.extract_twell(Z.cpu().numpy(), cfg.tile_cols, cfg.tile_slots, "bf16")
    assert_twell_equal(twell_views(bufs, T, w.f, cfg), tw, twell.classify(tw, cfg.ell_width))
    Yref, _ = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    Yd, _, _, _ = run_forward(w, use_wupt=True, use_wdownt=True, dense=True)
    assert rel_l2(to_f64(Yd), Yref) <= 2e-2


@pytest.mark.parametrize("T,d,f,Tn,S,K", [(300, 256, 320, 256, 32, 40), (65, 128, 1024, 64, 8, 24),
                                            (1, 512, 2048, 128, 16, 64), (513, 64, 192, 64, 64, 192)])
def test_ragged_shapes_bf16(T, d, f, Tn, S, K):
    w = wl.make_ffn("ragged", "bf16", T, d, f, seed=T + f, sparsity=0.9, tile_cols=Tn, tile_slots=S, ell_width=K)
    Y, bufs, stats, cfg = run_forward(w)
    Yref, Z = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    check_pattern(twell_views(bufs, T, f, cfg), Z, np.arange(min(T, 64)), f, Tn, S)


def test_all_active_and_all_inactive_rows():
    w = wl.make_ffn("extremes", "bf16", 96, 256, 512, seed=3, sparsity=0.95, ell_width=32)
    w.shift_t[:8] = 100.0     # every unit active -> dense-backup rows
    w.shift_t[8:16] = -100.0  # no unit active -> exact zeros
    Y, bufs, stats, cfg = run_forward(w)
    Yref, Z = oracle_rows(w, np.arange(w.T))
    got = twell_views(bufs, w.T, w.f, cfg)
    assert got["row_ovf"][:8].all() and (got["row_nnz"][:8] == w.f).all()
    assert (to_f64(Y)[8:16] == 0).all()
    assert rel_l2(to_f64(Y), Yref) <= 2e-2


@pytest.mark.parametrize("T,d,copies", [(128, 256, False), (48, 512, True), (48, 512, False), (1536, 512, False)])
def test_capacity_exceeded_flag_then_enough_capacity(T, d, copies):
    """More dense-backup rows than the capacity: the flag, the count and the first `capacity`
    rows of the ascending list, which at most 64 rows with a slice-major gather are built by
    the gather's first block, from 1024 rows (tokens sorted by row count) by a second
    workgroup of the sort's launch, else by the list kernel; the entry total, which the
    classification's blocks leave to whichever of them builds the list."""
    w = wl.make_ffn("capacity", "bf16", T, d, 512, seed=4, sparsity=0.95, ell_width=16)
    w.shift_t[::4] = 100.0    # T / 4 dense-backup rows
    w.cfg["ovf_capacity"] = 10
    Y, bufs, stats, cfg = run_forward(w, use_wupt=copies, use_wdownt=copies)
    st = b.read_stats(stats)
    assert st["capacity_exceeded"] == 1 and st["n_ovf_rows"] >= T // 4
    got = twell_views(bufs, w.T, w.f, cfg)
    flagged = np.nonzero(got["row_ovf"])[0]
    assert got["n_ovf"] == st["n_ovf_rows"] == len(flagged)
    assert st["total_nnz"] == int(got["row_nnz"].astype(np.int64).sum())
    np.testing.assert_array_equal(got["ovf_rows"][:10], flagged[:10])  # ascending, the first `capacity`
    Yref, _ = oracle_rows(w, np.arange(w.T))
    done = got["ovf_rows"][:10]
    assert rel_l2(to_f64(Y)[done], Yref[done]) <= 2e-2
    sparse = np.nonzero(got["row_ovf"] == 0)[0]
    assert rel_l2(to_f64(Y)[sparse], Yref[sparse]) <= 2e-2
    w.cfg["ovf_capacity"] = 0
    Y2, _, stats2, _ = run_forward(w, use_wupt=copies, use_wdownt=copies)
    assert b.read_stats(stats2)["capacity_exceeded"] == 0
    assert rel_l2(to_f64(Y2), Yref) <= 2e-2


@pytest.mark.parametrize("T,copies,gated", [(1000, False, False), (200, True, False), (777, True, False),
                                            (300, True, True)])
def test_dense_baseline_matches_oracle(T, copies, gated):
    """The library's dense FFN: GEMMs whose 256 x 256 tiles fill at most half of the CUs
    split K (here every one: 2-8 ranges, ragged row counts), with row-contiguous weights
    and with K-contiguous copies, non-gated and gated."""
    w = wl.make_ffn("dense", "bf16", T, 512, 2048, seed=9 + T, sparsity=0.95, gated=gated)
    Y, _, _, _ = run_forward(w, dense=True, use_wupt=copies, use_wdownt=copies, use_wgatet=copies and gated)
    Yref, _ = oracle_rows(w, np.arange(w.T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    if T != 1000:
        return
    w32 = wl.c1_small_fp32()
    Y32, _, _, _ = run_forward(w32, dense=True)
    Yref32, _ = oracle_rows(w32, np.arange(w32.T))
    assert rel_l2(to_f64(Y32), Yref32) <= 1e-5


@pytest.mark.parametrize("T", [32, 700])
def test_gated_forward(T):
    w = wl.c3_gated(T=T, d=1024, f=4096)
    Y, bufs, stats, cfg = run_forward(w)
    Yref, G = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    Yd, _, _, _ = run_forward(w, dense=True)
    assert rel_l2(to_f64(Yd), Yref) <= 2e-2
    # with caller-provided W_up^T, or slice-major copies of W_up and W_down, the result is
    # identical (the same kernels read copies made outside instead of inside the call)
    Y2, _, _, _ = run_forward(w, use_wupt=True)
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))
    Y3, _, _, _ = run_forward(w, packed_up=True, packed_down=True)
    assert torch.equal(Y.view(torch.int16), Y3.view(torch.int16))
    Y4, _, _, _ = run_forward(w)
    assert torch.equal(Y.view(torch.int16), Y4.view(torch.int16))  # deterministic


def test_gated_c3_sampled():
    w = wl.c3_gated()
    Y, bufs, stats, cfg = run_forward(w)
    got = twell_views(bufs, w.T, w.f, cfg)
    rows = sample_rows(w.T, 128, 3, extra=np.nonzero(got["row_ovf"])[0][:32])
    Yref, _ = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y)[rows], Yref) <= 2e-2


def test_forward_deterministic():
    w = wl.make_ffn("det", "bf16", 1024, 1024, 4096, seed=11, sparsity=0.99, ell_width=128)
    Y1, b1, _, _ = run_forward(w)
    Y2, b2, _, _ = run_forward(w)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    for k in ("cnt", "row_nnz", "row_ovf"):
        assert torch.equal(b1[k], b2[k])


@pytest.mark.parametrize("T,Tn,S,K,s", [(4000, 64, 16, 64, 0.99), (4100, 128, 32, 640, 0.9)])
def test_large_ragged_batches_narrow_tiles(T, Tn, S, K, s):
    """Thousands of tokens, not a multiple of any block size, with tiles narrower than 256
    columns and (at 90%) long ELL rows: sampled rows (overflow rows included) against the
    oracle, and run-to-run identical output."""
    w = wl.make_ffn("ragged-large", "bf16", T, 2048, 4096, seed=21, sparsity=s, tile_cols=Tn, tile_slots=S,
                    ell_width=K)
    Y, bufs, stats, cfg = run_forward(w, packed_down=True)
    got = twell_views(bufs, w.T, w.f, cfg)
    ovf = np.nonzero(got["row_ovf"])[0]
    assert len(ovf) < 0.01 * T
    rows = sample_rows(w.T, 96, 5, extra=[0, 255, 256, T - 1, *ovf[:8]])
    Yref, _ = oracle_rows(w, rows)
    for i, t in enumerate(rows):
        assert rel_l2(to_f64(Y)[t], Yref[i]) <= 2e-2, t
    Y2, _, _, _ = run_forward(w, packed_down=True)
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))


@pytest.mark.parametrize("dtype,gated", [("bf16", False), ("f32", False), ("bf16", True)])
def test_empty_batch(dtype, gated):
    """T = 0: the forward and the dense FFN succeed with every zero-size buffer NULL (an
    empty tensor's pointer), write a dense-backup count of 0 and leave the statistics at 0."""
    w = wl.make_ffn("empty", dtype, 0, 512, 1024, seed=3, gated=gated, sparsity=0.99, ell_width=32)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    assert X.numel() == 0
    Wg = dev(w.W_gate) if gated else None
    cfg = b.make_cfg(**w.cfg)
    bufs = {k: None for k in b.alloc_twell(1, w.f, dtype, cfg)}
    bufs["n_ovf"] = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    stats = b.alloc_stats()
    Y = torch.empty((0, w.d), dtype=X.dtype, device="cuda")
    for dense in (False, True):
        args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, W_gate=Wg, stats=stats)
        ws = torch.empty(max(1, b.sfl_workspace_size(args, 2 if dense else 0)), dtype=torch.uint8, device="cuda")
        args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, W_gate=Wg, stats=stats, workspace=ws)
        (b.sfl_dense_ffn_baseline if dense else b.sfl_ffn_forward)(args)
        torch.cuda.synchronize()
    assert int(bufs["n_ovf"].item()) == 0
    st = b.read_stats(stats)
    assert st["total_nnz"] == 0 and st["n_ovf_rows"] == 0 and st["l1_sum"] == 0.0
    assert st["capacity_exceeded"] == 0


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("rows,cols", [(64, 64), (100, 132), (4096, 1024), (99, 130), (1, 7), (130, 4)])
def test_transpose_copies_bit_exact(rows, cols, dtype):
    """sfl_transpose against torch's transpose, bit for bit: 2- and 4-byte elements, shapes
    whose sides are multiples of 4 (the 16-byte path for 4-byte elements), of the 64 x 64
    tile, and neither."""
    g = torch.Generator().manual_seed(rows * 1000 + cols)
    x = torch.randn(rows, cols, generator=g).to(dtype).cuda()
    out = torch.full((cols, rows), float("nan"), dtype=dtype, device="cuda")
    b.sfl_transpose(x, out)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                       x.t().contiguous().view(torch.int16 if dtype == torch.bfloat16 else torch.int32))


def test_packed_down_weights_layout_and_equivalence():
    w = wl.make_ffn("packed", "bf16", 300, 1024, 2048, seed=12, sparsity=0.98, ell_width=96)
    Wd = dev(w.W_down)
    P = torch.empty_like(Wd)
    b.sfl_pack_down_weights(Wd, P)
    torch.cuda.synchronize()
    want = w.W_down.reshape(w.f, w.d // 64, 64).transpose(1, 0, 2).reshape(-1)
    np.testing.assert_array_equal(host_bits(P).reshape(-1), want)
    Y1, _, _, _ = run_forward(w)
    Y2, _, _, _ = run_forward(w, packed_down=True)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    Yref, _ = oracle_rows(w, np.arange(w.T))
    assert rel_l2(to_f64(Y1), Yref) <= 2e-2


@pytest.mark.parametrize("T,d,f", [(777, 512, 2048), (8192, 4096, 16384)])
def test_transposed_up_weights_match_row_contiguous_ones(T, d, f):
    """W_up^T routes the up projection to the K-contiguous GEMM (16x16x32 MFMAs) instead
    of the row-contiguous one (32x32x16): the float32 pre-activations agree to summation
    order, and the outputs meet the oracle."""
    w = wl.make_ffn("wupt", "bf16", T, d, f, seed=13, sparsity=0.99, ell_width=256)
    X, Wu = dev(w.X), dev(w.W_up)
    WupT = torch.empty((f, d), dtype=X.dtype, device="cuda")
    b.sfl_transpose(Wu, WupT)
    cfg = b.make_cfg(**w.cfg)
    Z1 = torch.empty((T, f), dtype=torch.float32, device="cuda")
    Z2 = torch.empty_like(Z1)
    b.sfl_up_projection(b.ffn_args(X, Wu, dev(w.W_down), cfg, shift_t=dev(w.shift_t)), Z1)
    b.sfl_up_projection(b.ffn_args(X, Wu, dev(w.W_down), cfg, shift_t=dev(w.shift_t), W_upT=WupT), Z2)
    torch.cuda.synchronize()
    scale = Z1.abs().max().item()
    assert (Z1 - Z2).abs().max().item() <= 1e-5 * scale
    Y2, b2, _, _ = run_forward(w, use_wupt=True)
    rows = sample_rows(T, 64, 5)
    Yref, Zref = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y2)[rows], Yref) <= 2e-2
    check_pattern(twell_views(b2, T, f, cfg), Zref, rows, f, cfg.tile_cols, cfg.tile_slots)


@pytest.mark.parametrize("gated", [False, True])
def test_transposed_gate_and_down_copies(gated):
    """W_gate^T and W_down^T move the gate projection, the dense-backup down GEMM and the
    dense baseline's GEMMs to the K-contiguous kernel; results still meet the oracle and the
    activity pattern. Rows forced active exercise the dense-backup rows."""
    if gated:
        w = wl.make_ffn("wt-gated", "bf16", 700, 512, 2048, seed=21, sparsity=0.99, ell_width=64, gated=True)
    else:
        w = wl.make_ffn("wt", "bf16", 700, 512, 2048, seed=22, sparsity=0.99, ell_width=64)
    w.shift_t[:40] = 100.0  # dense-backup rows
    rows = sample_rows(w.T, 96, 9, extra=range(0, 40, 3))
    Yref, Zref = oracle_rows(w, rows)
    cfg = b.make_cfg(**w.cfg)
    for dense in (False, True):
        Y0, b0, _, _ = run_forward(w, dense=dense)
        Y1, b1, st1, _ = run_forward(w, dense=dense, use_wupt=True, use_wgatet=gated, use_wdownt=True)
        assert rel_l2(to_f64(Y1)[rows], Yref) <= 2e-2
        assert rel_l2(to_f64(Y1), to_f64(Y0)) <= 1e-2
        if not dense:
            assert b.read_stats(st1)["n_ovf_rows"] >= 40
            check_pattern(twell_views(b1, w.T, w.f, cfg), Zref, rows, w.f, cfg.tile_cols, cfg.tile_slots)


def test_decode_forward_replays_from_a_hip_graph():
    """The decode-shaped gated forward captured in a HIP graph: every replay, with eager
    work and synchronisations between replays, equals the eager call bit for bit."""
    w = wl.c3_gated(T=32, d=1024, f=4096)
    X, Wu, Wd, Wg = dev(w.X), dev(w.W_up), dev(w.W_down), dev(w.W_gate)
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    Y = torch.zeros((w.T, w.d), dtype=torch.bfloat16, device="cuda")
    kw = dict(Y=Y, bufs=bufs, W_gate=Wg, W_upT=transposed(Wu), W_gateT=transposed(Wg), W_downT=transposed(Wd),
              shift_t=dev(w.shift_t))
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw))), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws)
    b.sfl_ffn_forward(args)
    torch.cuda.synchronize()
    Yeager = Y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        b.sfl_ffn_forward(args, torch.cuda.current_stream())
    for i in range(3):
        Y.fill_(float("nan"))
        bufs["row_nnz"].fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int16), Yeager.view(torch.int16)), i
        _ = (X.float() @ X.float().t()).sum().item()  # unrelated eager work between replays
    Yref, _ = oracle_rows(w, np.arange(w.T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2


@pytest.mark.parametrize("gated", [False, True])
def test_prefill_forward_replays_from_a_hip_graph(gated):
    """A forward above 256 tokens with dense-backup rows of both kinds (rebuilt from the
    slabs and recomputed through the need list, whose counter the first kernel zeroes): the
    eager call against the oracle, a second eager call equal to the first bit for bit, and
    the forward captured in a HIP graph replaying to the same bits, with eager work between
    replays."""
    T = 600
    sr = np.full(T, 0.99)
    sr[::7] = 0.5    # half of the units active: overflowing tiles, recomputed by the GEMM
    sr[3::7] = 0.95  # more than K = 64 active units but no tile over S: rebuilt from the slabs
    w = wl.make_ffn("fork", "bf16", T, 512, 2048, seed=5 + gated, gated=gated, sparsity_rows=sr, ell_width=64)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    Wg = dev(w.W_gate) if gated else None
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    Y = torch.zeros((w.T, w.d), dtype=torch.bfloat16, device="cuda")
    kw = dict(Y=Y, bufs=bufs, W_gate=Wg, W_upT=transposed(Wu), W_gateT=transposed(Wg) if gated else None,
              W_downT=transposed(Wd), shift_t=dev(w.shift_t))
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw))), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws)
    b.sfl_ffn_forward(args)
    torch.cuda.synchronize()
    Yeager = Y.clone()
    got = twell_views(bufs, T, w.f, cfg)
    tile_ovf = (got["cnt"] > cfg.tile_slots).any(axis=1)
    assert got["n_ovf"] == 2 * len(range(0, T, 7)) and 0 < tile_ovf.sum() < got["n_ovf"]
    Yref, _ = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    ovf = np.nonzero(got["row_ovf"])[0]
    assert rel_l2(to_f64(Y)[ovf], Yref[ovf]) <= 2e-2
    Y.fill_(float("nan"))
    b.sfl_ffn_forward(args)
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.int16), Yeager.view(torch.int16))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        b.sfl_ffn_forward(args, torch.cuda.current_stream())
    for i in range(3):
        Y.fill_(float("nan"))
        bufs["row_nnz"].fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int16), Yeager.view(torch.int16)), i
        _ = (X.float() @ X.float().t()).sum().item()  # unrelated eager work between replays


def test_c4_headline_in_the_bench_configuration():
    """The headline workload as bench.py launches it: W_up^T and W_down^T copies, slice-major
    W_down; sampled rows and their patterns against the oracle, and the dense baseline."""
    w = wl.c4_sweep(0.99)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    got = twell_views(bufs, w.T, w.f, cfg)
    rows = sample_rows(w.T, 128, 21, extra=np.nonzero(got["row_ovf"])[0][:16])
    Yref, Z = oracle_rows(w, rows)
    Yg = to_f64(Y)[rows]
    assert rel_l2(Yg, Yref) <= 2e-2
    for i, t in enumerate(rows):
        assert rel_l2(Yg[i], Yref[i]) <= 2e-2, t
    check_pattern(got, Z, rows, w.f, cfg.tile_cols, cfg.tile_slots)
    Yd, _, _, _ = run_forward(w, dense=True, use_wupt=True, use_wdownt=True)
    Ydg = to_f64(Yd)[rows]
    for i, t in enumerate(rows):
        assert rel_l2(Ydg[i], Yref[i]) <= 2e-2, t


def test_c3_gated_in_the_bench_configuration():
    """The gated prefill workload as bench.py launches it (transposed and slice-major copies
    of all weights); sampled rows against the oracle, and the dense baseline."""
    w = wl.c3_gated()
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wgatet=True, use_wdownt=True, packed_down=True,
                                      packed_up=True)
    got = twell_views(bufs, w.T, w.f, cfg)
    rows = sample_rows(w.T, 128, 22, extra=np.nonzero(got["row_ovf"])[0][:16])
    Yref, G = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y)[rows], Yref) <= 2e-2
    check_pattern(got, G, rows[:48], w.f, cfg.tile_cols, cfg.tile_slots)
    Yd, _, _, _ = run_forward(w, dense=True, use_wupt=True, use_wgatet=True, use_wdownt=True)
    assert rel_l2(to_f64(Yd)[rows], Yref) <= 2e-2


@pytest.mark.parametrize("force_ovf", [False, True])
def test_c3_decode_in_the_bench_configuration(force_ovf):
    """The gated decode workload (T=32, d=4096, f=14336) as bench.py launches it: every
    row against the oracle, sparse and dense. With a quarter of the rows made all-active,
    the dense-backup GEMMs of that width split K over the CUs and the last block of each
    output tile adds the partial sums; two calls in a row reuse the tile counters."""
    w = wl.c3_gated(T=32)
    if force_ovf:
        w.shift_t[::4] = 100.0
    rows = np.arange(w.T)
    Yref, G = oracle_rows(w, rows)
    for _ in range(2 if force_ovf else 1):
        Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wgatet=True, use_wdownt=True, packed_down=True,
                                          packed_up=True)
        got = twell_views(bufs, w.T, w.f, cfg)
        if force_ovf:
            assert got["row_ovf"][::4].all() and got["n_ovf"] >= 8
        assert rel_l2(to_f64(Y), Yref) <= 2e-2
        sparse = np.nonzero(~got["row_ovf"].astype(bool))[0]
        assert rel_l2(to_f64(Y)[sparse], Yref[sparse]) <= 2e-2
        check_pattern(got, G[sparse[:8]], sparse[:8], w.f, cfg.tile_cols, cfg.tile_slots)
    Yd, _, _, _ = run_forward(w, dense=True, use_wupt=True, use_wgatet=True, use_wdownt=True)
    assert rel_l2(to_f64(Yd), Yref) <= 2e-2


@pytest.mark.parametrize("kind", ["tp8", "dp8"])
def test_shard_shapes_in_the_bench_configuration(kind):
    """One GPU's share of the headline layer split eight ways, over hidden units (f = 2048,
    K = 64; the up GEMM is a single round of 256 tiles) or over tokens (T = 1024): sampled
    rows and their patterns against the oracle, and the dense baseline."""
    w = wl.c4_shard(kind)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    got = twell_views(bufs, w.T, w.f, cfg)
    rows = sample_rows(w.T, 128, 23, extra=np.nonzero(got["row_ovf"])[0][:16])
    Yref, Z = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y)[rows], Yref) <= 2e-2
    check_pattern(got, Z, rows[:48], w.f, cfg.tile_cols, cfg.tile_slots)
    Yd, _, _, _ = run_forward(w, dense=True, use_wupt=True, use_wdownt=True)
    assert rel_l2(to_f64(Yd)[rows], Yref) <= 2e-2


@pytest.mark.parametrize("T,K", [(1, 64), (9, 32), (777, 64), (1024, 64), (1031, 256), (2053, 48), (4100, 128)])
def test_token_group_walk_short_rows(T, K):
    """Batches of at least 1024 tokens with ELL widths of at most 256 take the token-group
    walk of the down projection (8 tokens per work item, each lane group on its own token;
    smaller batches the per-token walk): ragged batches whose last group is partly empty,
    all-active rows (dense backup, skipped by the walk) and all-inactive rows (Y exactly 0)
    among ordinary rows of about 20 entries."""
    w = wl.make_ffn("short-rows", "bf16", T, 1024, 2048, seed=T + K, sparsity=0.99, ell_width=K)
    zero = np.setdiff1d(np.arange(3, T, 5), np.arange(1, T, 7))
    if T > 2:
        w.shift_t[3::5] = -100.0
        w.shift_t[1::7] = 100.0
    Y, bufs, stats, cfg = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    got = twell_views(bufs, T, w.f, cfg)
    Yref, Z = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y), Yref) <= 2e-2
    ovf = got["row_ovf"].astype(bool)
    if T > 2:
        assert ovf[1::7].all() and int(got["row_nnz"][zero].max()) == 0
        assert (host_bits(Y)[zero] == 0).all()
    sparse = np.nonzero(~ovf)[0]
    assert len(sparse) > 0 and rel_l2(to_f64(Y)[sparse], Yref[sparse]) <= 2e-2


@pytest.mark.parametrize("T,d,f,splits", [(700, 1024, 4096, (1, 2)), (300, 4096, 2048, (1, 2, 4, 8))])
def test_rowwise_down_projection_variant(T, d, f, splits):
    """The paper-shaped down projection (one wave per token and segment of d) on the ELL rows
    the forward saved: sparse rows equal the oracle, and the forward's own Y to summation order;
    dense-backup rows are left untouched."""
    w = wl.make_ffn("rowwise", "bf16", T, d, f, seed=T + d, sparsity=0.99, ell_width=64)
    w.shift_t[::50] = 10.0  # dense-backup rows
    Y, bufs, stats, cfg = run_forward(w)
    got = twell_views(bufs, T, f, cfg)
    ovf = got["row_ovf"].astype(bool)
    assert ovf.sum() >= T // 50
    sparse = np.nonzero(~ovf)[0]
    Yref, _ = oracle_rows(w, sparse)
    for split in splits:
        Y2 = torch.full_like(Y, float("nan"))
        args = b.ffn_args(dev(w.X), dev(w.W_up), dev(w.W_down), cfg, Y=Y2, bufs=bufs)
        b.sfl_down_projection_rowwise(args, split)
        torch.cuda.synchronize()
        Yg = to_f64(Y2)
        assert np.isnan(Yg[ovf]).all()
        for i, t in enumerate(sparse):
            assert rel_l2(Yg[t], Yref[i]) <= 2e-2, (split, t)
        assert rel_l2(Yg[sparse], to_f64(Y)[sparse]) <= 1e-2
    args = b.ffn_args(dev(w.X), dev(w.W_up), dev(w.W_down), cfg, Y=Y, bufs=bufs)
    with pytest.raises(b.SflError) as e:
        b.sfl_down_projection_rowwise(args, 3)
    assert e.value.code == b.SFL_E_UNSUPPORTED


@pytest.mark.parametrize("T,gated,K", [(1500, False, 64), (700, False, 96), (32, True, 128), (600, True, 96)])
def test_descending_nnz_token_order_gives_identical_results(T, gated, K, monkeypatch):
    """SFL_TOKEN_ORDER=nnz deals the sparse down projection's (and the gated up-dots') tokens
    by descending row count (the default for batches of >= 1024 tokens with K <= 256),
    SFL_TOKEN_ORDER=token in token order: the outputs are bit-identical (every token
    is handled exactly once, by the same arithmetic), with dense-backup rows and rows of
    widely varying length (token-group walk at 1500 tokens, per-token walk below 1024)."""
    r = np.random.default_rng(T)
    sp = np.where(r.random(T) < 0.5, 0.995, 0.98)
    w = wl.make_ffn("order", "bf16", T, 512, 2048, seed=T + K, gated=gated, sparsity_rows=sp, ell_width=K)
    w.shift_t[::37] = 10.0  # dense-backup rows
    monkeypatch.setenv("SFL_TOKEN_ORDER", "token")
    Y1, b1, _, cfg = run_forward(w, packed_down=True)
    monkeypatch.setenv("SFL_TOKEN_ORDER", "nnz")
    Y2, b2, _, _ = run_forward(w, packed_down=True)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    monkeypatch.delenv("SFL_TOKEN_ORDER")  # the default (by batch size and ELL width)
    Y3, _, _, _ = run_forward(w, packed_down=True)
    assert torch.equal(Y1.view(torch.int16), Y3.view(torch.int16))
    got = twell_views(b2, T, w.f, cfg)
    assert got["n_ovf"] >= T // 37
    rows = sample_rows(T, 48, 4, extra=np.nonzero(got["row_ovf"])[0][:4])
    Yref, _ = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y2)[rows], Yref) <= 2e-2


@pytest.mark.parametrize("sparsity,K,dense_expected", [(0.9, 640, True), (0.99, 64, False)])
def test_dense_fallback_choice_and_results(sparsity, K, dense_expected, monkeypatch):
    """ELL width K >= f / 32 makes a call a dense-fallback candidate: the up projection also
    writes H, and a batch whose mean row count exceeds f / 64 takes one dense down GEMM instead
    of the gather (the sparse rows' entries against T f / 64). Both choices meet the oracle; the TwELL, classification and the
    dense-backup rows' outputs are the same as with the fallback disabled; a candidate that
    keeps the gather gives the disabled run's output bit for bit."""
    T, d, f = 1000, 512, 2048
    w = wl.make_ffn("fallback", "bf16", T, d, f, seed=int(sparsity * 1000), sparsity=sparsity, ell_width=K)
    w.shift_t[::50] = 10.0  # dense-backup rows
    monkeypatch.setenv("SFL_DENSE_FALLBACK", "off")
    Y0, b0, st0, cfg = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    monkeypatch.delenv("SFL_DENSE_FALLBACK")
    Y1, b1, st1, _ = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    for k in ("cnt", "row_nnz", "row_ovf"):
        assert torch.equal(b0[k], b1[k]), k
    got = twell_views(b1, T, f, cfg)
    got0 = twell_views(b0, T, f, cfg)
    for t in np.nonzero(got["row_ovf"] == 0)[0][::7]:  # ELL rows: the specified entries
        c = int(got["row_nnz"][t])
        np.testing.assert_array_equal(got["ell_idx"][t, :c], got0["ell_idx"][t, :c])
        np.testing.assert_array_equal(got["ell_val"][t, :c], got0["ell_val"][t, :c])
    gather_entries = got["row_nnz"][got["row_ovf"] == 0].sum()
    assert (gather_entries * 64 > T * f) == dense_expected
    ovf = np.nonzero(got["row_ovf"])[0]
    assert len(ovf) >= T // 50
    assert torch.equal(Y0.view(torch.int16)[ovf], Y1.view(torch.int16)[ovf])  # dense-backup rows
    if dense_expected:
        assert rel_l2(to_f64(Y1), to_f64(Y0)) <= 1e-2
    else:
        assert torch.equal(Y0.view(torch.int16), Y1.view(torch.int16))
    s0, s1 = b.read_stats(st0), b.read_stats(st1)
    assert s0["total_nnz"] == s1["total_nnz"] and abs(s0["l1_sum"] - s1["l1_sum"]) <= 1e-6 * s0["l1_sum"]
    rows = sample_rows(T, 64, 8, extra=ovf[:4])
    Yref, _ = oracle_rows(w, rows)
    for i, t in enumerate(rows):
        assert rel_l2(to_f64(Y1)[t], Yref[i]) <= 2e-2, t
    monkeypatch.setenv("SFL_DENSE_FALLBACK", "on")  # every eligible call takes the dense GEMM
    Y2, _, _, _ = run_forward(w, use_wupt=True, use_wdownt=True, packed_down=True)
    assert rel_l2(to_f64(Y2)[rows], Yref) <= 2e-2
    if dense_expected:
        assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
