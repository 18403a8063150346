"""The L1 statistic of the forward (stats.l1_sum) against the oracle's eq. l1.

l1_sum * lambda / (T f) must equal `oracle.ffn.l1_penalty(H, lambda)` for one layer, with
H the fp64 activations: ReLU(Z) for the non-gated layer, ReLU(G) * U for the gated one
(eq. l1 puts the penalty on h; the gated h is signed, so the sum is of |h|).

Tolerance. Every term of the sum is non-negative, so the relative error of the sum is at
most the largest relative error of a term. The GPU's terms are stored activations:
non-gated, one round-to-nearest-even to bf16 of the fp32 pre-activation (2^-9 relative);
gated, bf16(bf16(g) * u) (two roundings, 2^-8 together) with u summed in fp32. Add the
fp32 accumulation of z and u (relative 1e-5 or so for terms that are not within rounding
of 0, which contribute next to nothing) and float64 atomics: 5e-3 bounds it. A dropped or
doubled group of rows, gate values summed in place of h, or signed h summed over the
dense-backup rows each move the sum by far more."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import ffn, twell
from tests.gpu_util import dev, twell_views

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")
from tests.test_gpu_forward import run_forward  # noqa: E402

LAM = 2e-5
RTOL = 5e-3


def oracle_h(w):
    X = w.as_f64(w.X)
    if w.gated:
        _, G, U, H = ffn.ffn_gated_dense(X, w.as_f64(w.W_gate), w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f,
                                         w.shift_t)
        return H, G
    _, Z, H = ffn.ffn_dense(X, w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, w.shift_t)
    return H, Z


def mixed_rows(T, seed, frac_rebuilt=0.04, frac_recomputed=0.04):
    """Per-row sparsity: mostly 99 %, some rows at 95 % (more than K = 64 active units but no
    tile over S = 32: dense-backup rows rebuilt from the slabs) and some at 50 % (tiles over
    S: recomputed by the GEMM)."""
    r = np.random.default_rng(seed)
    s = np.full(T, 0.99)
    u = r.random(T)
    s[u < frac_rebuilt] = 0.95
    s[(u >= frac_rebuilt) & (u < frac_rebuilt + frac_recomputed)] = 0.5
    return s


def check_l1(st, w, H, rows=None):
    got = st["l1_sum"] * LAM / (w.T * w.f)
    Hs = H if rows is None else H[rows]
    # l1_penalty normalises by the rows and columns of its argument; keep the layer's T f
    want = ffn.l1_penalty(Hs, LAM) * (Hs.shape[0] * Hs.shape[1]) / (w.T * w.f)
    assert want > 0
    assert abs(got - want) <= RTOL * want, (got, want, got / want)


@pytest.mark.parametrize("T,copies", [(700, False), (700, True), (200, True), (200, False), (48, True), (48, False)])
def test_l1_non_gated_with_both_kinds_of_dense_backup_rows(T, copies):
    """Non-gated: sparse rows (the TwELL values summed by the classification) and dense-backup
    rows; above 256 tokens some are rebuilt from the slabs and some recomputed by the GEMM,
    at or below 256 tokens all are recomputed (with W_up^T, through the split-K GEMM; at
    most 64 rows, whose last blocks sum the rows they store)."""
    w = wl.make_ffn("l1", "bf16", T, 512, 2048, seed=31 + T, sparsity_rows=mixed_rows(T, T), ell_width=64)
    Y, bufs, stats, cfg = run_forward(w, use_wupt=copies, use_wdownt=copies)
    st = b.read_stats(stats)
    got = twell_views(bufs, w.T, w.f, cfg)
    H, Z = oracle_h(w)
    tw = twell.extract_twell(Z, cfg.tile_cols, cfg.tile_slots, "bf16")
    hy = twell.classify(tw, cfg.ell_width)
    np.testing.assert_array_equal(got["ovf_rows"][:got["n_ovf"]], hy.ovf_rows)
    tile_ovf = (tw.cnt > cfg.tile_slots).any(axis=1)
    assert 0 < tile_ovf.sum() < len(hy.ovf_rows)  # both kinds of dense-backup row
    assert st["capacity_exceeded"] == 0
    check_l1(st, w, H)


@pytest.mark.parametrize("T", [700, 32])
def test_l1_gated_sums_absolute_h(T):
    """Gated: h = ReLU(g) * u is signed. The sparse rows' |h| is summed where h is formed (not
    the gate values), the dense-backup rows' after the multiplication by u, as |h|."""
    w = wl.make_ffn("l1-gated", "bf16", T, 512, 2048, seed=41 + T, gated=True, sparsity_rows=mixed_rows(T, 7 + T, 0.1, 0.1),
                    ell_width=64)
    Y, bufs, stats, cfg = run_forward(w)
    st = b.read_stats(stats)
    H, G = oracle_h(w)
    assert (H < 0).sum() > 0.3 * (H != 0).sum()  # many negative h: a signed sum would fail
    got = twell_views(bufs, w.T, w.f, cfg)
    assert got["n_ovf"] > 0
    check_l1(st, w, H)
    # the same call with K-contiguous copies of every weight
    Y2, _, stats2, _ = run_forward(w, use_wupt=True, use_wgatet=True, use_wdownt=True, packed_down=True,
                                   packed_up=True)
    check_l1(b.read_stats(stats2), w, H)


@pytest.mark.parametrize("gated", [False, True])
def test_l1_capacity_exceeded_counts_only_computed_rows(gated):
    """More dense-backup rows than the capacity: only the first `capacity` of them are
    computed, and only they (with the sparse rows) enter the sum."""
    T = 128
    w = wl.make_ffn("l1-cap", "bf16", T, 512, 512, seed=5, gated=gated, sparsity=0.99, ell_width=16)
    w.shift_t[::4] = 0.0  # about half of every such row active: 32 dense-backup rows
    w.cfg["ovf_capacity"] = 10
    Y, bufs, stats, cfg = run_forward(w)
    st = b.read_stats(stats)
    assert st["capacity_exceeded"] == 1
    got = twell_views(bufs, w.T, w.f, cfg)
    ovf = np.nonzero(got["row_ovf"])[0]
    assert len(ovf) >= 32
    computed = np.setdiff1d(np.arange(T), ovf[10:])
    H, _ = oracle_h(w)
    check_l1(st, w, H, rows=computed)


def test_l1_of_the_standalone_pack():
    """sfl_pack_twell sums the stored values of its sparse rows (ReLU(Z), bf16-rounded)."""
    w = wl.make_ffn("l1-pack", "bf16", 300, 256, 1024, seed=9, sparsity=0.97, ell_width=48)
    w.shift_t[:5] = 50.0  # dense-backup rows
    H, Z = oracle_h(w)
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    stats = b.alloc_stats()
    b.sfl_pack_twell(torch.from_numpy(Z.astype(np.float32)).cuda(), "bf16", cfg, bufs, stats)
    torch.cuda.synchronize()
    st = b.read_stats(stats)
    tw = twell.extract_twell(Z.astype(np.float32), cfg.tile_cols, cfg.tile_slots, "bf16")
    hy = twell.classify(tw, cfg.ell_width)
    sparse = np.nonzero(~hy.is_ovf)[0]
    assert len(sparse) < w.T  # some dense-backup rows, left out of the pack's sum
    check_l1(st, w, H, rows=sparse)


@pytest.mark.parametrize("T,gated,copies", [(32, True, True), (48, False, True), (48, True, False), (700, False, True)])
def test_statistics_and_counters_are_cleared_by_the_call(T, gated, copies):
    """Every forward clears its statistics and workspace counters itself (a batch of at most
    64 tokens with K-contiguous weights in its first GEMM, others in a clearing kernel): the
    same call with the statistics and the workspace filled with 0xff bytes beforehand gives
    the statistics of a clean start, and the same Y bit for bit. Rows with dense-backup rows,
    so that the per-tile counters and the recompute list are in use."""
    w = wl.make_ffn("clear", "bf16", T, 512, 2048, seed=3 + T, gated=gated,
                    sparsity_rows=mixed_rows(T, T, 0.15, 0.15), ell_width=64)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    Wg = dev(w.W_gate) if gated else None
    tr = lambda W: None if (W is None or not copies) else W.t().contiguous()
    cfg = b.make_cfg(**w.cfg)
    out = []
    for dirty in (False, True):
        bufs = b.alloc_twell(T, w.f, "bf16", cfg)
        Y = torch.empty((T, w.d), dtype=torch.bfloat16, device="cuda")
        stats = b.alloc_stats()
        kw = dict(Y=Y, bufs=bufs, W_gate=Wg, W_upT=tr(Wu), W_gateT=tr(Wg), W_downT=tr(Wd), shift_t=dev(w.shift_t),
                  stats=stats)
        ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw))), dtype=torch.uint8,
                         device="cuda")
        if dirty:
            stats.fill_(0xff)
            ws.fill_(0xff)
        b.sfl_ffn_forward(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws))
        torch.cuda.synchronize()
        out.append((Y, b.read_stats(stats), twell_views(bufs, T, w.f, cfg)["n_ovf"]))
    (Y0, s0, n0), (Y1, s1, n1) = out
    assert n0 == n1 > 0
    assert torch.equal(Y0.view(torch.int16), Y1.view(torch.int16))
    for k in ("total_nnz", "n_ovf_rows", "n_tile_ovf", "capacity_exceeded"):
        assert s0[k] == s1[k], k
    assert abs(s1["l1_sum"] - s0["l1_sum"]) <= 1e-6 * abs(s0["l1_sum"])
