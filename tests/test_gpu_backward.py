"""sfl_ffn_backward on the GPU against the fp64 oracle (non-gated, with the L1 term).

The oracle consumes the activity pattern the GPU forward saved (its fp32 pre-activation
decides z > 0, which may differ from fp64 within rounding), then applies the chain rule of
the loss sum(dY * Y) + lambda/(T f) sum|h|. Bar: relative L2 <= 2e-2 for dX, dW_up, dW_down."""
import numpy as np
import pytest
import scipy.sparse as sp
import torch

import workloads as wl
from oracle import ffn
from tests.gpu_util import dev, host_bits, rel_l2, to_f64, twell_views

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")


def run_fwd_bwd(w, lam, with_wupt=False, with_packed=False):
    X, Wu, Wd, dY = dev(w.X), dev(w.W_up), dev(w.W_down), dev(w.dY)
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    Y = torch.empty((w.T, w.d), dtype=torch.bfloat16, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=dev(w.shift_t))
    ws = torch.empty(max(1, b.sfl_workspace_size(args)), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=dev(w.shift_t), workspace=ws)
    b.sfl_ffn_forward(args)
    dX = torch.full((w.T, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dWu = torch.full((w.d, w.f), float("nan"), dtype=torch.float32, device="cuda")
    dWd = torch.full((w.f, w.d), float("nan"), dtype=torch.float32, device="cuda")
    WupT = None
    if with_wupt:
        WupT = torch.empty((w.f, w.d), dtype=torch.bfloat16, device="cuda")
        b.sfl_transpose(Wu, WupT)
    pk = {}
    if with_packed:
        pk["W_down_packed"] = torch.empty_like(Wd)
        b.sfl_pack_down_weights(Wd, pk["W_down_packed"])
        WuT = torch.empty((w.f, w.d), dtype=torch.bfloat16, device="cuda")
        b.sfl_transpose(Wu, WuT)
        pk["W_up_packed"] = torch.empty_like(Wu)
        b.sfl_pack_down_weights(WuT, pk["W_up_packed"])
    ba = b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd, W_upT=WupT, **pk)
    bws = torch.empty(max(1, b.sfl_workspace_size(ba, 1)), dtype=torch.uint8, device="cuda")
    ba = b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd, W_upT=WupT, workspace=bws, **pk)
    b.sfl_ffn_backward(ba)
    torch.cuda.synchronize()
    return dX, dWu, dWd, bufs, cfg


def gpu_pattern(bufs, w, cfg):
    """Sparse [T, f] boolean activity saved by the GPU forward: ELL rows and dense-backup rows."""
    got = twell_views(bufs, w.T, w.f, cfg)
    rows, cols = [], []
    for t in np.nonzero(got["row_ovf"] == 0)[0]:
        c = int(got["row_nnz"][t])
        rows.append(np.full(c, t))
        cols.append(got["ell_idx"][t, :c].astype(np.int64))
    n_ovf = got["n_ovf"]
    dense = host_bits(bufs["ovf_dense"])[: n_ovf * w.f].reshape(n_ovf, w.f)
    for i, t in enumerate(got["ovf_rows"][:n_ovf]):
        c = np.nonzero(dense[i].view(np.int16) > 0)[0]
        rows.append(np.full(len(c), t))
        cols.append(c)
    r = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    c = np.concatenate(cols) if cols else np.zeros(0, np.int64)
    return sp.csr_matrix((np.ones(len(r), dtype=bool), (r, c)), shape=(w.T, w.f))


def oracle_full(w, active, lam):
    X, Wu, Wd, dY = w.as_f64(w.X), w.as_f64(w.W_up), w.as_f64(w.W_down), w.as_f64(w.dY)
    Z = ffn.preactivation(X, Wu, None, w.shift_t)
    act = active.toarray()
    H = np.where(act, Z, 0.0)
    dX, dWu, dWd, _ = ffn.ffn_backward(X, Wu, Wd, dY, H, act, lam)
    return dX, dWu, dWd


@pytest.mark.parametrize("T,d,f,K,S,lam_scale", [(300, 512, 2048, 96, 32, 0.0), (300, 512, 2048, 96, 32, 1e-3),
                                                 (129, 1024, 1024, 24, 8, 1e-3), (64, 512, 512, 512, 64, 0.0)])
def test_backward_small_full(T, d, f, K, S, lam_scale):
    w = wl.make_ffn("bwd", "bf16", T, d, f, seed=T + d, sparsity=0.97, ell_width=K, tile_slots=S, with_dy=True)
    w.shift_t[:3] = 10.0   # dense-backup rows
    lam = lam_scale * T * f
    dX, dWu, dWd, bufs, cfg = run_fwd_bwd(w, lam)
    act = gpu_pattern(bufs, w, cfg)
    rdX, rdWu, rdWd = oracle_full(w, act, lam)
    assert rel_l2(to_f64(dX), rdX) <= 2e-2
    assert rel_l2(to_f64(dWu), rdWu) <= 2e-2
    assert rel_l2(to_f64(dWd), rdWd) <= 2e-2
    ovf = np.nonzero(twell_views(bufs, w.T, w.f, cfg)["row_ovf"])[0]
    assert len(ovf) >= 3
    assert rel_l2(to_f64(dX)[ovf], rdX[ovf]) <= 2e-2


def test_backward_empty_batch():
    """T = 0: the weight gradients are zero (overwriting what the buffers held)."""
    w = wl.make_ffn("empty", "bf16", 0, 512, 1024, seed=4, sparsity=0.99, ell_width=32, with_dy=True)
    dX, dWu, dWd, bufs, cfg = run_fwd_bwd(w, 0.0)
    assert dX.shape == (0, 512)
    assert torch.count_nonzero(dWu).item() == 0 and torch.count_nonzero(dWd).item() == 0


def test_backward_widest_f():
    """f = 65472, the widest multiple of 64 the uint16 column index allows: the transposed
    pattern spans four windows of per-unit token masks; two dense-backup rows."""
    T, d, f = 96, 512, 65472
    w = wl.make_ffn("wide", "bf16", T, d, f, seed=23, sparsity=0.99, ell_width=1024, with_dy=True)
    w.shift_t[:2] = 10.0
    lam = 1e-3 * T * f
    dX, dWu, dWd, bufs, cfg = run_fwd_bwd(w, lam)
    act = gpu_pattern(bufs, w, cfg)
    rdX, rdWu, rdWd = oracle_full(w, act, lam)
    assert rel_l2(to_f64(dX), rdX) <= 2e-2
    assert rel_l2(to_f64(dWu), rdWu) <= 2e-2
    assert rel_l2(to_f64(dWd), rdWd) <= 2e-2


def test_backward_hot_units_exceed_staged_lists():
    """Units active in every token have lists longer than one block's LDS stage, so their
    per-unit gathers read the lists from global memory; results still meet the oracle."""
    T, d, f = 12800, 512, 1024
    w = wl.make_ffn("hot", "bf16", T, d, f, seed=17, sparsity=0.99, ell_width=64, with_dy=True)
    w.bias_f = np.zeros(f, dtype=np.float32)
    w.bias_f[[5, 6, 700]] = 100.0  # always active
    X, Wu, Wd, dY = dev(w.X), dev(w.W_up), dev(w.W_down), dev(w.dY)
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(T, f, "bf16", cfg)
    Y = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    kw = dict(Y=Y, bufs=bufs, bias_f=dev(w.bias_f), shift_t=dev(w.shift_t))
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw))), dtype=torch.uint8, device="cuda")
    b.sfl_ffn_forward(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws))
    lam = 1e-3 * T * f
    dX = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    dWu = torch.empty((d, f), dtype=torch.float32, device="cuda")
    dWd = torch.empty((f, d), dtype=torch.float32, device="cuda")
    ba = b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd)
    bws = torch.empty(max(1, b.sfl_workspace_size(ba, 1)), dtype=torch.uint8, device="cuda")
    b.sfl_ffn_backward(b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd, workspace=bws))
    torch.cuda.synchronize()
    act = gpu_pattern(bufs, w, cfg)
    assert act[:, 5].sum() == T and act[:, 700].sum() == T
    Xd, Wud, Wdd, dYd = w.as_f64(w.X), w.as_f64(w.W_up), w.as_f64(w.W_down), w.as_f64(w.dY)
    Z = ffn.preactivation(Xd, Wud, w.bias_f, w.shift_t)
    A = act.toarray()
    rdX, rdWu, rdWd, _ = ffn.ffn_backward(Xd, Wud, Wdd, dYd, np.where(A, Z, 0.0), A, lam)
    assert rel_l2(to_f64(dWd), rdWd) <= 2e-2
    assert rel_l2(to_f64(dWu), rdWu) <= 2e-2
    assert rel_l2(to_f64(dX), rdX) <= 2e-2
    for n in (5, 700):  # the long lists themselves
        assert rel_l2(to_f64(dWd)[n], rdWd[n]) <= 2e-2
        assert rel_l2(to_f64(dWu)[:, n], rdWu[:, n]) <= 2e-2


def test_backward_lambda_term_is_injected():
    """With dY = 0 the gradients come from the L1 term alone: dZ = lambda/(T f) on the pattern."""
    w = wl.make_ffn("l1", "bf16", 200, 512, 1024, seed=5, sparsity=0.95, ell_width=128, with_dy=True)
    w.dY[:] = 0
    lam = 1e-3 * w.T * w.f
    dX, dWu, dWd, bufs, cfg = run_fwd_bwd(w, lam)
    act = gpu_pattern(bufs, w, cfg)
    rdX, rdWu, rdWd = oracle_full(w, act, lam)
    assert np.abs(to_f64(dWd)).max() == 0.0
    assert rel_l2(to_f64(dWu), rdWu) <= 2e-2
    assert rel_l2(to_f64(dX), rdX) <= 2e-2


def test_backward_deterministic_and_weight_copies():
    """Bitwise reproducible, and identical whether W_up^T / the slice-major weight copies
    come from the caller or are built inside the call."""
    w = wl.make_ffn("bdet", "bf16", 512, 1024, 2048, seed=8, sparsity=0.98, ell_width=128, with_dy=True)
    a = run_fwd_bwd(w, 2e-5)
    for other in (run_fwd_bwd(w, 2e-5, with_wupt=True), run_fwd_bwd(w, 2e-5, with_packed=True),
                  run_fwd_bwd(w, 2e-5)):
        for x, y in zip(a[:3], other[:3]):
            assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))


def test_backward_c5_sampled():
    """Training shape: T=16384, d=4096, f=16384, ~99% sparse, K=256; sampled units (dW_up
    columns, dW_down rows) and sampled rows (dX) against the oracle's per-unit and per-row
    gradients on the pattern the GPU saved, each unit and row on its own."""
    w = wl.c5_training()
    lam = 1e-3 * w.T * w.f   # per-element injection 1e-3, visible in bf16
    dX, dWu, dWd, bufs, cfg = run_fwd_bwd(w, lam)
    act = gpu_pattern(bufs, w, cfg).tocsc()
    r = np.random.default_rng(0)
    X, Wu, Wd, dY = w.as_f64(w.X), w.as_f64(w.W_up), w.as_f64(w.W_down), w.as_f64(w.dY)
    units = r.choice(w.f, size=48, replace=False)
    dWu_ref, dWd_ref = ffn.ffn_backward_units(X, Wu, Wd, dY, units, act[:, units].toarray(), lam, None, w.shift_t)
    gWu, gWd = to_f64(dWu)[:, units], to_f64(dWd)[units]
    assert rel_l2(gWd, dWd_ref) <= 2e-2 and rel_l2(gWu, dWu_ref) <= 2e-2
    for j in range(len(units)):
        assert rel_l2(gWd[j], dWd_ref[j]) <= 2e-2, units[j]
        assert rel_l2(gWu[:, j], dWu_ref[:, j]) <= 2e-2, units[j]
    got = twell_views(bufs, w.T, w.f, cfg)
    rows = np.unique(np.concatenate([r.choice(w.T, size=64, replace=False),
                                     np.nonzero(got["row_ovf"])[0][:8]]))
    dX_ref = ffn.ffn_backward_rows(X, Wu, Wd, dY, rows, act.tocsr()[rows].toarray(), lam)
    gX = to_f64(dX)[rows]
    for i, t in enumerate(rows):
        assert rel_l2(gX[i], dX_ref[i]) <= 2e-2, t


# ---- gated block (eq. sec3:eq:all_other_gradients with eq. l1 on h = ReLU(g) h_u) --------

def run_gated_fwd_bwd(w, lam, copies=False):
    X, Wg, Wu, Wd, dY = dev(w.X), dev(w.W_gate), dev(w.W_up), dev(w.W_down), dev(w.dY)
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    Y = torch.empty((w.T, w.d), dtype=torch.bfloat16, device="cuda")
    kw = dict(Y=Y, bufs=bufs, W_gate=Wg, bias_f=dev(w.bias_f), shift_t=dev(w.shift_t))
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw))), dtype=torch.uint8, device="cuda")
    b.sfl_ffn_forward(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws))
    dX = torch.full((w.T, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dWg = torch.full((w.d, w.f), float("nan"), dtype=torch.float32, device="cuda")
    dWu = torch.full((w.d, w.f), float("nan"), dtype=torch.float32, device="cuda")
    dWd = torch.full((w.f, w.d), float("nan"), dtype=torch.float32, device="cuda")
    extra = {}
    if copies:
        def tr(W):
            out = torch.empty((W.shape[1], W.shape[0]), dtype=W.dtype, device="cuda")
            b.sfl_transpose(W, out)
            return out

        def pk(Wt):
            out = torch.empty_like(Wt)
            b.sfl_pack_down_weights(Wt, out)
            return out
        extra = dict(W_upT=tr(Wu), W_gateT=tr(Wg), W_down_packed=pk(Wd))
        extra["W_up_packed"] = pk(extra["W_upT"])
        extra["W_gate_packed"] = pk(extra["W_gateT"])
    bkw = dict(W_gate=Wg, dW_gate=dWg, bias_f=dev(w.bias_f), shift_t=dev(w.shift_t), **extra)
    ba = b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd, **bkw)
    bws = torch.empty(max(1, b.sfl_workspace_size(ba, 1)), dtype=torch.uint8, device="cuda")
    b.sfl_ffn_backward(b.bwd_args(X, Wu, Wd, dY, cfg, bufs, lam, dX, dWu, dWd, workspace=bws, **bkw))
    torch.cuda.synchronize()
    return dX, dWg, dWu, dWd, bufs, cfg


def gated_oracle(w, bufs, cfg, lam):
    """The fp64 gated gradients on the gate pattern the GPU saved (ELL rows); dense-backup
    rows keep the fp64 pattern G > 0 (the GPU recomputes them)."""
    X, Wg, Wu, Wd, dY = (w.as_f64(a) for a in (w.X, w.W_gate, w.W_up, w.W_down, w.dY))
    G = ffn.preactivation(X, Wg, w.bias_f, w.shift_t)
    U = X @ Wu
    got = twell_views(bufs, w.T, w.f, cfg)
    act = G > 0
    for t in np.nonzero(got["row_ovf"] == 0)[0]:
        act[t] = False
        act[t, got["ell_idx"][t, :int(got["row_nnz"][t])].astype(np.int64)] = True
    Gm = np.where(act, np.maximum(G, 1e-30), np.minimum(G, 0.0))
    return ffn.ffn_gated_backward(X, Wg, Wu, Wd, dY, Gm, U, lam), got


@pytest.mark.parametrize("T,d,f,K,lam_scale", [(300, 512, 2048, 96, 0.0), (300, 512, 2048, 96, 1e-3),
                                               (129, 1024, 1024, 48, 1e-3)])
def test_gated_backward_small_full(T, d, f, K, lam_scale):
    w = wl.make_ffn("gbwd", "bf16", T, d, f, seed=T + f, gated=True, sparsity=0.97, ell_width=K, with_dy=True)
    w.shift_t[:3] = 10.0   # dense-backup rows (every gate unit active)
    lam = lam_scale * T * f
    dX, dWg, dWu, dWd, bufs, cfg = run_gated_fwd_bwd(w, lam)
    (rdX, rdWg, rdWu, rdWd), got = gated_oracle(w, bufs, cfg, lam)
    assert got["row_ovf"][:3].all()
    for gpu, ref in ((dX, rdX), (dWg, rdWg), (dWu, rdWu), (dWd, rdWd)):
        assert rel_l2(to_f64(gpu), ref) <= 2e-2
    assert rel_l2(to_f64(dX)[:3], rdX[:3]) <= 2e-2          # the dense-backup rows
    sparse = np.nonzero(got["row_ovf"] == 0)[0]
    assert rel_l2(to_f64(dX)[sparse], rdX[sparse]) <= 2e-2


def test_gated_backward_copies_and_determinism():
    """Identical with caller-provided transposed / slice-major copies, and run to run."""
    w = wl.make_ffn("gbdet", "bf16", 400, 1024, 2048, seed=31, gated=True, sparsity=0.98, ell_width=96,
                    with_dy=True)
    w.shift_t[:2] = 10.0
    a = run_gated_fwd_bwd(w, 2e-5)
    for other in (run_gated_fwd_bwd(w, 2e-5, copies=True), run_gated_fwd_bwd(w, 2e-5)):
        for x, y in zip(a[:4], other[:4]):
            assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))


def test_backward_c5_bench_configuration_is_identical():
    """bench.py passes W_up^T and slice-major W_down / W_up^T to the backward at the training
    shape; the gradients equal those of the copy-free call (sampled-oracle checked above)."""
    w = wl.c5_training()
    a = run_fwd_bwd(w, 2e-5)
    c = run_fwd_bwd(w, 2e-5, with_wupt=True, with_packed=True)
    for x, y in zip(a[:3], c[:3]):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))


def test_gated_training_bench_configuration_sampled():
    """The gated training step as bench.py runs it (T=8192, d=4096, f=14336, dense backup of
    T/8 rows, all weight copies): sampled units of dW_gate, dW_up, dW_down and sampled rows
    of dX, each on its own, against the oracle's per-unit and per-row gradients on the gate
    pattern the GPU saved (ELL rows; fp64 G > 0 on the dense-backup rows, which the GPU
    recomputes)."""
    w = wl.gated_training()
    w.shift_t[:4] = 10.0  # a few dense-backup rows
    lam = 1e-3 * w.T * w.f
    dX, dWg, dWu, dWd, bufs, cfg = run_gated_fwd_bwd(w, lam, copies=True)
    got = twell_views(bufs, w.T, w.f, cfg)
    assert got["row_ovf"][:4].all()
    X, Wg, Wu, Wd, dY = (w.as_f64(a) for a in (w.X, w.W_gate, w.W_up, w.W_down, w.dY))
    sparse_rows = np.nonzero(got["row_ovf"] == 0)[0]

    def pattern(rows_sel, cols):
        """GPU pattern on ELL rows, fp64 G > 0 on dense-backup rows, for [rows_sel][cols]."""
        act = ffn.preactivation(X[rows_sel], Wg[:, cols], None, w.shift_t[rows_sel]) > 0
        colpos = {int(c): j for j, c in enumerate(cols)}
        for i, t in enumerate(rows_sel):
            if got["row_ovf"][t]:
                continue
            act[i] = False
            for n in got["ell_idx"][t, :int(got["row_nnz"][t])]:
                j = colpos.get(int(n))
                if j is not None:
                    act[i, j] = True
        return act

    r = np.random.default_rng(5)
    units = r.choice(w.f, size=32, replace=False)
    A = pattern(np.arange(w.T), units)
    rWg, rWu, rWd = ffn.ffn_gated_backward_units(X, Wg, Wu, Wd, dY, units, A, lam, None, w.shift_t)
    gWg, gWu, gWd = to_f64(dWg)[:, units], to_f64(dWu)[:, units], to_f64(dWd)[units]
    for j in range(len(units)):
        assert rel_l2(gWd[j], rWd[j]) <= 2e-2, units[j]
        assert rel_l2(gWu[:, j], rWu[:, j]) <= 2e-2, units[j]
        assert rel_l2(gWg[:, j], rWg[:, j]) <= 2e-2, units[j]
    rows = np.concatenate([r.choice(sparse_rows, size=24, replace=False), np.arange(4)])
    Ar = pattern(rows, np.arange(w.f))
    rX = ffn.ffn_gated_backward_rows(X, Wg, Wu, Wd, dY, rows, Ar, lam, None, w.shift_t)
    gX = to_f64(dX)[rows]
    for i, t in enumerate(rows):
        assert rel_l2(gX[i], rX[i]) <= 2e-2, t
