"""The packed 32-bit TwELL layout (Appendix A's single-load inference format) on the GPU.

Per (row, tile) 32 words: the true count in word 0, then column | bf16 value << 16 for the
first min(count, 31) active columns in ascending order. Bars: the standalone pack and the
fused GEMM epilogue write the same words as the oracle's encoder (`oracle.twell.pack32`) of
its extraction from the same float32 pre-activations, bit for bit (words past a tile's stored
entries are unspecified and masked); the classification and the forward's output are those
of the planes layout with 31 slots, bit for bit."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import ffn, twell
from tests.gpu_util import assert_twell_equal, dev, host_bits, rel_l2, to_f64, twell_views

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")
from tests.test_gpu_forward import oracle_rows, run_forward, sample_rows, transposed  # noqa: E402

PK = b.SFL_TWELL_PACKED32


def got_words(bufs, T, f, Tn):
    NT = -(-f // Tn)
    return bufs["val"].cpu().numpy().view(np.uint32)[:T * NT * 32].reshape(T, NT * 32)


def assert_words_equal(got, want, rows=None):
    """Counts (word 0) everywhere; entry words 1 .. min(count, 31)."""
    T, W = want.shape
    rows = np.arange(T) if rows is None else rows
    NT = W // 32
    for j in range(NT):
        c = want[rows, j * 32].astype(np.int64)
        np.testing.assert_array_equal(got[rows, j * 32], want[rows, j * 32])
        for s in range(31):
            sel = rows[np.minimum(c, 31) > s]
            if len(sel) == 0:
                break
            np.testing.assert_array_equal(got[sel, j * 32 + 1 + s], want[sel, j * 32 + 1 + s])


@pytest.mark.parametrize("T,f,Tn", [(300, 1000, 256), (77, 4096, 64), (5, 640, 40)])
def test_standalone_pack_packed_words(T, f, Tn):
    r = np.random.default_rng(T + f)
    Z = r.standard_normal((T, f)).astype(np.float32) - 2.0
    Z[::7, :200] = 3.0                       # tiles over 31 entries: dense-backup rows
    Z[1, 5] = np.float32(1e-42)              # a positive subnormal is active
    Z[2, 6] = -0.0
    cfg = b.make_cfg(tile_cols=Tn, tile_slots=31, ell_width=64, layout=PK)
    bufs = b.alloc_twell(T, f, "bf16", cfg)
    b.sfl_pack_twell(torch.from_numpy(Z).cuda(), "bf16", cfg, bufs)
    torch.cuda.synchronize()
    tw = twell.extract_twell(Z, Tn, 31, "bf16")
    hy = twell.classify(tw, 64)
    assert_words_equal(got_words(bufs, T, f, Tn), twell.pack32(tw))
    g = {"row_nnz": host_bits(bufs["row_nnz"])[:T], "row_ovf": host_bits(bufs["row_ovf"])[:T]}
    np.testing.assert_array_equal(g["row_nnz"], hy.row_nnz)
    np.testing.assert_array_equal(g["row_ovf"].astype(bool), hy.is_ovf)
    ell_i = host_bits(bufs["ell_idx"])[:T * 64].reshape(T, 64)
    ell_v = host_bits(bufs["ell_val"])[:T * 64].reshape(T, 64)
    for t in np.nonzero(~hy.is_ovf)[0]:
        c = int(hy.row_nnz[t])
        np.testing.assert_array_equal(ell_i[t, :c], hy.ell_idx[t, :c])
        np.testing.assert_array_equal(ell_v[t, :c], hy.ell_val[t, :c])
    assert int(bufs["n_ovf"].item()) == len(hy.ovf_rows)


@pytest.mark.parametrize("use_wupt", [False, True])
@pytest.mark.parametrize("T,f", [(700, 2048), (2048, 16384)])
def test_fused_epilogue_packed_words_and_forward(T, f, use_wupt):
    """The up projection's epilogue writes the packed words (several tiles per persistent
    block at T = 2048, f = 16384; per-column bias and per-row shift) bit-identical to the
    oracle's encoding of the same main loop's Z; the forward's output equals the planes
    layout's (31 slots) bit for bit, dense-backup rows (rebuilt from the words) included."""
    K, s_rebuilt = (64, 0.95) if f == 2048 else (256, 0.98)
    w = wl.make_ffn("packed", "bf16", T, 512, f, seed=T + 3, sparsity=0.99, tile_slots=31, ell_width=K)
    r = np.random.default_rng(T)
    w.bias_f = (r.standard_normal(f) * 0.02).astype(np.float32)
    w.shift_t[::97] = 0.0  # about half active: tiles over 31, recomputed dense-backup rows
    # more than K active but no tile over 31: dense-backup rows rebuilt from the words
    w.shift_t[1::97] = wl.row_shift_for_sparsity(w.as_f32(w.X)[1::97], s_rebuilt)
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    WupT = transposed(Wu) if use_wupt else None
    cfg = b.make_cfg(**w.cfg)
    kw = dict(bias_f=dev(w.bias_f), shift_t=dev(w.shift_t), W_upT=WupT)
    Z = torch.empty((T, f), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, b.sfl_workspace_size(b.ffn_args(X, Wu, Wd, cfg, **kw), 0)), dtype=torch.uint8,
                     device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws), Z)
    Y1, b1, _, cfg1 = run_forward(w, use_wupt=use_wupt)            # planes, 31 slots
    w.cfg["layout"] = PK
    Y2, b2, st2, cfg2 = run_forward(w, use_wupt=use_wupt)          # packed
    tw = twell.extract_twell(Z.cpu().numpy(), 256, 31, "bf16")
    assert_words_equal(got_words(b2, T, f, 256), twell.pack32(tw))
    g1, g2 = twell_views(b1, T, f, cfg1), b2
    np.testing.assert_array_equal(host_bits(g2["row_nnz"])[:T], g1["row_nnz"])
    np.testing.assert_array_equal(host_bits(g2["row_ovf"])[:T], g1["row_ovf"])
    n_ovf = g1["n_ovf"]
    assert n_ovf >= 2 * (T // 97)
    tile_ovf = (g1["cnt"][g1["ovf_rows"][:n_ovf]] > 31).any(axis=1)
    assert 0 < tile_ovf.sum() < n_ovf  # both kinds of dense-backup row
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    d1 = host_bits(b1["ovf_dense"])[:n_ovf * f]
    d2 = host_bits(b2["ovf_dense"])[:n_ovf * f]
    np.testing.assert_array_equal(d1, d2)
    rows = sample_rows(T, 32, 6, extra=g1["ovf_rows"][:4])
    Yref, _ = oracle_rows(w, rows)
    assert rel_l2(to_f64(Y2)[rows], Yref) <= 2e-2


@pytest.mark.parametrize("T", [1, 40, 256])
def test_small_batch_packed(T):
    """Batches of at most 256 tokens with W_up^T pack the words from the split-K partial sums:
    the same words as the oracle's encoding of the fp32 pre-activations, and Y as the planes."""
    w = wl.make_ffn("packed-small", "bf16", T, 1024, 2048, seed=T, sparsity=0.97, tile_slots=31, ell_width=128)
    w.shift_t[::8] = 10.0
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    WupT = transposed(Wu)
    w.cfg["layout"] = PK
    cfg = b.make_cfg(**w.cfg)
    Z = torch.empty((T, w.f), dtype=torch.float32, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, shift_t=dev(w.shift_t), W_upT=WupT)
    ws = torch.empty(max(1, b.sfl_workspace_size(args, 0)), dtype=torch.uint8, device="cuda")
    b.sfl_up_projection(b.ffn_args(X, Wu, Wd, cfg, shift_t=dev(w.shift_t), W_upT=WupT, workspace=ws), Z)
    Y2, b2, _, _ = run_forward(w, use_wupt=True, use_wdownt=True)
    tw = twell.extract_twell(Z.cpu().numpy(), 256, 31, "bf16")
    assert_words_equal(got_words(b2, T, w.f, 256), twell.pack32(tw))
    w.cfg["layout"] = 0
    Y1, _, _, _ = run_forward(w, use_wupt=True, use_wdownt=True)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    Yref, _ = oracle_rows(w, np.arange(T))
    assert rel_l2(to_f64(Y2), Yref) <= 2e-2
