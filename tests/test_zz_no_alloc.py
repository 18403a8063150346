"""sfl_ffn_forward_noalloc (the forward for callers that cannot allocate, its workspace taken
from the library's fixed device scratch) against sfl_ffn_forward on the same inputs: the
same kernels, so every output is bit-identical, and both meet the fp64 oracle. Two calls in
a row, the second with a smaller batch, so that the second starts from the scratch contents
the first left behind (counters included)."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import ffn
from tests.gpu_util import dev, rel_l2, to_f64

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")

SCRATCH = 64 << 20


def transposed(W):
    out = torch.empty((W.shape[1], W.shape[0]), dtype=W.dtype, device="cuda")
    b.sfl_transpose(W, out)
    return out


def setup(w):
    """Device inputs, weight copies and two sets of outputs for one workload."""
    X, Wu, Wd = dev(w.X), dev(w.W_up), dev(w.W_down)
    Wg = dev(w.W_gate) if w.gated else None
    WdP = torch.empty_like(Wd)
    b.sfl_pack_down_weights(Wd, WdP)
    WupT = transposed(Wu)
    WuP = None
    if w.gated:
        WuP = torch.empty_like(Wu)
        b.sfl_pack_down_weights(WupT, WuP)
    cfg = b.make_cfg(**w.cfg)
    kw = dict(W_gate=Wg, W_upT=WupT, W_gateT=transposed(Wg) if w.gated else None, W_downT=transposed(Wd),
              W_down_packed=WdP, W_up_packed=WuP, bias_f=dev(w.bias_f), shift_t=dev(w.shift_t))
    return X, Wu, Wd, cfg, kw


def outputs(w, cfg):
    bufs = b.alloc_twell(w.T, w.f, "bf16", cfg)
    for t in bufs.values():
        if t is not None and t.numel():
            t.view(torch.uint8).fill_(0xA5)  # stale contents: every output must be written
    Y = torch.full((w.T, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    return Y, bufs, b.alloc_stats()


def run_pair(w):
    X, Wu, Wd, cfg, kw = setup(w)
    Y1, bufs1, st1 = outputs(w, cfg)
    a1 = b.ffn_args(X, Wu, Wd, cfg, Y=Y1, bufs=bufs1, stats=st1, **kw)
    nbytes = b.sfl_workspace_size(a1, 0)
    assert 0 < nbytes <= SCRATCH, nbytes
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b.sfl_ffn_forward(b.ffn_args(X, Wu, Wd, cfg, Y=Y1, bufs=bufs1, stats=st1, workspace=ws, **kw))
    Y2, bufs2, st2 = outputs(w, cfg)
    # no workspace: the call takes its scratch from the library
    b.sfl_ffn_forward_noalloc(b.ffn_args(X, Wu, Wd, cfg, Y=Y2, bufs=bufs2, stats=st2, **kw))
    torch.cuda.synchronize()
    return (Y1, bufs1, st1), (Y2, bufs2, st2)


def assert_same(ref, got, w):
    (Y1, bufs1, st1), (Y2, bufs2, st2) = ref, got
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    n_ovf = int(bufs1["n_ovf"].item())
    assert int(bufs2["n_ovf"].item()) == n_ovf
    for k in ("cnt", "row_nnz", "row_ovf"):
        assert torch.equal(bufs1[k], bufs2[k]), k
    cap = min(n_ovf, bufs1["ovf_rows"].numel())
    assert torch.equal(bufs1["ovf_rows"][:cap], bufs2["ovf_rows"][:cap])
    dense1 = bufs1["ovf_dense"].view(torch.int16).reshape(-1, w.f)[:cap]
    dense2 = bufs2["ovf_dense"].view(torch.int16).reshape(-1, w.f)[:cap]
    assert torch.equal(dense1, dense2)
    s1, s2 = b.read_stats(st1), b.read_stats(st2)
    for k in ("total_nnz", "n_ovf_rows", "n_tile_ovf", "capacity_exceeded"):
        assert s1[k] == s2[k], k
    assert abs(s1["l1_sum"] - s2["l1_sum"]) <= 1e-6 * abs(s1["l1_sum"])  # float64 atomics: order varies
    return n_ovf


def oracle_y(w):
    X = w.as_f64(w.X)
    if w.gated:
        return ffn.ffn_gated_dense(X, w.as_f64(w.W_gate), w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f,
                                   w.shift_t)[0]
    return ffn.ffn_dense(X, w.as_f64(w.W_up), w.as_f64(w.W_down), w.bias_f, w.shift_t)[0]


@pytest.mark.parametrize("gated", [False, True])
def test_noalloc_forward_equals_the_workspace_forward_on_two_calls(gated):
    """First a batch above 256 tokens (fused TwELL epilogue, dense-backup rows rebuilt from the
    slabs or recomputed, split-K partial sums in the scratch), then a smaller one of 40 tokens
    (split-K up projection packed from partial sums, dense-backup GEMMs of at most 64 rows
    that count finished blocks in per-tile counters held in the scratch)."""
    for T, seed in ((600, 3), (40, 4)):
        w = wl.make_ffn("noalloc", "bf16", T, 512, 2048, seed=seed + 10 * gated, gated=gated, sparsity=0.98,
                        ell_width=96)
        w.shift_t[::9] = 10.0  # dense-backup rows
        ref, got = run_pair(w)
        n_ovf = assert_same(ref, got, w)
        assert n_ovf >= T // 9
        assert rel_l2(to_f64(got[0]), oracle_y(w)) <= 2e-2


def test_noalloc_gated_decode_then_smaller_batch():
    """The decode shape of the gated layer (T = 32, d = 4096, f = 14336, every weight copy
    given) fits the scratch; then a batch of 8 tokens."""
    for T in (32, 8):
        w = wl.c3_gated(T=T)
        w.shift_t[::4] = 10.0
        ref, got = run_pair(w)
        assert_same(ref, got, w)
        assert rel_l2(to_f64(got[0]), oracle_y(w)) <= 2e-2


def test_noalloc_rejects_a_call_larger_than_its_scratch():
    w = wl.make_ffn("noalloc-big", "bf16", 4096, 512, 4096, seed=5, sparsity=0.99, ell_width=128)
    X, Wu, Wd, cfg, kw = setup(w)
    Y, bufs, st = outputs(w, cfg)
    a = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, stats=st, **kw)
    assert b.sfl_workspace_size(a, 0) > SCRATCH
    with pytest.raises(b.SflError) as e:
        b.sfl_ffn_forward_noalloc(a)
    assert e.value.code == b.SFL_E_WORKSPACE
