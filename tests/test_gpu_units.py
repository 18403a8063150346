"""Dead-unit record and targeted re-initialisation on the GPU against the oracle.

sfl_track_active_units: bit-exact against the units the oracle's own TwELL extraction
stores (slots s < min(cnt, S)) plus the positive entries of the stored dense-backup
rows; on random pre-activations with overflowing rows this is exactly the oracle's set
of active units. sfl_reinit_dead_units: within one bf16 unit in the last place (bf16,
the fp32 intermediate may round once more than the fp64 oracle) or 1e-6 relative (fp32)
of the oracle's interpolation, live units bit-identical."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import bf16, training, twell
from tests.gpu_util import dev, host_bits

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")


def slot_units(tw, f):
    """Units named by the stored slots of the oracle's extraction."""
    S = tw.tile_slots
    seen = np.zeros(f, dtype=bool)
    for j in range(tw.cnt.shape[1]):
        c = np.minimum(tw.cnt[:, j], S)
        for s in range(S):
            rows = np.nonzero(c > s)[0]
            seen[tw.idx[rows, j * S + s].astype(np.int64)] = True
    return seen


def pattern_z(T, f, seed, density):
    r = np.random.default_rng(seed)
    Z = r.standard_normal((T, f)).astype(np.float32)
    Z -= np.float32(np.quantile(Z, 1 - density))
    if T > 2:
        Z[1, :f // 2] = 1.0                       # an overflowing row: its tiles full
    Z[:, 3::17] = -np.abs(Z[:, 3::17]) - 1.0      # units never active in this batch
    return Z


@pytest.mark.parametrize("T,f,Tn,S,K,dt", [(300, 1000, 128, 8, 40, "bf16"), (129, 777, 64, 4, 12, "f32"),
                                            (64, 4096, 256, 32, 64, "bf16")])
def test_track_pack_path(T, f, Tn, S, K, dt):
    Z = pattern_z(T, f, seed=T + f, density=0.03)
    cfg = b.make_cfg(tile_cols=Tn, tile_slots=S, ell_width=K)
    bufs = b.alloc_twell(T, f, dt, cfg)
    b.sfl_pack_twell(dev(Z), dt, cfg, bufs)
    tw = twell.extract_twell(Z, Tn, S, dt)
    hy = twell.classify(tw, K)
    assert len(hy.ovf_rows) > 0 and (tw.cnt > S).any()
    # slots only (no dense-backup rows): the stored slots' units; earlier steps kept
    last = torch.full((f,), -1, dtype=torch.int64, device="cuda")
    last[::2] = 7
    no_dense = dict(bufs)
    no_dense["ovf_dense"] = None
    b.sfl_track_active_units(no_dense, T, f, dt, cfg, 9, last)
    torch.cuda.synchronize()
    want = np.where(slot_units(tw, f), 9, np.where(np.arange(f) % 2 == 0, 7, -1))
    np.testing.assert_array_equal(last.cpu().numpy(), want)
    # with the dense-backup rows stored (as the forward stores them): every active unit
    dense = np.maximum(Z[hy.ovf_rows].astype(np.float64), 0.0)
    if dt == "bf16":
        stored = bf16.to_bf16_bits(dense)
    else:
        stored = dense.astype(np.float32)
    bufs["ovf_dense"][:stored.size].copy_(dev(stored.reshape(-1)))
    last2 = torch.zeros((f,), dtype=torch.int64, device="cuda")
    b.sfl_track_active_units(bufs, T, f, dt, cfg, 1, last2)
    torch.cuda.synchronize()
    got = last2.cpu().numpy() == 1
    np.testing.assert_array_equal(got, training.active_units(Z))
    assert not got[3::17].any()


def test_track_forward_two_batches_then_reinit():
    """Two batches of one step through sfl_ffn_forward (bf16, lognormal row counts, so
    there are dense-backup rows, stored by the forward), then the dead units' W_up
    columns re-initialised. Units with an all-zero W_up column only see the (negative)
    row shift and are never active."""
    T, d, f = 384, 512, 2048
    base = wl.make_ffn("units", "bf16", T, d, f, seed=11)
    Wu_bits = base.W_up.copy()
    Wu_bits[:, 5::9] = 0
    Wu, Wd = dev(Wu_bits), dev(base.W_down)
    cfg = b.make_cfg(tile_cols=256, tile_slots=16, ell_width=96)
    last = torch.full((f,), -1, dtype=torch.int64, device="cuda")
    seen = np.zeros(f, dtype=bool)
    unsure = np.zeros(f, dtype=bool)
    for batch in range(2):
        X = wl.make_ffn("units", "bf16", T, d, f, seed=100 + batch).X
        shift = wl.row_shift_for_sparsity(wl.f32_from_bf16_bits(X), wl.lognormal_row_counts(T, f, 5 + batch))
        Xd, sh = dev(X), dev(shift)
        bufs = b.alloc_twell(T, f, "bf16", cfg)
        Y = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
        args = b.ffn_args(Xd, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=sh)
        ws = torch.empty(max(1, b.sfl_workspace_size(args, 0)), dtype=torch.uint8, device="cuda")
        b.sfl_ffn_forward(b.ffn_args(Xd, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=sh, workspace=ws))
        b.sfl_track_active_units(bufs, T, f, "bf16", cfg, 3, last)
        Z = torch.empty((T, f), dtype=torch.float32, device="cuda")
        b.sfl_up_projection(b.ffn_args(Xd, Wu, Wd, cfg, shift_t=sh), Z)
        torch.cuda.synchronize()
        assert int(host_bits(bufs["n_ovf"])[0]) > 0
        Zn = Z.cpu().numpy().astype(np.float64)
        zmax = Zn.max(axis=0)
        tol = 1e-4 * np.sqrt(np.mean(Zn ** 2))
        seen |= zmax > tol
        unsure |= np.abs(zmax) <= tol     # within rounding of 0: may go either way
    got = last.cpu().numpy() == 3
    sure = ~unsure | seen
    np.testing.assert_array_equal(got[sure], seen[sure])
    assert not got[5::9].any() and got.sum() > f // 2
    # targeted re-initialisation of the units dead for step 3
    noise = torch.randn((d, f), dtype=torch.float32, device="cuda", generator=torch.Generator("cuda").manual_seed(1))
    W = Wu.clone()
    b.sfl_reinit_dead_units(W, last, 3, 0.1, 0.02, noise)
    torch.cuda.synchronize()
    dead = training.dead_units(last.cpu().numpy(), 3)
    assert dead[5::9].all()
    want = training.reinit_dead(wl.f32_from_bf16_bits(Wu_bits).astype(np.float64), dead, 0.1, 0.02,
                                noise.cpu().numpy(), bf16_out=True)
    check_bf16_close(wl.f32_from_bf16_bits(host_bits(W)).astype(np.float64), want)
    np.testing.assert_array_equal(host_bits(W)[:, ~dead], Wu_bits[:, ~dead])


def check_bf16_close(out, want):
    ulp = np.ldexp(1.0, np.frexp(np.abs(want))[1] - 8)
    assert (np.abs(out - want) <= ulp + 1e-30).all()


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("units_on_rows", [False, True])
@pytest.mark.parametrize("R,C", [(64, 1000), (3, 7), (1, 1)])
def test_reinit_matches_oracle(dt, units_on_rows, R, C):
    r = np.random.default_rng(R * C + units_on_rows)
    W64 = r.normal(size=(R, C)) * 0.02
    nz = r.standard_normal((R, C)).astype(np.float32)
    n_units = R if units_on_rows else C
    last = r.integers(0, 6, size=n_units).astype(np.int64)
    step = 4
    if dt == "bf16":
        Wst = bf16.to_bf16_bits(W64)
        W0 = wl.f32_from_bf16_bits(Wst).astype(np.float64)
    else:
        Wst = W64.astype(np.float32)
        W0 = Wst.astype(np.float64)
    W = dev(Wst)
    b.sfl_reinit_dead_units(W, dev(last), step, 0.1, 0.02, dev(nz), units_on_rows=units_on_rows)
    torch.cuda.synchronize()
    dead = training.dead_units(last, step)
    want = training.reinit_dead(W0, dead, 0.1, 0.02, nz, units_on_rows=units_on_rows, bf16_out=dt == "bf16")
    got = host_bits(W)
    live = (~dead)[:, None] if units_on_rows else (~dead)[None, :]
    live = np.broadcast_to(live, (R, C))
    np.testing.assert_array_equal(got[live], Wst[live])
    if dt == "bf16":
        check_bf16_close(wl.f32_from_bf16_bits(got).astype(np.float64), want)
    else:
        np.testing.assert_allclose(got.astype(np.float64), want, rtol=1e-6, atol=4e-9)


def test_empty_inputs_are_no_ops():
    cfg = b.make_cfg()
    last = torch.full((10,), 4, dtype=torch.int64, device="cuda")
    b.sfl_track_active_units({}, 0, 10, "bf16", cfg, 9, last)
    W = torch.empty((0, 10), dtype=torch.bfloat16, device="cuda")
    b.sfl_reinit_dead_units(W, last, 9, 0.1, 0.02, torch.empty((0, 10), device="cuda"))
    torch.cuda.synchronize()
    assert (last.cpu() == 4).all()
