"""sfl_pack_twell on the GPU is bit-exact against the oracle's extractor and classifier
on the same float32 pre-activations (Alg. 1 + the hybrid classification of Sec. 3.4)."""
import numpy as np
import pytest
import torch

from oracle import twell
from tests.gpu_util import assert_twell_equal, dev, twell_views

pytestmark = pytest.mark.gpu

b = pytest.importorskip("paper_2603_23198_amd.binding")


def special_z(T, f, seed, density=0.05):
    r = np.random.default_rng(seed)
    Z = r.standard_normal((T, f)).astype(np.float32)
    if Z.size == 0:
        return Z
    Z -= np.float32(np.quantile(Z, 1 - density))
    n = T * f
    pick = r.choice(n, size=min(n, 200), replace=False)
    specials = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1e-45, -1e-45, 1.1754942e-38,
                         3.4028235e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8], dtype=np.float32)
    Z.reshape(-1)[pick] = specials[np.arange(len(pick)) % len(specials)]
    return Z


CASES = [
    # T, f, T_n, S, K, cap, dtype
    (37, 300, 256, 32, 8, 0, "bf16"),
    (64, 1024, 256, 32, 32, 0, "f32"),
    (129, 777, 64, 4, 12, 0, "bf16"),
    (50, 97, 3, 2, 5, 0, "f32"),
    (33, 12, 5, 1, 2, 0, "bf16"),
    (300, 4096, 128, 8, 100, 7, "bf16"),     # capacity below the number of overflow rows
    (1, 65535, 256, 32, 2000, 0, "bf16"),    # largest index
    (0, 256, 256, 32, 8, 0, "bf16"),         # empty
    # up to 256 rows with f a multiple of 64: one workgroup per row packs and classifies
    (200, 2048, 64, 16, 40, 0, "bf16"),
    (256, 4096, 128, 8, 100, 7, "bf16"),     # capacity below the number of overflow rows
    (3, 1984, 256, 32, 64, 0, "bf16"),       # partial last tile
    (17, 320, 128, 128, 500, 0, "f32"),      # every column of a tile kept
    (2, 24576, 256, 32, 400, 0, "bf16"),     # a row of 96 KB of fp32 in LDS
]


@pytest.mark.parametrize("T,f,Tn,S,K,cap,dt", CASES)
def test_pack_bit_exact(T, f, Tn, S, K, cap, dt):
    Z = special_z(T, f, seed=T * 7 + f)
    if T > 3:
        Z[1] = 1.0        # all-active row: tile and row overflow
        Z[2] = -1.0       # all-inactive row
    cfg = b.make_cfg(tile_cols=Tn, tile_slots=S, ell_width=K, ovf_capacity=cap)
    bufs = b.alloc_twell(T, f, dt, cfg)
    stats = b.alloc_stats()
    b.sfl_pack_twell(dev(Z), dt, cfg, bufs, stats)
    torch.cuda.synchronize()
    tw = twell.extract_twell(Z, Tn, S, dt)
    hy = twell.classify(tw, K)
    got = twell_views(bufs, T, f, cfg)
    assert_twell_equal(got, tw, hy)
    n_ovf = len(hy.ovf_rows)
    assert got["n_ovf"] == n_ovf
    capv = cap if cap else T
    np.testing.assert_array_equal(got["ovf_rows"][:min(n_ovf, capv)], hy.ovf_rows[:capv])
    st = b.read_stats(stats)
    assert st["total_nnz"] == int(tw.cnt.sum())
    assert st["n_ovf_rows"] == n_ovf
    assert st["n_tile_ovf"] == hy.n_tile_ovf
    assert st["capacity_exceeded"] == int(n_ovf > capv)


def test_pack_is_deterministic():
    Z = special_z(512, 4096, seed=5, density=0.02)
    cfg = b.make_cfg(tile_cols=256, tile_slots=32, ell_width=128)
    outs = []
    for _ in range(3):
        bufs = b.alloc_twell(512, 4096, "bf16", cfg)
        for v in bufs.values():
            if v is not None:
                v.zero_()
        b.sfl_pack_twell(dev(Z), "bf16", cfg, bufs)
        torch.cuda.synchronize()
        outs.append({k: v.cpu().clone() for k, v in bufs.items() if v is not None})
    for o in outs[1:]:
        for k in o:
            assert torch.equal(o[k].view(torch.uint8), outs[0][k].view(torch.uint8)), k
