"""Helpers shared by the GPU parity tests: numpy <-> torch marshalling of stored inputs
and comparison of library outputs with the oracle."""
import numpy as np
import torch

from paper_2603_23198_amd import binding as b


def dev(a, dtype=None):
    """numpy stored array -> device tensor (uint16 bf16 bits -> torch.bfloat16)."""
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_bits(t):
    """device tensor -> numpy (bf16 as uint16 bits)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.int16:
        return t.numpy().view(np.uint16)
    return t.numpy()


def to_f64(t):
    t = t.detach().cpu()
    return t.float().double().numpy() if t.dtype == torch.bfloat16 else t.double().numpy()


def rel_l2(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(a - ref) / (den if den > 0 else 1.0)


def twell_views(bufs, T, f, cfg):
    """Reshape flat buffers to their documented shapes (numpy, on host)."""
    NT = -(-f // cfg.tile_cols)
    S, K = cfg.tile_slots, cfg.ell_width
    out = {
        "val": host_bits(bufs["val"])[:T * NT * S].reshape(T, NT * S),
        "idx": host_bits(bufs["idx"])[:T * NT * S].reshape(T, NT * S),
        "cnt": host_bits(bufs["cnt"])[:T * NT].reshape(T, NT),
        "row_nnz": host_bits(bufs["row_nnz"])[:T],
        "row_ovf": host_bits(bufs["row_ovf"])[:T],
        "n_ovf": int(host_bits(bufs["n_ovf"])[0]),
        "ovf_rows": host_bits(bufs["ovf_rows"]),
    }
    if bufs.get("ell_val") is not None:
        out["ell_val"] = host_bits(bufs["ell_val"])[:T * K].reshape(T, K)
        out["ell_idx"] = host_bits(bufs["ell_idx"])[:T * K].reshape(T, K)
    return out


def assert_twell_equal(got, tw, hy, rows=None, check_ell=True):
    """Bit-exact comparison on the specified (unique) parts: counts, the valid slots,
    row_nnz, the overflow set and list, and the ELL rows of sparse rows."""
    S = tw.tile_slots
    rows = np.arange(tw.cnt.shape[0]) if rows is None else rows
    np.testing.assert_array_equal(got["cnt"][rows], tw.cnt[rows])
    np.testing.assert_array_equal(got["row_nnz"][rows], hy.row_nnz[rows])
    np.testing.assert_array_equal(got["row_ovf"][rows].astype(bool), hy.is_ovf[rows])
    for j in range(tw.n_tiles):
        nv = np.minimum(tw.cnt[rows, j], S)
        for s in range(S):
            sel = rows[nv > s]
            if len(sel) == 0:
                break
            np.testing.assert_array_equal(got["idx"][sel, j * S + s], tw.idx[sel, j * S + s])
            np.testing.assert_array_equal(got["val"][sel, j * S + s].view(tw.val.dtype), tw.val[sel, j * S + s])
    if check_ell and "ell_idx" in got:
        for t in rows:
            if hy.is_ovf[t]:
                continue
            c = int(hy.row_nnz[t])
            np.testing.assert_array_equal(got["ell_idx"][t, :c], hy.ell_idx[t, :c])
            np.testing.assert_array_equal(got["ell_val"][t, :c].view(hy.ell_val.dtype), hy.ell_val[t, :c])
