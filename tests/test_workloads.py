"""The synthetic generators hit the activity levels they are meant to stand in for."""
import numpy as np

import workloads as wl
from oracle import ffn


def test_bf16_storage_rounding_is_rne():
    from oracle import bf16
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    np.testing.assert_array_equal(wl.bf16_bits_from_f32(x), bf16.to_bf16_bits(x))


def test_row_shift_hits_target_sparsity():
    w = wl.make_ffn("probe", "bf16", 96, 1024, 4096, seed=3, sparsity=0.99)
    Z = ffn.preactivation(w.as_f64(w.X), w.as_f64(w.W_up), None, w.shift_t)
    frac = (Z > 0).mean()
    assert 0.008 < frac < 0.012, frac


def test_c1_bias_gives_sub_percent_activity():
    w = wl.c1_small_fp32()
    assert w.X.dtype == np.float32 and w.bias_f[0] == np.float32(-0.8)
    Z = ffn.preactivation(w.X, w.W_up, w.bias_f, None)
    assert 0.002 < (Z > 0).mean() < 0.012


def test_lognormal_counts_shape():
    s = wl.lognormal_row_counts(4096, 8192, seed=0)
    n = (1 - s) * 8192
    assert 70 < n.mean() < 90 and n.max() <= 1000 and n.min() >= 1
    assert 0.10 < (n > 128).mean() < 0.22
