"""Pins for the oracle's bf16 rounding: IEEE round-to-nearest-even, checked against
torch's float32 -> bfloat16 conversion (a library routine) and hand-worked bit patterns."""
import numpy as np
import torch

from oracle import bf16


def torch_bits(x32):
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_hand_worked_patterns():
    one = np.float32(1.0)
    cases = [
        (1.0, 0x3F80),
        (-2.0, 0xC000),
        (0.0, 0x0000),
        (-0.0, 0x8000),
        (float(one + np.float32(2.0 ** -8)), 0x3F80),           # tie, even stays
        (float(one + np.float32(3 * 2.0 ** -8)), 0x3F82),       # tie, rounds up to even
        (float(one + np.float32(2.0 ** -8 + 2.0 ** -20)), 0x3F81),  # above the tie
        (float(np.float32(3.3895314e38)), 0x7F7F),              # max finite bf16
        (float(np.float32(3.4028235e38)), 0x7F80),              # rounds to +inf
        (float("inf"), 0x7F80),
        (float("-inf"), 0xFF80),
        (2.0 ** -133, 0x0001),                                   # smallest bf16 subnormal
        (2.0 ** -134, 0x0000),                                   # tie to even (zero)
        (3 * 2.0 ** -134, 0x0002),                               # tie to even (2)
    ]
    for x, want in cases:
        got = int(bf16.to_bf16_bits(np.array([x]))[0])
        assert got == want, (x, hex(got), hex(want))
    assert bf16.to_bf16_bits(np.array([np.nan]))[0] & 0x7FFF > 0x7F80


def test_against_library_random_and_edges():
    r = np.random.default_rng(0)
    x = np.concatenate([
        r.standard_normal(200000).astype(np.float32),
        (r.standard_normal(20000) * 1e-39).astype(np.float32),   # fp32 subnormals
        (r.standard_normal(20000) * 1e38).astype(np.float32),
        # exact ties: bf16 value + half ulp
        (np.arange(1, 5000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
    ])
    np.testing.assert_array_equal(bf16.to_bf16_bits(x.astype(np.float64)), torch_bits(x))


def test_roundtrip_is_exact():
    b = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    v = bf16.from_bf16_bits(b)
    finite = np.isfinite(v)
    np.testing.assert_array_equal(bf16.to_bf16_bits(v[finite]), b[finite])
