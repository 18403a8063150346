"""Overflow probability of a TwELL tile (Appendix A, TwELL matmul discussion).

With n active units per token spread uniformly over N hidden units, the count
in one tile of T_n columns is Binomial(T_n, n/N). The packed inference layout
keeps T_n/C - 1 slots (one word holds the count), so a tile overflows when it
holds T_n/C or more non-zeros.
"""
from __future__ import annotations

from scipy.stats import binom


def tile_overflow_probability(nnz_per_token, hidden, tile_cols=256, compression=8, count_word=True):
    slots = tile_cols // compression - (1 if count_word else 0)
    return float(binom.sf(slots, tile_cols, nnz_per_token / hidden))
