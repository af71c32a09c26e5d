"""Helpers for the oracle's pin tests: brute-force constructions written
directly from the paper's statements, independent of the oracle's code."""

from fractions import Fraction

import numpy as np


def eq1_rows_brute(H, n, i0, p):
    """Boolean per-row mask of the key/value context of 0-based patch i0,
    marked literally from Eq. 1 with the paper's 1-based patch numbers.

    The number of rows "p h" is the exact rational floor of p*h, with p
    read as the decimal it was written as (reading R2 without floating
    point)."""
    h = H // n
    I = i0 + 1  # paper's 1-based index
    ph = int(Fraction(str(p)) * h // 1)
    ph = min(ph, h)
    mask = np.zeros(H, dtype=bool)
    for row in range(H):
        patch = row // h + 1
        pos = row % h
        if patch == I:
            mask[row] = True                      # the local patch itself
        if I > 1 and patch == I - 1 and pos >= h - ph:
            mask[row] = True                      # lower ph of x^(i-1)
        if I < n and patch == I + 1 and pos < ph:
            mask[row] = True                      # upper ph of x^(i+1)
    return mask


def eq1_token_ids_brute(H, W, n, i0, p):
    mask = eq1_rows_brute(H, n, i0, p)
    grid = np.zeros((H, W), dtype=bool)
    grid[mask, :] = True
    return np.flatnonzero(grid.reshape(-1)).astype(np.int32)


def full_grid(cfg, kind, local, variant, synth):
    """[B, H*W, C] float64 grid where row band `local` holds the fresh draw
    and every other band its stale copy."""
    bands = []
    for j in range(cfg.n):
        bands.append(synth.patch_tensor(cfg, j, kind, stale=(j != local), variant=variant))
    return np.concatenate(bands, axis=1)
