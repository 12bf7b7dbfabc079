"""Top-rho selection of later-chunk tokens (paper Section 2, after Eq. 5).

The top rho fraction of later-chunk tokens by deviation is recomputed.
Readings: candidates are all tokens of chunks 2..N (t >= chunk_start[1]); the
count is k = 0 for rho = 0, else min(n, ceil(rho * n - 1e-9)); selection is
global across the later chunks; equal scores are broken toward the lower token
index; the result is returned in ascending token order.
"""
import math

import numpy as np


def n_select(rho, n):
    """Number of repaired tokens for fraction rho of n candidates."""
    rho = float(rho)
    if not (0.0 <= rho <= 1.0):
        raise ValueError("rho must lie in [0, 1]")
    if rho == 0.0 or n == 0:
        return 0
    return min(int(n), int(math.ceil(rho * n - 1e-9)))


def select_top(scores, k, cs1):
    """Ascending global indices of the k largest scores (lower index wins ties).

    scores : [n] score of token cs1 + r at position r
    """
    scores = np.asarray(scores)
    n = scores.shape[0]
    idx = np.arange(n)
    order = np.lexsort((idx, -scores.astype(np.float64)))   # primary: score desc, then index asc
    return np.sort(order[:k]).astype(np.int64) + int(cs1)
