"""Per-token key deviation (paper Section 2, Eq. 5).

delta_t = || k_t^{1,recomp} - k_t^{1,stored} ||_2 for every later-chunk token
t in [chunk_start[1], T).  Readings: the norm covers the whole key of token t
at the scoring layer, i.e. all H_kv heads x D dims concatenated; the stored key
is the rebased one (scoring happens after composition).

The selection decision is taken on float32 scores: delta is computed in
float64 and rounded once to float32, the precision the GPU path ranks in.
"""
import numpy as np


def deviation_f64(k_stored_layer, k_fresh, cs1):
    """delta_t in float64.

    k_stored_layer : float64 [H_kv, T, D]   stored (rebased) keys at the scoring layer
    k_fresh        : float64 [H_kv, n, D]   recomputed keys, row r <-> token cs1 + r
    returns        : float64 [n]
    """
    d = k_fresh - k_stored_layer[:, cs1:, :]
    return np.sqrt(np.sum(d * d, axis=(0, 2)))


def deviation_f32(k_stored_layer, k_fresh, cs1):
    """delta_t rounded once to float32 (the values the selection ranks)."""
    return deviation_f64(k_stored_layer, k_fresh, cs1).astype(np.float32)
