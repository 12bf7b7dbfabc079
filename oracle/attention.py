"""Scatter of fresh K/V, then causal GQA attention of the repaired rows
(paper Section 2: Eq. 1 and the repair step after Eq. 5).

The selected tokens are recomputed through every layer while attending
causally to the full composed cache, and their new keys and values are
scattered back; all other rows stay as stored.

Readings: within a layer the fresh rows are scattered first and the selected
rows then attend over the post-scatter cache (they are recomputed jointly, so
row t sees fresh K/V for selected rows j <= t and stored K/V elsewhere); key j
is visible to row t iff j <= t in cache order (self included); the scale is
1/sqrt(D) with no bias, cap or window; q-head h reads kv-head h // (H_q/H_kv).
"""
import numpy as np


def scatter_rows(cache, fresh, sel, cs1):
    """cache [H, T, D] with rows sel replaced by fresh[:, sel - cs1] (returns a copy)."""
    out = np.array(cache, copy=True)
    sel = np.asarray(sel, dtype=np.int64)
    out[:, sel, :] = fresh[:, sel - cs1, :]
    return out


def attend_rows(q_fresh, k_cache, v_cache, sel, cs1, block=64):
    """Causal softmax attention of the selected rows, float64.

    q_fresh  : [H_q, n, D]    fresh queries, row r <-> token cs1 + r
    k_cache  : [H_kv, T, D]   post-scatter keys
    v_cache  : [H_kv, T, D]   post-scatter values
    sel      : [k] ascending token indices (>= cs1)
    returns  : o [H_q, k, D] and lse [H_q, k] (natural-log sum of exp scores)

    Rows are independent; they are processed ``block`` at a time with an
    explicit causal mask so that memory stays bounded.
    """
    Hq, _, D = q_fresh.shape
    Hkv, T, _ = k_cache.shape
    G = Hq // Hkv
    sel = np.asarray(sel, dtype=np.int64)
    k = sel.shape[0]
    o = np.zeros((Hq, k, D))
    lse = np.zeros((Hq, k))
    scale = 1.0 / np.sqrt(D)
    keys = np.arange(T)
    for b0 in range(0, k, block):
        rows = sel[b0:b0 + block]
        tmax = int(rows[-1]) + 1
        visible = keys[None, :tmax] <= rows[:, None]            # [b, tmax]
        for h in range(Hq):
            kv = h // G
            q = q_fresh[h, rows - cs1, :]                        # [b, D]
            s = (q @ k_cache[kv, :tmax, :].T) * scale            # [b, tmax]
            s = np.where(visible, s, -np.inf)
            m = np.max(s, axis=1, keepdims=True)
            w = np.exp(s - m)
            z = np.sum(w, axis=1, keepdims=True)
            o[h, b0:b0 + len(rows), :] = (w @ v_cache[kv, :tmax, :]) / z
            lse[h, b0:b0 + len(rows)] = (m + np.log(z))[:, 0]
    return o, lse
