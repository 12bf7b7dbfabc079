"""The hot path chained in the paper's order (paper Section 2, closing summary):
shift coordinates -> delta-rotate stored keys -> (concatenation is the layout)
-> score later-chunk tokens -> select the top rho -> per layer: scatter the
fresh rows, then the selected rows attend over the composed cache.

Storage dtypes: 'bf16' arrays are uint16 bit patterns, 'f32' arrays float32.
"""
import numpy as np

from . import attention, bf16, rebase, rope, score, select


def decode(x, dtype):
    return bf16.decode(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64)


def encode(x, dtype):
    return bf16.encode(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64).astype(np.float32)


def global_coords(local_coords, chunk_start, chunk_offsets):
    """p' = p + Delta_c for every token of chunk c (Section 2, before Eq. 3)."""
    g = np.array(local_coords, dtype=np.int64, copy=True)
    off = np.asarray(chunk_offsets, dtype=np.int64).reshape(-1, 3)
    for c in range(len(chunk_start) - 1):
        g[int(chunk_start[c]):int(chunk_start[c + 1])] += off[c]
    return g


def compose(dtype, head_dim, sections, base, chunk_start, chunk_offsets,
            k_stored, v_stored, q_fresh, k_fresh, v_fresh, rho, score_layer,
            layers=None):
    """Run every stage; returns a dict of stage outputs.

    k_stored, v_stored : [L, H_kv, T, D] storage dtype (post-rotary K at local coords)
    q_fresh            : [L, H_q, n, D]  storage dtype, fresh queries of the candidates
    k_fresh, v_fresh   : [L, H_kv, n, D] storage dtype, fresh keys / values of the candidates
    layers             : iterable of layers to attend (default: all)
    """
    theta = rope.inv_freq(head_dim, base)
    sigma = rope.axis_of_pair(sections)
    cs1 = int(chunk_start[1])
    T = int(chunk_start[-1])
    n = T - cs1
    L = k_stored.shape[0]

    k_reb = rebase.rebase_stored(k_stored, dtype, chunk_start, chunk_offsets, theta, sigma)
    scores = score.deviation_f32(decode(k_reb[score_layer], dtype),
                                 decode(k_fresh[score_layer], dtype), cs1)
    k = select.n_select(rho, n)
    sel = select.select_top(scores, k, cs1)

    k_post = np.array(k_reb, copy=True)
    v_post = np.array(v_stored, copy=True)
    out = {}
    for layer in (range(L) if layers is None else layers):
        k_post[layer] = attention.scatter_rows(k_reb[layer], k_fresh[layer], sel, cs1)
        v_post[layer] = attention.scatter_rows(v_stored[layer], v_fresh[layer], sel, cs1)
        o, lse = attention.attend_rows(decode(q_fresh[layer], dtype),
                                       decode(k_post[layer], dtype),
                                       decode(v_post[layer], dtype), sel, cs1)
        out[layer] = (o, lse)
    return {"k_rebased": k_reb, "scores": scores, "sel": sel,
            "k_post": k_post, "v_post": v_post, "attn": out}
