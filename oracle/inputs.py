"""Post-rotary caches for the parity tests, built from the generator's draws
with the oracle's own Eq. 2 (test infrastructure only).

Noise model for the fresh rows (the model's recompute is out of scope, so its
output is synthetic): for candidate token t with pre-rotary stored key x_t,
  fresh key    = f(x_t + s_t z_t, p'_t)     (rotated at GLOBAL coordinates)
  fresh value  = v_t + s_t z'_t
  fresh query  = f(q_t, p'_t),  q_t ~ N(0, 1)
with z, z' ~ N(0, 0.1^2) per element and s_t ~ LogNormal(0, 1) per token,
shared by all layers and heads.  Stored keys are f(x_t, p_t) at LOCAL
coordinates.  Everything is rounded once to the storage dtype.
"""
import numpy as np

from . import bf16, compose, rope


def _enc(x, dtype):
    return bf16.encode(x) if dtype == "bf16" else x.astype(np.float32)


def build(w, layers=None, synth=None, q_layers=None):
    """Storage-dtype arrays of a workload for the given layers (default: all).

    Returns dict with k_stored, v_stored [L', H_kv, T, D], q_fresh [L', H_q, n, D],
    k_fresh, v_fresh [L', H_kv, n, D], plus chunk_start, chunk_offsets,
    local_coords, global_coords and the list of layers drawn.

    q_layers: layers whose fresh queries are drawn (default: all).  The other
    layers get a copy of the queries of the first layer in q_layers, which
    keeps large test inputs cheap to build where only some layers' attention
    is compared against the oracle.
    """
    if synth is None:
        from paper_2607_19547_amd import synth
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    theta = rope.inv_freq(w.head_dim, w.base)
    sigma = rope.axis_of_pair(w.sections)
    cs = w.chunk_start
    off = synth.chunk_offsets(w)
    loc = synth.local_coords(w)
    glob = compose.global_coords(loc, cs, off)
    cs1 = int(cs[1])
    s = synth.draw_token_scale(w)[None, :, None]
    q_layers = layers if q_layers is None else [l for l in layers if l in set(q_layers)]
    out = {k: [] for k in ("k_stored", "v_stored", "q_fresh", "k_fresh", "v_fresh")}
    q_first = None
    for layer in layers:
        draw_q = layer in q_layers
        which = [t for t in synth.LAYER_TENSORS if t != "q_pre" or draw_q]
        d = synth.draw_layer(w, layer, which)
        out["k_stored"].append(_enc(rope.apply_mrope(d["k_pre"], loc, theta, sigma), w.dtype))
        out["v_stored"].append(_enc(d["v"], w.dtype))
        kf = d["k_pre"][:, cs1:, :] + s * d["zk"]
        out["k_fresh"].append(_enc(rope.apply_mrope(kf, glob[cs1:], theta, sigma), w.dtype))
        out["v_fresh"].append(_enc(d["v"][:, cs1:, :] + s * d["zv"], w.dtype))
        if draw_q:
            out["q_fresh"].append(_enc(rope.apply_mrope(d["q_pre"], glob[cs1:], theta, sigma), w.dtype))
            if q_first is None:
                q_first = out["q_fresh"][-1]
        else:
            out["q_fresh"].append(None)
    out["q_fresh"] = [q_first if q is None else q for q in out["q_fresh"]]
    res = {k: np.stack(v) for k, v in out.items()}
    res.update(chunk_start=cs, chunk_offsets=off, local_coords=loc, global_coords=glob,
               layers=layers)
    return res
