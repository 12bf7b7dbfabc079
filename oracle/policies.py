"""Position policies of Section 3 (Table 1) and the layer-0 key-fidelity
diagnostic (test infrastructure only).

The policies differ only in the coordinate each stored token is moved to:
  * three-axis re-basing (the method): chunk c moves by its own offset,
    p' = p + Delta_c, as a joint prefill of the composed sequence would place it;
  * Scalar1D: the visual tokens are flattened to consecutive scalar positions,
    the way text tokens are placed: token j of the composed cache (0-based, in
    cache order) goes to (j, j, j) on all three axes;
  * naive concatenation: no re-basing, every chunk stays at its local coordinates.
At layer 0 a key depends only on its token's embedding and position (Section 3),
so the joint prefill's layer-0 key of a token is the key rotated to the
three-axis target; the diagnostic compares a policy's keys with those by the
cosine similarity of each key vector (averaged) and by the relative mean
squared error sum ||k - k_joint||^2 / sum ||k_joint||^2.
"""
import numpy as np

POLICIES = ("three_axis", "scalar1d", "naive")


def target_coords(policy, local_coords, chunk_start, chunk_offsets):
    """Target coordinate [T, 3] (int64) of every token under a policy."""
    loc = np.asarray(local_coords, dtype=np.int64).reshape(-1, 3)
    T = loc.shape[0]
    if policy == "naive":
        return loc.copy()
    if policy == "scalar1d":
        j = np.arange(T, dtype=np.int64)
        return np.stack([j, j, j], axis=1)
    if policy == "three_axis":
        off = np.asarray(chunk_offsets, dtype=np.int64).reshape(-1, 3)
        out = loc.copy()
        for c in range(len(chunk_start) - 1):
            out[int(chunk_start[c]):int(chunk_start[c + 1])] += off[c]
        return out
    raise ValueError(policy)


def token_offsets(policy, local_coords, chunk_start, chunk_offsets):
    """Per-token offset p' - p [T, 3] (int64) that moves each stored key to its target."""
    loc = np.asarray(local_coords, dtype=np.int64).reshape(-1, 3)
    return target_coords(policy, loc, chunk_start, chunk_offsets) - loc


def fidelity(k, k_ref):
    """(mean cosine, relative MSE) of key vectors k against k_ref, both [..., D] float."""
    a = np.asarray(k, dtype=np.float64).reshape(-1, np.shape(k)[-1])
    b = np.asarray(k_ref, dtype=np.float64).reshape(-1, np.shape(k_ref)[-1])
    na, nb = np.linalg.norm(a, axis=1), np.linalg.norm(b, axis=1)
    cos = np.sum(a * b, axis=1) / (na * nb)
    rel = np.sum((a - b) ** 2) / np.sum(b * b)
    return float(np.mean(cos)), float(rel)
