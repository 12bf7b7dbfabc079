"""Three-axis delta rotation of stored post-rotary keys (paper Section 2, Eq. 3).

Every chunk was prefilled from local coordinates; composition gives chunk c a
global coordinate interval, p' = p + Delta_c for all of its tokens (the offset
is per chunk).  Because planar rotations compose additively, the stored key
f(W_k x, p) is moved to f(W_k x, p') by one more rotation, pair i turning by
Delta_i = Delta_c[sigma(i)] * theta_i.  Values are never rotated.

Cache layout: [L][H_kv][T][D], chunks are contiguous token ranges
[chunk_start[c], chunk_start[c+1]).

The same rotation with one offset per TOKEN (``rebase_tokens_*``) moves each
token to its own target coordinate; it serves the position policies compared
in Section 3 (Table 1), e.g. the scalar re-basing, whose offset differs from
token to token.
"""
import numpy as np

from . import bf16 as _bf16
from .rope import rotate_pairs


def chunk_phases(chunk_offsets, theta, sigma):
    """Delta angles [N, D/2] in float64: Delta_c[sigma(i)] * theta_i."""
    off = np.asarray(chunk_offsets, dtype=np.float64).reshape(-1, 3)
    return off[:, sigma] * theta[None, :]


def rebase_f64(k, chunk_start, chunk_offsets, theta, sigma):
    """Rotate float64 keys k [..., T, D]; returns a new float64 array (no rounding)."""
    k = np.array(k, dtype=np.float64, copy=True)
    phases = chunk_phases(chunk_offsets, theta, sigma)
    for c in range(len(chunk_start) - 1):
        s0, s1 = int(chunk_start[c]), int(chunk_start[c + 1])
        if not np.any(np.asarray(chunk_offsets).reshape(-1, 3)[c]):
            continue
        k[..., s0:s1, :] = rotate_pairs(k[..., s0:s1, :], phases[c])
    return k


def rebase_stored(k_stored, dtype, chunk_start, chunk_offsets, theta, sigma):
    """Rebase a stored cache and round the result back to the storage dtype.

    dtype 'bf16': k_stored is uint16 bf16 bits; decoded exactly, rotated in
    float64 and rounded float64 -> bf16 (RNE) once.
    dtype 'f32' : k_stored is float32; rotated in float64, rounded to float32.
    Chunks with Delta_c = 0 are returned bit-identical.
    """
    off = np.asarray(chunk_offsets).reshape(-1, 3)
    out = np.array(k_stored, copy=True)
    for c in range(len(chunk_start) - 1):
        if not np.any(off[c]):
            continue
        s0, s1 = int(chunk_start[c]), int(chunk_start[c + 1])
        seg = out[..., s0:s1, :]
        x = _bf16.decode(seg) if dtype == "bf16" else seg.astype(np.float64)
        phi = chunk_phases(off[c:c + 1], theta, sigma)[0]
        y = rotate_pairs(x, phi)
        out[..., s0:s1, :] = _bf16.encode(y) if dtype == "bf16" else y.astype(np.float32)
    return out



def token_phases(token_offsets, theta, sigma):
    """Delta angles [T, D/2] in float64 for per-token offsets [T, 3]."""
    off = np.asarray(token_offsets, dtype=np.float64).reshape(-1, 3)
    return off[:, sigma] * theta[None, :]


def rebase_tokens_f64(k, token_offsets, theta, sigma):
    """Rotate float64 keys k [..., T, D] by a per-token offset; float64, no rounding."""
    k = np.asarray(k, dtype=np.float64)
    return rotate_pairs(k, token_phases(token_offsets, theta, sigma))


def rebase_tokens_stored(k_stored, dtype, token_offsets, theta, sigma):
    """Per-token rebase of a stored cache, rounded back to the storage dtype once.

    Tokens whose offset is (0, 0, 0) are returned bit-identical; every other row
    is decoded exactly, rotated in float64 and rounded once (bf16 RNE or float32).
    """
    off = np.asarray(token_offsets).reshape(-1, 3)
    moved = np.any(off != 0, axis=1)
    out = np.array(k_stored, copy=True)
    if not moved.any():
        return out
    seg = out[..., moved, :]
    x = _bf16.decode(seg) if dtype == "bf16" else seg.astype(np.float64)
    y = rotate_pairs(x, token_phases(off[moved], theta, sigma))
    out[..., moved, :] = _bf16.encode(y) if dtype == "bf16" else y.astype(np.float32)
    return out
