"""Three-axis multimodal RoPE primitives (paper Section 2, Eq. 2).

A visual token has coordinate p = (p_t, p_h, p_w).  Each rotary frequency i is
assigned to one axis sigma(i), and its rotation angle is p_sigma(i) * theta_i;
f(x, p) rotates every frequency pair of x by its angle.

Readings where the paper is silent (each listed in the design notes):
  * theta_i = base ** (-2 i / D), i = 0 .. D/2 - 1, in float64 (Qwen convention;
    base = 1e6 for the workloads here).
  * sigma follows the section sizes in order: the first s_t frequencies are
    temporal, the next s_h height, the last s_w width (Section 3 gives 16/24/24).
  * pair i is the element pair (i, i + D/2) ("rotate-half" layout of the model).
  * R(phi)(a, b) = (a cos phi - b sin phi, a sin phi + b cos phi), i.e. a
    counter-clockwise rotation of the point (a, b).
"""
import numpy as np

AXIS_T, AXIS_H, AXIS_W = 0, 1, 2


def inv_freq(head_dim, base):
    """theta_i for i in [0, D/2), float64."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * i / head_dim)


def axis_of_pair(sections):
    """sigma: axis index (0=t, 1=h, 2=w) of every rotary pair, from the section sizes."""
    st, sh, sw = (int(s) for s in sections)
    return np.array([AXIS_T] * st + [AXIS_H] * sh + [AXIS_W] * sw, dtype=np.int64)


def angles(coords, theta, sigma):
    """alpha_i(p) = p_sigma(i) * theta_i for every token.  coords [..., 3] -> [..., D/2]."""
    c = np.asarray(coords, dtype=np.float64)
    return c[..., sigma] * theta


def rotate_pairs(x, phi):
    """Apply R(phi_i) to pair i = (x_i, x_{i+D/2}) of the last axis.  float64."""
    x = np.asarray(x, dtype=np.float64)
    P = x.shape[-1] // 2
    a, b = x[..., :P], x[..., P:]
    c, s = np.cos(phi), np.sin(phi)
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def apply_mrope(x, coords, theta, sigma):
    """f(x, p) of Eq. 2: rotate x [..., T, D] at per-token coordinates coords [T, 3]."""
    return rotate_pairs(x, angles(coords, theta, sigma))
