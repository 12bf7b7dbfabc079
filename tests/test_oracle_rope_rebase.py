"""Pins for the oracle's mRoPE primitives (Eq. 2) and the delta rotation (Eq. 3).

Independent anchors: complex multiplication (textbook planar rotation), the
relative-position property of RoPE, the closed form of the Qwen frequency
table, and the paper's own invariants for re-basing: re-based keys equal keys
rotated directly at the global coordinate, rotations compose additively,
norms are preserved, Delta = 0 is the identity and values are never touched.
"""
import numpy as np
import pytest

from oracle import bf16, compose, rebase, rope
from paper_2607_19547_amd import synth

QW = synth.WORKLOADS["qwen8k"]


def test_inv_freq_closed_form():
    th = rope.inv_freq(128, 1e6)
    assert th.shape == (64,) and th[0] == 1.0
    assert th[32] == pytest.approx(1e-3, rel=1e-14)         # 1e6 ** (-64/128)
    r = th[1:] / th[:-1]
    assert np.allclose(r, 1e6 ** (-2 / 128), rtol=1e-13)   # geometric with ratio base^(-2/D)


def test_axis_assignment_sections():
    s = rope.axis_of_pair((16, 24, 24))
    assert s.tolist() == [0] * 16 + [1] * 24 + [2] * 24
    assert rope.axis_of_pair((2, 3, 3)).tolist() == [0, 0, 1, 1, 1, 2, 2, 2]


def test_rotation_is_complex_multiplication():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 16))
    phi = rng.uniform(-50, 50, (5, 8))
    y = rope.rotate_pairs(x, phi)
    z = (x[:, :8] + 1j * x[:, 8:]) * np.exp(1j * phi)
    assert np.allclose(y[:, :8], z.real, atol=1e-13) and np.allclose(y[:, 8:], z.imag, atol=1e-13)
    # counter-clockwise: (1, 0) turned by pi/2 is (0, 1)
    e = np.zeros(2); e[0] = 1.0
    out = rope.rotate_pairs(e, np.array([np.pi / 2]))
    assert np.allclose(out, [0.0, 1.0], atol=1e-15)


def test_single_axis_coordinates_touch_only_their_sections():
    th, sg = rope.inv_freq(16, 1e6), rope.axis_of_pair((2, 3, 3))
    x = np.random.default_rng(1).standard_normal((3, 16))
    for axis, pairs in ((0, [0, 1]), (1, [2, 3, 4]), (2, [5, 6, 7])):
        p = np.zeros((3, 3)); p[:, axis] = 7
        y = rope.apply_mrope(x, p, th, sg)
        moved = [i for i in range(8) if not (np.allclose(y[:, i], x[:, i]) and np.allclose(y[:, i + 8], x[:, i + 8]))]
        assert moved == pairs


def test_relative_position_property():
    # <f(q,p), f(k,p')> depends only on p' - p, per axis
    th, sg = rope.inv_freq(128, 1e6), rope.axis_of_pair((16, 24, 24))
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((2, 128))
    p, pp, d = np.array([3, 5, 7]), np.array([40, 2, 11]), np.array([1000, -4, 9])
    a = rope.apply_mrope(q, p, th, sg) @ rope.apply_mrope(k, pp, th, sg)
    b = rope.apply_mrope(q, p + d, th, sg) @ rope.apply_mrope(k, pp + d, th, sg)
    assert a == pytest.approx(b, rel=1e-10, abs=1e-10)


def _setup(w, seed=0):
    th, sg = rope.inv_freq(w.head_dim, w.base), rope.axis_of_pair(w.sections)
    loc = synth.local_coords(w)
    off = synth.chunk_offsets(w)
    cs = w.chunk_start
    x = synth.draw_normal((2, w.n_tokens, w.head_dim), seed, 0, 0, 0)
    return th, sg, loc, off, cs, x


@pytest.mark.parametrize("name", ["tiny", "qwen8k", "rebase8k"])
def test_rebase_equals_direct_rotation_f64(name):
    """I1 (Eq. 3): R(Delta) f(x, p) = f(x, p')."""
    w = synth.WORKLOADS[name]
    th, sg, loc, off, cs, x = _setup(w)
    stored = rope.apply_mrope(x, loc, th, sg)
    glob = compose.global_coords(loc, cs, off)
    direct = rope.apply_mrope(x, glob, th, sg)
    reb = rebase.rebase_f64(stored, cs, off, th, sg)
    assert np.max(np.abs(reb - direct)) < 1e-9      # angles up to ~1e5 rad: fp64 rounding of the angle


def test_rebase_composes_additively_and_preserves_norm():
    """I2 and I3: rebase(a) then rebase(b) == rebase(a + b); pair norms unchanged."""
    w = synth.WORKLOADS["rebase8k"]
    th, sg, loc, off, cs, x = _setup(w)
    off2 = np.random.default_rng(5).integers(-50, 50, off.shape)
    two = rebase.rebase_f64(rebase.rebase_f64(x, cs, off, th, sg), cs, off2, th, sg)
    one = rebase.rebase_f64(x, cs, off + off2, th, sg)
    assert np.max(np.abs(two - one)) < 1e-9
    P = w.head_dim // 2
    n0 = np.hypot(x[..., :P], x[..., P:])
    n1 = np.hypot(two[..., :P], two[..., P:])
    assert np.allclose(n0, n1, rtol=1e-12, atol=1e-12)


def test_zero_offset_is_bit_identity_and_values_untouched():
    """I4: chunks with Delta = 0 come back bit-identical (both storage dtypes)."""
    w = synth.WORKLOADS["qwen8k"]
    th, sg, loc, off, cs, x = _setup(w)
    bits = bf16.encode(x)
    out = rebase.rebase_stored(bits, "bf16", cs, off, th, sg)
    assert np.array_equal(out[:, :int(cs[1])], bits[:, :int(cs[1])])     # chunk 0 has Delta = 0
    assert not np.array_equal(out[:, int(cs[1]):], bits[:, int(cs[1]):])
    zero = np.zeros_like(off)
    assert np.array_equal(rebase.rebase_stored(bits, "bf16", cs, zero, th, sg), bits)
    f32 = x.astype(np.float32)
    assert np.array_equal(rebase.rebase_stored(f32, "f32", cs, zero, th, sg), f32)


def test_bf16_rebase_within_one_rounding_of_exact():
    """I1 in bf16: rebased storage differs from the exact rotation of the stored
    value by at most half an ulp of the result, so by <= 2^-8 |pair|."""
    w = synth.WORKLOADS["rebase8k"]
    th, sg, loc, off, cs, x = _setup(w)
    bits = bf16.encode(rope.apply_mrope(x, loc, th, sg))
    exact = rebase.rebase_f64(bf16.decode(bits), cs, off, th, sg)
    got = bf16.decode(rebase.rebase_stored(bits, "bf16", cs, off, th, sg))
    P = w.head_dim // 2
    pn = np.hypot(exact[..., :P], exact[..., P:])
    pn = np.concatenate([pn, pn], axis=-1)
    assert np.all(np.abs(got - exact) <= 2.0 ** -8 * pn + 2.0 ** -133)
    # and it is the correctly rounded value (single rounding)
    assert np.array_equal(bf16.encode(exact), bf16.encode(got))


def test_layer0_fidelity_ordering_table1():
    """Table 1, layer 0 (qualitative): 3-axis re-basing reconstructs the keys of
    a joint prefill (rotation at global coordinates) to rounding level, while
    naive concatenation (no re-basing) is far off."""
    w = synth.WORKLOADS["qwen8k"]
    th, sg, loc, off, cs, x = _setup(w)
    glob = compose.global_coords(loc, cs, off)
    joint = rope.apply_mrope(x, glob, th, sg)
    stored = bf16.encode(rope.apply_mrope(x, loc, th, sg))
    three = bf16.decode(rebase.rebase_stored(stored, "bf16", cs, off, th, sg))
    naive = bf16.decode(stored)

    def rel_mse(a):
        return np.sum((a - joint) ** 2) / np.sum(joint ** 2)
    assert rel_mse(three) < 1e-4          # bf16 rounding level (two roundings)
    assert rel_mse(naive) > 1e-2
    assert rel_mse(three) < rel_mse(naive) * 1e-2


def test_float32_angles_fail_at_large_offsets():
    """P2: why the delta angles are formed in float64.  At Delta_t = 1e5 the
    temporal pairs turn by up to 1e5 rad, where float32 spacing is 2^-7 rad;
    forming Delta_t * theta_i in float32 moves the rotated key by more than a
    bf16 ulp, while the float64 angles of the oracle keep the single rounding."""
    th, sg = rope.inv_freq(128, 1e6), rope.axis_of_pair((16, 24, 24))
    rng = np.random.default_rng(21)
    x = bf16.decode(bf16.encode(rng.standard_normal((4096, 128))))
    off = np.array([[100000, 0, 0]])
    exact_phi = rebase.chunk_phases(off, th, sg)[0]
    phi32 = (np.float32(off[0, 0]) * th.astype(np.float32)).astype(np.float64)
    phi32 = np.where(sg == 0, phi32, exact_phi)          # only the temporal pairs move
    exact = rope.rotate_pairs(x, exact_phi)
    via32 = bf16.decode(bf16.encode(rope.rotate_pairs(x, phi32)))
    via64 = bf16.decode(rebase.rebase_stored(bf16.encode(x), "bf16", np.array([0, 4096]), off, th, sg))
    _, e = np.frexp(np.abs(exact))
    ulp = np.ldexp(1.0, np.maximum(e - 1, -126) - 7)    # bf16 spacing at each exact value
    assert np.max(np.abs(via32 - exact) / ulp) > 1.0    # float32 angles: beyond one bf16 ulp
    assert np.all(np.abs(via64 - exact) <= 0.5 * ulp)   # float64 angles: one correct rounding
    assert np.array_equal(via64, bf16.decode(bf16.encode(exact)))
