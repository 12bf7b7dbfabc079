"""Pins for the per-token rebase (Eq. 3 with one offset per token) and the
position policies of Section 3 with their layer-0 fidelity diagnostic (Table 1).

Independent anchors: rotating a stored key by its token's offset equals
rotating the pre-rotary key directly at the target coordinate (Eq. 2 applied
once); the per-chunk rebase (pinned elsewhere) for chunk-wise offsets; the
global coordinates of the composition (compose.global_coords); closed forms of
the cosine and relative error; the expectation of the naive policy's error for
isotropic keys, sum over pairs of 2 (1 - cos phi) per unit energy; and the
ordering the paper reports at layer 0: three-axis at rounding level, Scalar1D
worse than naive.
"""
import numpy as np
import pytest

from oracle import bf16, compose, policies, rebase, rope
from paper_2607_19547_amd import synth


def _frame(n_chunks=3, grid=(2, 4, 4)):
    t, h, w = grid
    per = t * h * w
    loc = np.array([(a, b, c) for a in range(t) for b in range(h) for c in range(w)] * n_chunks, dtype=np.int64)
    cs = np.arange(n_chunks + 1, dtype=np.int64) * per
    return loc, cs


def test_per_token_rebase_equals_direct_rotation():
    rng = np.random.default_rng(3)
    th, sg = rope.inv_freq(16, 1e4), rope.axis_of_pair((2, 3, 3))
    loc = rng.integers(0, 40, (57, 3))
    off = rng.integers(-100000, 100000, (57, 3))
    x = rng.standard_normal((2, 57, 16))
    stored = rope.apply_mrope(x, loc, th, sg)
    got = rebase.rebase_tokens_f64(stored, off, th, sg)
    want = rope.apply_mrope(x, loc + off, th, sg)
    assert np.allclose(got, want, atol=1e-9)


def test_per_token_equals_per_chunk_for_chunkwise_offsets():
    w = synth.WORKLOADS["qwen8k"]
    th, sg = rope.inv_freq(128, w.base), rope.axis_of_pair(w.sections)
    rng = np.random.default_rng(4)
    cs = np.array([0, 100, 230, 333, 500])
    coff = np.array([[0, 0, 0], [8, 0, 0], [99991, -7, 13], [3, 2, 1]])
    tok = np.repeat(coff, np.diff(cs), axis=0)
    k = bf16.encode(rng.standard_normal((2, 3, 500, 128)))
    a = rebase.rebase_tokens_stored(k, "bf16", tok, th, sg)
    b = rebase.rebase_stored(k, "bf16", cs, coff, th, sg)
    assert np.array_equal(a, b)
    assert np.array_equal(a[:, :, :100], k[:, :, :100])          # Delta = 0 rows bit-identical


def test_policy_targets():
    loc, cs = _frame()
    off = np.array([[0, 0, 0], [5, 0, 0], [11, 2, -3]])
    tgt = policies.target_coords("three_axis", loc, cs, off)
    assert np.array_equal(tgt, compose.global_coords(loc, cs, off))
    s1 = policies.target_coords("scalar1d", loc, cs, off)
    j = np.arange(len(loc))
    assert np.array_equal(s1, np.stack([j, j, j], axis=1))
    assert np.array_equal(policies.target_coords("naive", loc, cs, off), loc)
    for p in policies.POLICIES:
        assert np.array_equal(loc + policies.token_offsets(p, loc, cs, off), policies.target_coords(p, loc, cs, off))
    # same-frame patches share a temporal coordinate but Scalar1D gives them different times
    same_frame = (loc[:, 0] == 0) & (np.arange(len(loc)) < 32)
    assert len(np.unique(loc[same_frame, 0])) == 1 and len(np.unique(s1[same_frame, 0])) == same_frame.sum()


def test_fidelity_closed_forms():
    rng = np.random.default_rng(5)
    k = rng.standard_normal((40, 16))
    assert policies.fidelity(k, k) == (pytest.approx(1.0), pytest.approx(0.0))
    c, r = policies.fidelity(k, 3.0 * k)
    assert c == pytest.approx(1.0) and r == pytest.approx((1 - 3.0) ** 2 / 9.0)
    a = np.zeros((2, 4)); a[:, 0] = 1.0
    b = np.zeros((2, 4)); b[:, 1] = 1.0
    assert policies.fidelity(a, b) == (pytest.approx(0.0), pytest.approx(2.0))


def test_naive_error_matches_expectation_for_isotropic_keys():
    """E||R(phi) v - v||^2 = 2 (1 - cos phi) E||v||^2 per pair: the naive policy's
    relative error is the mean of 2 (1 - cos phi) over tokens and pairs."""
    th, sg = rope.inv_freq(128, 1e6), rope.axis_of_pair((16, 24, 24))
    loc, cs = _frame(n_chunks=4, grid=(2, 8, 8))
    off = np.array([[0, 0, 0], [8, 0, 0], [16, 3, 0], [24, 0, 5]])
    rng = np.random.default_rng(6)
    x = rng.standard_normal((64, len(loc), 128))
    stored = rope.apply_mrope(x, loc, th, sg)
    joint = rope.apply_mrope(x, policies.target_coords("three_axis", loc, cs, off), th, sg)
    _, rel = policies.fidelity(stored, joint)
    phi = rebase.token_phases(policies.token_offsets("three_axis", loc, cs, off), th, sg)
    assert rel == pytest.approx(np.mean(2.0 * (1.0 - np.cos(phi))), rel=0.03)


@pytest.mark.parametrize("name", ["qwen8k", "long65k"])
def test_table1_layer0_ordering(name):
    """Layer 0 (keys = position-rotated embeddings), bf16 storage: three-axis
    re-basing reproduces the joint keys to rounding, naive concatenation does
    not, and the scalar collapse is worse than naive (Table 1, first row)."""
    w = synth.WORKLOADS[name]
    th, sg = rope.inv_freq(128, w.base), rope.axis_of_pair(w.sections)
    loc, cs, off = synth.local_coords(w), w.chunk_start, synth.chunk_offsets(w)
    pick = np.sort(np.random.default_rng(7).choice(w.n_tokens, 4096, replace=False))
    x = np.random.default_rng(8).standard_normal((2, w.n_tokens, 128))[:, pick]
    stored = bf16.encode(rope.apply_mrope(x, loc[pick], th, sg))
    joint = rope.apply_mrope(x, policies.target_coords("three_axis", loc, cs, off)[pick], th, sg)
    res = {}
    for p in policies.POLICIES:
        toff = policies.token_offsets(p, loc, cs, off)[pick]
        res[p] = policies.fidelity(bf16.decode(rebase.rebase_tokens_stored(stored, "bf16", toff, th, sg)), joint)
    assert res["three_axis"][1] < 1e-4 and res["three_axis"][0] > 0.9999
    assert res["naive"][1] > 1e-2
    assert res["scalar1d"][1] > res["naive"][1] and res["scalar1d"][0] < res["naive"][0]
