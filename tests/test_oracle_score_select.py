"""Pins for the deviation score (Eq. 5) and the top-rho selection.

Anchors: a 3-4-5 closed form across the two KV heads, invariance of the L2
norm under a common rotation, a brute-force sort with Python's sorted(), the
special cases rho = 0 / rho = 1 / k = 1 (numpy argmax, which returns the first
maximum), all-equal scores, and the repair-fraction arithmetic of Section 2
(rho = 0.35 of the later chunks of a 4-chunk cache is about 25% of it)."""
import math

import numpy as np
import pytest

from oracle import rope, score, select


def test_score_closed_form_spans_all_heads():
    H, T, D, cs1 = 2, 10, 8, 4
    k = np.zeros((H, T, D))
    kf = np.zeros((H, T - cs1, D))
    kf[0, 2, 3] = 3.0          # token cs1 + 2: head 0 differs by 3
    kf[1, 2, 7] = -4.0         # ... and head 1 by 4
    kf[1, 5, 0] = 1.5          # token cs1 + 5
    d = score.deviation_f64(k, kf, cs1)
    assert d.tolist() == [0, 0, 5.0, 0, 0, 1.5]


def test_score_invariant_under_common_rotation():
    rng = np.random.default_rng(0)
    th, sg = rope.inv_freq(16, 1e6), rope.axis_of_pair((2, 3, 3))
    k = rng.standard_normal((2, 40, 16))
    kf = k[:, 8:] + 0.1 * rng.standard_normal((2, 32, 16))
    p = rng.integers(0, 1000, (40, 3))
    a = score.deviation_f64(k, kf, 8)
    b = score.deviation_f64(rope.apply_mrope(k, p, th, sg), rope.apply_mrope(kf, p[8:], th, sg), 8)
    assert np.allclose(a, b, rtol=1e-12)


def test_n_select():
    assert select.n_select(0.0, 100) == 0
    assert select.n_select(1.0, 100) == 100
    assert select.n_select(0.1, 6144) == 615
    assert select.n_select(0.1, 63488) == 6349
    assert select.n_select(0.25, 32) == 8
    assert select.n_select(1e-9, 5) == 1
    with pytest.raises(ValueError):
        select.n_select(1.5, 10)


def _brute(scores, k, cs1):
    order = sorted(range(len(scores)), key=lambda i: (-float(scores[i]), i))
    return sorted(i + cs1 for i in order[:k])


@pytest.mark.parametrize("seed", range(5))
def test_select_matches_sorted(seed):
    rng = np.random.default_rng(seed)
    n = 500
    s = rng.lognormal(0, 1, n).astype(np.float32)
    s[rng.integers(0, n, 60)] = s[7]            # plenty of ties
    for k in (0, 1, 2, 37, 250, 499, 500):
        assert select.select_top(s, k, 1000).tolist() == _brute(s, k, 1000)


def test_select_special_cases():
    rng = np.random.default_rng(9)
    s = rng.lognormal(0, 1, 64).astype(np.float32)
    s[40] = s.max()                               # duplicate maximum: first one wins
    assert select.select_top(s, 1, 32).tolist() == [32 + int(np.argmax(s))]
    assert select.select_top(s, 64, 32).tolist() == list(range(32, 96))
    assert select.select_top(s, 0, 32).tolist() == []
    eq = np.full(64, 2.5, dtype=np.float32)
    assert select.select_top(eq, 10, 32).tolist() == list(range(32, 42))


def test_repair_fraction_of_composed_cache():
    """Candidates are the later chunks only: with 4 equal chunks, rho = 0.35 of
    them is 0.35 * 3/4 = 26.25% of the whole cache, which the paper calls
    approximately 25% (Section 2)."""
    chunk, N = 2048, 4
    n = chunk * (N - 1)
    k = select.n_select(0.35, n)
    assert abs(k / (chunk * N) - 0.2625) < 1e-3
    assert math.isclose(0.35 * 3 / 4, 0.2625)
