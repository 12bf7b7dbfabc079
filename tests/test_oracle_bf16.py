"""Pins for the oracle's bfloat16 codec: torch's float32->bfloat16 conversion
(round to nearest even), exact rational brute force, and known bit patterns."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import bf16


def _torch_bits(x32):
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_known_patterns():
    assert bf16.encode(np.array([1.0, -2.0, 0.0, -0.0]))[:].tolist() == [0x3F80, 0xC000, 0x0000, 0x8000]
    assert bf16.decode(np.array([0x0001], dtype=np.uint16))[0] == 2.0 ** -133
    assert bf16.decode(np.array([0x7F7F], dtype=np.uint16))[0] == (2 - 2.0 ** -7) * 2.0 ** 127
    assert np.isinf(bf16.decode(np.array([0x7F80], dtype=np.uint16))[0])


def test_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(200_000),
        rng.standard_normal(20_000) * 1e-39,          # subnormal range
        np.clip(rng.standard_normal(20_000), -3, 3) * 1.1e38,   # near overflow
        np.ldexp(rng.integers(1, 1 << 20, 20_000).astype(np.float64), -20),
    ]).astype(np.float32)
    # exact midpoints between neighbouring bf16 values (ties)
    b = rng.integers(0, 0x7F7F, 20_000).astype(np.uint32)
    mid = (((b << 16) | 0x8000).astype(np.uint32)).view(np.float32)
    x = np.concatenate([x, mid, -mid])
    assert np.array_equal(bf16.encode(x.astype(np.float64)), _torch_bits(x))


def _brute(xf):
    """Nearest bf16 by exact rational comparison of the two neighbours (ties to even)."""
    x = Fraction(xf)
    sign = 1 if x >= 0 else -1
    a = abs(x)
    # the two representable neighbours of a in its binade (quantum q)
    e = math.frexp(float(a))[1] - 1
    q = Fraction(2) ** (max(e, -126) - 7)
    lo = (a // q) * q
    hi = lo + q
    dl, dh = a - lo, hi - a
    if dl < dh:
        best = lo
    elif dh < dl:
        best = hi
    else:
        best = lo if (lo / q) % 2 == 0 else hi
    return sign * best


def test_brute_force_rational_rounding():
    rng = np.random.default_rng(1)
    vals = list(rng.standard_normal(3000)) + list(rng.standard_normal(500) * 1e-38)
    # fp64 values just around bf16 midpoints: a float32 detour would round twice
    for b in rng.integers(0x0080, 0x7F00, 300):
        m = float(np.array([(int(b) << 16) | 0x8000], dtype=np.uint32).view(np.float32)[0])
        vals += [m, math.nextafter(m, math.inf), math.nextafter(m, -math.inf),
                 m * (1 + 2.0 ** -30), m * (1 - 2.0 ** -30)]
    x = np.array(vals, dtype=np.float64)
    got = bf16.decode(bf16.encode(x))
    want = np.array([float(_brute(v)) for v in vals])
    assert np.array_equal(got, want)


def test_single_rounding_not_double():
    # 1 + 2^-8 + 2^-30 lies just above the midpoint of 1 and 1 + 2^-7.
    # Rounded once it goes up; via float32 (which drops 2^-30) it would tie to 1.0.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert bf16.encode(np.array([x]))[0] == 0x3F81
    assert _torch_bits(np.array([x], dtype=np.float32))[0] == 0x3F80


def test_roundtrip_representable():
    bits = np.arange(0, 0x7F80, dtype=np.uint16)
    assert np.array_equal(bf16.encode(bf16.decode(bits)), bits)
    assert np.array_equal(bf16.encode(bf16.decode(bits | 0x8000)), bits | 0x8000)
