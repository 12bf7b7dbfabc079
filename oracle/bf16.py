"""Exact bfloat16 codec for the oracle (test infrastructure only).

bfloat16 keeps the float32 sign and 8-bit exponent and 7 stored significand
bits.  The paper does not state the cache dtype; the stored cache is taken to
be bfloat16 with round-to-nearest-even (ties to even) for the Qwen-shaped
workloads.  Values are carried as uint16 bit patterns because numpy has no
bfloat16 type.

``encode`` rounds a float64 value to bfloat16 in ONE step (no detour through
float32, which would round twice).
"""
import numpy as np

_EXP_MIN = -126          # smallest normal exponent of bfloat16 (same as float32)
_MANT_BITS = 7           # stored significand bits
_CHUNK = 1 << 16         # elements per slice in encode


def decode(bits):
    """uint16 bf16 bit patterns -> float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def encode(x):
    """float64 -> uint16 bf16 bit patterns, round to nearest, ties to even.

    For |x| with leading-bit exponent e the representable spacing (quantum) is
    2**(e - 7) for normals and 2**(-126 - 7) in the subnormal range.  Scaling
    by the inverse quantum is exact (a power of two), numpy.rint rounds half
    to even, and the rounded value times the quantum is exactly representable
    in bf16 (and in float32), so its float32 bit pattern shifted right by 16
    is the answer.  The exponent e is read from the float64 bit pattern.
    """
    x = np.asarray(x, dtype=np.float64)
    if x.size > _CHUNK:  # elementwise: the same steps, one cache-sized slice at a time
        flat = x.reshape(-1)
        out = np.empty(flat.shape, dtype=np.uint16)
        for i in range(0, flat.size, _CHUNK):
            out[i:i + _CHUNK] = encode(flat[i:i + _CHUNK])
        return out.reshape(x.shape)
    a = np.abs(x)
    ebits = (a.view(np.uint64) >> np.uint64(52)).astype(np.int64)   # biased exponent
    lead = np.where(ebits == 0, -1075, ebits - 1023)                 # fp64 subnormals: far below bf16 range
    qexp = np.maximum(lead, _EXP_MIN) - _MANT_BITS
    q = ((qexp + 1023).astype(np.uint64) << np.uint64(52)).view(np.float64)       # 2**qexp
    iq = ((1023 - qexp).astype(np.uint64) << np.uint64(52)).view(np.float64)      # 2**-qexp
    with np.errstate(over="ignore", invalid="ignore"):
        y = np.rint(a * iq) * q
        ovf = ~(y < 2.0 ** 128)                                      # overflow, inf and nan
        hb = (np.where(ovf, 0.0, y).astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    hb = np.where(ovf, np.uint16(0x7F80), hb)
    hb = np.where(np.isnan(x), np.uint16(0x7FC0), hb)
    sign = np.where(np.signbit(x), np.uint16(0x8000), np.uint16(0))
    return (hb | sign).astype(np.uint16)


def round_f64(x):
    """float64 -> float64 value of its bf16 rounding."""
    return decode(encode(x))
