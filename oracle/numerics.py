"""Storage roundings used by the COBS descriptor (oracle side).

Sec. 5.5 of the paper stores the block mean in bf16 and the scaled
eigenvectors in FP4 E2M1 with one fp32 scale per eigenvector.  The paper does
not fix the scale rule or the rounding; the reading used throughout is:

* fp32 storage: round-to-nearest-even (RNE) of the exact value.
* bf16 storage: RNE of the exact value to 8 significant bits.
* E2M1 storage of a vector x (one fp32 scale per vector):
    1. x is held in fp32 (RNE),
    2. scale = fp32(max_i |x_i|) / 6, one correctly rounded fp32 division,
    3. y_i = x_i / scale, one correctly rounded fp32 division each,
    4. |y_i| is clamped to 6 and rounded to the nearest point of the E2M1
       magnitude grid {0, 0.5, 1, 1.5, 2, 3, 4, 6}; a tie goes to the grid
       point with the even 3-bit code,
    5. the sign is kept in bit 3 unless the magnitude code is 0 (no -0),
    6. max|x| == 0 gives scale 0 and all codes 0,
    7. element 2j sits in the low nibble of byte j, element 2j+1 in the high.
  Decoding is code value times scale, computed in float64 (exact).

This module is test infrastructure (see the package docstring).
"""

import numpy as np

# E2M1 magnitudes indexed by the 3-bit code (exponent bits e1 e0, mantissa bit m).
E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)


def round_fp32(x):
    """RNE of float64 values to float32 (returned as float64)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_bf16(x):
    """RNE of float64 values to bfloat16 (8 significant bits), returned as float64.

    Written from the definition: x = m * 2**e with 0.5 <= |m| < 1, keep
    round_half_even(m * 2**8) / 2**8.  Inputs are assumed to lie in the normal
    bf16 range (true for every descriptor value the library stores).
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def bf16_bits(x):
    """uint16 bit patterns of bf16 values (x must already be bf16-representable)."""
    v = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def bf16_from_bits(bits):
    """float64 values of uint16 bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def _e2m1_magnitude_code(mag):
    """Nearest E2M1 grid index for each non-negative fp32 magnitude (<= 6), ties to even code."""
    mag = np.asarray(mag, dtype=np.float64)
    lo = np.searchsorted(E2M1_GRID, mag, side="right") - 1   # largest i with grid[i] <= mag
    lo = np.clip(lo, 0, 7)
    hi = np.clip(lo + 1, 0, 7)
    d_lo = mag - E2M1_GRID[lo]
    d_hi = E2M1_GRID[hi] - mag
    code = np.where(d_lo < d_hi, lo, hi)
    tie = (d_lo == d_hi) & (hi != lo)
    even = np.where(lo % 2 == 0, lo, hi)
    code = np.where(tie, even, code)
    return np.where(hi == lo, lo, code).astype(np.uint8)


def e2m1_encode(x):
    """Encode vectors (last axis) to E2M1 codes with one fp32 scale per vector.

    Returns (codes uint8 [..., dim] with values 0..15, scales float32 [...]).
    Arithmetic is float32, as fixed in the module docstring.
    """
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    absmax = np.max(np.abs(x32), axis=-1)
    scale = (absmax / np.float32(6.0)).astype(np.float32)
    safe = np.where(scale > 0, scale, np.float32(1.0)).astype(np.float32)
    y = (x32 / safe[..., None]).astype(np.float32)
    mag = np.minimum(np.abs(y), np.float32(6.0))
    mcode = _e2m1_magnitude_code(mag)
    sign = ((y < 0) & (mcode != 0)).astype(np.uint8)
    codes = (sign << 3) | mcode
    codes = np.where((scale > 0)[..., None], codes, 0).astype(np.uint8)
    return codes, scale


def e2m1_decode(codes, scales):
    """float64 values code_value * scale (exact in float64)."""
    codes = np.asarray(codes, dtype=np.uint8)
    mag = E2M1_GRID[codes & 7]
    sign = np.where(codes & 8, -1.0, 1.0)
    return sign * mag * np.asarray(scales, dtype=np.float32).astype(np.float64)[..., None]


def pack_nibbles(codes):
    """Pack codes [..., dim] (dim even) into bytes [..., dim/2]; element 2j in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[..., 0::2] | (codes[..., 1::2] << 4)).astype(np.uint8)


def unpack_nibbles(packed):
    """Inverse of pack_nibbles."""
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 0xF
    out[..., 1::2] = packed >> 4
    return out
