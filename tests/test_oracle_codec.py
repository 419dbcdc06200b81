"""Pins of the oracle's storage roundings: bf16, FP4 E2M1 (Sec. 5.5) and the record layout.

The E2M1 value of each code is taken from the format's bit-field definition
(1 sign bit, 2 exponent bits with bias 1, 1 mantissa bit, subnormal at exponent
0), written here independently of the oracle's grid table.  bf16 rounding is
checked against torch's float32 -> bfloat16 conversion (round to nearest even).
"""

import numpy as np
import torch

from oracle import numerics as nx
from oracle import records as R


def _e2m1_from_bits(code):
    s = -1.0 if code & 8 else 1.0
    e = (code >> 1) & 3
    m = code & 1
    if e == 0:
        return s * (m / 2.0)
    return s * 2.0 ** (e - 1) * (1.0 + m / 2.0)


def test_every_code_decodes_to_its_bitfield_value():
    codes = np.arange(16, dtype=np.uint8)
    got = nx.e2m1_decode(codes[None], np.array([1.0], np.float32))[0]
    want = np.array([_e2m1_from_bits(int(c)) for c in codes])
    np.testing.assert_array_equal(got, want)


def test_grid_points_encode_exactly():
    vals = np.array([_e2m1_from_bits(c) for c in range(16) if c != 8])    # no -0
    x = np.concatenate([vals, [6.0]])                                     # absmax 6 -> scale 1
    codes, scale = nx.e2m1_encode(x[None])
    assert scale[0] == np.float32(1.0)
    np.testing.assert_array_equal(nx.e2m1_decode(codes, scale)[0], x)
    for sc in (0.37, 3.0e-3, 17.5):                                       # scaled copies round-trip too
        codes, scale = nx.e2m1_encode((x * sc)[None])
        back = nx.e2m1_decode(codes, scale)[0]
        np.testing.assert_allclose(back, x * np.float64(scale[0]), rtol=0, atol=0)


def test_midpoints_round_to_even_code_and_neighbours_to_nearest():
    mids = {0.25: 0, 0.75: 2, 1.25: 2, 1.75: 4, 2.5: 4, 3.5: 6, 5.0: 6}
    for m, code in mids.items():
        c, s = nx.e2m1_encode(np.array([[6.0, m, -m]]))
        assert s[0] == 1.0
        assert c[0, 1] == code, (m, c)
        assert c[0, 2] == (code | 8 if code else 0), (m, c)
        up = float(np.nextafter(np.float32(m), np.float32(10)))
        dn = float(np.nextafter(np.float32(m), np.float32(-10)))
        cu, _ = nx.e2m1_encode(np.array([[6.0, up]]))
        cd, _ = nx.e2m1_encode(np.array([[6.0, dn]]))
        grid = [abs(_e2m1_from_bits(k)) for k in range(8)]
        lo = max(k for k in range(8) if grid[k] < m)
        hi = min(k for k in range(8) if grid[k] > m)
        assert cu[0, 1] == hi and cd[0, 1] == lo, (m, cu, cd)


def test_scale_rule_zero_vector_and_no_negative_zero():
    x = np.array([[-3.0, 1.0, 0.5, -0.01]])
    codes, scale = nx.e2m1_encode(x)
    assert scale[0] == np.float32(np.float32(3.0) / np.float32(6.0))
    assert codes[0, 0] == (8 | 7)                        # the absmax element maps to -6
    assert codes[0, 3] == 0                               # |y| < 0.25 rounds to +0, not -0
    codes, scale = nx.e2m1_encode(np.zeros((2, 8)))
    assert np.all(scale == 0) and np.all(codes == 0)


def test_round_trip_error_within_half_step():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((200, 128)) * np.exp(rng.normal(0, 2, (200, 1)))
    codes, scale = nx.e2m1_encode(x)
    back = nx.e2m1_decode(codes, scale)
    y = np.abs(x) / scale[:, None].astype(np.float64)
    half = np.where(y <= 2.0, 0.25, np.where(y <= 4.0, 0.5, 1.0)) * scale[:, None]
    assert np.all(np.abs(back - x) <= half * (1 + 1e-6))


def test_nibble_order():
    packed = nx.pack_nibbles(np.array([[1, 2, 15, 0]], dtype=np.uint8))
    assert packed.tolist() == [[0x21, 0x0F]]
    np.testing.assert_array_equal(nx.unpack_nibbles(packed), [[1, 2, 15, 0]])


def test_bf16_rounding_matches_library_rne():
    rng = np.random.default_rng(6)
    x = (rng.standard_normal(20000) * np.exp(rng.normal(0, 4, 20000))).astype(np.float32)
    # exact midpoints between neighbouring bf16 values, both parities
    mids = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(2 + 2.0 ** -7), 3.0 * (1 + 2.0 ** -8)], np.float32)
    x = np.concatenate([x, mids])
    lib = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(nx.round_bf16(x.astype(np.float64)), lib)
    np.testing.assert_array_equal(nx.bf16_from_bits(nx.bf16_bits(lib)), lib)


def test_record_round_trip_every_dtype_pair():
    rng = np.random.default_rng(8)
    nb, d, r = 5, 128, 4
    counts = np.array([64, 64, 64, 64, 17])
    means = rng.standard_normal((nb, d))
    factors = rng.standard_normal((nb, r, d))
    for md in R.DTYPES:
        for fd in R.DTYPES:
            buf = R.encode(counts, means, factors, md, fd)
            assert buf.shape == (nb, R.layout(d, r, md, fd)["total"])
            c2, m2, f2 = R.decode(buf, d, r, md, fd)
            np.testing.assert_array_equal(c2, counts)
            ref_m = {"f32": nx.round_fp32, "bf16": nx.round_bf16,
                     "e2m1": lambda v: nx.e2m1_decode(*nx.e2m1_encode(v))}[md](means)
            np.testing.assert_array_equal(m2, ref_m)
            # decoding what was decoded and re-encoded is a fixed point
            buf2 = R.encode(c2, m2, f2, md, fd)
            np.testing.assert_array_equal(buf, buf2)
