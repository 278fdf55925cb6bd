"""Pins for the oracle's element and scale codecs (Sec. 3.1, Eq. 1-3).

Each oracle codec finds the nearest representable value by comparing exact distances. The
references here are written differently, so that a mistake in either shows up:
  * E2M1: a threshold table derived by hand from the midpoints of the grid {0, .5, 1, 1.5, 2, 3, 4, 6}
    and the ties-to-even rule, checked exhaustively over every fp32 value in the decision range.
  * E8M0 (rounded up): ceil(log2(s)) in float64, over whole binades and every exponent's edges.
  * E4M3: the integer round-half-to-even trick on the fp32 bit pattern, exhaustively over the
    whole E4M3 range, plus the format's published extremes (max 448, min subnormal 2^-9).
  * bfloat16 rounding: torch's own float32 -> bfloat16 conversion.
"""
import numpy as np
import pytest
import torch

E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def binade(e: int, sign: int = 0) -> np.ndarray:
    """Every fp32 value 2^e <= |x| < 2^(e+1) of one sign (normal e only)."""
    mant = np.arange(1 << 23, dtype=np.uint32)
    bits = (np.uint32(sign) << np.uint32(31)) | (np.uint32(e + 127) << np.uint32(23)) | mant
    return bits.view(np.float32)


def e2m1_index_by_thresholds(a: np.ndarray) -> np.ndarray:
    # midpoints 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5; at a midpoint the even index wins, so the
    # comparison is strict where the lower neighbour is even and inclusive where it is odd
    a = a.astype(np.float64)
    return ((a > 0.25).astype(np.int32) + (a >= 0.75) + (a > 1.25) + (a >= 1.75) + (a > 2.5)
            + (a >= 3.5) + (a > 5.0))


@pytest.mark.parametrize("sign", [0, 1])
def test_e2m1_exhaustive_decision_range(oracle, sign):
    # every fp32 with 2^-3 <= |u| < 2^3 (all thresholds lie inside), both signs
    for e in range(-3, 3):
        u = binade(e, sign)
        q, code = oracle.e2m1(u)
        idx = e2m1_index_by_thresholds(np.abs(u))
        np.testing.assert_array_equal(code & 7, idx)
        np.testing.assert_array_equal(code >> 3, sign)
        ref = E2M1_GRID[idx] * (-1.0 if sign else 1.0)
        np.testing.assert_array_equal(q.astype(np.float64), ref)


def test_e2m1_outside_range_and_specials(oracle):
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 2**32, size=4_000_000, dtype=np.uint64).astype(np.uint32)
    u = bits.view(np.float32)
    u = u[~np.isnan(u)]
    u = np.concatenate([u, np.array([0.0, -0.0, np.inf, -np.inf, 6.0, -6.0, 1e-45, -1e-45,
                                     np.float32(3.4e38)], np.float32)])
    q, code = oracle.e2m1(u)
    idx = e2m1_index_by_thresholds(np.minimum(np.abs(u.astype(np.float64)), 1e30))
    np.testing.assert_array_equal(code & 7, idx)
    np.testing.assert_array_equal(code >> 3, np.signbit(u).astype(np.uint8))
    # P1: every value lies on the E2M1 grid
    assert np.isin(np.abs(q.astype(np.float64)), E2M1_GRID).all()
    assert np.abs(q).max() == 6.0


def test_e2m1_ties_and_grid_points(oracle):
    ties = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    q, code = oracle.e2m1(ties)
    # the even neighbour wins: 0, 1, 1, 2, 2, 4, 4
    np.testing.assert_array_equal(q, [0.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0])
    q, code = oracle.e2m1(E2M1_GRID.astype(np.float32))
    np.testing.assert_array_equal(q, E2M1_GRID)
    np.testing.assert_array_equal(code, np.arange(8))
    np.testing.assert_array_equal(oracle.e2m1_decode(np.arange(16)),
                                  np.concatenate([E2M1_GRID, -E2M1_GRID]))


def e8m0_ceil_reference(s: np.ndarray) -> np.ndarray:
    s64 = s.astype(np.float64)
    with np.errstate(divide="ignore"):
        e = np.ceil(np.log2(np.where(s64 > 0, s64, 1.0)))
    e = np.where(s64 > 0, e, -127)
    return (np.clip(e, -127, 127) + 127).astype(np.uint8)


def test_e8m0_ceiling_whole_binades(oracle):
    # subnormals in full, the clamp edges, and a spread of normal binades in full
    sub = np.arange(1, 1 << 23, dtype=np.uint32).view(np.float32)
    np.testing.assert_array_equal(oracle.e8m0_ceil(sub), e8m0_ceil_reference(sub))
    for e in (-126, -125, -20, -9, -1, 0, 1, 7, 125, 126, 127):
        s = binade(e)
        np.testing.assert_array_equal(oracle.e8m0_ceil(s), e8m0_ceil_reference(s))


def test_e8m0_ceiling_every_exponent(oracle):
    rng = np.random.default_rng(2)
    mant = np.concatenate([np.array([0, 1, 2, 1 << 22, (1 << 23) - 1], np.uint32),
                           rng.integers(0, 1 << 23, size=2048).astype(np.uint32)])
    for E in range(1, 255):
        s = ((np.uint32(E) << np.uint32(23)) | mant).view(np.float32)
        np.testing.assert_array_equal(oracle.e8m0_ceil(s), e8m0_ceil_reference(s))
    special = np.array([0.0, -0.0, -1.0, -np.inf, np.inf, 2.0**-127, 2.0**-126, 6.0], np.float32)
    # non-positive -> 2^-127 (byte 0); +inf saturates to 2^127 (byte 254); exact powers stay put
    np.testing.assert_array_equal(oracle.e8m0_ceil(special), [0, 0, 0, 0, 254, 0, 1, 130])


def e4m3_reference(x: np.ndarray) -> np.ndarray:
    """Round-half-to-even onto OCP E4M3FN by integer arithmetic on the fp32 bits; 0 <= x < 2^127."""
    x = np.asarray(x, np.float32)
    bits = x.view(np.uint32)  # non-negative and below 2^127, so the additions cannot overflow
    # normal range (x >= 2^-6): keep 3 mantissa bits (drop 20), round half to even
    r = (bits + np.uint32(0x7FFFF) + ((bits >> 20) & 1)) & np.uint32(0xFFF00000)
    exp = (r >> 23).astype(np.int32) - 127
    man = ((r >> 20) & 7).astype(np.int32)
    byte_n = np.where((exp > 8) | ((exp == 8) & (man > 6)), 126, (exp + 7) * 8 + man)
    # subnormal range: multiples of 2^-9, round half to even
    small = np.minimum(x, np.float32(2.0**-6)).astype(np.float64)
    byte_s = np.rint(small * 512.0).astype(np.int32)
    return np.where(x >= np.float32(2.0**-6), byte_n, byte_s).astype(np.uint8)


def test_e4m3_exhaustive_range(oracle):
    # every positive fp32 from 2^-11 to 2^9: below 2^-10 everything rounds to 0, above 464 to 448
    for e in range(-11, 9):
        x = binade(e)
        np.testing.assert_array_equal(oracle.e4m3(x), e4m3_reference(x))


def test_e4m3_published_points(oracle):
    vals = oracle.e4m3_decode(np.arange(127))
    assert np.all(np.diff(vals) > 0)  # codes 0x00..0x7E increase monotonically
    assert vals[0x7E] == 448.0 and vals[1] == 2.0**-9 and vals[8] == 2.0**-6 and vals[0x38] == 1.0
    x = np.array([448, 464, 500, 1e30, np.inf, 0, -1, -np.inf, 2.0**-9, 2.0**-10, 1.5 * 2.0**-10,
                  1.0625, 1.1875, 0.3], np.float32)
    expect = [126, 126, 126, 126, 126, 0, 0, 0, 1, 0, 1, 0x38, 0x3A, 42]
    np.testing.assert_array_equal(oracle.e4m3(x), expect)


def test_bf16_round_matches_torch(oracle):
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2**32, size=8_000_000, dtype=np.uint64).astype(np.uint32)
    # add every tie pattern (low half exactly 0x8000) for a spread of high halves
    hi = rng.integers(0, 2**16, size=200_000, dtype=np.uint64).astype(np.uint32)
    bits = np.concatenate([bits, (hi << 16) | 0x8000, (hi << 16) | 0x7FFF, (hi << 16) | 0x8001,
                           np.array([0x7F7F8000, 0x7F7FFFFF, 0xFF7F8000, 0x7F800000, 0], np.uint32)])
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    ours = oracle.bf16_round(x)
    theirs = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(ours.view(np.uint32), theirs.view(np.uint32))
