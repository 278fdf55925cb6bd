"""Pins of the oracle's OCP floor mode for E8M0 scales (an f4 variant of Q_E8M0, Sec. 3.1 Eq. 3, whose
paper default rounds up).

  * the floor codec against the exponent field of the fp32 encoding (normal numbers) and the bit
    length of the mantissa (subnormals), over every binade and its edges, plus the specials;
  * activation fake quantisation in floor mode against a separately written OCP MX quantiser
    (shared exponent floor(log2 amax) - 2, elements scaled, rounded to nearest E2M1 with ties to the
    even grid index, saturating at 6), bit for bit;
  * weight fake quantisation at the floor-mode initialisation (S_fp = amax / 4, c = 1) against the
    same quantiser: learned-scale fake quantisation starts exactly at OCP MX quantisation.
"""
import numpy as np
import pytest

from oracle import focus_oracle as O

GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def floor_exponent_by_bits(s: np.ndarray) -> np.ndarray:
    b = s.astype(np.float32).view(np.uint32).astype(np.int64)
    E, man = (b >> 23) & 0xFF, b & 0x7FFFFF
    sub = np.array([int(m).bit_length() - 1 - 149 if m else -1000 for m in man])
    e = np.where(E > 0, E - 127, sub)
    return np.clip(e, -127, 127)


def test_floor_codec_every_binade():
    vals = []
    for e in range(-149, 128):
        base = np.float32(2.0) ** np.float32(e) if e >= -126 else np.float32(np.ldexp(1.0, e))
        vals += [base, np.nextafter(base, np.float32(np.inf)), base * np.float32(1.5),
                 np.nextafter(base * np.float32(2), np.float32(0)) if e < 127 else base]
    s = np.array(vals, np.float32)
    s = s[np.isfinite(s) & (s > 0)]
    got = O.e8m0_floor(s).astype(np.int64) - 127
    np.testing.assert_array_equal(got, floor_exponent_by_bits(s))
    specials = np.array([0.0, -0.0, -1.0, np.inf, -np.inf], np.float32)
    np.testing.assert_array_equal(O.e8m0_floor(specials), [0, 0, 0, 254, 0])


def ocp_mx_quantise(X: np.ndarray) -> np.ndarray:
    """OCP MX (v1.0) quantisation of rows of 32-element blocks to E2M1 with an E8M0 shared scale."""
    M, K = X.shape
    out = np.empty_like(X)
    for r in range(M):
        for b in range(0, K, 32):
            x = X[r, b:b + 32].astype(np.float64)
            amax = np.max(np.abs(x))
            e = -127 if amax == 0 else int(np.clip(np.floor(np.log2(amax)) - 2, -127, 127))
            scale = np.ldexp(1.0, e)
            u = np.abs(x) / scale
            d = np.abs(u[:, None] - GRID[None, :])
            best = np.zeros(32, np.int64)
            for j in range(32):
                cand = np.nonzero(d[j] == d[j].min())[0]
                best[j] = cand[0] if len(cand) == 1 or cand[0] % 2 == 0 else cand[1]
            q = np.where(u >= 6.0, 6.0, GRID[best])
            out[r, b:b + 32] = np.copysign(q * scale, x)
    return out.astype(np.float32)


@pytest.mark.parametrize("seed", [0, 1])
def test_floor_activation_equals_ocp_mx(seed):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((24, 256)) * np.exp2(rng.integers(-20, 20, (24, 1)))).astype(np.float32)
    X[:, ::37] *= 40.0
    X[3, :32] = 0.0
    X[5, 32:64] = np.float32(2.0) ** -100  # exponent near the bottom, not clamped
    x_hat, _, _, _ = O.fq_act(X, 0, e8m0_floor=True)
    np.testing.assert_array_equal(x_hat.view(np.uint32), ocp_mx_quantise(X).view(np.uint32))
    # and the ceiling mode differs (it never clips): the pin would catch a mode that is ignored
    x_ceil, _, _, _ = O.fq_act(X, 0)
    assert not np.array_equal(x_ceil, x_hat)


def test_floor_weight_init_equals_ocp_mx():
    rng = np.random.default_rng(2)
    W = (rng.standard_normal((40, 320)) * 0.02).astype(np.float32)
    W.ravel()[rng.choice(W.size, 30, replace=False)] *= 10.0
    s, c, a = O.init_scales(W, 0, 8, e8m0_floor=True)
    np.testing.assert_array_equal(s, (np.abs(W).reshape(40, 10, 32).max(axis=2) / np.float32(4.0)).astype(np.float32))
    fq = O.fq_weight(W, 0, 8, s, c, a, e8m0_floor=True)
    np.testing.assert_array_equal(fq.w_hat.view(np.uint32), ocp_mx_quantise(W).view(np.uint32))
    # scale bytes are the OCP exponents
    amax = np.abs(W).reshape(40, 10, 32).max(axis=2).astype(np.float64)
    np.testing.assert_array_equal(fq.scale_bytes.astype(np.int64) - 127, np.floor(np.log2(amax)).astype(np.int64) - 2)
