"""Pins for the oracle's fake quantisation: hand-worked examples and the properties the paper fixes.

  * golden: hand-derived examples (tests/golden/fake_quant_examples.json), each citing its equations
  * P5  c = 1 with absmax scales is plain round-to-nearest MXFP4 / NVFP4 (Sec. 3.2, Sec. 3.3)
  * P6  one coefficient per block (K = 1) is CRS: sub-blocks with equal coefficients give the same
        result (Sec. 3.4, Table "dgs_granularity": sub-block size = block size reduces DGS to CRS)
  * P7  fixed-scale idempotence; MXFP4 idempotence with re-derived scales
  * P8  power-of-two equivariance; P9 sign symmetry; P10 packed-export round trip (Fig. 3(d))
  * dynamic activation quantisation is the weight path with absmax scales and c = 1
"""
import numpy as np
import pytest

from test_oracle_codecs import E2M1_GRID, e2m1_index_by_thresholds, e4m3_reference

MX, NV = 0, 1


def as_f32(v):
    return np.array(v, dtype=np.float32)


@pytest.mark.parametrize("idx", range(5))
def test_golden_examples(oracle, golden_cases, idx):
    case = golden_cases[idx]
    fmt = MX if case["fmt"] == "mxfp4" else NV
    sb = case["sub_block"]
    rows = case.get("rows", 1)
    W = as_f32(case["w"]).reshape(rows, -1)
    c = as_f32(case["c"]).reshape(rows, -1)
    if "s_fp" in case:
        s_fp, alpha = as_f32(case["s_fp"]).reshape(rows, -1), 1.0
    else:
        s_fp, c_init, alpha = oracle.init_scales(W, fmt, sb)
        np.testing.assert_array_equal(c_init, np.ones_like(c_init))
    if "expect_s_fp" in case:
        np.testing.assert_array_equal(s_fp.ravel(), case["expect_s_fp"])
    if "expect_alpha" in case:
        assert alpha == case["expect_alpha"]
    fq = oracle.fq_weight(W, fmt, sb, s_fp, c, alpha)
    assert fq.domain_error == 0
    np.testing.assert_array_equal(fq.scale_bytes.ravel(), case["expect_scale_byte"])
    if "expect_s_dq" in case:
        np.testing.assert_array_equal(fq.s_dq.ravel(), case["expect_s_dq"])
    if "expect_codes" in case:
        np.testing.assert_array_equal(fq.codes.ravel(), case["expect_codes"])
        got = fq.w_hat.ravel()
        exp = as_f32(case["expect_w_hat"])
        np.testing.assert_array_equal(got, exp)
        np.testing.assert_array_equal(np.signbit(got), np.signbit(exp))  # signed zeros too
    else:
        blocks = W.reshape(-1, 16 if fmt == NV else 32)
        codes = fq.codes.reshape(blocks.shape)
        what = fq.w_hat.reshape(blocks.shape)
        for b, (cp, wp) in enumerate(zip(case["expect_codes_prefix"], case["expect_w_hat_prefix"])):
            np.testing.assert_array_equal(codes[b, :len(cp)], cp)
            np.testing.assert_array_equal(what[b, :len(wp)], as_f32(wp))
    if "expect_mask" in case:
        np.testing.assert_array_equal(fq.m.ravel(), case["expect_mask"])


def textbook_rtn(W: np.ndarray, fmt: int):
    """Round-to-nearest FP4 with absmax block scales, written from Eq. (1)-(3) directly."""
    B = 32 if fmt == MX else 16
    N, K = W.shape
    blocks = W.reshape(N, K // B, B).astype(np.float32)
    amax = np.abs(blocks).max(axis=2)
    if fmt == MX:
        s = (amax / np.float32(6.0)).astype(np.float32)
        with np.errstate(divide="ignore"):
            e = np.where(s > 0, np.ceil(np.log2(np.where(s > 0, s, 1).astype(np.float64))), -127)
        e = np.clip(e, -127, 127).astype(np.int32)
        S = np.ldexp(np.float32(1.0), e).astype(np.float32)
        byte = (e + 127).astype(np.uint8)
    else:
        A = np.float32(np.abs(W).max())
        alpha = np.float32(A / np.float32(2688.0)) if A > 0 else np.float32(1.0)
        d = (amax / np.float32(alpha * np.float32(6.0))).astype(np.float32)
        byte = e4m3_reference(d)
        E, m = (byte >> 3).astype(np.int32), (byte & 7).astype(np.float64)
        delta = np.where(E == 0, m / 8 * 2.0**-6, (1 + m / 8) * np.exp2(E - 7.0)).astype(np.float32)
        S = (alpha * delta).astype(np.float32)
    Sb = np.repeat(S, B, axis=1).reshape(N, K // B, B)
    with np.errstate(divide="ignore", invalid="ignore"):
        u = np.where(Sb > 0, blocks / np.where(Sb > 0, Sb, 1), 0).astype(np.float32)
    idx = e2m1_index_by_thresholds(np.abs(u))
    sign = np.signbit(blocks)
    val = np.where(sign, -E2M1_GRID[idx], E2M1_GRID[idx]).astype(np.float32)
    what = (val * Sb).astype(np.float32)
    codes = (sign.astype(np.uint8) << 3) | idx.astype(np.uint8)
    return codes.reshape(N, K), byte, what.reshape(N, K)


def weights(seed, N=64, K=256, sigma=0.02, outliers=20, f=10.0):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((N, K)) * sigma).astype(np.float32)
    idx = rng.choice(N * K, size=outliers, replace=False)
    W.ravel()[idx] *= f
    return W


@pytest.mark.parametrize("fmt", [MX, NV])
@pytest.mark.parametrize("sb", [8, 16])
def test_p5_c_one_is_round_to_nearest(oracle, fmt, sb):
    W = weights(5 + fmt)
    W[3, :32] = 0.0  # an all-zero block
    s_fp, c, alpha = oracle.init_scales(W, fmt, sb)
    fq = oracle.fq_weight(W, fmt, sb, s_fp, c, alpha)
    codes, byte, what = textbook_rtn(W, fmt)
    np.testing.assert_array_equal(fq.codes, codes)
    np.testing.assert_array_equal(fq.scale_bytes, byte)
    np.testing.assert_array_equal(fq.w_hat.view(np.uint32), what.view(np.uint32))
    # with c = 1 the quantisation scale is the dequantisation scale (Eq. 5 baseline)
    np.testing.assert_array_equal(fq.s_q, np.repeat(fq.s_dq, (32 if fmt == MX else 16) // sb, axis=1))
    # P1 on a real tensor: w_hat / S_dq lies on the grid
    B = 32 if fmt == MX else 16
    S = np.repeat(fq.s_dq, B, axis=1)
    live = S > 0
    assert np.isin(np.abs(fq.w_hat[live].astype(np.float64) / S[live]), E2M1_GRID).all() or fmt == NV


def perturbed(seed, s_fp, c):
    rng = np.random.default_rng(seed)
    s = (s_fp * np.exp2(rng.uniform(-0.5, 0.5, s_fp.shape))).astype(np.float32)
    cc = rng.uniform(0.75, 1.25, c.shape).astype(np.float32)
    return s, cc


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p6_one_coefficient_per_block_is_crs(oracle, fmt):
    B = 32 if fmt == MX else 16
    W = weights(11)
    s_fp, c, alpha = oracle.init_scales(W, fmt, 8)
    s_fp, c8 = perturbed(12, s_fp, c)
    c_block = c8[:, :: B // 8].copy()                 # one coefficient per block
    c_bcast = np.repeat(c_block, B // 8, axis=1)      # the same value on every sub-block
    a = oracle.fq_weight(W, fmt, B, s_fp, c_block, alpha)
    b = oracle.fq_weight(W, fmt, 8, s_fp, c_bcast, alpha)
    np.testing.assert_array_equal(a.codes, b.codes)
    np.testing.assert_array_equal(a.w_hat, b.w_hat)
    np.testing.assert_array_equal(a.m, b.m)
    # changing one sub-block's coefficient only moves codes inside that sub-block
    c_one = c_bcast.copy()
    c_one[:, 1] *= np.float32(1.5)
    d = oracle.fq_weight(W, fmt, 8, s_fp, c_one, alpha)
    changed = np.nonzero((d.codes != b.codes).any(axis=0))[0]
    assert len(changed) > 0 and changed.min() >= 8 and changed.max() < 16


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p7_fixed_scale_idempotence(oracle, fmt):
    W = weights(21)
    s_fp, c, alpha = oracle.init_scales(W, fmt, 8)
    s_fp, c = perturbed(22, s_fp, c)
    first = oracle.fq_weight(W, fmt, 8, s_fp, c, alpha)
    ones = np.ones_like(c)
    second = oracle.fq_weight(first.w_hat, fmt, 8, s_fp, ones, alpha)
    np.testing.assert_array_equal(second.codes, first.codes)
    np.testing.assert_array_equal(second.w_hat, first.w_hat)


def test_p7_mxfp4_rederived_scale_idempotence(oracle):
    W = weights(31)
    s_fp, c, _ = oracle.init_scales(W, MX, 8)
    s_fp, c = perturbed(32, s_fp, c)
    first = oracle.fq_weight(W, MX, 8, s_fp, c, 1.0)
    s2, c2, _ = oracle.init_scales(first.w_hat, MX, 8)
    second = oracle.fq_weight(first.w_hat, MX, 8, s2, c2, 1.0)
    np.testing.assert_array_equal(second.w_hat, first.w_hat)


@pytest.mark.parametrize("fmt", [MX, NV])
@pytest.mark.parametrize("k", [-3, 2])
def test_p8_power_of_two_equivariance(oracle, fmt, k):
    W = weights(41)
    s_fp, c, alpha = oracle.init_scales(W, fmt, 8)
    s_fp, c = perturbed(42, s_fp, c)
    base = oracle.fq_weight(W, fmt, 8, s_fp, c, alpha)
    f = np.float32(2.0**k)
    if fmt == MX:
        moved = oracle.fq_weight(W * f, fmt, 8, s_fp * f, c, alpha)
        np.testing.assert_array_equal(moved.scale_bytes.astype(int), base.scale_bytes.astype(int) + k)
    else:
        moved = oracle.fq_weight(W * f, fmt, 8, s_fp, c, alpha * f)
        np.testing.assert_array_equal(moved.scale_bytes, base.scale_bytes)
    np.testing.assert_array_equal(moved.codes, base.codes)
    np.testing.assert_array_equal(moved.w_hat, base.w_hat * f)


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p9_sign_symmetry(oracle, fmt):
    W = weights(51)
    s_fp, c, alpha = oracle.init_scales(W, fmt, 8)
    s_fp, c = perturbed(52, s_fp, c)
    a = oracle.fq_weight(W, fmt, 8, s_fp, c, alpha)
    b = oracle.fq_weight(-W, fmt, 8, s_fp, c, alpha)
    np.testing.assert_array_equal(b.w_hat, -a.w_hat)
    np.testing.assert_array_equal(b.codes, a.codes ^ 8)


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p10_packed_export_round_trip(oracle, fmt):
    W = weights(61)
    s_fp, c, alpha = oracle.init_scales(W, fmt, 8)
    s_fp, c = perturbed(62, s_fp, c)
    fq = oracle.fq_weight(W, fmt, 8, s_fp, c, alpha)
    packed = oracle.pack_codes(fq.codes)
    assert packed.shape == (W.shape[0], W.shape[1] // 2)
    np.testing.assert_array_equal(packed & 15, fq.codes[:, 0::2])
    np.testing.assert_array_equal(packed >> 4, fq.codes[:, 1::2])
    np.testing.assert_array_equal(oracle.unpack_codes(packed), fq.codes)
    dec = oracle.decode_packed(fmt, packed, fq.scale_bytes, alpha)
    np.testing.assert_array_equal(dec.view(np.uint32), fq.w_hat.view(np.uint32))


@pytest.mark.parametrize("fmt", [MX, NV])
def test_dynamic_activation_is_absmax_weight_path(oracle, fmt):
    rng = np.random.default_rng(71)
    X = rng.standard_normal((40, 256)).astype(np.float32)
    X[:, 7] *= 30
    X[5, 32:64] = 0.0
    xh, codes, sbytes, alpha = oracle.fq_act(X, fmt)
    s_fp, c, alpha_w = oracle.init_scales(X, fmt, 32 if fmt == MX else 16)
    ref = oracle.fq_weight(X, fmt, 32 if fmt == MX else 16, s_fp, c, alpha_w)
    assert alpha == alpha_w
    np.testing.assert_array_equal(codes, ref.codes)
    np.testing.assert_array_equal(sbytes, ref.scale_bytes)
    np.testing.assert_array_equal(xh.view(np.uint32), ref.w_hat.view(np.uint32))


@pytest.mark.parametrize("fmt", [MX, NV])
def test_all_zero_tensor(oracle, fmt):
    Z = np.zeros((2, 64), np.float32)
    Z[1, 3] = -0.0
    s_fp, c, alpha = oracle.init_scales(Z, fmt, 8)
    assert alpha == 1.0
    fq = oracle.fq_weight(Z, fmt, 8, s_fp, c, alpha)
    assert (fq.codes & 7).max() == 0 and fq.codes[1, 3] == 8 and (fq.w_hat == 0).all()
    assert fq.m.max() == 0 or fmt == MX
    xh, codes, sbytes, a = oracle.fq_act(Z, fmt)
    assert a == 1.0 and (xh == 0).all() and codes[1, 3] == 8
