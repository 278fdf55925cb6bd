"""Weight fake quantisation of bf16 weights at quotients that sit on the E2M1 decision points, bit-exact.

For bf16 weights the library forms u = W / S_q (Eq. 7, 8) from one correctly rounded reciprocal of
S_q per sub-block and two FMA corrections instead of a division per element, and falls back to true
division for a wave whose operands leave the range where that is exact. The codes can only come
out wrong where u lies on or next to a rounding midpoint of E2M1 (0.25, 0.75, 1.25, 1.75, 2.5, 3.5,
5) or next to the saturation point 6, so here every sub-block places one weight within +-3 units in
the last place of such a point: S_q is chosen as fl32(|w| / t) moved by -3 .. +3 ulps and the
coefficient c is set so that fl32(S_dq c) is that S_q (exactly, under MXFP4, where S_dq is a power of
two). Other rows force the fallback: infinite, NaN and huge (> 2^80) weights, and scales outside
[2^-40, 2^40]. Codes, scale bytes and W_hat (bf16 and fp32) are compared bit for bit with the
oracle, in both scale layouts, MXFP4 and NVFP4, at sub-blocks 8 and 2.
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, host_bits16, host_bits32, require_gpu

pytestmark = pytest.mark.gpu

POINTS = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0]


def bf16_round(x):
    from oracle import focus_oracle as O
    return O.bf16_round(np.asarray(x, np.float32))


def step_ulps(x: np.float32, k: int) -> np.float32:
    d = np.float32(np.inf) if k > 0 else np.float32(0.0)
    for _ in range(abs(k)):
        x = np.nextafter(x, d)
    return x


def build_case(fmt, sb, N, K, seed):
    """bf16 weights W, learnable scales s_fp and coefficients c (as fp32 arrays) and NVFP4's alpha."""
    rng = np.random.default_rng(seed)
    B = 32 if fmt == 0 else 16
    W = bf16_round(rng.standard_normal((N, K)).astype(np.float32) * 0.02)
    alpha = 1.0
    if fmt == 0:
        # S_dq = 2^e exactly: s_fp a power of two
        s = np.exp2(rng.integers(-9, -4, size=(N, K // B))).astype(np.float32)
        sdq = s.copy()
    else:
        alpha = float(np.float32(0.02 * 1.7 / 2688.0))
        s = rng.uniform(20.0, 440.0, size=(N, K // B)).astype(np.float32)  # Delta_fp (E4M3 domain)
        from oracle import focus_oracle as O
        # the dequantisation scale the oracle forms from s (E4M3 rounding, then alpha times it)
        fq0 = O.fq_weight(np.zeros((N, K), np.float32), fmt, sb, s, np.ones((N, K // sb), np.float32), alpha)
        sdq = fq0.s_dq
    c = rng.uniform(0.75, 1.25, size=(N, K // sb)).astype(np.float32)
    sub = np.arange(K // sb)
    for n in range(N):
        for k in sub:
            j = k * sb + (k * 5 + n) % sb       # the element placed on a decision point
            t = POINTS[(k + 3 * n) % len(POINTS)]
            delta = int((k + n) % 7) - 3
            w = W[n, j]
            if w == 0:
                w = W[n, j] = np.float32(0.015625)
            sq = step_ulps(np.float32(abs(w) / np.float32(t)), delta)
            d = sdq[n, k * sb // B]
            cv = np.float32(sq / d)
            if not (0.0 < cv < np.inf):
                continue
            c[n, k] = cv
    return W, s, c, alpha


def add_fallback_rows(W, s, c, fmt):
    """Rows whose waves must leave the fast path: non-finite and huge weights, out-of-range scales."""
    W[0, 3] = np.inf
    W[0, 70] = -np.inf
    W[1, 5] = np.nan
    W[2, 9] = np.float32(2.0 ** 90)
    W[3, 17] = np.float32(-(2.0 ** 100))
    c[4, :] = np.float32(2.0 ** -60)        # S_q far below 2^-40
    c[5, :] = np.float32(2.0 ** 60)         # S_q far above 2^40
    if fmt == 1:
        s[6, 0] = 0.0                        # Delta = 0: a zero-scale block
    else:
        s[6, 0] = np.float32(2.0 ** -120)    # S_dq = 2^-120


@pytest.mark.parametrize("fmt,sb", [(0, 8), (0, 2), (1, 8), (1, 2)])
def test_bf16_weights_on_decision_points(fmt, sb):
    F = require_gpu()
    from oracle import focus_oracle as O
    N, K = 96, 512
    W, s, c, alpha = build_case(fmt, sb, N, K, seed=31 + fmt * 10 + sb)
    add_fallback_rows(W, s, c, fmt)
    announce(f"divisor cases fmt={fmt} sb={sb} N={N} K={K}")
    Wg = torch.from_numpy(W).to(torch.bfloat16).cuda()
    W = Wg.float().cpu().numpy()  # exactly the values the library sees (NaN payloads included)
    s_d, c_d = torch.from_numpy(s).cuda(), torch.from_numpy(c).cuda()
    a_d = torch.tensor([alpha], dtype=torch.float32, device="cuda") if fmt == 1 else None
    fq = O.fq_weight(W, fmt, sb, s, c, alpha)
    ref_codes = O.pack_codes(fq.codes)
    for layout in (0, 1):
        w16, codes, sbytes, _ = F.fakequant_fwd(Wg, fmt, sb, s_d, c_d, a_d, want_codes=True, want_scale_bytes=True,
                                                scale_layout=layout)
        w32, _, _, _ = F.fakequant_fwd(Wg, fmt, sb, s_d, c_d, a_d, out_dtype=torch.float32)
        packed, ebytes = F.export_packed(Wg, fmt, sb, s_d, c_d, a_d, scale_layout=layout)
        torch.cuda.synchronize()
        ref_bytes = fq.scale_bytes if layout == 0 else np.ascontiguousarray(fq.scale_bytes.T)
        assert_bits_equal(codes.cpu().numpy(), ref_codes, f"codes (layout {layout})")
        assert_bits_equal(packed.cpu().numpy(), ref_codes, f"export codes (layout {layout})")
        assert_bits_equal(sbytes.cpu().numpy(), ref_bytes, f"scale bytes (layout {layout})")
        assert_bits_equal(ebytes.cpu().numpy(), ref_bytes, f"export scale bytes (layout {layout})")
        assert_bits_equal(host_bits32(w32), fq.w_hat.view(np.uint32), "W_hat fp32")
        assert_bits_equal(host_bits16(w16), O.bf16_bits(O.bf16_round(fq.w_hat)), "W_hat bf16")
    # the decision points were hit: many quotients round onto a midpoint or to within an ulp of it
    u = np.abs(fq.u[~np.isnan(fq.u)])
    mids = np.array(POINTS[:-1], np.float32)
    on_mid = np.isin(u, mids).sum()
    assert on_mid >= 20, on_mid
