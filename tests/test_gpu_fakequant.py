"""GPU parity of the fake-quantisation kernels against the CPU oracle (bit-exact).

Covered: absmax initialisation (s_fp, c, alpha bits), weight fake quantisation with learned scales
(W_hat bits, packed codes, scale bytes) at the initial and a perturbed state, dynamic activation
fake quantisation (X_hat, codes, bytes, alpha), export (packed codes + bytes, decoding back to
W_hat), the straight-through backward from a given G (1e-5 relative: fp32 sums vs float64), the
domain flag, and edge cases (all-zero blocks, subnormal / huge scales, exact ties, signed zeros,
one row, ragged row counts).
"""
import numpy as np
import pytest
import torch

from gpu_common import (announce, assert_bits_equal, assert_close, device_bits, host_bits32, host_f32,
                        oracle_bits, require_gpu)

pytestmark = pytest.mark.gpu

MX, NV = 0, 1
B = {MX: 32, NV: 16}


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


def make_weight(seed, N, K, fmt, edge=False):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    idx = rng.choice(N * K, size=max(1, N * K // 1000), replace=False)
    W.ravel()[idx] *= 10
    if edge and N >= 6:
        bs = B[fmt]
        W[0, :bs] = 0.0                                  # all-zero block
        W[0, bs:2 * bs] = -0.0                           # negative zeros
        W[1, :bs] = rng.standard_normal(bs) * 1e-39      # subnormal magnitudes
        W[2, :bs] = rng.standard_normal(bs) * 1e30       # huge magnitudes
        # exact E2M1 ties at unit scale: block max 6 -> S = 1
        ties = np.array([6, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5, -5, -6])
        W[3, :16] = ties
        W[3, 16:bs] = 0.5
        W[4, :] = 0.0                                    # an all-zero row
    return W


def to_dev(a: np.ndarray, dtype) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dtype).contiguous()


def perturb(seed, s_fp, c):
    rng = np.random.default_rng(seed)
    s = (s_fp * np.exp2(rng.uniform(-0.5, 0.5, s_fp.shape))).astype(np.float32)
    cc = rng.uniform(0.75, 1.25, c.shape).astype(np.float32)
    return s, cc


WEIGHT_CASES = [(MX, 8), (MX, 32), (MX, 16), (MX, 4), (MX, 2), (NV, 8), (NV, 16), (NV, 4), (NV, 2)]


@pytest.mark.parametrize("fmt,sb", WEIGHT_CASES)
@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_weight_fakequant_bitexact(F, O, fmt, sb, dt):
    for (N, K, edge) in [(37, 3 * B[fmt], False), (8, 4 * B[fmt], True), (1, B[fmt], False), (300, 2560, False)]:
        announce(f"weight fq fmt={fmt} sb={sb} dt={dt} N={N} K={K} edge={edge}")
        Wn = make_weight(N * 7 + K + sb, N, K, fmt, edge)
        Wg = to_dev(Wn, dt)
        Wh = host_f32(Wg)  # the exact values the device holds
        s_g, c_g, a_g = F.scales_init(Wg, fmt, sb)
        s_o, c_o, a_o = O.init_scales(Wh, fmt, sb)
        torch.cuda.synchronize()
        assert_bits_equal(host_bits32(s_g), s_o.view(np.uint32), "s_fp init")
        assert_bits_equal(host_bits32(c_g), c_o.view(np.uint32), "c init")
        assert_bits_equal(host_bits32(a_g), np.array([a_o], np.float32).view(np.uint32), "alpha init")
        for state in ("init", "perturbed"):
            if state == "perturbed":
                s_o, c_o = perturb(N + K, s_o, c_o)
            s_d, c_d = to_dev(s_o, torch.float32), to_dev(c_o, torch.float32)
            w_hat, codes, sbytes, _ = F.fakequant_fwd(Wg, fmt, sb, s_d, c_d, a_g, out_dtype=dt,
                                                      want_codes=True, want_scale_bytes=True)
            fq = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o)
            tag = f"{state} N={N} K={K}"
            assert_bits_equal(device_bits(w_hat), oracle_bits(fq.w_hat, dt), f"W_hat {tag}")
            assert_bits_equal(codes.cpu().numpy(), O.pack_codes(fq.codes), f"codes {tag}")
            assert_bits_equal(sbytes.cpu().numpy(), fq.scale_bytes, f"scale bytes {tag}")
            packed, eb = F.export_packed(Wg, fmt, sb, s_d, c_d, a_g)
            assert_bits_equal(packed.cpu().numpy(), O.pack_codes(fq.codes), f"export codes {tag}")
            assert_bits_equal(eb.cpu().numpy(), fq.scale_bytes, f"export bytes {tag}")
            dec = O.decode_packed(fmt, packed.cpu().numpy(), eb.cpu().numpy(), a_o)
            assert_bits_equal(dec.view(np.uint32), fq.w_hat.view(np.uint32), f"decoded export {tag}")


def make_activation(seed, M, K, kind="normal"):
    rng = np.random.default_rng(seed)
    if kind == "student_t3":
        z = rng.standard_normal((M, K))
        X = z / np.sqrt((rng.standard_normal((M, K, 3)) ** 2).sum(-1) / 3)
    else:
        X = rng.standard_normal((M, K))
        ch = rng.choice(K, size=max(1, K // 100), replace=False)
        X[:, ch] *= 30
    X = X.astype(np.float32)
    if M > 4:
        X[1] = 0.0
        X[2, :16] = -0.0
        X[3, :32] *= 1e-40
    return X


@pytest.mark.parametrize("fmt", [MX, NV])
@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_activation_fakequant_bitexact(F, O, fmt, dt):
    for (M, K) in [(1, 64), (5, 96 if fmt == MX else 80), (1000, 2560), (333, 4096)]:
        announce(f"act fq fmt={fmt} dt={dt} M={M} K={K}")
        Xn = make_activation(M + K, M, K, "student_t3" if fmt == NV else "normal")
        Xg = to_dev(Xn, dt)
        Xh = host_f32(Xg)
        x_hat, codes, sbytes, a_x = F.fakequant_fwd(Xg, fmt, 8, want_codes=True, want_scale_bytes=True,
                                                    want_alpha=True)
        xo, co, so, ao = O.fq_act(Xh, fmt)
        tag = f"M={M} K={K}"
        assert_bits_equal(device_bits(x_hat), oracle_bits(xo, dt), f"X_hat {tag}")
        assert_bits_equal(codes.cpu().numpy(), O.pack_codes(co), f"codes {tag}")
        assert_bits_equal(sbytes.cpu().numpy(), so, f"scale bytes {tag}")
        if fmt == NV:
            assert_bits_equal(host_bits32(a_x), np.array([ao], np.float32).view(np.uint32), "alpha_x")


def test_activation_all_zero_tensor(F, O):
    for fmt in (MX, NV):
        Xg = torch.zeros(3, 64, device="cuda", dtype=torch.bfloat16)
        x_hat, codes, _, a_x = F.fakequant_fwd(Xg, fmt, 8, want_codes=True, want_alpha=True)
        assert not x_hat.float().abs().max().item()
        if fmt == NV:
            assert a_x.item() == 1.0


@pytest.mark.parametrize("fmt,sb", [(MX, 8), (MX, 32), (MX, 4), (NV, 8), (NV, 16), (NV, 2)])
@pytest.mark.parametrize("clip", [1, 0])
def test_fakequant_bwd_matches_oracle(F, O, fmt, sb, clip):
    N, K = 64, 8 * B[fmt]
    announce(f"fq bwd fmt={fmt} sb={sb} clip={clip}")
    Wn = make_weight(99 + sb, N, K, fmt, edge=True)
    Wg = to_dev(Wn, torch.bfloat16)
    Wh = host_f32(Wg)
    s_o, c_o, a_o = O.init_scales(Wh, fmt, sb)
    s_o, c_o = perturb(5, s_o, c_o)
    G = np.random.default_rng(7).standard_normal((N, K)).astype(np.float32)
    a_d = torch.tensor([a_o], device="cuda", dtype=torch.float32)
    gs, gc = F.fakequant_bwd(to_dev(G, torch.float32), Wg, fmt, sb, to_dev(s_o, torch.float32),
                             to_dev(c_o, torch.float32), a_d, ste_clip=clip)
    fq = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o, ste_clip=bool(clip))
    rs, rc = O.ste_gradients_from_G(G.astype(np.float64), fq, fmt, sb, a_o)
    assert_close(host_f32(gs), rs, 1e-5, "grad_s")
    assert_close(host_f32(gc), rc, 1e-5, "grad_c")


def test_domain_flag(F, O):
    announce("domain flag")
    fmt, sb, N, K = MX, 8, 4, 64
    Wg = to_dev(make_weight(1, N, K, fmt), torch.bfloat16)
    s, c, a = F.scales_init(Wg, fmt, sb)
    ws = F.workspace(F.workspace_size(F.CALL_FAKEQUANT_FWD, F.qconfig(fmt, sb)))
    F.fakequant_fwd(Wg, fmt, sb, s, c, a, ws=ws)
    assert F.check_flags(ws) == F.OK
    c_bad = c.clone()
    c_bad[1, 3] = 0.0
    c_bad[2, 0] = -1.0
    F.fakequant_fwd(Wg, fmt, sb, s, c_bad, a, ws=ws)
    assert F.check_flags(ws) == F.ERR_DOMAIN
    assert F.check_flags(ws) == F.OK  # the check clears the flag
    s_bad = s.clone()
    s_bad[0, 0] = float("nan")
    F.fakequant_fwd(Wg, fmt, sb, s_bad, c, a, ws=ws)
    assert F.check_flags(ws) == F.ERR_DOMAIN
