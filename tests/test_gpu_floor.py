"""GPU parity of the OCP floor mode of the E8M0 scales (MXFP4) against the CPU oracle.

  * absmax initialisation in floor mode (S_fp = amax / 4) bit for bit;
  * weight fake quantisation (W_hat, packed codes, scale bytes, export) at the initial and a
    perturbed state, sub-blocks 8 and 32, bf16 and fp32 weights, with zero, subnormal and huge
    blocks: bit-exact;
  * dynamic activation fake quantisation (exponent floor(log2 amax) - 2, saturation at 6) with
    zero rows and subnormal blocks: bit-exact;
  * the fused backward in floor mode on the bf16 MFMA path (2e-2) and the fp32 path (1e-5).
"""
import numpy as np
import pytest
import torch

from gpu_common import (announce, assert_bits_equal, assert_close, device_bits, host_bits32, host_f32,
                        oracle_bits, require_gpu)
from test_gpu_fakequant import make_activation, make_weight, perturb, to_dev

pytestmark = pytest.mark.gpu

MX = 0
FLOOR = 1


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


@pytest.mark.parametrize("sb", [8, 32])
@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_floor_weight_bitexact(F, O, sb, dt):
    for (N, K, edge) in [(37, 96, False), (8, 128, True), (300, 2560, False)]:
        announce(f"floor weight fq sb={sb} dt={dt} N={N} K={K}")
        Wg = to_dev(make_weight(N * 3 + K + sb, N, K, MX, edge), dt)
        Wh = host_f32(Wg)
        s_g, c_g, a_g = F.scales_init(Wg, MX, sb, e8m0_rounding=FLOOR)
        s_o, c_o, a_o = O.init_scales(Wh, MX, sb, e8m0_floor=True)
        torch.cuda.synchronize()
        assert_bits_equal(host_bits32(s_g), s_o.view(np.uint32), "s_fp init (floor)")
        for state in ("init", "perturbed"):
            if state == "perturbed":
                s_o, c_o = perturb(N + K + 1, s_o, c_o)
            s_d, c_d = to_dev(s_o, torch.float32), to_dev(c_o, torch.float32)
            w_hat, codes, sbytes, _ = F.fakequant_fwd(Wg, MX, sb, s_d, c_d, a_g, out_dtype=dt, want_codes=True,
                                                      want_scale_bytes=True, e8m0_rounding=FLOOR)
            fq = O.fq_weight(Wh, MX, sb, s_o, c_o, a_o, e8m0_floor=True)
            tag = f"{state} N={N} K={K}"
            assert_bits_equal(device_bits(w_hat), oracle_bits(fq.w_hat, dt), f"W_hat {tag}")
            assert_bits_equal(codes.cpu().numpy(), O.pack_codes(fq.codes), f"codes {tag}")
            assert_bits_equal(sbytes.cpu().numpy(), fq.scale_bytes, f"scale bytes {tag}")
            packed, eb = F.export_packed(Wg, MX, sb, s_d, c_d, a_g, e8m0_rounding=FLOOR)
            assert_bits_equal(packed.cpu().numpy(), O.pack_codes(fq.codes), f"export codes {tag}")
            assert_bits_equal(eb.cpu().numpy(), fq.scale_bytes, f"export bytes {tag}")


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_floor_activation_bitexact(F, O, dt):
    for (M, K) in [(1, 64), (5, 96), (1000, 2560)]:
        announce(f"floor act fq dt={dt} M={M} K={K}")
        Xg = to_dev(make_activation(M * 5 + K, M, K), dt)
        Xh = host_f32(Xg)
        x_hat, codes, sbytes, _ = F.fakequant_fwd(Xg, MX, 8, want_codes=True, want_scale_bytes=True,
                                                  e8m0_rounding=FLOOR)
        xo, co, so, _ = O.fq_act(Xh, MX, e8m0_floor=True)
        tag = f"M={M} K={K}"
        assert_bits_equal(device_bits(x_hat), oracle_bits(xo, dt), f"X_hat {tag}")
        assert_bits_equal(codes.cpu().numpy(), O.pack_codes(co), f"codes {tag}")
        assert_bits_equal(sbytes.cpu().numpy(), so, f"scale bytes {tag}")


@pytest.mark.parametrize("dt,tol", [(torch.bfloat16, 2e-2), (torch.float32, 1e-5)], ids=["bf16", "f32"])
def test_floor_fused_backward(F, O, dt, tol):
    M, N, K, sb = 300, 264, 256, 8
    announce(f"floor fused bwd dt={dt}")
    rng = np.random.default_rng(11)
    Xg = to_dev(make_activation(7, M, K), dt)
    Wg = to_dev(make_weight(8, N, K, MX), dt)
    Xh, Wh = host_f32(Xg), host_f32(Wg)
    Y = to_dev((Xh.astype(np.float64) @ Wh.astype(np.float64).T).astype(np.float32), dt)
    s_o, c_o, a_o = O.init_scales(Wh, MX, sb, e8m0_floor=True)
    s_o, c_o = perturb(12, s_o, c_o)
    s_d, c_d = to_dev(s_o, torch.float32), to_dev(c_o, torch.float32)
    x_hat = F.fakequant_fwd(Xg, MX, sb, e8m0_rounding=FLOOR)[0]
    w_hat = F.fakequant_fwd(Wg, MX, sb, s_d, c_d, None, e8m0_rounding=FLOOR)[0]
    dY, loss, _ = F.recon_gemm_fwd(x_hat, w_hat, Y)
    gs, gc, _ = F.recon_gemm_bwd(dY, x_hat, Wg, MX, sb, s_d, c_d, None, e8m0_rounding=FLOOR)
    torch.cuda.synchronize()
    xo = O.fq_act(Xh, MX, e8m0_floor=True)[0]
    fq = O.fq_weight(Wh, MX, sb, s_o, c_o, 1.0, e8m0_floor=True)
    bf = dt == torch.bfloat16
    X_op = O.bf16_round(xo) if bf else xo
    W_op = O.bf16_round(fq.w_hat) if bf else fq.w_hat
    res = O.recon_layer(X_op, W_op, host_f32(Y).astype(np.float64), fq, MX, sb, 1.0)
    assert abs(loss.item() - res.loss_part) <= tol * res.loss_part
    assert_close(host_f32(gs), res.grad_s, tol, "grad_s (floor)")
    assert_close(host_f32(gc), res.grad_c, tol, "grad_c (floor)")
