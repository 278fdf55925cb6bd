"""GPU parity of the reconstruction GEMMs' main loops at every step count their schedules tell apart.

Both GEMMs read each half-step's operand fragments one step ahead, into three register sets that
rotate with a period of three steps. Their loops therefore run whole groups of three steps plus a
remainder of zero, one or two, and the forward renames its sets once before the steps that bring in
the Y_ref tile. These cases check each such count against the oracle:
  * forward, FP4 operands and the bf16-operand forward through the same check: K in {512, 640, 768,
    1152} gives the FP4 kernel 1, 2, 3 and 6 operand steps before its Y_ref steps, and the bf16 kernel
    12, 16, 20 and 32;
  * forward, bf16 operands alone: K in {96, 128, 160, 192, 224} runs 3 to 7 steps, which is fewer
    than, as many as, and just more than its Y_ref steps;
  * backward, packed MXFP4 and bf16 operands, compared bit for bit with each other and against the
    oracle: a 4096 x 4096 layer fills the chip with one token split, so M in {32, 64, 96, 128, 160, 224}
    tokens runs 1 to 7 steps of 32 tokens in every workgroup.
"""
import zlib

import numpy as np
import pytest
import torch

import test_gpu_recon_bwd_mx as bwd_mx
import test_gpu_recon_mx as fwd_mx
from gpu_common import announce, assert_close, host_f32, require_gpu

pytestmark = pytest.mark.gpu

MX = 0
TOL = 2e-2


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


def operands(M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    X = torch.randn(M, K, generator=g)
    X[:, :: max(1, K // 20)] *= 30
    W = torch.randn(N, K, generator=g) * 0.02
    Xd, Wd = X.to(torch.bfloat16).cuda(), W.to(torch.bfloat16).cuda()
    Y = (Xd.float() @ Wd.float().t()).to(torch.bfloat16)
    return Xd, Wd, Y


@pytest.mark.parametrize("K", [512, 640, 768, 1152])
def test_forward_operand_steps(F, O, K):
    M, N = 300, 264
    announce(f"forward steps M={M} N={N} K={K}")
    Xd, Wd, Y = operands(M, N, K, 7 * K + 1)
    fwd_mx.check_layer(F, O, Xd, Wd, Y, 8, "perturbed", f"steps {M}x{N}x{K}")


@pytest.mark.parametrize("K", [96, 128, 160, 192, 224])
def test_bf16_forward_short_k(F, O, K):
    M, N, sb = 260, 264, 8
    announce(f"bf16 forward steps M={M} N={N} K={K}")
    Xd, Wd, Y = operands(M, N, K, 11 * K + 3)
    Xh, Wh = host_f32(Xd), host_f32(Wd)
    s_o, c_o, a_o = O.init_scales(Wh, MX, sb)
    s_o, c_o = fwd_mx.perturb(zlib.crc32(f"short {K}".encode()), s_o, c_o)
    s_d, c_d = torch.from_numpy(s_o).cuda(), torch.from_numpy(c_o).cuda()
    _, _, a_d = F.scales_init(Wd, MX, sb)
    x_hat = F.fakequant_fwd(Xd, MX, sb)[0]
    w_hat = F.fakequant_fwd(Wd, MX, sb, s_d, c_d, a_d)[0]
    dY, loss, col_sq = F.recon_gemm_fwd(x_hat, w_hat, Y, want_col_sq=True)
    torch.cuda.synchronize()
    xo, _, _, _ = O.fq_act(Xh, MX)
    fq = O.fq_weight(Wh, MX, sb, s_o, c_o, a_o)
    res = O.recon_layer(xo, fq.w_hat, host_f32(Y).astype(np.float64), fq, MX, sb, a_o, keep_dy=True)
    assert abs(loss.item() - res.loss_part) <= TOL * res.loss_part, (K, loss.item(), res.loss_part)
    assert_close(host_f32(dY), res.d_y, TOL, f"dY K={K}")
    assert_close(col_sq.cpu().numpy(), res.col_sq, TOL, f"col_sq K={K}")


@pytest.mark.parametrize("M", [32, 64, 96, 128, 160, 224])
def test_backward_token_steps(F, O, M):
    N = K = 4096
    announce(f"backward steps M={M} N={N} K={K}")
    Xd, Wd, Y = operands(M, N, K, 13 * M + 5)
    rows = np.sort(np.random.default_rng(M).choice(N, size=96, replace=False))
    bwd_mx.check_layer(F, O, Xd, Wd, Y, 8, "perturbed", f"steps M={M}", rows=rows)
