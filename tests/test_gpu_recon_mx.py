"""GPU parity of the forward reconstruction GEMM from packed MXFP4 operands.

Under MXFP4 the fake-quantised operands are exactly E2M1 codes times E8M0 block scales (Sec. 3.1,
Eq. 1 and 3), so the forward can run on the block-scaled FP4 MFMA from the codes and scale bytes
that the library's fake quantisation returns. Checked here:
  * against the oracle (its own fake quantisation, fp64 products): loss, column sums of D^2 and
    dY within 2e-2 (the bf16 GEMM tolerance; dY is bf16), on ragged shapes (token counts and
    output features off the 256 tile, one and several 128-wide K steps) and a hidden-2560 decoder
    block narrowed 4x, at the initial and a perturbed parameter state;
  * against the bf16 forward on the same operands: the two compute the same sums and differ only
    in the fp32 accumulation order (1e-4 on the loss and column sums);
  * the plain product mode (no Y_ref) returns Y_hat;
  * the block-major scale bytes the forward reads are the transpose of the row-major ones, for
    activations (MXFP4 and NVFP4), weights and the export;
  * at full size (hidden-2560 gate_proj, 65,536 tokens) on sampled output rows.
"""
import zlib

import numpy as np
import pytest
import torch

from gpu_common import to_k_slabs, announce, assert_close, host_f32, require_gpu

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


def perturb(seed, s_fp, c):
    rng = np.random.default_rng(seed)
    s = (s_fp * np.exp2(rng.uniform(-0.5, 0.5, s_fp.shape))).astype(np.float32)
    cc = rng.uniform(0.75, 1.25, c.shape).astype(np.float32)
    return s, cc


def device_operands(F, X, W, sb, s_d, c_d, a_d):
    """bf16 X_hat, W_hat and the packed operands of both (X codes row-major, W codes in K-slabs, scale bytes
    block-major), from the library."""
    bm, slab = F.SCALES_BLOCK_MAJOR, F.CODES_K_SLAB
    x_hat, xc, xs, _ = F.fakequant_fwd(X, MX, sb, want_codes=True, want_scale_bytes=True, scale_layout=bm)
    w_hat, wc, ws, _ = F.fakequant_fwd(W, MX, sb, s_d, c_d, a_d, want_codes=True, want_scale_bytes=True,
                                       scale_layout=bm, code_layout=slab)
    return x_hat, w_hat, xc, xs, wc, ws


def check_layer(F, O, X, W, Y, sb, state, tag, rows=None):
    Xh, Wh = host_f32(X), host_f32(W)
    s_d, c_d, a_d = F.scales_init(W, MX, sb)
    s_o, c_o, a_o = O.init_scales(Wh, MX, sb)
    if state == "perturbed":
        s_o, c_o = perturb(zlib.crc32(tag.encode()), s_o, c_o)
        s_d, c_d = torch.from_numpy(s_o).cuda(), torch.from_numpy(c_o).cuda()
    x_hat, w_hat, xc, xs, wc, ws = device_operands(F, X, W, sb, s_d, c_d, a_d)
    dY, loss, col_sq = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y, want_col_sq=True)
    dYb, lossb, col_sqb = F.recon_gemm_fwd(x_hat, w_hat, Y, want_col_sq=True)
    torch.cuda.synchronize()
    # the same sums as the bf16 path up to the accumulation order
    assert abs(loss.item() - lossb.item()) <= 1e-4 * lossb.item(), (tag, loss.item(), lossb.item())
    assert_close(col_sq.cpu().numpy(), col_sqb.cpu().numpy(), 1e-4, f"col_sq vs bf16 {tag}")
    # against the oracle
    xo, _, _, _ = O.fq_act(Xh, MX)
    fq = O.fq_weight(Wh, MX, sb, s_o, c_o, a_o)
    if rows is None:
        res = O.recon_layer(xo, fq.w_hat, host_f32(Y).astype(np.float64), fq, MX, sb, a_o, keep_dy=True)
        assert abs(loss.item() - res.loss_part) <= TOL * res.loss_part, (tag, loss.item(), res.loss_part)
        assert_close(host_f32(dY), res.d_y, TOL, f"dY {tag}")
    else:
        Yr = host_f32(Y[:, torch.from_numpy(rows).cuda()])
        res = O.recon_layer(xo, fq.w_hat, None, fq, MX, sb, a_o, rows=rows, y_ref_cols=Yr)
        assert abs(loss.item() - col_sq.cpu().numpy().sum() / (X.shape[0] * W.shape[0])) <= 1e-9 * loss.item()
    assert_close(col_sq.cpu().numpy()[res.rows], res.col_sq, TOL, f"col_sq {tag}")


SHAPES = [(300, 264, 256), (64, 8, 128), (516, 520, 384), (1000, 1024, 2560)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("state", ["init", "perturbed"])
def test_mx_forward_shapes(F, O, M, N, K, state):
    announce(f"mx fwd M={M} N={N} K={K} {state}")
    g = torch.Generator().manual_seed(M * 31 + N + K)
    X = torch.randn(M, K, generator=g)
    X[:, :: max(1, K // 20)] *= 30
    W = torch.randn(N, K, generator=g) * 0.02
    Xd, Wd = X.to(torch.bfloat16).cuda(), W.to(torch.bfloat16).cuda()
    Y = (Xd.float() @ Wd.float().t()).to(torch.bfloat16)
    check_layer(F, O, Xd, Wd, Y, 8, state, f"{M}x{N}x{K}")


def test_mx_forward_small_block(F, O):
    from paper_2608_01847_amd import synth
    w = synth.scaled(synth.WORKLOADS["block2560_mxfp4"], M=1000, hidden_div=4)  # every K a multiple of 128
    acts = {src: synth.activation(w, src, device="cuda") for src in w.inputs}
    for lin in w.linears:
        announce(f"mx fwd small block {lin.name}")
        W = synth.weight(w, lin, device="cuda")
        Y = synth.reference_output(acts[lin.source], W)
        check_layer(F, O, acts[lin.source], W, Y, w.sub_block, "perturbed", lin.name)


def test_mx_forward_plain_product(F):
    announce("mx fwd plain product")
    g = torch.Generator().manual_seed(5)
    X = (torch.randn(384, 512, generator=g)).to(torch.bfloat16).cuda()
    W = (torch.randn(136, 512, generator=g) * 0.02).to(torch.bfloat16).cuda()
    s, c, a = F.scales_init(W, MX, 8)
    x_hat, w_hat, xc, xs, wc, ws = device_operands(F, X, W, 8, s, c, a)
    y_mx, _, _ = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, None)
    y_bf, _, _ = F.recon_gemm_fwd(x_hat, w_hat, None)
    ref = x_hat.double() @ w_hat.double().t()
    assert_close(host_f32(y_mx), ref.cpu().numpy(), 1e-2, "Y_hat (mx) vs fp64")
    assert_close(host_f32(y_mx), host_f32(y_bf), 1e-2, "Y_hat (mx) vs bf16 path")


def test_mx_forward_fullsize_gate(F, O):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    lin = next(l for l in w.linears if l.name == "gate_proj")
    announce(f"mx fwd fullsize gate M={w.M} N={lin.N} K={lin.K}")
    X = synth.activation(w, lin.source, device="cuda")
    outl = []
    W = synth.weight(w, lin, device="cuda", outlier_rows=outl)
    Y = synth.reference_output(X, W)
    rng = np.random.default_rng(7)
    rows = np.array(sorted({0, lin.N - 1} | set(rng.choice(lin.N, 24, replace=False).tolist()) | set(outl[:6])))
    check_layer(F, O, X, W, Y, w.sub_block, "perturbed", "fullsize gate", rows=rows)


def test_gemm_layouts_are_permutations(F):
    """Block-major scale bytes are the transpose of the row-major ones, K-slab codes the row-major codes
    rearranged, for every call that writes them."""
    announce("block-major scale bytes and K-slab codes")
    g = torch.Generator().manual_seed(9)
    X = torch.randn(300, 640, generator=g).to(torch.bfloat16).cuda()
    W = (torch.randn(72, 640, generator=g) * 0.02).to(torch.bfloat16).cuda()
    bm, slab = F.SCALES_BLOCK_MAJOR, F.CODES_K_SLAB
    for fmt in (0, 1):
        _, c0, s0, _ = F.fakequant_fwd(X, fmt, 8, want_codes=True, want_scale_bytes=True)
        _, c1, s1, _ = F.fakequant_fwd(X, fmt, 8, want_codes=True, want_scale_bytes=True, scale_layout=bm)
        assert torch.equal(c0, c1) and torch.equal(s0.t().contiguous(), s1), f"activation fmt {fmt}"
        _, c2, _, _ = F.fakequant_fwd(X, fmt, 8, want_codes=True, code_layout=slab)
        assert torch.equal(to_k_slabs(c0), c2), f"activation K-slabs fmt {fmt}"
        s, c, a = F.scales_init(W, fmt, 8)
        _, w0, t0, _ = F.fakequant_fwd(W, fmt, 8, s, c, a, want_codes=True, want_scale_bytes=True)
        _, w1, t1, _ = F.fakequant_fwd(W, fmt, 8, s, c, a, want_codes=True, want_scale_bytes=True, scale_layout=bm)
        assert torch.equal(w0, w1) and torch.equal(t0.t().contiguous(), t1), f"weight fmt {fmt}"
        _, w2, _, _ = F.fakequant_fwd(W, fmt, 8, s, c, a, want_codes=True, code_layout=slab)
        assert torch.equal(to_k_slabs(w0), w2), f"weight K-slabs fmt {fmt}"
        p0, e0 = F.export_packed(W, fmt, 8, s, c, a)
        p1, e1 = F.export_packed(W, fmt, 8, s, c, a, scale_layout=bm)
        assert torch.equal(p0, p1) and torch.equal(e0.t().contiguous(), e1), f"export fmt {fmt}"
        p2, _ = F.export_packed(W, fmt, 8, s, c, a, code_layout=slab)
        assert torch.equal(to_k_slabs(p0), p2), f"export K-slabs fmt {fmt}"
        g2 = [dict(W=W, s_fp=s, c=c, alpha=a, codes=torch.empty_like(p2))]
        F.fakequant_weights(g2, fmt, 8, code_layout=slab)
        assert torch.equal(g2[0]["codes"], p2), f"grouped K-slabs fmt {fmt}"
        # fp32 inputs take the one-chunk-per-thread kernels
        _, c3, _, _ = F.fakequant_fwd(X.float(), fmt, 8, want_codes=True, want_x_hat=False, code_layout=slab)
        assert torch.equal(c3, c2), f"fp32 activation K-slabs fmt {fmt}"
        _, w3, _, _ = F.fakequant_fwd(W.float(), fmt, 8, s, c, a, want_codes=True, want_x_hat=False,
                                      code_layout=slab)
        _, w4, _, _ = F.fakequant_fwd(W.float(), fmt, 8, s, c, a, want_codes=True, want_x_hat=False)
        assert torch.equal(to_k_slabs(w4), w3), f"fp32 weight K-slabs fmt {fmt}"
