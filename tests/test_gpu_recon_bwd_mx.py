"""GPU parity of the fused backward from packed MXFP4 activations (focus_recon_gemm_bwd_mxfp4).

Under MXFP4, X_hat is exactly an E2M1 code times its block's E8M0 power of two (Sec. 3.1, Eq. 1
and 3). The backward rebuilds the bf16 operand from the codes and scale bytes that the activation
fake quantisation returns, so checked here:
  * bit-identical gradients to the backward on the bf16 X_hat (same operand values, same tiles,
    splits and accumulation order), on ragged shapes (token counts off the 32-token step and the
    split length, K off the 256 tile, one 32-wide block, N off the tile), every sub-block size and
    the baseline without coefficients, at the initial and a perturbed parameter state;
  * against the oracle (its own fake quantisation, fp64 products): grad_s, grad_c within 2e-2, the
    bf16 GEMM tolerance;
  * the OCP floor rule for the scale bytes of the activations and the weights;
  * at full size (hidden-2560 gate_proj, 65,536 tokens): bit-identical to the bf16 path, and the
    oracle on sampled rows.
"""
import zlib

import numpy as np
import pytest
import torch

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


def perturb(seed, s_fp, c):
    rng = np.random.default_rng(seed)
    s = (s_fp * np.exp2(rng.uniform(-0.5, 0.5, s_fp.shape))).astype(np.float32)
    cc = rng.uniform(0.75, 1.25, c.shape).astype(np.float32)
    return s, cc


def same_bits(a, b, what):
    a, b = a.contiguous().view(torch.int32), b.contiguous().view(torch.int32)
    bad = (a != b).nonzero()
    assert bad.numel() == 0, f"{what}: {bad.shape[0]} words differ, first at {bad[:3].tolist()}"


def check_layer(F, O, X, W, Y, sb, state, tag, rows=None, coeff=True, rnd=0):
    Xh, Wh = host_f32(X), host_f32(W)
    s_d, c_d, a_d = F.scales_init(W, MX, sb, e8m0_rounding=rnd)
    s_o, c_o, a_o = O.init_scales(Wh, MX, sb, e8m0_floor=bool(rnd))
    if state == "perturbed":
        s_o, c_o = perturb(zlib.crc32(tag.encode()), s_o, c_o)
        s_d, c_d = torch.from_numpy(s_o).cuda(), torch.from_numpy(c_o).cuda()
    cf = c_d if coeff else None
    x_hat, xc, xs, _ = F.fakequant_fwd(X, MX, sb, want_codes=True, want_scale_bytes=True,
                                       scale_layout=F.SCALES_BLOCK_MAJOR, e8m0_rounding=rnd)
    w_hat, _, _, _ = F.fakequant_fwd(W, MX, sb, s_d, cf, a_d, e8m0_rounding=rnd)
    dY, _, _ = F.recon_gemm_fwd(x_hat, w_hat, Y)
    gs, gc = F.recon_gemm_bwd_mxfp4(dY, xc, xs, W, sb, s_d, cf, e8m0_rounding=rnd)
    gsb, gcb, _ = F.recon_gemm_bwd(dY, x_hat, W, MX, sb, s_d, cf, a_d, e8m0_rounding=rnd)
    torch.cuda.synchronize()
    same_bits(gs, gsb, f"grad_s vs bf16 path {tag}")
    same_bits(gc, gcb, f"grad_c vs bf16 path {tag}")
    # against the oracle, from the device dY (the backward's input): G = dY^T X_op in float64, then
    # the oracle's straight-through gradients
    xo, _, _, _ = O.fq_act(Xh, MX, e8m0_floor=bool(rnd))
    fq = O.fq_weight(Wh, MX, sb, s_o, c_o if coeff else None, a_o, e8m0_floor=bool(rnd))
    r = np.arange(W.shape[0]) if rows is None else np.asarray(rows)
    G = host_f32(dY).astype(np.float64)[:, r].T @ O.gemm_operand(xo, True).astype(np.float64)
    gs_o, gc_o = O.ste_gradients_from_G(G, fq, MX, sb, a_o, rows=r)
    assert_close(host_f32(gs)[r], gs_o, TOL, f"grad_s {tag}")
    assert_close(host_f32(gc)[r], gc_o, TOL, f"grad_c {tag}")


SHAPES = [(300, 264, 256), (64, 8, 32), (516, 520, 384), (1000, 1024, 2560), (4100, 96, 640)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("state", ["init", "perturbed"])
def test_mx_backward_shapes(F, O, M, N, K, state):
    announce(f"mx bwd M={M} N={N} K={K} {state}")
    g = torch.Generator().manual_seed(M * 31 + N + K)
    X = torch.randn(M, K, generator=g)
    X[:, :: max(1, K // 20)] *= 30
    W = torch.randn(N, K, generator=g) * 0.02
    Xd, Wd = X.to(torch.bfloat16).cuda(), W.to(torch.bfloat16).cuda()
    Y = (Xd.float() @ Wd.float().t()).to(torch.bfloat16)
    check_layer(F, O, Xd, Wd, Y, 8, state, f"{M}x{N}x{K}")


@pytest.mark.parametrize("sb,coeff,rnd", [(2, True, 0), (4, True, 0), (16, True, 0), (32, True, 0),
                                         (8, False, 0), (8, True, 1)])
def test_mx_backward_variants(F, O, sb, coeff, rnd):
    announce(f"mx bwd variant sb={sb} coeff={coeff} floor={rnd}")
    g = torch.Generator().manual_seed(17 + sb)
    X = torch.randn(520, 384, generator=g)
    X[:, ::19] *= 30
    W = torch.randn(136, 384, generator=g) * 0.02
    Xd, Wd = X.to(torch.bfloat16).cuda(), W.to(torch.bfloat16).cuda()
    Y = (Xd.float() @ Wd.float().t()).to(torch.bfloat16)
    check_layer(F, O, Xd, Wd, Y, sb, "perturbed", f"variant {sb} {coeff} {rnd}", coeff=coeff, rnd=rnd)


def test_mx_backward_fp32_weights(F):
    announce("mx bwd fp32 weights")
    g = torch.Generator().manual_seed(23)
    X = (torch.randn(260, 256, generator=g) * 3).to(torch.bfloat16).cuda()
    W = (torch.randn(40, 256, generator=g) * 0.02).cuda()
    s, c, a = F.scales_init(W, MX, 8)
    x_hat, xc, xs, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True,
                                       scale_layout=F.SCALES_BLOCK_MAJOR)
    dY = (torch.randn(260, 40, generator=g) * 1e-3).to(torch.bfloat16).cuda()
    gs, gc = F.recon_gemm_bwd_mxfp4(dY, xc, xs, W, 8, s, c)
    gsb, gcb, _ = F.recon_gemm_bwd(dY, x_hat, W, MX, 8, s, c, a)
    same_bits(gs, gsb, "grad_s fp32 W")
    same_bits(gc, gcb, "grad_c fp32 W")


def test_mx_backward_fullsize_gate(F, O):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    lin = next(l for l in w.linears if l.name == "gate_proj")
    announce(f"mx bwd fullsize gate M={w.M} N={lin.N} K={lin.K}")
    X = synth.activation(w, lin.source, device="cuda")
    outl = []
    W = synth.weight(w, lin, device="cuda", outlier_rows=outl)
    Y = synth.reference_output(X, W)
    rng = np.random.default_rng(11)
    rows = np.array(sorted({0, lin.N - 1} | set(rng.choice(lin.N, 16, replace=False).tolist()) | set(outl[:4])))
    check_layer(F, O, X, W, Y, w.sub_block, "perturbed", "fullsize gate", rows=rows)


def test_codes_only_activation_quant(F):
    """The packed form without X_hat gives the same codes and scale bytes as with it."""
    announce("codes-only activation fake-quant")
    g = torch.Generator().manual_seed(29)
    X = (torch.randn(300, 640, generator=g) * 2).to(torch.bfloat16).cuda()
    for rnd in (0, 1):
        x_hat, c0, s0, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True,
                                           scale_layout=F.SCALES_BLOCK_MAJOR, e8m0_rounding=rnd)
        none, c1, s1, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                          scale_layout=F.SCALES_BLOCK_MAJOR, e8m0_rounding=rnd)
        assert none is None and x_hat is not None
        assert torch.equal(c0, c1) and torch.equal(s0, s1), f"rounding {rnd}"


def test_packed_step_is_deterministic(F):
    """The packed-operand step (fixed-order reductions, no atomics) repeats bit for bit."""
    from paper_2608_01847_amd import synth
    w = synth.scaled(synth.WORKLOADS["block2560_mxfp4"], M=3000, hidden_div=4)
    lin = w.linears[4]  # gate_proj 2432 x 640
    announce(f"packed determinism {lin.name} M={w.M} N={lin.N} K={lin.K}")
    X = synth.activation(w, lin.source, device="cuda")
    W = synth.weight(w, lin, device="cuda")
    Y = synth.reference_output(X, W)
    bm = F.SCALES_BLOCK_MAJOR
    outs = []
    for _ in range(2):
        _, xc, xs, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                       scale_layout=bm)
        s, c, a = F.scales_init(W, MX, 8)
        wc, ws = F.export_packed(W, MX, 8, s, c, a, scale_layout=bm, code_layout=F.CODES_K_SLAB)
        dY, loss, col = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y, want_col_sq=True)
        gs, gc = F.recon_gemm_bwd_mxfp4(dY, xc, xs, W, 8, s, c)
        outs.append([t.cpu().clone() for t in (dY, loss, col, gs, gc)])
    for a_, b_ in zip(*outs):
        assert torch.equal(a_.view(torch.uint8), b_.view(torch.uint8))


@pytest.mark.parametrize("M", [0, 4, 36])
def test_backward_short_token_ranges(F, O, M):
    """No tokens gives zero gradients; a few tokens (less than one 32-token step, or one step and a
    ragged tail) give the oracle's, from both backward entry points."""
    announce(f"short token range M={M}")
    g = torch.Generator().manual_seed(41 + M)
    K, N = 256, 72
    X = (torch.randn(max(M, 1), K, generator=g) * 2)[:M].to(torch.bfloat16).cuda()
    W = (torch.randn(N, K, generator=g) * 0.02).to(torch.bfloat16).cuda()
    dY = (torch.randn(max(M, 1), N, generator=g) * 1e-3)[:M].to(torch.bfloat16).cuda()
    s, c, a = F.scales_init(W, MX, 8)
    x_hat, xc, xs, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True,
                                       scale_layout=F.SCALES_BLOCK_MAJOR)
    gs, gc = F.recon_gemm_bwd_mxfp4(dY, xc, xs, W, 8, s, c)
    gsb, gcb, _ = F.recon_gemm_bwd(dY, x_hat, W, MX, 8, s, c, a)
    torch.cuda.synchronize()
    same_bits(gs, gsb, f"grad_s M={M}")
    same_bits(gc, gcb, f"grad_c M={M}")
    if M == 0:
        assert not gs.any() and not gc.any()
        return
    Wh = host_f32(W)
    so, co, ao = O.init_scales(Wh, MX, 8)
    fq = O.fq_weight(Wh, MX, 8, so, co, ao)
    xo, _, _, _ = O.fq_act(host_f32(X), MX)
    G = host_f32(dY).astype(np.float64).T @ xo.astype(np.float64)
    gs_o, gc_o = O.ste_gradients_from_G(G, fq, MX, 8, ao)
    assert_close(host_f32(gs), gs_o, TOL, f"grad_s M={M}")
    assert_close(host_f32(gc), gc_o, TOL, f"grad_c M={M}")
