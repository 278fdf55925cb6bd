"""GPU parity at the full benchmark sizes, in the launch configuration the benchmark times.

For each decoder-block workload (hidden 2560 MXFP4 and NVFP4 with 65,536 tokens, hidden 4096
MXFP4 with 262,144 tokens, hidden 8192 MXFP4 with 131,072 tokens) a few layers are run end to end
on the GPU with the seeded inputs at their real shapes:
  * bit-exact on every element: activation fake-quant X_hat, weight fake-quant W_hat (initial and
    perturbed state), and for the hidden-8192 block the exported packed codes and scale bytes;
  * loss and straight-through gradients on sampled output rows (first, last, 30 seeded rows and
    rows holding injected weight outliers), against the oracle computed row by row (loss and
    gradients of an output row depend only on that row), within 2e-2 relative, at the initial
    state (absmax S_fp, c = 1: the state the benchmark times) and at a perturbed one;
  * for the MXFP4 blocks also the packed-operand step the benchmark times there: activation codes
    and block-major E8M0 bytes without X_hat and the weights' export, bit-exact against the
    oracle's codes and scale bytes; the FP4-MFMA forward and the backward from the packed
    activations, loss and gradients on the sampled rows against the same oracle results.
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, assert_close, host_f32, require_gpu, to_k_slabs

pytestmark = pytest.mark.gpu

TOL = 2e-2
CASES = [
    ("block2560_mxfp4", "k_proj"), ("block2560_mxfp4", "down_proj"),
    ("block2560_nvfp4", "q_proj"), ("block2560_nvfp4", "down_proj"),
    ("block4096_mxfp4", "v_proj"), ("block4096_mxfp4", "o_proj"),
    ("block8192_mxfp4", "k_proj"), ("block8192_mxfp4", "gate_proj"),
    # the largest K of any workload (and the largest per-launch offsets)
    ("block4096_mxfp4", "down_proj"), ("block8192_mxfp4", "down_proj"),
]


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


def sample_rows(N, outliers, seed):
    rng = np.random.default_rng(seed)
    rows = {0, N - 1} | set(rng.choice(N, size=min(30, N), replace=False).tolist())
    rows |= set(outliers[:8])
    return np.array(sorted(rows), dtype=np.int64)


def device_values_equal(dev_bf16: torch.Tensor, oracle_fp32: np.ndarray, O, exact_in_bf16: bool, what: str):
    """Bit comparison of a bf16 device tensor with oracle fp32 values rounded to bf16."""
    got = dev_bf16.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    if exact_in_bf16:
        # MXFP4 values are codes times powers of two: the oracle's fp32 value is bf16-exact, so its
        # upper 16 bits are the expected bf16 pattern (a value that were not would mismatch)
        ref = (oracle_fp32.view(np.uint32) >> 16).astype(np.uint16)
        lost = (oracle_fp32.view(np.uint32) & 0xFFFF) != 0
        assert not lost.any(), f"{what}: oracle value not representable in bf16"
    else:
        ref = O.bf16_bits(O.bf16_round(oracle_fp32))
    assert_bits_equal(got, ref, what)


@pytest.mark.parametrize("name,layer", CASES)
def test_fullsize_layer(F, O, name, layer):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[name]
    lin = next(l for l in w.linears if l.name == layer)
    fmt, sb = w.fmt, w.sub_block
    mx = fmt == synth.MXFP4
    announce(f"fullsize {name} {layer} M={w.M} N={lin.N} K={lin.K}")
    X = synth.activation(w, lin.source, device="cuda")
    outl = []
    W = synth.weight(w, lin, device="cuda", outlier_rows=outl)
    Y = synth.reference_output(X, W)
    torch.cuda.synchronize()

    # activations: every element
    x_hat, _, _, a_x = F.fakequant_fwd(X, fmt, sb, want_alpha=True)
    Xh = host_f32(X)
    xo, _, _, ao = O.fq_act(Xh, fmt)
    device_values_equal(x_hat, xo, O, mx, f"X_hat {name} {layer}")
    if not mx:
        assert a_x.item() == ao
    del Xh

    # weights: initial state from both sides (bit-compared), then a perturbed state
    Wh = host_f32(W)
    s_d, c_d, a_d = F.scales_init(W, fmt, sb)
    s_o, c_o, a_o = O.init_scales(Wh, fmt, sb)
    assert_bits_equal(s_d.cpu().numpy().view(np.uint32), s_o.view(np.uint32), "s_fp init")
    assert np.all(c_d.cpu().numpy() == 1.0) and np.all(c_o == 1.0)
    rows = sample_rows(lin.N, outl, 5)
    Yr = host_f32(Y[:, torch.from_numpy(rows).cuda()])
    X_op = xo if mx else O.gemm_operand(xo, True)  # MXFP4 operands are bf16-exact already

    # the initial state: loss and gradients on the sampled rows, through the path the benchmark times
    # (packed operands under MXFP4, bf16 operands under NVFP4)
    announce(f"fullsize init state {name} {layer}")
    fq0 = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o)
    res0 = O.recon_layer(X_op, fq0.w_hat if mx else O.gemm_operand(fq0.w_hat, True), None, fq0, fmt, sb, a_o,
                         rows=rows, y_ref_cols=Yr)
    if mx:
        bm = F.SCALES_BLOCK_MAJOR
        _, xc0, xs0, _ = F.fakequant_fwd(X, fmt, sb, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                         scale_layout=bm)
        wc0, ws0 = F.export_packed(W, fmt, sb, s_d, c_d, a_d, scale_layout=bm, code_layout=F.CODES_K_SLAB)
        dY0, loss0, col0 = F.recon_gemm_fwd_mxfp4(xc0, xs0, wc0, ws0, Y, want_col_sq=True)
        gs0, gc0 = F.recon_gemm_bwd_mxfp4(dY0, xc0, xs0, W, sb, s_d, c_d)
        del xc0, xs0, wc0, ws0
    else:
        w_hat0, _, _, _ = F.fakequant_fwd(W, fmt, sb, s_d, c_d, a_d)
        dY0, loss0, col0 = F.recon_gemm_fwd(x_hat, w_hat0, Y, want_col_sq=True)
        gs0, gc0, _ = F.recon_gemm_bwd(dY0, x_hat, W, fmt, sb, s_d, c_d, a_d)
        del w_hat0
    torch.cuda.synchronize()
    col0 = col0.cpu().numpy()
    assert_close(col0[rows], res0.col_sq, TOL, "col_sq (init)")
    assert abs(loss0.item() - col0.sum() / (w.M * lin.N)) <= 1e-9 * loss0.item()
    assert_close(host_f32(gs0)[rows], res0.grad_s, TOL, "grad_s (init)")
    assert_close(host_f32(gc0)[rows], res0.grad_c, TOL, "grad_c (init)")
    del dY0, res0, fq0

    rng = np.random.default_rng(11)
    s_o = (s_o * np.exp2(rng.uniform(-0.5, 0.5, s_o.shape))).astype(np.float32)
    c_o = rng.uniform(0.75, 1.25, c_o.shape).astype(np.float32)
    s_d, c_d = torch.from_numpy(s_o).cuda(), torch.from_numpy(c_o).cuda()
    w_hat, _, _, _ = F.fakequant_fwd(W, fmt, sb, s_d, c_d, a_d)
    fq = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o)
    device_values_equal(w_hat, fq.w_hat, O, mx, f"W_hat {name} {layer}")
    if name == "block8192_mxfp4":
        packed, sbytes = F.export_packed(W, fmt, sb, s_d, c_d, a_d)
        assert_bits_equal(packed.cpu().numpy(), O.pack_codes(fq.codes), "export codes")
        assert_bits_equal(sbytes.cpu().numpy(), fq.scale_bytes, "export scale bytes")
        dec = O.decode_packed(fmt, packed.cpu().numpy(), sbytes.cpu().numpy(), a_o)
        assert_bits_equal(dec.view(np.uint32), fq.w_hat.view(np.uint32), "decoded export")

    # reconstruction step, compared on sampled output rows
    dY, loss, col_sq = F.recon_gemm_fwd(x_hat, w_hat, Y, want_col_sq=True)
    gs, gc, _ = F.recon_gemm_bwd(dY, x_hat, W, fmt, sb, s_d, c_d, a_d)
    torch.cuda.synchronize()
    del xo
    W_op = fq.w_hat if mx else O.gemm_operand(fq.w_hat, True)
    res = O.recon_layer(X_op, W_op, None, fq, fmt, sb, a_o, rows=rows, y_ref_cols=Yr)
    col = col_sq.cpu().numpy()  # float64
    assert_close(col[rows], res.col_sq, TOL, "col_sq")
    # the loss is the mean over all columns of the device's column sums
    assert abs(loss.item() - col.sum() / (w.M * lin.N)) <= 1e-9 * loss.item()
    assert_close(host_f32(gs)[rows], res.grad_s, TOL, "grad_s")
    assert_close(host_f32(gc)[rows], res.grad_c, TOL, "grad_c")

    if not mx:
        return
    # the packed-operand step (the benchmark's default for MXFP4): codes and block-major bytes only
    announce(f"fullsize packed-operand step {name} {layer}")
    bm = F.SCALES_BLOCK_MAJOR
    _, xc, xs, _ = F.fakequant_fwd(X, fmt, sb, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                   scale_layout=bm)
    wc, ws = F.export_packed(W, fmt, sb, s_d, c_d, a_d, scale_layout=bm, code_layout=F.CODES_K_SLAB)
    _, xcodes_o, xbytes_o, _ = O.fq_act(host_f32(X), fmt)
    assert_bits_equal(xc.cpu().numpy(), O.pack_codes(xcodes_o), "activation codes")
    assert_bits_equal(xs.cpu().numpy(), np.ascontiguousarray(xbytes_o.T), "activation scale bytes (block-major)")
    del xcodes_o, xbytes_o
    assert_bits_equal(wc.cpu().numpy(), to_k_slabs(O.pack_codes(fq.codes)), "weight codes (K-slabs)")
    assert_bits_equal(ws.cpu().numpy(), np.ascontiguousarray(fq.scale_bytes.T), "weight scale bytes (block-major)")
    dYm, lossm, colm = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y, want_col_sq=True)
    gsm, gcm = F.recon_gemm_bwd_mxfp4(dYm, xc, xs, W, sb, s_d, c_d)
    torch.cuda.synchronize()
    colm = colm.cpu().numpy()
    assert_close(colm[rows], res.col_sq, TOL, "col_sq (packed)")
    assert abs(lossm.item() - colm.sum() / (w.M * lin.N)) <= 1e-9 * lossm.item()
    assert abs(lossm.item() - loss.item()) <= 1e-4 * loss.item(), (lossm.item(), loss.item())
    assert_close(host_f32(gsm)[rows], res.grad_s, TOL, "grad_s (packed)")
    assert_close(host_f32(gcm)[rows], res.grad_c, TOL, "grad_c (packed)")
