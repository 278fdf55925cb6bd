"""GPU parity of the benchmark's packed-operand step on every linear of the hidden-8192 MXFP4 block
(131,072 tokens), at the initial parameter state the benchmark times (absmax S_fp, c = 1).

k_proj, gate_proj and down_proj are covered in full detail (bf16 and packed paths, initial and
perturbed states) by the full-size layer test; this one runs the other four linears (q_proj,
v_proj, o_proj, up_proj) exactly as one benchmark step does: activation fake quantisation to codes
+ block-major E8M0 bytes (bit-exact against the oracle on every element), the weights' export
(bit-exact), the FP4-MFMA forward with the MSE epilogue and the backward from the packed
activations, whose loss and straight-through gradients are compared with the oracle on sampled
output rows (first, last, 30 seeded rows and rows holding injected weight outliers) within 2e-2.
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, assert_close, host_f32, require_gpu, to_k_slabs

pytestmark = pytest.mark.gpu

TOL = 2e-2
WORKLOAD = "block8192_mxfp4"
LAYERS = ["q_proj", "v_proj", "o_proj", "up_proj"]


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


@pytest.fixture(scope="module")
def oracle_acts():
    """The oracle's activation fake quantisation of each block input, computed once per input."""
    return {}


def sample_rows(N, outliers, seed):
    rng = np.random.default_rng(seed)
    rows = {0, N - 1} | set(rng.choice(N, size=min(30, N), replace=False).tolist())
    rows |= set(outliers[:8])
    return np.array(sorted(rows), dtype=np.int64)


@pytest.mark.parametrize("layer", LAYERS)
def test_packed_step_init_state(F, O, oracle_acts, layer):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[WORKLOAD]
    lin = next(l for l in w.linears if l.name == layer)
    fmt, sb = w.fmt, w.sub_block
    announce(f"fullsize packed step {WORKLOAD} {layer} M={w.M} N={lin.N} K={lin.K}")
    X = synth.activation(w, lin.source, device="cuda")
    outl = []
    W = synth.weight(w, lin, device="cuda", outlier_rows=outl)
    Y = synth.reference_output(X, W)
    bm = F.SCALES_BLOCK_MAJOR
    _, xc, xs, _ = F.fakequant_fwd(X, fmt, sb, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                   scale_layout=bm)
    s_d, c_d, a_d = F.scales_init(W, fmt, sb)
    wc, ws = F.export_packed(W, fmt, sb, s_d, c_d, a_d, scale_layout=bm, code_layout=F.CODES_K_SLAB)
    dY, loss, col = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y, want_col_sq=True)
    gs, gc = F.recon_gemm_bwd_mxfp4(dY, xc, xs, W, sb, s_d, c_d)
    torch.cuda.synchronize()

    if lin.source not in oracle_acts:
        oracle_acts.clear()  # one input held at a time (the layers are ordered by input)
        xo, codes, sbytes, _ = O.fq_act(host_f32(X), fmt)
        oracle_acts[lin.source] = (xo, O.pack_codes(codes), np.ascontiguousarray(sbytes.T))
        del codes, sbytes
    xo, xcodes_o, xbytes_o = oracle_acts[lin.source]
    assert_bits_equal(xc.cpu().numpy(), xcodes_o, "activation codes")
    assert_bits_equal(xs.cpu().numpy(), xbytes_o, "activation scale bytes (block-major)")
    del X, xc, xs, dY

    Wh = host_f32(W)
    s_o, c_o, a_o = O.init_scales(Wh, fmt, sb)
    assert_bits_equal(s_d.cpu().numpy().view(np.uint32), s_o.view(np.uint32), "s_fp init")
    fq = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o)
    assert_bits_equal(wc.cpu().numpy(), to_k_slabs(O.pack_codes(fq.codes)), "weight codes (K-slabs)")
    assert_bits_equal(ws.cpu().numpy(), np.ascontiguousarray(fq.scale_bytes.T), "weight scale bytes (block-major)")

    rows = sample_rows(lin.N, outl, 7)
    Yr = host_f32(Y[:, torch.from_numpy(rows).cuda()])
    # MXFP4 operands are exact in bf16 (codes times powers of two), so no operand rounding applies
    res = O.recon_layer(xo, fq.w_hat, None, fq, fmt, sb, a_o, rows=rows, y_ref_cols=Yr)
    col = col.cpu().numpy()
    assert_close(col[rows], res.col_sq, TOL, "col_sq")
    assert abs(loss.item() - col.sum() / (w.M * lin.N)) <= 1e-9 * loss.item()
    assert_close(host_f32(gs)[rows], res.grad_s, TOL, "grad_s")
    assert_close(host_f32(gc)[rows], res.grad_c, TOL, "grad_c")
