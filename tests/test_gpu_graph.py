"""A scale-learning step replayed from a HIP graph gives the eager step's results bit for bit.

Every entry point of the step is ordered on the caller's stream, synchronises nothing and allocates
nothing (outputs and workspaces come from the caller), so a caller can capture a whole step once
and replay it. Checked on the fp32 layer (VALU kernels), on a bf16 MXFP4 layer with bf16 operands
(MFMA kernels) and with packed operands (FP4-MFMA forward, backward from packed activations): the
step captured with torch.cuda.graph, then three replays, each after eager work of the program's own
and a synchronisation, each compared with the eager step on loss, dY and both gradients. The weight
pass goes through the grouped call (focus_fakequant_weights), as the benchmark's step does.
"""
import pytest
import torch

from gpu_common import announce, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def F():
    return require_gpu()


def layer_step(F, w, lin, packed):
    from paper_2608_01847_amd import synth
    fmt, sb, M = w.fmt, w.sub_block, w.M
    X = synth.activation(w, lin.source, device="cuda")
    W = synth.weight(w, lin, device="cuda")
    Y = synth.reference_output(X, W)
    s, c, a = F.scales_init(W, fmt, sb)
    N, K = W.shape
    q = F.qconfig(fmt, sb)
    ws_fq = F.workspace(F.workspace_size(F.CALL_FAKEQUANT_FWD, q, 0, max(M, N), K))
    ws_fwd = F.workspace(F.workspace_size(F.CALL_RECON_GEMM_FWD, q, M, N, K))
    ws_bwd = F.workspace(F.workspace_size(F.CALL_RECON_GEMM_BWD, q, M, N, K))
    out = {"dY": torch.empty(M, N, dtype=X.dtype, device="cuda"),
           "loss": torch.empty(1, dtype=torch.float64, device="cuda"),
           "gs": torch.empty_like(s), "gc": torch.empty_like(c)}
    bm = F.SCALES_BLOCK_MAJOR
    if packed:
        xc = torch.empty(M, K // 2, dtype=torch.uint8, device="cuda")
        xs = torch.empty(K // 32, M, dtype=torch.uint8, device="cuda")
        wc = torch.empty(*F.codes_shape(N, K, F.CODES_K_SLAB), dtype=torch.uint8, device="cuda")
        wsb = torch.empty(K // 32, N, dtype=torch.uint8, device="cuda")

        def step():
            F.fakequant_fwd(X, fmt, sb, ws=ws_fq, want_x_hat=False, codes_out=xc, scales_out=xs, scale_layout=bm)
            F.fakequant_weights([dict(W=W, s_fp=s, c=c, alpha=a, codes=wc, scale_bytes=wsb)], fmt, sb, ws=ws_fq,
                                scale_layout=bm, code_layout=F.CODES_K_SLAB)
            F.recon_gemm_fwd_mxfp4(xc, xs, wc, wsb, Y, ws=ws_fwd, out=out["dY"], loss=out["loss"])
            F.recon_gemm_bwd_mxfp4(out["dY"], xc, xs, W, sb, s, c, ws=ws_bwd, out=(out["gs"], out["gc"]))
    else:
        xh, wh = torch.empty_like(X), torch.empty_like(W)

        def step():
            F.fakequant_fwd(X, fmt, sb, ws=ws_fq, out=xh)
            F.fakequant_weights([dict(W=W, s_fp=s, c=c, alpha=a, W_hat=wh)], fmt, sb, ws=ws_fq)
            F.recon_gemm_fwd(xh, wh, Y, ws=ws_fwd, out=out["dY"], loss=out["loss"])
            F.recon_gemm_bwd(out["dY"], xh, W, fmt, sb, s, c, a, ws=ws_bwd, out=(out["gs"], out["gc"]))
    return step, out, X


def same_bits(a, b):
    if a.dtype in (torch.bfloat16, torch.float16):
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    if a.dtype == torch.float64:
        return torch.equal(a.view(torch.int64), b.view(torch.int64))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


CASES = [("linear256_mxfp4_f32", 0, 0, False), ("block2560_mxfp4", 512, 4, False), ("block2560_mxfp4", 512, 4, True)]


@pytest.mark.parametrize("name,M,div,packed", CASES)
def test_graph_replays_equal_eager(F, name, M, div, packed):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[name]
    if div:
        w = synth.scaled(w, M=M, hidden_div=div, name="graph")
    lin = w.linears[1] if len(w.linears) > 1 else w.linears[0]
    announce(f"graph {name} M={w.M} N={lin.N} K={lin.K} packed={packed}")
    step, out, X = layer_step(F, w, lin, packed)
    step()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in out.items()}
    for v in out.values():
        v.zero_()
    # capture on a side stream of default priority after a warm-up there, as torch recommends
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    other = torch.empty_like(X)
    for r in range(3):
        # the program's own eager work between replays: a library call and a torch kernel
        F.fakequant_fwd(X * 0.5, w.fmt, w.sub_block, out=other)
        for v in out.values():
            v.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in out:
            assert same_bits(out[k], eager[k]), f"replay {r}: {k} differs from the eager step"
    del g
