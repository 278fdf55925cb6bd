"""Benchmark of the FOCUS scale-learning step on one MI355X.

One step = one fwd+bwd scale-learning pass over one decoder block for one batch of calibration
tokens: dynamic activation fake-quant of the block's four distinct inputs, then for each of the
seven linears the weight fake-quant with learned scales, the reconstruction GEMM with the MSE
epilogue, and the fused straight-through backward to the scales and coefficients. Inputs are
seeded synthetic tensors resident in HBM before timing starts. Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import hashlib
import json
import os
import sys
import time

REPO = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, REPO)

METRIC = "ms per fwd+bwd scale-learning step per decoder block; fake-quant GB/s"
DEFAULT_WORKLOAD = "block8192_mxfp4"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP4_TFLOPS = 10100.0   # MI355X dense MXFP4 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector (the fp32 operand path runs on VALU FMAs)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--summarize-trace", metavar="DIR",
                   help="write profiles/ summaries from a rocprofv3 --kernel-trace --stats output directory and exit")
    p.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="write profiles/traffic.json and the HBM traffic summary from the two rocprofv3 --pmc "
                        "output directories (FETCH_SIZE, WRITE_SIZE) of a --steps 1 --warmup 0 "
                        "--copy-calibration run and exit")
    p.add_argument("--summarize-mfma", metavar="DIR",
                   help="write the MFMA-utilisation summary from the rocprofv3 --pmc output directory of a "
                        "--steps 1 --warmup 0 --copy-calibration run with the counters of PMC_MFMA and exit")
    p.add_argument("--summarize-memory", metavar="DIR",
                   help="write profiles/gemm_memory_<workload>.md from a rocprofv3 --pmc run of PMC_MEM")
    p.add_argument("--summarize-stalls", metavar="DIR",
                   help="write the wave-cycle breakdown of the GEMMs from the rocprofv3 --pmc output directory of a "
                        "--steps 1 --warmup 0 run with the counters of PMC_STALL and exit")
    p.add_argument("--summarize-extras", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="write profiles/hbm_traffic_extras_<workload>.md (the chaining and optimizer kernels) from "
                        "two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of a full --steps 1 --warmup 0 "
                        "--copy-calibration run and exit")
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--tokens", type=int, default=0, help="override the token count (0 = the workload's)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample-tokens", type=int, default=32768)
    p.add_argument("--cpu-sample-rows", type=int, default=512)
    p.add_argument("--fwd-operands", choices=("auto", "bf16", "mxfp4"), default="auto",
                   help="forward reconstruction GEMM from bf16 X_hat / W_hat, or (MXFP4 workloads) from their "
                        "packed FP4 codes and E8M0 scales on the block-scaled FP4 MFMA; auto = mxfp4 where the "
                        "workload's format and shapes allow it, else bf16")
    p.add_argument("--sub-block", type=int, default=0, help="elements per coefficient c (0 = the workload's)")
    p.add_argument("--no-coeff", action="store_true", help="the baseline mode: no coefficients (c = 1)")
    p.add_argument("--weights-per-layer", action="store_true",
                   help="fake-quantise each linear's weights with its own call instead of one grouped call")
    p.add_argument("--e8m0", choices=("ceil", "floor"), default="ceil",
                   help="MXFP4 scale rounding: up (the paper's) or the OCP floor rule")
    p.add_argument("--step-only", action="store_true",
                   help="time the step only (no graph replay, cold-cache pass, other operands, chaining, optimizer, "
                        "export or attainable rates): for profiling runs")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run an untimed 1 GiB device copy first (a known-size reference for HBM counters)")
    return p.parse_args()


class Timer:
    """HIP events on the current stream around each library call, grouped by kernel family. With
    `before`, before(name) runs ahead of each call's start event (untimed), e.g. a cache flush."""

    def __init__(self, torch, before=None):
        self.torch = torch
        self.spans = {}
        self.before = before

    def run(self, name, fn, units):
        t = self.torch
        if self.before is not None:
            self.before(name)
        a, b = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
        a.record()
        out = fn()
        b.record()
        self.spans.setdefault(name, []).append((a, b, units))
        return out

    def summary(self):
        res = {}
        for name, spans in self.spans.items():
            ms = [a.elapsed_time(b) for a, b, _ in spans]
            res[name] = {"launches": len(ms), "total_ms": sum(ms), "avg_ms": sum(ms) / len(ms),
                         "units": sum(u for _, _, u in spans)}
        return res


def kernel_source_hash(csrc_dir=None):
    """Hash of the library sources with comments and whitespace removed: a change of code changes
    it, a change of comments does not."""
    import re
    csrc_dir = csrc_dir or os.path.join(REPO, "paper_2608_01847_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(csrc_dir)):
        with open(os.path.join(csrc_dir, f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(f.encode() + " ".join(text.split()).encode())
    return h.hexdigest()[:16]


def traffic_path(workload):
    return os.path.join(REPO, "profiles", f"traffic_{workload}.json")


def traffic_from_profile(kernel: str, src_hash: str, path):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it is current."""
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    entry = data.get(kernel)
    if not entry or entry.get("source_hash") != src_hash:
        return None
    return entry.get("bytes_per_launch")


def main():
    args = parse()
    if (args.summarize_trace or args.summarize_counters or args.summarize_mfma or args.summarize_stalls
            or args.summarize_memory or args.summarize_extras):
        if args.summarize_extras:
            summarize_extras(*args.summarize_extras, args.workload)
        if args.summarize_trace:
            summarize_trace(args.summarize_trace, args.workload)
        if args.summarize_counters:
            summarize_counters(*args.summarize_counters, args.workload)
        if args.summarize_mfma:
            summarize_mfma(args.summarize_mfma, args.workload)
        if args.summarize_stalls:
            summarize_stalls(args.summarize_stalls, args.workload)
        if args.summarize_memory:
            summarize_memory(args.summarize_memory, args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the data-parallel path across GPUs is not built "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_01847_amd import focus as F
    from paper_2608_01847_amd import synth

    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    w = synth.WORKLOADS[args.workload]
    if args.tokens:
        w = synth.scaled(w, M=args.tokens, name=w.name)
    dev = "cuda"
    torch.cuda.set_device(0)
    fmt, sb, M = w.fmt, args.sub_block or w.sub_block, w.M
    rnd = 1 if args.e8m0 == "floor" else 0
    B = w.block

    # ---- inputs and state, resident in HBM before timing (untimed) ----
    acts = {src: synth.activation(w, src, device=dev) for src in w.inputs}
    layers = []
    for lin in w.linears:
        W = synth.weight(w, lin, device=dev)
        Y = synth.reference_output(acts[lin.source], W)
        s, c, a = F.scales_init(W, fmt, sb, e8m0_rounding=rnd)
        layers.append(dict(lin=lin, W=W, Y=Y, s=s, c=c, cf=None if args.no_coeff else c, a=a,
                           W_hat=torch.empty_like(W),
                           gs=torch.empty_like(s), gc=torch.empty_like(c),
                           loss=torch.empty(1, dtype=torch.float64, device=dev)))
    x_hat = {src: torch.empty_like(x) for src, x in acts.items()}  # bf16 X_hat (the bf16-operand step)
    mx_possible = (fmt == 0 and w.dtype == "bf16" and M % 4 == 0
                   and all(l.K % 128 == 0 and l.N % 8 == 0 for l in w.linears))
    if args.fwd_operands == "mxfp4" and not mx_possible:
        print("--fwd-operands mxfp4 needs an MXFP4 workload whose shapes the FP4 forward takes", file=sys.stderr)
        sys.exit(2)
    mx_primary = args.fwd_operands == "mxfp4" or (args.fwd_operands == "auto" and mx_possible)
    if mx_possible:  # packed operands of the MXFP4 GEMMs, in the layouts they read: activation codes
        # [M][K/2], weight codes in K-slabs [K/128][N][64], E8M0 bytes block-major [K/32][rows]
        slab = F.CODES_K_SLAB
        x_codes = {src: torch.empty(M, x.shape[1] // 2, dtype=torch.uint8, device=dev) for src, x in acts.items()}
        x_scales = {src: torch.empty(x.shape[1] // 32, M, dtype=torch.uint8, device=dev) for src, x in acts.items()}
        for L in layers:
            N_, K_ = L["W"].shape
            L["Wc"] = torch.empty(*F.codes_shape(N_, K_, slab), dtype=torch.uint8, device=dev)
            L["Ws"] = torch.empty(K_ // 32, N_, dtype=torch.uint8, device=dev)
    max_n = max(l.N for l in w.linears)
    dY_buf = torch.empty(M * max_n, dtype=acts[w.linears[0].source].dtype, device=dev)
    q = F.qconfig(fmt, sb)
    ws_fq = F.workspace(F.workspace_size(F.CALL_FAKEQUANT_FWD, q, 0, M, max(w.inputs.values())))
    ws_fwd = F.workspace(max(F.workspace_size(F.CALL_RECON_GEMM_FWD, q, M, l.N, l.K) for l in w.linears))
    ws_bwd = F.workspace(max(F.workspace_size(F.CALL_RECON_GEMM_BWD, q, M, l.N, l.K) for l in w.linears))
    torch.cuda.synchronize()

    n_weights = sum(l.N * l.K for l in w.linears)
    # the weight pass: every linear's fake quantisation in one grouped call (one launch), or with
    # --weights-per-layer one call per linear
    group_mx = [dict(W=L["W"], s_fp=L["s"], c=L["cf"], alpha=L["a"], codes=L.get("Wc"), scale_bytes=L.get("Ws"))
                for L in layers]
    group_bf = [dict(W=L["W"], s_fp=L["s"], c=L["cf"], alpha=L["a"], W_hat=L["W_hat"]) for L in layers]

    def weight_pass(timer, mx_fwd):
        if mx_fwd:
            # the forward's weight operand is the deployable export: codes + E8M0 bytes, no bf16 W_hat
            timer.run("fakequant_weight", lambda: F.fakequant_weights(group_mx, fmt, sb, ws=ws_fq,
                                                                      scale_layout=F.SCALES_BLOCK_MAJOR,
                                                                      e8m0_rounding=rnd, code_layout=F.CODES_K_SLAB),
                      n_weights)
        else:
            timer.run("fakequant_weight", lambda: F.fakequant_weights(group_bf, fmt, sb, ws=ws_fq, e8m0_rounding=rnd),
                      n_weights)

    def step(timer, mx_fwd):
        for src, x in acts.items():
            rows, K = x.shape
            if mx_fwd:
                # the packed form only: both GEMMs read the codes and E8M0 bytes, no bf16 X_hat
                timer.run("fakequant_act", lambda: F.fakequant_fwd(x, fmt, sb, ws=ws_fq, want_x_hat=False,
                                                                   e8m0_rounding=rnd, codes_out=x_codes[src],
                                                                   scales_out=x_scales[src],
                                                                   scale_layout=F.SCALES_BLOCK_MAJOR),
                          rows * K)
            else:
                timer.run("fakequant_act", lambda: F.fakequant_fwd(x, fmt, sb, ws=ws_fq, out=x_hat[src], e8m0_rounding=rnd),
                          rows * K)
        if not args.weights_per_layer:
            weight_pass(timer, mx_fwd)
        for L in layers:
            lin = L["lin"]
            xh = x_hat[lin.source]
            dY = dY_buf[:M * lin.N].view(M, lin.N)
            if mx_fwd and args.weights_per_layer:
                timer.run("fakequant_weight",
                          lambda: F.export_packed(L["W"], fmt, sb, L["s"], L["cf"], L["a"], ws=ws_fq,
                                                  out=(L["Wc"], L["Ws"]), scale_layout=F.SCALES_BLOCK_MAJOR,
                                                  e8m0_rounding=rnd, code_layout=F.CODES_K_SLAB),
                          lin.N * lin.K)
            elif args.weights_per_layer:
                timer.run("fakequant_weight",
                          lambda: F.fakequant_fwd(L["W"], fmt, sb, L["s"], L["cf"], L["a"], ws=ws_fq, out=L["W_hat"],
                                                  e8m0_rounding=rnd),
                          lin.N * lin.K)
            if mx_fwd:
                timer.run("recon_gemm_fwd",
                          lambda: F.recon_gemm_fwd_mxfp4(x_codes[lin.source], x_scales[lin.source], L["Wc"], L["Ws"],
                                                         L["Y"], ws=ws_fwd, out=dY, loss=L["loss"]),
                          2 * M * lin.N * lin.K)
            else:
                timer.run("recon_gemm_fwd",
                          lambda: F.recon_gemm_fwd(xh, L["W_hat"], L["Y"], ws=ws_fwd, out=dY, loss=L["loss"]),
                          2 * M * lin.N * lin.K)
            if mx_fwd:
                timer.run("recon_gemm_bwd",
                          lambda: F.recon_gemm_bwd_mxfp4(dY, x_codes[lin.source], x_scales[lin.source], L["W"], sb,
                                                         L["s"], L["cf"], ws=ws_bwd, e8m0_rounding=rnd,
                                                         out=(L["gs"], L["gc"])),
                          2 * M * lin.N * lin.K)
            else:
                timer.run("recon_gemm_bwd",
                          lambda: F.recon_gemm_bwd(dY, xh, L["W"], fmt, sb, L["s"], L["cf"], L["a"], ws=ws_bwd,
                                                   e8m0_rounding=rnd, out=(L["gs"], L["gc"])),
                          2 * M * lin.N * lin.K)

    def cold_fakequant(mx_fwd, steps):
        """The step again with the caches flushed before every fake-quant call: a kernel reads a 1 GiB
        buffer (4x the 256 MB Infinity Cache, far beyond the L2s) ahead of the call's start event, so
        each call streams its tensors from HBM. The flush reads rather than writes: written lines would
        be written back to HBM inside the timed call. Only the fake-quant spans are used."""
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        sink = torch.empty((), dtype=torch.float32, device=dev)

        def before(name):
            if name.startswith("fakequant"):
                torch.sum(flush, dim=0, out=sink)

        for _ in range(steps):
            timer = Timer(torch, before)
            step(timer, mx_fwd)
        torch.cuda.synchronize()
        del flush
        return timer.summary()

    def run(mx_fwd):
        """Warm-up, then exactly args.steps timed steps; -> (ms per step, per-family summary)."""
        for _ in range(args.warmup):
            step(Timer(torch), mx_fwd)
        torch.cuda.synchronize()
        if F.check_flags(ws_fq) != F.OK:
            raise RuntimeError("domain error in the warm-up steps")
        timer = Timer(torch)
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        marks[0].record()
        for i in range(args.steps):
            step(timer, mx_fwd)
            marks[i + 1].record()
        torch.cuda.synchronize()
        per_step = [marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)]
        run.per_step = per_step
        return marks[0].elapsed_time(marks[-1]) / args.steps, timer.summary()

    class Direct:
        """The library calls without the per-call events (for graph capture)."""

        def run(self, name, fn, units):
            return fn()

    def graph_run(mx_fwd):
        """The same step captured once in a HIP graph and replayed: warm-up replays, then exactly
        args.steps timed replays. Every call of the step is stream-ordered and allocates nothing."""
        side = torch.cuda.Stream()  # default priority
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(Direct(), mx_fwd)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(Direct(), mx_fwd)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(args.steps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / args.steps
        loss = float(sum(L["loss"].item() for L in layers))
        del g
        return ms, loss

    mx_fwd = mx_primary
    ms_per_step, kern = run(mx_fwd)
    per_step = sorted(run.per_step)
    block_loss = float(sum(L["loss"].item() for L in layers))
    if args.step_only:
        print(json.dumps({"metric": METRIC, "value": round(ms_per_step, 4), "unit": "ms per step", "n_gpus": 1,
                          "steps": args.steps, "warmup": args.warmup, "step_only": True, "block_loss": block_loss,
                          "config": {"workload": w.name, "tokens": M},
                          "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]}
                                      for k, v in kern.items()}}), flush=True)
        return
    clocks = gpu_clocks()
    kern_cold = cold_fakequant(mx_fwd, 2)
    try:
        graph_ms, graph_loss = graph_run(mx_fwd)
        graph_res = {"ms_per_step": round(graph_ms, 4), "replays": args.steps, "same_loss": graph_loss == block_loss}
    except RuntimeError as e:  # the eager line stands on its own; report why the replay is missing
        torch.cuda.synchronize()
        graph_res = {"error": str(e).splitlines()[0][:200]}

    # ---- algorithmic work ----
    # fake quantisation bytes per element: activations read 2 + write 2 (bf16) (+2 for the NVFP4
    # tensor-absmax pass; the MXFP4-operand step writes codes 0.5 + scale bytes 1/32 instead of X_hat);
    # weights read W 2 + S_fp 4/B + c 4/sb, write W_hat 2 (or, for the MXFP4-operand step, codes 0.5 +
    # bytes 1/32)
    esz = 2 if w.dtype == "bf16" else 4
    act_b = (esz + 0.5 + 1.0 / 32) if mx_fwd else (2 * esz + (esz if fmt == 1 else 0))
    c_b = 0.0 if args.no_coeff else 4.0 / sb
    wt_b = esz + 4.0 / B + c_b + ((0.5 + 1.0 / 32) if mx_fwd else esz)
    fq_bytes = kern["fakequant_act"]["units"] * act_b + kern["fakequant_weight"]["units"] * wt_b
    fq_ms = kern["fakequant_act"]["total_ms"] + kern["fakequant_weight"]["total_ms"]
    fq_cold_ms = kern_cold["fakequant_act"]["total_ms"] + kern_cold["fakequant_weight"]["total_ms"]
    fq_cold_bytes = kern_cold["fakequant_act"]["units"] * act_b + kern_cold["fakequant_weight"]["units"] * wt_b

    if esz == 4:  # fp32 operands: the VALU kernels
        peaks = {"recon_gemm_fwd": PEAK_FP32_TFLOPS, "recon_gemm_bwd": PEAK_FP32_TFLOPS}
    else:
        peaks = {"recon_gemm_fwd": PEAK_FP4_TFLOPS if mx_fwd else PEAK_BF16_TFLOPS, "recon_gemm_bwd": PEAK_BF16_TFLOPS}
    gemm = {k: {"TFLOPs": round(kern[k]["units"] / (kern[k]["total_ms"] * 1e-3) / 1e12, 1), "peak": peaks[k],
                "frac": round(kern[k]["units"] / (kern[k]["total_ms"] * 1e-3) / 1e12 / peaks[k], 4)}
            for k in ("recon_gemm_fwd", "recon_gemm_bwd")}
    dominant = max(("recon_gemm_fwd", "recon_gemm_bwd"), key=lambda k: kern[k]["total_ms"])
    d = kern[dominant]
    per_launch_flops = d["units"] / d["launches"]
    achieved = per_launch_flops / (d["avg_ms"] * 1e-3) / 1e12
    src_hash = kernel_source_hash()
    if esz == 4:
        kname = {"recon_gemm_fwd": "fwd_valu_kernel", "recon_gemm_bwd": "bwd_valu_kernel"}[dominant]
    else:
        kname = {"recon_gemm_fwd": "fwd_mfma_kernel_mx" if mx_fwd else "fwd_mfma_kernel",
                 "recon_gemm_bwd": "bwd_mfma_mx_kernel" if mx_fwd else "bwd_mfma_kernel"}[dominant]
    roofline = {"bound": "alu" if esz == 4 else "mfma", "achieved": round(achieved, 2), "peak": peaks[dominant],
                "unit": "TFLOP/s", "frac": round(achieved / peaks[dominant], 4),
                "traffic": traffic_from_profile(kname, src_hash, traffic_path(w.name)),
                "kernel": kname, "avg_launch_ms": round(d["avg_ms"], 4), "launches": d["launches"],
                "flops_per_launch": per_launch_flops}

    result = {
        "metric": METRIC, "value": round(ms_per_step, 4), "unit": "ms per step", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": ("mxfp4+bf16" if mx_fwd else "bf16") if esz == 2 else "f32",
        "data": "synthetic (seeded; shapes and distributions of the calibration workload)",
        "config": {"workload": w.name, "tokens": M, "format": "mxfp4" if fmt == 0 else "nvfp4", "sub_block": sb,
                   "coefficients": not args.no_coeff, "e8m0": args.e8m0,
                   "fwd_operands": "mxfp4" if mx_fwd else "bf16",
                   "linears": {l.name: [l.N, l.K] for l in w.linears}},
        "roofline": roofline,
        "fakequant_GBps": round(fq_bytes / (fq_ms * 1e-3) / 1e9, 1),
        "fakequant_frac_hbm": round(fq_bytes / (fq_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        # each family on its own: algorithmic bytes per element and GB/s against the HBM peak, in the
        # timed step and with the caches flushed before every call
        "fakequant": {k: {"bytes_per_element": round(b, 4),
                          "GBps": round(kern[k]["units"] * b / (kern[k]["total_ms"] * 1e-3) / 1e9, 1),
                          "frac_hbm": round(kern[k]["units"] * b / (kern[k]["total_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                          "cold_GBps": round(kern_cold[k]["units"] * b / (kern_cold[k]["total_ms"] * 1e-3) / 1e9, 1),
                          "cold_frac_hbm": round(kern_cold[k]["units"] * b / (kern_cold[k]["total_ms"] * 1e-3) / 1e9
                                                 / PEAK_HBM_GBPS, 4)}
                      for k, b in (("fakequant_act", act_b), ("fakequant_weight", wt_b))},
        "fakequant_cold_GBps": round(fq_cold_bytes / (fq_cold_ms * 1e-3) / 1e9, 1),
        "fakequant_cold_frac_hbm": round(fq_cold_bytes / (fq_cold_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        # each reconstruction GEMM against the peak of the MFMA it runs on
        "gemm": gemm,
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "total_ms_per_step": round(v["total_ms"] / args.steps, 4),
                        "launches_per_step": v["launches"] // args.steps} for k, v in kern.items()},
        "step_ms": {"median": round(per_step[len(per_step) // 2], 4), "min": round(per_step[0], 4),
                    "max": round(per_step[-1], 4)},
        "block_loss": block_loss,
        # the same step as one HIP graph (no per-call events, no launch gaps); same results
        "graph": graph_res,
        "source_hash": src_hash,
        "device": device_info(torch, clocks),
    }
    if mx_possible:
        # the same step with the other forward operands, same inputs: under MXFP4, X_hat and W_hat
        # are exactly E2M1 codes times power-of-two block scales, so the bf16 and the block-scaled FP4
        # MFMA form the same exact products and differ only in the fp32 accumulation order
        alt = not mx_fwd
        alt_ms, alt_kern = run(alt)
        alt_loss = float(sum(L["loss"].item() for L in layers))
        f = alt_kern["recon_gemm_fwd"]
        peak = PEAK_FP4_TFLOPS if alt else PEAK_BF16_TFLOPS
        tf = f["units"] / (f["total_ms"] * 1e-3) / 1e12
        result["mxfp4_forward" if alt else "bf16_forward"] = {
            "ms_per_step": round(alt_ms, 4), "block_loss": alt_loss,
            "recon_gemm_fwd": {"TFLOPs": round(tf, 1), "peak": peak, "frac": round(tf / peak, 4)},
            "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "total_ms_per_step": round(v["total_ms"] / args.steps, 4)}
                        for k, v in alt_kern.items()}}
    result["chain"] = chain_costs(torch, F, layers, acts, x_hat, fmt, sb, M, ws_fwd, rnd)
    opt = optimizer_and_export(torch, F, layers, fmt, sb, B, esz, ws_fq, rnd, c_b)
    result["optimizer"] = {"adamw": opt["adamw"]}
    # the deployable export of every linear (Fig. 3(d)), timed on its own outside the step
    result["export"] = opt["export"]
    big = max(w.linears, key=lambda l: l.N * l.K)
    result["attainable"] = attainable(torch, fq_GBps=fq_bytes / (fq_ms * 1e-3) / 1e9,
                                      layer=(M, big.N, big.K) if esz == 2 else None, mx=mx_possible)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_tokens, args.cpu_sample_rows)
    print(json.dumps(result), flush=True)


def optimizer_and_export(torch, F, layers, fmt, sb, B, esz, ws, rnd, c_b, reps=5):
    """Outside the step (as the optimizer and the export are): one AdamW step on every linear's S_fp
    and c (log2 domain, the paper's learning rates), and the deployable export of every linear.
    AdamW moves 28 B per parameter (p, g, m, v read; p, m, v written); the export reads W, S_fp and
    c and writes the packed codes and scale bytes."""
    lr_s, lr_c = {0: (2e-2, 5e-2), 1: (5e-3, 1e-3)}[fmt]
    moms = [(torch.zeros_like(L["s"]), torch.zeros_like(L["s"]), torch.zeros_like(L["c"]), torch.zeros_like(L["c"]))
            for L in layers]
    outs = [(torch.empty(L["W"].shape[0], L["W"].shape[1] // 2, dtype=torch.uint8, device=L["W"].device),
             torch.empty(L["W"].shape[0], L["W"].shape[1] // B, dtype=torch.uint8, device=L["W"].device))
            for L in layers]
    s0 = [(L["s"].clone(), L["c"].clone()) for L in layers]

    def adam_all(t):
        for L, (ms, vs, mc, vc) in zip(layers, moms):
            F.adamw_step(L["s"], L["gs"], ms, vs, t, lr_s, log2_domain=True, ws=ws)
            F.adamw_step(L["c"], L["gc"], mc, vc, t, lr_c, log2_domain=True, ws=ws)

    group = [dict(W=L["W"], s_fp=L["s"], c=L["cf"], alpha=L["a"], codes=o[0], scale_bytes=o[1])
             for L, o in zip(layers, outs)]

    def export_all():
        # one grouped call: every linear's export in one launch
        F.fakequant_weights(group, fmt, sb, ws=ws, e8m0_rounding=rnd)

    def export_per_layer():
        for L, o in zip(layers, outs):
            F.export_packed(L["W"], fmt, sb, L["s"], L["cf"], L["a"], ws=ws, out=o, e8m0_rounding=rnd)

    def export_cold():
        """The grouped export with the caches flushed first (a kernel reading 1 GiB)."""
        flush = torch.ones(1 << 28, dtype=torch.float32, device=layers[0]["W"].device)
        sink = torch.empty((), dtype=torch.float32, device=flush.device)
        torch.sum(flush, dim=0, out=sink)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        export_all()
        b.record()
        torch.cuda.synchronize()
        del flush
        return a.elapsed_time(b)

    res = {}
    for name, fn in (("adamw", lambda t: adam_all(t)), ("export", lambda t: export_all()),
                     ("export_per_layer", lambda t: export_per_layer())):
        fn(1)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for t in range(reps):
            fn(t + 2)
        b.record()
        torch.cuda.synchronize()
        res[name] = a.elapsed_time(b) / reps
    res["export_cold"] = min(export_cold() for _ in range(2))
    if F.check_flags(ws) != F.OK:
        raise RuntimeError("domain error in the optimizer step")
    for L, (s, c) in zip(layers, s0):  # leave the timed state as it was
        L["s"].copy_(s)
        L["c"].copy_(c)
    n_params = sum(L["s"].numel() + L["c"].numel() for L in layers)
    n_w = sum(L["W"].numel() for L in layers)
    adam_bytes = 28 * n_params
    exp_bytes = n_w * (esz + 4.0 / B + c_b + 0.5 + 1.0 / B)
    return {"adamw": {"ms_per_block": round(res["adamw"], 4), "params": n_params, "launches": 2 * len(layers),
                      "GBps": round(adam_bytes / (res["adamw"] * 1e-3) / 1e9, 1),
                      "frac_hbm": round(adam_bytes / (res["adamw"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)},
            "export": {"ms_per_block": round(res["export"], 4), "weights": n_w, "launches": 1,
                       "per_layer_calls_ms_per_block": round(res["export_per_layer"], 4),
                       "bytes_per_weight": round(exp_bytes / n_w, 4), "scale_layout": "row-major",
                       "GBps": round(exp_bytes / (res["export"] * 1e-3) / 1e9, 1),
                       "frac_hbm": round(exp_bytes / (res["export"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                       "cold_ms_per_block": round(res["export_cold"], 4),
                       "cold_GBps": round(exp_bytes / (res["export_cold"] * 1e-3) / 1e9, 1),
                       "cold_frac_hbm": round(exp_bytes / (res["export_cold"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}}


def chain_costs(torch, F, layers, acts, x_hat, fmt, sb, M, ws, rnd, reps=3):
    """Outside the step: what end-to-end chaining adds per block (the input gradient dX_hat = dY W_hat
    of every linear, 2 M N K flops each, and the activation straight-through backward of every block
    input), and the KL-Top loss on a vocabulary-sized logit tensor (8192 tokens x 151,936 logits,
    k = 1000; algorithmic bytes: read both logit rows, write dZ)."""
    dev = acts[layers[0]["lin"].source].device
    max_n = max(L["lin"].N for L in layers)
    dY = (torch.randn(M, max_n, device=dev) * 1e-3).to(acts[layers[0]["lin"].source].dtype)
    ws_dx = F.workspace(max(F.workspace_size(F.CALL_RECON_GEMM_DX, F.qconfig(fmt, sb), M, L["lin"].N, L["lin"].K)
                            for L in layers))
    dxs = {src: torch.empty_like(x) for src, x in acts.items()}
    W_hats = [F.fakequant_fwd(L["W"], fmt, sb, L["s"], L["cf"], L["a"], e8m0_rounding=rnd)[0] for L in layers]

    def dx_all():
        for L, Wh in zip(layers, W_hats):
            lin = L["lin"]
            F.recon_gemm_dx(dY.view(-1)[:M * lin.N].view(M, lin.N), Wh, ws=ws_dx, out=dxs[lin.source])

    def act_all():
        for src, x in acts.items():
            F.fakequant_act_bwd(x, dxs[src], fmt, e8m0_rounding=rnd, ws=ws, out=dxs[src])

    T, V = 8192, 151936
    Zt = (torch.randn(T, V, device=dev) * 3).to(torch.bfloat16)
    Zs = (Zt.float() + torch.randn(T, V, device=dev)).to(torch.bfloat16)
    dZ = torch.empty_like(Zs)
    ws_kl = F.workspace(F.workspace_size(F.CALL_KL_TOP, F.qconfig(fmt, sb), T, V, 0))
    res = {}
    for name, fn in (("dx", dx_all), ("act_bwd", act_all), ("kl_top", lambda: F.kl_top(Zs, Zt, 1000, ws=ws_kl, out=dZ))):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / reps
    if F.check_flags(ws_kl) != F.OK:
        raise RuntimeError("domain error in the KL-Top timing")
    dx_flops = sum(2 * M * L["lin"].N * L["lin"].K for L in layers)
    act_elems = sum(x.numel() for x in acts.values())
    esz = acts[layers[0]["lin"].source].element_size()
    del Zt, Zs, dZ, dY
    return {"dx": {"ms_per_block": round(res["dx"], 4), "TFLOPs": round(dx_flops / (res["dx"] * 1e-3) / 1e12, 1),
                   "frac_bf16": round(dx_flops / (res["dx"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
            "act_bwd": {"ms_per_block": round(res["act_bwd"], 4),
                        "GBps": round(act_elems * 3 * esz / (res["act_bwd"] * 1e-3) / 1e9, 1)},
            "kl_top": {"tokens": T, "vocab": V, "k": 1000, "ms": round(res["kl_top"], 4),
                       "us_per_token": round(res["kl_top"] * 1e3 / T, 3),
                       "GBps": round(T * V * 6 / (res["kl_top"] * 1e-3) / 1e9, 1)}}


def under_profiler():
    """Whether rocprofv3 runs this process: its tool library is preloaded and its settings are in the
    environment."""
    return "rocprof" in os.environ.get("LD_PRELOAD", "") or any(k.startswith("ROCPROF") for k in os.environ)


def gpu_clocks():
    """The GPU's clocks as rocm-smi reports them (current levels of sclk, mclk, fclk, socclk), or why
    they could not be read. Under rocprofv3 no child program is started: the profiler has initialised
    the GPU in this process before it began, and a child that execs after such a start is refused."""
    import subprocess
    if under_profiler():
        return {"skipped": "under rocprofv3"}
    try:
        r = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True, text=True, timeout=30)
        data = json.loads(r.stdout)
    except Exception as e:  # noqa: BLE001 (reported, never fatal)
        return {"error": str(e)[:120]}
    card = next(iter(data.values()), {}) if isinstance(data, dict) else {}
    return {k: v for k, v in card.items() if "clock" in k.lower() or "clk" in k.lower()}


def device_info(torch, clocks=None):
    """What ran the measurement: the GPU, its architecture and CU count, the HIP runtime of torch,
    and the clocks rocm-smi reported right after the timed steps."""
    prop = torch.cuda.get_device_properties(0)
    return {"name": prop.name, "arch": getattr(prop, "gcnArchName", ""), "compute_units": prop.multi_processor_count,
            "memory_GiB": round(prop.total_memory / 2 ** 30, 1), "hip": torch.version.hip,
            "clocks_after_timed_steps": clocks}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def attainable(torch, fq_GBps, layer=None, mx=False):
    """Measured attainable rates on this GPU as secondary denominators (not the product's code): a
    1 GiB device copy, a large bf16 library GEMM (torch.mm, 8192^3, random data) and, for `layer`
    = (M, N, K), the library GEMM on that layer's forward ([M][K] x [K][N]) and backward
    ([K][M] x [M][N]) shapes, plain products without the fused epilogues; with `mx`, also the
    library's block-scaled MXFP4 GEMM on the forward shape (torch._scaled_mm on E2M1 operands with
    E8M0 scales per 32, bf16 out; null where this torch build does not offer it)."""
    src = torch.randn(1 << 28, device="cuda").to(torch.bfloat16)
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    bt = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)  # contiguous operands only
    res = {}
    cases = [("copy", lambda: dst.copy_(src), 2 * src.numel() * 2), ("gemm", lambda: torch.mm(a, bt), 2 * 8192 ** 3)]
    if layer:
        M, N, K = layer
        xf = torch.randn(M, K, device="cuda").to(torch.bfloat16)
        wf = torch.randn(K, N, device="cuda").to(torch.bfloat16)
        xb = torch.randn(K, M, device="cuda").to(torch.bfloat16)
        yb = torch.randn(M, N, device="cuda").to(torch.bfloat16)
        cases += [("layer_fwd", lambda: torch.mm(xf, wf), 2 * M * N * K), ("layer_bwd", lambda: torch.mm(xb, yb), 2 * M * N * K)]
    for name, fn, work in cases:
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(10):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = work / (e0.elapsed_time(e1) / 10 * 1e-3)
    del src, dst, a, bt
    copy_GBps, gemm_TF = res["copy"] / 1e9, res["gemm"] / 1e12
    out = {"copy_GBps": round(copy_GBps, 1), "library_bf16_gemm_TFLOPs": round(gemm_TF, 1),
           "fakequant_frac_of_copy": round(fq_GBps / copy_GBps, 4)}
    if layer:
        out["library_layer_gemm"] = {"shape_MNK": list(layer), "fwd_TFLOPs": round(res["layer_fwd"] / 1e12, 1),
                                     "bwd_TFLOPs": round(res["layer_bwd"] / 1e12, 1)}
        del xf, wf, xb, yb
    if layer and mx:
        out["library_layer_gemm"]["fwd_mxfp4_TFLOPs"] = None
        try:
            M, N, K = layer
            u8 = dict(dtype=torch.uint8, device="cuda")
            a4 = torch.randint(0, 256, (M, K // 2), **u8).view(torch.float4_e2m1fn_x2)
            b4 = torch.randint(0, 256, (N, K // 2), **u8).view(torch.float4_e2m1fn_x2)
            sa = torch.randint(118, 124, (M, K // 32), **u8).view(torch.float8_e8m0fnu)
            sb = torch.randint(118, 124, (N, K // 32), **u8).view(torch.float8_e8m0fnu)
            fn = lambda: torch._scaled_mm(a4, b4.t(), sa, sb, out_dtype=torch.bfloat16)
            fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(5):
                fn()
            e1.record()
            torch.cuda.synchronize()
            tf = 2 * M * N * K / (e0.elapsed_time(e1) / 5 * 1e-3) / 1e12
            out["library_layer_gemm"]["fwd_mxfp4_TFLOPs"] = round(tf, 1)
            out["library_layer_gemm"]["fwd_mxfp4_frac"] = round(tf / PEAK_FP4_TFLOPS, 4)
            del a4, b4, sa, sb
        except (RuntimeError, AttributeError, TypeError) as e:  # no MX path in this torch build
            out["library_layer_gemm"]["fwd_mxfp4_error"] = str(e)[:200]
    return out


def cpu_baseline(w, sample_tokens, sample_rows):
    """The CPU oracle on a bounded sample of the same step, extrapolated linearly to the full step.

    Sample: for every input, `sample_tokens` tokens are fake-quantised; for every linear,
    `sample_rows` weight rows are fake-quantised and their reconstruction loss and gradients are
    computed over those tokens. Each part is linear in the tokens and/or rows it covers, so the
    full-step time is each part's time scaled by the covered fraction."""
    import numpy as np
    import torch

    from oracle import focus_oracle as O
    from paper_2608_01847_amd import synth

    O._lib()
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    Ms = min(sample_tokens, w.M)
    full_ms = 0.0
    sample_s = 0.0
    xs = {}
    for src, K in w.inputs.items():
        X = synth.activation(w, src, M=Ms, device="cpu").float().numpy()
        t0 = time.perf_counter()
        xo, _, _, _ = O.fq_act(X, w.fmt)
        dt = time.perf_counter() - t0
        sample_s += dt
        full_ms += dt * 1e3 * (w.M / Ms)
        xs[src] = (X, O.gemm_operand(xo, w.dtype == "bf16"))
    for lin in w.linears:
        R = min(sample_rows, lin.N)
        W = synth.weight(synth.scaled(w, M=Ms, name=w.name), lin, device="cpu")[:R].float().numpy()
        X, X_op = xs[lin.source]
        Y = (X.astype(np.float64) @ W.astype(np.float64).T)
        t0 = time.perf_counter()
        s, c, a = O.init_scales(W, w.fmt, w.sub_block)
        fq = O.fq_weight(W, w.fmt, w.sub_block, s, c, a)
        t1 = time.perf_counter()
        O.recon_layer(X_op, O.gemm_operand(fq.w_hat, w.dtype == "bf16"), Y, fq, w.fmt, w.sub_block, a)
        t2 = time.perf_counter()
        sample_s += t2 - t0
        full_ms += (t1 - t0) * 1e3 * (lin.N / R) + (t2 - t1) * 1e3 * (lin.N / R) * (w.M / Ms)
    return {"value": round(full_ms, 1), "unit": "ms per step", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"{Ms} of {w.M} tokens per input; {sample_rows} weight rows per linear "
                      f"({sample_s:.1f} s measured), extrapolated linearly to the full step"}


# ---- rocprofv3 summaries (host only) ------------------------------------------------------------
# Library kernels by the name bench.py reports them under, and the rocprofv3 name prefix of each.
# The commands below write into OUT, any output directory; the summaries are made from it.
GEMM_KERNELS = {"bwd_mfma_mx_kernel": "void focus::bwd_mfma_mx_kernel<",
                "fwd_mfma_kernel_mx": "void focus::fwd_mfma_kernel<true, true>",
                "fwd_mfma_kernel": "void focus::fwd_mfma_kernel<true, false>",
                "bwd_mfma_kernel": "void focus::bwd_mfma_kernel<"}
FAKEQUANT_KERNELS = {"fq_act_mx_kernel": "void focus::fq_act_mx_kernel<",
                     "absmax_partial_kernel": "void focus::absmax_partial_kernel<",
                     "fq_act_nv_kernel": "void focus::fq_act_nv_kernel<",
                     "fq_weight_kernel": "void focus::fq_weight_kernel<",
                     "fq_weight_group_kernel": "void focus::fq_weight_group_kernel<"}
PROFILED = {**GEMM_KERNELS, **FAKEQUANT_KERNELS}
TRACE_CMD = ("rocprofv3 --kernel-trace --stats -d OUT/prof_trace -o run --output-format csv -- "
             "python3 -u bench.py --steps 5 --warmup 2 --no-cpu-baseline --copy-calibration{wl}")
PMC_CMD = ("rocprofv3 --pmc {c} -d OUT/prof_{d} -o run --output-format csv -- "
           "python3 -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --step-only --copy-calibration{wl}")


# one counter pass (6 SQ and 1 GRBM counters, within what one rocprofv3 pass can collect on gfx950);
# MfmaUtil is rocprofv3's own metric: MFMA-busy cycles summed over SIMDs / (GPU-busy cycles x SIMDs)
PMC_MFMA = ("MfmaUtil SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_MOPS_F8 "
            "SQ_BUSY_CYCLES SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE")  # pass as one --pmc argument list


# where the GEMM waves' cycles go (8 SQ counters, one pass)
PMC_STALL = ("SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_WAIT_INST_LDS SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_VMEM "
             "SQ_LDS_DATA_FIFO_FULL SQ_LDS_CMD_FIFO_FULL")
STALL_CMD = ("rocprofv3 --pmc {c} -d OUT/prof_stall -o run --output-format csv -- "
             "python3 -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --step-only{wl}")

# the GEMMs' memory side (2 TCC, 2 TA, 4 TCP and 1 GRBM counters, one pass)
PMC_MEM = ("TCC_HIT_sum TCC_MISS_sum TA_BUSY_avr TA_ADDR_STALLED_BY_TC_CYCLES_sum TCP_PENDING_STALL_CYCLES_sum "
           "TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCP_TOTAL_CACHE_ACCESSES_sum GRBM_GUI_ACTIVE")
MEM_CMD = ("rocprofv3 --pmc {c} -d OUT/prof_mem -o run --output-format csv -- "
           "python3 -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --step-only{wl}")


def wl_arg(workload):
    """The --workload argument of a profiling command (none for the default workload)."""
    return "" if workload == DEFAULT_WORKLOAD else f" --workload {workload}"


def algorithmic_bytes(kernel, M, N, K, sb, fmt=0):
    """Bytes each input is read and each output written once, per launch: one linear for the GEMMs
    (M tokens, N x K weights); for the fake-quant kernels one [N][K] bf16 tensor as the default step
    runs them (MXFP4: activations and weights written as packed codes + E8M0 bytes; NVFP4: as bf16)."""
    B = 32 if fmt == 0 else 16
    grads = N * K // B * 4 + N * K // sb * 4
    wparams = 2 * N * K + N * K // B * 4 + N * K // sb * 4
    packed = N * (K // 2 + K // 32)
    return {"fwd_mfma_kernel": 2 * M * K + 2 * N * K + 4 * M * N,
            "fwd_mfma_kernel_mx": (M + N) * (K // 2 + K // 32) + 4 * M * N,
            "bwd_mfma_kernel": 2 * M * N + 2 * M * K + wparams + grads,
            "bwd_mfma_mx_kernel": 2 * M * N + M * (K // 2 + K // 32) + wparams + grads,
            "fq_act_mx_kernel": 2 * N * K + packed,
            "absmax_partial_kernel": 2 * N * K,
            "fq_act_nv_kernel": 4 * N * K,
            "fq_weight_kernel": wparams + (packed if fmt == 0 else 2 * N * K)}[kernel]


def launch_algorithmic_bytes(kernel, w, shape):
    """algorithmic_bytes of one launch as step_launches lists it; a grouped weight launch covers every
    linear of the block (its shape entry lists them)."""
    label, rows, K = shape
    if kernel == "fq_weight_group_kernel":
        return sum(algorithmic_bytes("fq_weight_kernel", w.M, n, k, w.sub_block, w.fmt) for n, k in rows)
    return algorithmic_bytes(kernel, w.M, rows, K, w.sub_block, w.fmt)


def step_launches(kernel, w):
    """How a kernel's launches in a `--steps 1 --warmup 0` run map to tensors: (launches before the
    step, [(label, rows, K)] of the step's launches in order). The step fake-quantises the four
    block inputs, then the weights of all linears in one grouped launch (or, with --weights-per-layer,
    each linear's weights); the NVFP4 weight initialisation runs one tensor-absmax pass per linear before
    the step."""
    if kernel in GEMM_KERNELS:
        return 0, [(f"{l.N}x{l.K}", l.N, l.K) for l in w.linears]
    if kernel == "fq_weight_kernel":  # one call per linear (--weights-per-layer)
        return 0, [(f"{l.name} {l.N}x{l.K}", l.N, l.K) for l in w.linears]
    if kernel == "fq_weight_group_kernel":  # the default step: all linears in one launch
        return 0, [(f"all {len(w.linears)} linears", [(l.N, l.K) for l in w.linears], None)]
    acts = [(f"{src} {w.M}x{K}", w.M, K) for src, K in w.inputs.items()]
    return (len(w.linears) if kernel == "absmax_partial_kernel" else 0), acts


def summarize_trace(trace_dir, workload, out_dir=None):
    import csv
    rows = [r for r in csv.DictReader(open(os.path.join(trace_dir, "run_kernel_stats.csv")))
            if "focus::" in r["Name"]]
    out = os.path.join(out_dir or os.path.join(REPO, "profiles"), f"step_{workload}_kernel_stats.md")
    with open(out, "w") as f:
        f.write(f"# Kernel-trace summary: scale-learning steps of the {workload} workload\n\n")
        f.write("Command (from the repository root on one MI355X; OUT is any output directory):\n\n    " +
                TRACE_CMD.format(wl=wl_arg(workload)) + "\n\n")
        other = (" and then the same step with the other forward and backward operands" if workload.endswith("_mxfp4")
                 else "")
        f.write(f"The run times the step (2 warm-up + 5 timed){other}, and the calls outside the step (chaining, "
                f"AdamW, export); library kernels only, source hash `{kernel_source_hash()}`:\n\n")
        f.write("| Kernel | Calls | Avg us | Min us | Max us | Share of GPU time |\n|---|---|---|---|---|---|\n")
        for r in rows:
            name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")
            f.write(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | {float(r['MinNs']) / 1e3:.1f} | "
                    f"{float(r['MaxNs']) / 1e3:.1f} | {float(r['Percentage']):.2f}% |\n")
    print(out)


def summarize_counters(fetch_dir, write_dir, workload, out_dir=None):
    import csv

    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    runs = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv")))
                if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        # the untimed 1 GiB device copy of --copy-calibration is the run's first copy kernel
        copy = next(r for r in rows if "copyBuffer" in r["Kernel_Name"])
        scale = (1 << 30) / (float(copy["Counter_Value"]) * 1024)
        per = {}
        for k, pre in PROFILED.items():
            skip, shapes = step_launches(k, w)
            vals = [float(r["Counter_Value"]) * 1024 * scale for r in rows if r["Kernel_Name"].startswith(pre)]
            per[k] = vals[skip:skip + len(shapes)]
        runs[counter] = (scale, per, float(copy["Counter_Value"]))
    fscale, fetch, fraw = runs["FETCH_SIZE"]
    wscale, write, wraw = runs["WRITE_SIZE"]
    src = kernel_source_hash()
    data = {"_calibration": {"copy_bytes": 1 << 30, "fetch_scale": fscale, "write_scale": wscale,
                             "note": "scales = known bytes of a 1 GiB device copy / what FETCH_SIZE and WRITE_SIZE "
                                     "read for it"}}
    md = [f"# HBM-side traffic of the reconstruction GEMMs and fake-quant kernels ({workload}, {w.M:,} tokens)\n",
          "Commands (one counter per run, from the repository root on one MI355X; OUT is any output directory):\n",
          "    " + PMC_CMD.format(c="FETCH_SIZE", d="fetch", wl=wl_arg(workload)),
          "    " + PMC_CMD.format(c="WRITE_SIZE", d="write", wl=wl_arg(workload)) + "\n",
          f"Calibration with the untimed 1 GiB device copy in the same runs: FETCH_SIZE reads {fraw:.0f} KiB (scale "
          f"{fscale:.3f}), WRITE_SIZE reads {wraw:.0f} KiB (scale {wscale:.3f}). The counters count L2 misses (traffic "
          f"to the Infinity Cache / HBM), per dispatch. Algorithmic bytes: every input read and every output written "
          f"once (fake-quant kernels: the default step's outputs, packed codes + E8M0 bytes under MXFP4, bf16 "
          f"under NVFP4). Source hash of the kernels: `{src}`.\n",
          "| Kernel | Tensor (rows x K) | fetched MB | written MB | algorithmic MB | ratio |", "|---|---|---|---|---|---|"]
    for k in PROFILED:
        if not fetch[k]:
            continue
        n = min(len(fetch[k]), len(write[k]))
        tot = [fetch[k][i] + write[k][i] for i in range(n)]
        algs = [launch_algorithmic_bytes(k, w, sh) for sh in step_launches(k, w)[1][:n]]
        data[k] = {"bytes_per_launch": sum(tot) / n, "algorithmic_bytes_per_launch": sum(algs) / n,
                   "source_hash": src, "launches": n}
        for i, (label, rows, K) in enumerate(step_launches(k, w)[1][:n]):
            md.append(f"| `{k}` | {label} | {fetch[k][i] / 1e6:.0f} | {write[k][i] / 1e6:.0f} | {algs[i] / 1e6:.0f} | "
                      f"{tot[i] / algs[i]:.2f} |")
    out_dir = out_dir or os.path.join(REPO, "profiles")
    with open(os.path.join(out_dir, f"traffic_{workload}.json"), "w") as f:
        json.dump(data, f, indent=1)
    out = os.path.join(out_dir, f"hbm_traffic_{workload}.md")
    with open(out, "w") as f:
        f.write("\n".join(md) + "\n")
    print(out)


EXTRA_KERNELS = {"transpose_kernel": "transpose_kernel<", "fq_act_bwd_kernel": "fq_act_bwd_kernel<",
                 "kl_top_kernel": "kl_top_kernel<", "adamw_kernel": "adamw_kernel"}
EXTRAS_CMD = ("rocprofv3 --pmc {c} -d OUT/prof_extras_{d} -o run --output-format csv -- "
              "python3 -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --copy-calibration{wl}")


def extra_launches(kernel, w):
    """One call's launches of a kernel outside the step, in order, with their algorithmic bytes: the
    transposes of dX (every linear's bf16 W_hat read and written once), the activation straight-through
    backward (every bf16 block input: X and dX_hat read, dX written), KL-Top (8,192 x 151,936 bf16 logits:
    both rows read, dZ written) and AdamW (S_fp, then c, of every linear: p, g, m, v read, p, m, v written,
    28 B per fp32 parameter). The bench repeats each call, so a position's launches are pooled."""
    if kernel == "transpose_kernel":
        return [(f"{l.name} {l.N}x{l.K}", 4 * l.N * l.K) for l in w.linears]
    if kernel == "fq_act_bwd_kernel":
        return [(f"{src} {w.M}x{K}", 6 * w.M * K) for src, K in w.inputs.items()]
    if kernel == "kl_top_kernel":
        return [("8192 x 151936 bf16, k = 1000", 8192 * 151936 * 6)]
    out = []
    for l in w.linears:
        out.append((f"{l.name} S_fp {l.N}x{l.K // w.block}", 28 * l.N * (l.K // w.block)))
        out.append((f"{l.name} c {l.N}x{l.K // w.sub_block}", 28 * l.N * (l.K // w.sub_block)))
    return out


def summarize_extras(fetch_dir, write_dir, workload, out_dir=None):
    """HBM-side bytes of the calls outside the step (chaining, AdamW) against their algorithmic bytes:
    for each launch position of a call, the median over the bench's repetitions of that call."""
    import csv
    import statistics

    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    got = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv")))
                if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        copy = next(r for r in rows if "copyBuffer" in r["Kernel_Name"])
        scale = (1 << 30) / (float(copy["Counter_Value"]) * 1024)
        per = {}
        for k, pat in EXTRA_KERNELS.items():
            vals = [float(r["Counter_Value"]) * 1024 * scale for r in rows if pat in r["Kernel_Name"]]
            n = len(extra_launches(k, w))
            per[k] = [statistics.median(vals[i::n]) for i in range(n)] if len(vals) >= n else []
        got[counter] = (scale, per)
    md = [f"# HBM-side traffic of the chaining and optimizer kernels ({workload}, {w.M:,} tokens)\n",
          "Commands (one counter per run, from the repository root on one MI355X; OUT is any output directory):\n",
          "    " + EXTRAS_CMD.format(c="FETCH_SIZE", d="fetch", wl=wl_arg(workload)),
          "    " + EXTRAS_CMD.format(c="WRITE_SIZE", d="write", wl=wl_arg(workload)) + "\n",
          f"Each counter scaled by what it reads for the untimed 1 GiB device copy of the same run (FETCH_SIZE "
          f"x{got['FETCH_SIZE'][0]:.3f}, WRITE_SIZE x{got['WRITE_SIZE'][0]:.3f}); per launch position of a call, the "
          f"median over the bench's repetitions of the call. Algorithmic bytes: every input read and every output "
          f"written once (bf16 tensors; AdamW 28 B per fp32 parameter). Source hash of the kernels: "
          f"`{kernel_source_hash()}`.\n",
          "| Kernel | Tensor | fetched MB | written MB | algorithmic MB | ratio |", "|---|---|---|---|---|---|"]
    fetch, write = got["FETCH_SIZE"][1], got["WRITE_SIZE"][1]
    for k in EXTRA_KERNELS:
        if not fetch[k] or not write[k]:
            continue
        for (label, alg), f, wr in zip(extra_launches(k, w), fetch[k], write[k]):
            md.append(f"| `{k}` | {label} | {f / 1e6:.1f} | {wr / 1e6:.1f} | {alg / 1e6:.1f} | {(f + wr) / alg:.2f} |")
    out = os.path.join(out_dir or os.path.join(REPO, "profiles"), f"hbm_traffic_extras_{workload}.md")
    with open(out, "w") as f:
        f.write("\n".join(md) + "\n")
    print(out)


def summarize_mfma(pmc_dir, workload, out_dir=None):
    import csv

    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    vals = {}  # (dispatch, kernel name) -> {counter: value, "ns": duration}
    for r in csv.DictReader(open(os.path.join(pmc_dir, "run_counter_collection.csv"))):
        d = vals.setdefault((int(r["Dispatch_Id"]), r["Kernel_Name"]), {})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    simds = 256 * 4
    md = [f"# MFMA utilisation of the reconstruction GEMMs ({workload}, {w.M:,} tokens)\n",
          "Command (from the repository root on one MI355X; OUT is any output directory):\n",
          "    " + PMC_CMD.format(c=PMC_MFMA, d="mfma", wl=wl_arg(workload)) + "\n",
          "Per launch (one linear layer), the first launches of each kernel in the run (the default step's). "
          "`MFMA busy` is rocprofv3's MfmaUtil: cycles in which a SIMD's matrix unit is busy, summed over the "
          "1,024 SIMDs, over GPU-busy cycles x 1,024. `clock` is the GPU-busy cycle count (the counter's maximum over "
          "instances, recovered from MfmaUtil and the MFMA-busy sum) over the launch's duration in the counter run. "
          "`executed / algorithmic` compares the MFMA work the counters saw with 2 M N K: bf16 MOPS x 512, and for "
          "the FP4 kernel, whose block-scaled MFMA no MOPS counter records, its busy cycles / 32 (a 32x32x64 FP4 "
          "MFMA occupies its SIMD's matrix unit for 32 cycles, as a 32x32x16 bf16 one does) x 131,072 flops. `frac of peak` = algorithmic flops / duration / the dense "
          "peak (bf16 2.5 PFLOP/s, FP4 10.1, both at 2.4 GHz); `frac at the clock` = frac of peak x 2.4 GHz / clock, "
          "the fraction of what the matrix units deliver at the clock they ran at. The clock is as good as the "
          "counter window: where the derived figure exceeds the chip's 2.4 GHz the window was longer than the "
          "kernel's timestamps, and that row's busy share and clock are approximate. LDS conflicts: bank-"
          f"conflict cycles / LDS-active cycles. Source hash of the kernels: `{kernel_source_hash()}`.\n",
          "| Kernel | Layer (N x K) | us | MFMA busy | clock GHz | executed / algorithmic | TFLOP/s | frac of peak | "
          "frac at the clock | LDS conflicts |", "|---|---|---|---|---|---|---|---|---|---|"]
    for k, pre in GEMM_KERNELS.items():
        runs = [(disp, v) for (disp, name), v in sorted(vals.items()) if name.startswith(pre)][:len(w.linears)]
        fp4 = k == "fwd_mfma_kernel_mx"
        peak = PEAK_FP4_TFLOPS if fp4 else PEAK_BF16_TFLOPS
        for (disp, v), lin in zip(runs, w.linears):
            alg = 2.0 * w.M * lin.N * lin.K
            util = v.get("MfmaUtil", 0.0)
            busy = v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            gui = busy * 100.0 / (util * simds) if util > 0 else 0.0
            ghz = gui / v["ns"] if v["ns"] > 0 else 0.0
            mops = busy / 32 * 131072 if fp4 else v.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512
            tf = alg / v["ns"] / 1e3
            frac = tf / peak
            lds = v.get("SQ_LDS_BANK_CONFLICT", 0.0) / max(v.get("SQ_LDS_IDX_ACTIVE", 0.0), 1.0)
            md.append(f"| `{k}` | {lin.N}x{lin.K} | {v['ns'] / 1e3:.0f} | {util:.1f}% | {ghz:.2f} | "
                      f"{mops / alg:.3f} | {tf:.0f} | {frac:.3f} | {frac * 2.4 / ghz if ghz else 0:.3f} | {100 * lds:.1f}% |")
    out = os.path.join(out_dir or os.path.join(REPO, "profiles"), f"mfma_util_{workload}.md")
    with open(out, "w") as f:
        f.write("\n".join(md) + "\n")
    print(out)


def summarize_memory(pmc_dir, workload, out_dir=None):
    """The GEMMs' memory side per launch: L2 hit rate, how busy the texture-address units are, how
    long their address path waits on the L1 and the L1 on L2 data, and the L1->L2 read latency."""
    import csv

    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    vals = {}
    for r in csv.DictReader(open(os.path.join(pmc_dir, "run_counter_collection.csv"))):
        d = vals.setdefault((int(r["Dispatch_Id"]), r["Kernel_Name"]), {})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    cus = 256  # one texture-address unit (TA) and one L1 (TCP) per CU
    md = [f"# Memory side of the reconstruction GEMMs ({workload}, {w.M:,} tokens)\n",
          "Command (from the repository root on one MI355X; OUT is any output directory):\n",
          "    " + MEM_CMD.format(c=PMC_MEM, wl=wl_arg(workload)) + "\n",
          "Per launch (one linear layer; the first launches of each kernel, the default step's). `L2 hit` = TCC_HIT / "
          "(TCC_HIT + TCC_MISS); `TA busy` = TA_BUSY_avr / GRBM_GUI_ACTIVE (share of GPU-busy cycles in which a "
          "CU's texture-address unit works); `TA waits on L1` = TA_ADDR_STALLED_BY_TC_CYCLES_sum / (256 GRBM_GUI_ACTIVE); "
          "`L1 waits on L2` = TCP_PENDING_STALL_CYCLES_sum / (256 GRBM_GUI_ACTIVE); `L1->L2 latency` = "
          "TCP_TCC_READ_REQ_LATENCY_sum / TCP_TCC_READ_REQ_sum (cycles per read request); `L1 reads / KB` = L1->L2 "
          "read requests per KB of the launch's algorithmic operand bytes (each operand read once), i.e. how often "
          f"the tiles re-fetch operands from L2. Source hash of the kernels: `{kernel_source_hash()}`.\n",
          "| Kernel | Layer (N x K) | us | L2 hit | TA busy | TA waits on L1 | L1 waits on L2 | L1->L2 latency | "
          "L1 reads / KB |", "|---|---|---|---|---|---|---|---|---|"]
    for k, pre in GEMM_KERNELS.items():
        runs = [v for (disp, name), v in sorted(vals.items()) if name.startswith(pre)][:len(w.linears)]
        for v, lin in zip(runs, w.linears):
            gui = max(v.get("GRBM_GUI_ACTIVE", 0.0), 1.0)
            hit, miss = v.get("TCC_HIT_sum", 0.0), v.get("TCC_MISS_sum", 0.0)
            req = max(v.get("TCP_TCC_READ_REQ_sum", 0.0), 1.0)
            op_bytes = algorithmic_bytes(k, w.M, lin.N, lin.K, w.sub_block, w.fmt)
            md.append(f"| `{k}` | {lin.N}x{lin.K} | {v['ns'] / 1e3:.0f} | {hit / max(hit + miss, 1.0):.3f} | "
                      f"{v.get('TA_BUSY_avr', 0.0) / gui:.3f} | {v.get('TA_ADDR_STALLED_BY_TC_CYCLES_sum', 0.0) / (cus * gui):.3f} | "
                      f"{v.get('TCP_PENDING_STALL_CYCLES_sum', 0.0) / (cus * gui):.3f} | "
                      f"{v.get('TCP_TCC_READ_REQ_LATENCY_sum', 0.0) / req:.0f} | {req / (op_bytes / 1024):.2f} |")
    out = os.path.join(out_dir or os.path.join(REPO, "profiles"), f"gemm_memory_{workload}.md")
    with open(out, "w") as f:
        f.write("\n".join(md) + "\n")
    print(out)


def summarize_stalls(pmc_dir, workload, out_dir=None):
    import csv

    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    vals = {}
    for r in csv.DictReader(open(os.path.join(pmc_dir, "run_counter_collection.csv"))):
        d = vals.setdefault((int(r["Dispatch_Id"]), r["Kernel_Name"]), {})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    cols = [("SQ_WAIT_ANY", "waiting (waitcnt, barrier)"), ("SQ_WAIT_INST_ANY", "waiting to issue"),
            ("SQ_WAIT_INST_LDS", "waiting to issue LDS"), ("SQ_ACTIVE_INST_LDS", "issuing LDS"),
            ("SQ_ACTIVE_INST_VMEM", "issuing VMEM"), ("SQ_LDS_CMD_FIFO_FULL", "LDS command FIFO full"),
            ("SQ_LDS_DATA_FIFO_FULL", "LDS data FIFO full")]
    md = [f"# Where the GEMM waves' cycles go ({workload}, {w.M:,} tokens)\n",
          "Command (from the repository root on one MI355X; OUT is any output directory):\n",
          "    " + STALL_CMD.format(c=PMC_STALL, wl=wl_arg(workload)) + "\n",
          "Per launch (one linear layer; the first launches of each kernel, the default step's): each counter as a "
          "fraction of SQ_WAVE_CYCLES (cycles the kernel's waves are resident). With one wave per SIMD, a wave "
          "waiting to issue is mostly its next MFMA waiting for the matrix unit; waiting on counters or the barrier "
          "is time in which, unless MFMAs are still in flight, the unit idles. The columns overlap (an LDS or "
          f"memory instruction issues while an MFMA runs). Source hash of the kernels: `{kernel_source_hash()}`.\n",
          "| Kernel | Layer (N x K) | us | " + " | ".join(c for _, c in cols) + " |",
          "|---|---|---|" + "---|" * len(cols)]
    for k, pre in GEMM_KERNELS.items():
        runs = [v for (disp, name), v in sorted(vals.items()) if name.startswith(pre)][:len(w.linears)]
        for v, lin in zip(runs, w.linears):
            wc = max(v.get("SQ_WAVE_CYCLES", 0.0), 1.0)
            md.append(f"| `{k}` | {lin.N}x{lin.K} | {v['ns'] / 1e3:.0f} | " +
                      " | ".join(f"{100 * v.get(c, 0.0) / wc:.1f}%" for c, _ in cols) + " |")
    out = os.path.join(out_dir or os.path.join(REPO, "profiles"), f"gemm_stalls_{workload}.md")
    with open(out, "w") as f:
        f.write("\n".join(md) + "\n")
    print(out)


if __name__ == "__main__":
    main()
