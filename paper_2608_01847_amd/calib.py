"""Calibration epoch of a decoder block: the scale-learning step followed by AdamW, over the batches
of one epoch (Sec. 4.1: AdamW, constant learning rate, one epoch of 1,248 samples at batch 32, i.e.
39 steps; MXFP4 learning rates 2e-2 for the block scales and 5e-2 for the coefficients c, NVFP4
5e-3 and 1e-3).

Every step runs in libfocus: activation fake quantisation of each block input, then per linear the
reference output (the GEMM's plain-product mode on the unquantised operands), weight fake
quantisation, the reconstruction GEMM with the MSE epilogue, the fused straight-through backward and
one AdamW call each for the scales and the coefficients. This module only orders the calls and
holds the tensors.

Variants (a synthetic analogue of the paper's ablation, Table "ablation"):
  rtn      absmax scales (Sec. 3.2 initialisation), c = 1, nothing learned;
  scale    the block scales learned, c = 1 throughout (the baseline of Sec. 3.2, S_q = S_dq);
  crs      scales and one coefficient per block learned (Coupled-Relaxation Scaling, Sec. 3.3);
  crs_dgs  scales and one coefficient per sub-block learned (Dual-Granularity Scaling, Sec. 3.4).

The scales and the coefficients are both stepped in the log2 domain (the stored parameters stay
S_fp, or Delta_fp for NVFP4, and c): the paper does not say in which domain they are learned; an
absolute step of 2e-2 on a scale near 1e-2 cannot be meant, and a linear-domain c stepped at 5e-2
runs through zero within an epoch once its gradient keeps one sign (every element of the sub-block
clamps, its straight-through gradient vanishes and momentum carries c on). Near c = 1 the log2 step
changes c by about ln 2 times the learning rate, close to the linear step the rates were set for.
Inputs are the seeded synthetic batches of `synth`.

With independent activation channels (X^T X nearly diagonal) the coefficients cannot lower the
per-layer loss: c = 1 is round-to-nearest onto the dequantisation grid S_dq * E2M1, optimal for every
element, and a moved threshold only helps through correlations between input channels. The
low-rank activation kind gives the inputs such correlations.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import time
from dataclasses import dataclass

import torch

from . import focus as F
from . import synth

LEARNING_RATES = {F.MXFP4: (2e-2, 5e-2), F.NVFP4: (5e-3, 1e-3)}  # (scales, coefficients)
VARIANTS = ("rtn", "scale", "crs", "crs_dgs")
EPOCH_STEPS = 39  # 1,248 samples / batch 32
EVAL_STEP = 1_000_000  # batch index of the held-out evaluation batch


@dataclass
class Hyper:
    lr_s: float
    lr_c: float
    betas: tuple = (0.9, 0.999)
    eps: float = 1e-8
    weight_decay: float = 0.0
    log2_scales: bool = True
    log2_coeffs: bool = True


def variant_setup(w: synth.Workload, variant: str) -> tuple[int, bool, bool, bool]:
    """-> (sub_block, learn_scales, learn_c, use_c)."""
    if variant == "rtn":
        return w.sub_block, False, False, False
    if variant == "scale":
        return w.sub_block, True, False, False
    if variant == "crs":
        return w.block, True, True, True
    if variant == "crs_dgs":
        return w.sub_block, True, True, True
    raise ValueError(f"unknown variant {variant!r}")


class LayerState:
    """Frozen weights, learnable parameters and AdamW moments of one linear."""

    def __init__(self, W: torch.Tensor, fmt: int, sub_block: int, ws: torch.Tensor):
        self.W = W
        self.s, self.c, self.alpha = F.scales_init(W, fmt, sub_block, ws=ws)
        self.ms, self.vs = torch.zeros_like(self.s), torch.zeros_like(self.s)
        self.mc, self.vc = torch.zeros_like(self.c), torch.zeros_like(self.c)


class BlockCalibrator:
    """Holds a block's layers and runs steps of one variant on the current stream."""

    def __init__(self, w: synth.Workload, variant: str, hyper: Hyper | None = None, device="cuda",
                 max_tokens: int | None = None):
        self.w, self.variant, self.device = w, variant, device
        self.sb, self.learn_s, self.learn_c, self.use_c = variant_setup(w, variant)
        lr_s, lr_c = LEARNING_RATES[w.fmt]
        self.hyper = hyper or Hyper(lr_s, lr_c)
        q = F.qconfig(w.fmt, self.sb)
        M = max(w.M, max_tokens or 0)
        self.ws = F.workspace(max(F.workspace_size(F.CALL_FAKEQUANT_FWD, q),
                                  max(F.workspace_size(F.CALL_RECON_GEMM_BWD, q, M, l.N, l.K) for l in w.linears),
                                  max(F.workspace_size(F.CALL_RECON_GEMM_FWD, q, M, l.N, l.K) for l in w.linears)),
                              device)
        self.layers = {l.name: LayerState(synth.weight(w, l, device=device), w.fmt, self.sb, self.ws)
                       for l in w.linears}
        self.t = 0

    def _c(self, L: LayerState):
        return L.c if self.use_c else None

    def layer_step(self, L: LayerState, x_hat: torch.Tensor, X: torch.Tensor, learn: bool,
                   Y_ref: torch.Tensor | None = None) -> torch.Tensor:
        """Forward (+ backward and AdamW when `learn`) of one linear on one batch -> loss (device fp64).
        Y_ref defaults to the unquantised layer's output X W^T (the GEMM's plain-product mode)."""
        w, ws = self.w, self.ws
        if Y_ref is None:
            Y_ref, _, _ = F.recon_gemm_fwd(X, L.W, None, ws=ws)
        w_hat, _, _, _ = F.fakequant_fwd(L.W, w.fmt, self.sb, L.s, self._c(L), L.alpha, ws=ws)
        dY, loss, _ = F.recon_gemm_fwd(x_hat, w_hat, Y_ref, ws=ws)
        if learn:
            gs, gc, _ = F.recon_gemm_bwd(dY, x_hat, L.W, w.fmt, self.sb, L.s, self._c(L), L.alpha, ws=ws)
            h = self.hyper
            if self.learn_s:
                F.adamw_step(L.s, gs, L.ms, L.vs, self.t, h.lr_s, h.betas, h.eps, h.weight_decay, h.log2_scales, ws)
            if self.learn_c:
                F.adamw_step(L.c, gc, L.mc, L.vc, self.t, h.lr_c, h.betas, h.eps, h.weight_decay, h.log2_coeffs, ws)
        return loss

    def run_batch(self, batch: int, M: int, learn: bool) -> dict:
        """One pass over the block on batch `batch` -> {layer: loss}."""
        w = self.w
        if learn:
            self.t += 1
        acts = {src: synth.activation_batch(w, src, batch, M, device=self.device) for src in w.inputs}
        x_hat = {src: F.fakequant_fwd(x, w.fmt, self.sb, ws=self.ws)[0] for src, x in acts.items()}
        losses = {l.name: self.layer_step(self.layers[l.name], x_hat[l.source], acts[l.source], learn)
                  for l in w.linears}
        return {k: float(v.item()) for k, v in losses.items()}

    def check_domain(self) -> None:
        st = F.check_flags(self.ws)
        if st != F.OK:
            raise F.FocusError(st, f"calibration ({self.variant})")


def calibrate(w: synth.Workload, variant: str, steps: int = EPOCH_STEPS, M: int | None = None,
              eval_M: int | None = None, hyper: Hyper | None = None, device="cuda") -> dict:
    """One epoch of `steps` batches -> held-out losses per layer before and after, the training curve."""
    M = M or w.M
    eval_M = eval_M or M
    cal = BlockCalibrator(w, variant, hyper, device, max_tokens=max(M, eval_M))
    before = cal.run_batch(EVAL_STEP, eval_M, learn=False)
    curve = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    learn = variant != "rtn"
    for b in range(steps if learn else 0):
        losses = cal.run_batch(b, M, learn=True)
        curve.append(sum(losses.values()) / len(losses))
    torch.cuda.synchronize()
    seconds = time.perf_counter() - t0
    after = cal.run_batch(EVAL_STEP, eval_M, learn=False)
    cal.check_domain()
    return {"variant": variant, "steps": steps if learn else 0, "tokens_per_step": M, "eval_tokens": eval_M,
            "seconds": seconds, "eval_before": before, "eval_after": after, "train_curve": curve,
            "params": {name: {"s": L.s, "c": L.c} for name, L in cal.layers.items()}}


def ablation(w: synth.Workload, steps: int = EPOCH_STEPS, M: int | None = None, eval_M: int | None = None,
             variants=VARIANTS, device="cuda") -> dict:
    """Held-out reconstruction MSE of every variant, per layer and relative to RTN."""
    out = {}
    for v in variants:
        r = calibrate(w, v, steps, M, eval_M, device=device)
        r.pop("params")
        out[v] = r
    rtn = out["rtn"]["eval_after"] if "rtn" in out else None
    for v, r in out.items():
        if rtn:
            r["rel_to_rtn"] = {k: r["eval_after"][k] / rtn[k] for k in rtn}
            r["block_rel_to_rtn"] = sum(r["rel_to_rtn"].values()) / len(r["rel_to_rtn"])
    return out


class KLTopStack:
    """A synthetic two-linear stack trained end to end on KL-Top (Sec. 4.1; f1 of the hot path's
    extensions): X0 [M][h] -> "up" (h -> h) -> "head" (h -> V) -> logits. The teacher is the same
    stack unquantised; the student quantises every activation and weight. One training step:

        forward:  X0_hat, W_up_hat -> Y1 -> Y1_hat, W_head_hat -> Z     (plain-product GEMMs)
        loss:     KL-Top(Z, Z_teacher), dZ
        backward: head: grad_s, grad_c from dZ (fused straight-through epilogue);
                  dY1 = STE_act(Y1, dZ W_head_hat); up: grad_s, grad_c from dY1
        update:   AdamW on both layers' S_fp and c (log2 domain)

    Every arithmetic step runs in libfocus."""

    def __init__(self, fmt: int, variant: str, hidden: int = 2560, vocab: int = 32000, tokens: int = 4096,
                 k: int = 1000, x_kind: str = "lowrank", hyper: Hyper | None = None, device="cuda"):
        from .synth import Linear, Workload
        self.w = Workload(name=f"klstack{hidden}x{vocab}", fmt=fmt, sub_block=8, M=tokens,
                          linears=(Linear("up", hidden, hidden, "x"), Linear("head", vocab, hidden, "y")),
                          inputs={"x": hidden, "y": hidden}, x_kind=x_kind, x_outlier_p=0.01, x_outlier_f=30.0)
        self.variant, self.k, self.device = variant, k, device
        self.sb, self.learn_s, self.learn_c, self.use_c = variant_setup(self.w, variant)
        lr_s, lr_c = LEARNING_RATES[fmt]
        self.hyper = hyper or Hyper(lr_s, lr_c)
        q = F.qconfig(fmt, self.sb)
        M = tokens
        self.ws = F.workspace(max(F.workspace_size(F.CALL_FAKEQUANT_FWD, q),
                                  max(F.workspace_size(F.CALL_RECON_GEMM_BWD, q, M, l.N, l.K) for l in self.w.linears),
                                  max(F.workspace_size(F.CALL_RECON_GEMM_FWD, q, M, l.N, l.K) for l in self.w.linears),
                                  F.workspace_size(F.CALL_RECON_GEMM_DX, q, M, vocab, hidden),
                                  F.workspace_size(F.CALL_KL_TOP, q, M, vocab, 0)), device)
        self.layers = {l.name: LayerState(synth.weight(self.w, l, device=device), fmt, self.sb, self.ws)
                       for l in self.w.linears}
        self.t = 0

    def _c(self, L):
        return L.c if self.use_c else None

    def _update(self, L, gs, gc):
        h = self.hyper
        if self.learn_s:
            F.adamw_step(L.s, gs, L.ms, L.vs, self.t, h.lr_s, h.betas, h.eps, h.weight_decay, h.log2_scales, self.ws)
        if self.learn_c:
            F.adamw_step(L.c, gc, L.mc, L.vc, self.t, h.lr_c, h.betas, h.eps, h.weight_decay, h.log2_coeffs, self.ws)

    def run_batch(self, batch: int, learn: bool) -> float:
        """KL-Top loss of the stack on batch `batch` (and one training step when `learn`)."""
        fmt, sb, ws, w = self.w.fmt, self.sb, self.ws, self.w
        up, head = self.layers["up"], self.layers["head"]
        X0 = synth.activation_batch(w, "x", batch, w.M, device=self.device)
        Zt = F.recon_gemm_fwd(F.recon_gemm_fwd(X0, up.W, None, ws=ws)[0], head.W, None, ws=ws)[0]
        x0h = F.fakequant_fwd(X0, fmt, sb, ws=ws)[0]
        w_up = F.fakequant_fwd(up.W, fmt, sb, up.s, self._c(up), up.alpha, ws=ws)[0]
        Y1 = F.recon_gemm_fwd(x0h, w_up, None, ws=ws)[0]
        y1h = F.fakequant_fwd(Y1, fmt, sb, ws=ws)[0]
        w_head = F.fakequant_fwd(head.W, fmt, sb, head.s, self._c(head), head.alpha, ws=ws)[0]
        Z = F.recon_gemm_fwd(y1h, w_head, None, ws=ws)[0]
        dZ, loss = F.kl_top(Z, Zt, self.k, ws=ws)
        if learn:
            self.t += 1
            gs2, gc2, _ = F.recon_gemm_bwd(dZ, y1h, head.W, fmt, sb, head.s, self._c(head), head.alpha, ws=ws)
            dY1 = F.fakequant_act_bwd(Y1, F.recon_gemm_dx(dZ, w_head, ws=ws), fmt, ws=ws)
            gs1, gc1, _ = F.recon_gemm_bwd(dY1, x0h, up.W, fmt, sb, up.s, self._c(up), up.alpha, ws=ws)
            self._update(head, gs2, gc2)
            self._update(up, gs1, gc1)
        return float(loss.item())


def kl_top_epoch(fmt: int, variant: str, steps: int = EPOCH_STEPS, **kw) -> dict:
    """One epoch of the KL-Top stack -> held-out KL-Top before and after, and the training curve."""
    stack = KLTopStack(fmt, variant, **kw)
    before = stack.run_batch(EVAL_STEP, learn=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    curve = [stack.run_batch(b, learn=True) for b in range(steps if variant != "rtn" else 0)]
    torch.cuda.synchronize()
    seconds = time.perf_counter() - t0
    after = stack.run_batch(EVAL_STEP, learn=False)
    st = F.check_flags(stack.ws)
    if st != F.OK:
        raise F.FocusError(st, f"KL-Top stack ({variant})")
    return {"variant": variant, "eval_before": before, "eval_after": after, "train_curve": curve, "seconds": seconds}


def main() -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="block2560_mxfp4", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--steps", type=int, default=EPOCH_STEPS)
    ap.add_argument("--tokens", type=int, default=None, help="tokens per step (default: the workload's)")
    ap.add_argument("--eval-tokens", type=int, default=None)
    ap.add_argument("--variants", default=",".join(VARIANTS))
    ap.add_argument("--x-kind", default=None, choices=("normal", "student_t3", "lowrank"),
                    help="activation distribution (default: the workload's)")
    ap.add_argument("--kl-top-stack", action="store_true",
                    help="train the synthetic two-linear stack end to end on KL-Top instead")
    ap.add_argument("--vocab", type=int, default=32000)
    a = ap.parse_args()
    if not torch.cuda.is_available():
        raise SystemExit("the calibration epoch runs on the GPU")
    w = synth.WORKLOADS[a.workload]
    if a.kl_top_stack:
        hidden = w.inputs[w.linears[0].source]
        out = {"stack": f"hidden {hidden} -> {hidden} -> vocab {a.vocab}", "x_kind": a.x_kind or "lowrank",
               "steps": a.steps, "tokens_per_step": a.tokens or 4096, "results": {}}
        for v in a.variants.split(","):
            r = kl_top_epoch(w.fmt, v, a.steps, hidden=hidden, vocab=a.vocab, tokens=a.tokens or 4096,
                             x_kind=a.x_kind or "lowrank")
            out["results"][v] = {"eval_before": r["eval_before"], "eval_after": r["eval_after"],
                                 "seconds": round(r["seconds"], 3), "train_first_last": r["train_curve"][:1] + r["train_curve"][-1:]}
        print(json.dumps(out))
        return
    if a.x_kind:
        w = dataclasses.replace(w, x_kind=a.x_kind)
    res = ablation(w, a.steps, a.tokens, a.eval_tokens, tuple(a.variants.split(",")))
    summary = {"workload": a.workload, "x_kind": w.x_kind, "steps": a.steps, "tokens_per_step": a.tokens or w.M,
               "results": {v: {"block_rel_to_rtn": r.get("block_rel_to_rtn"), "seconds": round(r["seconds"], 3),
                               "rel_to_rtn": {k: round(x, 4) for k, x in r.get("rel_to_rtn", {}).items()},
                               "eval_after": r["eval_after"],
                               "train_first_last": (r["train_curve"][:1] + r["train_curve"][-1:])}
                           for v, r in res.items()}}
    print(json.dumps(summary))


if __name__ == "__main__":
    main()
