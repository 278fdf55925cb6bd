"""CPU oracle for end-to-end chaining -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this module; the HIP
library and its Python binding never do, and the two share no code.

Paper passages followed (FOCUS, arXiv 2608.01847):
  * Sec. 4.1: the model is trained end to end with the KL-Top loss, k = 1000 (the loss of the
    method the paper cites for it): the KL divergence between the full-precision model's and the
    quantised model's output distributions, restricted to the full-precision model's k largest
    logits. The paper gives no formula; the reading here: per token, I = the teacher's top-k
    indices (ties at the k-th value in increasing index order), both distributions renormalised over
    I by a softmax of the logits there, KL(p_teacher || p_student), averaged over tokens.
  * Sec. 3.2: straight-through estimation through every non-differentiable operation, here the
    activation fake quantisation: the gradient passes where the clamp does not act (|x / S| <= 6),
    and not through the absmax scale.
A linear layer's input gradient is the plain product dX_hat = dY W_hat (float64).
"""
from __future__ import annotations

import numpy as np

from . import focus_oracle as O


def kl_top(Zs, Zt, k: int):
    """-> (loss, dZs) in float64: loss = mean over rows of KL(p_t || p_s) on the teacher's top-k."""
    Zs = np.asarray(Zs, np.float64)
    Zt = np.asarray(Zt, np.float64)
    T, V = Zs.shape
    loss = 0.0
    dZ = np.zeros_like(Zs)
    for r in range(T):
        order = np.argsort(-Zt[r], kind="stable")  # largest first, equal values by index
        idx = order[:min(k, V)]
        a, b = Zt[r, idx], Zs[r, idx]
        lpt = a - (a.max() + np.log(np.sum(np.exp(a - a.max()))))
        lps = b - (b.max() + np.log(np.sum(np.exp(b - b.max()))))
        pt, ps = np.exp(lpt), np.exp(lps)
        loss += float(np.sum(pt * (lpt - lps)))
        dZ[r, idx] = (ps - pt) / T
    return loss / T, dZ


def recon_dx(dY, W_hat):
    """dX_hat = dY W_hat (the input gradient of Y_hat = X_hat W_hat^T)."""
    return np.asarray(dY, np.float64) @ np.asarray(W_hat, np.float64)


def act_ste_mask(X, fmt: int, e8m0_floor: bool = False, ste_clip: bool = True) -> np.ndarray:
    """Straight-through mask of the activation fake quantisation: [|x / S| <= 6] with S the block
    scale the forward uses (0 where S is 0; all ones without the clamp except zero-scale blocks)."""
    X = np.asarray(X, np.float32)
    M, K = X.shape
    B = O.block_size(fmt)
    _, _, sbytes, alpha = O.fq_act(X, fmt, e8m0_floor=e8m0_floor)
    if fmt == 0:
        S = np.ldexp(np.float32(1.0), sbytes.astype(np.int64) - 127).astype(np.float32)
    else:
        S = (np.float32(alpha) * O.e4m3_decode(sbytes).astype(np.float32)).astype(np.float32)
    Sx = np.repeat(S, B, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        u = (X / np.where(Sx == 0, np.float32(1), Sx)).astype(np.float32)
    m = (np.abs(u) <= 6.0) if ste_clip else np.ones_like(u, bool)
    return (m & (Sx != 0)).astype(np.float64)


def chain_layer_backward(X, W, Zt, fmt: int, sb: int, s_fp, c, alpha: float, k: int, bf16: bool,
                         e8m0_floor: bool = False):
    """The top layer of a stack trained on KL-Top: X [M][K] its input, W [N][K] its weight, Zt [M][N]
    the teacher logits. Forward: X_hat, W_hat fake-quantised, Z = X_hat W_hat^T (rounded to bf16 when
    the path is bf16, as the library writes it); KL-Top -> dZ (bf16-rounded likewise); backward:
    grad_s, grad_c through the fused straight-through epilogue of dZ^T X_hat, and dX = m * (dZ W_hat).
    -> dict(loss, dZ, grad_s, grad_c, dX)."""
    x_hat = O.fq_act(X, fmt, e8m0_floor=e8m0_floor)[0]
    fq = O.fq_weight(W, fmt, sb, s_fp, c, alpha, e8m0_floor=e8m0_floor)
    X_op = O.bf16_round(x_hat) if bf16 else x_hat
    W_op = O.bf16_round(fq.w_hat) if bf16 else fq.w_hat
    Z = X_op.astype(np.float64) @ W_op.astype(np.float64).T
    Z = O.bf16_round(Z.astype(np.float32)) if bf16 else Z
    loss, dZ = kl_top(Z, Zt, k)
    dZ_op = O.bf16_round(dZ.astype(np.float32)).astype(np.float64) if bf16 else dZ
    G = dZ_op.T @ X_op.astype(np.float64)
    grad_s, grad_c = O.ste_gradients_from_G(G, fq, fmt, sb, alpha)
    dX_hat = recon_dx(dZ_op, W_op)
    dX = act_ste_mask(X, fmt, e8m0_floor) * dX_hat
    return {"loss": loss, "dZ": dZ, "grad_s": grad_s, "grad_c": grad_c, "dX": dX}
