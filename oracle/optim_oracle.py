"""CPU oracle for the optimizer and the calibration step -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this module; the HIP
library and its Python binding never do, and the two share no code.

Paper passages followed (FOCUS, arXiv 2608.01847):
  * Sec. 4.1: AdamW with a constant learning rate; MXFP4 learning rates 2e-2 (block scales) and
    5e-2 (coefficients c), NVFP4 5e-3 and 1e-3; one epoch over the calibration batches.
  * Sec. 3.2-3.4 (Eq. 4-8): the scale-learning step itself, taken from focus_oracle.
AdamW is written as Loshchilov & Hutter state it (decoupled weight decay, bias-corrected first and
second moments m_hat = m / (1 - beta1^t), v_hat = v / (1 - beta2^t)), in float64. The paper does not
give beta1, beta2, eps or the weight decay; the defaults below are the common AdamW defaults, with
no weight decay. The block scales and the coefficients may be stepped in the log2 domain
(theta = log2 p): the paper does not say in which domain they are learned, an absolute step of 2e-2
on a linear scale of about 1e-2 could not be what it describes, and a linear-domain c stepped at 5e-2
can run through zero.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import focus_oracle as O


def adamw(p, g, m, v, t: int, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
          weight_decay: float = 0.0, log2_domain: bool = False):
    """One AdamW step -> (p_new, m_new, v_new), float64. In the log2 domain the moments belong to
    theta = log2(p) and the gradient is carried over by the chain rule, dL/dtheta = dL/dp * p * ln 2."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    if log2_domain:
        theta = np.log2(p)
        g = g * p * np.log(2.0)
    else:
        theta = p
    theta = theta - lr * weight_decay * theta
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    theta = theta - lr * m_hat / (np.sqrt(v_hat) + eps)
    return (np.exp2(theta) if log2_domain else theta), m, v


@dataclass
class LayerParams:
    """Learnable state of one linear, stored in fp32 as the library stores it."""
    s: np.ndarray
    c: np.ndarray
    alpha: float
    ms: np.ndarray
    vs: np.ndarray
    mc: np.ndarray
    vc: np.ndarray

    @staticmethod
    def init(W, fmt: int, sb: int) -> "LayerParams":
        s, c, alpha = O.init_scales(W, fmt, sb)
        z = np.zeros_like
        return LayerParams(s, c, alpha, z(s), z(s), z(c), z(c))


def calib_step(X, W, Y_ref, fmt: int, sb: int, P: LayerParams, t: int, lr_s: float, lr_c: float,
               learn_s: bool, learn_c: bool, use_c: bool, bf16: bool, log2_scales: bool = True,
               betas=(0.9, 0.999), eps: float = 1e-8, weight_decay: float = 0.0, log2_coeffs: bool = True):
    """One scale-learning step of one linear followed by AdamW -> (loss, new LayerParams).

    X [M][K], W [N][K], Y_ref [M][N] as fp32 arrays of the values the library sees; bf16 operands
    are rounded to bf16 after fake quantisation, as the GEMM consumes them."""
    x_hat = O.fq_act(X, fmt)[0]
    fq = O.fq_weight(W, fmt, sb, P.s, P.c if use_c else None, P.alpha)
    X_op = O.bf16_round(x_hat) if bf16 else x_hat
    W_op = O.bf16_round(fq.w_hat) if bf16 else fq.w_hat
    res = O.recon_layer(X_op, W_op, np.asarray(Y_ref, np.float64), fq, fmt, sb, P.alpha)
    s, ms, vs, c, mc, vc = P.s, P.ms, P.vs, P.c, P.mc, P.vc
    f32 = lambda a: np.asarray(a, np.float64).astype(np.float32)
    if learn_s:
        s, ms, vs = map(f32, adamw(P.s, res.grad_s, P.ms, P.vs, t, lr_s, betas[0], betas[1], eps, weight_decay,
                                   log2_scales))
    if learn_c:
        c, mc, vc = map(f32, adamw(P.c, res.grad_c, P.mc, P.vc, t, lr_c, betas[0], betas[1], eps, weight_decay,
                                   log2_coeffs))
    return res.loss_part, LayerParams(s, c, P.alpha, ms, vs, mc, vc), res
