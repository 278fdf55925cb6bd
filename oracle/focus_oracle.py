"""CPU oracle for the FOCUS scale-learning step -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this module; the
HIP library and its Python binding never do, and the two share no code. The element and block
codecs and the fake quantisation are plain C loops in ``focus_oracle.c`` (built with gcc, no fast
math, no FMA contraction); the reconstruction GEMM, the MSE loss and the straight-through
gradients are written here in float64 with numpy, using a BLAS matmul only as the matrix product.

Paper (FOCUS, arXiv 2608.01847) passages followed:
  * Sec. 3.1, Eq. (1)-(3): E2M1 elements, NVFP4 two-level scales, MXFP4 E8M0 scales.
  * Sec. 3.2, Eq. (4)-(5): learnable full-precision scale copies quantised on the fly, STE applied
    to every non-differentiable operation, alpha frozen for NVFP4.
  * Sec. 3.3, Eq. (6)-(7): Coupled-Relaxation Scaling, S_q = S_dq * c.
  * Sec. 3.4, Eq. (8): Dual-Granularity Scaling, one coefficient per sub-block of 8.
  * Sec. 4.1: weights and activations of every linear layer quantised; activations dynamic.
The per-layer objective is the mean squared error between the quantised layer output and the
full-precision output, L = sum((Y_hat - Y_ref)^2) / (M * N).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from pathlib import Path

import numpy as np

ORACLE_DIR = Path(__file__).resolve().parent
SOURCE = ORACLE_DIR / "focus_oracle.c"
LIBRARY = ORACLE_DIR / "liboracle.so"

MXFP4 = 0
NVFP4 = 1


def block_size(fmt: int) -> int:
    """Hardware block size: 32 for MXFP4 (Eq. 3), 16 for NVFP4 (Eq. 2)."""
    return 32 if fmt == MXFP4 else 16


def build(force: bool = True) -> Path:
    """Compile the C half of the oracle with gcc."""
    if force or not LIBRARY.exists():
        tmp = LIBRARY.with_suffix(".so.tmp")
        cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-std=c11",
               "-shared", "-fPIC", str(SOURCE), "-o", str(tmp), "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIBRARY)
    return LIBRARY


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not LIBRARY.exists():
            build(force=False)
        lib = ctypes.CDLL(str(LIBRARY))
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        i32 = ctypes.c_int
        f32 = ctypes.c_float
        lib.oracle_e2m1_array.argtypes = [p, i64, p, p]
        lib.oracle_e2m1_decode_array.argtypes = [p, i64, p]
        lib.oracle_e8m0_ceil_array.argtypes = [p, i64, p]
        lib.oracle_e4m3_array.argtypes = [p, i64, p]
        lib.oracle_e4m3_decode_array.argtypes = [p, i64, p]
        lib.oracle_bf16_round_array.argtypes = [p, i64, p]
        lib.oracle_init_scales.argtypes = [i32, i32, i32, p, i64, i64, p, p, p]
        lib.oracle_fq_weight.argtypes = [i32, i32, i32, i32, p, i64, i64, p, p, f32, p, p, p, p, p, p, p]
        lib.oracle_fq_act.argtypes = [i32, i32, p, i64, i64, p, p, p, p]
        lib.oracle_e8m0_floor_array.argtypes = [p, i64, p]
        lib.oracle_pack_codes.argtypes = [p, i64, i64, p]
        lib.oracle_unpack_codes.argtypes = [p, i64, i64, p]
        lib.oracle_decode_packed.argtypes = [i32, p, p, f32, i64, i64, p]
        for name in ("oracle_e8m0_ceil_array", "oracle_e8m0_floor_array", "oracle_e4m3_array", "oracle_init_scales",
                     "oracle_fq_weight", "oracle_fq_act"):
            getattr(lib, name).restype = ctypes.c_int
        _LIB = lib
    return _LIB


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


# ---------------------------------------------------------------------------------------------
# Codecs (Sec. 3.1)
# ---------------------------------------------------------------------------------------------

def e2m1(u) -> tuple[np.ndarray, np.ndarray]:
    """Q_E2M1 (Eq. 1): nearest E2M1 value, ties to the even code, saturating at 6. -> (value, code)."""
    u = _f32(u)
    q = np.empty_like(u)
    code = np.empty(u.shape, np.uint8)
    _lib().oracle_e2m1_array(_ptr(u), u.size, _ptr(q), _ptr(code))
    return q, code


def e2m1_decode(code) -> np.ndarray:
    code = np.ascontiguousarray(code, dtype=np.uint8)
    v = np.empty(code.shape, np.float32)
    _lib().oracle_e2m1_decode_array(_ptr(code), code.size, _ptr(v))
    return v


def e8m0_floor(s) -> np.ndarray:
    """Q_E8M0 rounded down (the OCP MX rule): the byte e + 127 of the largest 2^e <= s."""
    s = _f32(s)
    out = np.empty(s.shape, np.uint8)
    _lib().oracle_e8m0_floor_array(_ptr(s), s.size, _ptr(out))
    return out


def e8m0_ceil(s) -> np.ndarray:
    """Q_E8M0 with the ceiling reading of Eq. (3): the byte e + 127 of the smallest 2^e >= s."""
    s = _f32(s)
    out = np.empty(s.shape, np.uint8)
    _lib().oracle_e8m0_ceil_array(_ptr(s), s.size, _ptr(out))
    return out


def e4m3(x) -> np.ndarray:
    """Q_E4M3 (Eq. 2): nearest OCP E4M3FN code, ties to even, saturating at 448, x <= 0 -> 0."""
    x = _f32(x)
    out = np.empty(x.shape, np.uint8)
    _lib().oracle_e4m3_array(_ptr(x), x.size, _ptr(out))
    return out


def e4m3_decode(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint8)
    v = np.empty(b.shape, np.float32)
    _lib().oracle_e4m3_decode_array(_ptr(b), b.size, _ptr(v))
    return v


def bf16_round(x) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 (ties to even); returned as fp32."""
    x = _f32(x)
    y = np.empty_like(x)
    _lib().oracle_bf16_round_array(_ptr(x), x.size, _ptr(y))
    return y


def bf16_bits(x_bf16_valued: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are already bfloat16-representable."""
    return (np.ascontiguousarray(x_bf16_valued, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    return (np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------------------------
# Scale initialisation and fake quantisation
# ---------------------------------------------------------------------------------------------

def init_scales(W, fmt: int, sb: int, e8m0_floor: bool = False):
    """Absmax initialisation (Sec. 3.2) -> (s_fp [N][K/B], c [N][K/sb] = 1, alpha)."""
    W = _f32(W)
    N, K = W.shape
    B = block_size(fmt)
    s_fp = np.empty((N, K // B), np.float32)
    c = np.empty((N, K // sb), np.float32)
    alpha = np.ones(1, np.float32)
    _lib().oracle_init_scales(fmt, sb, int(e8m0_floor), _ptr(W), N, K, _ptr(s_fp), _ptr(c), _ptr(alpha))
    return s_fp, c, float(alpha[0])


@dataclass
class WeightFQ:
    """Everything the forward produces for one weight tensor (Eq. 4, 6-8)."""
    w_hat: np.ndarray        # fp32 [N][K] dequantised weights
    codes: np.ndarray        # uint8 [N][K] 4-bit codes, one per element
    scale_bytes: np.ndarray  # uint8 [N][K/B] E8M0 or E4M3 bytes of S_dq
    u: np.ndarray            # fp32 [N][K] w / S_q
    m: np.ndarray            # uint8 [N][K] straight-through clamp mask [|u| <= 6]
    s_dq: np.ndarray         # fp32 [N][K/B]
    s_q: np.ndarray          # fp32 [N][K/sb]
    domain_error: int
    w: np.ndarray            # fp32 [N][K] the (frozen) input weights
    c: np.ndarray | None     # fp32 [N][K/sb] the coefficients used (None means all ones)


def fq_weight(W, fmt: int, sb: int, s_fp, c, alpha: float = 1.0, ste_clip: bool = True,
              e8m0_floor: bool = False) -> WeightFQ:
    W = _f32(W)
    N, K = W.shape
    B = block_size(fmt)
    s_fp = _f32(s_fp)
    c = None if c is None else _f32(c)
    out = WeightFQ(np.empty((N, K), np.float32), np.empty((N, K), np.uint8),
                   np.empty((N, K // B), np.uint8), np.empty((N, K), np.float32),
                   np.empty((N, K), np.uint8), np.empty((N, K // B), np.float32),
                   np.empty((N, K // sb), np.float32), 0, W, c)
    out.domain_error = _lib().oracle_fq_weight(
        fmt, sb, int(ste_clip), int(e8m0_floor), _ptr(W), N, K, _ptr(s_fp), _ptr(c), float(alpha),
        _ptr(out.w_hat), _ptr(out.codes), _ptr(out.scale_bytes), _ptr(out.u), _ptr(out.m),
        _ptr(out.s_dq), _ptr(out.s_q))
    return out


def fq_act(X, fmt: int, e8m0_floor: bool = False):
    """Dynamic activation fake quantisation -> (x_hat fp32, codes, scale_bytes, alpha)."""
    X = _f32(X)
    M, K = X.shape
    B = block_size(fmt)
    x_hat = np.empty_like(X)
    codes = np.empty((M, K), np.uint8)
    sb = np.empty((M, K // B), np.uint8)
    alpha = np.ones(1, np.float32)
    _lib().oracle_fq_act(fmt, int(e8m0_floor), _ptr(X), M, K, _ptr(x_hat), _ptr(codes), _ptr(sb), _ptr(alpha))
    return x_hat, codes, sb, float(alpha[0])


def pack_codes(codes) -> np.ndarray:
    """Export layout (Fig. 3(d)): two codes per byte, even k in the low nibble."""
    codes = np.ascontiguousarray(codes, np.uint8)
    N, K = codes.shape
    packed = np.empty((N, K // 2), np.uint8)
    _lib().oracle_pack_codes(_ptr(codes), N, K, _ptr(packed))
    return packed


def unpack_codes(packed) -> np.ndarray:
    packed = np.ascontiguousarray(packed, np.uint8)
    N, K2 = packed.shape
    codes = np.empty((N, 2 * K2), np.uint8)
    _lib().oracle_unpack_codes(_ptr(packed), N, 2 * K2, _ptr(codes))
    return codes


def decode_packed(fmt: int, packed, scale_bytes, alpha: float = 1.0) -> np.ndarray:
    packed = np.ascontiguousarray(packed, np.uint8)
    scale_bytes = np.ascontiguousarray(scale_bytes, np.uint8)
    N, K2 = packed.shape
    out = np.empty((N, 2 * K2), np.float32)
    _lib().oracle_decode_packed(fmt, _ptr(packed), _ptr(scale_bytes), float(alpha), N, 2 * K2,
                                _ptr(out))
    return out


# ---------------------------------------------------------------------------------------------
# Reconstruction GEMM, MSE loss and straight-through gradients (float64)
# ---------------------------------------------------------------------------------------------

def gemm_operand(values_fp32: np.ndarray, bf16: bool) -> np.ndarray:
    """The GEMM operand: the fake-quantised tensor, rounded to bfloat16 on the bf16 path."""
    return bf16_round(values_fp32) if bf16 else _f32(values_fp32)


@dataclass
class LayerResult:
    rows: np.ndarray       # output features n the results below are for
    col_sq: np.ndarray     # float64 [|rows|]: sum over tokens of (Y_hat - Y_ref)^2
    d_y: np.ndarray | None  # float64 [M][|rows|]: dL/dY_hat = 2 (Y_hat - Y_ref) / (M N), if kept
    G: np.ndarray          # float64 [|rows|][K]: dL/dW_hat = D^T X_op
    grad_s: np.ndarray     # float64 [|rows|][K/B]
    grad_c: np.ndarray     # float64 [|rows|][K/sb]
    loss_part: float       # sum(col_sq) / (M N); the full loss when rows covers every n


def recon_layer(X_op: np.ndarray, W_op: np.ndarray, Y_ref, fq: WeightFQ, fmt: int,
                sb: int, alpha: float = 1.0, rows=None, keep_dy: bool = False,
                chunk: int = 8192, y_ref_cols: np.ndarray | None = None) -> LayerResult:
    """One layer of the scale-learning step, computed for the output features ``rows``.

    X_op [M][K] and W_op [N][K] are the GEMM operands (fp32 arrays holding the exact operand
    values); Y_ref [M][N] is the full-precision reference output. Forward Y_hat = X_op W_op^T
    and the loss are in float64. Backward (STE, Sec. 3.2, through Eq. 6-8):
        G_j         = sum_t D[t, n] X_op[t, j]                         (dL/dW_hat)
        dW_hat/dc   = -m_j w_j / c^2                                   (Q_E2M1 -> identity in [-6, 6])
        dW_hat/dS_dq = q_j - m_j w_j / S_q                             (S_dq appears in S_q and in W_hat)
        grad_c[k]   = sum over sub-block k of G_j dW_hat/dc
        grad_S_dq   = sum over the block of G_j dW_hat/dS_dq
        grad S_fp   = grad_S_dq (MXFP4, STE through Q_E8M0); alpha * grad_S_dq (NVFP4, Delta_fp)
    Loss and gradients for output feature n depend only on row n of W and column n of Y_ref, so a
    subset of rows is exact for those rows. `y_ref_cols` may carry Y_ref already restricted to the
    columns `rows` ([M][|rows|]); Y_ref is then not used.
    """
    M, K = X_op.shape
    N = W_op.shape[0]
    B = block_size(fmt)
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    R = len(rows)
    WR = W_op[rows].astype(np.float64)
    scale = 2.0 / (M * N)
    col_sq = np.zeros(R, np.float64)
    G = np.zeros((R, K), np.float64)
    d_y = np.empty((M, R), np.float64) if keep_dy else None
    for t0 in range(0, M, chunk):
        Xc = X_op[t0:t0 + chunk].astype(np.float64)
        Yc = Xc @ WR.T
        Yr = y_ref_cols[t0:t0 + chunk] if y_ref_cols is not None else Y_ref[t0:t0 + chunk][:, rows]
        Dc = Yc - Yr.astype(np.float64)
        col_sq += (Dc * Dc).sum(axis=0)
        Dc *= scale
        if keep_dy:
            d_y[t0:t0 + chunk] = Dc
        G += Dc.T @ Xc

    return _ste_gradients(rows, col_sq, d_y, G, fq, fmt, sb, alpha, M, N)


def ste_gradients_from_G(G: np.ndarray, fq: WeightFQ, fmt: int, sb: int, alpha: float = 1.0,
                         rows=None):
    """grad_s, grad_c (float64) from a given dL/dW_hat G [|rows|][K] (the unfused backward)."""
    N, K = fq.w.shape
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    B = block_size(fmt)
    R = len(rows)
    w = fq.w[rows].astype(np.float64)
    m = fq.m[rows].astype(np.float64)
    q = e2m1_decode(fq.codes[rows]).astype(np.float64)  # the signed E2M1 value Q(u)
    c = (np.ones((R, K // sb)) if fq.c is None else fq.c[rows].astype(np.float64))
    s_q = fq.s_q[rows].astype(np.float64).repeat(sb, axis=1)
    live = s_q != 0
    w_over_sq = np.where(live, w / np.where(live, s_q, 1.0), 0.0)
    # d W_hat / d c_k = -m w / c^2 ;  d W_hat / d S_dq = q - m w / S_q
    grad_c = -(G * m * w).reshape(R, K // sb, sb).sum(axis=2) / (c * c)
    grad_s = (G * (q - m * w_over_sq)).reshape(R, K // B, B).sum(axis=2)
    dead = (fq.s_dq[rows] == 0)
    grad_s[dead] = 0.0
    grad_c[np.repeat(dead, B // sb, axis=1)] = 0.0
    if fmt == NVFP4:
        grad_s = grad_s * alpha  # S_dq = alpha * Q_E4M3(Delta_fp), alpha frozen
    return grad_s, grad_c


def _ste_gradients(rows, col_sq, d_y, G, fq, fmt, sb, alpha, M, N) -> LayerResult:
    grad_s, grad_c = ste_gradients_from_G(G, fq, fmt, sb, alpha, rows)
    return LayerResult(rows=rows, col_sq=col_sq, d_y=d_y, G=G, grad_s=grad_s, grad_c=grad_c,
                       loss_part=float(col_sq.sum() / (M * N)))
