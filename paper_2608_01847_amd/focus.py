"""Thin ctypes binding of libfocus (include/focus.h) for torch tensors.

Argument marshalling only: every computation runs in the library's HIP kernels on the caller's
current torch stream. PyTorch provides device memory and streams. Importing this module loads
nothing; the first call opens libfocus.so and raises if it is not built.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

LIBRARY = Path(__file__).resolve().parent / "libfocus.so"

MXFP4, NVFP4 = 0, 1
F32, BF16 = 0, 1
CALL_SCALES_INIT, CALL_FAKEQUANT_FWD, CALL_FAKEQUANT_BWD = 0, 1, 2
CALL_RECON_GEMM_FWD, CALL_RECON_GEMM_BWD, CALL_EXPORT_PACKED, CALL_ADAMW = 3, 4, 5, 6
CALL_RECON_GEMM_DX, CALL_FAKEQUANT_ACT_BWD, CALL_KL_TOP, CALL_FAKEQUANT_WEIGHTS = 7, 8, 9, 10
MAX_WEIGHT_LAYERS = 16

OK, ERR_NULL, ERR_SHAPE, ERR_DTYPE, ERR_CONFIG, ERR_WORKSPACE, ERR_DOMAIN, ERR_HIP, ERR_SCRATCH = range(9)

EXPORTED = ("focus_workspace_size", "focus_scales_init", "focus_fakequant_fwd", "focus_fakequant_bwd",
            "focus_recon_gemm_fwd", "focus_recon_gemm_fwd_mxfp4", "focus_recon_gemm_fwd_mxfp4_noalloc",
            "focus_recon_gemm_bwd",
            "focus_recon_gemm_bwd_mxfp4", "focus_export_packed", "focus_fakequant_weights", "focus_recon_gemm_dx",
            "focus_fakequant_act_bwd", "focus_kl_top", "focus_adamw_step", "focus_check_flags", "focus_status_string")


class QConfig(ctypes.Structure):
    _fields_ = [("format", ctypes.c_int32), ("sub_block", ctypes.c_int32),
                ("ste_clip", ctypes.c_int32), ("scale_layout", ctypes.c_int32), ("e8m0_rounding", ctypes.c_int32),
                ("code_layout", ctypes.c_int32)]


class WeightLayer(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("rows", ctypes.c_int64), ("K", ctypes.c_int64),
                ("s_fp", ctypes.c_void_p), ("c", ctypes.c_void_p), ("alpha", ctypes.c_void_p),
                ("W_hat", ctypes.c_void_p), ("codes", ctypes.c_void_p), ("scale_bytes", ctypes.c_void_p)]


class AdamWConfig(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float), ("log2_domain", ctypes.c_int32)]


class FocusError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_LIB = None


def lib() -> ctypes.CDLL:
    """Opens libfocus.so (built by __graft_entry__.build()); raises if it is missing."""
    global _LIB
    if _LIB is None:
        if not LIBRARY.exists():
            raise RuntimeError(f"{LIBRARY} is not built: run __graft_entry__.build() first")
        L = ctypes.CDLL(str(LIBRARY))
        p, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
        q = ctypes.POINTER(QConfig)
        L.focus_workspace_size.argtypes = [i32, q, i64, i64, i64]
        L.focus_workspace_size.restype = sz
        L.focus_scales_init.argtypes = [q, p, i32, i64, i64, p, p, p, p, sz, p]
        L.focus_fakequant_fwd.argtypes = [q, p, i32, i64, i64, p, p, p, p, i32, p, p, p, p, sz, p]
        L.focus_fakequant_bwd.argtypes = [q, p, i64, i64, p, i32, p, p, p, p, p, p, sz, p]
        L.focus_recon_gemm_fwd.argtypes = [p, p, i32, i64, i64, i64, p, p, p, p, p, sz, p]
        L.focus_recon_gemm_fwd_mxfp4.argtypes = [p, p, p, p, i64, i64, i64, p, p, p, p, p, sz, p]
        L.focus_recon_gemm_fwd_mxfp4_noalloc.argtypes = [p, p, p, p, i64, i64, i64, p, p, p, p, p]
        L.focus_recon_gemm_bwd.argtypes = [q, p, p, i32, i64, i64, i64, p, i32, p, p, p, p, p, p, p, sz, p]
        L.focus_recon_gemm_bwd_mxfp4.argtypes = [q, p, p, p, i64, i64, i64, p, i32, p, p, p, p, p, sz, p]
        L.focus_export_packed.argtypes = [q, p, i32, i64, i64, p, p, p, p, p, p, sz, p]
        L.focus_fakequant_weights.argtypes = [q, i32, i32, ctypes.POINTER(WeightLayer), i32, p, sz, p]
        L.focus_recon_gemm_dx.argtypes = [p, p, i32, i64, i64, i64, p, p, sz, p]
        L.focus_fakequant_act_bwd.argtypes = [q, p, i32, i64, i64, p, i32, p, p, sz, p]
        L.focus_kl_top.argtypes = [p, p, i32, i64, i64, i32, p, p, p, sz, p]
        L.focus_adamw_step.argtypes = [ctypes.POINTER(AdamWConfig), i64, i64, p, p, p, p, p, sz, p]
        L.focus_check_flags.argtypes = [p, p]
        L.focus_status_string.argtypes = [i32]
        L.focus_status_string.restype = ctypes.c_char_p
        for name in ("focus_scales_init", "focus_fakequant_fwd", "focus_fakequant_bwd", "focus_recon_gemm_fwd",
                     "focus_recon_gemm_fwd_mxfp4", "focus_recon_gemm_fwd_mxfp4_noalloc", "focus_recon_gemm_bwd",
                     "focus_recon_gemm_bwd_mxfp4",
                     "focus_export_packed", "focus_fakequant_weights", "focus_adamw_step", "focus_check_flags", "focus_recon_gemm_dx", "focus_fakequant_act_bwd",
                     "focus_kl_top"):
            getattr(L, name).restype = ctypes.c_int
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().focus_status_string(status).decode()


SCALES_ROW_MAJOR, SCALES_BLOCK_MAJOR = 0, 1
E8M0_CEIL, E8M0_FLOOR = 0, 1
CODES_ROW_MAJOR, CODES_K_SLAB = 0, 1


def qconfig(fmt: int, sub_block: int, ste_clip: int = 1, scale_layout: int = SCALES_ROW_MAJOR,
            e8m0_rounding: int = 0, code_layout: int = CODES_ROW_MAJOR) -> QConfig:
    return QConfig(fmt, sub_block, ste_clip, scale_layout, e8m0_rounding, code_layout)


def codes_shape(rows: int, K: int, code_layout: int = CODES_ROW_MAJOR) -> tuple:
    """Shape of a packed-code tensor: [rows][K/2], or K-slabs [K/128][rows][64]."""
    return (rows, K // 2) if code_layout == CODES_ROW_MAJOR else (K // 128, rows, 64)


def _slab_dims(codes: torch.Tensor) -> tuple:
    """(rows, K) of codes in K-slabs [K/128][rows][64], the layout of the MXFP4 forward's W operand."""
    if codes.dim() != 3 or codes.shape[2] != 64:
        raise ValueError("the MXFP4 forward takes W codes in K-slabs [K/128][N][64] (code_layout=CODES_K_SLAB)")
    return codes.shape[1], codes.shape[0] * 128


def block_size(fmt: int) -> int:
    return 32 if fmt == MXFP4 else 16


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: torch.Tensor | None):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libfocus must be contiguous")
    return t.data_ptr()


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(status: int, where: str) -> None:
    if status != OK:
        raise FocusError(status, where)


def workspace_size(call: int, q: QConfig, M: int = 0, N: int = 0, K: int = 0) -> int:
    return int(lib().focus_workspace_size(call, ctypes.byref(q), M, N, K))


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """A zero-filled workspace (torch's device allocations are at least 256-byte aligned)."""
    ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def _ws(ws: torch.Tensor | None, call: int, q: QConfig, M: int, N: int, K: int, device) -> torch.Tensor:
    need = workspace_size(call, q, M, N, K)
    if ws is None or ws.numel() < need:
        ws = workspace(need, device)
    return ws


def scales_init(W: torch.Tensor, fmt: int, sub_block: int, ws=None, out=None, e8m0_rounding: int = 0):
    """Absmax initialisation -> (s_fp [N][K/B], c [N][K/sb] = 1, alpha [1])."""
    N, K = W.shape
    q = qconfig(fmt, sub_block, 1, SCALES_ROW_MAJOR, e8m0_rounding)
    if out is None:
        s_fp = torch.empty(N, K // block_size(fmt), dtype=torch.float32, device=W.device)
        c = torch.empty(N, K // sub_block, dtype=torch.float32, device=W.device)
        alpha = torch.ones(1, dtype=torch.float32, device=W.device)
    else:
        s_fp, c, alpha = out
    ws = _ws(ws, CALL_SCALES_INIT, q, 0, N, K, W.device)
    _check(lib().focus_scales_init(ctypes.byref(q), _ptr(W), _dt(W), N, K, _ptr(s_fp), _ptr(c), _ptr(alpha),
                                   _ptr(ws), ws.numel(), _stream()), "focus_scales_init")
    return s_fp, c, alpha


def fakequant_fwd(X: torch.Tensor, fmt: int, sub_block: int = 8, s_fp=None, c=None, alpha=None,
                  out_dtype=None, want_codes: bool = False, want_scale_bytes: bool = False,
                  want_alpha: bool = False, ste_clip: int = 1, ws=None, out=None, codes_out=None,
                  scales_out=None, scale_layout: int = SCALES_ROW_MAJOR, e8m0_rounding: int = 0,
                  want_x_hat: bool = True, code_layout: int = CODES_ROW_MAJOR):
    """Fake quantisation forward. Weight mode when s_fp is given, dynamic activation mode otherwise.
    codes_out / scales_out: preallocated code and scale-byte outputs (they imply want_codes /
    want_scale_bytes). scale_layout: [rows][K/B] (row-major) or [K/B][rows] (block-major); code_layout:
    [rows][K/2] (row-major) or [K/128][rows][64] (K-slabs). want_x_hat=False (with codes) writes the
    packed form only.

    Returns (x_hat or None, packed_codes or None, scale_bytes or None, alpha_x or None)."""
    rows, K = X.shape
    q = qconfig(fmt, sub_block, ste_clip, scale_layout, e8m0_rounding, code_layout)
    out_dtype = out_dtype or X.dtype
    x_hat = out if out is not None else (torch.empty(rows, K, dtype=out_dtype, device=X.device) if want_x_hat
                                         else None)
    codes = codes_out
    if codes is None and want_codes:
        codes = torch.empty(*codes_shape(rows, K, code_layout), dtype=torch.uint8, device=X.device)
    sbytes = scales_out
    if sbytes is None and want_scale_bytes:
        shape = (rows, K // block_size(fmt)) if scale_layout == SCALES_ROW_MAJOR else (K // block_size(fmt), rows)
        sbytes = torch.empty(*shape, dtype=torch.uint8, device=X.device)
    alpha_out = torch.empty(1, dtype=torch.float32, device=X.device) if want_alpha else None
    ws = _ws(ws, CALL_FAKEQUANT_FWD, q, 0, rows, K, X.device)
    _check(lib().focus_fakequant_fwd(ctypes.byref(q), _ptr(X), _dt(X), rows, K, _ptr(s_fp), _ptr(c), _ptr(alpha),
                                     _ptr(x_hat), _dt(x_hat) if x_hat is not None else _dt(X), _ptr(codes),
                                     _ptr(sbytes), _ptr(alpha_out),
                                     _ptr(ws), ws.numel(), _stream()), "focus_fakequant_fwd")
    return x_hat, codes, sbytes, alpha_out


def fakequant_bwd(G: torch.Tensor, W: torch.Tensor, fmt: int, sub_block: int, s_fp, c=None, alpha=None,
                  ste_clip: int = 1, ws=None, e8m0_rounding: int = 0):
    """Straight-through backward from G = dL/dW_hat (fp32) -> (grad_s, grad_c)."""
    N, K = W.shape
    q = qconfig(fmt, sub_block, ste_clip, SCALES_ROW_MAJOR, e8m0_rounding)
    grad_s = torch.empty(N, K // block_size(fmt), dtype=torch.float32, device=W.device)
    grad_c = torch.empty(N, K // sub_block, dtype=torch.float32, device=W.device)
    ws = _ws(ws, CALL_FAKEQUANT_BWD, q, 0, N, K, W.device)
    _check(lib().focus_fakequant_bwd(ctypes.byref(q), _ptr(G), N, K, _ptr(W), _dt(W), _ptr(s_fp), _ptr(c),
                                     _ptr(alpha), _ptr(grad_s), _ptr(grad_c), _ptr(ws), ws.numel(), _stream()),
           "focus_fakequant_bwd")
    return grad_s, grad_c


def recon_gemm_fwd(X_hat: torch.Tensor, W_hat: torch.Tensor, Y_ref=None, want_col_sq: bool = False, ws=None,
                   out=None, loss=None):
    """Y_hat = X_hat W_hat^T with the MSE epilogue -> (dY (or Y_hat when Y_ref is None), loss, col_sq)."""
    M, K = X_hat.shape
    N = W_hat.shape[0]
    dY = out if out is not None else torch.empty(M, N, dtype=X_hat.dtype, device=X_hat.device)
    loss_t = None
    if Y_ref is not None:
        loss_t = loss if loss is not None else torch.empty(1, dtype=torch.float64, device=X_hat.device)
    col_sq = torch.empty(N, dtype=torch.float64, device=X_hat.device) if want_col_sq else None
    q = qconfig(MXFP4, 8)
    ws = _ws(ws, CALL_RECON_GEMM_FWD, q, M, N, K, X_hat.device)
    _check(lib().focus_recon_gemm_fwd(_ptr(X_hat), _ptr(W_hat), _dt(X_hat), M, N, K, _ptr(Y_ref), _ptr(dY),
                                      _ptr(loss_t), _ptr(col_sq), _ptr(ws), ws.numel(), _stream()),
           "focus_recon_gemm_fwd")
    return dY, loss_t, col_sq


def recon_gemm_fwd_mxfp4(X_codes: torch.Tensor, X_scales: torch.Tensor, W_codes: torch.Tensor, W_scales: torch.Tensor,
                         Y_ref=None, want_col_sq: bool = False, ws=None, out=None, loss=None):
    """The forward from packed MXFP4 operands (X codes [M][K/2], W codes in K-slabs [K/128][N][64],
    block-major E8M0 bytes [K/32][rows]) -> as recon_gemm_fwd."""
    M, K = X_codes.shape[0], X_codes.shape[1] * 2
    N = _slab_dims(W_codes)[0]
    dev = X_codes.device
    dY = out if out is not None else torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    loss_t = None
    if Y_ref is not None:
        loss_t = loss if loss is not None else torch.empty(1, dtype=torch.float64, device=dev)
    col_sq = torch.empty(N, dtype=torch.float64, device=dev) if want_col_sq else None
    ws = _ws(ws, CALL_RECON_GEMM_FWD, qconfig(MXFP4, 8), M, N, K, dev)
    _check(lib().focus_recon_gemm_fwd_mxfp4(_ptr(X_codes), _ptr(X_scales), _ptr(W_codes), _ptr(W_scales), M, N, K,
                                            _ptr(Y_ref), _ptr(dY), _ptr(loss_t), _ptr(col_sq), _ptr(ws), ws.numel(),
                                            _stream()),
           "focus_recon_gemm_fwd_mxfp4")
    return dY, loss_t, col_sq


def recon_gemm_fwd_mxfp4_noalloc(X_codes: torch.Tensor, X_scales: torch.Tensor, W_codes: torch.Tensor,
                                 W_scales: torch.Tensor, Y_ref=None, col_sq=None, out=None, loss=None):
    """recon_gemm_fwd_mxfp4 without a workspace (the library's fixed device scratch instead). The
    library allocates nothing; the caller passes dY (`out`), `loss` when Y_ref is given, and
    optionally `col_sq` [N] float64. -> (dY, loss, col_sq)."""
    M, K = X_codes.shape[0], X_codes.shape[1] * 2
    N = _slab_dims(W_codes)[0]
    if out is None or (Y_ref is not None and loss is None):
        raise ValueError("recon_gemm_fwd_mxfp4_noalloc: pass the outputs (out, and loss with Y_ref)")
    _check(lib().focus_recon_gemm_fwd_mxfp4_noalloc(_ptr(X_codes), _ptr(X_scales), _ptr(W_codes), _ptr(W_scales),
                                                    M, N, K, _ptr(Y_ref), _ptr(out), _ptr(loss), _ptr(col_sq),
                                                    _stream()),
           "focus_recon_gemm_fwd_mxfp4_noalloc")
    return out, loss, col_sq


def recon_gemm_bwd(dY: torch.Tensor, X_hat: torch.Tensor, W: torch.Tensor, fmt: int, sub_block: int, s_fp,
                   c=None, alpha=None, ste_clip: int = 1, want_G: bool = False, ws=None, out=None,
                   e8m0_rounding: int = 0):
    """Fused backward -> (grad_s, grad_c, G or None)."""
    M, K = X_hat.shape
    N = W.shape[0]
    q = qconfig(fmt, sub_block, ste_clip, SCALES_ROW_MAJOR, e8m0_rounding)
    if out is None:
        grad_s = torch.empty(N, K // block_size(fmt), dtype=torch.float32, device=W.device)
        grad_c = torch.empty(N, K // sub_block, dtype=torch.float32, device=W.device)
    else:
        grad_s, grad_c = out
    G = torch.empty(N, K, dtype=torch.float32, device=W.device) if want_G else None
    ws = _ws(ws, CALL_RECON_GEMM_BWD, q, M, N, K, W.device)
    _check(lib().focus_recon_gemm_bwd(ctypes.byref(q), _ptr(dY), _ptr(X_hat), _dt(X_hat), M, N, K, _ptr(W),
                                      _dt(W), _ptr(s_fp), _ptr(c), _ptr(alpha), _ptr(grad_s), _ptr(grad_c),
                                      _ptr(G), _ptr(ws), ws.numel(), _stream()), "focus_recon_gemm_bwd")
    return grad_s, grad_c, G


def recon_gemm_bwd_mxfp4(dY: torch.Tensor, X_codes: torch.Tensor, X_scales: torch.Tensor, W: torch.Tensor,
                         sub_block: int, s_fp, c=None, ste_clip: int = 1, ws=None, out=None, e8m0_rounding: int = 0):
    """Fused backward with X_hat as packed MXFP4 (codes [M][K/2], block-major E8M0 bytes [K/32][M])
    -> (grad_s, grad_c)."""
    M, K = X_codes.shape[0], X_codes.shape[1] * 2
    N = W.shape[0]
    q = qconfig(MXFP4, sub_block, ste_clip, SCALES_ROW_MAJOR, e8m0_rounding)
    if out is None:
        grad_s = torch.empty(N, K // 32, dtype=torch.float32, device=W.device)
        grad_c = torch.empty(N, K // sub_block, dtype=torch.float32, device=W.device)
    else:
        grad_s, grad_c = out
    ws = _ws(ws, CALL_RECON_GEMM_BWD, q, M, N, K, W.device)
    _check(lib().focus_recon_gemm_bwd_mxfp4(ctypes.byref(q), _ptr(dY), _ptr(X_codes), _ptr(X_scales), M, N, K,
                                            _ptr(W), _dt(W), _ptr(s_fp), _ptr(c), _ptr(grad_s), _ptr(grad_c),
                                            _ptr(ws), ws.numel(), _stream()), "focus_recon_gemm_bwd_mxfp4")
    return grad_s, grad_c


def export_packed(W: torch.Tensor, fmt: int, sub_block: int, s_fp, c=None, alpha=None, ws=None, out=None,
                  scale_layout: int = SCALES_ROW_MAJOR, e8m0_rounding: int = 0, code_layout: int = CODES_ROW_MAJOR):
    """Deployable export -> (packed codes [N][K/2] or, in K-slabs, [K/128][N][64]; scale bytes [N][K/B] or,
    block-major, [K/B][N])."""
    N, K = W.shape
    q = qconfig(fmt, sub_block, 1, scale_layout, e8m0_rounding, code_layout)
    if out is None:
        packed = torch.empty(*codes_shape(N, K, code_layout), dtype=torch.uint8, device=W.device)
        shape = (N, K // block_size(fmt)) if scale_layout == SCALES_ROW_MAJOR else (K // block_size(fmt), N)
        sbytes = torch.empty(*shape, dtype=torch.uint8, device=W.device)
    else:
        packed, sbytes = out
    ws = _ws(ws, CALL_EXPORT_PACKED, q, 0, N, K, W.device)
    _check(lib().focus_export_packed(ctypes.byref(q), _ptr(W), _dt(W), N, K, _ptr(s_fp), _ptr(c), _ptr(alpha),
                                     _ptr(packed), _ptr(sbytes), _ptr(ws), ws.numel(), _stream()),
           "focus_export_packed")
    return packed, sbytes


def fakequant_weights(layers, fmt: int, sub_block: int, w_dtype=None, what_dtype=None, ws=None,
                      scale_layout: int = SCALES_ROW_MAJOR, e8m0_rounding: int = 0,
                      code_layout: int = CODES_ROW_MAJOR) -> None:
    """Weight fake quantisation of several layers in one call (focus_fakequant_weights). `layers` is a
    sequence of dicts with keys W, s_fp and optionally c, alpha, W_hat, codes, scale_bytes (device
    tensors; the outputs are written in place). w_dtype / what_dtype default to the first layer's W /
    W_hat dtype."""
    q = qconfig(fmt, sub_block, 1, scale_layout, e8m0_rounding, code_layout)
    arr = (WeightLayer * max(1, len(layers)))()
    for i, l in enumerate(layers):
        W = l["W"]
        arr[i] = WeightLayer(_ptr(W), W.shape[0], W.shape[1], _ptr(l["s_fp"]), _ptr(l.get("c")), _ptr(l.get("alpha")),
                             _ptr(l.get("W_hat")), _ptr(l.get("codes")), _ptr(l.get("scale_bytes")))
    if w_dtype is None:
        w_dtype = _dt(layers[0]["W"]) if layers else BF16
    if what_dtype is None:
        wh = next((l["W_hat"] for l in layers if l.get("W_hat") is not None), None)
        what_dtype = _dt(wh) if wh is not None else w_dtype
    device = layers[0]["W"].device if layers else "cuda"
    ws = _ws(ws, CALL_FAKEQUANT_WEIGHTS, q, 0, 0, 0, device)
    _check(lib().focus_fakequant_weights(ctypes.byref(q), w_dtype, what_dtype, arr, len(layers), _ptr(ws), ws.numel(),
                                         _stream()), "focus_fakequant_weights")


def recon_gemm_dx(dY: torch.Tensor, W_hat: torch.Tensor, ws=None, out=None) -> torch.Tensor:
    """dX_hat = dY W_hat (the input gradient of a linear) -> [M][K] in dY's dtype."""
    M, N = dY.shape
    K = W_hat.shape[1]
    assert W_hat.shape[0] == N and W_hat.dtype == dY.dtype
    dX = out if out is not None else torch.empty(M, K, dtype=dY.dtype, device=dY.device)
    need = workspace_size(CALL_RECON_GEMM_DX, qconfig(MXFP4, 8), M, N, K)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dY.device)
    _check(lib().focus_recon_gemm_dx(_ptr(dY), _ptr(W_hat), _dt(dY), M, N, K, _ptr(dX), _ptr(ws), ws.numel(),
                                     _stream()), "focus_recon_gemm_dx")
    return dX


def fakequant_act_bwd(X: torch.Tensor, dX_hat: torch.Tensor, fmt: int, ste_clip: int = 1, e8m0_rounding: int = 0,
                      ws=None, out=None) -> torch.Tensor:
    """Straight-through backward of the activation fake quantisation -> dX (dX_hat's dtype)."""
    rows, K = X.shape
    q = qconfig(fmt, 8, ste_clip, SCALES_ROW_MAJOR, e8m0_rounding)  # the sub-block plays no part here
    dX = out if out is not None else torch.empty_like(dX_hat)
    ws = _ws(ws, CALL_FAKEQUANT_ACT_BWD, q, 0, rows, K, X.device)
    _check(lib().focus_fakequant_act_bwd(ctypes.byref(q), _ptr(X), _dt(X), rows, K, _ptr(dX_hat), _dt(dX_hat),
                                         _ptr(dX), _ptr(ws), ws.numel(), _stream()), "focus_fakequant_act_bwd")
    return dX


def kl_top(Z_student: torch.Tensor, Z_teacher: torch.Tensor, k: int = 1000, ws=None, out=None, loss=None):
    """KL-Top loss of student logits against teacher logits -> (dZ_student, loss [1] fp64)."""
    T, V = Z_student.shape
    assert Z_teacher.shape == Z_student.shape and Z_teacher.dtype == Z_student.dtype
    dZ = out if out is not None else torch.empty_like(Z_student)
    loss_t = loss if loss is not None else torch.empty(1, dtype=torch.float64, device=Z_student.device)
    need = workspace_size(CALL_KL_TOP, qconfig(MXFP4, 8), T, V, 0)
    if ws is None or ws.numel() < need:
        ws = workspace(need, Z_student.device)
    _check(lib().focus_kl_top(_ptr(Z_student), _ptr(Z_teacher), _dt(Z_student), T, V, k, _ptr(dZ), _ptr(loss_t),
                              _ptr(ws), ws.numel(), _stream()), "focus_kl_top")
    return dZ, loss_t


def adamw_step(param: torch.Tensor, grad: torch.Tensor, exp_avg: torch.Tensor, exp_avg_sq: torch.Tensor, t: int,
               lr: float, betas=(0.9, 0.999), eps: float = 1e-8, weight_decay: float = 0.0,
               log2_domain: bool = False, ws=None) -> None:
    """One in-place AdamW step on fp32 `param` (moments in exp_avg / exp_avg_sq, t the 1-based step)."""
    for x in (param, grad, exp_avg, exp_avg_sq):
        assert x.dtype == torch.float32 and x.is_contiguous() and x.numel() == param.numel()
    cfg = AdamWConfig(lr, betas[0], betas[1], eps, weight_decay, int(log2_domain))
    if ws is None:
        ws = workspace(256, param.device)
    _check(lib().focus_adamw_step(ctypes.byref(cfg), t, param.numel(), _ptr(param), _ptr(grad), _ptr(exp_avg),
                                  _ptr(exp_avg_sq), _ptr(ws), ws.numel(), _stream()), "focus_adamw_step")


def check_flags(ws: torch.Tensor) -> int:
    """Synchronises the current stream; returns OK or ERR_DOMAIN (and clears the flag)."""
    return int(lib().focus_check_flags(_ptr(ws), _stream()))
