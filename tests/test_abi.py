"""The C ABI on the CPU: libfocus loads, exports every function include/focus.h declares, and its
host-side checks reject bad arguments with the documented status before anything is launched.

No test here launches a kernel: every call carries an argument that a check must refuse, and the
pointers are never dereferenced. On a machine with a visible GPU the argument-check tests are
skipped (they belong to the CPU suite).
"""
import ctypes
import os
import re

import pytest

from paper_2608_01847_amd import focus

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "focus.h")


def declared_functions():
    text = open(HEADER).read()
    # declarations: a return type at the start of a line, then the function name and "("
    return sorted(set(re.findall(r"^(?:focus_status|size_t|const char \*)\s*(focus_[a-z0-9_]+)\(", text, re.M)))


@pytest.fixture(scope="module")
def L():
    if not focus.LIBRARY.exists():
        pytest.skip("libfocus.so is not built")
    return focus.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(focus.EXPORTED)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    for s in range(9):
        assert focus.status_string(s) and focus.status_string(s) != "unknown status"
    assert focus.status_string(99) == "unknown status"


def test_workspace_sizes_host_only(L):
    q = focus.qconfig(focus.MXFP4, 8)
    assert focus.workspace_size(focus.CALL_FAKEQUANT_BWD, q) == 256
    assert focus.workspace_size(focus.CALL_FAKEQUANT_FWD, q) >= 256 + 4 * 1024
    fwd = focus.workspace_size(focus.CALL_RECON_GEMM_FWD, q, 1000, 300, 256)
    assert fwd >= 256 + 8 * 300 * (1000 // 256)
    bwd = focus.workspace_size(focus.CALL_RECON_GEMM_BWD, q, 65536, 1024, 2560)
    assert bwd >= 256 + 4 * 1024 * (2560 // 32 + 2560 // 8)
    # invalid configurations size to 0
    assert focus.workspace_size(focus.CALL_RECON_GEMM_BWD, focus.qconfig(focus.NVFP4, 32), 1, 1, 16) == 0
    assert focus.workspace_size(focus.CALL_RECON_GEMM_BWD, q, 16, 4, 48) == 0  # K % 32
    assert focus.workspace_size(99, q) == 0


BOGUS = ctypes.c_void_p(1 << 20)  # never dereferenced: every call below fails a host check first


@pytest.fixture()
def cpu_only():
    import torch
    if torch.cuda.is_available():
        pytest.skip("argument-check tests run in the CPU suite only")


def fq_fwd(L, q, K=64, rows=4, x_dt=1, xh_dt=1, X=BOGUS, s_fp=None, c=None, alpha=None, ws=BOGUS, ws_bytes=1 << 20):
    return L.focus_fakequant_fwd(ctypes.byref(q), X, x_dt, rows, K, s_fp, c, alpha, BOGUS, xh_dt, None, None,
                                 None, ws, ws_bytes, None)


def test_argument_checks(L, cpu_only):
    mx = focus.qconfig(focus.MXFP4, 8)
    assert fq_fwd(L, focus.qconfig(2, 8)) == focus.ERR_CONFIG
    assert fq_fwd(L, focus.qconfig(focus.MXFP4, 3)) == focus.ERR_CONFIG
    assert fq_fwd(L, focus.qconfig(focus.NVFP4, 32)) == focus.ERR_CONFIG  # sub-block larger than the block
    assert fq_fwd(L, focus.qconfig(focus.MXFP4, 8, 2)) == focus.ERR_CONFIG
    assert fq_fwd(L, focus.QConfig(0, 8, 1, 5)) == focus.ERR_CONFIG  # no such scale layout
    assert fq_fwd(L, focus.QConfig(0, 8, 1, 0, 2)) == focus.ERR_CONFIG  # no such E8M0 rounding
    assert fq_fwd(L, focus.QConfig(1, 8, 1, 0, 1), K=64) == focus.ERR_CONFIG  # floor E8M0 is MXFP4 only
    assert fq_fwd(L, focus.QConfig(0, 8, 1, 0, 0, 2)) == focus.ERR_CONFIG  # no such code layout
    slab = focus.qconfig(focus.MXFP4, 8, code_layout=focus.CODES_K_SLAB)
    # K-slab codes need whole slabs of 128 elements (only where codes are written)
    assert L.focus_fakequant_fwd(ctypes.byref(slab), BOGUS, 1, 4, 96, None, None, None, BOGUS, 1, BOGUS, None, None,
                                 BOGUS, 1 << 20, None) == focus.ERR_SHAPE
    assert L.focus_export_packed(ctypes.byref(slab), BOGUS, 1, 4, 96, BOGUS, None, None, BOGUS, BOGUS, BOGUS, 1 << 20,
                                 None) == focus.ERR_SHAPE
    assert fq_fwd(L, mx, X=None) == focus.ERR_NULL
    # an empty tensor may come as NULL pointers (nothing is launched)
    assert L.focus_fakequant_fwd(ctypes.byref(mx), None, 1, 0, 64, None, None, None, None, 1, None, None, None,
                                 BOGUS, 1 << 20, None) == focus.OK
    # X_hat may be left out only when the codes are asked for
    assert L.focus_fakequant_fwd(ctypes.byref(mx), BOGUS, 1, 4, 64, None, None, None, None, 1, None, BOGUS, None,
                                 BOGUS, 1 << 20, None) == focus.ERR_NULL
    assert fq_fwd(L, mx, x_dt=7) == focus.ERR_DTYPE
    assert fq_fwd(L, mx, K=48) == focus.ERR_SHAPE          # not a multiple of 32
    assert fq_fwd(L, mx, rows=-1) == focus.ERR_SHAPE
    assert fq_fwd(L, mx, rows=1 << 31) == focus.ERR_SHAPE
    assert fq_fwd(L, mx, ws=None) == focus.ERR_WORKSPACE
    assert fq_fwd(L, mx, ws=ctypes.c_void_p((1 << 20) + 8)) == focus.ERR_WORKSPACE  # misaligned
    assert fq_fwd(L, mx, ws_bytes=16) == focus.ERR_WORKSPACE
    assert fq_fwd(L, mx, c=BOGUS) == focus.ERR_CONFIG       # activation mode takes no coefficients
    nv = focus.qconfig(focus.NVFP4, 8)
    assert fq_fwd(L, nv, K=64, s_fp=BOGUS) == focus.ERR_NULL  # NVFP4 weights need alpha
    # fused backward
    assert L.focus_recon_gemm_bwd(ctypes.byref(mx), BOGUS, BOGUS, 1, 64, 4, 40, BOGUS, 1, BOGUS, None, None,
                                  BOGUS, BOGUS, None, BOGUS, 1 << 30, None) == focus.ERR_SHAPE
    assert L.focus_recon_gemm_bwd(ctypes.byref(mx), BOGUS, BOGUS, 1, 64, 4, 64, BOGUS, 1, None, None, None,
                                  BOGUS, BOGUS, None, BOGUS, 1 << 30, None) == focus.ERR_NULL
    assert L.focus_recon_gemm_bwd(ctypes.byref(mx), BOGUS, BOGUS, 1, 64, 4, 64, BOGUS, 1, BOGUS, None, None,
                                  BOGUS, BOGUS, None, BOGUS, 16, None) == focus.ERR_WORKSPACE
    # forward GEMM
    assert L.focus_recon_gemm_fwd(BOGUS, BOGUS, 1, 8, 8, 24, None, BOGUS, None, None, BOGUS, 1 << 30,
                                  None) == focus.ERR_SHAPE
    assert L.focus_recon_gemm_fwd(BOGUS, BOGUS, 1, 8, 8, 32, BOGUS, BOGUS, None, None, BOGUS, 1 << 30,
                                  None) == focus.ERR_NULL  # MSE mode needs loss_out
    assert L.focus_recon_gemm_fwd(BOGUS, BOGUS, 3, 8, 8, 32, None, BOGUS, None, None, BOGUS, 1 << 30,
                                  None) == focus.ERR_DTYPE
    # no tokens or no output features: nothing is launched and nothing is written (the loss, a mean over
    # no elements, keeps whatever the caller's buffer held); the workspace is still checked
    loss = ctypes.c_double(-7.0)
    for M, N in ((0, 8), (8, 0)):
        assert L.focus_recon_gemm_fwd(BOGUS, BOGUS, 1, M, N, 32, BOGUS, BOGUS, ctypes.byref(loss), None, BOGUS,
                                      1 << 30, None) == focus.OK
        assert L.focus_recon_gemm_fwd_mxfp4(BOGUS, BOGUS, BOGUS, BOGUS, M, N, 128, BOGUS, BOGUS, ctypes.byref(loss),
                                            None, BOGUS, 1 << 30, None) == focus.OK
    assert loss.value == -7.0
    assert L.focus_recon_gemm_fwd(BOGUS, BOGUS, 1, 0, 8, 32, BOGUS, BOGUS, ctypes.byref(loss), None, BOGUS, 8,
                                  None) == focus.ERR_WORKSPACE
    # forward GEMM from packed MXFP4 operands
    mxf = L.focus_recon_gemm_fwd_mxfp4
    assert mxf(BOGUS, BOGUS, BOGUS, BOGUS, 8, 8, 64, None, BOGUS, None, None, BOGUS, 1 << 30,
               None) == focus.ERR_SHAPE   # K not a multiple of 128
    assert mxf(BOGUS, BOGUS, BOGUS, BOGUS, 8, 12, 128, None, BOGUS, None, None, BOGUS, 1 << 30,
               None) == focus.ERR_SHAPE   # N not a multiple of 8
    assert mxf(BOGUS, BOGUS, BOGUS, BOGUS, 6, 8, 128, None, BOGUS, None, None, BOGUS, 1 << 30,
               None) == focus.ERR_SHAPE   # M not a multiple of 4
    assert mxf(BOGUS, None, BOGUS, BOGUS, 8, 8, 128, None, BOGUS, None, None, BOGUS, 1 << 30,
               None) == focus.ERR_NULL
    assert mxf(BOGUS, BOGUS, BOGUS, BOGUS, 8, 8, 128, BOGUS, BOGUS, None, None, BOGUS, 1 << 30,
               None) == focus.ERR_NULL    # MSE mode needs loss_out
    assert mxf(BOGUS, ctypes.c_void_p((1 << 20) + 2), BOGUS, BOGUS, 8, 8, 128, None, BOGUS, None, None, BOGUS,
               1 << 30, None) == focus.ERR_SHAPE  # scale bytes not 4-byte aligned
    assert mxf(BOGUS, BOGUS, BOGUS, BOGUS, 8, 8, 128, None, BOGUS, None, None, BOGUS, 16,
               None) == focus.ERR_WORKSPACE
    # its allocation-free variant: the same argument checks, then the fixed 32 MiB scratch bounds the sizes
    # (256 + 8 (ceil(M / 256) N + N) bytes, the column sums dropped when the caller passes col_sq)
    nal = L.focus_recon_gemm_fwd_mxfp4_noalloc
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, 8, 8, 64, None, BOGUS, None, None, None) == focus.ERR_SHAPE
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, 8, 12, 128, None, BOGUS, None, None, None) == focus.ERR_SHAPE
    assert nal(BOGUS, None, BOGUS, BOGUS, 8, 8, 128, None, BOGUS, None, None, None) == focus.ERR_NULL
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, 8, 8, 128, BOGUS, BOGUS, None, None, None) == focus.ERR_NULL
    limit = 32 << 20
    M = 65536                      # 256 m-tiles
    n_max = (limit - 256) // 8 // (256 + 1) // 8 * 8
    assert 256 + 8 * (256 * n_max + n_max) <= limit < 256 + 8 * (256 * (n_max + 8) + n_max + 8)
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, M, n_max + 8, 128, BOGUS, BOGUS, BOGUS, None, None) == focus.ERR_SCRATCH
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, M, 28672, 8192, BOGUS, BOGUS, BOGUS, BOGUS, None) == focus.ERR_SCRATCH
    # with the caller's col_sq the N column sums leave the scratch: one more width step fits
    n_col = (limit - 256) // 8 // 256 // 8 * 8
    assert n_col > n_max
    assert nal(BOGUS, BOGUS, BOGUS, BOGUS, M, n_col + 8, 128, BOGUS, BOGUS, BOGUS, BOGUS, None) == focus.ERR_SCRATCH
    # fused backward from packed MXFP4 activations
    mxb = L.focus_recon_gemm_bwd_mxfp4
    def bwd_mx(q, M=8, N=8, K=128, scales=BOGUS, ws_bytes=1 << 30, w_dt=1):
        return mxb(ctypes.byref(q), BOGUS, BOGUS, scales, M, N, K, BOGUS, w_dt, BOGUS, None, BOGUS, BOGUS, BOGUS,
                   ws_bytes, None)
    assert bwd_mx(nv) == focus.ERR_CONFIG                   # MXFP4 only
    assert bwd_mx(mx, K=48) == focus.ERR_SHAPE               # K not a multiple of 32
    assert bwd_mx(mx, N=12) == focus.ERR_SHAPE               # N not a multiple of 8
    assert bwd_mx(mx, M=6) == focus.ERR_SHAPE                # M not a multiple of 4
    assert bwd_mx(mx, scales=None) == focus.ERR_NULL
    assert mxb(ctypes.byref(mx), BOGUS, BOGUS, BOGUS, 8, 8, 64, None, 1, BOGUS, None, BOGUS, BOGUS, BOGUS,
               1 << 30, None) == focus.ERR_NULL  # W is needed even for no tokens
    assert bwd_mx(mx, scales=ctypes.c_void_p((1 << 20) + 2)) == focus.ERR_SHAPE  # scale bytes not 4-byte aligned
    assert bwd_mx(mx, w_dt=5) == focus.ERR_DTYPE
    assert bwd_mx(mx, ws_bytes=16) == focus.ERR_WORKSPACE
    # export and init
    assert L.focus_export_packed(ctypes.byref(mx), BOGUS, 1, 4, 64, BOGUS, None, None, None, BOGUS, BOGUS,
                                 1 << 20, None) == focus.ERR_NULL
    assert L.focus_scales_init(ctypes.byref(nv), BOGUS, 1, 4, 64, BOGUS, BOGUS, None, BOGUS, 1 << 20,
                               None) == focus.ERR_NULL
    assert L.focus_fakequant_bwd(ctypes.byref(mx), BOGUS, 4, 64, BOGUS, 0, BOGUS, None, None, BOGUS, BOGUS,
                                 BOGUS, 8, None) == focus.ERR_WORKSPACE
    # AdamW
    def adam(cfg, t=1, n=16, ptr=BOGUS, ws=BOGUS, ws_bytes=256):
        return L.focus_adamw_step(ctypes.byref(cfg), t, n, ptr, BOGUS, BOGUS, BOGUS, ws, ws_bytes, None)
    good = focus.AdamWConfig(1e-2, 0.9, 0.999, 1e-8, 0.0, 1)
    assert adam(good, t=0) == focus.ERR_CONFIG
    assert adam(focus.AdamWConfig(-1e-2, 0.9, 0.999, 1e-8, 0.0, 0)) == focus.ERR_CONFIG
    assert adam(focus.AdamWConfig(1e-2, 1.0, 0.999, 1e-8, 0.0, 0)) == focus.ERR_CONFIG
    assert adam(focus.AdamWConfig(1e-2, 0.9, 0.999, 0.0, 0.0, 0)) == focus.ERR_CONFIG
    assert adam(focus.AdamWConfig(float("nan"), 0.9, 0.999, 1e-8, 0.0, 0)) == focus.ERR_CONFIG
    assert adam(focus.AdamWConfig(1e-2, 0.9, 0.999, 1e-8, 0.0, 2)) == focus.ERR_CONFIG
    assert L.focus_adamw_step(None, 1, 16, BOGUS, BOGUS, BOGUS, BOGUS, BOGUS, 256, None) == focus.ERR_NULL
    assert adam(good, n=-1) == focus.ERR_SHAPE
    assert adam(good, n=(1 << 40) + 1) == focus.ERR_SHAPE
    assert adam(good, ptr=None) == focus.ERR_NULL
    assert adam(good, ptr=ctypes.c_void_p((1 << 20) + 4)) == focus.ERR_SHAPE  # not 16-byte aligned
    assert adam(good, ws_bytes=8) == focus.ERR_WORKSPACE
    assert focus.workspace_size(focus.CALL_ADAMW, focus.qconfig(focus.MXFP4, 8)) == 256
    assert L.focus_check_flags(None, None) == focus.ERR_WORKSPACE
    # KL-Top: k >= 1, at least one token row and 1 <= V <= 2^31
    def kl(T=4, V=64, k=8, ptr=BOGUS):
        return L.focus_kl_top(ptr, BOGUS, 1, T, V, k, BOGUS, BOGUS, BOGUS, 1 << 30, None)
    assert kl(k=0) == focus.ERR_CONFIG
    assert kl(T=0) == focus.ERR_SHAPE
    assert kl(V=0) == focus.ERR_SHAPE
    assert kl(V=(1 << 31) + 1, T=1) == focus.ERR_SHAPE
    assert kl(ptr=None) == focus.ERR_NULL
    assert kl(ptr=ctypes.c_void_p((1 << 20) + 1)) == focus.ERR_SHAPE  # not element-aligned (bf16)


def test_grouped_weight_argument_checks(L, cpu_only):
    """focus_fakequant_weights checks the group size, then every layer as focus_fakequant_fwd checks a
    weight-mode call, then the workspace; a bad layer anywhere in the table fails the whole call."""
    mx, nv = focus.qconfig(focus.MXFP4, 8), focus.qconfig(focus.NVFP4, 8)
    assert focus.workspace_size(focus.CALL_FAKEQUANT_WEIGHTS, mx) == 256

    def table(n, over=None):
        arr = (focus.WeightLayer * max(n, 1))()
        for i in range(n):
            arr[i] = focus.WeightLayer(BOGUS.value, 4, 64, BOGUS.value, None, None, None, BOGUS.value, BOGUS.value)
        for (i, field), v in (over or {}).items():
            setattr(arr[i], field, v)
        return arr

    def call(q, arr, n, w_dt=1, wh_dt=1, ws=BOGUS, ws_bytes=1 << 20):
        return L.focus_fakequant_weights(ctypes.byref(q), w_dt, wh_dt, arr, n, ws, ws_bytes, None)

    n = focus.MAX_WEIGHT_LAYERS
    assert call(mx, table(n + 1), n + 1) == focus.ERR_SHAPE
    assert call(mx, table(1), -1) == focus.ERR_SHAPE
    assert L.focus_fakequant_weights(ctypes.byref(mx), 1, 1, None, 2, BOGUS, 1 << 20, None) == focus.ERR_NULL
    assert call(focus.qconfig(2, 8), table(2), 2) == focus.ERR_CONFIG
    assert call(mx, table(2), 2, w_dt=7) == focus.ERR_DTYPE
    assert call(mx, table(2), 2, wh_dt=7) == focus.ERR_DTYPE
    # a bad last layer fails the call
    assert call(mx, table(n, {(n - 1, "K"): 48}), n) == focus.ERR_SHAPE
    assert call(mx, table(n, {(n - 1, "rows"): 1 << 31}), n) == focus.ERR_SHAPE
    assert call(mx, table(3, {(2, "W"): None}), 3) == focus.ERR_NULL
    assert call(mx, table(3, {(1, "s_fp"): None}), 3) == focus.ERR_NULL
    assert call(mx, table(3, {(1, "codes"): None}), 3) == focus.ERR_NULL   # W_hat and codes both NULL
    assert call(mx, table(3, {(0, "W"): BOGUS.value + 8}), 3) == focus.ERR_SHAPE  # not 16-byte aligned
    assert call(nv, table(3), 3) == focus.ERR_NULL                           # NVFP4 needs alpha
    slab = focus.qconfig(focus.MXFP4, 8, code_layout=focus.CODES_K_SLAB)
    assert call(slab, table(3, {(1, "K"): 96}), 3) == focus.ERR_SHAPE        # K-slab codes need K % 128 == 0
    # a layer that writes no codes may have any K: the call gets as far as the workspace check
    w_hat_only = table(3, {(0, "K"): 128, (2, "K"): 128, (1, "K"): 96, (1, "codes"): None,
                           (1, "W_hat"): BOGUS.value})
    assert call(slab, w_hat_only, 3, ws_bytes=16) == focus.ERR_WORKSPACE
    assert call(mx, table(3), 3, ws=None) == focus.ERR_WORKSPACE
    assert call(mx, table(3), 3, ws_bytes=16) == focus.ERR_WORKSPACE
    # no layers, or only empty layers (NULL pointers allowed): nothing is launched
    assert call(mx, table(0), 0) == focus.OK
    empty = table(2, {(0, "rows"): 0, (0, "W"): None, (0, "s_fp"): None, (0, "codes"): None,
                        (1, "rows"): 0, (1, "W"): None})
    assert call(mx, empty, 2) == focus.OK
