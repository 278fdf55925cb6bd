"""GPU test of the allocation-free forward (focus_recon_gemm_fwd_mxfp4_noalloc) through the C ABI.

It runs the same kernels as focus_recon_gemm_fwd_mxfp4, with the library's fixed device scratch in
place of a workspace, so its outputs must equal that entry point's bit for bit: dY, the loss and
the column sums of D^2 in MSE mode (with and without the caller's col_sq), Y_hat in the plain
product mode. Two calls in a row, the second on smaller sizes, show that what the first call left in
the shared scratch does not reach the second's results. Sizes beyond the scratch are refused on the
host before anything is launched.
"""
import pytest
import torch

from gpu_common import announce, assert_bits_equal, device_bits, require_gpu

pytestmark = pytest.mark.gpu

MX = 0


@pytest.fixture(scope="module")
def F():
    return require_gpu()


def operands(F, M, N, K, seed):
    """Packed MXFP4 codes (W in K-slabs) + block-major E8M0 bytes of a seeded X [M][K] and W [N][K], and Y_ref."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    X = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
    W = (torch.randn(N, K, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    Y = (X.float() @ W.float().T).to(torch.bfloat16)
    bm = F.SCALES_BLOCK_MAJOR
    _, xc, xs, _ = F.fakequant_fwd(X, MX, 8, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                   scale_layout=bm)
    _, wc, ws, _ = F.fakequant_fwd(W, MX, 8, want_codes=True, want_scale_bytes=True, want_x_hat=False,
                                   scale_layout=bm, code_layout=F.CODES_K_SLAB)
    return xc, xs, wc, ws, Y


def nan_like(shape, dtype):
    return torch.full(shape, float("nan"), dtype=dtype, device="cuda")


def check_case(F, M, N, K, seed):
    xc, xs, wc, ws, Y = operands(F, M, N, K, seed)
    # the entry point with a workspace
    ref_dy, ref_loss, ref_col = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y, want_col_sq=True)
    ref_plain, _, _ = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, None)
    _, ref_loss_only, _ = F.recon_gemm_fwd_mxfp4(xc, xs, wc, ws, Y)
    # the allocation-free one, outputs pre-filled with NaN so a value it failed to write shows
    announce(f"noalloc forward M={M} N={N} K={K} (MSE with col_sq)")
    dy = nan_like((M, N), torch.bfloat16)
    loss = nan_like((1,), torch.float64)
    col = nan_like((N,), torch.float64)
    F.recon_gemm_fwd_mxfp4_noalloc(xc, xs, wc, ws, Y, col_sq=col, out=dy, loss=loss)
    announce(f"noalloc forward M={M} N={N} K={K} (MSE, column sums in the scratch)")
    dy2 = nan_like((M, N), torch.bfloat16)
    loss2 = nan_like((1,), torch.float64)
    F.recon_gemm_fwd_mxfp4_noalloc(xc, xs, wc, ws, Y, out=dy2, loss=loss2)
    announce(f"noalloc forward M={M} N={N} K={K} (plain product)")
    plain = nan_like((M, N), torch.bfloat16)
    F.recon_gemm_fwd_mxfp4_noalloc(xc, xs, wc, ws, None, out=plain)
    torch.cuda.synchronize()
    assert_bits_equal(device_bits(dy), device_bits(ref_dy), f"dY {M}x{N}x{K}")
    assert_bits_equal(device_bits(dy2), device_bits(ref_dy), f"dY (no col_sq) {M}x{N}x{K}")
    assert_bits_equal(device_bits(plain), device_bits(ref_plain), f"Y_hat {M}x{N}x{K}")
    assert loss.item() == ref_loss.item() and loss2.item() == ref_loss_only.item()
    assert torch.equal(col, ref_col)
    assert torch.isfinite(loss).all() and ref_loss.item() > 0


def test_noalloc_matches_the_workspace_forward_twice(F):
    # first call: ragged in every dimension (4 token tiles, the last 232 rows; 3 column tiles, the last
    # 8 wide; 3 K steps); second call smaller, so the scratch still holds the first call's partials
    check_case(F, 1000, 520, 384, seed=11)
    check_case(F, 260, 136, 256, seed=12)


def test_noalloc_refuses_sizes_beyond_the_scratch(F):
    xc = torch.empty(65536, 64, dtype=torch.uint8, device="cuda")  # K = 128
    xs = torch.empty(4, 65536, dtype=torch.uint8, device="cuda")
    wc = torch.empty(1, 20480, 64, dtype=torch.uint8, device="cuda")  # K-slabs
    ws = torch.empty(4, 20480, dtype=torch.uint8, device="cuda")
    Y = torch.empty(1, dtype=torch.bfloat16, device="cuda")  # never read: the size check comes first
    dy = torch.empty(1, dtype=torch.bfloat16, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    with pytest.raises(F.FocusError) as e:
        F.recon_gemm_fwd_mxfp4_noalloc(xc, xs, wc, ws, Y, out=dy, loss=loss)
    assert e.value.status == F.ERR_SCRATCH
