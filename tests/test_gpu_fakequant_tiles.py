"""GPU parity of the tiled fake-quant kernels at the edges of their tiles (bit-exact).

The bf16 fake-quant kernels work on 64-row x 256-element tiles and write a tile's scale bytes as
4-byte words where the four bytes are valid and the address is word aligned, single bytes otherwise.
Shapes here put every kind of edge under both scale layouts: a last column tile holding 1, 3 or 5
blocks, a last row tile of 1, 2 or 63 rows, row counts that are not multiples of 4 (block-major runs
not word aligned), a single row, and tensors of exactly one and of several whole tiles. For the
activation kernels (MXFP4 and NVFP4) and the weight kernel (learned scales, perturbed state,
sub-blocks 8 and 2): X_hat / W_hat bits, packed codes and scale bytes against the oracle.
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, device_bits, host_f32, oracle_bits, require_gpu

pytestmark = pytest.mark.gpu

MX, NV = 0, 1
B = {MX: 32, NV: 16}


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def O():
    from oracle import focus_oracle
    return focus_oracle


def shapes(fmt):
    b = B[fmt]
    return [(1, b), (2, 256 + b), (63, 256 + 3 * b), (64, 256), (65, 512 + 5 * b), (130, 2560 + b),
            (129, 256 * 3), (200, 8 * b)]


def data(seed, rows, K, heavy):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((rows, K))
    if heavy:
        X = X / np.sqrt((rng.standard_normal((rows, K, 3)) ** 2).sum(-1) / 3)
    X = X.astype(np.float32)
    X[rng.random((rows, K)) < 0.002] *= 25
    return torch.from_numpy(X).to(torch.bfloat16).cuda()


def block_major(a):
    return np.ascontiguousarray(a.T)


@pytest.mark.parametrize("fmt", [MX, NV])
def test_activation_tiles(F, O, fmt):
    for rows, K in shapes(fmt):
        announce(f"act tiles fmt={fmt} rows={rows} K={K}")
        X = data(rows * 31 + K, rows, K, fmt == NV)
        xo, co, so, _ = O.fq_act(host_f32(X), fmt)
        for layout in (0, 1):
            x_hat, codes, sbytes, _ = F.fakequant_fwd(X, fmt, 8, want_codes=True, want_scale_bytes=True,
                                                      scale_layout=layout)
            _, codes2, sbytes2, _ = F.fakequant_fwd(X, fmt, 8, want_codes=True, want_scale_bytes=True,
                                                    want_x_hat=False, scale_layout=layout)
            torch.cuda.synchronize()
            tag = f"rows={rows} K={K} layout={layout}"
            ref_b = so if layout == 0 else block_major(so)
            assert_bits_equal(device_bits(x_hat), oracle_bits(xo, torch.bfloat16), f"X_hat {tag}")
            for c_, s_ in ((codes, sbytes), (codes2, sbytes2)):
                assert_bits_equal(c_.cpu().numpy(), O.pack_codes(co), f"codes {tag}")
                assert_bits_equal(s_.cpu().numpy(), ref_b, f"scale bytes {tag}")


@pytest.mark.parametrize("fmt,sb", [(MX, 8), (MX, 2), (NV, 8), (NV, 2)])
def test_weight_tiles(F, O, fmt, sb):
    rng = np.random.default_rng(7 + sb + fmt)
    for rows, K in shapes(fmt):
        announce(f"weight tiles fmt={fmt} sb={sb} rows={rows} K={K}")
        W = (data(rows * 17 + K, rows, K, False).float() * 0.02).to(torch.bfloat16)
        Wh = host_f32(W)
        s_d, c_d, a_d = F.scales_init(W, fmt, sb)
        s_o, c_o, a_o = O.init_scales(Wh, fmt, sb)
        s_o = (s_o * np.exp2(rng.uniform(-0.5, 0.5, s_o.shape))).astype(np.float32)
        c_o = rng.uniform(0.75, 1.25, c_o.shape).astype(np.float32)
        s_d, c_d = torch.from_numpy(s_o).cuda(), torch.from_numpy(c_o).cuda()
        fq = O.fq_weight(Wh, fmt, sb, s_o, c_o, a_o)
        for layout in (0, 1):
            w_hat, codes, sbytes, _ = F.fakequant_fwd(W, fmt, sb, s_d, c_d, a_d, want_codes=True,
                                                      want_scale_bytes=True, scale_layout=layout)
            packed, eb = F.export_packed(W, fmt, sb, s_d, c_d, a_d, scale_layout=layout)
            torch.cuda.synchronize()
            tag = f"rows={rows} K={K} layout={layout}"
            ref_b = fq.scale_bytes if layout == 0 else block_major(fq.scale_bytes)
            assert_bits_equal(device_bits(w_hat), oracle_bits(fq.w_hat, torch.bfloat16), f"W_hat {tag}")
            for c_, s_ in ((codes, sbytes), (packed, eb)):
                assert_bits_equal(c_.cpu().numpy(), O.pack_codes(fq.codes), f"codes {tag}")
                assert_bits_equal(s_.cpu().numpy(), ref_b, f"scale bytes {tag}")


def test_nvfp4_activation_exact_ties(F, O):
    """NVFP4 activations whose quotients x / S are exactly E2M1 midpoints: a global maximum of 2688
    makes alpha = 1, a block maximum of 6 Delta (Delta an E4M3 value) makes S = Delta, and every
    t Delta (t a midpoint or a grid value, either sign) is exact in bf16, so u = t exactly and the tie
    rule decides each code (through the FMA-corrected quotient: S is in its range)."""
    deltas = [1.0, 1.125, 1.25, 1.375, 1.5, 1.625, 1.75, 1.875, 0.125, 0.3125, 2.5, 3.75, 0.0625, 7.0, 0.5625, 13.0]
    ts = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5, -5.0, 0.5, -3.0]
    rows, K = 66, 256
    X = np.zeros((rows, K), np.float32)
    X[0, 0] = 2688.0
    for r in range(1, rows):
        for b in range(K // 16):
            d = deltas[(r + b) % len(deltas)]
            blk = X[r, 16 * b:16 * (b + 1)]
            blk[0] = 6.0 * d if (r + b) % 2 == 0 else -6.0 * d  # the block maximum
            for j in range(1, 16):
                blk[j] = ts[(j + r + 3 * b) % len(ts)] * d
    Xg = torch.from_numpy(X).to(torch.bfloat16).cuda()
    assert np.array_equal(Xg.float().cpu().numpy(), X), "every value exact in bf16"
    announce(f"nvfp4 exact ties rows={rows} K={K}")
    x_hat, codes, sbytes, a_x = F.fakequant_fwd(Xg, NV, 8, want_codes=True, want_scale_bytes=True, want_alpha=True)
    torch.cuda.synchronize()
    xo, co, so, ao = O.fq_act(X, NV)
    assert ao == 1.0 and a_x.item() == 1.0
    assert_bits_equal(codes.cpu().numpy(), O.pack_codes(co), "codes")
    assert_bits_equal(sbytes.cpu().numpy(), so, "scale bytes")
    assert_bits_equal(device_bits(x_hat), oracle_bits(xo, torch.bfloat16), "X_hat")
    # the ties were really ties: |x| / S is a midpoint for at least half the elements past row 0
    S = np.repeat(np.array([[d for d in [deltas[(r + b) % len(deltas)] for b in range(K // 16)]]
                            for r in range(1, rows)], np.float32), 16, axis=1)
    u = np.abs(X[1:] / S)
    assert np.isin(u, [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]).mean() > 0.5
