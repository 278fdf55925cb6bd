"""E2M1 rounding of the HIP path on every bf16 value and around every grid midpoint (bit-exact).

Weight fake quantisation with S_fp = 1 and c = 1 under MXFP4 gives S_dq = 2^0 = 1 and u = w
exactly (Sec. 3.1, Eq. 1 and Eq. 6-7 with c = 1), so the codes the library returns are Q_E2M1(w)
of each weight element. The weights are fp32: all 65,536 bf16 bit patterns (signed zeros,
subnormals, infinities and NaNs included) and, for each grid value and each rounding midpoint
(0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5), its 16 nearest fp32 neighbours on either side, in both signs.
Codes, packed bytes and W_hat are compared bit for bit with the oracle's own threshold form of the
rounding (nearest, ties to the even index, saturation at 6, NaN to index 0).
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, host_bits32, require_gpu

pytestmark = pytest.mark.gpu

MX = 0


def grid_inputs() -> np.ndarray:
    patterns = (np.arange(65536, dtype=np.uint32) << 16).view(np.float32)
    points = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    near = []
    for p in points:
        up = dn = np.float32(p)
        near.append(up)
        for _ in range(16):
            up = np.nextafter(up, np.float32(np.inf))
            dn = np.nextafter(dn, np.float32(0.0))
            near += [up, dn]
    near = np.array(near, np.float32)
    vals = np.concatenate([patterns, near, -near])
    vals = np.concatenate([vals, np.zeros((-len(vals)) % 32, np.float32)])
    return vals.reshape(-1, 32)


def test_e2m1_rounding_every_bf16_and_midpoint():
    F = require_gpu()
    from oracle import focus_oracle as O
    W = grid_inputs()
    N, K = W.shape
    s = np.ones((N, K // 32), np.float32)
    c = np.ones((N, K // 8), np.float32)
    announce(f"e2m1 grid N={N} K={K}")
    Wg = torch.from_numpy(W).cuda()
    s_d, c_d = torch.from_numpy(s).cuda(), torch.from_numpy(c).cuda()
    w_hat, codes, sbytes, _ = F.fakequant_fwd(Wg, MX, 8, s_d, c_d, None, out_dtype=torch.float32,
                                              want_codes=True, want_scale_bytes=True)
    packed, _ = F.export_packed(Wg, MX, 8, s_d, c_d, None)
    torch.cuda.synchronize()
    fq = O.fq_weight(W, MX, 8, s, c, 1.0)
    ref_codes = O.pack_codes(fq.codes)
    assert_bits_equal(codes.cpu().numpy(), ref_codes, "codes")
    assert_bits_equal(packed.cpu().numpy(), ref_codes, "export codes")
    assert_bits_equal(host_bits32(w_hat), fq.w_hat.view(np.uint32), "W_hat")
    assert_bits_equal(sbytes.cpu().numpy(), fq.scale_bytes, "scale bytes")
