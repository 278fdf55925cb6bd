"""GPU parity of the end-to-end chaining calls at the benchmark's full sizes, on sampled rows.

Each sampled output row depends only on its own input row (and, under NVFP4, on the tensor-wide
absmax), so the oracle computes the sampled rows one by one: the first, the last and seeded rows in
between (the last row exercises the largest offsets of each tensor).
  * focus_recon_gemm_dx on the hidden-8192 block's largest linears, gate_proj (28672 x 8192) and
    down_proj (8192 x 28672), at 131,072 tokens: dX_hat = dY W_hat within 2e-2 on the sampled rows
    (bf16 output). The W_hat operand is the layer's seeded synthetic weight itself: any bf16 matrix
    exercises the same product, and no input of the oracle comes from the library;
  * focus_fakequant_act_bwd on the widest block input the benchmark passes, down_in of the hidden-8192
    block (131,072 x 28,672, MXFP4 with the rounded-up and the OCP floor E8M0 rule), and on the NVFP4
    block's down_in (65,536 x 9,728, Student-t(3) activations): dX bit for bit on the sampled rows.
    The NVFP4 mask needs the tensor scale of the whole tensor: its absmax is taken on the host and
    given to the oracle as one extra row, so the oracle forms alpha from it as it does for any input;
  * focus_kl_top on 8,192 tokens x 151,936 logits with k = 1000 in bf16 (the benchmark's call): dZ on
    the sampled rows within 2e-2 and exactly zero off each row's teacher top-k set. (The loss, a mean
    over all rows, is checked against the oracle at the smaller sizes of the chaining tests.)
"""
import numpy as np
import pytest
import torch

from gpu_common import announce, assert_bits_equal, assert_close, device_bits, host_f32, require_gpu

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def C():
    from oracle import chain_oracle
    return chain_oracle


def sample_rows(M, seed, n=6):
    rng = np.random.default_rng(seed)
    return np.array(sorted({0, M - 1} | set(rng.choice(M, size=n, replace=False).tolist())), dtype=np.int64)


def seeded_randn(shape, seed, scale, dtype=torch.bfloat16):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn(*shape, generator=g, device="cuda") * scale).to(dtype)


@pytest.mark.parametrize("name", ["gate_proj", "down_proj"])
def test_dx_fullsize(F, C, name):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block8192_mxfp4"]
    lin = next(l for l in w.linears if l.name == name)
    M, N, K = w.M, lin.N, lin.K
    announce(f"dx full size block8192_mxfp4 {name}: M={M} N={N} K={K}")
    W_hat = synth.weight(w, lin, device="cuda")
    dY = seeded_randn((M, N), 101 + N, 1e-3)
    dX = F.recon_gemm_dx(dY, W_hat)
    torch.cuda.synchronize()
    rows = sample_rows(M, N + K)
    idx = torch.from_numpy(rows).cuda()
    got = host_f32(dX.index_select(0, idx))
    ref = C.recon_dx(host_f32(dY.index_select(0, idx)), host_f32(W_hat))
    assert_close(got, ref, TOL, f"dX_hat rows {rows.tolist()}")


def host_absmax(X, chunk=8192):
    """max |X| over the whole device tensor, taken on the host chunk by chunk (exact)."""
    m = 0.0
    for i in range(0, X.shape[0], chunk):
        m = max(m, float(X[i:i + chunk].cpu().float().abs().max()))
    return m


@pytest.mark.parametrize("workload,fmt,floor", [("block8192_mxfp4", 0, 0), ("block8192_mxfp4", 0, 1),
                                                ("block2560_nvfp4", 1, 0)], ids=["mx", "mx_floor", "nv"])
def test_act_bwd_fullsize(F, C, workload, fmt, floor):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    X = synth.activation(w, "down_in", device="cuda")
    M, K = X.shape
    announce(f"act bwd full size {workload} down_in: M={M} K={K} fmt={fmt} floor={floor}")
    g = seeded_randn((M, K), 7 + K + floor, 1.0)
    dX = F.fakequant_act_bwd(X, g, fmt, e8m0_rounding=floor)
    torch.cuda.synchronize()
    rows = sample_rows(M, K + fmt + floor)
    idx = torch.from_numpy(rows).cuda()
    Xr = host_f32(X.index_select(0, idx))
    if fmt == 1:
        # the tensor scale comes from the whole tensor: one extra row carrying its absmax
        amax = host_absmax(X)
        assert amax >= np.abs(Xr).max()
        extra = np.zeros((1, K), np.float32)
        extra[0, 0] = amax
        m = C.act_ste_mask(np.vstack([Xr, extra]), fmt)[:-1]
    else:
        m = C.act_ste_mask(Xr, fmt, e8m0_floor=bool(floor))
    gr = host_f32(g.index_select(0, idx))
    ref = np.where(m != 0, gr, np.float32(0.0)).astype(np.float32)  # a dropped gradient is +0
    got = dX.index_select(0, idx)
    assert_bits_equal(device_bits(got), device_bits(torch.from_numpy(ref).to(torch.bfloat16)), f"dX rows {rows.tolist()}")
    if fmt == 0 and not floor:
        assert np.all(m[Xr != 0] == 1.0)  # rounded-up E8M0: no element clips
    else:
        assert (m == 0).any()


def test_kl_top_fullsize(F, C):
    T, V, k = 8192, 151936, 1000
    announce(f"kl_top full size T={T} V={V} k={k} bf16")
    Zt = seeded_randn((T, V), 11, 3.0)
    Zs = (Zt.float() + seeded_randn((T, V), 12, 1.0, torch.float32)).to(torch.bfloat16)
    dZ, loss = F.kl_top(Zs, Zt, k)
    torch.cuda.synchronize()
    assert np.isfinite(loss.item()) and loss.item() > 0
    rows = sample_rows(T, 13)
    idx = torch.from_numpy(rows).cuda()
    Zs_r, Zt_r = host_f32(Zs.index_select(0, idx)), host_f32(Zt.index_select(0, idx))
    got = host_f32(dZ.index_select(0, idx))
    for i, r in enumerate(rows):
        _, d1 = C.kl_top(Zs_r[i:i + 1], Zt_r[i:i + 1], k)  # one row: dZ scaled by 1 / 1
        ref = d1[0] / T                                       # the full call's 1 / T (a power of two)
        assert_close(got[i:i + 1], ref[None], TOL, f"dZ row {r}")
        assert not np.any((got[i] != 0) & (ref == 0)), f"dZ row {r} nonzero off the teacher's top-k set"
