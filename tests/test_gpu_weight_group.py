"""GPU parity of the grouped weight fake quantisation (focus_fakequant_weights), bit-exact.

One call fake-quantises several linear layers in one launch. Checked here: layers of different
shapes in one group (ragged row and column tiles, a one-row layer, an empty layer) against the oracle
in both scale layouts and for every output combination (codes + bytes, W_hat, all three); the group
against one focus_fakequant_fwd / focus_export_packed call per layer on the full-size linears of the
hidden-8192 MXFP4 block and of the hidden-2560 NVFP4 block; the sixteen-layer maximum; fp32 weights
(one launch per layer behind the same call); the domain flag raised by one bad layer of a group.
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


def block_major(a):
    return np.ascontiguousarray(a.T)


def shapes(fmt):
    b = B[fmt]
    return [(63, 256 + 3 * b), (1, b), (64, 256), (0, 256), (130, 2560 + b), (200, 8 * b), (5, 512)]


def perturbed_state(O, Wh, fmt, sb, rng):
    s, c, a = O.init_scales(Wh, fmt, sb)
    s = (s * np.exp2(rng.uniform(-0.5, 0.5, s.shape))).astype(np.float32)
    c = rng.uniform(0.75, 1.25, c.shape).astype(np.float32)
    return s, c, a


def weights(seed, rows, K, dtype=torch.bfloat16):
    g = torch.Generator().manual_seed(seed)
    W = torch.randn(rows, K, generator=g) * 0.02
    W[torch.rand(rows, K, generator=g) < 0.002] *= 25
    return W.to(dtype).cuda()


@pytest.mark.parametrize("fmt,sb", [(MX, 8), (MX, 2), (NV, 8), (NV, 2)])
def test_group_matches_oracle(F, O, fmt, sb):
    rng = np.random.default_rng(11 + 3 * fmt + sb)
    layers, refs = [], []
    for i, (rows, K) in enumerate(shapes(fmt)):
        W = weights(100 * i + K, rows, K)
        _, _, a_d = F.scales_init(W, fmt, sb) if rows else (None, None, torch.ones(1, device="cuda"))
        Wh = host_f32(W)
        s, c, a = perturbed_state(O, Wh, fmt, sb, rng) if rows else (
            np.zeros((0, K // B[fmt]), np.float32), np.zeros((0, K // sb), np.float32), 1.0)
        if rows:
            assert float(a_d.item()) == float(a)
        layers.append(dict(W=W, s_fp=torch.from_numpy(s).cuda(), c=torch.from_numpy(c).cuda(), alpha=a_d))
        refs.append(O.fq_weight(Wh, fmt, sb, s, c, a) if rows else None)
    for layout in (0, 1):
        for mode in ("packed", "w_hat", "all"):
            announce(f"weight group fmt={fmt} sb={sb} layout={layout} outputs={mode}")
            group = []
            for l in layers:
                rows, K = l["W"].shape
                g = dict(l)
                if mode != "w_hat":
                    g["codes"] = torch.empty(rows, K // 2, dtype=torch.uint8, device="cuda")
                    nb = K // B[fmt]
                    g["scale_bytes"] = torch.empty(*((rows, nb) if layout == 0 else (nb, rows)), dtype=torch.uint8,
                                                   device="cuda")
                if mode != "packed":
                    g["W_hat"] = torch.empty(rows, K, dtype=torch.bfloat16, device="cuda")
                group.append(g)
            F.fakequant_weights(group, fmt, sb, scale_layout=layout)
            torch.cuda.synchronize()
            for i, (g, ref) in enumerate(zip(group, refs)):
                if ref is None:
                    continue
                tag = f"layer {i} {tuple(g['W'].shape)} layout={layout} {mode}"
                if "W_hat" in g:
                    assert_bits_equal(device_bits(g["W_hat"]), oracle_bits(ref.w_hat, torch.bfloat16), f"W_hat {tag}")
                if "codes" in g:
                    assert_bits_equal(g["codes"].cpu().numpy(), O.pack_codes(ref.codes), f"codes {tag}")
                    want = ref.scale_bytes if layout == 0 else block_major(ref.scale_bytes)
                    assert_bits_equal(g["scale_bytes"].cpu().numpy(), want, f"scale bytes {tag}")


def full_size_layers(F, workload, perturb):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS[workload]
    out = []
    for lin in w.linears:
        W = synth.weight(w, lin, device="cuda")
        s, c, a = F.scales_init(W, w.fmt, w.sub_block)
        if perturb:
            g = torch.Generator(device="cuda").manual_seed(lin.N + lin.K)
            s = s * torch.exp2(torch.rand(s.shape, generator=g, device="cuda") - 0.5)
            c = 0.75 + 0.5 * torch.rand(c.shape, generator=g, device="cuda")
        out.append((lin, dict(W=W, s_fp=s, c=c, alpha=a)))
    return w, out


def test_group_equals_per_layer_export_hidden8192(F):
    """The benchmark's packed step: every linear of the hidden-8192 MXFP4 block in one launch, K-slab codes
    and block-major bytes, against one export call per linear (whole tensors, on the device)."""
    for perturb in (False, True):
        w, layers = full_size_layers(F, "block8192_mxfp4", perturb)
        announce(f"weight group vs per-layer export, block8192_mxfp4, perturbed={perturb}")
        group, ref = [], []
        for lin, l in layers:
            N, K = l["W"].shape
            g = dict(l, codes=torch.empty(*F.codes_shape(N, K, F.CODES_K_SLAB), dtype=torch.uint8, device="cuda"),
                     scale_bytes=torch.empty(K // 32, N, dtype=torch.uint8, device="cuda"))
            group.append(g)
            ref.append(F.export_packed(l["W"], w.fmt, w.sub_block, l["s_fp"], l["c"], l["alpha"],
                                       scale_layout=F.SCALES_BLOCK_MAJOR, code_layout=F.CODES_K_SLAB))
        F.fakequant_weights(group, w.fmt, w.sub_block, scale_layout=F.SCALES_BLOCK_MAJOR, code_layout=F.CODES_K_SLAB)
        torch.cuda.synchronize()
        for (lin, _), g, (codes, sbytes) in zip(layers, group, ref):
            assert torch.equal(g["codes"], codes), f"codes {lin.name}"
            assert torch.equal(g["scale_bytes"], sbytes), f"scale bytes {lin.name}"
        del layers, group, ref
        torch.cuda.empty_cache()


def test_group_equals_per_layer_nvfp4_w_hat(F):
    """The NVFP4 block's bf16-operand step: W_hat of every linear in one launch against fakequant_fwd."""
    w, layers = full_size_layers(F, "block2560_nvfp4", True)
    announce("weight group vs per-layer fakequant_fwd, block2560_nvfp4 W_hat")
    group = [dict(l, W_hat=torch.empty_like(l["W"])) for _, l in layers]
    F.fakequant_weights(group, w.fmt, w.sub_block)
    torch.cuda.synchronize()
    for (lin, l), g in zip(layers, group):
        ref = F.fakequant_fwd(l["W"], w.fmt, w.sub_block, l["s_fp"], l["c"], l["alpha"])[0]
        assert torch.equal(g["W_hat"].view(torch.int16), ref.view(torch.int16)), f"W_hat {lin.name}"


def test_sixteen_layers_and_fp32_weights(F):
    fmt, sb = MX, 8
    for dtype in (torch.bfloat16, torch.float32):
        announce(f"weight group of 16 layers, {dtype}")
        group, ref = [], []
        for i in range(F.MAX_WEIGHT_LAYERS):
            rows, K = 3 + 17 * i, 32 * (1 + i % 5)
            W = weights(7 * i + 1, rows, K, dtype)
            s, c, a = F.scales_init(W, fmt, sb)
            c = 0.8 + 0.4 * torch.rand(c.shape, device="cuda")
            group.append(dict(W=W, s_fp=s, c=c, codes=torch.empty(rows, K // 2, dtype=torch.uint8, device="cuda"),
                              scale_bytes=torch.empty(rows, K // 32, dtype=torch.uint8, device="cuda"),
                              W_hat=torch.empty(rows, K, dtype=dtype, device="cuda")))
            ref.append(F.fakequant_fwd(W, fmt, sb, s, c, want_codes=True, want_scale_bytes=True))
        F.fakequant_weights(group, fmt, sb)
        torch.cuda.synchronize()
        for i, (g, (w_hat, codes, sbytes, _)) in enumerate(zip(group, ref)):
            assert np.array_equal(device_bits(g["W_hat"]), device_bits(w_hat)), f"W_hat layer {i}"
            assert torch.equal(g["codes"], codes) and torch.equal(g["scale_bytes"], sbytes), f"packed layer {i}"
    with pytest.raises(F.FocusError) as e:
        F.fakequant_weights(group + group[:1], fmt, sb)
    assert e.value.status == F.ERR_SHAPE


def test_group_domain_flag(F):
    fmt, sb = MX, 8
    announce("weight group domain flag")
    ws = F.workspace(F.workspace_size(F.CALL_FAKEQUANT_WEIGHTS, F.qconfig(fmt, sb)))
    group = []
    for i in range(3):
        W = weights(i, 64 + i, 256)
        s, c, a = F.scales_init(W, fmt, sb)
        group.append(dict(W=W, s_fp=s, c=c, codes=torch.empty(64 + i, 128, dtype=torch.uint8, device="cuda")))
    F.fakequant_weights(group, fmt, sb, ws=ws)
    assert F.check_flags(ws) == F.OK
    group[2]["c"] = group[2]["c"].clone()
    group[2]["c"][5, 7] = 0.0
    F.fakequant_weights(group, fmt, sb, ws=ws)
    assert F.check_flags(ws) == F.ERR_DOMAIN
    assert F.check_flags(ws) == F.OK
