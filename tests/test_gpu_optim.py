"""GPU parity of the AdamW kernel and of the calibration step (Sec. 4.1: AdamW, constant learning
rate) against the CPU oracle.

  * focus_adamw_step on ragged lengths (1 to 2^20 + 3 elements), linear and log2 domain, with and
    without weight decay, five chained steps from the same inputs: parameter and both moments
    within 1e-5 (fp32 arithmetic against float64);
  * the benchmark's largest optimizer tensor (29.4 M coefficients), sampled elements after three
    chained steps on the whole tensor, within 1e-5;
  * the log2 domain's guard: non-positive or non-finite parameters raise the domain flag and stay
    unchanged, the rest are updated;
  * the calibration step of calib.BlockCalibrator, teacher-forced: at each of three steps the GPU
    starts from the oracle's state (scales, coefficients, moments); loss and moments within 1e-5,
    and the stepped log2 parameters within 1e-5 plus what the gradient's own 1e-5 tolerance can move
    an AdamW step (its division by sqrt(v_hat) + eps magnifies gradients near eps), for the
    learned-scale, CRS and CRS+DGS variants under MXFP4 and NVFP4 on the fp32 256x256 layer;
  * one epoch (39 steps of 16,384 tokens) on the hidden-2560 MXFP4 block with correlated (low-rank)
    inputs: the held-out reconstruction loss of every learned variant ends below RTN's, the
    training loss falls, and CRS+DGS ends below the learned-scale baseline.
"""
import dataclasses

import numpy as np
import pytest
import torch

from gpu_common import announce, assert_close, host_f32, require_gpu

pytestmark = pytest.mark.gpu

TOL = 1e-5


def f32(x: float) -> float:
    """The library's hyper-parameters are fp32 (focus_adamw_config): the oracle gets the same values."""
    return float(np.float32(x))


B1, B2, EPS = f32(0.9), f32(0.999), f32(1e-8)


@pytest.fixture(scope="module")
def F():
    return require_gpu()


@pytest.fixture(scope="module")
def OO():
    from oracle import optim_oracle
    return optim_oracle


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1027, (1 << 20) + 3])
@pytest.mark.parametrize("log2", [False, True])
@pytest.mark.parametrize("wd", [0.0, 1e-2])
def test_adamw_kernel(F, OO, n, log2, wd):
    announce(f"adamw n={n} log2={log2} wd={wd}")
    rng = np.random.default_rng(n * 7 + int(log2) * 3 + int(wd * 100))
    p0 = (np.exp2(rng.normal(-7, 2, n)) if log2 else rng.normal(1, 0.2, n)).astype(np.float32)
    grads = [(rng.normal(size=n) * 10.0 ** rng.uniform(-10, -2, n)).astype(np.float32) for _ in range(5)]
    lr, wd = f32(2e-2 if log2 else 5e-2), f32(wd)
    p, m, v = (torch.from_numpy(a).cuda() for a in (p0, np.zeros(n, np.float32), np.zeros(n, np.float32)))
    ws = F.workspace(256)
    po, mo, vo = p0.astype(np.float64), np.zeros(n), np.zeros(n)
    for t, g in enumerate(grads, start=1):
        F.adamw_step(p, torch.from_numpy(g).cuda(), m, v, t, lr, weight_decay=wd, log2_domain=log2, ws=ws)
        po, mo, vo = OO.adamw(po, g, mo, vo, t, lr, B1, B2, EPS, weight_decay=wd, log2_domain=log2)
        torch.cuda.synchronize()
        assert_close(host_f32(p), po, TOL, f"param t={t}")
        assert_close(host_f32(m), mo, TOL, f"exp_avg t={t}")
        assert_close(host_f32(v), vo, TOL, f"exp_avg_sq t={t}")
    assert F.check_flags(ws) == F.OK


def test_adamw_fullsize_sampled(F, OO):
    """The largest tensor the benchmark steps: the coefficients of the hidden-8192 block's gate_proj
    (28,672 x 1,024 = 29.4 M, sub-blocks of 8) in the log2 domain at the paper's MXFP4 rate, three
    chained steps on the whole tensor; parameter and moments of sampled elements (the first, the last
    and 4,096 seeded ones) within 1e-5 of the oracle's element-wise steps."""
    n = 28672 * (8192 // 8)
    announce(f"adamw full size n={n} log2")
    rng = np.random.default_rng(17)
    idx = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 4096, replace=False)])).astype(np.int64)
    di = torch.from_numpy(idx).cuda()
    g = torch.Generator(device="cuda").manual_seed(19)
    p = torch.exp2(torch.randn(n, generator=g, device="cuda") * 0.1)  # coefficients near 1
    m, v = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    lr = f32(5e-2)
    ws = F.workspace(256)
    po, mo, vo = host_f32(p.index_select(0, di)).astype(np.float64), np.zeros(len(idx)), np.zeros(len(idx))
    for t in range(1, 4):
        grad = torch.randn(n, generator=g, device="cuda") * 1e-4
        F.adamw_step(p, grad, m, v, t, lr, log2_domain=True, ws=ws)
        po, mo, vo = OO.adamw(po, host_f32(grad.index_select(0, di)), mo, vo, t, lr, B1, B2, EPS, log2_domain=True)
        torch.cuda.synchronize()
        assert_close(host_f32(p.index_select(0, di)), po, TOL, f"param t={t}")
        assert_close(host_f32(m.index_select(0, di)), mo, TOL, f"exp_avg t={t}")
        assert_close(host_f32(v.index_select(0, di)), vo, TOL, f"exp_avg_sq t={t}")
    assert F.check_flags(ws) == F.OK


def test_adamw_log2_domain_guard(F, OO):
    announce("adamw log2 guard")
    p0 = np.array([0.5, 0.0, -1.0, np.inf, np.nan, 2.0, 1e-30, 3.0], np.float32)
    g = np.full(8, 0.1, np.float32)
    p, m, v = torch.from_numpy(p0).cuda(), torch.zeros(8, device="cuda"), torch.zeros(8, device="cuda")
    ws = F.workspace(256)
    F.adamw_step(p, torch.from_numpy(g).cuda(), m, v, 1, 2e-2, log2_domain=True, ws=ws)
    assert F.check_flags(ws) == F.ERR_DOMAIN
    got = host_f32(p)
    bad = [1, 2, 3, 4]
    np.testing.assert_array_equal(got[bad], p0[bad])
    good = [0, 5, 6, 7]
    ref, _, _ = OO.adamw(p0[good].astype(np.float64), g[good], np.zeros(4), np.zeros(4), 1, f32(2e-2), B1, B2, EPS,
                         log2_domain=True)
    assert_close(got[good], ref, TOL, "guarded step")
    assert F.check_flags(ws) == F.OK  # the flag was cleared


def step_bound(OO, p, g, m, v, t, lr, log2):
    """Error bound of the stepped parameter (in log2 p when log2, else p) given the gradient
    tolerance: AdamW divides by sqrt(v_hat) + eps, so where |g| is near eps a gradient within
    TOL * max(|g|, rms g) of the oracle's moves the step by up to the difference below (taken
    from the oracle at g -/+ that tolerance), on top of TOL relative to the parameter itself."""
    g = np.asarray(g, np.float64)
    gtol = TOL * np.maximum(np.abs(g), np.sqrt(np.mean(g * g)))
    fwd = (lambda x: np.log2(x)) if log2 else (lambda x: x)
    th = lambda gg: fwd(OO.adamw(p, gg, m, v, t, lr, B1, B2, EPS, 0.0, log2)[0])
    base = th(g)
    spread = np.maximum(np.abs(th(g + gtol) - base), np.abs(th(g - gtol) - base))
    # TOL relative on the fp32 parameter p; in log2 p that is TOL / ln 2 absolute
    own = TOL / np.log(2.0) if log2 else TOL * np.maximum(np.abs(base), np.sqrt(np.mean(base * base)))
    return base, spread + own


def assert_within(got, ref, bound, what):
    err = np.abs(np.asarray(got, np.float64) - ref)
    worst = float(np.max(err / bound))
    assert worst <= 1.0, f"{what}: error {float(err.max()):.3e}, {worst:.2f} x its bound"


def fp32_layer(fmt):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["linear256_mxfp4_f32"]
    if fmt == 1:
        w = dataclasses.replace(w, name="linear256_nvfp4_f32", fmt=1)
    return w


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("variant", ["scale", "crs", "crs_dgs"])
def test_calibration_step_teacher_forced(F, OO, fmt, variant):
    from oracle import focus_oracle as O
    from paper_2608_01847_amd import calib, synth
    w = fp32_layer(fmt)
    lin = w.linears[0]
    announce(f"calib step fmt={fmt} {variant}")
    cal = calib.BlockCalibrator(w, variant)
    L = cal.layers[lin.name]
    W = host_f32(L.W)
    lr_s, lr_c = (f32(x) for x in calib.LEARNING_RATES[fmt])
    P = OO.LayerParams.init(W, fmt, cal.sb)
    for k in range(3):
        X = synth.activation_batch(w, lin.source, k, device="cpu")
        Xh = X.numpy()
        Y_ref = (Xh.astype(np.float64) @ W.astype(np.float64).T).astype(np.float32)
        loss_o, P_next, res = OO.calib_step(Xh, W, Y_ref, fmt, cal.sb, P, k + 1, lr_s, lr_c, cal.learn_s,
                                            cal.learn_c, cal.use_c, bf16=False, betas=(B1, B2), eps=EPS)
        # the GPU starts from the oracle's state
        for name in ("s", "c", "ms", "vs", "mc", "vc"):
            getattr(L, name).copy_(torch.from_numpy(getattr(P, name)))
        cal.t = k + 1
        Xd = X.cuda()
        x_hat = F.fakequant_fwd(Xd, fmt, cal.sb, ws=cal.ws)[0]
        loss = cal.layer_step(L, x_hat, Xd, True, Y_ref=torch.from_numpy(Y_ref).cuda())
        torch.cuda.synchronize()
        assert abs(loss.item() - loss_o) <= TOL * loss_o, (k, loss.item(), loss_o)
        if cal.learn_s:
            ref, bound = step_bound(OO, P.s, res.grad_s, P.ms, P.vs, k + 1, lr_s, True)
            assert_within(np.log2(host_f32(L.s)), ref, bound, f"log2 s step {k}")
            assert_close(host_f32(L.ms), P_next.ms, TOL, f"m_s step {k}")
            assert_close(host_f32(L.vs), P_next.vs, TOL, f"v_s step {k}")
        if cal.learn_c:
            ref, bound = step_bound(OO, P.c, res.grad_c, P.mc, P.vc, k + 1, lr_c, True)
            assert_within(np.log2(host_f32(L.c)), ref, bound, f"log2 c step {k}")
            assert_close(host_f32(L.mc), P_next.mc, TOL, f"m_c step {k}")
        else:
            np.testing.assert_array_equal(host_f32(L.c), P.c)
        P = P_next
    cal.check_domain()


def test_epoch_on_correlated_inputs_lowers_the_loss(F):
    # with correlated input channels every learned variant ends below RTN on the held-out batch and
    # the finer coefficients help most (the ordering of the paper's ablation); with independent
    # channels c = 1 is already optimal per element, so no such claim is made there
    from paper_2608_01847_amd import calib, synth
    # (the hidden-2560 block itself: on blocks narrowed to a few hundred input features the
    # coefficients' gain is not reliable)
    w = dataclasses.replace(synth.WORKLOADS["block2560_mxfp4"], x_kind="lowrank")
    announce("calib epoch, hidden-2560 block, low-rank inputs, 16384 tokens per step")
    res = calib.ablation(w, steps=calib.EPOCH_STEPS, M=16384, eval_M=16384)
    rel = {v: r.get("block_rel_to_rtn") for v, r in res.items()}
    print(rel)
    for v in ("scale", "crs", "crs_dgs"):
        assert rel[v] < 1.0, (v, res[v]["rel_to_rtn"])
        assert res[v]["train_curve"][-1] < res[v]["train_curve"][0], (v, res[v]["train_curve"])
    assert rel["crs_dgs"] < rel["scale"], rel
