"""Pins for the oracle's reconstruction step: loss, dL/dW_hat and the straight-through gradients.

  * P11 finite differences: the STE gradient (Sec. 3.2, applied through Eq. 6-8) is the exact
    gradient of a smooth surrogate in which every rounding is replaced by its frozen residual
    (q = clamp(u, -6, 6) + r, S_dq = S_fp + (Q_fmt(S_fp0) - S_fp0)); central differences of that
    surrogate, written here independently, must reproduce the oracle's gradients. A dropped term,
    a wrong sign, a missing 1/c^2, a wrong alpha factor or a mis-indexed sub-block fails it.
  * brute force: the forward product, the mean-squared-error loss and dL/dW_hat in plain Python
    loops on a tiny layer.
  * P13 row separability: results for a subset of output rows equal the full computation's rows.
"""
import numpy as np
import pytest

MX, NV = 0, 1


def layer_inputs(oracle, fmt, seed, N=3, K=64, M=6, power_of_two_alpha=False):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    if power_of_two_alpha:
        # make max|W| = 2688 * 2^-12 so alpha = 2^-12 and every S_dq * c product is exact in fp32
        W = np.clip(W, -0.6, 0.6)
        W[0, 5] = np.float32(2688 * 2.0**-12)
    X = rng.standard_normal((M, K)).astype(np.float32)
    X[:, 3] *= 8
    x_hat, _, _, _ = oracle.fq_act(X, fmt)
    Y = (X.astype(np.float64) @ W.astype(np.float64).T)  # full-precision output of the layer
    return W, x_hat.astype(np.float64), Y


def perturbed_state(oracle, W, fmt, sb, seed):
    s_fp, c, alpha = oracle.init_scales(W, fmt, sb)
    rng = np.random.default_rng(seed)
    s_fp = (s_fp * np.exp2(rng.uniform(-0.5, 0.5, s_fp.shape))).astype(np.float32)
    # coefficients on a 1/64 grid keep S_dq * c exact in fp32 for the surrogate comparison
    c = (np.round(rng.uniform(0.75, 1.25, c.shape) * 64) / 64).astype(np.float32)
    return s_fp, c, alpha


class Surrogate:
    """Smooth stand-in for the fake-quantised layer around theta0 = (s_fp0, c0), in float64."""

    def __init__(self, oracle, W, X, Y, fmt, sb, s_fp0, c0, alpha):
        self.W = W.astype(np.float64)
        self.X, self.Y, self.fmt, self.sb, self.alpha = X, Y, fmt, sb, alpha
        self.B = 32 if fmt == MX else 16
        fq = oracle.fq_weight(W, fmt, sb, s_fp0, c0, alpha)
        q0 = oracle.e2m1_decode(fq.codes).astype(np.float64)
        # frozen residual of the scale format: S_dq(theta) = S_fp(theta) + (Q_fmt(S_fp0) - S_fp0)
        if fmt == MX:
            self.scale_resid = fq.s_dq.astype(np.float64) - s_fp0.astype(np.float64)
        else:
            delta = fq.s_dq.astype(np.float64) / alpha
            self.scale_resid = delta - s_fp0.astype(np.float64)
        u0 = self.w_over_sq(s_fp0.astype(np.float64), c0.astype(np.float64))
        self.r = q0 - np.clip(u0, -6.0, 6.0)  # frozen E2M1 rounding residual
        self.min_dist_to_clip = np.abs(np.abs(u0) - 6.0).min()

    def s_dq(self, s_fp):
        if self.fmt == MX:
            return s_fp + self.scale_resid
        return self.alpha * (s_fp + self.scale_resid)

    def w_over_sq(self, s_fp, c):
        sq = np.repeat(self.s_dq(s_fp), self.B // self.sb, axis=1) * c
        return self.W / np.repeat(sq, self.sb, axis=1)

    def loss(self, s_fp, c):
        q = np.clip(self.w_over_sq(s_fp, c), -6.0, 6.0) + self.r
        w_hat = q * np.repeat(self.s_dq(s_fp), self.B, axis=1)
        D = self.X @ w_hat.T - self.Y
        return (D * D).sum() / D.size


def central_differences(f, theta, rel_h=1e-6):
    g = np.zeros_like(theta)
    for i in range(theta.size):
        h = rel_h * max(abs(theta.flat[i]), 1e-30)
        tp, tm = theta.copy(), theta.copy()
        tp.flat[i] += h
        tm.flat[i] -= h
        g.flat[i] = (f(tp) - f(tm)) / (2 * h)
    return g


def assert_grad_close(got, ref, tol):
    scale = max(np.sqrt(np.mean(ref * ref)), 1e-300)
    err = np.abs(got - ref)
    assert np.all(err <= tol * np.maximum(np.abs(ref), scale)), (err.max(), scale)
    assert np.linalg.norm(got - ref) <= tol * np.linalg.norm(ref)


@pytest.mark.parametrize("fmt,sb", [(MX, 32), (MX, 8), (NV, 16), (NV, 8)])
@pytest.mark.parametrize("seed", [1, 2])
def test_p11_ste_gradients_match_surrogate_finite_differences(oracle, fmt, sb, seed):
    W, X, Y = layer_inputs(oracle, fmt, seed, power_of_two_alpha=(fmt == NV))
    s_fp0, c0, alpha = perturbed_state(oracle, W, fmt, sb, seed + 100)
    if fmt == NV:
        assert alpha == 2.0**-12
    sur = Surrogate(oracle, W, X, Y, fmt, sb, s_fp0, c0, alpha)
    assert sur.min_dist_to_clip > 1e-3  # no element sits on the clamp kink
    fq = oracle.fq_weight(W, fmt, sb, s_fp0, c0, alpha)
    res = oracle.recon_layer(X.astype(np.float32), fq.w_hat, Y, fq, fmt, sb, alpha)
    s64, c64 = s_fp0.astype(np.float64), c0.astype(np.float64)
    # the surrogate reproduces the oracle's loss at theta0
    assert abs(sur.loss(s64, c64) - res.loss_part) <= 1e-12 * res.loss_part
    fd_s = central_differences(lambda t: sur.loss(t, c64), s64)
    fd_c = central_differences(lambda t: sur.loss(s64, t), c64)
    assert_grad_close(res.grad_s, fd_s, 1e-6)
    assert_grad_close(res.grad_c, fd_c, 1e-6)


def test_bruteforce_loss_and_weight_gradient(oracle):
    W, X, Y = layer_inputs(oracle, MX, 7, N=2, K=32, M=3)
    s_fp, c, alpha = perturbed_state(oracle, W, MX, 8, 8)
    fq = oracle.fq_weight(W, MX, 8, s_fp, c, alpha)
    res = oracle.recon_layer(X.astype(np.float32), fq.w_hat, Y, fq, MX, 8, alpha, keep_dy=True)
    M, K = X.shape
    N = W.shape[0]
    yhat = [[sum(float(X[t][k]) * float(fq.w_hat[n][k]) for k in range(K)) for n in range(N)]
            for t in range(M)]
    loss = sum((yhat[t][n] - Y[t][n]) ** 2 for t in range(M) for n in range(N)) / (M * N)
    assert abs(loss - res.loss_part) <= 1e-12 * loss
    for n in range(N):
        for k in range(K):
            g = sum(2.0 * (yhat[t][n] - Y[t][n]) / (M * N) * float(X[t][k]) for t in range(M))
            assert abs(g - res.G[n, k]) <= 1e-12 * max(abs(g), 1e-30) + 1e-300
        for t in range(M):
            assert abs(2.0 * (yhat[t][n] - Y[t][n]) / (M * N) - res.d_y[t, n]) <= 1e-15


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p13_row_subset_equals_full(oracle, fmt):
    W, X, Y = layer_inputs(oracle, fmt, 9, N=12, K=96 if fmt == MX else 80, M=40)
    s_fp, c, alpha = perturbed_state(oracle, W, fmt, 8, 10)
    fq = oracle.fq_weight(W, fmt, 8, s_fp, c, alpha)
    full = oracle.recon_layer(X.astype(np.float32), fq.w_hat, Y, fq, fmt, 8, alpha, chunk=7)
    rows = [0, 5, 11]
    part = oracle.recon_layer(X.astype(np.float32), fq.w_hat, Y, fq, fmt, 8, alpha, rows=rows)
    np.testing.assert_allclose(part.grad_s, full.grad_s[rows], rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(part.grad_c, full.grad_c[rows], rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(part.col_sq, full.col_sq[rows], rtol=1e-12)
    assert abs(full.col_sq.sum() / (40 * 12) - full.loss_part) <= 1e-12 * full.loss_part


@pytest.mark.parametrize("fmt", [MX, NV])
def test_p6_block_coefficient_gradient_is_sum_of_subblocks(oracle, fmt):
    B = 32 if fmt == MX else 16
    W, X, Y = layer_inputs(oracle, fmt, 13, N=4, K=64, M=8)
    s_fp, c8, alpha = perturbed_state(oracle, W, fmt, 8, 14)
    c_block = c8[:, :: B // 8].copy()
    c_bcast = np.repeat(c_block, B // 8, axis=1)
    fa = oracle.fq_weight(W, fmt, B, s_fp, c_block, alpha)
    fb = oracle.fq_weight(W, fmt, 8, s_fp, c_bcast, alpha)
    ra = oracle.recon_layer(X.astype(np.float32), fa.w_hat, Y, fa, fmt, B, alpha)
    rb = oracle.recon_layer(X.astype(np.float32), fb.w_hat, Y, fb, fmt, 8, alpha)
    np.testing.assert_allclose(ra.grad_c, rb.grad_c.reshape(4, -1, B // 8).sum(axis=2),
                               rtol=1e-12, atol=1e-14 * np.abs(ra.grad_c).max())
    np.testing.assert_allclose(ra.grad_s, rb.grad_s, rtol=1e-12)


def test_zero_residual_gives_zero_loss_and_gradients(oracle):
    W, X, _ = layer_inputs(oracle, MX, 15, N=4, K=64, M=8)
    s_fp, c, alpha = perturbed_state(oracle, W, MX, 8, 16)
    fq = oracle.fq_weight(W, MX, 8, s_fp, c, alpha)
    Y = X @ fq.w_hat.astype(np.float64).T  # the quantised layer reproduces its target exactly
    res = oracle.recon_layer(X.astype(np.float32), fq.w_hat, Y, fq, MX, 8, alpha)
    assert res.loss_part == 0.0 and not res.grad_s.any() and not res.grad_c.any()
