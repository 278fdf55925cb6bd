"""Pins of the optimizer oracle (Sec. 4.1: AdamW, constant learning rate) against what fixes it from
outside: PyTorch's own AdamW implementation (float64, CPU), the closed form of the first step, and
finite differences for the log2-domain chain rule.

A planted mistake in the oracle (a dropped bias correction, a weight decay applied after the step or
coupled into the gradient, a missing ln 2, the root of the uncorrected second moment) fails one of
these; test_planted_mistakes_are_caught checks that on copies of the formula.
"""
import numpy as np
import pytest
import torch

from oracle import optim_oracle as OO


def torch_adamw(p0, grads, lr, betas, eps, wd):
    p = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=lr, betas=betas, eps=eps, weight_decay=wd, foreach=False)
    out = []
    for g in grads:
        opt.zero_grad()
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        st = opt.state[p]
        out.append((p.detach().numpy().copy(), st["exp_avg"].numpy().copy(), st["exp_avg_sq"].numpy().copy()))
    return out


@pytest.mark.parametrize("wd", [0.0, 1e-2])
@pytest.mark.parametrize("betas,eps", [((0.9, 0.999), 1e-8), ((0.8, 0.95), 1e-6)])
def test_matches_torch_adamw(wd, betas, eps):
    rng = np.random.default_rng(3)
    p0 = rng.normal(size=257)
    grads = [rng.normal(size=257) * 10.0 ** rng.uniform(-9, 0, 257) for _ in range(6)]
    ref = torch_adamw(p0, grads, 5e-2, betas, eps, wd)
    p, m, v = p0, np.zeros_like(p0), np.zeros_like(p0)
    for t, (g, (rp, rm, rv)) in enumerate(zip(grads, ref), start=1):
        p, m, v = OO.adamw(p, g, m, v, t, 5e-2, betas[0], betas[1], eps, wd)
        np.testing.assert_allclose(p, rp, rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(m, rm, rtol=1e-13, atol=0)
        np.testing.assert_allclose(v, rv, rtol=1e-13, atol=0)


def test_first_step_closed_form():
    # t = 1: m_hat = g and v_hat = g^2, so the step is lr * g / (|g| + eps) after the decay
    rng = np.random.default_rng(4)
    p = rng.normal(size=100)
    g = rng.normal(size=100) * 10.0 ** rng.uniform(-10, 1, 100)
    lr, eps, wd = 2e-2, 1e-8, 0.1
    p1, _, _ = OO.adamw(p, g, np.zeros(100), np.zeros(100), 1, lr, eps=eps, weight_decay=wd)
    np.testing.assert_allclose(p1, p * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-12, atol=1e-16)


def loss_and_grad(p, a, b):
    """A smooth loss of a positive parameter and its gradient in p."""
    return np.sum(a * (np.log(p) - b) ** 2 + 0.1 * p), 2 * a * (np.log(p) - b) / p + 0.1


def test_log2_domain_follows_finite_differences():
    # in the log2 domain the oracle must be AdamW on theta = log2 p with dL/dtheta; here dL/dtheta is
    # taken by central differences of L(2^theta) and the theta-trajectory comes from PyTorch's AdamW
    rng = np.random.default_rng(5)
    n = 64
    a, b = rng.uniform(0.5, 2, n), rng.normal(size=n)
    p0 = np.exp2(rng.normal(-6, 1, n))
    lr = 2e-2
    theta = torch.tensor(np.log2(p0), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([theta], lr=lr, weight_decay=0.0, foreach=False)
    p, m, v = p0, np.zeros(n), np.zeros(n)
    h = 1e-6
    for t in range(1, 6):
        th = theta.detach().numpy()
        fd = np.array([(loss_and_grad(np.exp2(th[i] + h), a[i], b[i])[0] - loss_and_grad(np.exp2(th[i] - h), a[i], b[i])[0])
                       / (2 * h) for i in range(n)])
        opt.zero_grad()
        theta.grad = torch.tensor(fd)
        opt.step()
        _, gp = loss_and_grad(p, a, b)
        p, m, v = OO.adamw(p, gp, m, v, t, lr, log2_domain=True)
        np.testing.assert_allclose(np.log2(p), theta.detach().numpy(), rtol=0, atol=1e-7)
    assert np.all(p > 0)


def test_log2_domain_steps_are_multiplicative():
    # a step changes log2 p by at most lr (t = 1), whatever the gradient's size
    rng = np.random.default_rng(6)
    p = np.exp2(rng.normal(-7, 2, 1000))
    g = rng.normal(size=1000) * 10.0 ** rng.uniform(-6, 6, 1000)
    p1, _, _ = OO.adamw(p, g, np.zeros(1000), np.zeros(1000), 1, 2e-2, log2_domain=True)
    d = np.log2(p1) - np.log2(p)
    assert np.all(np.abs(d) <= 2e-2 * (1 + 1e-12)) and np.all(np.sign(d) == -np.sign(g))


def test_zero_learning_rate_keeps_parameters():
    p = np.array([0.5, 2.0, 3.0])
    p1, m1, v1 = OO.adamw(p, np.array([1.0, -1.0, 0.0]), np.zeros(3), np.zeros(3), 1, 0.0, weight_decay=0.5)
    np.testing.assert_array_equal(p1, p)
    assert m1[0] > 0 and v1[1] > 0


def test_planted_mistakes_are_caught():
    rng = np.random.default_rng(7)
    p0 = rng.normal(size=64)
    grads = [rng.normal(size=64) for _ in range(4)]
    ref = torch_adamw(p0, grads, 1e-2, (0.9, 0.999), 1e-8, 1e-2)

    def run(step):
        p, m, v = p0, np.zeros(64), np.zeros(64)
        for t, g in enumerate(grads, start=1):
            p, m, v = step(p, g, m, v, t)
        return p

    def planted(kind):
        def step(p, g, m, v, t, lr=1e-2, b1=0.9, b2=0.999, eps=1e-8, wd=1e-2):
            if kind == "coupled_decay":
                g = g + wd * p
            else:
                p = p - lr * wd * p
            m = b1 * m + (1 - b1) * g
            v = b2 * v + (1 - b2) * g * g
            mh = m if kind == "no_bias1" else m / (1 - b1 ** t)
            vh = v if kind == "no_bias2" else v / (1 - b2 ** t)
            return p - lr * mh / (np.sqrt(vh) + eps), m, v
        return step

    good = run(lambda p, g, m, v, t: OO.adamw(p, g, m, v, t, 1e-2, weight_decay=1e-2))
    np.testing.assert_allclose(good, ref[-1][0], rtol=1e-13)
    for kind in ("coupled_decay", "no_bias1", "no_bias2"):
        assert not np.allclose(run(planted(kind)), ref[-1][0], rtol=1e-6), kind
