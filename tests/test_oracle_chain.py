"""Pins of the chaining oracle: the KL-Top loss (Sec. 4.1), the input gradient of a linear and the
straight-through mask of the activation fake quantisation (Sec. 3.2).

  * a hand-worked KL-Top example (teacher [ln 3, 0, -5], k = 2: p_t = (3/4, 1/4); student [0, 0, 7]:
    p_s = (1/2, 1/2); KL = 3/4 ln(3/2) - 1/4 ln 2; dZ = p_s - p_t on the set, 0 off it);
  * with k >= V, KL-Top is the full KL divergence of the two softmaxes, computed by PyTorch's
    kl_div; KL >= 0, zero for equal logits, unchanged by adding a constant to a row;
  * ties at the k-th value are taken in increasing index order;
  * the gradient against central differences of the loss (the index set depends on the teacher only);
  * dX_hat = dY W_hat against central differences of the MSE of X_hat W_hat^T;
  * the activation mask: all ones under rounded-up E8M0 (|x| <= amax <= 6 S), and under the OCP floor
    rule zero exactly where |x| > 6 * 2^(floor(log2 amax) - 2).
"""
import math

import numpy as np
import torch

from oracle import chain_oracle as C


def test_kl_top_hand_example():
    Zt = np.array([[math.log(3.0), 0.0, -5.0]])
    Zs = np.array([[0.0, 0.0, 7.0]])
    loss, dZ = C.kl_top(Zs, Zt, 2)
    assert abs(loss - (0.75 * math.log(1.5) - 0.25 * math.log(2.0))) < 1e-15
    np.testing.assert_allclose(dZ, [[-0.25, 0.25, 0.0]], atol=1e-15)


def test_full_k_is_the_kl_divergence():
    rng = np.random.default_rng(0)
    Zt, Zs = rng.normal(size=(5, 40)) * 3, rng.normal(size=(5, 40)) * 3
    loss, _ = C.kl_top(Zs, Zt, 40)
    ref = torch.nn.functional.kl_div(torch.log_softmax(torch.tensor(Zs), 1), torch.log_softmax(torch.tensor(Zt), 1),
                                     reduction="batchmean", log_target=True).item()
    assert abs(loss - ref) < 1e-12 * max(1.0, abs(ref))
    assert C.kl_top(Zs, Zt, 1000)[0] == loss


def test_kl_top_invariants():
    rng = np.random.default_rng(1)
    Zt, Zs = rng.normal(size=(6, 300)), rng.normal(size=(6, 300))
    loss, dZ = C.kl_top(Zs, Zt, 50)
    assert loss > 0
    assert C.kl_top(Zt, Zt, 50)[0] == 0.0
    shifted = Zs + rng.normal(size=(6, 1)) * 10
    assert abs(C.kl_top(shifted, Zt, 50)[0] - loss) < 1e-12
    np.testing.assert_allclose(dZ.sum(axis=1), 0.0, atol=1e-15)   # p_s and p_t both sum to 1 on the set
    assert np.all((dZ != 0).sum(axis=1) == 50)


def test_ties_in_index_order():
    Zt = np.array([[1.0, 3.0, 3.0, 2.0, 3.0, 3.0]])
    Zs = np.zeros((1, 6))
    _, dZ = C.kl_top(Zs, Zt + 0.0, 3)
    assert list(np.nonzero(dZ[0])[0]) == [1, 2, 4]


def test_kl_top_gradient_by_finite_differences():
    rng = np.random.default_rng(2)
    Zt, Zs = rng.normal(size=(3, 60)) * 2, rng.normal(size=(3, 60)) * 2
    _, dZ = C.kl_top(Zs, Zt, 20)
    h = 1e-6
    for r, i in [(0, int(np.argmax(Zt[0]))), (1, 5), (2, int(np.argsort(-Zt[2])[19])), (2, int(np.argmin(Zt[2])))]:
        P, M = Zs.copy(), Zs.copy()
        P[r, i] += h
        M[r, i] -= h
        fd = (C.kl_top(P, Zt, 20)[0] - C.kl_top(M, Zt, 20)[0]) / (2 * h)
        assert abs(fd - dZ[r, i]) < 1e-8, (r, i, fd, dZ[r, i])


def test_dx_by_finite_differences():
    rng = np.random.default_rng(3)
    X, W, Y = rng.normal(size=(7, 12)), rng.normal(size=(5, 12)), rng.normal(size=(7, 5))

    def loss(Xv):
        D = Xv @ W.T - Y
        return np.sum(D * D) / D.size

    dY = 2 * (X @ W.T - Y) / Y.size
    dX = C.recon_dx(dY, W)
    h = 1e-6
    for (a, b) in [(0, 0), (3, 7), (6, 11)]:
        P, M = X.copy(), X.copy()
        P[a, b] += h
        M[a, b] -= h
        assert abs((loss(P) - loss(M)) / (2 * h) - dX[a, b]) < 1e-8


def test_activation_mask():
    rng = np.random.default_rng(4)
    X = (rng.normal(size=(16, 128)) * np.exp2(rng.integers(-8, 8, (16, 1)))).astype(np.float32)
    X[:, ::17] *= 30
    assert np.all(C.act_ste_mask(X, 0) == 1.0)
    m = C.act_ste_mask(X, 0, e8m0_floor=True)
    amax = np.abs(X).reshape(16, 4, 32).max(axis=2).astype(np.float64)
    lim = np.repeat(6.0 * np.exp2(np.floor(np.log2(amax)) - 2), 32, axis=1)
    np.testing.assert_array_equal(m, (np.abs(X) <= lim).astype(np.float64))
    assert (m == 0).any()
