"""Pins of the diffusion-style step oracle (App. A.4): the noise schedule,
the linear special case in closed form, the step Jacobian by central
differences, a one-step example by hand, and Newton's fixed point and prefix
exactness on the denoising chain."""
import math

import numpy as np
import pytest

import oracle
from oracle import diffusion_oracle as D
from paper_2309_16318_amd import synth


def test_schedule():
    beta, alpha, alphabar = D.schedule(5)
    np.testing.assert_allclose(beta, [1e-4, 0.0050750, 0.010050, 0.0150250, 0.02], rtol=1e-12)
    prod = 1.0
    for t in range(5):
        prod *= 1.0 - beta[t]
        assert alphabar[t] == pytest.approx(prod, rel=1e-15)
    assert np.all(np.diff(alphabar) < 0)


def test_one_step_by_hand():
    # L = 1 (t = 1: beta = 1e-4), w = h = 1
    p = {"W1": np.array([[0.5]]), "b1": np.array([0.1]), "W2": np.array([[2.0]]),
         "b2": np.array([-0.3]), "temb": np.array([[0.2]])}
    zT = np.array([[0.7]])
    eps = np.array([[[1.5]]])
    beta = 1e-4
    alpha = 1.0 - beta
    g = 2.0 * math.tanh(0.5 * 0.7 + 0.1 + 0.2) - 0.3
    c = (1.0 - alpha) / math.sqrt(1.0 - alpha)
    want = (0.7 - c * g) / math.sqrt(alpha) + math.sqrt(beta) * 1.5
    assert D.seq_sample(p, zT, eps)[0, 0, 0] == pytest.approx(want, rel=1e-14)
    th = math.tanh(0.5 * 0.7 + 0.1 + 0.2)
    jwant = (1.0 - c * 2.0 * (1.0 - th * th) * 0.5) / math.sqrt(alpha)
    assert D.step_jacobian(p, 0, zT)[0, 0, 0] == pytest.approx(jwant, rel=1e-14)


def test_linear_chain_closed_form():
    """g = 0 (W2 = 0, b2 = 0): z_j = a_j z_{j-1} + s_j eps_j with
    a_j = 1/sqrt(alpha_t), s_j = sqrt(beta_t), so
    z_j = (prod_{i<=j} a_i) z_T + sum_{i<=j} (prod_{i<k<=j} a_k) s_i eps_i."""
    B, L, w, h = 2, 9, 3, 4
    d = dict(synth.diffusion_inputs(B, L, w, h, seed=5))
    d["W2"] = np.zeros_like(d["W2"])
    d["b2"] = np.zeros_like(d["b2"])
    Z = D.seq_sample(d, d["zT"], d["eps"])
    beta, alpha, _ = D.schedule(L)
    t = L - np.arange(L)                     # schedule index of step j
    a = 1.0 / np.sqrt(alpha[t - 1])
    s = np.sqrt(beta[t - 1])
    zT = d["zT"].astype(np.float64)
    eps = d["eps"].astype(np.float64)
    for j in range(L):
        want = np.prod(a[:j + 1]) * zT
        for i in range(j + 1):
            want = want + np.prod(a[i + 1:j + 1]) * s[i] * eps[:, i]
        np.testing.assert_allclose(Z[:, j], want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("j", [0, 3, 7])
def test_step_jacobian_matches_central_differences(j):
    B, L, w, h = 2, 8, 4, 6
    d = synth.diffusion_inputs(B, L, w, h, seed=7)
    z = np.random.default_rng(1).standard_normal((B, w))
    J = D.step_jacobian(d, j, z)
    hstep = 1e-6
    for k in range(w):
        e = np.zeros(w)
        e[k] = hstep
        fd = (D.step(d, j, z + e, d["eps"][:, j]) - D.step(d, j, z - e, d["eps"][:, j])) / (2 * hstep)
        np.testing.assert_allclose(J[:, :, k], fd, rtol=1e-7, atol=1e-8)


@pytest.mark.parametrize("L,w,h", [(16, 4, 8), (64, 16, 32)])
def test_newton_fixed_point_is_sequential_sample(L, w, h):
    d = synth.diffusion_inputs(2, L, w, h, seed=11)
    ref = D.seq_sample(d, d["zT"], d["eps"])
    for solve in (oracle.seq_solve, oracle.pcr_solve):
        Z, k, ok, hist = D.newton_sample(d, d["zT"], d["eps"], 1e-12, 30, solve=solve)
        assert ok and k <= L
        np.testing.assert_allclose(Z, ref, rtol=1e-11, atol=1e-11)


def test_newton_prefix_exactness():
    B, L, w, h = 2, 7, 3, 5
    d = synth.diffusion_inputs(B, L, w, h, seed=13)
    ref = D.seq_sample(d, d["zT"], d["eps"])
    for k in range(1, L + 1):
        Z, it, ok, _ = D.newton_sample(d, d["zT"], d["eps"], 0.0, k, Z_init=np.zeros((B, L, w)))
        assert it == k and ok
        np.testing.assert_allclose(Z[:, :k], ref[:, :k], rtol=0, atol=1e-12)
