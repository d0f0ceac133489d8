"""Pins of the Newton start (App. F.2: every unknown begins as the output of
the first step) for the MLP, collapsed-skip ResNet and denoising-chain
oracles.

Each start is rebuilt here from one application of the first step, written
out with torch CPU float64 operations (not the oracle's layer code), and
compared exactly or to rounding.  The start that the Newton drivers actually
use is read back by running them for zero iterations.  A start taken from
another layer, from z0 itself, or a zero start fails these tests."""
import math

import numpy as np
import pytest

import oracle
from oracle import diffusion_oracle as D
from oracle import resnet_oracle as R
from paper_2309_16318_amd import synth

torch = pytest.importorskip("torch")

LAYER_KINDS = [(0, 1.0), (1, 0.1), (2, 1.0), (3, 0.3), (4, 1.0), (5, 0.2)]


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def _sigma(act, a):
    if act == 0:
        return torch.tanh(a)
    if act == 1:
        return torch.sigmoid(a)
    return torch.clamp(a, min=0.0)


def _mlp_first_layer(layer, alpha, W, bias, z0):
    """f_0(z0) for the post-activation layer kinds: sigma(W_0 z0 + b_0),
    plus z0 + alpha * (...) for the residual kinds."""
    a = _t(z0) @ _t(W[0]).T + _t(bias[0])
    s = _sigma(layer >> 1, a)
    out = _t(z0) + alpha * s if layer & 1 else s
    return out.numpy()


@pytest.mark.parametrize("layer,alpha", LAYER_KINDS)
def test_mlp_start_is_first_layer_output(layer, alpha):
    B, L, w = 3, 9, 5
    d = synth.mlp_inputs(B, L, w, seed=77 + layer)
    want = _mlp_first_layer(layer, alpha, d["W"], d["bias"], d["z0"])
    Z0 = oracle.initial_guess(layer, alpha, d["W"], d["bias"], d["z0"])
    assert Z0.shape == (B, L, w)
    for l in range(L):
        np.testing.assert_allclose(Z0[:, l], want, rtol=1e-14, atol=1e-15)
    # the first row of the sequential pass is the same vector
    seq = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"])
    np.testing.assert_array_equal(Z0, np.repeat(seq[:, :1], L, axis=1))
    # the start the Newton drivers use: zero iterations return it unchanged
    Zn, k, _, _ = oracle.newton_forward(layer, alpha, d["W"], d["bias"], d["z0"], 1e-5, 0)
    assert k == 0
    np.testing.assert_array_equal(Zn, Z0)
    Zr, k, _, _ = oracle.newton_forward_residual(layer, alpha, d["W"], d["bias"], d["z0"],
                                                 0.0, 0.0, 0)
    assert k == 0
    np.testing.assert_array_equal(Zr, Z0)


def test_mlp_start_rejects_wrong_layer():
    """The start differs from the output of layer 1 applied to z0 and from
    z0 itself, so a start built from either would fail the pin above."""
    d = synth.mlp_inputs(2, 4, 3, seed=5)
    Z0 = oracle.initial_guess(0, 1.0, d["W"], d["bias"], d["z0"])
    wrong = np.tanh(d["z0"].astype(np.float64) @ d["W"][1].T.astype(np.float64) + d["bias"][1])
    assert np.max(np.abs(Z0[:, 0] - wrong)) > 1e-3
    assert np.max(np.abs(Z0[:, 0] - d["z0"])) > 1e-3


@pytest.mark.parametrize("act", [R.ACT_TANH, R.ACT_SIGMOID, R.ACT_RELU])
@pytest.mark.parametrize("skip", [1, 2, 4])
def test_resnet_start_is_first_block_output(act, skip):
    B, G, w = 2, 5, 4
    L = G * skip
    d = synth.resnet_inputs(B, L, w, seed=31 + skip)
    W, bias, z0 = d["W"], d["bias"], d["z0"]
    # the first block by hand: skip pre-activation layers W sigma(z) + b,
    # then the skip connection adds the block input
    z = _t(z0)
    for j in range(skip):
        z = _sigma(act, z) @ _t(W[j]).T + _t(bias[j])
    want = (z + _t(z0)).numpy()
    X0 = R.resnet_initial_guess(act, skip, W, bias, z0)
    assert X0.shape == (B, G, w)
    for g in range(G):
        np.testing.assert_allclose(X0[:, g], want, rtol=1e-13, atol=1e-14)
    seq = R.resnet_seq_forward(act, skip, W, bias, z0)
    np.testing.assert_allclose(X0[:, 0], seq[:, skip - 1], rtol=1e-14, atol=1e-15)
    # Newton's start: zero iterations, block-output rows of the expansion
    Zn, k, _, _ = R.resnet_newton_forward(act, skip, W, bias, z0, 1e-5, 0)
    assert k == 0
    np.testing.assert_array_equal(Zn[:, skip - 1::skip], X0)


def test_diffusion_start_is_first_step_output():
    B, L, w, hdim = 2, 6, 3, 5
    p = synth.diffusion_inputs(B, L, w, hdim, seed=9)
    zT, eps = p["zT"], p["eps"]
    # step 0 uses schedule index t = L (linear betas from 1e-4 to 0.02)
    beta_t = 0.02
    alpha_t = 1.0 - beta_t
    alphabar_t = math.prod(1.0 - (1e-4 + (0.02 - 1e-4) * i / (L - 1)) for i in range(L))
    c = (1.0 - alpha_t) / math.sqrt(1.0 - alphabar_t)
    a = _t(zT) @ _t(p["W1"]).T + _t(p["b1"]) + _t(p["temb"][L - 1])
    g = torch.tanh(a) @ _t(p["W2"]).T + _t(p["b2"])
    want = ((_t(zT) - c * g) / math.sqrt(alpha_t) + math.sqrt(beta_t) * _t(eps[:, 0])).numpy()
    Z0 = D.initial_guess(p, zT, eps)
    assert Z0.shape == (B, L, w)
    for l in range(L):
        np.testing.assert_allclose(Z0[:, l], want, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(Z0[:, 0], D.seq_sample(p, zT, eps)[:, 0], rtol=1e-14, atol=1e-15)
    Zn, k, _, _ = D.newton_sample(p, zT, eps, 1e-5, 0)
    assert k == 0
    np.testing.assert_array_equal(Zn, Z0)
