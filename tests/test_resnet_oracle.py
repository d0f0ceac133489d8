"""Pins of the collapsed-skip ResNet oracle (App. A.3) against hand-worked
values, closed forms, finite differences, torch autograd and the
prefix-exactness property of Newton on a block lower-triangular system."""
import numpy as np
import pytest

from oracle import resnet_oracle as R
import oracle
from paper_2309_16318_amd import synth

ACTS = [R.ACT_TANH, R.ACT_SIGMOID, R.ACT_RELU]


def _hand_net():
    W = np.array([[[2.0]], [[-1.0]], [[0.5]], [[3.0]]])
    b = np.array([[0.1], [0.2], [-0.3], [0.4]])
    z0 = np.array([[0.5]])
    return W, b, z0


def test_forward_by_hand_relu():
    # s = 2: Z0 = 2 relu(.5) + .1 = 1.1;  Z1 = -relu(1.1) + .2 + z0 = -.4
    #        Z2 = .5 relu(-.4) - .3 = -.3; Z3 = 3 relu(-.3) + .4 + Z1 = 0
    W, b, z0 = _hand_net()
    Z = R.resnet_seq_forward(R.ACT_RELU, 2, W, b, z0)
    np.testing.assert_allclose(Z[0, :, 0], [1.1, -0.4, -0.3, 0.0], atol=1e-15)


def test_backward_by_hand_relu():
    # G = 1: lambda3 = 1; layer 3 sees relu'(-.3) = 0 and skips lambda3 to Z1;
    # layer 2 gets nothing; layer 1: relu'(1.1) = 1, lambda0 = W1 * 1 = -1 and
    # its skip sends 1 to z0; layer 0: dz0 += W0 * lambda0 = -2, so dz0 = -1.
    W, b, z0 = _hand_net()
    Z = R.resnet_seq_forward(R.ACT_RELU, 2, W, b, z0)
    lam, dz0, dW, db = R.resnet_seq_backward(R.ACT_RELU, 2, W, b, z0, Z, np.array([[1.0]]))
    np.testing.assert_allclose(lam[0, :, 0], [-1.0, 1.0, 0.0, 1.0], atol=1e-15)
    np.testing.assert_allclose(dz0[0], [-1.0], atol=1e-15)
    np.testing.assert_allclose(dW[:, 0, 0], [-0.5, 1.1, 0.0, 0.0], atol=1e-15)
    np.testing.assert_allclose(db[:, 0], [-1.0, 1.0, 0.0, 1.0], atol=1e-15)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("skip", [1, 2, 4])
def test_zero_weights_closed_form(act, skip):
    """W = 0: h_j = b_j, so X_g = z0 + sum_{g' <= g} b_{g's+s-1} and the rows
    inside a block are their biases."""
    B, L, w = 2, 4 * skip, 3
    rng = np.random.default_rng(5)
    W = np.zeros((L, w, w))
    b = rng.standard_normal((L, w))
    z0 = rng.standard_normal((B, w))
    Z = R.resnet_seq_forward(act, skip, W, b, z0)
    X = z0[:, None, :] + np.cumsum(b[skip - 1::skip], axis=0)[None]
    np.testing.assert_allclose(Z[:, skip - 1::skip], X, rtol=1e-14, atol=1e-14)
    for j in range(L):
        if not R.is_skip_layer(j, skip):
            np.testing.assert_array_equal(Z[:, j], np.broadcast_to(b[j], (B, w)))


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("skip", [1, 3, 4])
def test_group_step_is_the_block_of_the_sequential_pass(act, skip):
    d = synth.resnet_inputs(3, 6 * skip, 5, seed=11)
    Z = R.resnet_seq_forward(act, skip, d["W"], d["bias"], d["z0"])
    X = Z[:, skip - 1::skip]
    Xprev = R.block_inputs(X, d["z0"])
    for g in range(X.shape[1]):
        np.testing.assert_allclose(R.group_step(act, skip, d["W"], d["bias"], g, Xprev[:, g]),
                                   X[:, g], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(R.expand_blocks(act, skip, d["W"], d["bias"], d["z0"], X), Z,
                               rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("skip", [1, 2, 4])
def test_group_jacobian_matches_central_differences(act, skip):
    B, w = 2, 4
    d = synth.resnet_inputs(B, 3 * skip, w, seed=21)
    x = np.random.default_rng(2).standard_normal((B, w)) * 0.7
    J = R.group_jacobian(act, skip, d["W"], d["bias"], 1, x)
    h = 1e-6
    for k in range(w):
        e = np.zeros(w)
        e[k] = h
        fd = (R.group_step(act, skip, d["W"], d["bias"], 1, x + e)
              - R.group_step(act, skip, d["W"], d["bias"], 1, x - e)) / (2 * h)
        np.testing.assert_allclose(J[:, :, k], fd, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("skip", [1, 2, 4])
def test_newton_fixed_point_is_sequential_pass(act, skip):
    d = synth.resnet_inputs(2, 16 * skip, 6, seed=31)
    ref = R.resnet_seq_forward(act, skip, d["W"], d["bias"], d["z0"])
    for solve in (oracle.seq_solve, oracle.pcr_solve):
        Z, k, ok, hist = R.resnet_newton_forward(act, skip, d["W"], d["bias"], d["z0"], 1e-12,
                                                 40, solve=solve)
        assert ok and k <= 16
        np.testing.assert_allclose(Z, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("act", ACTS)
def test_newton_prefix_exactness_on_collapsed_system(act):
    """After k solves from a zero start, blocks 0..k-1 (and the rows computed
    from them) equal the sequential pass: the collapsed system is block
    lower-triangular too."""
    skip, G, w, B = 4, 7, 3, 2
    d = synth.resnet_inputs(B, skip * G, w, seed=41)
    ref = R.resnet_seq_forward(act, skip, d["W"], d["bias"], d["z0"])
    for k in range(1, G + 1):
        Z, it, ok, _ = R.resnet_newton_forward(act, skip, d["W"], d["bias"], d["z0"], 0.0, k,
                                               Z_init=np.zeros((B, skip * G, w)))
        assert it == k and ok
        np.testing.assert_allclose(Z[:, :k * skip], ref[:, :k * skip], rtol=0, atol=1e-13)


def test_newton_iterations_paper_shape():
    """w = 16, skip 4, ReLU, L = 256 (the paper's ResNet shape): a handful of
    Newton iterations (the paper reports about 6)."""
    d = synth.resnet_inputs(2, 256, 16, seed=0)
    Z, k, ok, hist = R.resnet_newton_forward(R.ACT_RELU, 4, d["W"], d["bias"], d["z0"], 1e-5, 20)
    ref = R.resnet_seq_forward(R.ACT_RELU, 4, d["W"], d["bias"], d["z0"])
    assert ok and 3 <= k <= 10
    np.testing.assert_allclose(Z, ref, atol=1e-8)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("skip,L", [(1, 3), (2, 4), (4, 8), (3, 6)])
def test_backward_matches_central_differences(act, skip, L):
    B, w = 2, 3
    d = synth.resnet_inputs(B, L, w, seed=51 + L)
    W, b, z0, G = (d[k].astype(np.float64) for k in ("W", "bias", "z0", "G"))
    Z = R.resnet_seq_forward(act, skip, W, b, z0)
    lam, dz0, dW, db = R.resnet_seq_backward(act, skip, W, b, z0, Z, G)
    h = 1e-6

    def fd(arr, idx):
        a0 = arr[idx]
        arr[idx] = a0 + h
        lp = R.resnet_loss(act, skip, W, b, z0, G)
        arr[idx] = a0 - h
        lm = R.resnet_loss(act, skip, W, b, z0, G)
        arr[idx] = a0
        return (lp - lm) / (2 * h)

    for idx in np.ndindex(W.shape):
        assert dW[idx] == pytest.approx(fd(W, idx), rel=1e-6, abs=1e-8)
    for idx in np.ndindex(b.shape):
        assert db[idx] == pytest.approx(fd(b, idx), rel=1e-6, abs=1e-8)
    for idx in np.ndindex(z0.shape):
        assert dz0[idx] == pytest.approx(fd(z0, idx), rel=1e-6, abs=1e-8)


@pytest.mark.parametrize("act", ACTS)
def test_intermediate_adjoints_match_central_differences(act):
    """lambda_j = dLoss/dZ_j for every layer, block outputs and rows inside a
    block: perturb Z_j and run the rest of the network from it (skips into
    later blocks read the recomputed block outputs)."""
    skip, L, B, w = 3, 9, 1, 2
    d = synth.resnet_inputs(B, L, w, seed=61)
    W, b, z0, G = (d[k].astype(np.float64) for k in ("W", "bias", "z0", "G"))
    Z = R.resnet_seq_forward(act, skip, W, b, z0)
    lam, _, _, _ = R.resnet_seq_backward(act, skip, W, b, z0, Z, G)

    def loss_from(j, zj):
        Zp = Z.copy()
        Zp[:, j] = zj
        for k in range(j + 1, L):
            z = R.resnet_layer(act, W[k], b[k], Zp[:, k - 1])
            if R.is_skip_layer(k, skip):
                z = z + (Zp[:, k - skip] if k - skip >= 0 else z0)
            Zp[:, k] = z
        return float(np.sum(G * Zp[:, -1]))

    h = 1e-6
    for j in range(L):
        for i in range(w):
            e = np.zeros(w)
            e[i] = h
            g = (loss_from(j, Z[:, j] + e) - loss_from(j, Z[:, j] - e)) / (2 * h)
            assert lam[0, j, i] == pytest.approx(g, rel=1e-6, abs=1e-8)


@pytest.mark.parametrize("act", ACTS)
def test_forward_and_backward_match_torch_autograd(act):
    torch = pytest.importorskip("torch")
    skip, L, B, w = 4, 12, 3, 5
    d = synth.resnet_inputs(B, L, w, seed=71)
    fn = {R.ACT_TANH: torch.tanh, R.ACT_SIGMOID: torch.sigmoid, R.ACT_RELU: torch.relu}[act]
    W = torch.tensor(d["W"], dtype=torch.float64, requires_grad=True)
    b = torch.tensor(d["bias"], dtype=torch.float64, requires_grad=True)
    z0 = torch.tensor(d["z0"], dtype=torch.float64, requires_grad=True)
    Gt = torch.tensor(d["G"], dtype=torch.float64)
    outs = []
    z = z0
    for j in range(L):
        lin = torch.nn.functional.linear(fn(z), W[j], b[j])
        if (j + 1) % skip == 0:
            lin = lin + (outs[j - skip] if j - skip >= 0 else z0)
        z = lin
        outs.append(z)
    (Gt * outs[-1]).sum().backward()
    Z = R.resnet_seq_forward(act, skip, d["W"], d["bias"], d["z0"])
    np.testing.assert_allclose(Z, torch.stack(outs, 1).detach().numpy(), rtol=1e-13, atol=1e-13)
    lam, dz0, dW, db = R.resnet_seq_backward(act, skip, d["W"], d["bias"], d["z0"], Z, d["G"])
    np.testing.assert_allclose(dW, W.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dz0, z0.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_resnet_inputs_are_seeded_and_shaped():
    a = synth.resnet_inputs(2, 8, 4, seed=3)
    b = synth.resnet_inputs(2, 8, 4, seed=3)
    assert synth.digest(a) == synth.digest(b)
    assert a["W"].shape == (8, 4, 4) and a["W"].dtype == np.float32
    assert np.abs(a["W"]).max() <= 0.5 and np.abs(a["bias"]).max() <= 0.5
