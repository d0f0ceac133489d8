"""CPU oracle for the collapsed-skip ResNet (App. A.3): plain numpy float64.

TEST INFRASTRUCTURE, like the rest of this package: only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the GPU
library shares no code with it.

The network (Eq. resnet_seq of App. A.3, 0-indexed): layer j = 0..L-1 maps
Z[:, j-1] to
    Z[:, j] = h_j(Z[:, j-1])                      if (j + 1) % s != 0
    Z[:, j] = h_j(Z[:, j-1]) + Z[:, j-s]          if (j + 1) % s == 0
with h_j(z) = W_j sigma(z) + b_j (an MLP layer in the pre-activation form the
appendix writes), Z[:, -1] := z0 and a skip connection of length s; L is a
multiple of s.  Collapsing the s layers between two skips (App. A.3) gives a
Markov chain over the block outputs X_g = Z[:, g*s + s - 1], g = 0..L/s-1,
X_{-1} = z0:
    X_g = F_g(X_{g-1}) = h_{gs+s-1}( ... h_{gs}(X_{g-1}) ... ) + X_{g-1},
    dF_g/dX = I + J_{gs+s-1} ... J_{gs},   J_j = W_j diag(sigma'(Z_{j-1})),
to which Newton + PCR is applied with L/s unknowns.

Activations: 0 tanh, 1 logistic sigmoid, 2 ReLU (derivative 0 at 0).

Readings: the initial guess applies the rule of App. F.2 to the collapsed
steps (every X_g starts at F_0(z0)); the layer outputs inside a block are
recovered after convergence from the converged block inputs; the loss and the
batch reduction of the gradients are those of the MLP oracle
(Loss = sum_b <G_b, Z_{b, L-1}>, gradients summed over the batch), with the
pre-activation form of Eq. 10: dW_j = sum_b lambda_j sigma(Z_{j-1})^T,
db_j = sum_b lambda_j.
"""
from __future__ import annotations

import numpy as np

from .deeppcr_oracle import activation as _activation_of_layer
from .deeppcr_oracle import seq_solve

ACT_TANH, ACT_SIGMOID, ACT_RELU = 0, 1, 2


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def sigma(act: int, z):
    """sigma(z) and sigma'(z) (the MLP oracle's activations, code 2 * act)."""
    return _activation_of_layer(2 * act, z)


def resnet_layer(act: int, W_j, b_j, z_prev):
    """h_j(z) = W_j sigma(z) + b_j for a batch of states z [B, w]."""
    s, _ = sigma(act, z_prev)
    return s @ _f64(W_j).T + _f64(b_j)


def resnet_layer_jacobian(act: int, W_j, z_prev):
    """dh_j/dz = W_j diag(sigma'(z)) at z_prev, as [B, w, w]."""
    _, d = sigma(act, z_prev)
    return _f64(W_j)[None, :, :] * d[:, None, :]


def is_skip_layer(j: int, skip: int) -> bool:
    return (j + 1) % skip == 0


def resnet_seq_forward(act: int, skip: int, W, bias, z0):
    """The sequential pass of Eq. resnet_seq: every layer output [B, L, w]."""
    W, bias, z0 = _f64(W), _f64(bias), _f64(z0)
    L = W.shape[0]
    assert L % skip == 0
    B, w = z0.shape
    Z = np.empty((B, L, w))
    z = z0
    for j in range(L):
        z = resnet_layer(act, W[j], bias[j], z)
        if is_skip_layer(j, skip):
            z = z + (Z[:, j - skip] if j - skip >= 0 else z0)
        Z[:, j] = z
    return Z


def group_step(act: int, skip: int, W, bias, g: int, x_prev):
    """F_g(x_prev): the s layers of block g composed, plus the skip."""
    W, bias, x_prev = _f64(W), _f64(bias), _f64(x_prev)
    z = x_prev
    for t in range(skip):
        j = g * skip + t
        z = resnet_layer(act, W[j], bias[j], z)
    return z + x_prev


def group_jacobian(act: int, skip: int, W, bias, g: int, x_prev):
    """dF_g/dx at x_prev = I + J_{gs+s-1} ... J_{gs}, as [B, w, w]."""
    W, bias, x_prev = _f64(W), _f64(bias), _f64(x_prev)
    B, w = x_prev.shape
    z = x_prev
    P = np.broadcast_to(np.eye(w), (B, w, w)).copy()
    for t in range(skip):
        j = g * skip + t
        P = resnet_layer_jacobian(act, W[j], z) @ P
        z = resnet_layer(act, W[j], bias[j], z)
    return np.eye(w)[None] + P


def block_inputs(X, z0):
    """Xprev[:, g] = X[:, g-1] with Xprev[:, 0] = z0."""
    X, z0 = _f64(X), _f64(z0)
    return np.concatenate([z0[:, None, :], X[:, :-1, :]], axis=1)


def expand_blocks(act: int, skip: int, W, bias, z0, X):
    """All layer outputs from the block outputs X: inside block g the layers
    run from X_{g-1}; the block's last row is X_g itself."""
    W, bias, X = _f64(W), _f64(bias), _f64(X)
    B, G, w = X.shape
    Xprev = block_inputs(X, z0)
    Z = np.empty((B, G * skip, w))
    for g in range(G):
        z = Xprev[:, g]
        for t in range(skip - 1):
            j = g * skip + t
            z = resnet_layer(act, W[j], bias[j], z)
            Z[:, j] = z
        Z[:, g * skip + skip - 1] = X[:, g]
    return Z


def resnet_initial_guess(act: int, skip: int, W, bias, z0):
    """Start of Newton on the block chain: App. F.2 copies the output of the
    first step into every unknown; the first step of the collapsed chain is
    the first block F_0, so every X_g starts at F_0(z0).  Returns X [B, L/s, w]."""
    W, bias, z0 = _f64(W), _f64(bias), _f64(z0)
    G = W.shape[0] // skip
    f0 = group_step(act, skip, W, bias, 0, z0)
    return np.repeat(f0[:, None, :], G, axis=1)


def resnet_newton_forward(act: int, skip: int, W, bias, z0, tol: float, max_iter: int,
                          Z_init=None, solve=seq_solve):
    """Newton on the collapsed system (App. A.3 with Sec. 2, Eqs. 2-3).

    Unknowns X_g, g = 0..L/s-1; each iteration evaluates every block step and
    its Jacobian at the iterate, solves the block-bidiagonal system of Eq. 3
    (sub-diagonal blocks dF_g/dX) and updates.  Stopping rule of the MLP
    oracle: max|dX| < tol * max(1, max|X|) after the update, or max_iter
    solves (tol = 0: exactly max_iter).  Z_init, if given, supplies the start
    X^0 = Z_init[:, s-1::s].
    Returns (Z [B, L, w], solves, converged, [max|dX| per iteration]).
    """
    W, bias, z0 = _f64(W), _f64(bias), _f64(z0)
    G = W.shape[0] // skip
    if Z_init is None:
        X = resnet_initial_guess(act, skip, W, bias, z0)
    else:
        X = _f64(Z_init)[:, skip - 1::skip].copy()
    history = []
    for k in range(1, max_iter + 1):
        Xprev = block_inputs(X, z0)
        F = np.stack([group_step(act, skip, W, bias, g, Xprev[:, g]) for g in range(G)], axis=1)
        J = np.stack([group_jacobian(act, skip, W, bias, g, Xprev[:, g]) for g in range(G)],
                     axis=1)
        dX = solve(J, F - X)
        X = X + dX
        m = float(np.max(np.abs(dX)))
        history.append(m)
        if tol > 0 and m < tol * max(1.0, float(np.max(np.abs(X)))):
            return expand_blocks(act, skip, W, bias, z0, X), k, True, history
    return expand_blocks(act, skip, W, bias, z0, X), max_iter, tol == 0, history


def resnet_seq_backward(act: int, skip: int, W, bias, z0, Z, G):
    """Reverse-mode pass through Eq. resnet_seq for Loss = sum_b <G_b, Z_{b, L-1}>.

    Layers are visited from L-1 down to 0; layer j sends diag(sigma'(Z_{j-1}))
    W_j^T lambda_j to its input and, for a skip layer, lambda_j to Z_{j-s}
    (z0 when j - s = -1).  Returns (Lambda = dLoss/dZ [B, L, w],
    dz0 [B, w], dW [L, w, w], db [L, w]) with dW_j = sum_b lambda_j
    sigma(Z_{j-1})^T and db_j = sum_b lambda_j (Eq. 10, pre-activation form).
    """
    W, bias, z0, Z, G = _f64(W), _f64(bias), _f64(z0), _f64(Z), _f64(G)
    B, L, w = Z.shape
    lam = np.zeros((B, L, w))
    lam[:, L - 1] = G
    dz0 = np.zeros((B, w))
    dW = np.empty((L, w, w))
    db = np.empty((L, w))
    for j in range(L - 1, -1, -1):
        zin = Z[:, j - 1] if j >= 1 else z0
        s, d = sigma(act, zin)
        dW[j] = lam[:, j].T @ s
        db[j] = lam[:, j].sum(axis=0)
        back = (lam[:, j] @ W[j]) * d
        if j >= 1:
            lam[:, j - 1] += back
        else:
            dz0 += back
        if is_skip_layer(j, skip):
            if j - skip >= 0:
                lam[:, j - skip] += lam[:, j]
            else:
                dz0 += lam[:, j]
    return lam, dz0, dW, db


def resnet_loss(act: int, skip: int, W, bias, z0, G):
    Z = resnet_seq_forward(act, skip, W, bias, z0)
    return float(np.sum(_f64(G) * Z[:, -1]))
