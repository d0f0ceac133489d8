"""DeepPCR CPU oracle: plain, slow, obviously correct, numpy float64.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The GPU library never calls it, and
the two share no code: the oracle takes float32 arrays (from the seeded input
generators), upcasts them to float64 and works from the paper's definitions.

Indexing is 0-based, as at the library boundary.  Layer l = 0..L-1 maps
Z[:, l-1] to Z[:, l], with Z[:, -1] := z0 (a given input, so its Newton update
is identically zero; the paper's row 0 of the collated system).  J_l denotes
dZ[:, l] / dZ[:, l-1].

Functions and the passages they follow
  step, step_jacobian   App. A.1, Eqs. 7-9 (MLP layer and its Jacobian), in the
                        post-activation form Z_l = sigma(W_l Z_{l-1} + b_l),
                        sigma in {tanh, sigmoid, ReLU}; and the residual step
                        Z_l = Z_{l-1} + alpha*sigma(...) (App. A.3 with a skip
                        of length 1).
  seq_forward           Sec. 2, Eq. 1: the sequence applied one step at a time;
                        it is the unique root of F(z) = 0.
  seq_solve             Sec. 3: forward substitution of the block-bidiagonal
                        system of Eq. 3 (and back substitution of its
                        transpose, App. A.2, Eq. 12).
  pcr_solve             Sec. 3, Alg. 1 and Eqs. 4-6: Parallel Cyclic Reduction,
                        level by level, every row of a level reading the
                        previous level's values.
  newton_forward        Sec. 2, Eqs. 2-3: Newton on F with the linear system
                        solved by seq_solve (or pcr_solve); initial guess of
                        App. F.2 (every row set to the first layer's output).
  newton_forward_residual
                        the same iteration stopped by the residual rule of the
                        solver-parameter table of App. F.1 (absolute and
                        relative infinity-norm thresholds on F(z^k)).
  seq_backward          App. A.2, Eqs. 10-12: adjoints by back substitution and
                        the parameter gradients.

Readings of the paper taken here (each is listed with its reason in the
design notes of the repository):
  * Sign: the sub-diagonal operator is A^0_l := +J_l (Eq. 4), so one PCR level
    is r_l <- r_l + A_l r_{l-s} and A_l <- A_l A_{l-s}.  Alg. 1 prints minus
    signs, which match the convention A := -J; with A^0 := +J, substituting
    Eq. 4 into itself gives plus signs (Eqs. 5-6 print a minus there).
  * Levels: strides s = 1, 2, 4, ... while s < L, i.e. ceil(log2 L) levels;
    row l is updated at stride s iff l >= s.
  * z0 is an input, so the unknowns are Z[:, 0..L-1] and J_0 couples row 0 to
    an unknown that is identically zero: J[:, 0] is ignored (treated as 0).
  * The Jacobians of the backward pass are evaluated at the stored inputs
    Z_{l-1} of each layer (Eq. 11); sigma' is recomputed from the
    pre-activation for every layer kind.  ReLU'(0) is taken as 0.
  * Residual stopping rule: the table gives an absolute and a relative
    threshold without saying how they combine; either one met stops the
    iteration (res <= atol or res <= rtol * res_0), checked on the iterate
    before each solve, and the iteration count is the number of solves.
  * Parameter gradients are summed over the batch for
    Loss = sum_b <G_b, Z_{b, L-1}>.

Parity status: every function here is pinned by CPU tests (hand-derived
systems, dense LAPACK solves, closed forms, the prefix-exactness property of
Newton on Eq. 3, and central finite differences for the backward pass).
"""
from __future__ import annotations

import numpy as np

# layer code = 2 * activation + residual; activation 0 tanh, 1 sigmoid, 2 ReLU
TANH_MLP, TANH_RESIDUAL, SIGMOID_MLP, SIGMOID_RESIDUAL, RELU_MLP, RELU_RESIDUAL = range(6)


def is_residual(layer: int) -> bool:
    return layer % 2 == 1


def activation(layer: int, a):
    """sigma(a) and sigma'(a) for the layer's activation (ReLU' (0) := 0)."""
    a = _f64(a)
    act = layer // 2
    if act == 0:
        t = np.tanh(a)
        return t, 1.0 - t * t
    if act == 1:
        s = 1.0 / (1.0 + np.exp(-a))
        return s, s * (1.0 - s)
    if act == 2:
        return np.maximum(a, 0.0), (a > 0).astype(np.float64)
    raise ValueError(f"unknown layer kind {layer}")


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------
# Layers (App. A.1, Eqs. 7-9; App. A.3 with skip length 1)
# ----------------------------------------------------------------------------

def preactivation(W_l, b_l, z_prev):
    """a = W_l z_prev + b_l for every batch row; z_prev is [B, w]."""
    return _f64(z_prev) @ _f64(W_l).T + _f64(b_l)


def step(layer: int, alpha: float, W_l, b_l, z_prev):
    """f_l(z_prev) for a batch of states z_prev [B, w]."""
    y, _ = activation(layer, preactivation(W_l, b_l, z_prev))
    return _f64(z_prev) + alpha * y if is_residual(layer) else y


def step_jacobian(layer: int, alpha: float, W_l, b_l, z_prev):
    """df_l/dz evaluated at z_prev, as explicit [B, w, w] matrices.

    plain:     J = diag(sigma'(a)) W_l               (Eq. 8)
    residual:  J = I + alpha * diag(sigma'(a)) W_l
    """
    _, d = activation(layer, preactivation(W_l, b_l, z_prev))
    J = d[:, :, None] * _f64(W_l)[None, :, :]
    if is_residual(layer):
        w = J.shape[-1]
        return np.eye(w)[None] + alpha * J
    return J


def seq_forward(layer: int, alpha: float, W, bias, z0):
    """The sequential pass Z[:, l] = f_l(Z[:, l-1]), Z[:, -1] = z0 (Eq. 1)."""
    W, bias, z = _f64(W), _f64(bias), _f64(z0)
    L = W.shape[0]
    B, w = z.shape
    Z = np.empty((B, L, w))
    for l in range(L):
        z = step(layer, alpha, W[l], bias[l], z)
        Z[:, l] = z
    return Z


def layer_inputs(Z, z0):
    """Zprev[:, l] = Z[:, l-1] with Zprev[:, 0] = z0."""
    Z, z0 = _f64(Z), _f64(z0)
    return np.concatenate([z0[:, None, :], Z[:, :-1, :]], axis=1)


def all_jacobians(layer: int, alpha: float, W, bias, Zprev):
    """J[:, l] = df_l/dz at Zprev[:, l], for every layer: [B, L, w, w]."""
    L = W.shape[0]
    return np.stack([step_jacobian(layer, alpha, W[l], bias[l], Zprev[:, l])
                     for l in range(L)], axis=1)


def all_steps(layer: int, alpha: float, W, bias, Zprev):
    """F[:, l] = f_l(Zprev[:, l]), for every layer: [B, L, w]."""
    L = W.shape[0]
    return np.stack([step(layer, alpha, W[l], bias[l], Zprev[:, l])
                     for l in range(L)], axis=1)


# ----------------------------------------------------------------------------
# Linear solves of the block-bidiagonal system (Eq. 3) and its transpose
# ----------------------------------------------------------------------------

def seq_solve(J, r, transpose: bool = False):
    """Substitution (Sec. 3, the sequential solve).

    transpose=False:  x_l = J_l x_{l-1} + r_l,      l = 0..L-1, x_{-1} = 0
    transpose=True:   x_l = J_{l+1}^T x_{l+1} + r_l, l = L-1..0, x_L = 0
    J is [B, L, w, w], r is [B, L, w]; J[:, 0] never enters.
    """
    J, r = _f64(J), _f64(r)
    B, L, w = r.shape
    x = np.empty_like(r)
    if not transpose:
        x[:, 0] = r[:, 0]
        for l in range(1, L):
            x[:, l] = np.einsum("bij,bj->bi", J[:, l], x[:, l - 1]) + r[:, l]
    else:
        x[:, L - 1] = r[:, L - 1]
        for l in range(L - 2, -1, -1):
            x[:, l] = np.einsum("bji,bj->bi", J[:, l + 1], x[:, l + 1]) + r[:, l]
    return x


def reversed_transposed_system(J, r):
    """The transposed system of Eq. 12 written again in lower block-bidiagonal
    form by reversing the row order: row m = L-1-l has sub-diagonal operator
    J_{L-m}^T (m >= 1) and right-hand side r_{L-1-m}."""
    J, r = _f64(J), _f64(r)
    B, L, w = r.shape
    Jr = np.zeros_like(J)
    for m in range(1, L):
        Jr[:, m] = np.swapaxes(J[:, L - m], -1, -2)
    return Jr, r[:, ::-1].copy()


def pcr_solve(J, r, transpose: bool = False, record_levels: list | None = None):
    """Parallel Cyclic Reduction for the block-bidiagonal system (Alg. 1).

    Initialisation: A_l = J_l (row 0 has no coupling: A_0 = 0), r_l = r_l.
    For s = 1, 2, 4, ... while s < L, every row l >= s is reduced in parallel,
    all reads seeing the previous level:
        r_l <- r_l + A_l r_{l-s}
        A_l <- A_l A_{l-s}
    Afterwards r holds the solution.  If ``record_levels`` is a list, a tuple
    (s, A, r) is appended after each level.
    """
    if transpose:
        A, R = reversed_transposed_system(J, r)
    else:
        A, R = _f64(J).copy(), _f64(r).copy()
    A[:, 0] = 0.0
    L = R.shape[1]
    s = 1
    while s < L:
        A_prev, R_prev = A.copy(), R.copy()          # the level's inputs
        R[:, s:] = R_prev[:, s:] + np.einsum("blij,blj->bli", A_prev[:, s:], R_prev[:, :-s])
        A[:, s:] = np.einsum("blij,bljk->blik", A_prev[:, s:], A_prev[:, :-s])
        if record_levels is not None:
            record_levels.append((s, A.copy(), R.copy()))
        s *= 2
    return R[:, ::-1].copy() if transpose else R


def num_levels(L: int) -> int:
    """ceil(log2 L): the number of PCR levels (0 for L = 1)."""
    k, s = 0, 1
    while s < L:
        s *= 2
        k += 1
    return k


# ----------------------------------------------------------------------------
# Newton on F(z) = 0 (Sec. 2, Eqs. 2-3)
# ----------------------------------------------------------------------------

def initial_guess(layer: int, alpha: float, W, bias, z0):
    """Every row set to the first layer's output f_0(z0) (App. F.2)."""
    f0 = step(layer, alpha, W[0], bias[0], z0)
    L = W.shape[0]
    return np.repeat(f0[:, None, :], L, axis=1)


def newton_forward(layer: int, alpha: float, W, bias, z0, tol: float, max_iter: int,
                   Z_init=None, solve=seq_solve):
    """Newton iterations z^{k+1} = z^k + dz^k with J_F(z^k) dz^k = -F(z^k).

    Each iteration evaluates all L layers and their Jacobians at the current
    iterate, forms the residual r_l = f_l(Z_{l-1}) - Z_l (right-hand side of
    Eq. 3) and solves the block-bidiagonal system.  Stops once
    max|dZ| < tol * max(1, max|Z|) after the update, or after max_iter solves;
    tol = 0 runs exactly max_iter solves.

    Returns (Z, iterations, converged, [max|dZ| per iteration]).
    """
    W, bias, z0 = _f64(W), _f64(bias), _f64(z0)
    Z = initial_guess(layer, alpha, W, bias, z0) if Z_init is None else _f64(Z_init).copy()
    history = []
    for k in range(1, max_iter + 1):
        Zprev = layer_inputs(Z, z0)
        F = all_steps(layer, alpha, W, bias, Zprev)
        J = all_jacobians(layer, alpha, W, bias, Zprev)
        dZ = solve(J, F - Z)
        Z = Z + dZ
        m = float(np.max(np.abs(dZ)))
        history.append(m)
        if tol > 0 and m < tol * max(1.0, float(np.max(np.abs(Z)))):
            return Z, k, True, history
    return Z, max_iter, tol == 0, history



def residual_norm(layer: int, alpha: float, W, bias, z0, Z) -> float:
    """max |F(Z)| with F_l = f_l(Z_{l-1}) - Z_l: the infinity norm of the
    Newton solver's residual (Eq. 1 at the iterate)."""
    W, bias, z0, Z = _f64(W), _f64(bias), _f64(z0), _f64(Z)
    F = all_steps(layer, alpha, W, bias, layer_inputs(Z, z0)) - Z
    return float(np.max(np.abs(F))) if F.size else 0.0


def newton_forward_residual(layer: int, alpha: float, W, bias, z0, atol: float, rtol: float,
                            max_iter: int, Z_init=None, solve=seq_solve):
    """Newton on F(z) = 0 with the residual-based stopping rule of the
    solver-parameter table (App. F.1): the infinity norm of the residual
    F(z^k) is compared with an absolute threshold and with a threshold
    relative to the first iterate's residual norm.

    At k = 0, 1, ...: res_k = max|F(z^k)|; stop with z^k when
    res_k <= atol or res_k <= rtol * res_0 (either criterion suffices);
    otherwise, if k == max_iter, stop without convergence; otherwise solve
    Eq. 3 for dz^k and set z^{k+1} = z^k + dz^k.

    Returns (Z, solves, converged, [res_0, res_1, ...]).
    """
    W, bias, z0 = _f64(W), _f64(bias), _f64(z0)
    Z = initial_guess(layer, alpha, W, bias, z0) if Z_init is None else _f64(Z_init).copy()
    history = []
    for k in range(max_iter + 1):
        Zprev = layer_inputs(Z, z0)
        F = all_steps(layer, alpha, W, bias, Zprev) - Z
        res = float(np.max(np.abs(F))) if F.size else 0.0
        history.append(res)
        if res <= atol or res <= rtol * history[0]:
            return Z, k, True, history
        if k == max_iter:
            break
        J = all_jacobians(layer, alpha, W, bias, Zprev)
        Z = Z + solve(J, F)
    return Z, max_iter, False, history

# ----------------------------------------------------------------------------
# Backward pass (App. A.2, Eqs. 10-12)
# ----------------------------------------------------------------------------

def seq_backward(layer: int, alpha: float, W, bias, z0, Z, G):
    """Adjoints and parameter gradients for Loss = sum_b <G_b, Z_{b, L-1}>.

    lambda_{L-1} = G, lambda_l = J_{l+1}^T lambda_{l+1} (Eq. 11), with J_l
    evaluated at the stored layer input Z_{l-1}; dz0 = J_0^T lambda_0.
    With d_l = sigma'(W_l Z_{l-1} + b_l) and c = 1 (plain) or alpha
    (residual), Eq. 10 in the post-activation form reads
        dW_l = c * sum_b (d_l * lambda_l) Z_{l-1}^T,   db_l = c * sum_b d_l * lambda_l.
    Returns (Lambda [B, L, w], dz0 [B, w], dW [L, w, w], db [L, w]).
    """
    W, bias, z0, Z, G = _f64(W), _f64(bias), _f64(z0), _f64(Z), _f64(G)
    B, L, w = Z.shape
    Zprev = layer_inputs(Z, z0)
    lam = np.empty((B, L, w))
    lam[:, L - 1] = G
    for l in range(L - 2, -1, -1):
        J_next = step_jacobian(layer, alpha, W[l + 1], bias[l + 1], Zprev[:, l + 1])
        lam[:, l] = np.einsum("bji,bj->bi", J_next, lam[:, l + 1])
    J_0 = step_jacobian(layer, alpha, W[0], bias[0], Zprev[:, 0])
    dz0 = np.einsum("bji,bj->bi", J_0, lam[:, 0])
    c = alpha if is_residual(layer) else 1.0
    dW = np.empty((L, w, w))
    db = np.empty((L, w))
    for l in range(L):
        _, d = activation(layer, preactivation(W[l], bias[l], Zprev[:, l]))
        g = c * d * lam[:, l]                        # dLoss / d(pre-activation)
        dW[l] = g.T @ Zprev[:, l]
        db[l] = g.sum(axis=0)
    return lam, dz0, dW, db


def loss(layer: int, alpha: float, W, bias, z0, G):
    """Loss = sum_b <G_b, Z_{b, L-1}> through the sequential pass."""
    Z = seq_forward(layer, alpha, W, bias, z0)
    return float(np.sum(_f64(G) * Z[:, -1]))
