"""CPU oracle for a diffusion-style step function (App. A.4): numpy float64.

TEST INFRASTRUCTURE, like the rest of this package: only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the GPU
library shares no code with it.

Denoising as a Markov chain (Eq. denoising_step of App. A.4).  Step
j = 0..L-1 (the paper's l = j + 1) uses the noise-schedule index
t = L - j (denoising runs from t = L down to t = 1):
    z_j = f_j(z_{j-1}) = (z_{j-1} - c_t g(z_{j-1}, t)) / sqrt(alpha_t) + sqrt(beta_t) eps_j,
    c_t = (1 - alpha_t) / sqrt(1 - alphabar_t),
starting from z_{-1} = z_T (pure noise), with the normal samples eps_j drawn
once and passed in.  Schedule (the linear one of Ho et al., 2020, over
T = L steps): beta_t from 1e-4 to 0.02, alpha_t = 1 - beta_t,
alphabar_t = alpha_1 ... alpha_t.  The denoiser g is a synthetic, untrained
one-hidden-layer network with a time embedding e_t:
    g(z, t) = W2 tanh(W1 z + b1 + e_t) + b2,
so that df_j/dz = (I - c_t W2 diag(1 - tanh(a)^2) W1) / sqrt(alpha_t).

Readings: the step's parenthesis prints z_l where the previous state
z_{l-1} is meant (the step maps z_{l-1} to z_l); the printed Jacobian drops
the 1/sqrt(alpha) factor of the denoiser term, so the Jacobian here is the
derivative of the step as written.
"""
from __future__ import annotations

import numpy as np

from .deeppcr_oracle import seq_solve


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def schedule(L: int):
    """(beta, alpha, alphabar) indexed by t = 1..L (entry t-1)."""
    beta = np.linspace(1e-4, 0.02, L) if L > 1 else np.array([1e-4])
    alpha = 1.0 - beta
    alphabar = np.cumprod(alpha)
    return beta, alpha, alphabar


def denoiser(p: dict, z, t: int):
    """g(z, t) = W2 tanh(W1 z + b1 + e_t) + b2 for a batch z [B, w]; returns
    (g, 1 - tanh(a)^2)."""
    a = _f64(z) @ _f64(p["W1"]).T + _f64(p["b1"]) + _f64(p["temb"])[t - 1]
    th = np.tanh(a)
    return th @ _f64(p["W2"]).T + _f64(p["b2"]), 1.0 - th * th


def step(p: dict, j: int, z_prev, eps_j):
    """f_j(z_prev) for step j (schedule index t = L - j)."""
    L = _f64(p["temb"]).shape[0]
    t = L - j
    beta, alpha, alphabar = schedule(L)
    c = (1.0 - alpha[t - 1]) / np.sqrt(1.0 - alphabar[t - 1])
    g, _ = denoiser(p, z_prev, t)
    return (_f64(z_prev) - c * g) / np.sqrt(alpha[t - 1]) + np.sqrt(beta[t - 1]) * _f64(eps_j)


def step_jacobian(p: dict, j: int, z_prev):
    """df_j/dz at z_prev as [B, w, w]."""
    L = _f64(p["temb"]).shape[0]
    t = L - j
    _, alpha, alphabar = schedule(L)
    c = (1.0 - alpha[t - 1]) / np.sqrt(1.0 - alphabar[t - 1])
    _, d = denoiser(p, z_prev, t)
    W1, W2 = _f64(p["W1"]), _f64(p["W2"])
    Jg = np.einsum("ik,bk,kj->bij", W2, d, W1)
    w = W1.shape[1]
    return (np.eye(w)[None] - c * Jg) / np.sqrt(alpha[t - 1])


def seq_sample(p: dict, zT, eps):
    """The sequential denoising pass: Z[:, j] = f_j(Z[:, j-1]), Z[:, -1] = zT."""
    eps = _f64(eps)
    B, L, w = eps.shape
    Z = np.empty((B, L, w))
    z = _f64(zT)
    for j in range(L):
        z = step(p, j, z, eps[:, j])
        Z[:, j] = z
    return Z


def initial_guess(p: dict, zT, eps):
    """Start of Newton on the denoising chain (App. F.2): every row holds the
    first step's output f_0(z_T).  Returns [B, L, w]."""
    eps = _f64(eps)
    L = eps.shape[1]
    f0 = step(p, 0, _f64(zT), eps[:, 0])
    return np.repeat(f0[:, None, :], L, axis=1)


def newton_sample(p: dict, zT, eps, tol: float, max_iter: int, Z_init=None, solve=seq_solve):
    """Newton on the denoising chain (Sec. 2, Eqs. 2-3) with the update rule
    max|dZ| < tol * max(1, max|Z|); start Z_init or f_0(zT) in every row
    (App. F.2).  Returns (Z, solves, converged, [max|dZ|])."""
    eps = _f64(eps)
    B, L, w = eps.shape
    zT = _f64(zT)
    if Z_init is None:
        Z = initial_guess(p, zT, eps)
    else:
        Z = _f64(Z_init).copy()
    hist = []
    for k in range(1, max_iter + 1):
        Zprev = np.concatenate([zT[:, None, :], Z[:, :-1]], axis=1)
        F = np.stack([step(p, j, Zprev[:, j], eps[:, j]) for j in range(L)], axis=1)
        J = np.stack([step_jacobian(p, j, Zprev[:, j]) for j in range(L)], axis=1)
        dZ = solve(J, F - Z)
        Z = Z + dZ
        m = float(np.max(np.abs(dZ)))
        hist.append(m)
        if tol > 0 and m < tol * max(1.0, float(np.max(np.abs(Z)))):
            return Z, k, True, hist
    return Z, max_iter, tol == 0, hist
