"""Newton + PCR for step functions the caller evaluates (Sec. 2, Eqs. 1-3).

DeepPCR needs, per Newton iteration, the step values f_l(z_{l-1}) and the
Jacobians df_l/dz at the current iterate, for all steps at once; everything
after that (the residual, the block-bidiagonal solve of Eq. 3 by PCR, the
update and the convergence measures) is the library's
`deeppcr_newton_step`.  `newton_generic` runs that loop for step and
Jacobian functions written in PyTorch (or anything that fills device
tensors), which is how the paper treats general sequences such as denoising
(App. A.4, Jacobians from autograd).  `denoising_steps` builds such a pair
for a diffusion-style step with a small untrained denoiser network.
"""
from __future__ import annotations

from . import deeppcr


def newton_generic(step_fn, jac_fn, z_start, L: int, tol: float = 1e-5, max_iter: int = 20,
                   Z_init=None, workspace=None, stream=None) -> deeppcr.ForwardResult:
    """Solve z_l = f_l(z_{l-1}), l = 0..L-1, z_{-1} = z_start [B, w].

    step_fn(Zprev) -> F [B, L, w] with F[:, l] = f_l(Zprev[:, l]);
    jac_fn(Zprev) -> J [B, L, w, w] with J[:, l] = df_l/dz at Zprev[:, l].
    Start: Z_init, or f_0(z_start) in every row (App. F.2).  Stops once
    max|dZ| < tol * max(1, max|Z|) (tol = 0: exactly max_iter iterations).
    """
    torch = deeppcr._torch()
    B, w = z_start.shape
    if Z_init is not None:
        Z = Z_init.clone().contiguous()
    else:
        F0 = step_fn(z_start[:, None, :].expand(B, L, w).contiguous())
        Z = F0[:, :1, :].expand(B, L, w).contiguous()
    if workspace is None:
        workspace = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w),
                                dtype=torch.uint8, device=z_start.device)
    last = 0.0
    for k in range(1, max_iter + 1):
        Zprev = torch.cat([z_start[:, None, :], Z[:, :-1, :]], dim=1)
        F = step_fn(Zprev).contiguous()
        J = jac_fn(Zprev).contiguous()
        r = deeppcr.deeppcr_newton_step(J, F, Z, tol=tol, workspace=workspace, stream=stream)
        last = r.max_update
        # the library's test: OK once converged, ENOCONV to go on
        if r.status != deeppcr.ENOCONV:
            return deeppcr.ForwardResult(Z, k, last, r.status)
    # tol = 0 asks for exactly max_iter iterations, which is not a failure
    return deeppcr.ForwardResult(Z, max_iter, last, deeppcr.ENOCONV if tol > 0 else deeppcr.OK)


def denoising_steps(p: dict, eps):
    """Step and Jacobian functions of a diffusion-style sampler (App. A.4).

    Step l (schedule index t = L - l, denoising from t = L to 1):
        z_l = (z_{l-1} - c_t g(z_{l-1}, t)) / sqrt(alpha_t) + sqrt(beta_t) eps_l,
        c_t = (1 - alpha_t) / sqrt(1 - alphabar_t),
    linear beta schedule from 1e-4 to 0.02 over L steps, and the denoiser
    g(z, t) = W2 tanh(W1 z + b1 + temb_t) + b2.  p holds device tensors W1
    [h, w], b1 [h], W2 [w, h], b2 [w], temb [L, h]; eps [B, L, w] are the
    normal samples the steps add.
    """
    torch = deeppcr._torch()
    W1, b1, W2, b2, temb = p["W1"], p["b1"], p["W2"], p["b2"], p["temb"]
    L = temb.shape[0]
    w = W1.shape[1]
    dev = W1.device
    beta = torch.linspace(1e-4, 0.02, L, dtype=torch.float64, device=dev)
    alpha = 1.0 - beta
    alphabar = torch.cumprod(alpha, 0)
    t = L - torch.arange(L, device=dev)          # schedule index of step l
    c = ((1.0 - alpha[t - 1]) / torch.sqrt(1.0 - alphabar[t - 1])).float()[:, None]
    isa = (1.0 / torch.sqrt(alpha[t - 1])).float()[:, None]
    sb = torch.sqrt(beta[t - 1]).float()[:, None]
    te = temb[t - 1]                              # [L, h]
    # W2 diag(d) W1 = sum_k d_k W2[:, k] W1[k, :]: the h rank-one products,
    # K[k] = W2[:, k] W1[k, :] flattened [h, w*w], so that the Jacobians of
    # all steps are one GEMM of the activation slopes against K
    K = (W2.t()[:, :, None] * W1[:, None, :]).reshape(W1.shape[0], w * w).contiguous()
    neg_ci = -(c * isa)                           # [L, 1]

    def pre(Zprev):
        return torch.matmul(Zprev, W1.t().contiguous()) + b1 + te

    def step_fn(Zprev):
        g = torch.matmul(torch.tanh(pre(Zprev)), W2.t().contiguous()) + b2
        return (Zprev - c * g) * isa + sb * eps

    def jac_fn(Zprev):
        th = torch.tanh(pre(Zprev))
        d = 1.0 - th * th                         # [B, L, h]
        # (I - c_t W2 diag(d) W1) / sqrt(alpha_t): the products' part in one
        # GEMM, then 1 / sqrt(alpha_t) on the diagonal
        J = torch.matmul(d * neg_ci, K).view(*d.shape[:-1], w, w)   # [B, L, w, w]
        J.diagonal(dim1=-2, dim2=-1).add_(isa)
        return J

    return step_fn, jac_fn
