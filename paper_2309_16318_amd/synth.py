"""Seeded synthetic inputs for the DeepPCR workloads.

This module only draws random numbers and shapes them; it holds none of the
method's arithmetic (no layer evaluation, no Jacobians, no solves).  Both the
GPU path's tests/bench and the CPU oracle receive the arrays produced here.

Distributions follow the workload definitions.  N(m, v) is read as mean m and
VARIANCE v (N(0, 1/w) only makes sense as a variance), so W has standard
deviation 1/sqrt(w) and the bias sqrt(0.1).  Every array is drawn in float64
from ``numpy.random.default_rng(seed)`` (PCG64) in a fixed order and then
rounded to float32, so every consumer sees bit-identical float32 inputs.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

# layer codes (2 * activation + residual; activation 0 tanh, 1 sigmoid, 2 ReLU)
TANH_MLP, TANH_RESIDUAL, SIGMOID_MLP, SIGMOID_RESIDUAL, RELU_MLP, RELU_RESIDUAL = range(6)


@dataclass(frozen=True)
class Workload:
    """One named workload: shapes, layer kind and Newton settings."""

    name: str
    kind: str            # "pcr" (standalone solve) or "mlp"
    B: int
    L: int
    w: int
    layer: int = TANH_MLP
    alpha: float = 1.0
    tol: float = 1e-5
    max_iter: int = 20
    transpose: int = 1   # standalone solve: backward-pass (transposed) form
    passes: tuple = field(default=("fwd",))
    seed: int = 0
    skip: int = 1        # collapsed-skip ResNet: layers per block
    act: int = 2         # collapsed-skip ResNet activation: 0 tanh, 1 sigmoid, 2 ReLU
    hidden: int = 0      # diffusion-style sampler: denoiser width
    chunks: int = 1      # row-chunked solve: chunks of the depth split


# The measured workloads (tanh MLPs / residual nets with
# random weights, a standalone block-bidiagonal solve, and the collapsed-skip
# ResNet).
WORKLOADS = {
    "tiny_fwd": Workload("tiny_fwd", "mlp", B=1, L=16, w=4, passes=("fwd",)),
    "pcr_solve": Workload("pcr_solve", "pcr", B=64, L=1024, w=16, transpose=1,
                          passes=("pcr",)),
    "mlp_fwd": Workload("mlp_fwd", "mlp", B=256, L=256, w=32, passes=("fwd",)),
    "mlp_bwd": Workload("mlp_bwd", "mlp", B=64, L=1024, w=64, passes=("bwd",)),
    "resnet_fwd_bwd": Workload("resnet_fwd_bwd", "mlp", B=16, L=1024, w=128,
                               layer=TANH_RESIDUAL, alpha=0.1,
                               passes=("fwd", "bwd")),
    # the paper's ResNet (App. A.3): width 16, ReLU, a skip every 4 layers,
    # depth 1024, Newton + PCR forward and the transposed backward
    "resnet_skip4_fwd_bwd": Workload("resnet_skip4_fwd_bwd", "resnet", B=64, L=1024, w=16,
                                     passes=("fwd", "bwd"), skip=4, act=2),
    # the standalone solve's system computed over 8 row chunks (the
    # single-GPU part of a depth split over 8 devices)
    "pcr_solve_chunked": Workload("pcr_solve_chunked", "pcr", B=64, L=1024, w=16, transpose=1,
                                  passes=("pcr",), chunks=8),
    # the paper's widest MLP width (Sec. 4.1): tiled block products
    "mlp_wide_fwd_bwd": Workload("mlp_wide_fwd_bwd", "mlp", B=1, L=256, w=1024,
                                 passes=("fwd", "bwd")),
    # a diffusion-style sampler (App. A.4): 1024 denoising steps of a 64-wide
    # latent with a synthetic 128-wide denoiser, steps evaluated by the caller
    "diffusion_generic": Workload("diffusion_generic", "diffusion", B=16, L=1024, w=64,
                                  passes=("fwd",), hidden=128, max_iter=30),
}


def _f32(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def mlp_inputs(B: int, L: int, w: int, seed: int = 0) -> dict:
    """Random MLP parameters, input and output cotangent.

    Draw order: W, bias, z0, G.
      W[L, w, w]  ~ N(0, 1/w)   (row-major, W[l] acts on column vectors)
      bias[L, w]  ~ N(0, 0.1)
      z0[B, w]    ~ N(0, 1)
      G[B, w]     ~ N(0, 1)     (dLoss/dZ_{L-1} for Loss = sum_b <G_b, Z_{b,L-1}>)
    """
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((L, w, w)) / np.sqrt(w)
    bias = rng.standard_normal((L, w)) * np.sqrt(0.1)
    z0 = rng.standard_normal((B, w))
    G = rng.standard_normal((B, w))
    return {"W": _f32(W), "bias": _f32(bias), "z0": _f32(z0), "G": _f32(G)}


def resnet_inputs(B: int, L: int, w: int, seed: int = 0) -> dict:
    """Random fully connected ResNet parameters (the collapsed-skip network).

    Draw order: W, bias, z0, G.  Weights and biases follow the default
    initialization of a fully connected layer in PyTorch (uniform on
    [-1/sqrt(w), 1/sqrt(w)] for both), the usual starting point of the
    training runs the network is used in:
      W[L, w, w]  ~ U(-1/sqrt(w), 1/sqrt(w))
      bias[L, w]  ~ U(-1/sqrt(w), 1/sqrt(w))
      z0[B, w]    ~ N(0, 1)
      G[B, w]     ~ N(0, 1)
    """
    rng = np.random.default_rng(seed)
    bound = 1.0 / np.sqrt(w)
    W = rng.uniform(-bound, bound, size=(L, w, w))
    bias = rng.uniform(-bound, bound, size=(L, w))
    z0 = rng.standard_normal((B, w))
    G = rng.standard_normal((B, w))
    return {"W": _f32(W), "bias": _f32(bias), "z0": _f32(z0), "G": _f32(G)}


def diffusion_inputs(B: int, L: int, w: int, h: int, seed: int = 0) -> dict:
    """A synthetic, untrained one-hidden-layer denoiser and the noise of one
    denoising run.

    Draw order: W1, b1, W2, b2, temb, zT, eps.
      W1[h, w], b1[h]  ~ U(-1/sqrt(w), 1/sqrt(w))   (default fully connected init)
      W2[w, h], b2[w]  ~ U(-1/sqrt(h), 1/sqrt(h))
      temb[L, h]       ~ N(0, 1)    (time embedding of schedule index t = 1..L)
      zT[B, w]         ~ N(0, 1)    (the starting noise)
      eps[B, L, w]     ~ N(0, 1)    (the normal sample each step adds)
    """
    rng = np.random.default_rng(seed)
    bw, bh = 1.0 / np.sqrt(w), 1.0 / np.sqrt(h)
    W1 = rng.uniform(-bw, bw, size=(h, w))
    b1 = rng.uniform(-bw, bw, size=(h,))
    W2 = rng.uniform(-bh, bh, size=(w, h))
    b2 = rng.uniform(-bh, bh, size=(w,))
    temb = rng.standard_normal((L, h))
    zT = rng.standard_normal((B, w))
    eps = rng.standard_normal((B, L, w))
    return {"W1": _f32(W1), "b1": _f32(b1), "W2": _f32(W2), "b2": _f32(b2),
            "temb": _f32(temb), "zT": _f32(zT), "eps": _f32(eps)}


def haar_orthogonal(rng: np.random.Generator, shape_prefix: tuple, w: int) -> np.ndarray:
    """Haar-distributed orthogonal w x w matrices: QR of a Gaussian, with the
    signs of R's diagonal folded into Q."""
    g = rng.standard_normal(shape_prefix + (w, w))
    q, rr = np.linalg.qr(g)
    sgn = np.sign(np.diagonal(rr, axis1=-2, axis2=-1))
    sgn[sgn == 0] = 1.0
    return q * sgn[..., None, :]


def pcr_inputs(B: int, L: int, w: int, seed: int = 0) -> dict:
    """Standalone block-bidiagonal system.

    Draw order: the Gaussian for QR, then u, then r.
      J[b, l] = 0.9 * Q[b, l] @ diag(u[b, l]),  Q Haar orthogonal, u ~ U(0, 1)
      r[B, L, w] ~ N(0, 1)
    """
    rng = np.random.default_rng(seed)
    q = haar_orthogonal(rng, (B, L), w)
    u = rng.uniform(0.0, 1.0, size=(B, L, w))
    r = rng.standard_normal((B, L, w))
    J = 0.9 * q * u[..., None, :]
    return {"J": _f32(J), "r": _f32(r)}


def random_system(B: int, L: int, w: int, seed: int, scale: float = 1.0) -> dict:
    """Generic random system for shape sweeps: J ~ N(0, scale^2 / w), r ~ N(0, 1)."""
    rng = np.random.default_rng(seed)
    J = rng.standard_normal((B, L, w, w)) * (scale / np.sqrt(w))
    r = rng.standard_normal((B, L, w))
    return {"J": _f32(J), "r": _f32(r)}


def workload_inputs(wl: Workload) -> dict:
    if wl.kind == "pcr":
        return pcr_inputs(wl.B, wl.L, wl.w, wl.seed)
    if wl.kind == "resnet":
        return resnet_inputs(wl.B, wl.L, wl.w, wl.seed)
    if wl.kind == "diffusion":
        return diffusion_inputs(wl.B, wl.L, wl.w, wl.hidden, wl.seed)
    return mlp_inputs(wl.B, wl.L, wl.w, wl.seed)


def digest(arrays: dict) -> str:
    """sha256 over the named float32 arrays, in sorted-name order."""
    h = hashlib.sha256()
    for k in sorted(arrays):
        a = np.ascontiguousarray(arrays[k])
        h.update(k.encode())
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()
