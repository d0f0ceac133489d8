"""ctypes binding of libdeeppcr.so (include/deeppcr.h).

Argument marshalling only: torch tensors provide device memory and the
current HIP stream; every step of the computation runs in the library's
kernels.  There is no CPU fallback: if the library is missing, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

OK, EINVAL, ENOCONV, ENONFINITE, EHIP, EWORKSPACE = range(6)
TANH_MLP, TANH_RESIDUAL, SIGMOID_MLP, SIGMOID_RESIDUAL, RELU_MLP, RELU_RESIDUAL = range(6)
OP_PCR, OP_FWD, OP_BWD = 0, 1, 2
ACT_TANH, ACT_SIGMOID, ACT_RELU = 0, 1, 2
(KCLASS_PCR_LEVEL, KCLASS_LAYER, KCLASS_UPDATE, KCLASS_WGRAD, KCLASS_OTHER, KCLASS_SEQUENTIAL,
 KCLASS_PCR_TAIL) = range(7)
KCLASS_NAMES = ("pcr_level", "layer", "update", "wgrad", "other", "sequential", "pcr_tail")
MAX_WIDTH = 1024
MAX_BLOCK_WIDTH = 128  # collapsed-skip ResNet and the chunked solve

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdeeppcr.so")

# Every symbol declared in include/deeppcr.h, with its ctypes signature.
_c = ctypes
SIGNATURES = {
    "deeppcr_workspace_bytes": (_c.c_size_t, [_c.c_int, _c.c_int, _c.c_int, _c.c_int]),
    "deeppcr_status_string": (_c.c_char_p, [_c.c_int]),
    "deeppcr_last_error": (_c.c_char_p, []),
    "pcr_solve_block_bidiag": (_c.c_int, [_c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_int,
                                          _c.c_int, _c.c_int, _c.c_int, _c.c_void_p,
                                          _c.c_size_t, _c.c_void_p]),
    "pcr_solve_block_bidiag_noalloc": (_c.c_int, [_c.c_void_p, _c.c_void_p, _c.c_void_p,
                                                  _c.c_int, _c.c_int, _c.c_int, _c.c_int,
                                                  _c.c_void_p]),
    "deeppcr_noalloc_scratch_bytes": (_c.c_size_t, []),
    "deeppcr_chunked_workspace_bytes": (_c.c_size_t, [_c.c_int] * 4),
    "pcr_solve_block_bidiag_chunked": (_c.c_int, [_c.c_void_p] * 3 + [_c.c_int] * 5 +
                                       [_c.c_void_p, _c.c_size_t, _c.c_void_p]),
    "deeppcr_mlp_forward": (_c.c_int, [_c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_void_p,
                                       _c.c_int, _c.c_int, _c.c_int, _c.c_int, _c.c_float,
                                       _c.c_float, _c.c_int, _c.c_void_p, _c.c_void_p,
                                       _c.c_size_t, _c.POINTER(_c.c_int),
                                       _c.POINTER(_c.c_float), _c.c_void_p]),
    "deeppcr_newton_step": (_c.c_int, [_c.c_void_p] * 3 + [_c.c_int] * 3 +
                            [_c.c_float, _c.c_void_p, _c.c_size_t] +
                            [_c.POINTER(_c.c_float)] * 3 + [_c.c_void_p]),
    "deeppcr_release_thread_state": (None, []),
    "deeppcr_mlp_forward_residual": (_c.c_int, [_c.c_void_p, _c.c_void_p, _c.c_void_p,
                                                _c.c_void_p, _c.c_int, _c.c_int, _c.c_int,
                                                _c.c_int, _c.c_float, _c.c_float, _c.c_float,
                                                _c.c_int, _c.c_void_p, _c.c_void_p, _c.c_size_t,
                                                _c.POINTER(_c.c_int), _c.POINTER(_c.c_float),
                                                _c.c_void_p]),
    "deeppcr_mlp_backward": (_c.c_int, [_c.c_void_p] * 9 + [_c.c_int, _c.c_int, _c.c_int,
                                                           _c.c_int, _c.c_float, _c.c_void_p,
                                                           _c.c_size_t, _c.c_void_p]),
    "deeppcr_resnet_workspace_bytes": (_c.c_size_t, [_c.c_int] * 5),
    "deeppcr_resnet_forward": (_c.c_int, [_c.c_void_p] * 4 + [_c.c_int] * 5 +
                               [_c.c_float, _c.c_int, _c.c_void_p, _c.c_void_p, _c.c_size_t,
                                _c.POINTER(_c.c_int), _c.POINTER(_c.c_float), _c.c_void_p]),
    "deeppcr_resnet_backward": (_c.c_int, [_c.c_void_p] * 8 + [_c.c_int] * 5 +
                                [_c.c_void_p, _c.c_size_t, _c.c_void_p]),
    "deeppcr_resnet_seq_forward": (_c.c_int, [_c.c_void_p] * 4 + [_c.c_int] * 6 + [_c.c_void_p]),
    "deeppcr_resnet_seq_backward": (_c.c_int, [_c.c_void_p] * 6 + [_c.c_int] * 6 +
                                    [_c.c_void_p]),
    "deeppcr_seq_forward": (_c.c_int, [_c.c_void_p] * 4 + [_c.c_int] * 4 + [_c.c_float, _c.c_int,
                                                                          _c.c_void_p]),
    "deeppcr_seq_backward": (_c.c_int, [_c.c_void_p] * 7 + [_c.c_int] * 4 + [_c.c_float, _c.c_int,
                                                                           _c.c_void_p]),
    "deeppcr_profile_enable": (_c.c_int, [_c.c_int]),
    "deeppcr_profile_select": (_c.c_int, [_c.c_uint]),
    "deeppcr_profile_reset": (None, []),
    "deeppcr_profile_read": (_c.c_int, [_c.c_int, _c.POINTER(_c.c_longlong),
                                        _c.POINTER(_c.c_double), _c.POINTER(_c.c_double),
                                        _c.POINTER(_c.c_double)]),
}

_lib = None


class DeepPCRError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = f"{where}: {status_string(status)} (status {status})"
        if status == EHIP:
            msg += f": {lib().deeppcr_last_error().decode()}"
        super().__init__(msg)


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2309_16318_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def status_string(status: int) -> str:
    return lib().deeppcr_status_string(status).decode()


def workspace_bytes(op: int, B: int, L: int, w: int) -> int:
    return int(lib().deeppcr_workspace_bytes(op, B, L, w))


# ------------------------------------------------------------------ helpers
def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(t, shape, name):
    torch = _torch()
    if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _workspace(op, B, L, w, workspace, device):
    torch = _torch()
    n = workspace_bytes(op, B, L, w)
    if workspace is None:
        workspace = torch.empty(n, dtype=torch.uint8, device=device)
    return workspace, workspace.numel() * workspace.element_size()


# ------------------------------------------------------------- entry points
def pcr_solve_block_bidiag(J, r, x=None, transpose: int = 0, workspace=None, stream=None):
    """x with M x = r (transpose=0) or M^T x = r (transpose=1); J [B, L, w, w], r [B, L, w]."""
    torch = _torch()
    B, L, w = r.shape
    _check(J, (B, L, w, w), "J")
    _check(r, (B, L, w), "r")
    if x is None:
        x = torch.empty_like(r)
    _check(x, (B, L, w), "x")
    ws, nbytes = _workspace(OP_PCR, B, L, w, workspace, r.device)
    st = lib().pcr_solve_block_bidiag(_ptr(J), _ptr(r), _ptr(x), B, L, w, int(transpose),
                                      _ptr(ws), nbytes, _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "pcr_solve_block_bidiag")
    return x


def pcr_solve_block_bidiag_noalloc(J, r, x, transpose: int = 0, stream=None):
    """The same solve into the caller's x without a workspace: the library
    uses its own fixed scratch array and allocates nothing."""
    B, L, w = r.shape
    _check(J, (B, L, w, w), "J")
    _check(r, (B, L, w), "r")
    _check(x, (B, L, w), "x")
    st = lib().pcr_solve_block_bidiag_noalloc(_ptr(J), _ptr(r), _ptr(x), B, L, w, int(transpose),
                                              _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "pcr_solve_block_bidiag_noalloc")
    return x


def pcr_solve_block_bidiag_chunked(J, r, G: int, x=None, transpose: int = 0, workspace=None,
                                   stream=None):
    """The same solve computed over G row chunks (chunk-local PCR keeping each
    chunk's coupling, a pass over the chunk ends, then the apply)."""
    torch = _torch()
    B, L, w = r.shape
    _check(J, (B, L, w, w), "J")
    _check(r, (B, L, w), "r")
    if x is None:
        x = torch.empty_like(r)
    _check(x, (B, L, w), "x")
    n = int(lib().deeppcr_chunked_workspace_bytes(B, L, w, int(G)))
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=r.device)
    nbytes = workspace.numel() * workspace.element_size()
    st = lib().pcr_solve_block_bidiag_chunked(_ptr(J), _ptr(r), _ptr(x), B, L, w, int(transpose),
                                              int(G), _ptr(workspace), nbytes, _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "pcr_solve_block_bidiag_chunked")
    return x


@dataclass
class ForwardResult:
    Z: object
    iters: int
    last_update: float
    status: int


def deeppcr_mlp_forward(W, bias, z0, Z=None, layer: int = TANH_MLP, alpha: float = 1.0,
                        tol: float = 1e-5, max_iter: int = 20, Z_init=None, workspace=None,
                        stream=None) -> ForwardResult:
    """Newton + PCR forward pass; raises on EINVAL/EHIP/EWORKSPACE and returns
    ENOCONV / ENONFINITE in ``status``."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    _check(W, (L, w, w), "W")
    _check(bias, (L, w), "bias")
    _check(z0, (B, w), "z0")
    if Z is None:
        Z = torch.empty((B, L, w), dtype=torch.float32, device=z0.device)
    _check(Z, (B, L, w), "Z")
    if Z_init is not None:
        _check(Z_init, (B, L, w), "Z_init")
    ws, nbytes = _workspace(OP_FWD, B, L, w, workspace, z0.device)
    iters = ctypes.c_int(0)
    last = ctypes.c_float(0.0)
    st = lib().deeppcr_mlp_forward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), B, L, w, int(layer),
                                   float(alpha), float(tol), int(max_iter), _ptr(Z_init),
                                   _ptr(ws), nbytes, ctypes.byref(iters), ctypes.byref(last),
                                   _stream(stream))
    if st not in (OK, ENOCONV, ENONFINITE):
        raise DeepPCRError(st, "deeppcr_mlp_forward")
    return ForwardResult(Z, iters.value, last.value, st)


@dataclass
class NewtonStepResult:
    residual: float
    max_update: float
    max_abs: float
    status: int


def deeppcr_newton_step(J, F, Z, tol: float = 1e-5, workspace=None,
                        stream=None) -> NewtonStepResult:
    """One Newton + PCR iteration for caller-evaluated step values F and
    Jacobians J at the iterate Z (updated in place); ``status`` is OK once
    the update meets ``tol``, ENOCONV before, ENONFINITE on a NaN/Inf."""
    B, L, w = Z.shape
    _check(J, (B, L, w, w), "J")
    _check(F, (B, L, w), "F")
    _check(Z, (B, L, w), "Z")
    ws, nbytes = _workspace(OP_PCR, B, L, w, workspace, Z.device)
    res, mx, mz = ctypes.c_float(0.0), ctypes.c_float(0.0), ctypes.c_float(0.0)
    st = lib().deeppcr_newton_step(_ptr(J), _ptr(F), _ptr(Z), B, L, w, float(tol), _ptr(ws),
                                   nbytes, ctypes.byref(res), ctypes.byref(mx), ctypes.byref(mz),
                                   _stream(stream))
    if st not in (OK, ENOCONV, ENONFINITE):
        raise DeepPCRError(st, "deeppcr_newton_step")
    return NewtonStepResult(res.value, mx.value, mz.value, st)


@dataclass
class ResidualForwardResult:
    Z: object
    iters: int
    residual: float
    status: int


def deeppcr_mlp_forward_residual(W, bias, z0, Z=None, layer: int = TANH_MLP, alpha: float = 1.0,
                                 atol: float = 1e-4, rtol: float = 1e-4, max_iter: int = 15,
                                 Z_init=None, workspace=None,
                                 stream=None) -> ResidualForwardResult:
    """Newton + PCR forward pass stopped by the residual rule (defaults: the
    paper's forward-pass solver settings); raises on EINVAL/EHIP/EWORKSPACE
    and returns ENOCONV / ENONFINITE in ``status``."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    _check(W, (L, w, w), "W")
    _check(bias, (L, w), "bias")
    _check(z0, (B, w), "z0")
    if Z is None:
        Z = torch.empty((B, L, w), dtype=torch.float32, device=z0.device)
    _check(Z, (B, L, w), "Z")
    if Z_init is not None:
        _check(Z_init, (B, L, w), "Z_init")
    ws, nbytes = _workspace(OP_FWD, B, L, w, workspace, z0.device)
    iters = ctypes.c_int(0)
    res = ctypes.c_float(0.0)
    st = lib().deeppcr_mlp_forward_residual(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), B, L, w,
                                            int(layer), float(alpha), float(atol), float(rtol),
                                            int(max_iter), _ptr(Z_init), _ptr(ws), nbytes,
                                            ctypes.byref(iters), ctypes.byref(res),
                                            _stream(stream))
    if st not in (OK, ENOCONV, ENONFINITE):
        raise DeepPCRError(st, "deeppcr_mlp_forward_residual")
    return ResidualForwardResult(Z, iters.value, res.value, st)


def deeppcr_mlp_backward(W, bias, z0, Z, G, layer: int = TANH_MLP, alpha: float = 1.0,
                         Lambda=None, dz0=None, dW=None, db=None, workspace=None, stream=None):
    """Transposed-PCR backward pass; returns (Lambda, dz0, dW, db)."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    for t, shp, n in ((W, (L, w, w), "W"), (bias, (L, w), "bias"), (z0, (B, w), "z0"),
                      (Z, (B, L, w), "Z"), (G, (B, w), "G")):
        _check(t, shp, n)
    dev = z0.device
    Lambda = torch.empty((B, L, w), dtype=torch.float32, device=dev) if Lambda is None else Lambda
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev) if dz0 is None else dz0
    dW = torch.empty((L, w, w), dtype=torch.float32, device=dev) if dW is None else dW
    db = torch.empty((L, w), dtype=torch.float32, device=dev) if db is None else db
    for t, shp, n in ((Lambda, (B, L, w), "Lambda"), (dz0, (B, w), "dz0"), (dW, (L, w, w), "dW"),
                      (db, (L, w), "db")):
        _check(t, shp, n)
    ws, nbytes = _workspace(OP_BWD, B, L, w, workspace, dev)
    st = lib().deeppcr_mlp_backward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), _ptr(G),
                                    _ptr(Lambda), _ptr(dz0), _ptr(dW), _ptr(db), B, L, w,
                                    int(layer), float(alpha), _ptr(ws), nbytes, _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_mlp_backward")
    return Lambda, dz0, dW, db


def resnet_workspace_bytes(op: int, B: int, L: int, w: int, skip: int) -> int:
    return int(lib().deeppcr_resnet_workspace_bytes(op, B, L, w, skip))


def deeppcr_resnet_forward(W, bias, z0, skip: int, act: int = ACT_RELU, Z=None,
                           tol: float = 1e-5, max_iter: int = 20, Z_init=None, workspace=None,
                           stream=None) -> ForwardResult:
    """Newton + PCR forward pass of the collapsed-skip ResNet; raises on
    EINVAL/EHIP/EWORKSPACE and returns ENOCONV / ENONFINITE in ``status``."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    _check(W, (L, w, w), "W")
    _check(bias, (L, w), "bias")
    _check(z0, (B, w), "z0")
    if Z is None:
        Z = torch.empty((B, L, w), dtype=torch.float32, device=z0.device)
    _check(Z, (B, L, w), "Z")
    if Z_init is not None:
        _check(Z_init, (B, L, w), "Z_init")
    n = resnet_workspace_bytes(OP_FWD, B, L, w, skip)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=z0.device)
    nbytes = workspace.numel() * workspace.element_size()
    iters = ctypes.c_int(0)
    last = ctypes.c_float(0.0)
    st = lib().deeppcr_resnet_forward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), B, L, w, int(skip),
                                      int(act), float(tol), int(max_iter), _ptr(Z_init),
                                      _ptr(workspace), nbytes, ctypes.byref(iters),
                                      ctypes.byref(last), _stream(stream))
    if st not in (OK, ENOCONV, ENONFINITE):
        raise DeepPCRError(st, "deeppcr_resnet_forward")
    return ForwardResult(Z, iters.value, last.value, st)


def deeppcr_resnet_backward(W, z0, Z, G, skip: int, act: int = ACT_RELU, Lambda=None, dz0=None,
                            dW=None, db=None, workspace=None, stream=None):
    """Backward pass of the collapsed-skip ResNet; returns (Lambda, dz0, dW, db)."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    for t, shp, n in ((W, (L, w, w), "W"), (z0, (B, w), "z0"), (Z, (B, L, w), "Z"),
                      (G, (B, w), "G")):
        _check(t, shp, n)
    dev = z0.device
    Lambda = torch.empty((B, L, w), dtype=torch.float32, device=dev) if Lambda is None else Lambda
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev) if dz0 is None else dz0
    dW = torch.empty((L, w, w), dtype=torch.float32, device=dev) if dW is None else dW
    db = torch.empty((L, w), dtype=torch.float32, device=dev) if db is None else db
    for t, shp, n in ((Lambda, (B, L, w), "Lambda"), (dz0, (B, w), "dz0"), (dW, (L, w, w), "dW"),
                      (db, (L, w), "db")):
        _check(t, shp, n)
    n = resnet_workspace_bytes(OP_BWD, B, L, w, skip)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)
    nbytes = workspace.numel() * workspace.element_size()
    st = lib().deeppcr_resnet_backward(_ptr(W), _ptr(z0), _ptr(Z), _ptr(G), _ptr(Lambda),
                                       _ptr(dz0), _ptr(dW), _ptr(db), B, L, w, int(skip),
                                       int(act), _ptr(workspace), nbytes, _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_resnet_backward")
    return Lambda, dz0, dW, db


def deeppcr_resnet_seq_forward(W, bias, z0, skip: int, act: int = ACT_RELU, Z=None,
                               launch_per_layer: bool = False, stream=None):
    """Sequential GPU pass of the collapsed-skip ResNet; returns Z."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    Z = torch.empty((B, L, w), dtype=torch.float32, device=z0.device) if Z is None else Z
    _check(Z, (B, L, w), "Z")
    st = lib().deeppcr_resnet_seq_forward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), B, L, w,
                                          int(skip), int(act), int(bool(launch_per_layer)),
                                          _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_resnet_seq_forward")
    return Z


def deeppcr_resnet_seq_backward(W, z0, Z, G, skip: int, act: int = ACT_RELU, Lambda=None,
                                dz0=None, launch_per_layer: bool = False, stream=None):
    """Sequential GPU adjoints of the collapsed-skip ResNet; returns (Lambda, dz0)."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    dev = z0.device
    Lambda = torch.empty((B, L, w), dtype=torch.float32, device=dev) if Lambda is None else Lambda
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev) if dz0 is None else dz0
    st = lib().deeppcr_resnet_seq_backward(_ptr(W), _ptr(z0), _ptr(Z), _ptr(G), _ptr(Lambda),
                                           _ptr(dz0), B, L, w, int(skip), int(act),
                                           int(bool(launch_per_layer)), _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_resnet_seq_backward")
    return Lambda, dz0


def deeppcr_seq_forward(W, bias, z0, Z=None, layer: int = TANH_MLP, alpha: float = 1.0,
                        launch_per_layer: bool = False, stream=None):
    """Sequential layer-by-layer forward pass on the GPU (the comparison baseline)."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    for t, shp, n in ((W, (L, w, w), "W"), (bias, (L, w), "bias"), (z0, (B, w), "z0")):
        _check(t, shp, n)
    if Z is None:
        Z = torch.empty((B, L, w), dtype=torch.float32, device=z0.device)
    _check(Z, (B, L, w), "Z")
    st = lib().deeppcr_seq_forward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), B, L, w, int(layer),
                                   float(alpha), int(bool(launch_per_layer)), _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_seq_forward")
    return Z


def deeppcr_seq_backward(W, bias, z0, Z, G, layer: int = TANH_MLP, alpha: float = 1.0,
                         Lambda=None, dz0=None, launch_per_layer: bool = False, stream=None):
    """Sequential adjoint pass on the GPU; returns (Lambda, dz0)."""
    torch = _torch()
    L, w, _ = W.shape
    B = z0.shape[0]
    for t, shp, n in ((W, (L, w, w), "W"), (bias, (L, w), "bias"), (z0, (B, w), "z0"),
                      (Z, (B, L, w), "Z"), (G, (B, w), "G")):
        _check(t, shp, n)
    dev = z0.device
    Lambda = torch.empty((B, L, w), dtype=torch.float32, device=dev) if Lambda is None else Lambda
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev) if dz0 is None else dz0
    _check(Lambda, (B, L, w), "Lambda")
    _check(dz0, (B, w), "dz0")
    st = lib().deeppcr_seq_backward(_ptr(W), _ptr(bias), _ptr(z0), _ptr(Z), _ptr(G), _ptr(Lambda),
                                    _ptr(dz0), B, L, w, int(layer), float(alpha),
                                    int(bool(launch_per_layer)), _stream(stream))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_seq_backward")
    return Lambda, dz0


def release_thread_state() -> None:
    """Frees the calling thread's pinned read-back buffer and profiler events."""
    lib().deeppcr_release_thread_state()


# ---------------------------------------------------------- instrumentation
def profile_enable(on: bool = True) -> None:
    lib().deeppcr_profile_enable(1 if on else 0)


def profile_select(kclasses) -> None:
    """Times only the given kernel classes (KCLASS_* values) while enabled."""
    mask = 0
    for c in kclasses:
        mask |= 1 << int(c)
    lib().deeppcr_profile_select(mask)


def profile_reset() -> None:
    lib().deeppcr_profile_reset()


def profile_read(kclass: int) -> dict:
    n = ctypes.c_longlong(0)
    ms = ctypes.c_double(0)
    by = ctypes.c_double(0)
    fl = ctypes.c_double(0)
    st = lib().deeppcr_profile_read(kclass, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(by),
                                    ctypes.byref(fl))
    if st != OK:
        raise DeepPCRError(st, "deeppcr_profile_read")
    return {"launches": n.value, "ms": ms.value, "bytes": by.value, "flops": fl.value}
