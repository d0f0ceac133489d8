"""The C ABI loads, exports every function include/deeppcr.h declares, and
rejects invalid arguments before any HIP call (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2309_16318_amd import deeppcr

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "deeppcr.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"defined"})


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("pcr_solve_block_bidiag", "deeppcr_mlp_forward", "deeppcr_mlp_forward_residual",
              "deeppcr_mlp_backward", "deeppcr_workspace_bytes"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = deeppcr.lib()
    for n in declared_functions():
        assert hasattr(lib, n), n
        assert n in deeppcr.SIGNATURES, n


def test_workspace_sizes():
    f = deeppcr.workspace_bytes
    B, L, w = 3, 7, 5
    nA = B * L * w * w * 4
    nr = B * L * w * 4
    up = lambda x: (x + 255) // 256 * 256
    red = 3 * 256 * 4  # three sets of 256 reduction slots (max|dZ|, max|Z|, max|F|)
    assert f(deeppcr.OP_PCR, B, L, w) == 2 * up(nA) + 2 * up(nr) + red
    assert f(deeppcr.OP_FWD, B, L, w) == 2 * up(nA) + 2 * up(nr) + red
    assert f(deeppcr.OP_BWD, B, L, w) == 2 * up(nA) + 3 * up(nr) + red
    for bad in ((0, 1, 1), (1, 0, 1), (1, 1, 0), (1, 1, 1025), (-1, 4, 4)):
        assert f(deeppcr.OP_PCR, *bad) == 0
    assert f(7, 1, 1, 1) == 0


def test_status_strings():
    for s in range(6):
        assert deeppcr.status_string(s)
    assert deeppcr.status_string(99) == "unknown status"


# Fake, non-overlapping "device" addresses: validation must reject before use.
P = [ctypes.c_void_p(0x10000000 * (i + 1)) for i in range(12)]
BIG = 1 << 40


def _pcr(J=P[0], r=P[1], x=P[2], B=2, L=8, w=4, tr=0, ws=P[3], nws=BIG):
    return deeppcr.lib().pcr_solve_block_bidiag(J, r, x, B, L, w, tr, ws, nws, None)


def test_pcr_solve_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    assert _pcr(J=None) == E
    assert _pcr(r=None) == E
    assert _pcr(x=None) == E
    assert _pcr(ws=None) == E
    assert _pcr(B=0) == E
    assert _pcr(L=0) == E
    assert _pcr(w=0) == E
    assert _pcr(w=1025) == E
    assert _pcr(tr=2) == E
    # x overlapping J, workspace overlapping r
    assert _pcr(x=ctypes.c_void_p(P[0].value + 64)) == E
    assert _pcr(ws=ctypes.c_void_p(P[1].value - 16)) == E
    # x partially overlapping r (exact aliasing is allowed)
    assert _pcr(x=ctypes.c_void_p(P[1].value + 16)) == E
    assert _pcr(nws=deeppcr.workspace_bytes(deeppcr.OP_PCR, 2, 8, 4) - 1) == deeppcr.EWORKSPACE


def test_noalloc_solve_rejects_invalid_arguments_and_oversized_problems():
    E = deeppcr.EINVAL
    f = deeppcr.lib().pcr_solve_block_bidiag_noalloc

    def call(J=P[0], r=P[1], x=P[2], B=2, L=8, w=4, tr=0):
        return f(J, r, x, B, L, w, tr, None)

    assert deeppcr.lib().deeppcr_noalloc_scratch_bytes() == 64 << 20
    for k in ("J", "r", "x"):
        assert call(**{k: None}) == E
        assert call(**{k: ctypes.c_void_p(dict(J=P[0], r=P[1], x=P[2])[k].value + 4)}) == E
    assert call(w=1025) == E
    assert call(tr=2) == E
    assert call(x=ctypes.c_void_p(P[0].value + 64)) == E       # x over J
    assert call(x=ctypes.c_void_p(P[1].value + 16)) == E       # x partly over r
    # past the fixed scratch: the workspace the solve would need exceeds it
    cap = 64 << 20
    assert deeppcr.workspace_bytes(deeppcr.OP_PCR, 1, 512, 128) > cap
    assert call(B=1, L=512, w=128) == deeppcr.EWORKSPACE
    assert call(B=64, L=1024, w=16) == deeppcr.EWORKSPACE


def _fwd(W=P[0], b=P[1], z0=P[2], Z=P[3], B=2, L=8, w=4, layer=0, alpha=1.0, tol=1e-5,
         max_iter=20, Zi=None, ws=P[5], nws=BIG):
    it = ctypes.c_int(-1)
    lu = ctypes.c_float(-1)
    return deeppcr.lib().deeppcr_mlp_forward(W, b, z0, Z, B, L, w, layer, alpha, tol, max_iter,
                                             Zi, ws, nws, ctypes.byref(it), ctypes.byref(lu),
                                             None)


def test_forward_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    assert _fwd(W=None) == E
    assert _fwd(Z=None) == E
    assert _fwd(layer=6) == E
    assert _fwd(layer=-1) == E
    assert _fwd(max_iter=0) == E
    assert _fwd(tol=-1.0) == E
    assert _fwd(tol=float("nan")) == E
    assert _fwd(tol=float("inf")) == E
    assert _fwd(alpha=float("nan")) == E
    assert _fwd(w=1025) == E
    assert _fwd(Zi=ctypes.c_void_p(P[3].value + 16)) == E     # partial overlap with Z
    assert _fwd(ws=ctypes.c_void_p(P[3].value)) == E          # workspace over Z
    assert _fwd(nws=100) == deeppcr.EWORKSPACE


def _fwd_res(W=P[0], b=P[1], z0=P[2], Z=P[3], B=2, L=8, w=4, layer=0, alpha=1.0, atol=1e-4,
             rtol=1e-4, max_iter=15, Zi=None, ws=P[5], nws=BIG):
    it = ctypes.c_int(-1)
    res = ctypes.c_float(-1)
    return deeppcr.lib().deeppcr_mlp_forward_residual(W, b, z0, Z, B, L, w, layer, alpha, atol,
                                                      rtol, max_iter, Zi, ws, nws,
                                                      ctypes.byref(it), ctypes.byref(res), None)


def test_forward_residual_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    assert _fwd_res(W=None) == E
    assert _fwd_res(b=None) == E
    assert _fwd_res(z0=None) == E
    assert _fwd_res(Z=None) == E
    assert _fwd_res(ws=None) == E
    assert _fwd_res(layer=6) == E
    assert _fwd_res(max_iter=-1) == E
    for bad in (-1.0, float("nan"), float("inf")):
        assert _fwd_res(atol=bad) == E
        assert _fwd_res(rtol=bad) == E
    assert _fwd_res(alpha=float("nan")) == E
    assert _fwd_res(B=0) == E
    assert _fwd_res(w=1025) == E
    assert _fwd_res(Zi=ctypes.c_void_p(P[3].value + 16)) == E
    assert _fwd_res(ws=ctypes.c_void_p(P[0].value)) == E      # workspace over W
    assert _fwd_res(nws=100) == deeppcr.EWORKSPACE


def _bwd(ptrs=None, B=2, L=8, w=4, layer=0, alpha=1.0, ws=P[10], nws=BIG):
    p = list(P[:9]) if ptrs is None else ptrs
    return deeppcr.lib().deeppcr_mlp_backward(*p, B, L, w, layer, alpha, ws, nws, None)


def test_backward_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    for i in range(9):
        p = list(P[:9])
        p[i] = None
        assert _bwd(p) == E
    p = list(P[:9])
    p[5] = P[3]  # Lambda over Z
    assert _bwd(p) == E
    p = list(P[:9])
    p[7] = ctypes.c_void_p(P[8].value - 16)  # dW runs into db
    assert _bwd(p) == E
    assert _bwd(layer=-1) == E
    assert _bwd(layer=6) == E
    assert _bwd(w=0) == E
    assert _bwd(alpha=float("inf")) == E
    assert _bwd(nws=1) == deeppcr.EWORKSPACE


def test_profile_read_rejects_bad_class():
    st = deeppcr.lib().deeppcr_profile_read(99, None, None, None, None)
    assert st == deeppcr.EINVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(deeppcr, "_lib", None)
    monkeypatch.setattr(deeppcr, "LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(RuntimeError, match="missing"):
        deeppcr.lib()


def test_sequential_passes_reject_invalid_arguments():
    E = deeppcr.EINVAL
    f = deeppcr.lib().deeppcr_seq_forward
    assert f(None, P[1], P[2], P[3], 2, 8, 4, 0, 1.0, 0, None) == E
    assert f(P[0], P[1], P[2], P[3], 2, 8, 0, 0, 1.0, 0, None) == E
    assert f(P[0], P[1], P[2], P[3], 2, 8, 4, 6, 1.0, 0, None) == E
    assert f(P[0], P[1], P[2], P[3], 2, 8, 4, 0, 1.0, 2, None) == E
    assert f(P[0], P[1], P[2], ctypes.c_void_p(P[0].value + 16), 2, 8, 4, 0, 1.0, 0, None) == E
    g = deeppcr.lib().deeppcr_seq_backward
    assert g(*P[:6], None, 2, 8, 4, 0, 1.0, 0, None) == E
    assert g(*P[:7], 2, 8, 4, -1, 1.0, 0, None) == E
    assert g(*P[:5], P[3], P[6], 2, 8, 4, 0, 1.0, 0, None) == E   # Lambda over Z


def test_wide_widths_accepted_up_to_1024():
    """The plain entry points take 1 <= w <= 1024; the ResNet and chunked
    entry points stop at 128."""
    assert deeppcr.MAX_WIDTH == 1024 and deeppcr.MAX_BLOCK_WIDTH == 128
    for w in (129, 130, 256, 1000, 1024):
        assert deeppcr.workspace_bytes(deeppcr.OP_FWD, 1, 4, w) > 0
        assert _pcr(w=w, nws=10) == deeppcr.EWORKSPACE   # valid shape, short workspace
    assert deeppcr.lib().deeppcr_resnet_workspace_bytes(deeppcr.OP_FWD, 1, 8, 129, 4) == 0
    assert deeppcr.lib().deeppcr_chunked_workspace_bytes(1, 8, 129, 2) == 0


def test_resnet_workspace_sizes():
    f = deeppcr.resnet_workspace_bytes
    B, L, w, skip = 3, 12, 5, 4
    G = L // skip
    up = lambda x: (x + 255) // 256 * 256
    nA, nr = B * G * w * w * 4, B * G * w * 4
    red = 3 * 256 * 4
    assert f(deeppcr.OP_FWD, B, L, w, skip) == 2 * up(nA) + 3 * up(nr) + red
    assert f(deeppcr.OP_BWD, B, L, w, skip) == 2 * up(nA) + 2 * up(nr) + red
    assert f(deeppcr.OP_PCR, B, L, w, skip) == 0
    for bad in ((B, 10, w, 4), (B, L, w, 0), (0, L, w, 4), (B, L, 129, 4)):
        assert f(deeppcr.OP_FWD, *bad) == 0


def _rfwd(W=P[0], b=P[1], z0=P[2], Z=P[3], B=2, L=8, w=4, skip=4, act=2, tol=1e-5, max_iter=20,
          Zi=None, ws=P[5], nws=BIG):
    it = ctypes.c_int(-1)
    lu = ctypes.c_float(-1)
    return deeppcr.lib().deeppcr_resnet_forward(W, b, z0, Z, B, L, w, skip, act, tol, max_iter,
                                                Zi, ws, nws, ctypes.byref(it), ctypes.byref(lu),
                                                None)


def test_resnet_forward_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    for k in ("W", "b", "z0", "Z", "ws"):
        assert _rfwd(**{k: None}) == E
    assert _rfwd(skip=0) == E
    assert _rfwd(skip=3) == E            # L = 8 is not a multiple of 3
    assert _rfwd(act=3) == E
    assert _rfwd(act=-1) == E
    assert _rfwd(tol=-1.0) == E
    assert _rfwd(tol=float("nan")) == E
    assert _rfwd(max_iter=0) == E
    assert _rfwd(w=129) == E
    assert _rfwd(Zi=ctypes.c_void_p(P[3].value + 16)) == E
    assert _rfwd(ws=ctypes.c_void_p(P[1].value)) == E
    assert _rfwd(nws=100) == deeppcr.EWORKSPACE


def _rbwd(ptrs=None, B=2, L=8, w=4, skip=2, act=0, ws=P[10], nws=BIG):
    p = list(P[:8]) if ptrs is None else ptrs
    return deeppcr.lib().deeppcr_resnet_backward(*p, B, L, w, skip, act, ws, nws, None)


def test_resnet_backward_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    for i in range(8):
        p = list(P[:8])
        p[i] = None
        assert _rbwd(p) == E
    p = list(P[:8])
    p[4] = P[2]  # Lambda over Z
    assert _rbwd(p) == E
    p = list(P[:8])
    p[6] = ctypes.c_void_p(P[7].value - 16)  # dW runs into db
    assert _rbwd(p) == E
    assert _rbwd(skip=3) == E
    assert _rbwd(act=5) == E
    assert _rbwd(ws=ctypes.c_void_p(P[0].value)) == E
    assert _rbwd(nws=1) == deeppcr.EWORKSPACE


def test_resnet_sequential_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    f = deeppcr.lib().deeppcr_resnet_seq_forward
    assert f(None, P[1], P[2], P[3], 2, 8, 4, 4, 2, 0, None) == E
    assert f(P[0], P[1], P[2], P[3], 2, 8, 4, 3, 2, 0, None) == E      # L % skip != 0
    assert f(P[0], P[1], P[2], P[3], 2, 8, 4, 4, 7, 0, None) == E      # unknown activation
    assert f(P[0], P[1], P[2], P[0], 2, 8, 4, 4, 2, 0, None) == E      # Z over W
    assert f(P[0], P[1], P[2], P[3], 2, 8, 4, 4, 2, 2, None) == E      # launch_per_layer
    fb = deeppcr.lib().deeppcr_resnet_seq_backward
    assert fb(P[0], P[1], P[2], P[3], None, P[5], 2, 8, 4, 4, 2, 0, None) == E
    assert fb(P[0], P[1], P[2], P[3], P[2], P[5], 2, 8, 4, 4, 2, 0, None) == E  # Lambda over Z
    assert fb(P[0], P[1], P[2], P[3], P[4], P[5], 2, 8, 4, 0, 2, 0, None) == E
    assert fb(P[0], P[1], P[2], P[3], P[4], P[5], 2, 8, 4, 4, 2, -1, None) == E


def test_newton_step_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    f = deeppcr.lib().deeppcr_newton_step

    def call(J=P[0], F=P[1], Z=P[2], B=2, L=8, w=4, tol=1e-5, ws=P[3], nws=BIG):
        return f(J, F, Z, B, L, w, tol, ws, nws, None, None, None, None)

    assert call(J=None) == E
    assert call(F=None) == E
    assert call(Z=None) == E
    assert call(ws=None) == E
    assert call(w=1025) == E
    assert call(Z=ctypes.c_void_p(P[0].value + 64)) == E   # Z over J
    assert call(Z=P[1]) == E                                # Z over F
    assert call(ws=ctypes.c_void_p(P[2].value - 16)) == E   # workspace runs into Z
    assert call(nws=deeppcr.workspace_bytes(deeppcr.OP_PCR, 2, 8, 4) - 1) == deeppcr.EWORKSPACE
    for bad in (-1e-5, float("nan"), float("inf")):
        assert call(tol=bad) == E
    for k in ("J", "F", "Z", "ws"):
        assert call(**{k: ctypes.c_void_p(dict(J=P[0], F=P[1], Z=P[2], ws=P[3])[k].value + 4)}) == E


def _misaligned(p, off=4):
    return ctypes.c_void_p(p.value + off)


def test_every_entry_point_rejects_misaligned_pointers():
    """Every float array and the workspace must start on a 16-byte boundary;
    offsets of 4 and 8 bytes are rejected before any HIP call."""
    E = deeppcr.EINVAL
    for off in (4, 8):
        for i in range(4):
            args = dict(J=P[0], r=P[1], x=P[2], ws=P[3])
            k = list(args)[i]
            args[k] = _misaligned(args[k], off)
            assert _pcr(**args) == E, k
        for k, base in (("W", P[0]), ("b", P[1]), ("z0", P[2]), ("Z", P[3]), ("ws", P[5])):
            assert _fwd(**{k: _misaligned(base, off)}) == E, k
            assert _fwd_res(**{k: _misaligned(base, off)}) == E, k
            assert _rfwd(**{k: _misaligned(base, off)}) == E, k
        assert _fwd(Zi=_misaligned(P[6], off)) == E
        for i in range(9):
            p = list(P[:9])
            p[i] = _misaligned(p[i], off)
            assert _bwd(p) == E, i
        assert _bwd(ws=_misaligned(P[10], off)) == E
        for i in range(8):
            p = list(P[:8])
            p[i] = _misaligned(p[i], off)
            assert _rbwd(p) == E, i
        sf = deeppcr.lib().deeppcr_seq_forward
        sb = deeppcr.lib().deeppcr_seq_backward
        rf = deeppcr.lib().deeppcr_resnet_seq_forward
        rb = deeppcr.lib().deeppcr_resnet_seq_backward
        for i in range(4):
            p = list(P[:4])
            p[i] = _misaligned(p[i], off)
            assert sf(*p, 2, 8, 4, 0, 1.0, 0, None) == E, i
            assert rf(*p, 2, 8, 4, 4, 2, 0, None) == E, i
        for i in range(7):
            p = list(P[:7])
            p[i] = _misaligned(p[i], off)
            assert sb(*p, 2, 8, 4, 0, 1.0, 0, None) == E, i
        for i in range(6):
            p = list(P[:6])
            p[i] = _misaligned(p[i], off)
            assert rb(*p, 2, 8, 4, 4, 2, 0, None) == E, i


def test_release_thread_state_without_a_gpu():
    """Nothing was allocated on this thread (no Newton call ran): releasing
    is a no-op and can be repeated."""
    deeppcr.release_thread_state()
    deeppcr.release_thread_state()


def test_chunked_workspace_sizes():
    f = deeppcr.lib().deeppcr_chunked_workspace_bytes
    up = lambda x: (x + 255) // 256 * 256
    B, L, w = 3, 10, 5
    nA, nr = B * L * w * w * 4, B * L * w * 4
    # G = 4 over 10 rows: chunks of 3, so 4 chunks; G = 6: chunks of 2, 5 chunks
    assert f(B, L, w, 4) == 2 * up(nA) + 2 * up(nr) + up(B * 4 * w * 4)
    assert f(B, L, w, 6) == 2 * up(nA) + 2 * up(nr) + up(B * 5 * w * 4)
    assert f(B, L, w, 1) == 2 * up(nA) + 2 * up(nr) + up(B * w * 4)
    for bad in ((0, 4, 4, 2), (1, 0, 4, 2), (1, 4, 129, 2), (1, 4, 4, 0), (1, 4, 4, -3)):
        assert f(*bad) == 0


def test_chunked_solve_rejects_invalid_arguments():
    E = deeppcr.EINVAL
    fn = deeppcr.lib().pcr_solve_block_bidiag_chunked

    def call(J=P[0], r=P[1], x=P[2], B=2, L=8, w=4, tr=0, G=2, ws=P[3], nws=BIG):
        return fn(J, r, x, B, L, w, tr, G, ws, nws, None)

    for k in ("J", "r", "x", "ws"):
        assert call(**{k: None}) == E
        assert call(**{k: _misaligned(dict(J=P[0], r=P[1], x=P[2], ws=P[3])[k], 4)}) == E
    assert call(G=0) == E
    assert call(G=-1) == E
    assert call(tr=2) == E
    assert call(w=129) == E
    assert call(B=0) == E
    assert call(x=ctypes.c_void_p(P[0].value + 64)) == E       # x over J
    assert call(x=ctypes.c_void_p(P[1].value + 16)) == E       # x partly over r
    assert call(ws=ctypes.c_void_p(P[1].value - 16)) == E      # workspace over r
    need = deeppcr.lib().deeppcr_chunked_workspace_bytes(2, 8, 4, 2)
    assert call(nws=need - 1) == deeppcr.EWORKSPACE
