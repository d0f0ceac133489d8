"""Row-chunked (L-sharded) solve of the block-bidiagonal system: CPU oracle.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this module; the GPU library never calls it and
shares no code with it.  numpy float64.

The system is that of Eq. 3 (and its transpose, App. A.2, Eq. 12):
    transpose=False:  x_l = J_l x_{l-1} + r_l,       l = 0..L-1, x_{-1} = 0
    transpose=True:   x_l = J_{l+1}^T x_{l+1} + r_l, l = L-1..0, x_L = 0
Its rows are cut into consecutive chunks of Lc = ceil(L / G) rows (the last
chunk may be shorter), as a solve spread over G devices would hold them.
Substituting the equations of one chunk into each other (what PCR does
pairwise in Eqs. 4-6 of Sec. 3) leaves every row of the chunk an affine
function of the one unknown that couples the chunk to the rest of the system,
x_in (the row before the chunk, or after it for the transposed system):
    x_l = P_l x_in + q_l.
Forward chunk [a, e):    x_in = x_{a-1},  P_l = J_l J_{l-1} ... J_a,
                         q_l = x_l computed from x_{a-1} = 0.
Transposed chunk [a, e): x_in = x_e,      P_l = J_{l+1}^T J_{l+2}^T ... J_e^T,
                         q_l = x_l computed from x_e = 0.
The chunk holding row 0 (forward) or row L-1 (transposed) has no coupling
(x_{-1} = 0, x_L = 0; J_0 never enters): its P is 0.
The chunk-end maps chain the chunks: the carry-in of the next chunk (in the
direction of the substitution) is P x_in + q at the current chunk's last row,
starting from 0 at the first chunk; each row is then P_l x_in + q_l.

Parity status: pinned by CPU tests against dense LAPACK solves, against the
substitution (seq_solve), and by the closed forms of J = a I.
"""
from __future__ import annotations

import numpy as np


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def chunk_bounds(L: int, G: int) -> list[tuple[int, int]]:
    """The chunks [a, e) of rows 0..L-1: Lc = ceil(L / G) rows each, the last
    one shorter when G does not divide L (so there may be fewer than G)."""
    if L < 1 or G < 1:
        raise ValueError("L and G must be positive")
    Lc = -(-L // G)
    return [(a, min(L, a + Lc)) for a in range(0, L, Lc)]


def chunk_maps(J, r, a: int, e: int, transpose: bool = False):
    """(P, q) of the rows a..e-1: P [B, e-a, w, w], q [B, e-a, w], built by
    multiplying out the chunk's recurrence one row at a time."""
    J, r = _f64(J), _f64(r)
    B, L, w = r.shape
    n = e - a
    P = np.empty((B, n, w, w))
    q = np.empty((B, n, w))
    eye = np.broadcast_to(np.eye(w), (B, w, w))
    if not transpose:
        Pp, qp = eye, np.zeros((B, w))                  # x_{a-1} = I x_in + 0
        for l in range(a, e):
            if l > 0:
                P[:, l - a] = J[:, l] @ Pp
                q[:, l - a] = np.einsum("bij,bj->bi", J[:, l], qp) + r[:, l]
            else:                                       # x_{-1} = 0: J_0 never enters
                P[:, l - a] = 0.0
                q[:, l - a] = r[:, l]
            Pp, qp = P[:, l - a], q[:, l - a]
    else:
        Pp, qp = eye, np.zeros((B, w))                  # x_e = I x_in + 0
        for l in range(e - 1, a - 1, -1):
            if l + 1 < L:
                JT = np.swapaxes(J[:, l + 1], -1, -2)
                P[:, l - a] = JT @ Pp
                q[:, l - a] = np.einsum("bij,bj->bi", JT, qp) + r[:, l]
            else:                                       # x_L = 0: no coupling
                P[:, l - a] = 0.0
                q[:, l - a] = r[:, l]
            Pp, qp = P[:, l - a], q[:, l - a]
    return P, q


def chunked_solve(J, r, transpose: bool = False, G: int = 1, return_carry: bool = False):
    """x of the block-bidiagonal system, computed chunk by chunk: the chunk
    maps, a sequential pass over the chunk ends for the carry-ins, then
    x_l = P_l x_in + q_l.  With return_carry also the carry-in x_in of every
    chunk ([B, n_chunks, w], in chunk order)."""
    J, r = _f64(J), _f64(r)
    B, L, w = r.shape
    chunks = chunk_bounds(L, G)
    maps = [chunk_maps(J, r, a, e, transpose) for a, e in chunks]
    xin = np.zeros((B, len(chunks), w))
    order = range(len(chunks)) if not transpose else range(len(chunks) - 1, -1, -1)
    carry = np.zeros((B, w))
    for g in order:
        xin[:, g] = carry
        P, q = maps[g]
        end = -1 if not transpose else 0                # the chunk's last row in solve order
        carry = np.einsum("bij,bj->bi", P[:, end], carry) + q[:, end]
    x = np.empty((B, L, w))
    for g, (a, e) in enumerate(chunks):
        P, q = maps[g]
        x[:, a:e] = np.einsum("blij,bj->bli", P, xin[:, g]) + q
    return (x, xin) if return_carry else x
