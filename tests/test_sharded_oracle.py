"""Pins for the row-chunked solve of the oracle (the L-sharded layout of
Eq. 3): dense LAPACK solves, the substitution, closed forms of J = a I, and
the carry-in identity.  CPU only."""
import numpy as np
import pytest

import oracle
from oracle import sharded_oracle as so
from paper_2309_16318_amd import synth


def dense_matrix(J, transpose):
    """(L*w) x (L*w) matrix of Eq. 3: identity diagonal blocks, -J_l in block
    (l, l-1); optionally transposed."""
    L, w = J.shape[0], J.shape[1]
    M = np.eye(L * w)
    for l in range(1, L):
        M[l * w:(l + 1) * w, (l - 1) * w:l * w] = -J[l]
    return M.T if transpose else M


def dense_solve(J, r, transpose):
    B, L, w = r.shape
    x = np.empty((B, L, w))
    for b in range(B):
        M = dense_matrix(np.asarray(J[b], np.float64), transpose)
        x[b] = np.linalg.solve(M, np.asarray(r[b], np.float64).reshape(-1)).reshape(L, w)
    return x


def test_chunk_bounds():
    assert so.chunk_bounds(8, 4) == [(0, 2), (2, 4), (4, 6), (6, 8)]
    assert so.chunk_bounds(10, 4) == [(0, 3), (3, 6), (6, 9), (9, 10)]
    assert so.chunk_bounds(10, 3) == [(0, 4), (4, 8), (8, 10)]
    assert so.chunk_bounds(3, 8) == [(0, 1), (1, 2), (2, 3)]
    assert so.chunk_bounds(5, 1) == [(0, 5)]
    # 7 rows over 6 chunks of two: only 4 chunks exist
    assert so.chunk_bounds(7, 6) == [(0, 2), (2, 4), (4, 6), (6, 7)]
    with pytest.raises(ValueError):
        so.chunk_bounds(0, 2)


@pytest.mark.parametrize("L", [1, 2, 5, 8, 13])
@pytest.mark.parametrize("G", [1, 2, 3, 4, 8, 20])
@pytest.mark.parametrize("w", [1, 3])
@pytest.mark.parametrize("transpose", [False, True])
def test_chunked_solve_matches_dense_lapack(L, G, w, transpose):
    d = synth.random_system(2, L, w, seed=100 * L + 7 * G + w, scale=0.9)
    ref = dense_solve(d["J"], d["r"], transpose)
    got = so.chunked_solve(d["J"], d["r"], transpose, G)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("G", [2, 4, 7])
def test_chunked_solve_matches_substitution(transpose, G):
    d = synth.random_system(3, 61, 5, seed=G, scale=0.9)
    np.testing.assert_allclose(so.chunked_solve(d["J"], d["r"], transpose, G),
                               oracle.seq_solve(d["J"], d["r"], transpose),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("transpose", [False, True])
def test_carry_in_is_the_neighbouring_row(transpose):
    """x_in of a chunk is the solution at the row before it (after it, for the
    transposed system), and every row is P_l x_in + q_l with that x_in."""
    d = synth.random_system(2, 23, 4, seed=9, scale=0.9)
    x = dense_solve(d["J"], d["r"], transpose)
    _, xin = so.chunked_solve(d["J"], d["r"], transpose, 5, return_carry=True)
    for g, (a, e) in enumerate(so.chunk_bounds(23, 5)):
        nb = a - 1 if not transpose else e
        want = x[:, nb] if 0 <= nb < 23 else np.zeros((2, 4))
        np.testing.assert_allclose(xin[:, g], want, rtol=1e-11, atol=1e-12)
        P, q = so.chunk_maps(d["J"], d["r"], a, e, transpose)
        np.testing.assert_allclose(np.einsum("blij,bj->bli", P, want) + q, x[:, a:e],
                                   rtol=1e-11, atol=1e-12)


def test_chunk_maps_scaled_identity_closed_form():
    """J = a I: forward P_l = a^(l-a0+1) I, q_l = sum_{m=a0..l} a^(l-m) r_m;
    transposed P_l = a^(e-l) I, q_l = sum_{m=l..e-1} a^(m-l) r_m."""
    a, L, w = 0.7, 12, 2
    r = np.random.default_rng(3).standard_normal((1, L, w))
    J = np.broadcast_to(a * np.eye(w), (1, L, w, w)).copy()
    a0, e = 4, 9
    P, q = so.chunk_maps(J, r, a0, e, False)
    for l in range(a0, e):
        np.testing.assert_allclose(P[0, l - a0], a ** (l - a0 + 1) * np.eye(w), rtol=1e-14)
        np.testing.assert_allclose(q[0, l - a0], sum(a ** (l - m) * r[0, m] for m in range(a0, l + 1)),
                                   rtol=1e-13)
    P, q = so.chunk_maps(J, r, a0, e, True)
    for l in range(a0, e):
        np.testing.assert_allclose(P[0, l - a0], a ** (e - l) * np.eye(w), rtol=1e-14)
        np.testing.assert_allclose(q[0, l - a0], sum(a ** (m - l) * r[0, m] for m in range(l, e)),
                                   rtol=1e-13)


@pytest.mark.parametrize("transpose", [False, True])
def test_uncoupled_chunk_ignores_first_block(transpose):
    """J_0 never enters, whatever it holds (NaN included), for any chunking."""
    d = synth.random_system(2, 10, 3, seed=4)
    J2 = d["J"].copy()
    J2[:, 0] = np.nan
    for G in (1, 3, 10):
        x = so.chunked_solve(J2, d["r"], transpose, G)
        assert np.all(np.isfinite(x))
        np.testing.assert_allclose(x, oracle.seq_solve(d["J"], d["r"], transpose),
                                   rtol=1e-12, atol=1e-12)


def test_one_row_chunks_are_the_blocks():
    """G >= L: every chunk is one row, P_l = J_l (J_{l+1}^T transposed)."""
    d = synth.random_system(1, 6, 3, seed=8)
    for l in range(1, 6):
        P, q = so.chunk_maps(d["J"], d["r"], l, l + 1, False)
        np.testing.assert_array_equal(P[0, 0], np.asarray(d["J"][0, l], np.float64))
        np.testing.assert_array_equal(q[0, 0], np.asarray(d["r"][0, l], np.float64))
    for l in range(0, 5):
        P, _ = so.chunk_maps(d["J"], d["r"], l, l + 1, True)
        np.testing.assert_array_equal(P[0, 0], np.asarray(d["J"][0, l + 1], np.float64).T)
