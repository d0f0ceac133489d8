"""The no-allocation solve (pcr_solve_block_bidiag_noalloc, through the C
ABI) against the workspace entry point it shares its kernels with, and
against the oracle: two calls in a row on one GPU, the second smaller, in
both orientations, plus a problem that fills the fixed scratch array."""
import sys

import numpy as np
import pytest

import oracle
from paper_2309_16318_amd import deeppcr, synth
from tests._util import normwise_rel_err

pytestmark = pytest.mark.gpu
TOL = 1e-4
torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def g(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def h(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _both(d, dev, transpose):
    J, r = g(d["J"], dev), g(d["r"], dev)
    want = h(deeppcr.pcr_solve_block_bidiag(J, r, transpose=transpose))
    x = torch.full_like(r, float("nan"))
    got = h(deeppcr.pcr_solve_block_bidiag_noalloc(J, r, x, transpose=transpose))
    return got, want


@pytest.mark.parametrize("transpose", [0, 1])
def test_noalloc_matches_workspace_entry_point_twice(dev, transpose):
    cap = deeppcr.lib().deeppcr_noalloc_scratch_bytes()
    for B, L, w in ((6, 1000, 32), (3, 257, 16)):
        assert deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w) <= cap
        _say(f"noalloc B={B} L={L} w={w} transpose={transpose}")
        d = synth.random_system(B, L, w, seed=4000 + B + L + w + transpose, scale=0.9)
        got, want = _both(d, dev, transpose)
        assert np.array_equal(got, want)
        ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
        assert normwise_rel_err(got, ref) <= TOL


def test_noalloc_largest_problem_that_fits(dev):
    B, L, w = 1, 480, 128
    cap = deeppcr.lib().deeppcr_noalloc_scratch_bytes()
    assert deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w) <= cap
    assert deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L + 32, w) > cap
    _say(f"noalloc largest B={B} L={L} w={w}")
    d = synth.random_system(B, L, w, seed=4100, scale=0.9)
    got, want = _both(d, dev, 1)
    assert np.array_equal(got, want)
    assert normwise_rel_err(got, oracle.seq_solve(d["J"], d["r"], True)) <= TOL
    # one row more than fits: rejected, the output left untouched
    d = synth.random_system(B, L + 32, w, seed=4101, scale=0.9)
    J, r = g(d["J"], dev), g(d["r"], dev)
    x = torch.zeros_like(r)
    with pytest.raises(deeppcr.DeepPCRError, match="workspace"):
        deeppcr.pcr_solve_block_bidiag_noalloc(J, r, x)
    assert float(x.abs().max()) == 0.0
