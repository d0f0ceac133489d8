"""GPU parity of the row-chunked solve (pcr_solve_block_bidiag_chunked: the
single-GPU part of a solve whose rows are spread over G devices) against the
CPU oracle's substitution, on the same seeded float32 inputs.  Tolerance:
normwise relative error max_b ||x_b - ref_b||_inf / ||ref_b||_inf <= 1e-4."""
import sys

import numpy as np
import pytest

import oracle
from oracle import sharded_oracle
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


# widths of the MFMA strip kernel (32, 64, 128) and of the generic kernel
CASES = []
for w in (1, 4, 16, 17, 32, 64, 128):
    for L, B in ((1, 3), (2, 3), (7, 2), (64, 2), (100, 2), (257, 1)):
        if B * L * w * w > (1 << 22):
            continue
        for G in (1, 2, 3, 4, 8, L + 5):
            CASES.append((w, L, B, G))


@pytest.mark.parametrize("w,L,B,G", CASES)
@pytest.mark.parametrize("transpose", [0, 1])
def test_chunked_solve_matches_substitution(dev, w, L, B, G, transpose):
    _say(f"chunked w={w} L={L} B={B} G={G} transpose={transpose}")
    d = synth.random_system(B, L, w, seed=3000 + 11 * w + L + 97 * G, scale=0.9)
    x = h(deeppcr.pcr_solve_block_bidiag_chunked(g(d["J"], dev), g(d["r"], dev), G,
                                                 transpose=transpose))
    ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
    assert normwise_rel_err(x, ref) <= TOL
    # the oracle's own chunked solve reaches the same x (its pins tie it to
    # the substitution); checked here on the GPU's chunking
    np.testing.assert_allclose(sharded_oracle.chunked_solve(d["J"], d["r"], bool(transpose), G),
                               ref, rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("G", [2, 4, 8])
@pytest.mark.parametrize("transpose", [1, 0])
def test_chunked_solve_workload(dev, G, transpose):
    """The standalone-solve workload (B 64, L 1024, w 16, 0.9 Q diag(u) blocks)
    over 2, 4 and 8 chunks."""
    wl = synth.WORKLOADS["pcr_solve"]
    _say(f"chunked workload B={wl.B} L={wl.L} w={wl.w} G={G} transpose={transpose}")
    d = synth.workload_inputs(wl)
    x = h(deeppcr.pcr_solve_block_bidiag_chunked(g(d["J"], dev), g(d["r"], dev), G,
                                                 transpose=transpose))
    ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
    err = normwise_rel_err(x, ref)
    _say(f"  err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("w,L,B", [(128, 1024, 4), (64, 1024, 8), (32, 512, 16)])
@pytest.mark.parametrize("G", [2, 8])
@pytest.mark.parametrize("transpose", [1, 0])
def test_chunked_solve_wide_blocks(dev, w, L, B, G, transpose):
    _say(f"chunked w={w} L={L} B={B} G={G} transpose={transpose}")
    d = synth.random_system(B, L, w, seed=5000 + w + G, scale=0.9)
    x = h(deeppcr.pcr_solve_block_bidiag_chunked(g(d["J"], dev), g(d["r"], dev), G,
                                                 transpose=transpose))
    ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
    assert normwise_rel_err(x, ref) <= TOL


@pytest.mark.parametrize("w", [16, 64])
@pytest.mark.parametrize("transpose", [0, 1])
def test_chunked_solve_ignores_first_block_and_aliases(dev, w, transpose):
    """J[:, 0] is never read (NaN there changes nothing); x may alias r; the
    result is the same on a second call with the same workspace."""
    B, L, G = 2, 45, 4
    _say(f"chunked NaN J0 / alias w={w} transpose={transpose}")
    d = synth.random_system(B, L, w, seed=77 + w, scale=0.9)
    J = d["J"].copy()
    J[:, 0] = np.nan
    Jd, rd = g(J, dev), g(d["r"], dev)
    n = deeppcr.lib().deeppcr_chunked_workspace_bytes(B, L, w, G)
    ws = torch.empty(n, dtype=torch.uint8, device=dev)
    x1 = h(deeppcr.pcr_solve_block_bidiag_chunked(Jd, rd, G, transpose=transpose, workspace=ws))
    assert np.all(np.isfinite(x1))
    ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
    assert normwise_rel_err(x1, ref) <= TOL
    x2 = h(deeppcr.pcr_solve_block_bidiag_chunked(Jd, rd, G, x=rd, transpose=transpose,
                                                  workspace=ws))
    np.testing.assert_array_equal(x1, x2)
