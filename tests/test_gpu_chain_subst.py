"""GPU parity of the last levels' substitution pass (the chains left after
the first PCR levels, solved row by row) across the shapes where the number
of substituted levels changes (3 to 6), with odd depths (chains of unequal
length, the last shorter than the others) and short chains, for the
standalone solve (both orientations), the Newton forward (the pass adds the
solution to the iterate and reduces the stopping measures) and the backward.
Against the CPU oracle on the same seeded float32 inputs; normwise relative
error <= 1e-4."""
import sys

import numpy as np
import pytest

import oracle
from paper_2309_16318_amd import deeppcr, synth
from tests._util import normwise_rel_err, per_layer_rel_err

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


# (w, B, L): 3, 4, 5 and 6 substituted levels at w = 16, 32, 64, 128, odd L
SHAPES = [(16, 64, 1024), (16, 64, 17), (16, 64, 33), (16, 32, 65), (16, 16, 129),
          (16, 8, 300), (16, 4, 1000), (16, 256, 64),
          (32, 64, 33), (32, 64, 65), (32, 64, 127), (32, 64, 129), (32, 64, 300),
          (32, 16, 65), (32, 16, 257), (32, 16, 1000),
          (64, 32, 65), (64, 32, 129), (64, 32, 300), (64, 8, 257), (64, 8, 1000),
          (128, 16, 129), (128, 16, 200), (128, 4, 513)]


@pytest.mark.parametrize("w,B,L", SHAPES)
@pytest.mark.parametrize("transpose", [0, 1])
def test_substitution_pass_solve(dev, w, B, L, transpose):
    _say(f"substitution solve w={w} B={B} L={L} transpose={transpose}")
    d = synth.random_system(B, L, w, seed=11000 + w + L + B, scale=0.9)
    x = h(deeppcr.pcr_solve_block_bidiag(g(d["J"], dev), g(d["r"], dev), transpose=transpose))
    assert normwise_rel_err(x, oracle.seq_solve(d["J"], d["r"], bool(transpose))) <= TOL


@pytest.mark.parametrize("w,B,L", SHAPES)
def test_substitution_pass_forward_and_backward(dev, w, B, L):
    """Residual tanh layers (adjoints stay O(1) through depth, so every layer
    is judged), forward from the paper's start and backward on its states."""
    _say(f"substitution fwd/bwd w={w} B={B} L={L}")
    layer, alpha = 1, 0.1
    d = synth.mlp_inputs(B, L, w, seed=12000 + w + L + B)
    t = {k: g(v, dev) for k, v in d.items()}
    res = deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], layer=layer, alpha=alpha,
                                      tol=1e-5, max_iter=20)
    assert res.status == deeppcr.OK
    Zref = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"])
    assert normwise_rel_err(h(res.Z), Zref) <= TOL
    _, k_ref, ok, _ = oracle.newton_forward(layer, alpha, d["W"], d["bias"], d["z0"], 1e-5, 20)
    assert ok and abs(res.iters - k_ref) <= 1
    Z32 = Zref.astype(np.float32)
    lam, dz0, dW, db = deeppcr.deeppcr_mlp_backward(t["W"], t["bias"], t["z0"], g(Z32, dev),
                                                    t["G"], layer=layer, alpha=alpha)
    rl, rz, rW, rb = oracle.seq_backward(layer, alpha, d["W"], d["bias"], d["z0"], Z32, d["G"])
    lam, dz0 = h(lam), h(dz0)
    assert normwise_rel_err(np.concatenate([dz0[:, None], lam], 1),
                            np.concatenate([rz[:, None], rl], 1)) <= TOL
    assert per_layer_rel_err(lam, rl, layer_axis=1)[0] <= TOL
    assert normwise_rel_err(h(dW), rW, axes="all") <= TOL
    assert normwise_rel_err(h(db), rb, axes="all") <= TOL
