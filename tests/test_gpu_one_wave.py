"""GPU parity of the one-wave Newton + PCR solver (iterates of at most 64
entries, w in {1, 2, 4, 8}: the whole solve in one wave's registers, rows
exchanged by lane shuffles) against the CPU oracle, for every layer kind,
both stopping rules, a fixed iteration count, a warm start and the status
reports; beside it the workgroup solver one entry above (65 entries) on the
same kind of inputs.  Tolerance as elsewhere: normwise relative error
<= 1e-4; Newton counts within one of the oracle's."""
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


def _forward(d, dev, layer, alpha, tol=1e-5, max_iter=20, Z_init=None):
    return deeppcr.deeppcr_mlp_forward(g(d["W"], dev), g(d["bias"], dev), g(d["z0"], dev),
                                       layer=layer, alpha=alpha, tol=tol, max_iter=max_iter,
                                       Z_init=Z_init)


def _forward_res(d, dev, layer, alpha, atol=1e-4, rtol=1e-4, max_iter=15, Z_init=None):
    return deeppcr.deeppcr_mlp_forward_residual(g(d["W"], dev), g(d["bias"], dev),
                                                g(d["z0"], dev), layer=layer, alpha=alpha,
                                                atol=atol, rtol=rtol, max_iter=max_iter,
                                                Z_init=Z_init)


ALL_KINDS = [(0, 1.0), (1, 0.1), (2, 1.0), (3, 0.1), (4, 1.0), (5, 0.1)]
# (w, L, B): B L w = 64 at every width, partial waves, L = 1 and 2, and one
# entry past a wave (65: the workgroup solver)
SHAPES = [(1, 64, 1), (1, 7, 3), (2, 32, 1), (2, 5, 6), (4, 16, 1), (4, 3, 5), (4, 1, 16),
          (8, 8, 1), (8, 2, 4), (8, 1, 8), (1, 65, 1), (5, 13, 1)]


@pytest.mark.parametrize("w,L,B", SHAPES)
@pytest.mark.parametrize("layer,alpha", ALL_KINDS)
def test_one_wave_forward(dev, w, L, B, layer, alpha):
    _say(f"one-wave forward w={w} L={L} B={B} layer={layer}")
    d = synth.mlp_inputs(B, L, w, seed=2100 + 7 * w + L + 13 * B + layer)
    res = _forward(d, dev, layer, alpha)
    assert res.status == deeppcr.OK
    ref = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"])
    assert normwise_rel_err(h(res.Z), ref) <= TOL
    _, k_ref, ok, _ = oracle.newton_forward(layer, alpha, d["W"], d["bias"], d["z0"], 1e-5, 20)
    assert ok and abs(res.iters - k_ref) <= 1


@pytest.mark.parametrize("w,L,B", SHAPES)
@pytest.mark.parametrize("layer,alpha", [(0, 1.0), (3, 0.1), (4, 1.0)])
def test_one_wave_residual_rule(dev, w, L, B, layer, alpha):
    d = synth.mlp_inputs(B, L, w, seed=2300 + 7 * w + L + 13 * B + layer)
    res = _forward_res(d, dev, layer, alpha)
    assert res.status == deeppcr.OK
    _, k_ref, ok, _ = oracle.newton_forward_residual(layer, alpha, d["W"], d["bias"], d["z0"],
                                                     1e-4, 1e-4, 15)
    assert ok and abs(res.iters - k_ref) <= 1
    if res.iters == 0:
        Zk = oracle.initial_guess(layer, alpha, *(d[k].astype(np.float64)
                                                  for k in ("W", "bias", "z0")))
    else:
        Zk, _, _, _ = oracle.newton_forward(layer, alpha, d["W"], d["bias"], d["z0"], 0.0,
                                            res.iters)
    assert normwise_rel_err(h(res.Z), Zk) <= TOL
    r_own = oracle.residual_norm(layer, alpha, d["W"], d["bias"], d["z0"], h(res.Z))
    assert abs(res.residual - r_own) <= 1e-5 + 1e-3 * r_own


@pytest.mark.parametrize("w,L,B", [(1, 64, 1), (4, 16, 1), (8, 8, 1), (2, 5, 6)])
def test_one_wave_fixed_count_warm_start_and_status(dev, w, L, B):
    """tol = 0: exactly max_iter solves, the first k rows exact after k from a
    zero start; a start at the root converges in one solve; ENOCONV after
    max_iter; ENONFINITE from a NaN bias, after one solve."""
    d = dict(synth.mlp_inputs(B, L, w, seed=2500 + w + L))
    ref = oracle.seq_forward(0, 1.0, d["W"], d["bias"], d["z0"])
    for k in (1, 2, min(L, 5)):
        res = _forward(d, dev, 0, 1.0, tol=0.0, max_iter=k,
                       Z_init=torch.zeros((B, L, w), device=dev))
        assert res.status == deeppcr.OK and res.iters == k
        assert normwise_rel_err(h(res.Z)[:, :k], ref[:, :k]) <= 1e-6
    res = _forward(d, dev, 0, 1.0, Z_init=g(ref, dev))
    assert res.status == deeppcr.OK and res.iters == 1
    assert normwise_rel_err(h(res.Z), ref) <= TOL
    if L >= 3:
        res = _forward(d, dev, 0, 1.0, tol=1e-7, max_iter=1)
        assert res.status == deeppcr.ENOCONV and res.iters == 1
    d["bias"] = d["bias"].copy()
    d["bias"][L // 2, 0] = np.nan
    res = _forward(d, dev, 0, 1.0)
    assert res.status == deeppcr.ENONFINITE and res.iters == 1
    res = _forward_res(d, dev, 0, 1.0)
    assert res.status == deeppcr.ENONFINITE


def test_one_wave_matches_workgroup_solver_on_the_workload(dev):
    """The tiny workload (B 1, L 16, w 4) through the one-wave solver equals
    the oracle's Newton iterate after the same number of solves."""
    wl = synth.WORKLOADS["tiny_fwd"]
    d = synth.workload_inputs(wl)
    res = _forward(d, dev, wl.layer, wl.alpha, wl.tol, wl.max_iter)
    assert res.status == deeppcr.OK
    Zk, _, _, _ = oracle.newton_forward(wl.layer, wl.alpha, d["W"], d["bias"], d["z0"], 0.0,
                                        res.iters)
    assert normwise_rel_err(h(res.Z), Zk) <= 1e-6
