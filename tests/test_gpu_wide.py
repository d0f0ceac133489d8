"""GPU parity at widths 129..1024 (the tiled block-product kernels): the
standalone PCR solve, the Newton + PCR forward pass, the transposed-PCR
backward pass and the sequential passes, against the CPU oracle on the same
seeded float32 inputs.  Tolerance: normwise relative error 1e-4 per system
(dW, db over the whole tensor and per layer)."""
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


# 129, 130: scalar loads (w % 4 != 0) and one partial 128-tile; 200: partial
# tiles with vector loads; 256, 384, 512, 1024: whole tiles
PCR_CASES = [(129, 5, 2), (130, 17, 1), (200, 9, 2), (256, 1, 2), (256, 2, 2), (256, 3, 1),
             (256, 64, 2), (256, 130, 1), (384, 33, 1), (512, 20, 1), (1024, 9, 1),
             (1024, 33, 1)]


@pytest.mark.parametrize("w,L,B", PCR_CASES)
@pytest.mark.parametrize("transpose", [0, 1])
def test_wide_pcr_solve(dev, w, L, B, transpose):
    _say(f"wide pcr w={w} L={L} B={B} transpose={transpose}")
    d = synth.random_system(B, L, w, seed=9000 + w + L, scale=0.5)
    x = h(deeppcr.pcr_solve_block_bidiag(g(d["J"], dev), g(d["r"], dev), transpose=transpose))
    ref = oracle.seq_solve(d["J"], d["r"], bool(transpose))
    err = normwise_rel_err(x, ref)
    _say(f"  err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("w,L", [(256, 64), (1024, 16)])
def test_wide_pcr_solve_noalloc_and_nan_first_block(dev, w, L):
    """J[:, 0] is never read; the no-allocation entry point gives the
    workspace entry point's result bit for bit where the problem fits."""
    d = synth.random_system(1, L, w, seed=77, scale=0.5)
    J = d["J"].copy()
    J[:, 0] = np.nan
    Jd, rd = g(J, dev), g(d["r"], dev)
    for tr in (0, 1):
        x = h(deeppcr.pcr_solve_block_bidiag(Jd, rd, transpose=tr))
        assert np.all(np.isfinite(x))
        assert normwise_rel_err(x, oracle.seq_solve(d["J"], d["r"], bool(tr))) <= TOL
        if deeppcr.workspace_bytes(deeppcr.OP_PCR, 1, L, w) <= deeppcr.lib().deeppcr_noalloc_scratch_bytes():
            x2 = torch.empty_like(rd)
            deeppcr.pcr_solve_block_bidiag_noalloc(Jd, rd, x2, transpose=tr)
            np.testing.assert_array_equal(h(x2), x)


FWD_CASES = [(256, 24, 2, 0, 1.0), (256, 24, 2, 1, 0.1), (130, 20, 2, 0, 1.0),
             (512, 16, 1, 2, 1.0), (512, 16, 1, 5, 0.1), (1024, 12, 1, 0, 1.0),
             (1024, 12, 1, 1, 0.1)]


@pytest.mark.parametrize("w,L,B,layer,alpha", FWD_CASES)
def test_wide_forward(dev, w, L, B, layer, alpha):
    _say(f"wide forward w={w} L={L} B={B} layer={layer}")
    d = synth.mlp_inputs(B, L, w, seed=9100 + w + L + layer)
    res = deeppcr.deeppcr_mlp_forward(g(d["W"], dev), g(d["bias"], dev), g(d["z0"], dev),
                                      layer=layer, alpha=alpha, tol=1e-5, max_iter=20)
    assert res.status == deeppcr.OK
    ref = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"])
    err = normwise_rel_err(h(res.Z), ref)
    _, k_ref, ok, _ = oracle.newton_forward(layer, alpha, d["W"], d["bias"], d["z0"], 1e-5, 20)
    _say(f"  err {err:.2e} iters {res.iters} oracle {k_ref}")
    assert err <= TOL
    assert ok and abs(res.iters - k_ref) <= 1


@pytest.mark.parametrize("w,L,B,layer,alpha", [(256, 24, 2, 0, 1.0), (256, 20, 3, 1, 0.1),
                                               (130, 17, 2, 3, 0.1), (512, 16, 2, 0, 1.0),
                                               (1024, 10, 2, 1, 0.1), (1024, 10, 1, 4, 1.0)])
def test_wide_backward(dev, w, L, B, layer, alpha):
    _say(f"wide backward w={w} L={L} B={B} layer={layer}")
    d = synth.mlp_inputs(B, L, w, seed=9200 + w + L + layer)
    Z32 = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"]).astype(np.float32)
    lam, dz0, dW, db = deeppcr.deeppcr_mlp_backward(g(d["W"], dev), g(d["bias"], dev),
                                                    g(d["z0"], dev), g(Z32, dev), g(d["G"], dev),
                                                    layer=layer, alpha=alpha)
    rl, rz, rW, rb = oracle.seq_backward(layer, alpha, d["W"], d["bias"], d["z0"], Z32, d["G"])
    lam, dz0, dW, db = h(lam), h(dz0), h(dW), h(db)
    errs = (normwise_rel_err(np.concatenate([dz0[:, None], lam], 1),
                             np.concatenate([rz[:, None], rl], 1)),
            normwise_rel_err(dW, rW, axes="all"), normwise_rel_err(db, rb, axes="all"),
            per_layer_rel_err(lam, rl, layer_axis=1)[0],
            per_layer_rel_err(dW, rW, layer_axis=0)[0], per_layer_rel_err(db, rb, layer_axis=0)[0])
    _say(f"  errs {['%.2e' % e for e in errs]}")
    assert max(errs) <= TOL


@pytest.mark.parametrize("w,L,B,layer,alpha", [(256, 9, 3, 0, 1.0), (130, 7, 9, 1, 0.1),
                                               (1024, 6, 2, 3, 0.1)])
def test_wide_sequential_passes(dev, w, L, B, layer, alpha):
    """The sequential baseline at wide widths (one launch per layer)."""
    _say(f"wide sequential w={w} L={L} B={B} layer={layer}")
    d = synth.mlp_inputs(B, L, w, seed=9300 + w + L)
    t = {k: g(v, dev) for k, v in d.items()}
    ref = oracle.seq_forward(layer, alpha, d["W"], d["bias"], d["z0"])
    for per_layer in (False, True):
        Z = deeppcr.deeppcr_seq_forward(t["W"], t["bias"], t["z0"], layer=layer, alpha=alpha,
                                        launch_per_layer=per_layer)
        assert normwise_rel_err(h(Z), ref) <= TOL
    Z32 = ref.astype(np.float32)
    rl, rz, _, _ = oracle.seq_backward(layer, alpha, d["W"], d["bias"], d["z0"], Z32, d["G"])
    lam, dz0 = deeppcr.deeppcr_seq_backward(t["W"], t["bias"], t["z0"], g(Z32, dev), t["G"],
                                            layer=layer, alpha=alpha)
    assert normwise_rel_err(np.concatenate([h(dz0)[:, None], h(lam)], 1),
                            np.concatenate([rz[:, None], rl], 1)) <= TOL


def test_wide_newton_step_generic(dev):
    """deeppcr_newton_step (caller-evaluated steps) at w = 256: one Newton
    iteration against the oracle's Eq. 3 solve."""
    B, L, w = 2, 20, 256
    d = synth.random_system(B, L, w, seed=5, scale=0.5)
    F = np.random.default_rng(6).standard_normal((B, L, w)).astype(np.float32)
    Z0 = np.random.default_rng(7).standard_normal((B, L, w)).astype(np.float32)
    Z = g(Z0, dev)
    deeppcr.deeppcr_newton_step(g(d["J"], dev), g(F, dev), Z, tol=0.0)
    ref = Z0.astype(np.float64) + oracle.seq_solve(d["J"], F.astype(np.float64) - Z0, False)
    assert normwise_rel_err(h(Z), ref) <= TOL


def test_wide_forward_iterations_past_the_watch(dev):
    """Newton iterations long enough (w = 1024, L = 96, B = 1: about ten
    milliseconds each) that the host's 5 ms watch of the measures word runs
    out and the read-back falls back to waiting for the stream: the same
    solution and iteration count as the oracle's Newton run."""
    import time
    B, L, w, layer = 1, 96, 1024, 1
    d = synth.mlp_inputs(B, L, w, seed=9400)
    t = {k: g(v, dev) for k, v in d.items()}
    deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], layer=layer, alpha=0.1, tol=0.0,
                                max_iter=1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], layer=layer, alpha=0.1,
                                      tol=1e-5, max_iter=20)
    ms = (time.perf_counter() - t0) * 1e3
    assert res.status == deeppcr.OK
    ref = oracle.seq_forward(layer, 0.1, d["W"], d["bias"], d["z0"])
    err = normwise_rel_err(h(res.Z), ref)
    _, k_ref, ok, _ = oracle.newton_forward(layer, 0.1, d["W"], d["bias"], d["z0"], 1e-5, 20)
    _say(f"  {res.iters} iterations in {ms:.1f} ms ({ms / max(res.iters, 1):.1f} ms each), "
         f"err {err:.2e}, oracle {k_ref}")
    assert err <= TOL
    assert ok and abs(res.iters - k_ref) <= 1
