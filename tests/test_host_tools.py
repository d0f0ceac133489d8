"""Host-side measurement logic (no GPU): the HBM counter summary, the
staleness digest of the kernel source, and bench.py's roofline placement and
single-GPU guard."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2309_16318_amd import pmc_traffic  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _counter_dir(tmp_path, name, rows):
    d = tmp_path / name / "host" / "pid"
    d.mkdir(parents=True)
    with open(d / "run_counter_collection.csv", "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=FIELDS)
        wr.writeheader()
        for r in rows:
            wr.writerow(dict(zip(FIELDS, r)))
    return str(tmp_path / name)


def test_digest_ignores_comments_and_layout():
    a = "int f(int x) {\n  return x + 1;  // one more\n}\n"
    b = "// leading note\nint f(int x)\n{\n\treturn x+1;\n}\n"
    c = "int f(int x) {\n  return x + 2;\n}\n"
    assert pmc_traffic.code_digest(a) == pmc_traffic.code_digest(b)
    assert pmc_traffic.code_digest(a) != pmc_traffic.code_digest(c)


def test_digest_covers_every_kernel_source():
    for fn in pmc_traffic.KERNEL_SOURCES:
        assert os.path.exists(fn), fn
    assert len(pmc_traffic.kernel_source_sha256()) == 64


def test_per_kernel_counts_each_dispatch_once(tmp_path):
    # rocprofv3 can list a dispatch once per agent / sample; it must count once
    d = _counter_dir(tmp_path, "f", [
        (1, "void deeppcr::(anonymous namespace)::pcr_level2_tile<64, false, false>(a, b)",
         "FETCH_SIZE", 100.0),
        (1, "void deeppcr::(anonymous namespace)::pcr_level2_tile<64, false, false>(a, b)",
         "FETCH_SIZE", 100.0),
        (2, "void deeppcr::(anonymous namespace)::pcr_level2_tile<64, false, false>(a, b)",
         "FETCH_SIZE", 300.0),
        (3, "copy_kernel(x)", "WRITE_SIZE", 7.0),
    ])
    k = pmc_traffic.per_kernel(d, "FETCH_SIZE")
    assert k == {"pcr_level2_tile<64, false, false>": [2, 400.0]}


def test_summary_scales_by_the_copy_and_leaves_out_the_tail(tmp_path, monkeypatch):
    # copy of 1 MiB: FETCH_SIZE reads 512 units (2048 B per unit), WRITE_SIZE
    # 1024 units (1024 B per unit)
    cf = _counter_dir(tmp_path, "cf", [(1, "copyBuffer", "FETCH_SIZE", 512.0)])
    cw = _counter_dir(tmp_path, "cw", [(1, "copyBuffer", "WRITE_SIZE", 1024.0)])
    lvl, tail = "pcr_level2_tile<128, false, false>", "pcr_level_tail<128, 6, true>"
    f = _counter_dir(tmp_path, "f", [(1, lvl, "FETCH_SIZE", 10.0), (2, lvl, "FETCH_SIZE", 30.0),
                                     (3, tail, "FETCH_SIZE", 1000.0),
                                     (4, "other_kernel", "FETCH_SIZE", 5000.0)])
    w = _counter_dir(tmp_path, "w", [(1, lvl, "WRITE_SIZE", 4.0), (2, lvl, "WRITE_SIZE", 8.0),
                                     (3, tail, "WRITE_SIZE", 2.0),
                                     (4, "other_kernel", "WRITE_SIZE", 5000.0)])
    out = tmp_path / "t.json"
    monkeypatch.setattr(sys, "argv", [
        "pmc_traffic", "--workload", "x", "--fetch", f, "--write", w, "--copy-fetch", cf,
        "--copy-write", cw, "--copy-bytes", str(1 << 20), "--out", str(out)])
    pmc_traffic.main()
    t = json.loads(out.read_text())
    assert t["fetch_bytes_per_counter_unit"] == pytest.approx(2048.0)
    assert t["write_bytes_per_counter_unit"] == pytest.approx(1024.0)
    assert t["pcr_level_launches"] == 2
    assert t["read_bytes_per_launch"] == pytest.approx(20.0 * 2048)
    assert t["write_bytes_per_launch"] == pytest.approx(6.0 * 1024)
    assert t["traffic_bytes_per_launch"] == pytest.approx(20.0 * 2048 + 6.0 * 1024)
    assert set(t["by_kernel"]) == {lvl, tail}
    assert t["by_kernel"][tail]["read_bytes_per_launch"] == pytest.approx(1000.0 * 2048)
    assert t["kernel_source_sha256"] == pmc_traffic.kernel_source_sha256()


def test_bench_roofline_placement():
    import bench

    # 1 ms of 15.73 GFLOP and 0.1 GB: intensity 157 flop/B, MFMA-bound at 0.1
    r = bench.roofline({"flops": 15.73e9, "bytes": 1e8, "ms": 1.0}, 32)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["achieved"] == pytest.approx(15.73) and r["frac"] == pytest.approx(0.1)
    # 1 ms of 4 GB and 4 GFLOP: 1 flop/B, HBM-bound at 4000 GB/s = 0.5
    r = bench.roofline({"flops": 4e9, "bytes": 4e9, "ms": 1.0}, 16)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["achieved"] == pytest.approx(4000.0) and r["frac"] == pytest.approx(0.5)
    # w >= 64 is placed against the MFMA peak whatever the intensity
    assert bench.roofline({"flops": 4e9, "bytes": 4e9, "ms": 1.0}, 64)["bound"] == "mfma"


def test_bench_measured_traffic_only_for_the_current_kernels(tmp_path, monkeypatch):
    import bench

    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w") is None
    rec = {"kernel_source_sha256": pmc_traffic.kernel_source_sha256(),
           "traffic_bytes_per_launch": 1234.4}
    (prof / "pcr_level_hbm_traffic_w.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("w") == 1234
    rec["kernel_source_sha256"] = "0" * 64
    (prof / "pcr_level_hbm_traffic_w.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("w") is None


def test_bench_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_calibration_scales_by_the_copy_and_checks_the_add(tmp_path):
    # 1 MiB probe: the copy reads 1 MiB in 512 FETCH units (2048 B per unit)
    # and writes it in 1024 WRITE units; the add reads 0.5 MiB and writes
    # 0.25 MiB, here measured 1% high on reads
    cp = "__amd_rocclr_copyBuffer"
    add = "void at::native::vectorized_elementwise_kernel<4, at::native::AddFunctor<float>>"
    f = _counter_dir(tmp_path, "f", [(1, cp, "FETCH_SIZE", 512.0),
                                     (2, add + "(x)", "FETCH_SIZE", 256.0 * 1.01)])
    w = _counter_dir(tmp_path, "w", [(1, cp, "WRITE_SIZE", 1024.0),
                                     (2, add + "(x)", "WRITE_SIZE", 256.0)])
    out = pmc_traffic.calibrate(["--fetch", f, "--write", w, "--mib", "1",
                                 "--out", str(tmp_path / "c.json")])
    assert out["fetch_bytes_per_counter_unit"] == pytest.approx(2048.0)
    assert out["write_bytes_per_counter_unit"] == pytest.approx(1024.0)
    assert out["add_read_ratio"] == pytest.approx(1.01)
    assert out["add_write_ratio"] == pytest.approx(1.0)
    assert json.loads((tmp_path / "c.json").read_text())["add_kernel"].startswith("at::native")


def test_mfma_summary_weights_by_dispatch_and_splits_the_tail(tmp_path):
    pair, tail = "pcr_level2_tile<128, false, false>", "pcr_level_tail<128, 6, true>"
    rows = [(1, pair, "MfmaUtil", 70.0), (1, pair, "SQ_BUSY_CYCLES", 10.0),
            (2, pair, "MfmaUtil", 74.0), (2, pair, "SQ_BUSY_CYCLES", 30.0),
            (3, "pcr_level2_tile_layer<128>", "MfmaUtil", 60.0),
            (4, tail, "MfmaUtil", 50.0), (5, "other", "MfmaUtil", 1.0)]
    d = _counter_dir(tmp_path, "m", rows)
    out = pmc_traffic.mfma(["--workload", "x", "--dir", d, "--out", str(tmp_path / "m.json")])
    assert out["by_kernel"][pair]["launches"] == 2
    assert out["by_kernel"][pair]["MfmaUtil"] == pytest.approx(72.0)
    assert out["by_kernel"][pair]["SQ_BUSY_CYCLES"] == pytest.approx(20.0)
    assert out["pcr_level_mfma_util_pct"] == pytest.approx((70 + 74 + 60) / 3)
    assert out["pcr_tail_mfma_util_pct"] == pytest.approx(50.0)
    assert "other" not in out["by_kernel"]
    assert out["kernel_source_sha256"] == pmc_traffic.kernel_source_sha256()


def test_denoising_step_jacobians_match_autograd():
    """The sampler example's step Jacobians (one GEMM of the activation slopes
    against the denoiser's rank-one products, the 1/sqrt(alpha) diagonal added
    in place) equal autograd's Jacobian of its step function, on the CPU."""
    torch = pytest.importorskip("torch")
    from paper_2309_16318_amd import generic, synth
    B, L, w, h = 2, 6, 4, 8
    d = synth.diffusion_inputs(B, L, w, h, seed=3)
    p = {k: torch.from_numpy(d[k]).double() for k in ("W1", "b1", "W2", "b2", "temb")}
    eps = torch.from_numpy(d["eps"]).double()
    step_fn, jac_fn = generic.denoising_steps(p, eps)
    Zprev = torch.randn(B, L, w, dtype=torch.float64, generator=torch.Generator().manual_seed(4))
    J = jac_fn(Zprev)
    assert J.shape == (B, L, w, w)
    full = torch.autograd.functional.jacobian(step_fn, Zprev)   # [B, L, w, B, L, w]
    for b in range(B):
        for l in range(L):
            torch.testing.assert_close(J[b, l], full[b, l, :, b, l, :], rtol=1e-6, atol=1e-6)
