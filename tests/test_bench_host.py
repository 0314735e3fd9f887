"""Host-side checks of bench.py: the algorithmic byte counts behind every
GB/s figure, the committed HBM-traffic summary it reads for the roofline
line, and the one-GPU refusal of --gpus N > 1.  No GPU is touched."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_algorithmic_bytes_at_the_bench_shape():
    T, d = 32768, 4096
    # x bf16 read; one E4M3 code byte and 1/32 E8M0 byte written per element;
    # 4 bytes of rho per row
    assert bench.mxfp8_bytes(T, d) == T * d * 2 + T * d + T * d // 32 + 4 * T == 406_978_560
    # NVFP4: half a code byte and 1/16 scale byte per element
    assert bench.nvfp4_bytes(T, d) == T * d * 2 + T * d // 2 + T * d // 16 + 4 * T == 344_064_000
    # STE: x and grad_Z read, grad_x (bf16) written; rho per row; gamma in,
    # grad_gamma (float) out once
    assert bench.ste_bytes(T, d) == 6 * T * d + 4 * T + 2 * d + 4 * d
    # column cast of rho~ X: the same bytes as the row cast
    assert bench.cast_t_bytes(T, d) == bench.mxfp8_bytes(T, d)


def test_traffic_summary_is_well_formed():
    kv = {}
    with open(bench.TRAFFIC_FILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    for k in ("kernel_source_sha256_16", "fetch_kib_per_launch", "write_kib_per_launch",
              "fetch_calibration", "write_calibration", "hbm_bytes_per_launch"):
        assert k in kv, k
    fetch, write = float(kv["fetch_kib_per_launch"]), float(kv["write_kib_per_launch"])
    fc, wc = float(kv["fetch_calibration"]), float(kv["write_calibration"])
    # the copy kernel's counters scale to its known byte count: factors near 2 and 1
    assert 1.9 < fc < 2.1 and 0.95 < wc < 1.05
    hbm = float(kv["hbm_bytes_per_launch"])
    assert abs(hbm - (fetch * fc + write * wc) * 1024) < 2048
    # one read of x and one narrow write: within 1% of the algorithmic bytes
    alg = bench.mxfp8_bytes(32768, 4096)
    assert abs(hbm / alg - 1.0) < 0.01
    # the bench reports it only while the kernel source is the one profiled
    got = bench.measured_traffic()
    if kv["kernel_source_sha256_16"] == bench.source_hash():
        assert got == hbm
    else:
        assert got is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_reports_cores_model_and_every_config():
    import bench
    from paper_2603_13180_amd import synth
    w = synth.generate(bench.WORKLOAD, rows=range(512))
    r = bench.cpu_baseline(w.x, w.preset.d, budget_s=0.05, per_config_s=0.05, parallel_rows=256)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["unit"] == "GB/s" and r["value"] > 0
    assert r["nproc"] >= 1 and r["cores_available"] >= 1 and r["cpu_model"]
    assert set(r["per_config"]) == {name for name, _ in bench.CPU_CONFIGS}
    assert set(name for name, _ in bench.CPU_CONFIGS) == set(synth.PRESETS)
    for v in r["per_config"].values():
        assert v["rows"] > 0 and v["GB/s"] > 0
    assert r["row_parallel"]["threads"] >= 1 and r["row_parallel"]["rows"] == 256
