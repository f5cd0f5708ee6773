"""The command-line contract of bench.py: one JSON line with the fields the
benchmark record needs, a roofline object consistent with itself, the oracle's
CPU baseline, and a refusal (with a message, before any GPU work) of a
multi-GPU run."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT, capture_output=True,
                          text=True, timeout=timeout)


def test_bench_refuses_several_gpus():
    r = run_bench("--gpus", "2", timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr
    assert not any(line.startswith("{") for line in r.stdout.splitlines())


@pytest.mark.gpu
def test_bench_json_line():
    print("[bench contract] workload 2, 1 step, no warmup", flush=True)
    r = run_bench("--workload", "2", "--steps", "1", "--warmup", "0", "--cpu-seconds", "1", "--cpu-mode", "sample",
                  "--no-static", "--no-achievable", "--no-workloads")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [line for line in r.stdout.splitlines() if line.startswith("{")]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 1 and d["warmup"] == 0
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["vs_baseline"] is None and d["data"] == "synthetic" and d["dtype"] == "bf16"
    assert "workload" in d["config"]
    roof = d["roofline"]
    assert roof["bound"] in ("hbm", "mfma", "alu") and roof["unit"] in ("GB/s", "TFLOP/s")
    assert roof["peak"] > 0 and roof["achieved"] > 0
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) <= 1e-3 * roof["frac"] + 1e-4
    assert "traffic" in roof
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert cpu["unit"] == d["unit"] and cpu["sample"]


def test_algorithmic_bytes_follow_the_element_size():
    """Decode and prefill bytes per launch are counted at the workload's element size: the fp32 variant of
    a workload moves exactly twice the bytes of its bf16 variant for the same FLOPs."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2606_10537_amd import synth
    from paper_2606_10537_amd._lib import PD_BF16, PD_FP32
    w = synth.WORKLOADS[2]
    wb = synth.Workload(**{**w.__dict__, "dtype": PD_BF16})
    wf = synth.Workload(**{**w.__dict__, "dtype": PD_FP32})
    pfb, pbb, dfb, dbb = bench.algorithmic(wb, 1)
    pff, pbf, dff, dbf = bench.algorithmic(wf, 1)
    assert (pff, dff) == (pfb, dfb)
    assert pbf == 2 * pbb and dbf == 2 * dbb


def test_algorithmic_work_of_the_32k_workloads():
    """The work the roofline fractions are taken against, pinned to the figures derived by hand from the
    method's shapes (4 S_c^2 d FLOP per prefill (chunk, head); 4 L_d L_kv d per decode (sequence, head);
    decode bytes: K and V of the L_kv rows per KV head plus Q read and O written per query head)."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2606_10537_amd import synth
    # 32K, one layer, batch 8: S_c = 1 + 1024 + 128 + 512 = 1665, L_kv = 4 * 257 + 128 + 512 = 1668
    pf, pb, df, db = bench.algorithmic(synth.WORKLOADS[5], 1)
    assert pf == 4 * 1665 ** 2 * 128 * 8 * 32 * 32              # 11.63 TFLOP per layer
    assert abs(pf / (8 * 32 * 32) - 1.419e9) < 1e6              # 1.419 GFLOP per (chunk, head)
    assert df == 4 * 512 * 1668 * 128 * 8 * 32                  # 111.9 GFLOP per launch
    assert abs(df / (8 * 32) - 437.3e6) < 1e5                   # 437.3 MFLOP per (sequence, head)
    assert db == 2 * 128 * 8 * (2 * 1668 * 32 + 2 * 512 * 32)   # 285.7 MB per launch
    assert abs(db / (8 * 32) - 1.116e6) < 1e3                   # 1.116 MB per (sequence, head)
    assert 391 < df / db < 393                                  # arithmetic intensity, FLOP per byte
    # 32K batch 4 is the same per (sequence, head)
    pf4, _, df4, db4 = bench.algorithmic(synth.WORKLOADS[4], 1)
    assert (pf4, df4, db4) == (pf / 2, df / 2, db / 2)


def test_cpu_baseline_full_tiny_workload():
    """The oracle baseline of the tiny workload runs every unit of one job step on a process pool and
    reports the host it ran on."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2606_10537_amd import synth
    r = bench.cpu_baseline(synth.WORKLOADS[1], 1.0, "auto")
    assert r["mode"] == "full" and r["kind"] == "oracle" and r["value"] > 0
    assert 1 <= r["cores"] <= bench.CPU_SHARE and r["affinity_cpus"] >= 1 and r["os_cpu_count"] >= 1
    assert r["blas_threads_per_worker"] == 1 and r["numpy"] and r["sample"]
