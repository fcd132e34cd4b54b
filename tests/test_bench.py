"""bench.py contract: the one-GPU refusal, the algorithmic byte count, the traffic figure's gating on
the committed counter profile, and (GPU) the keys of the JSON line."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_attend_bytes_counts_kv_acc_and_io():
    # 7B shape, 32 sequences at 1536 cached slots + the appended row: per live slot K and V rows of
    # 4 KV heads x 128 dims in bf16 (4 x 128 x 2 B each) and the acc read + write (4 x 8 B); per
    # launch q read and out written (28 x 128 x 2 B each) and lse + suffix mass (28 x 8 B).
    lens = np.full(32, 1537)
    per_slot = 4 * 128 * 2 * 2 + 4 * 4 * 2
    per_seq_io = 28 * 128 * 2 * 2 + 28 * 4 * 2
    assert bench.attend_bytes(lens, 4, 28, 128, 2, 32) == 32 * 1537 * per_slot + 32 * per_seq_io
    # ragged lengths add up slot by slot
    lens = np.array([0, 1, 4096, 17])
    got = bench.attend_bytes(lens, 8, 32, 128, 2, 4)
    assert got == (4096 + 1 + 17) * (8 * 128 * 2 * 2 + 8 * 8) + 4 * (32 * 128 * 2 * 2 + 32 * 8)


def test_traffic_figure_follows_the_profile(tmp_path, monkeypatch):
    src = tmp_path / "lg_attend.hip"
    src.write_text("// kernel source\n")
    digest = hashlib.sha256(src.read_bytes()).hexdigest()
    prof = tmp_path / "traffic.md"
    prof.write_text("# counters\n\n- workload: 7B-shaped-b32\n- HBM bytes per lg_decode_attend "
                    "launch: 116144006\n- lg_attend.hip sha256: `%s`\n" % digest)
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(prof))
    monkeypatch.setattr(bench, "ATTEND_SOURCE", str(src))
    assert bench.measured_traffic("7B-shaped-b32") == 116144006.0
    assert bench.measured_traffic("ragged-b64") is None        # another workload
    src.write_text("// kernel source, edited\n")
    assert bench.measured_traffic("7B-shaped-b32") is None     # the kernel changed since
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "missing.md"))
    assert bench.measured_traffic("7B-shaped-b32") is None


@pytest.mark.gpu
def test_bench_json_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--config", "0",
                        "--steps", "3", "--warmup", "1", "--cpu-seconds", "1"],
                       capture_output=True, text=True, timeout=280, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    d = json.loads(lines[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline",
              "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["value"] > 0 and abs(d["value"] * d["ms_per_step"] - 1000.0) < 1e-6 * d["value"] * d["ms_per_step"] + 1e-3
    assert d["config"]["workload"] == "tiny-1layer-fp32" and d["dtype"] == "f32"
    roof = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in roof, k
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-12
    assert roof["traffic"] is None                      # counters were taken on another workload
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] == 1 and cpu["value"] > 0 and cpu["sample"]
    assert cpu["nproc"] >= 1 and cpu["layer_step_ms"] > 0
    assert abs(cpu["layer_step_ms"] * d["config"]["layers"] - cpu["sequence_step_ms"]) < 1e-9 * cpu["sequence_step_ms"] + 1e-12
    # tiny workload: 192 slots after the prefill reduction, budget 256, window 256: in 4 steps
    # nothing triggers and nothing overflows
    assert d["interventions"] == 0 and d["overflow_compactions"] == 0
    assert d["step_frac_of_copy"] > 0 and d["copy_gbps"] > 0
