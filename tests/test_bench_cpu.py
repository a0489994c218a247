"""Host logic of bench.py: rocprofv3 summaries and the traffic reader (CPU
only; synthetic counter files, no GPU)."""

import csv
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Grid_Size", "Workgroup_Size",
                                          "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, grid, value in rows:
            w.writerow({"Kernel_Name": name, "Grid_Size": grid * 256, "Workgroup_Size": 256,
                        "Counter_Name": counter, "Counter_Value": value})


def test_pmc_summary_scales_by_the_copy_probe(tmp_path):
    # the copy probe moves 4 GiB each way; the counters read half (fetch) and
    # all (write) of it, so fetch values are scaled x2 and write values x1
    copy_kib = (4 << 30) // 1024
    _write_counters(tmp_path / "f", "FETCH_SIZE", [
        ("void copy_probe_kernel(uint4 const*, uint4*, unsigned long)", 4096, copy_kib // 2),
        ("void stage_k::(anonymous namespace)::gemm_skinny_bf16<4, 1>(...)", 224, 1000.0),
        ("void stage_k::(anonymous namespace)::gemm_skinny_bf16<4, 1>(...)", 224, 1002.0)])
    _write_counters(tmp_path / "w", "WRITE_SIZE", [
        ("void copy_probe_kernel(uint4 const*, uint4*, unsigned long)", 4096, copy_kib),
        ("void stage_k::(anonymous namespace)::gemm_skinny_bf16<4, 1>(...)", 224, 10.0),
        ("void stage_k::(anonymous namespace)::gemm_skinny_bf16<4, 1>(...)", 224, 10.0)])
    text = bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), "t", ["c"], "alg")
    line = [l for l in text.splitlines() if l.startswith("TRAFFIC kernel=gemm_skinny")][0]
    kv = dict(t.split("=", 1) for t in line.split()[1:])
    assert float(kv["fetch_bytes"]) == pytest.approx(1001.0 * 1024 * 2)
    assert float(kv["write_bytes"]) == pytest.approx(10.0 * 1024)
    assert kv["grid"] == "224"


def test_traffic_is_null_when_the_kernel_sources_changed(tmp_path, monkeypatch):
    good = tmp_path / "profiles"
    good.mkdir()
    body = ("source_sha256: {sha}\n"
            "TRAFFIC kernel=gemm_skinny_bf16<4,1> grid=224 fetch_bytes=100 write_bytes=5\n")
    (good / "t.txt").write_text(body.format(sha=bench.kernel_source_sha()))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", "profiles/t.txt")
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "abc")
    (good / "t.txt").write_text(body.format(sha="abc"))
    val, _ = bench.committed_traffic(bench.GATE_UP_DECODE_KERNEL)
    assert val == 105
    (good / "t.txt").write_text(body.format(sha="def"))
    val, note = bench.committed_traffic(bench.GATE_UP_DECODE_KERNEL)
    assert val is None and "predate" in note


def test_gpus_above_one_exit_with_a_message():
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stderr


def test_oracle_step_timing_and_cpu_block():
    """The CPU-baseline helpers: one step of one layer of the oracle, timed,
    and its scaling to the stage's layers."""
    from paper_2606_18600_amd import synth
    sec, reps, spent = bench.oracle_layer_step(synth.TINY, [(20, 1), (0, 7), (33, 1)], 1,
                                               budget_s=0.2)
    assert sec > 0 and reps >= 1 and spent >= sec
    blk = bench.cpu_block(9, 20, 0.5, 3, 1.5, "a sample")
    assert blk["value"] == pytest.approx(9 / 10.0)
    assert blk["kind"] == "oracle" and blk["cores"] >= 1 and "x20 layers" in blk["sample"]
    info = bench.host_info()
    assert info["nproc"] >= 1 and "cpu_model" in info
