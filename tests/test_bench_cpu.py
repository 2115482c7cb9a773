"""Host logic of bench.py (CPU): the one-GPU refusal, the kernel-source hash
that keys the traffic record, the traffic record built from counter files, and
the CPU oracle baseline's phases."""
import csv
import json
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_code_only_drops_comments_keeps_strings():
    src = 'int a = 1; // note\n/* block\n comment */ const char* s = "x // y /* z */";\n'
    out = bench._code_only(src)
    assert "note" not in out and "block" not in out
    assert '"x // y /* z */"' in out and out.startswith("int a = 1;")


def test_source_hash_ignores_comment_edits_only(tmp_path, monkeypatch):
    src = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, src)
    monkeypatch.setattr(bench, "CSRC", str(src))
    h0 = bench.source_hash()
    f = src / "sparse_fwd.hip"
    text = f.read_text()
    f.write_text("// an added comment line\n" + text.replace("\n", "\n  ", 3))
    assert bench.source_hash() == h0
    f.write_text(text.replace("kSumBound = 1048576.0f", "kSumBound = 524288.0f"))
    assert bench.source_hash() != h0
    f.write_text(text)
    # the fp32 path is not among the recorded kernels
    g = src / "f32_path.hip"
    g.write_text(g.read_text().replace("constexpr int CK = 32;", "constexpr int CK = 16;"))
    assert bench.source_hash() == h0


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        w.writeheader()
        for d, name, val in rows:
            # two counter instances per dispatch: the record sums them
            w.writerow(dict(Dispatch_Id=d, Kernel_Name=name, Counter_Name=counter,
                            Counter_Value=val / 2))
            w.writerow(dict(Dispatch_Id=d, Kernel_Name=name, Counter_Name=counter,
                            Counter_Value=val / 2))


def test_record_traffic_scales_by_the_reference_copy(tmp_path, monkeypatch):
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    sparse = "_ZN4losa12_GLOBAL__N_122sparse_fwd_bf16_kernelILi128ELi128ELi128ELb0EEEvv"
    dense = "_ZN4losa12_GLOBAL__N_122sparse_fwd_bf16_kernelILi128ELi128ELi128ELb1EEEvv"
    mib = 256
    # the copy reads 256 MiB: FETCH_SIZE counts half of it, WRITE_SIZE all of it (KiB)
    fetch = [(1, bench.COPY_KERNEL, mib * 1024 / 2), (2, sparse, 1000.0), (3, sparse, 3000.0),
             (4, dense, 500.0)]
    write = [(1, bench.COPY_KERNEL, mib * 1024), (2, sparse, 10.0), (3, sparse, 30.0),
             (4, dense, 50.0)]
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE", fetch)
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE", write)
    bench.record_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), mib, "wan")
    rec = json.loads(out.read_text())
    assert rec["fetch_size_scale"] == pytest.approx(2.0)
    assert rec["write_size_scale"] == pytest.approx(1.0)
    sf = rec["kernels"]["sparse_fwd"]
    assert sf["launches"] == 2
    assert sf["fetch_bytes"] == int(2000.0 * 2.0 * 1024)     # mean KiB x scale x 1024
    assert sf["write_bytes"] == int(20.0 * 1024)
    assert rec["kernels"]["dense_fwd"]["fetch_bytes"] == int(500.0 * 2.0 * 1024)
    assert rec["bytes_per_launch"] == sf["fetch_bytes"] + sf["write_bytes"]
    assert rec["source_sha256_16"] == bench.source_hash()
    # reported only for the workload it was taken on, and for the current sources
    assert bench.measured_traffic("wan")["bytes_per_launch"] == rec["bytes_per_launch"]
    assert bench.measured_traffic("cog") is None
    rec["source_sha256_16"] = "0" * 16
    out.write_text(json.dumps(rec))
    assert bench.measured_traffic("wan") is None


def test_cpu_baseline_reports_three_phases():
    from oracle import losa_oracle as O
    from paper_2608_12032_amd import workload as W
    w = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(w, device="cpu")
    f64 = lambda x: x.double().numpy()  # noqa: E731
    m, _ = O.block_masses(f64(q), f64(k), w.N, w.block, w.bk, w.scale)
    rp, ci, _ = O.select_blocks(m, w.N, w.block, w.bk, w.tau)
    r = bench.cpu_baseline(w, q, k, v, torch.tensor(m, dtype=torch.float32),
                           torch.tensor(rp), torch.tensor(ci), 0.5)
    assert r["kind"] == "oracle" and r["unit"] == "ms/layer" and r["value"] > 0
    ph = r["phases_ms_per_layer"]
    assert set(ph) == {"calibrate", "select", "sparse_fwd"} and min(ph.values()) > 0
    assert r["value"] == ph["sparse_fwd"]
    assert r["host"]["nproc"] >= 1 and r["cores"] >= 1


def test_tiny_single_thread_times_the_whole_oracle():
    r = bench.tiny_single_thread()
    assert r["threads"] == 1 and r["workload"].startswith("tiny")
    assert set(r["ms"]) == {"calibrate", "select", "sparse_fwd"} and min(r["ms"].values()) > 0
