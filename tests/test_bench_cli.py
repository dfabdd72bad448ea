"""The measurement harness on the CPU: the one-GPU refusal, the algorithmic bytes the roofline
divides by, and the calibration of the traffic counters against a copy of known size."""
import csv
import importlib.util
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_attention_bytes_count_every_cached_row_once():
    bench = load_bench()
    from paper_2609_34370_amd import workloads as wl
    spec = wl.spec_with(1, batch=3)
    batch = wl.make_batch(spec, seed=4)
    D, hkv, hq, bs = spec.head_dim, spec.num_kv_heads, spec.num_q_heads, spec.block_size
    by_hand = 0
    for b in range(batch.B):
        S = int(batch.seq_lens[b])
        n = int(batch.qsl[b + 1] - batch.qsl[b])
        by_hand += S * hkv * D * 2 * 2            # K and V rows, bf16
        by_hand += n * hq * D * 2 * 2             # Q in, O out, bf16
        by_hand += -(-S // bs) * 4                # block ids used
    assert bench.attention_bytes(batch, spec) == by_hand


def write_counters(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, kib in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": kib})


def test_traffic_is_scaled_by_the_copy_reading(tmp_path, monkeypatch):
    # a copy of N bytes reads as N/2 KiB-counts of fetch and N of write: the factors 2 and 1 must
    # turn the attention kernels' readings into bytes; dispatches of a kernel are averaged, and
    # the call's two kernels summed
    bench = load_bench()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "_kernel_digest", lambda: "digest")
    (tmp_path / "profiles").mkdir()
    N = 1 << 30
    copy = "__amd_rocclr_copyBuffer"
    attn = "void spexis::verify_attn_kernel<128, 16, 1>(spexis::AttnParams)"
    merge = "void spexis::attn_merge_kernel<128>(spexis::AttnParams)"
    kib = 1.0 / 1024.0
    write_counters(tmp_path / "f.csv", "FETCH_SIZE", [(copy, N / 2 * kib), (copy, 10.0), (attn, 300e6 * kib),
                                                      (attn, 310e6 * kib), (merge, 5e6 * kib)])
    write_counters(tmp_path / "w.csv", "WRITE_SIZE", [(copy, N * kib), (attn, 1e6 * kib), (merge, 3e6 * kib)])
    bench.ingest_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 2, N)
    import json
    data = json.load(open(tmp_path / "profiles" / "traffic.json"))["workload2"]
    fetch = (305e6 + 5e6) * 2.0
    write = (1e6 + 3e6) * 1.0
    assert data["source_digest"] == "digest"
    np.testing.assert_allclose(data["bytes_per_launch"], fetch + write, rtol=1e-9)
    np.testing.assert_allclose(data["counters"]["FETCH_SIZE"]["factor"], 2.0)
    np.testing.assert_allclose(data["counters"]["WRITE_SIZE"]["factor"], 1.0)


def test_traffic_needs_the_copy_probe(tmp_path, monkeypatch):
    bench = load_bench()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    write_counters(tmp_path / "f.csv", "FETCH_SIZE", [("void spexis::verify_attn_kernel<128, 16, 1>", 1.0)])
    write_counters(tmp_path / "w.csv", "WRITE_SIZE", [("void spexis::verify_attn_kernel<128, 16, 1>", 1.0)])
    with pytest.raises(SystemExit):
        bench.ingest_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 2, 1 << 30)
