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
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, kib) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": kib})


def test_traffic_is_scaled_by_the_copy_reading(tmp_path, monkeypatch):
    # a copy of N bytes reads as N/2 KiB-counts of fetch and N of write: the factors 2 and 1 must
    # turn the kernels' readings into bytes; a call's launches are summed and divided by the
    # number of calls (the launches of its once-per-call kernel)
    bench = load_bench()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "_kernel_digest", lambda sources=(): "digest-" + sources[0])
    (tmp_path / "profiles").mkdir()
    N = 1 << 30
    copy = "__amd_rocclr_copyBuffer"
    attn = "void spexis::verify_attn_kernel<128, 16, 1>(spexis::AttnParams)"
    merge = "void spexis::attn_merge_kernel<128>(spexis::AttnParams)"
    stats = "spexis::accept_stats_kernel(spexis::AcceptParams, int)"
    decide = "spexis::accept_decide_kernel(spexis::AcceptParams, int, int, int, int)"
    search = "spexis::accept_search_kernel(spexis::AcceptParams)"
    kib = 1.0 / 1024.0
    # input copies (one larger than the probe), the three probe copies, then two calls of each:
    # attention + merge, and stats + two decide rounds + search
    write_counters(tmp_path / "f.csv", "FETCH_SIZE",
                   [(copy, 10.0), (copy, 3 * N * kib), (copy, N / 2 * kib), (copy, N / 2 * kib), (copy, N / 2 * kib),
                    (attn, 300e6 * kib), (merge, 5e6 * kib), (attn, 310e6 * kib),
                    (merge, 5e6 * kib), (stats, 60e6 * kib), (decide, 40e6 * kib), (decide, 8e6 * kib),
                    (search, 1e6 * kib), (stats, 60e6 * kib), (decide, 40e6 * kib), (decide, 10e6 * kib),
                    (search, 1e6 * kib)])
    write_counters(tmp_path / "w.csv", "WRITE_SIZE",
                   [(copy, 5 * N * kib), (copy, N * kib), (copy, N * kib), (copy, N * kib), (attn, 1e6 * kib), (merge, 3e6 * kib), (attn, 1e6 * kib), (merge, 3e6 * kib),
                    (stats, 1e5 * kib), (search, 1e4 * kib), (stats, 1e5 * kib), (search, 1e4 * kib)])
    bench.ingest_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 2, N)
    import json
    data = json.load(open(tmp_path / "profiles" / "traffic.json"))
    at, ac = data["workload2:verify_attention"], data["workload2:accept"]
    assert at["source_digest"] == "digest-attention.hip" and ac["source_digest"] == "digest-accept.hip"
    np.testing.assert_allclose(at["bytes_per_launch"], (305e6 + 5e6) * 2.0 + (1e6 + 3e6), rtol=1e-9)
    np.testing.assert_allclose(ac["bytes_per_launch"], (60e6 + 40e6 + 9e6 + 1e6) * 2.0 + (1e5 + 1e4), rtol=1e-9)
    np.testing.assert_allclose(at["counters"]["FETCH_SIZE"]["factor"], 2.0)
    np.testing.assert_allclose(at["counters"]["WRITE_SIZE"]["factor"], 1.0)
    assert ac["counters"]["FETCH_SIZE"]["calls"] == 2


def test_accept_bytes_follow_the_rows_a_sequence_reaches():
    # logits mode: both normalisers of rows 0..a (target and draft, the draft only up to k-1),
    # then the sampled rows again: residual (target + draft row a) or bonus (target row k)
    bench = load_bench()
    from paper_2609_34370_amd import workloads as wl
    spec = wl.spec_with(1, batch=3)
    batch = wl.make_batch(spec, seed=4, k=np.array([4, 4, 0], np.int32))
    V4 = 4 * spec.vocab
    accepted = np.array([0, 4, 0])
    expect = (V4 * 1 + V4 * 1 + 2 * V4) + (V4 * 5 + V4 * 4 + V4) + (V4 * 1 + 0 + V4)
    assert bench.accept_bytes(batch, spec, accepted) == expect


def test_traffic_needs_the_copy_probe(tmp_path, monkeypatch):
    bench = load_bench()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    write_counters(tmp_path / "f.csv", "FETCH_SIZE", [("void spexis::verify_attn_kernel<128, 16, 1>", 1.0)])
    write_counters(tmp_path / "w.csv", "WRITE_SIZE", [("void spexis::verify_attn_kernel<128, 16, 1>", 1.0)])
    with pytest.raises(SystemExit):
        bench.ingest_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 2, 1 << 30)
