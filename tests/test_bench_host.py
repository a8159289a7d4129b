"""Host-side logic of bench.py (CPU only): the algorithmic byte counts the
decode roofline divides by, the HBM-traffic record built from rocprofv3
counter files, the rule that a traffic record only counts for the decode
kernel it was taken on, and the one-GPU refusal."""
import argparse
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_25537_amd import workloads as wl  # noqa: E402


def _hand_bytes(Hkv, keys_per_seq_sum, B, Hq, Dh, kv_bytes):
    """One launch, counted by hand: every key row of every kv head is K and
    V (Dh elements each), the appended row is written once per (sequence,
    kv head), and q and out are Hq x Dh fp32 per sequence."""
    row = 2 * Dh * kv_bytes
    return Hkv * keys_per_seq_sum * row + B * Hkv * row + 2 * B * Hq * Dh * 4


def test_llama_layer_bytes_by_hand():
    # 8 kv heads x (256 pool + 512 ring) keys x 512 B, + 8 x 512 B appended, + 2 x 32 x 128 x 4 B
    assert 8 * 768 * 512 + 8 * 512 + 2 * 32 * 128 * 4 == 3_182_592
    assert bench.decode_bytes(wl.get("llama3_8b_layer")) == 3_182_592


@pytest.mark.parametrize("name,expected", [
    ("mistral7b_batch64", 405_012_480), ("long_wide_d256", 806_092_800), ("llama_stack32", 202_506_240),
    ("paper_scale_b8", 5_865_472), ("ragged_batch64", 388_317_184),
])
def test_workload_bytes(name, expected):
    """The per-launch byte counts the measurement notes quote, re-derived
    from the workload sizes (ragged: each sequence's own k_b + q_b pool
    rows)."""
    w = wl.get(name)
    if w.ragged:
        rs = wl.ragged_sizes(w)
        pool = int(np.minimum(rs["n_rows"], w.k).sum() + rs["q_rows"].sum())
    else:
        pool = w.B * w.k
    assert _hand_bytes(w.Hkv, pool + w.B * w.W, w.B, w.Hq, w.Dh, w.kv_bytes) == expected
    assert bench.decode_bytes(w) == expected


def test_partial_rings_count_filled_slots_only():
    """A ring holding c tokens contributes min(c + 1, W) rows (its filled
    slots plus the appended row), and several launches average."""
    w = wl.get("llama3_8b_layer")  # B = 1, W = 512
    full = bench.decode_bytes(w)
    row_all_heads = w.Hkv * 2 * w.Dh * w.kv_bytes
    assert bench.decode_bytes(w, [511]) == full
    assert bench.decode_bytes(w, [10_000]) == full
    assert bench.decode_bytes(w, [99]) == full - (512 - 100) * row_all_heads
    two = bench.decode_bytes(w, [[99], [199]])
    assert two == full - ((512 - 100) + (512 - 200)) / 2 * row_all_heads


def _counter_dir(tmp, name, counter, kernel, values):
    d = tmp / name
    d.mkdir()
    with open(d / "r_counter_collection.csv", "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for i, v in enumerate(values):
            wr.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": v})
        # another kernel's samples must be ignored
        wr.writerow({"Dispatch_Id": 99, "Kernel_Name": "other_kernel", "Counter_Name": counter, "Counter_Value": 1e9})
    return str(d)


def test_pmc_summary_record(tmp_path, monkeypatch):
    """Counter files -> traffic record: each counter scaled by known / counted
    bytes of the copy probe, the median dispatch taken, the algorithmic
    bytes of that dispatch's ring fill alongside."""
    traffic = tmp_path / "traffic.json"
    traffic.write_text(json.dumps({"other_workload": {"kept": True}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    kib = 1024 * 1024  # a 1 GiB copy
    copy_f = _counter_dir(tmp_path, "cf", "FETCH_SIZE", "__amd_rocclr_copyBuffer", [kib / 2] * 3)
    copy_w = _counter_dir(tmp_path, "cw", "WRITE_SIZE", "__amd_rocclr_copyBuffer", [kib] * 3)
    fetch = [2000.0, 1900.0, 2100.0, 1950.0, 2050.0]  # median 2000
    write = [40.0, 41.0, 39.0, 40.0, 40.0]             # median 40
    dec_f = _counter_dir(tmp_path, "df", "FETCH_SIZE", "decode_kernel<4, bf16>", fetch)
    dec_w = _counter_dir(tmp_path, "dw", "WRITE_SIZE", "decode_kernel<4, bf16>", write)
    args = argparse.Namespace(workload="llama3_8b_layer", pmc_summary=[dec_f, dec_w, copy_f, copy_w],
                              copy_probe_mib=1024)
    bench.pmc_summary(args)
    data = json.loads(traffic.read_text())
    assert data["other_workload"] == {"kept": True}
    rec = data["llama3_8b_layer"]
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["fetch_bytes"] == 2000 * 2 * 1024 and rec["write_bytes"] == 40 * 1024
    assert rec["bytes_per_launch"] == 2000 * 2 * 1024 + 40 * 1024
    assert rec["dispatches"] == [5, 5]
    assert rec["kernel_hash"] == bench.decode_kernel_hash()
    w = wl.get("llama3_8b_layer")
    _, _, cnt0 = wl.window_kv(w)
    assert rec["algorithmic_bytes"] == round(bench.decode_bytes(w, cnt0.astype(np.int64) + 2))
    assert rec["algorithmic_bytes_rings_full"] == bench.decode_bytes(w)


def test_traffic_counts_only_for_its_kernel(tmp_path, monkeypatch):
    traffic = tmp_path / "traffic.json"
    traffic.write_text(json.dumps({"llama3_8b_layer": {"kernel_hash": "abc", "bytes_per_launch": 123}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    w = wl.get("llama3_8b_layer")
    monkeypatch.setattr(bench, "decode_kernel_hash", lambda: "abc")
    assert bench.recorded_traffic(w) == 123
    monkeypatch.setattr(bench, "decode_kernel_hash", lambda: "def")
    assert bench.recorded_traffic(w) is None
    assert bench.recorded_traffic(wl.get("mistral7b_batch64")) is None


def test_kernel_hash_ignores_comments():
    """Editing a comment, or blank lines, keeps the code's hash; editing code
    does not."""
    src = "int a; // note\n/* block\ncomment */ int b;\n"
    same = "int a; // another note\n\n/* a different\nblock */ int b;\n"
    assert bench._strip_comments(src) == bench._strip_comments(same)
    assert bench._strip_comments(src) != bench._strip_comments("int a; // note\n/* block\ncomment */ int c;\n")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("workload", ["ragged_batch64", "llama_stack32"])
def test_selection_only_takes_uniform_single_layer_workloads(workload):
    """--selection-only times the uniform selection of one layer's batch; a
    ragged batch or a layer stack is refused before any GPU work."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--selection-only", "--workload", workload],
                       capture_output=True, text=True, timeout=180, cwd=ROOT)
    assert r.returncode == 2, r.stderr[-2000:]
    assert "uniform single-layer" in r.stderr
    assert r.stdout == ""
