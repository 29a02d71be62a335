"""bench.py on the CPU: the one-GPU refusal, the algorithmic bytes the roofline is priced with (from the model's
shapes, independently of the library), and the counter summaries made from rocprofv3-style CSV files."""

from __future__ import annotations

import csv
import json
import os
import subprocess
import sys

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


def weight_bytes_from_shapes(wl) -> int:
    """Packed bf16 weights of one tick: per layer W_q, W_k, W_v, W_o (A x d each), W_gate, W_up, W_down (F x d
    each); the head W [n_out][d]."""
    A, d, F = wl.n_heads * wl.head_dim, wl.d_model, wl.d_ffn
    return wl.n_layers * (4 * A * d + 3 * F * d) * 2 + wl.n_out * d * 2


@pytest.mark.parametrize("name,want", [("single_bf16_L224", 855_648_256), ("long_bf16_L4096_F64", 2_885_691_392),
                                       ("batched_bf16_B16_L1024", 9_328_142_336), ("ragged_fp8_B8", 26_769_631_232)])
def test_algorithmic_bytes_of_each_workload(name, want):
    wl = synth.WORKLOADS[name]
    assert weight_bytes_from_shapes(wl) == 738_207_744
    # K and V of every valid row, every layer, all heads: 2 B per bf16 element, 1 B per fp8 code
    es = 1 if wl.cache_dtype == "fp8" else 2
    assert sum(wl.lengths) * wl.n_layers * 2 * wl.n_heads * wl.head_dim * es + 738_207_744 == want
    assert bench.algorithmic_bytes(wl, weight_bytes_from_shapes(wl)) == want


def write_counters(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, c, v in rows:
            w.writerow({"Kernel_Name": k, "Counter_Name": c, "Counter_Value": v})


def test_counter_summary_averages_tick_launches_only(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    tick = "void fsx::k_tick<0, false>(fsx::TickArgs, fsx::TickParams, fsx::Dims)"
    write_counters(tmp_path / "a", [(tick, "SQ_INSTS_VALU", 100), (tick, "SQ_INSTS_VALU", 300),
                                    ("other_kernel", "SQ_INSTS_VALU", 7), (tick, "SQ_INSTS_MFMA", 10)])
    write_counters(tmp_path / "b", [(tick, "SQ_BUSY_CYCLES", 50), (tick, "SQ_BUSY_CYCLES", 70)])
    bench.summarize_counters([str(tmp_path / "a"), str(tmp_path / "b")], ["w1"], ["cmd a", "cmd b"])
    text = (tmp_path / "profiles" / "instructions_tick.md").read_text()
    row = [ln for ln in text.splitlines() if ln.startswith("| `w1`")][0].split("|")
    cols = ["", " workload "] + [c.replace("SQ_", "") for c in bench.INSTR_COUNTERS]
    vals = dict(zip([c.strip() for c in cols[1:]], [c.strip() for c in row[1:]]))
    assert vals["INSTS_VALU"] == "200" and vals["INSTS_MFMA"] == "10" and vals["BUSY_CYCLES"] == "60"
    assert vals["INSTS_LDS"] == "–"
    assert "cmd a" in text and "cmd b" in text


def test_traffic_summary_scales_by_the_copy_calibration(tmp_path, monkeypatch):
    real_hash = bench.source_hash()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_hash", lambda: real_hash)
    os.makedirs(tmp_path / "profiles")
    tick = "fsx::k_tick<1, false>"
    copy = "__amd_rocclr_copyBuffer"
    write_counters(tmp_path / "f", [(tick, "FETCH_SIZE", 1000), (tick, "FETCH_SIZE", 3000)])
    write_counters(tmp_path / "w", [(tick, "WRITE_SIZE", 500)])
    write_counters(tmp_path / "cf", [(copy, "FETCH_SIZE", 4000)])
    write_counters(tmp_path / "cw", [(copy, "WRITE_SIZE", 8000)])
    # a 1 MiB copy reads 4000 and writes 8000 units: 262.144 and 131.072 bytes per unit
    bench.summarize_traffic([str(tmp_path / x) for x in ("f", "w", "cf", "cw")], "wl", 1 << 20, ["c"])
    d = json.load(open(tmp_path / "profiles" / "traffic_wl.json"))
    assert d["fetch_bytes_per_launch"] == int(2000 * (1 << 20) / 4000)
    assert d["write_bytes_per_launch"] == int(500 * (1 << 20) / 8000)
    assert d["source_hash"] == real_hash


def test_attention_tail_separates_a_slow_xcd_from_a_late_slot():
    """A synthetic phase trace (256 workgroups, workgroup w on XCD w mod 8, slot w // 8): XCD 3 ends every layer's
    attention 5 µs late and slot 7 of every XCD 2 µs late."""
    np = pytest.importorskip("numpy")
    G, nl, t0 = 256, 4, 1000
    tr = np.zeros((G, 2 + 16 * nl + 1), dtype=np.int64)
    w = np.arange(G)
    for l in range(nl):
        start = t0 + 100_000 * l  # the previous layer's latest end
        extra = 5.0 * (w % 8 == 3) + 2.0 * (w // 8 == 7)
        tr[:, 2 + 16 * l + 1] = start + ((100.0 + extra) * 100).astype(np.int64)
        tr[:, 2 + 16 * l + 4] = t0 + 100_000 * (l + 1)  # every workgroup ends the layer at once
        tr[:, 2 + 16 * l + 5 + 4] = start + 50  # every workgroup ran an attention unit
    per_x, latest, slot_mean = bench.attention_tail(tr, nl, t0)
    assert per_x == pytest.approx([102.0] * 3 + [107.0] + [102.0] * 4)
    assert latest == pytest.approx(107.0)
    assert len(slot_mean) == 32
    assert slot_mean[7] == pytest.approx(2.0)
    assert all(v == pytest.approx(0.0) for k, v in enumerate(slot_mean) if k != 7)
