"""Host-side arithmetic of bench.py (no GPU): the algorithmic FLOPs per latent
and the per-step row counts that the roofline figures divide by, the
per-step latency histograms, and the one-GPU guard.

The FLOP pins are written out from the model's layer widths (Sec. II-A: the
masked context convolution over the causal taps, then the three 1x1 layers of
the entropy-parameter network with widths 640/512/2KM for M = 192 and
1066/853/2KM for M = 320); the step counts are the schedule length
T = W + lambda (H - 1) of Theorem 1 (lambda = 3 for the 5x5 mask, 2 relaxed).
"""
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
from paper_2607_19082_amd import inputs  # noqa: E402


def macs_by_hand(M, taps, d1, d2, K):
    # context: taps x M inputs -> 2M outputs; layer 1 over [psi (2M), ctx (2M)]
    return taps * M * 2 * M + 4 * M * d1 + d1 * d2 + d2 * (2 * K * M if K == 1 else 3 * K * M)


@pytest.mark.parametrize("name,taps,d1,d2,K,T,mflop", [
    ("minnen-16x16-m192", 12, 640, 512, 1, 16 + 3 * 15, 3.801088),
    ("minnen-kodak-48x32-m192", 12, 640, 512, 1, 48 + 3 * 31, 3.801088),
    ("cheng-gmm3-1080p-120x68-m192", 12, 640, 512, 3, 120 + 3 * 67, 5.177344),
    ("minnen-relaxed-b8-120x68-m192", 10, 640, 512, 1, 120 + 2 * 67, 3.506176),
    ("minnen-hr-4k-240x135-m320", 12, 1066, 853, 1, 240 + 3 * 134, 10.554596),
])
def test_flops_and_steps(name, taps, d1, d2, K, T, mflop):
    cfg = inputs.workload(name)
    assert (cfg["d1"], cfg["d2"], cfg["K"]) == (d1, d2, K)
    f = bench.flops_per_latent(cfg)
    assert f == 2 * macs_by_hand(cfg["M"], taps, d1, d2, K)
    assert abs(f / 1e6 - mflop) < 1e-6
    rows = bench.step_rows(cfg)
    assert len(rows) == T
    assert rows.sum() == cfg["B"] * cfg["H"] * cfg["W"]
    # rows grow by B per lambda steps up to min(H, ceil(W / lambda)) wavefront members
    lam = T - cfg["W"] if cfg["H"] == 2 else (T - cfg["W"]) // (cfg["H"] - 1)
    assert rows.max() == cfg["B"] * min(cfg["H"], -(-cfg["W"] // lam))
    assert rows[0] == cfg["B"] and rows[-1] == cfg["B"]


def test_grouped_rows_sum():
    cfg = inputs.workload("minnen-hr-4k-240x135-m320")
    for g in (2, 4, 8, 16):
        r = bench.step_rows(cfg, g)
        assert len(r) == -(-642 // g) and r.sum() == 32400


def test_latency_histogram_bins():
    h = bench.latency_histogram([0.5, 1.0, 1.9, 3.0, 100.0, 7.99], 1.0)
    assert h["counts"] == [1, 2, 1, 1, 0, 0, 0, 1]
    assert h["steps"] == 6 and abs(h["sum_ms"] - 0.11439) < 1e-9
    assert h["percentiles_us"]["p0"] == 0.5 and h["percentiles_us"]["p100"] == 100.0
    h2 = bench.latency_histogram([3.0, 3.0], 1.5)
    assert h2["counts"][2] == 2 and h2["median_over_L_floor"] == 2.0


def write_trace(path, spans):
    """A kernel trace of two calls, each k_set_call followed by the phase
    kernels given as (start, end) ns pairs (the second call's shifted by 1 ms
    and stretched by 2)."""
    fields = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        t0 = 0
        for call in range(2):
            w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": "wf::k_set_call(int)", "Start_Timestamp": t0,
                        "End_Timestamp": t0 + 10})
            w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": "void wf::k_hoist<wf::PF32>(x)",
                        "Start_Timestamp": t0 + 20, "End_Timestamp": t0 + 30})
            for a, b in spans:
                w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": "void wf::k_phase<wf::PF32, 1, false>(x)",
                            "Start_Timestamp": t0 + a * (call + 1), "End_Timestamp": t0 + b * (call + 1)})
            t0 += 1_000_000


def test_trace_step_latency(tmp_path):
    # two steps of three phases: busy 3+3+3 us and 1+1+1 us; spans 10 us and
    # 3.5 us (first kernel of step 2 to the last kernel's end)
    spans = [(1000, 4000), (4000, 7000), (7000, 10000), (11000, 12000), (12500, 13500), (13500, 14500)]
    p = tmp_path / "run_kernel_trace.csv"
    write_trace(p, spans)
    busy, span = bench.trace_step_latency(str(p), 0, 2, 2.0)
    assert busy["steps"] == 2 and span["steps"] == 2
    assert busy["percentiles_us"]["p0"] == 3.0 and busy["percentiles_us"]["p100"] == 9.0
    assert span["percentiles_us"]["p0"] == 3.5 and span["percentiles_us"]["p100"] == 10.0
    assert busy["counts"] == [0, 1, 0, 1, 0, 0, 0, 0]
    busy2, span2 = bench.trace_step_latency(str(p), 1, 2, 2.0)
    assert busy2["percentiles_us"]["p100"] == 18.0 and span2["percentiles_us"]["p0"] == 7.0
    # as three steps of two phases
    busy3, _ = bench.trace_step_latency(str(p), 0, 3, 1.0)
    assert busy3["steps"] == 3 and busy3["percentiles_us"]["p100"] == 6.0
    # a call that is not in the trace, or phases that do not split evenly into T steps
    assert bench.trace_step_latency(str(p), 2, 2, 2.0) is None
    write_trace(p, spans[:5])
    assert bench.trace_step_latency(str(p), 0, 2, 2.0) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_histogram_edges_cover_everything():
    x = np.array([0.0, 1e-9, 63.9, 64.0, 1e9])
    h = bench.latency_histogram(x, 1.0)
    assert sum(h["counts"]) == x.size


def test_stats_summary_leaves_out_the_persistent_leg(tmp_path):
    """A graph-driver run whose bench also traced persistent decodes: those
    dispatches stay out of the call count, the table and the per-call time."""
    d = tmp_path / "st"
    d.mkdir()
    stats = [("wf::k_set_call(x)", 5, 5e3), ("void wf::k_phase<wf::PF32, 1, false>(x)", 4 * 6, 24e6),
             ("void wf::k_hoist<wf::PF32>(x)", 4, 4e6), ("void wf::k_persistent<wf::PF32, 1>(x)", 1, 9e6),
             ("wf::k_zero_u32(x)", 1, 2e3)]
    total = sum(t for _, _, t in stats)
    with open(d / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs",
                                          "Percentage"])
        w.writeheader()
        for n, c, t in stats:
            w.writerow({"Name": n, "Calls": c, "TotalDurationNs": t, "AverageNs": t / c, "MinNs": t / c,
                        "MaxNs": t / c, "Percentage": 100.0 * t / total})
    # busy 9 us and 3 us: 6 and 2 times the floor of 1.5 us
    write_trace(d / "run_kernel_trace.csv",
                [(1000, 4000), (4000, 7000), (7000, 10000), (11000, 12000), (12500, 13500), (13500, 14500)])
    rec = {"metric": "m", "value": 1.0, "ms_per_step": 1.0, "warmup": 0, "steps": 1,
           "config": {"workload": "w", "precision": "fp32", "driver": "graph", "steps_T": 2},
           "roofline": {"launch_ms_events": 1.0}, "latency_roofline": {"L_floor_us": 1.0}}
    log = tmp_path / "st.log"
    log.write_text("noise\n" + json.dumps(rec) + "\n")
    out = tmp_path / "kernels_w_fp32_graph.md"
    bench.summarize_stats(str(d), str(log), str(out), "cmd", l_floor_us=1.5)
    txt = out.read_text()
    assert "The run makes 4 decode/encode calls" in txt
    assert "The 1 traced decodes of the persistent driver" in txt
    assert "k_persistent" not in txt.split("The 1 traced")[1]
    # (24 + 4) ms of phase and hoist kernels plus the set-call kernels over 4 calls
    assert "Decode kernels per call: 7.001 ms" in txt
    assert "L_floor = 1.50 us" in txt and "| steps | 0 | 0 | 1 | 1 | 0 | 0 | 0 | 0 |" in txt


def test_parity_record():
    import bench
    rng = np.random.default_rng(0)
    table = np.exp(np.linspace(np.log(0.11), np.log(256.0), 64)).astype(np.float32)
    sc = rng.uniform(0.2, 50.0, size=(1, 3, 5, 1, 4)).astype(np.float32)
    idx = np.searchsorted(table[:-1], sc, side="left").astype(np.int32)
    ref = {"y_hat": rng.normal(size=(1, 3, 5, 4)), "mean": rng.normal(size=(1, 3, 5, 4)), "scale": sc, "idx": idx}
    got = {k: v.copy() for k, v in ref.items()}
    r = bench.parity_record(got, ref, table, 1e-4)
    assert r["within_bar"] and r["idx_mismatch_unexcused"] == 0
    assert all(v == 0.0 for v in r["max_abs_err"].values())
    got["mean"] = got["mean"] + 2e-4
    r = bench.parity_record(got, ref, table, 1e-4)
    assert not r["within_bar"] and abs(r["max_abs_err"]["mean"] - 2e-4) < 1e-9
    # an index flip at a scale sitting on a level is excused and counted
    got = {k: v.copy() for k, v in ref.items()}
    ref["scale"][0, 0, 0, 0, 0] = table[10]
    ref["idx"][0, 0, 0, 0, 0] = 10
    got["idx"][0, 0, 0, 0, 0] = 11
    got["scale"][0, 0, 0, 0, 0] = table[10] * np.float32(1 + 5e-5)   # (its own decision: 11)
    r = bench.parity_record(got, ref, table, 1e-4)
    assert r["idx_mismatch_at_boundary"] == 1 and r["idx_mismatch_unexcused"] == 0 and r["within_bar"]
    assert r["idx_inconsistent_with_own_scale"] == 0
    # an index that does not follow the decode's own scale fails the bar
    bad = {k: v.copy() for k, v in got.items()}
    bad["idx"][0, 2, 2, 0, 2] += 1
    r = bench.parity_record(bad, ref, table, 1e-4)
    assert r["idx_inconsistent_with_own_scale"] == 1 and not r["within_bar"]
    # bf16: a level between the two scales (1e-3 apart, outside 1e-4 of the
    # level) excuses the flip and is counted apart; fp32 does not excuse it
    g2, r2 = {k: v.copy() for k, v in got.items()}, {k: v.copy() for k, v in ref.items()}
    r2["scale"][0, 1, 2, 0, 3] = table[20] * np.float32(1 - 1e-3)
    r2["idx"][0, 1, 2, 0, 3] = 20
    g2["scale"][0, 1, 2, 0, 3] = table[20] * np.float32(1 + 1e-3)
    g2["idx"][0, 1, 2, 0, 3] = 21
    rb = bench.parity_record(g2, r2, table, 1e-2, bf16=True)
    assert rb["idx_mismatch_bracketed"] == 1 and rb["idx_mismatch_unexcused"] == 0 and rb["within_bar"]
    assert bench.parity_record(g2, r2, table, 1e-2)["idx_mismatch_unexcused"] == 1
    got["idx"][0, 1, 1, 0, 1] += 1
    assert bench.parity_record(got, ref, table, 1e-4)["idx_mismatch_unexcused"] == 1
