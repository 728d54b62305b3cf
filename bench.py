"""Benchmark: wavefront decode of one 3840x2160 image's latent (240x135 latents,
M = 320 channels) through the C-ABI, on one MI355X.

One step = one whole decode of the latent grid: every wavefront step's tap
gather, context product, entropy-parameter network, parameter epilogue and
y_hat write, plus the pre-loop hyperprior product.  Inputs are seeded
synthetic arrays (weights N(0, 1/fan_in), hyperprior params N(0, 1), Laplace
symbols) already resident in HBM.  Prints one JSON line.

The default driver is the resident one (one cooperative k_resident launch per
decode, each workgroup's weight slice held in registers for the whole decode);
--driver picks another, and the context approximation (--group > 1) runs on
the graph driver.

roofline: one decode is one decode call (resident driver: counter reset,
hoist and the k_resident launch, which takes nearly all of it), one launch of
the plan's HIP graph (graph driver: the hoist, two context kernels and one
kernel per phase of every step) or of k_persistent (persistent driver), timed
with HIP events on the launch stream;
achieved = algorithmic FLOPs of a decode / that time, against the dense fp32
(or bf16) MFMA peak.  traffic = HBM bytes of one decode from the committed
rocprofv3 FETCH_SIZE / WRITE_SIZE summary for this workload, precision and
driver, scaled by the counters' reading for a plain copy of known size; null
when no summary exists or the kernel sources changed since it was taken.
latency_roofline adds the dependency floor: T_roof = hoist / peak + sum over
steps of max(F_t / peak, L_floor), with L_floor the measured minimal
dependent hop.

--summarize-traffic writes such a summary from rocprofv3 --pmc outputs.
"""
import argparse
import glob
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2500.0}
DEFAULT_WORKLOAD = "minnen-hr-4k-240x135-m320"
CSRC = os.path.join(ROOT, "paper_2607_19082_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
# kernels of one decode call (the rest of a bench run: the floor probes, torch)
DECODE_KERNELS = ("wf::k_phase", "wf::k_hoist", "wf::k_ctxo", "wf::k_set_call", "wf::k_persistent", "wf::k_zero_u32",
                  "wf::k_dataflow", "wf::k_zero_u128", "wf::k_resident", "wf::k_res_zero")


# kernels of the bench's per-step latency leg (one traced decode by the
# persistent driver); when another driver is timed they stay out of its summaries
LEG_KERNELS = ("wf::k_persistent", "wf::k_zero_u32")


def leg_kernel(k, driver):
    return driver != "persistent" and any(x in k for x in LEG_KERNELS)


# sources that no decode from symbols runs (the transforms, the entropy coder)
NOT_DECODE = ("wf_xform.hip", "wf_ec.hip")


def source_hash():
    """sha256 over the sources of the decode's kernels and plan: counters taken
    on other sources are stale."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(CSRC, "*.hip"))):
        if os.path.basename(f) in NOT_DECODE:
            continue
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_file(workload, precision, driver):
    return os.path.join(PROFILES, f"traffic_{workload}_{precision}_{driver}.md")


def read_traffic(workload, precision, driver):
    """HBM bytes of one decode from the committed counter summary, or None."""
    path = traffic_file(workload, precision, driver)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].strip().split(": ", 1)
                vals[k] = v.strip("`")
    if vals.get("source_sha256") != source_hash():
        return None
    return float(vals["hbm_bytes_per_decode"])


def _pmc_rows(d):
    import sqlite3
    db = glob.glob(os.path.join(d, "**", "*results.db"), recursive=True)[0]
    con = sqlite3.connect(db)
    return list(con.execute("select kernel_name, counter_name, value from counters_collection"))


def summarize_traffic(fetch_dir, write_dir, cal_fetch_dir, cal_write_dir, cal_bytes, out, command, driver):
    """Per-decode HBM bytes from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs
    (KiB per dispatch), each scaled by the same counter's reading for a plain
    copy of cal_bytes bytes."""
    def total(d, cname, pred):
        return sum(v for k, c, v in _pmc_rows(d) if c == cname and pred(k))
    is_copy = lambda k: "copyBuffer" in k or "copy" in k.lower()
    f_cal = cal_bytes / (1024.0 * total(cal_fetch_dir, "FETCH_SIZE", is_copy))
    w_cal = cal_bytes / (1024.0 * total(cal_write_dir, "WRITE_SIZE", is_copy))
    is_dec = lambda k: any(x in k for x in DECODE_KERNELS) and not leg_kernel(k, driver)
    fetch_rows = _pmc_rows(fetch_dir)
    decodes = sum(1 for k, c, v in fetch_rows if c == "FETCH_SIZE" and "k_set_call" in k) - \
        sum(1 for k, c, v in fetch_rows if c == "FETCH_SIZE" and "wf::k_persistent" in k and leg_kernel(k, driver))
    fetch = total(fetch_dir, "FETCH_SIZE", is_dec) * 1024.0 * f_cal / decodes
    write = total(write_dir, "WRITE_SIZE", is_dec) * 1024.0 * w_cal / decodes
    with open(out, "w") as f:
        f.write("# HBM traffic of one decode (rocprofv3 counters)\n\n")
        f.write("FETCH_SIZE and WRITE_SIZE summed over the dispatches of the decode call(s), per decode,\n")
        f.write("each scaled by the counter's reading for a plain device copy of a known size.\n\n")
        f.write(f"- decodes_profiled: {decodes}\n- fetch_scale: {f_cal:.4f}\n- write_scale: {w_cal:.4f}\n")
        f.write(f"- fetch_bytes_per_decode: {fetch:.0f}\n- write_bytes_per_decode: {write:.0f}\n")
        f.write(f"- hbm_bytes_per_decode: {fetch + write:.0f}\n- source_sha256: `{source_hash()}`\n\n")
        f.write("Commands:\n\n```\n" + command + "\n```\n")
    print(json.dumps({"fetch_scale": f_cal, "write_scale": w_cal, "fetch": fetch, "write": write,
                      "decodes": decodes}))


# wave-state counters of one --pmc pass (eight SQ counters at most; the
# pass also takes SQ_BUSY_CYCLES, which counts per shader engine, not per wave)
WAVE_STATE = ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU",
              "SQ_ACTIVE_INST_VMEM", "SQ_ACTIVE_INST_LDS")


def summarize_counters(dirs, out, command, driver):
    """MFMA utilisation and L2 hit rate of the decode's dispatches from
    rocprofv3 --pmc runs (one counter set per run): MfmaUtil (percent of the
    SIMDs' cycles with the matrix unit busy) weighted by dispatch duration,
    and TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum), overall and per kernel;
    with a pass of the WAVE_STATE counters also where the waves' cycles go."""
    import sqlite3
    rows = []
    for d in dirs:
        db = glob.glob(os.path.join(d, "**", "*results.db"), recursive=True)[0]
        con = sqlite3.connect(db)
        rows += list(con.execute("select kernel_name, counter_name, value, duration from counters_collection"))
    is_dec = lambda k: any(x in k for x in DECODE_KERNELS) and not leg_kernel(k, driver)
    short = lambda k: k.split("(")[0].replace("void ", "")
    per = {}
    for k, c, v, dur in rows:
        if not is_dec(k):
            continue
        e = per.setdefault(short(k), {"n": 0, "dur": 0.0, "mfma_w": 0.0, "mfma_dur": 0.0, "hit": 0.0, "miss": 0.0})
        if c == "MfmaUtil":
            e["n"] += 1
            e["dur"] += dur
            e["mfma_w"] += v * dur
            e["mfma_dur"] += dur
        elif c == "TCC_HIT_sum":
            e["hit"] += v
        elif c == "TCC_MISS_sum":
            e["miss"] += v
        elif c in WAVE_STATE:
            e[c] = e.get(c, 0.0) + v
    tot = {k: sum(e[k] for e in per.values()) for k in ("dur", "mfma_w", "mfma_dur", "hit", "miss")}
    mfma = tot["mfma_w"] / tot["mfma_dur"] if tot["mfma_dur"] else float("nan")
    hit = tot["hit"] / (tot["hit"] + tot["miss"]) if tot["hit"] + tot["miss"] else float("nan")
    with open(out, "w") as f:
        f.write("# MFMA utilisation and L2 hit rate of the decode (rocprofv3 counters)\n\n")
        f.write("MfmaUtil = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMDs), per dispatch, weighted by\n")
        f.write("dispatch duration; L2 hit rate = TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum).  The counters\n")
        f.write("serialise the dispatches, so durations here are longer than in a timed run.\n\n")
        f.write(f"- mfma_util_percent: {mfma:.2f}\n- l2_hit_rate: {hit:.4f}\n- source_sha256: `{source_hash()}`\n\n")
        f.write("| Kernel | Dispatches | MfmaUtil % | L2 hit rate |\n|---|---|---|---|\n")
        for k, e in sorted(per.items(), key=lambda kv: -kv[1]["dur"]):
            mu = e["mfma_w"] / e["mfma_dur"] if e["mfma_dur"] else float("nan")
            hr = e["hit"] / (e["hit"] + e["miss"]) if e["hit"] + e["miss"] else float("nan")
            f.write(f"| `{k}` | {e['n']} | {mu:.2f} | {hr:.4f} |\n")
        if any("SQ_WAVE_CYCLES" in e for e in per.values()):
            f.write("\nWave state (share of SQ_WAVE_CYCLES, the cycles waves were resident; the SQ_ACTIVE_INST_* "
                    "shares overlap with each other):\n\n| Kernel | " + " | ".join(WAVE_STATE[1:]) + " |\n|---|"
                    + "---|" * (len(WAVE_STATE) - 1) + "\n")
            for k, e in sorted(per.items(), key=lambda kv: -kv[1]["dur"]):
                if e.get("SQ_WAVE_CYCLES"):
                    f.write(f"| `{k}` | " + " | ".join(f"{e.get(c, 0.0) / e['SQ_WAVE_CYCLES']:.3f}"
                                                       for c in WAVE_STATE[1:]) + " |\n")
        f.write("\nCommands:\n\n```\n" + command + "\n```\n")
    print(json.dumps({"mfma_util_percent": mfma, "l2_hit_rate": hit}))


def summarize_stats(stats_dir, log, out, command, l_floor_us=None):
    """Kernel statistics of a profiled bench run (rocprofv3 --kernel-trace
    --stats): the per-kernel table, and the decode kernels' time per call next
    to the HIP-event time of one decode from the same run's bench line."""
    import csv
    rows = list(csv.DictReader(open(glob.glob(os.path.join(stats_dir, "**", "*kernel_stats.csv"), recursive=True)[0])))
    rec = json.loads([l for l in open(log) if l.startswith('{"metric"')][-1])
    cfg = rec["config"]
    leg = [r for r in rows if leg_kernel(r["Name"], cfg["driver"])]
    leg_calls = sum(int(r["Calls"]) for r in leg if "wf::k_persistent" in r["Name"])
    rows = [r for r in rows if r not in leg]
    calls = sum(int(r["Calls"]) for r in rows if "k_set_call" in r["Name"]) - leg_calls
    dec = sum(float(r["TotalDurationNs"]) for r in rows if any(x in r["Name"] for x in DECODE_KERNELS))
    lines = [f"# Kernel statistics: {cfg['workload']}, {cfg['precision']}, {cfg['driver']} driver"
             + (f", context approximation N = {cfg['context_approximation_group']}"
                if cfg.get("context_approximation_group", 1) > 1 else "")
             + (f", {cfg['mask']} mask" if cfg.get("mask") not in (None, "full", "relaxed") else "")
             + (", with the decode from rANS streams" if rec.get("entropy_decode") else "")
             + (", with the transforms" if rec.get("end_to_end") else ""), "",
             "Command (on one MI355X, from the repository root):", "", "```", command, "```", "",
             f"The run makes {calls} decode/encode calls (warm-up, timed decodes, encodes); per-call kernels appear "
             f"that many times.  k_empty and k_barrier_rounds are the latency-floor probes of the bench."
             + (f"  The {leg_calls} traced decodes of the persistent driver (the bench's per-step latency leg) "
                "are left out of this table." if leg_calls else ""), "",
             "| Kernel | Calls | Total (ms) | Average (us) | Min (us) | Max (us) | % |", "|---|---|---|---|---|---|---|"]
    # shares of the kernels in the table (the left-out leg's time excluded)
    total_ns = sum(float(r["TotalDurationNs"]) for r in rows)
    for r in rows:
        pct = 100.0 * float(r["TotalDurationNs"]) / total_ns
        if pct < 0.05:
            continue
        name = r["Name"].split("(")[0].replace("void ", "")
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                     f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                     f"{float(r['MaxNs']) / 1e3:.2f} | {pct:.2f} |")
    lines += ["", f"Decode kernels per call: {dec / max(calls, 1) / 1e6:.3f} ms of kernel time.  The same run's "
              f"HIP-event time of one decode (under the profiler) was {rec['roofline']['launch_ms_events']:.3f} ms; "
              f"bench line: {rec['ms_per_step']:.3f} ms per decode, {rec['value']:.0f} latents/s.  For the graph "
              "and stream drivers the difference is the gaps between kernels."]
    trace = glob.glob(os.path.join(stats_dir, "**", "*kernel_trace.csv"), recursive=True)
    traced_floor = rec.get("latency_roofline", {}).get("L_floor_us")
    lfloor = l_floor_us or traced_floor
    # the bench's first calls are its warm-up and timed decodes: take the last timed one
    hist = trace_step_latency(trace[0], rec["warmup"] + rec["steps"] - 1, cfg["steps_T"], lfloor) \
        if trace and lfloor and cfg["driver"] in ("graph", "stream") else None
    if hist:
        busy, span = hist
        src = (f"measured by a bench run without the profiler (the same probe under the tracer read "
               f"{traced_floor:.2f} us)" if l_floor_us else "measured in this run, under the tracer")
        lines += ["", "Per-step latency of the last timed decode in the trace, in multiples of the latency floor "
                  f"L_floor = {lfloor:.2f} us, one dependent hop between graph nodes, {src}.  Busy: the sum of "
                  "the step's phase kernels' durations.  Span: start of the step's first phase kernel to the "
                  "start of the next step's, gaps included (the tracer lengthens the gaps).", ""]
        lines += histogram_table(busy, "busy") + [""] + histogram_table(span, "span")
    ec = rec.get("entropy_decode")
    if ec:
        lines += ["", "This run also times the decode from rANS streams (`entropy_decode` in the bench line: "
                  f"{ec['ms_per_image']:.3f} ms per image, {ec['no_escapes']['ms_per_image']:.3f} ms for a stream "
                  "without escapes; the stream encoder "
                  f"{ec['encode_bits_ms_per_image']:.3f} ms).  Its phase C runs as `k_phase<…, true>` (one launch "
                  "per step), its stream set-up as `k_ec_init`; the stream encoder is `k_ec_encode`, `k_ec_scan`, "
                  "`k_ec_compact`.  The per-call line above then mixes both decodes."]
    e2e = rec.get("end_to_end")
    if e2e:
        lines += ["", "This run also times the transforms (`end_to_end` in the bench line): the hyper-decoder "
                  f"{e2e['hyper_decoder_ms_per_image']:.3f} ms and the synthesis {e2e['synthesis_ms_per_image']:.3f} "
                  f"ms per image ({e2e['ms_per_image']:.3f} ms end to end with the decode); their layers run as "
                  "`k_conv<P, mode, row tiles, column tiles, column waves>` (mode 0: transposed conv by output "
                  "class, 1: 3x3 conv, 2: inverse GDN, 3: the image layer with the classes as columns)."]
    # runs that also time the rANS decode or the transforms get a summary of their own
    out = out[:-len(".md")] + ("_entropy" if ec else "") + ("_transforms" if e2e else "") + ".md"
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({"calls": calls, "decode_kernel_ms_per_call": dec / max(calls, 1) / 1e6}))


def copy_calibration(nbytes):
    """A plain device copy of nbytes whose source is not cache resident (the
    source, then as many bytes of other writes, then the copy): the reference
    reading for FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = int(nbytes) // 4
    src = torch.ones(n, device="cuda")
    evict = torch.empty(n, device="cuda")
    dst = torch.empty_like(src)
    evict.fill_(2.0)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copied_bytes": n * 4}), flush=True)


# causal taps, shear and kernel radius of each mask (Def. 1; Sec. III-B)
MASK_TAPS = {"full": 12, "relaxed": 10, "3x3": 4, "7x7": 24}
MASK_SHEAR = {"full": 3, "relaxed": 2, "3x3": 2, "7x7": 4}
MASK_RADIUS = {"full": 2, "relaxed": 2, "3x3": 1, "7x7": 3}


def mask_of(cfg):
    return cfg.get("mask") or ("relaxed" if cfg["relaxed"] else "full")


# transform channels N of the hyper-latent and the synthesis (M -> N)
XFORM_N = {192: 128, 320: 192}


def synthesis_flops(N, M, lat):
    """2 x MACs of g_s per image of `lat` latents: four stride-2 transposed
    convs (25/4 taps per output pixel) and three inverse GDNs (N x N)."""
    px = [4 * lat, 16 * lat, 64 * lat, 256 * lat]
    macs = px[0] * N * M * 25 / 4 + (px[1] + px[2]) * N * N * 25 / 4 + px[3] * 3 * N * 25 / 4
    macs += (px[0] + px[1] + px[2]) * N * N
    return 2 * macs


def hyper_flops(N, M, lat):
    """2 x MACs of h_s (on the 4x-upsampled z grid, ~lat latents)."""
    c = M * 3 // 2
    return 2 * (lat / 4 * M * N * 25 / 4 + lat * c * M * 25 / 4 + lat * 2 * M * c * 9)


def flops_per_latent(cfg):
    """Algorithmic FLOPs of one latent (2 x MACs): the context product over the
    causal taps and the three layers of the entropy-parameter network."""
    M, d1, d2, n3 = cfg["M"], cfg["d1"], cfg["d2"], cfg["n3"]
    taps = MASK_TAPS[mask_of(cfg)]
    macs = taps * M * 2 * M + 4 * M * d1 + d1 * d2 + d2 * n3
    return 2 * macs


def hoistable_flops_per_latent(cfg):
    """The hyperprior half of layer 1 (computed before the step loop)."""
    return 2 * 2 * cfg["M"] * cfg["d1"]


def step_rows(cfg, group=1):
    """Latents per decoding step: per wavefront, or per group of `group`
    wavefronts under context approximation."""
    H, W, B = cfg["H"], cfg["W"], cfg["B"]
    lam = MASK_SHEAR[mask_of(cfg)]
    T = W + lam * (H - 1)
    rows = np.zeros(T, np.int64)
    for i in range(H):
        rows[lam * i:lam * i + W] += B
    if group > 1:
        rows = np.add.reduceat(rows, np.arange(0, T, group))
    return rows


def parity_record(got, ref, table, tol, bf16=False):
    """Element-wise comparison of the timed decode's outputs with the oracle's
    decode of the same latents: the largest absolute error per output, the
    scale indices within 1e-4 relative of a table level (where the index is
    excused and counted), for bf16 also those where a level lies between the
    two scales (counted apart), and the index mismatches outside them."""
    rec = {"bar_abs": tol}
    errs = {}
    for k in ("y_hat", "mean", "scale", "weight", "comp_mean"):
        if k in got and k in ref and got[k] is not None:
            g, r = np.asarray(got[k], np.float64), np.asarray(ref[k], np.float64)
            errs[k] = float(np.abs(g - r).max()) if g.size else 0.0
    rec["max_abs_err"] = errs
    t = np.asarray(table, np.float64)[:-1]
    s = np.asarray(ref["scale"], np.float64).reshape(-1)
    near = np.zeros(s.shape, bool)
    pos = np.searchsorted(t, s)
    for off in (-1, 0):
        q = np.clip(pos + off, 0, len(t) - 1)
        near |= np.abs(s - t[q]) <= 1e-4 * t[q]
    near &= s != np.float64(table[0])
    gi = np.asarray(got["idx"]).reshape(-1)
    mism = gi != np.asarray(ref["idx"]).reshape(-1)
    rec["idx_boundary_cases"] = int(near.sum())
    rec["idx_mismatch_at_boundary"] = int((mism & near).sum())
    # the index decided on the timed decode's own scale (in fp32, as the
    # kernel decides it) must hold exactly
    own = np.searchsorted(np.asarray(table, np.float32)[:-1],
                          np.asarray(got["scale"], np.float32).reshape(-1), side="left")
    rec["idx_inconsistent_with_own_scale"] = int((own != gi).sum())
    excused = near
    if bf16:
        # bf16: also where a level lies between the two scales (which agree to
        # the float bar), so that either side's decision is right; counted apart
        g = np.asarray(got["scale"], np.float64).reshape(-1)
        lo, hi = np.minimum(g, s), np.maximum(g, s)
        br = (np.searchsorted(t, hi, side="right") > np.searchsorted(t, lo, side="left")) & ~near
        rec["idx_mismatch_bracketed"] = int((mism & br).sum())
        excused = near | br
    rec["idx_mismatch_unexcused"] = int((mism & ~excused).sum())
    rec["within_bar"] = bool(all(v <= tol for v in errs.values()) and rec["idx_mismatch_unexcused"] == 0
                             and rec["idx_inconsistent_with_own_scale"] == 0)
    return rec


def cpu_baseline(name, rows, mask=None, group=1, precision="fp32", got=None):
    """Time the CPU oracle decoding the top `rows` grid rows of the same
    workload (the causal taps point up and left, so this is an exact decode of
    those latents).  With `got` (the timed decode's outputs, host arrays) the
    same oracle decode is also the parity reference of those rows; for bf16 the
    oracle's bf16 mode is run as well (the parity reference) and the distance
    to the fp32 oracle is reported beside it."""
    import oracle
    from paper_2607_19082_amd import inputs
    cfg, w, table, psi, sym = inputs.make_inputs(name)
    if mask:
        cfg["relaxed"] = mask == "relaxed"
        w = inputs.make_weights(cfg["M"], cfg["K"], radius=MASK_RADIUS[mask])
    psi, sym = psi[:, :rows].copy(), sym[:, :rows].copy()
    m = oracle.Model(w, table, rows, cfg["W"], cfg["B"], cfg["K"], relaxed=cfg["relaxed"], group=group)
    t0 = time.perf_counter()
    ref = m.decode(psi, sym)
    dt = time.perf_counter() - t0
    n = cfg["B"] * rows * cfg["W"]
    cpu = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    rec = {"value": n / dt, "unit": "latents/s", "cores": 1, "kind": "oracle",
           "sample": f"sequential raster decode (fp64 accumulate) of the top {rows} grid rows "
                     f"({n} latents) of {name}, one thread, {dt:.1f} s, on {cpu} "
                     f"({os.cpu_count()} logical cpus)",
           "ms_per_image_extrapolated": dt * 1e3 * (cfg["H"] / rows)}
    par = None
    if got is not None:
        top = {k: v[:, :rows] for k, v in got.items()}
        if precision == "bf16":
            mb = oracle.Model(w, table, rows, cfg["W"], cfg["B"], cfg["K"], relaxed=cfg["relaxed"], group=group,
                              bf16=True)
            par = parity_record(top, mb.decode(psi, sym), table, 1e-3, bf16=True)
            par["reference"] = "the oracle's bf16 mode (bf16 weights, bf16-pair activations)"
            par["max_abs_vs_fp32_oracle"] = parity_record(top, ref, table, 1e-2, bf16=True)["max_abs_err"]
        else:
            par = parity_record(top, ref, table, 1e-4)
            par["reference"] = "the oracle (fp64 accumulation)"
        par["latents"] = n
        par["rows"] = f"top {rows} grid rows of the last timed decode"
    return rec, par


# bin edges of the per-step latency histograms, in multiples of L_floor
HIST_EDGES = (0, 1, 2, 4, 8, 16, 32, 64, float("inf"))


def latency_histogram(us, lfloor):
    """Per-step latencies (microseconds) against the latency floor L_floor:
    percentiles, and counts in bins of [a, b) x L_floor."""
    us = np.asarray(us, dtype=np.float64)
    x = us / lfloor
    counts = [int(((x >= a) & (x < b)).sum()) for a, b in zip(HIST_EDGES[:-1], HIST_EDGES[1:])]
    pct = (0, 10, 50, 90, 99, 100)
    return {"L_floor_us": lfloor, "steps": int(us.size), "sum_ms": float(us.sum()) / 1e3,
            "percentiles_us": {f"p{q}": round(float(v), 3) for q, v in zip(pct, np.percentile(us, pct))},
            "median_over_L_floor": round(float(np.median(x)), 2),
            "bins_in_L_floor": [f"[{a:g}, {b:g})" for a, b in zip(HIST_EDGES[:-1], HIST_EDGES[1:])],
            "counts": counts}


def histogram_table(h, what):
    lines = [f"| {what} | " + " | ".join(h["bins_in_L_floor"]) + " |",
             "|---|" + "---|" * len(h["counts"]),
             "| steps | " + " | ".join(str(c) for c in h["counts"]) + " |"]
    p = h["percentiles_us"]
    lines += ["", f"{h['steps']} steps, {h['sum_ms']:.3f} ms in all; percentiles (us): "
              + ", ".join(f"{k} {v:.2f}" for k, v in p.items())
              + f"; median {h['median_over_L_floor']:.1f} x L_floor ({h['L_floor_us']:.2f} us)."]
    return lines


def trace_step_latency(trace_csv, call, T, lfloor):
    """Per-step latencies of decode call number `call` (0-based, in launch
    order) in a rocprofv3 kernel trace of the graph or stream driver: its
    phase kernels, in launch order, are an equal number per step for its T
    steps; a step's busy time is the sum of its phase kernels' durations, its
    span the time from the start of its first phase kernel to the start of the
    next step's (the last: to its last kernel's end), gaps included."""
    import csv
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    calls = [i for i, r in enumerate(rows) if "wf::k_set_call" in r["Kernel_Name"]]
    if call >= len(calls):
        return None
    ph = []
    for r in rows[calls[call] + 1:]:
        k = r["Kernel_Name"]
        if "wf::k_set_call" in k:
            break
        if "wf::k_phase" in k:
            ph.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    if not ph or len(ph) % T:
        return None
    s = np.array([a for a, _ in ph], dtype=np.float64).reshape(T, -1)
    e = np.array([b for _, b in ph], dtype=np.float64).reshape(T, -1)
    busy = (e - s).sum(1) / 1e3
    span = np.diff(np.append(s[:, 0], e[-1, -1])) / 1e3
    return latency_histogram(busy, lfloor), latency_histogram(span, lfloor)


def persistent_step_latency(w, table, cfg, precision, psi_d, sym_d, lfloor, torch, wf):
    """Per-step latencies of one decode by the persistent driver, from the
    device wall clock (100 MHz) that its trace hook records when workgroup 0
    leaves each device-wide barrier: steps begin at the release of the
    barrier before their first phase."""
    pp = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask_of(cfg), precision=precision,
                 driver="persistent")
    try:
        out = pp.alloc_out()
        needed, G = pp.trace(None)
        st = torch.zeros(needed, dtype=torch.int64, device="cuda")
        for _ in range(2):
            pp.decode(psi_d, sym_d, out=out)
        pp.sync()
        pp.trace(st)
        pp.decode(psi_d, sym_d, out=out)
        pp.sync()
        pp.trace(None)
        rel = st.cpu().numpy().reshape(-1, G + 1)[:, G].astype(np.float64)
    finally:
        pp.close()
    # two barriers before the first step, then one after each of a step's phases
    T = len(step_rows(cfg))
    phases = (rel.size - 2) // T
    assert rel.size == 2 + phases * T, (rel.size, T)
    starts = rel[1 + phases * np.arange(T + 1)]
    return latency_histogram(np.diff(starts) / 100.0, lfloor)


def resident_step_latency(w, table, cfg, precision, psi_d, sym_d, lfloor, torch, wf):
    """Per-step latencies of one decode by the resident driver, from the
    device wall clock (100 MHz) that its trace hook records per task and
    workgroup: a step is done when the last workgroup has published its part
    of the step's last task, and the latency of step t is the time from step
    t-1 done to step t done (the bands of a step overlap the steps around it,
    so this is the rate at which steps complete, not one step's span)."""
    pr = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask_of(cfg), precision=precision,
                 driver="resident")
    try:
        out = pr.alloc_out()
        needed, G = pr.trace(None)
        st = torch.zeros(needed, dtype=torch.int64, device="cuda")
        for _ in range(2):
            pr.decode(psi_d, sym_d, out=out)
        pr.sync()
        pr.trace(st)
        pr.decode(psi_d, sym_d, out=out)
        pr.sync()
        pr.trace(None)
        ends = st.cpu().numpy().reshape(-1, G, 3)[:, :, 2].max(axis=1).astype(np.float64)
    finally:
        pr.close()
    # tasks of each step in the global order: (image, 16-row band) pairs
    # holding a latent of the step
    H, W, B = cfg["H"], cfg["W"], cfg["B"]
    lam = MASK_SHEAR[mask_of(cfg)]
    T = W + lam * (H - 1)
    ntask = []
    for t in range(T):
        i0, i1 = max(0, -(-(t - W + 1) // lam)), min(H - 1, t // lam)
        ntask.append(B * (i1 // 16 - i0 // 16 + 1))
    assert sum(ntask) == ends.size, (sum(ntask), ends.size)
    kb = np.concatenate([[0], np.cumsum(ntask)])
    done = np.maximum.accumulate(np.array([ends[kb[t]:kb[t + 1]].max() for t in range(T)]))
    return latency_histogram(np.diff(done) / 100.0, lfloor)


def timed_calls(fn, steps, stream, torch):
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, [a.elapsed_time(b) for a, b in ev]


GMM_WORKLOAD = "cheng-gmm3-1080p-120x68-m192"


def entropy_leg(cfg, w, table, psi_d, sym, mask, precision, driver, steps, stream, torch, wf, inputs):
    """Time the decode that reads every symbol from its rANS stream (and the
    stream encoder) on one workload; the streams are those of an encode whose
    symbols are `sym`, and again of one whose symbols lie in {-1, 0, 1}."""
    pe = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask, precision=precision, driver=driver,
                 entropy_coder="rans")
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    bits = torch.zeros((2 + 4 * cfg["W"]) * cfg["B"] * cfg["H"] * cfg["M"], dtype=torch.int32, device="cuda")
    out_b = pe.alloc_out()
    sym_b = torch.empty(sym.shape, dtype=torch.int32, device="cuda")

    def measure(sym_np):
        # encoder input whose symbols are sym_np, then the timed decodes from its streams
        s_d = torch.from_numpy(sym_np).cuda()
        m = pe.decode(psi_d, s_d, stream=stream)["mean"]
        y_d = (torch.from_numpy(sym_np.astype(np.float32) + u).cuda() + m).contiguous()
        _, sym_e, offs = pe.encode_bits(psi_d, y_d, bits, stream=stream)
        pe.sync(stream)
        n_words = int(offs[-1].item())
        n_enc = max(3, steps // 4)
        ewall, _ = timed_calls(lambda: pe.encode_bits(psi_d, y_d, bits, stream=stream), n_enc, stream, torch)
        pe.sync(stream)

        def dec_bits():
            pe.decode_bits(psi_d, bits, offs, out=out_b, sym_out=sym_b, n_words=n_words, stream=stream)

        dec_bits()
        pe.sync(stream)
        bwall, bper = timed_calls(dec_bits, steps, stream, torch)
        pe.sync(stream)
        return {"ms_per_image": bwall * 1e3 / steps / cfg["B"], "launch_ms_events": float(np.mean(bper)),
                "encode_bits_ms_per_image": ewall * 1e3 / n_enc / cfg["B"],
                "stream_words": n_words, "bits_per_symbol": 32.0 * n_words / sym_np.size,
                "symbols_match": bool(torch.equal(sym_b, s_d)) and bool(torch.equal(sym_e, s_d))}

    rec = measure(sym)
    # symbols in {-1, 0, 1} lie inside every latent's coded symbols: no escapes
    rec["no_escapes"] = measure(np.clip(sym, -1, 1).astype(np.int32))
    rec["driver"] = driver
    rec["streams"] = ("one per (image, grid row, channel); 64-bit rANS state, 32-bit words, "
                      + ("2^-16 Gaussian tables per scale level" if cfg["K"] == 1 else
                         "2^-16 mixture frequencies per latent from quantised weights, offsets and scale levels")
                      + "; the workload's symbols do not follow the random model, so many of them escape")
    pe.close()
    del bits
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--driver", default=None, choices=["stream", "graph", "persistent", "dataflow", "resident"],
                    help="decode driver (default: resident; graph for --group > 1)")
    ap.add_argument("--precision", default="fp32", choices=["fp32", "bf16"])
    ap.add_argument("--mask", default=None, choices=sorted(MASK_TAPS),
                    help="causal mask (default: the workload's own), weights drawn for its kernel size")
    ap.add_argument("--group", type=int, default=1,
                    help="context approximation: decode N wavefronts per step (1: exact decode)")
    ap.add_argument("--cpu-rows", type=int, default=16, help="grid rows of the CPU-oracle sample (0: skip)")
    ap.add_argument("--no-encode", action="store_true")
    ap.add_argument("--no-transforms", action="store_true",
                    help="skip the hyper-decoder and synthesis timing (end-to-end decode)")
    ap.add_argument("--no-step-latency", action="store_true",
                    help="skip the per-step latency histogram (one traced decode by the resident driver when it "
                         "is the one timed, else by the persistent driver)")
    ap.add_argument("--no-entropy", action="store_true",
                    help="skip the decode from rANS streams (measured by default when the plan allows it)")
    ap.add_argument("--summarize-traffic", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="write the traffic summary of this workload/precision/driver from rocprofv3 outputs")
    ap.add_argument("--cal-bytes", type=float, default=float(1 << 30))
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only the plain copy of --cal-bytes that calibrates FETCH_SIZE / WRITE_SIZE")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS_DIR", "BENCH_LOG"),
                    help="write the kernel-statistics summary of this workload/precision/driver/group from a "
                         "rocprofv3 --kernel-trace --stats run of bench.py and its output")
    ap.add_argument("--summarize-counters", nargs="+", metavar="PMC_DIR",
                    help="write the MFMA-utilisation / L2-hit summary of this workload/precision/driver "
                         "from rocprofv3 --pmc outputs (MfmaUtil; TCC_HIT_sum TCC_MISS_sum)")
    ap.add_argument("--l-floor-us", type=float, default=None,
                    help="latency floor of an unprofiled bench run for --summarize-stats' step histograms")
    ap.add_argument("--command", default="", help="the commands that made the counter outputs (recorded)")
    args = ap.parse_args()
    driver_given = args.driver is not None
    if args.driver is None:
        args.driver = "resident" if args.group <= 1 else "graph"
    if args.copy_calibration:
        copy_calibration(args.cal_bytes)
        return
    if args.summarize_stats:
        g = f"_g{args.group}" if args.group > 1 else ""
        mk = f"_mask{args.mask}" if args.mask else ""
        summarize_stats(*args.summarize_stats,
                        os.path.join(PROFILES, f"kernels_{args.workload}_{args.precision}_{args.driver}{mk}{g}.md"),
                        args.command, args.l_floor_us)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters,
                           os.path.join(PROFILES, f"counters_{args.workload}_{args.precision}_{args.driver}.md"),
                           args.command, args.driver)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args.cal_bytes,
                          traffic_file(args.workload, args.precision, args.driver), args.command, args.driver)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py runs the decode on one GPU only (--gpus 1); a multi-GPU run is not "
                                   "part of it"}))
        sys.exit(2)

    import torch
    from paper_2607_19082_amd import inputs, wf

    assert torch.cuda.is_available(), "bench needs a GPU"
    torch.cuda.set_device(0)
    cfg, w, table, psi, sym = inputs.make_inputs(args.workload)
    own_mask = args.mask is None or args.mask == mask_of(cfg)
    if args.mask:
        cfg["mask"] = args.mask
        cfg["relaxed"] = args.mask == "relaxed"
        w = inputs.make_weights(cfg["M"], cfg["K"], radius=MASK_RADIUS[args.mask])
    try:
        plan = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask_of(cfg), precision=args.precision,
                       driver=args.driver, group=args.group)
    except wf.WfError as e:
        # the resident driver refuses plans whose weight slices exceed its
        # registers (e.g. the 7x7 mask at M = 320): by default, the graph driver
        if driver_given or e.code != wf.WF_E_UNSUPPORTED:
            raise
        args.driver = "graph"
        plan = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask_of(cfg), precision=args.precision,
                       driver=args.driver, group=args.group)
    psi_d = torch.from_numpy(psi).cuda()
    sym_d = torch.from_numpy(sym).cuda()
    out = plan.alloc_out()
    stream = torch.cuda.current_stream()

    def dec():
        plan.decode(psi_d, sym_d, out=out, stream=stream)

    for _ in range(args.warmup):
        dec()
    plan.sync(stream)
    wall, per = timed_calls(dec, args.steps, stream, torch)
    plan.sync(stream)

    rec_enc = None
    if not args.no_encode:
        u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
        y_d = (torch.from_numpy(sym.astype(np.float32) + u).cuda() + out["mean"]).contiguous()
        out_e = plan.alloc_out()
        sym_o = torch.empty_like(sym_d)

        def enc():
            plan.encode(psi_d, y_d, out=out_e, sym_out=sym_o, stream=stream)

        enc()
        plan.sync(stream)
        ewall, eper = timed_calls(enc, max(3, args.steps // 4), stream, torch)
        plan.sync(stream)
        rec_enc = {"ms_per_image": ewall * 1e3 / max(3, args.steps // 4) / cfg["B"],
                   "symbols_match_decode": bool(torch.equal(sym_o, sym_d))}

    # the last timed decode's top grid rows, for the parity record of the CPU-baseline leg
    got_host = {k: v[:, :args.cpu_rows].cpu().numpy() for k, v in out.items()} if args.cpu_rows > 0 else None
    node_us, bar_us = plan.measure_floor()
    plan.close()
    lfloor = min(x for x in (node_us, bar_us) if x > 0)

    rec_hist = None
    if not args.no_step_latency and args.group <= 1 and args.driver == "resident":
        rec_hist = {"driver": "resident (device clock per task and workgroup; a step's latency is the time "
                              "between the completions of consecutive steps)",
                    **resident_step_latency(w, table, cfg, args.precision, psi_d, sym_d, lfloor, torch, wf)}
    elif not args.no_step_latency and args.group <= 1:
        rec_hist = {"driver": "persistent (device clock at each device-wide barrier; the graph driver's "
                              "histogram is in its committed kernel-trace summary)",
                    **persistent_step_latency(w, table, cfg, args.precision, psi_d, sym_d, lfloor, torch, wf)}

    # the decode that reads every symbol from its rANS stream inside the step
    # loop (on the per-step kernels: the graph driver unless stream is timed),
    # for this workload and, when it is another, the 3-component mixture
    # model at 1080p
    rec_ec = rec_ec_gmm = None
    if not args.no_entropy and args.group <= 1:
        ec_driver = "stream" if args.driver == "stream" else "graph"
        rec_ec = entropy_leg(cfg, w, table, psi_d, sym, mask_of(cfg), args.precision, ec_driver, args.steps, stream,
                             torch, wf, inputs)
        if cfg["K"] == 1:
            g_cfg, g_w, g_table, g_psi, g_sym = inputs.make_inputs(GMM_WORKLOAD)
            g_psi_d = torch.from_numpy(g_psi).cuda()
            rec_ec_gmm = entropy_leg(g_cfg, g_w, g_table, g_psi_d, g_sym, mask_of(g_cfg), args.precision, ec_driver,
                                     args.steps, stream, torch, wf, inputs)
            # the same workload's decode from symbols, for comparison
            gp = wf.Plan(g_w, g_table, g_cfg["H"], g_cfg["W"], g_cfg["B"], g_cfg["K"], mask=mask_of(g_cfg),
                         precision=args.precision, driver=args.driver)
            g_out = gp.alloc_out()
            g_sym_d = torch.from_numpy(g_sym).cuda()
            gp.decode(g_psi_d, g_sym_d, out=g_out, stream=stream)
            gp.sync(stream)
            gwall, _ = timed_calls(lambda: gp.decode(g_psi_d, g_sym_d, out=g_out, stream=stream), args.steps, stream,
                                   torch)
            gp.sync(stream)
            gp.close()
            rec_ec_gmm["workload"] = GMM_WORKLOAD
            rec_ec_gmm["decode_from_symbols_ms_per_image"] = gwall * 1e3 / args.steps / g_cfg["B"]
            rec_ec_gmm["decode_from_symbols_driver"] = args.driver

    # the transforms around the decode: hyper-decoder (z_hat -> psi) and
    # synthesis (y_hat -> image), random weights, for an end-to-end timing
    rec_e2e = None
    if not args.no_transforms and args.group <= 1:
        N = XFORM_N.get(cfg["M"], 192)
        xf = wf.Xform(inputs.make_transform_weights(N, cfg["M"]), N, cfg["M"], cfg["B"], cfg["H"], cfg["W"],
                      args.precision)
        z_d = torch.from_numpy(inputs.make_zhat(cfg["B"], -(-cfg["H"] // 4), -(-cfg["W"] // 4), N)).cuda()
        psi_x = torch.empty_like(psi_d)
        img = torch.empty((cfg["B"], 16 * cfg["H"], 16 * cfg["W"], 3), dtype=torch.float32, device="cuda")
        xf.hyper_synthesis(z_d, psi=psi_x, stream=stream)
        xf.synthesis(out["y_hat"], image=img, stream=stream)
        torch.cuda.synchronize()
        n_x = max(3, args.steps // 4)
        hwall, hper = timed_calls(lambda: xf.hyper_synthesis(z_d, psi=psi_x, stream=stream), n_x, stream, torch)
        gwall, gper = timed_calls(lambda: xf.synthesis(out["y_hat"], image=img, stream=stream), n_x, stream, torch)
        finite = bool(torch.isfinite(img).all().item()) and bool(torch.isfinite(psi_x).all().item())
        xf.close()
        hs_ms, gs_ms = hwall * 1e3 / n_x / cfg["B"], gwall * 1e3 / n_x / cfg["B"]
        dec_img_ms = wall * 1e3 / args.steps / cfg["B"]
        rec_e2e = {"hyper_decoder_ms_per_image": hs_ms, "synthesis_ms_per_image": gs_ms,
                   "ar_decode_ms_per_image": dec_img_ms, "ms_per_image": hs_ms + dec_img_ms + gs_ms,
                   "N": N, "outputs_finite": finite,
                   "synthesis_gflop": synthesis_flops(N, cfg["M"], cfg["B"] * cfg["H"] * cfg["W"]) / 1e9,
                   "hyper_decoder_gflop": hyper_flops(N, cfg["M"], cfg["B"] * cfg["H"] * cfg["W"]) / 1e9}
        if rec_ec is not None:
            rec_e2e["ms_per_image_with_entropy_decode"] = hs_ms + rec_ec["ms_per_image"] + gs_ms
        del img

    lat = cfg["B"] * cfg["H"] * cfg["W"]
    ms = wall * 1e3 / args.steps
    value = lat / (ms * 1e-3)
    fl = flops_per_latent(cfg) * lat
    dec_ms = float(np.mean(per))
    peak = PEAK_TFLOPS[args.precision]
    achieved = fl / (dec_ms * 1e-3) / 1e12
    rows = step_rows(cfg, args.group)
    # the committed counter summaries cover the exact decode with the workload's own mask only
    traffic = read_traffic(args.workload, args.precision, args.driver) if args.group == 1 and own_mask else None
    f_step = rows * (flops_per_latent(cfg) - hoistable_flops_per_latent(cfg))
    t_roof_s = (hoistable_flops_per_latent(cfg) * lat) / (peak * 1e12) + np.maximum(
        f_step / (peak * 1e12), lfloor * 1e-6).sum()
    T = len(rows)
    rec = {
        "metric": "latents/s of a whole-image wavefront decode (ms per image = ms_per_step)",
        "value": value,
        "unit": "latents/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "paper_context": ("the paper reports more than 13x speed-up of encode plus decode from the wavefront "
                          "order alone over raster order (more than 26x with its tensorized rANS), with trained "
                          "weights on an RTX 3080 with an i7-8700K host (Table I); other hardware, context only"),
        "dtype": "f32" if args.precision == "fp32" else "bf16 operands, f32 accumulate",
        "data": "synthetic (seeded N(0,1/fan_in) weights, N(0,1) hyperprior params, Laplace symbols)",
        "config": {"workload": args.workload, "H": cfg["H"], "W": cfg["W"], "M": cfg["M"],
                   "B": cfg["B"], "K": cfg["K"], "mask": mask_of(cfg),
                   "steps_T": T, "driver": args.driver, "precision": args.precision,
                   "context_approximation_group": args.group,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "traffic_unit": "HBM bytes per launch (one decode)",
                     "traffic_GBps": None if traffic is None else traffic / (dec_ms * 1e-3) / 1e9,
                     "kernel": {"persistent": "k_persistent (one launch = one decode)",
                                "dataflow": "one decode call: counter reset, hoist and one k_dataflow launch",
                                "resident": "one decode call: counter reset, hoist and one k_resident launch",
                                "graph": "one replay of the decode graph (hoist, context, one k_phase per phase)",
                                "stream": "all kernels of one decode call"}[args.driver],
                     "algorithmic_gflop_per_launch": fl / 1e9, "launch_ms_events": dec_ms,
                     "mfma_floor_ms": fl / (peak * 1e12) * 1e3},
        "latency_roofline": {"L_floor_us": lfloor, "graph_node_us": node_us, "barrier_round_us": bar_us,
                             "hops_per_step_algorithmic": 1, "T_roof_ms": t_roof_s * 1e3,
                             "frac": t_roof_s * 1e3 / dec_ms,
                             "T_mfma_over_T_meas": fl / (peak * 1e12) * 1e3 / dec_ms,
                             "T_L_floor_over_T_meas": T * lfloor * 1e-3 / dec_ms},
        "latents_per_s": value,
        "symbols_per_s": value * cfg["M"],
        "step_latency": rec_hist,
        "ms_per_image": ms / cfg["B"],
        "encode": rec_enc,
        "entropy_decode": rec_ec,
        "entropy_decode_gmm": rec_ec_gmm,
        "end_to_end": rec_e2e,
    }
    if args.cpu_rows > 0:
        rec["cpu_baseline"], rec["parity"] = cpu_baseline(args.workload, args.cpu_rows, args.mask, args.group,
                                                          args.precision, got_host)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
