"""Benchmark: wavefront decode of one 3840x2160 image's latent (240x135, M=320)
through the C-ABI, on one GPU.

One step = one whole decode of the latent grid (every wavefront step: tap
gather, context product, entropy-parameter network, parameter epilogue and the
y_hat write).  Inputs are seeded synthetic arrays already resident in HBM.
Prints one JSON line.
"""
import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2500.0}


def flops_per_latent(cfg):
    """Algorithmic FLOPs of one latent: 2 x MACs of the context product over
    the causal taps and of the three network layers."""
    M, d1, d2, n3 = cfg["M"], cfg["d1"], cfg["d2"], cfg["n3"]
    taps = 10 if cfg["relaxed"] else 12
    macs = taps * M * 2 * M + 4 * M * d1 + d1 * d2 + d2 * n3
    return 2 * macs


def cpu_baseline(name, rows):
    """Time the CPU oracle decoding the top `rows` rows of the same workload
    (the AR dependencies point up and left, so this is an exact decode of
    those latents)."""
    import oracle
    from paper_2607_19082_amd import inputs
    cfg, w, table, psi, sym = inputs.make_inputs(name)
    psi, sym = psi[:, :rows].copy(), sym[:, :rows].copy()
    m = oracle.Model(w, table, rows, cfg["W"], cfg["B"], cfg["K"], relaxed=cfg["relaxed"])
    t0 = time.perf_counter()
    m.decode(psi, sym)
    dt = time.perf_counter() - t0
    n = cfg["B"] * rows * cfg["W"]
    return {"value": n / dt, "unit": "latents/s", "cores": 1, "kind": "oracle",
            "sample": f"sequential raster decode of the top {rows} rows ({n} latents) of {name}, "
                      f"single thread, {dt:.1f} s; host {platform.processor() or platform.machine()}, "
                      f"{os.cpu_count()} logical cpus"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="minnen-hr-4k-240x135-m320")
    ap.add_argument("--driver", default="graph", choices=["stream", "graph", "persistent"])
    ap.add_argument("--precision", default="fp32", choices=["fp32", "bf16"])
    ap.add_argument("--cpu-rows", type=int, default=8, help="rows of the CPU-oracle sample (0: skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    from paper_2607_19082_amd import inputs, wf

    assert torch.cuda.is_available(), "bench needs a GPU"
    torch.cuda.set_device(0)
    cfg, w, table, psi, sym = inputs.make_inputs(args.workload)
    plan = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"],
                   mask="relaxed" if cfg["relaxed"] else "full", precision=args.precision,
                   driver=args.driver)
    psi_d = torch.from_numpy(psi).cuda()
    sym_d = torch.from_numpy(sym).cuda()
    out = plan.alloc_out()
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        plan.decode(psi_d, sym_d, out=out, stream=stream)
    plan.sync(stream)

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        plan.decode(psi_d, sym_d, out=out, stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    plan.sync(stream)
    per = [a.elapsed_time(b) for a, b in ev]  # ms, HIP events on the launch stream

    lat = cfg["B"] * cfg["H"] * cfg["W"]
    ms = wall * 1e3 / args.steps
    value = lat / (ms * 1e-3)
    fl = flops_per_latent(cfg) * lat
    dec_ms = float(np.mean(per))
    achieved = fl / (dec_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[args.precision]
    T = cfg["W"] + (2 if cfg["relaxed"] else 3) * (cfg["H"] - 1)
    rec = {
        "metric": "latents/s of a whole-image wavefront decode (ms per image in ms_per_step)",
        "value": value,
        "unit": "latents/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.precision == "fp32" else "bf16 operands, f32 accumulate",
        "data": "synthetic (seeded N(0,1/fan_in) weights, N(0,1) hyperprior params, Laplace symbols)",
        "config": {"workload": args.workload, "H": cfg["H"], "W": cfg["W"], "M": cfg["M"],
                   "B": cfg["B"], "K": cfg["K"], "mask": "relaxed" if cfg["relaxed"] else "full",
                   "steps_T": T, "driver": args.driver, "precision": args.precision,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "whole decode (all step kernels, per decode call)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "algorithmic_gflop_per_decode": fl / 1e9, "decode_ms_events": dec_ms,
                     "mfma_floor_ms": fl / (peak * 1e12) * 1e3},
        "latents_per_s": value,
        "ms_per_image": ms / cfg["B"],
    }
    plan.close()
    if args.cpu_rows > 0:
        rec["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_rows)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
