"""GPU parity of the bf16 variant (bf16 weights, activations carried as bf16
hi+lo pairs, every product on bf16 MFMA with fp32 accumulation) against the
oracle's matching bf16 mode on the same seeded inputs.

Bars, as for fp32 but with the bf16 tolerance: means, scales and y_hat within
1e-3 absolute of the bf16 oracle's whole decode (and encode); the two evaluate
the same bf16 function in different summation orders, measured ~1e-4 apart,
and a single-rounded activation misses this bar by an order of magnitude
(tests/test_oracle.py).  Encode symbols bit-exact; scale indices identical
except scales within 1e-4 relative of a table level, and, counted apart,
where a level lies between the GPU's and the oracle's scales.  The wide grids
(40 x 120) put three row tiles on a wavefront; at the full 3840x2160 size the
oracle decodes the top 33 grid rows (an exact sub-decode, three row tiles of
the widest steps) and its per-latent function is evaluated on the GPU's own
reconstruction at sampled latents.  The distance to the fp32 oracle (the
effect of the bf16 weights, not of the kernels) is logged beside it.
"""
import sys

import numpy as np
import pytest

from paper_2607_19082_amd import inputs, wf

import oracle_refs
from gpu_helpers import (BF16_TOL, compare, gpu_plan, make_case, max_rows_per_step, oracle_model,
                         sample_latents, teacher_forced, to_np, top_rows_check)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

WIDE = [("cheng-gmm3-1080p-120x68-m192", 40, 120), ("minnen-hr-4k-240x135-m320", 40, 120)]
ROWS_4K = 33

if torch.cuda.is_available():
    oracle_refs.prefetch([("minnen-hr-4k-240x135-m320", None, None, None, ROWS_4K, True)]
                         + [(n, H, W, None, None, True) for n, H, W in WIDE]
                         + [(n, H, W, None, None, False) for n, H, W in WIDE])


@pytest.fixture(scope="module", autouse=True)
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wf.lib()  # fails loudly when the library is missing
    torch.cuda.set_device(0)
    return torch.device("cuda", 0)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def decode(cfg, w, table, psi, sym, driver):
    plan = gpu_plan(cfg, w, table, driver, "bf16")
    out = plan.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    plan.sync()
    res = to_np(out)
    plan.close()
    return res


def encode(cfg, w, table, psi, y, driver):
    plan = gpu_plan(cfg, w, table, driver, "bf16")
    out, s = plan.encode(torch.from_numpy(psi).cuda(), torch.from_numpy(y).cuda())
    plan.sync()
    res, s = to_np(out), s.cpu().numpy()
    plan.close()
    return res, s


def vs_fp32(cfg, w, table, psi, sym, got, ref=None):
    if ref is None:
        ref = oracle_model(cfg, w, table).decode(psi, sym)
    return {k: float(np.abs(got[k].astype(np.float64) - ref[k]).max()) for k in ("y_hat", "mean", "scale")}


SMALL = [
    ("minnen-16x16-m192", 7, 9, 1),
    ("minnen-16x16-m192", 5, 3, 2),
    ("cheng-gmm3-1080p-120x68-m192", 6, 11, 1),
    ("minnen-relaxed-b8-120x68-m192", 5, 7, 3),
    ("minnen-hr-4k-240x135-m320", 4, 10, 1),
]


@pytest.mark.parametrize("driver", ["stream", "graph", "persistent", "dataflow", "resident"])
@pytest.mark.parametrize("name,H,W,B", SMALL)
def test_bf16_small_decode_encode(name, H, W, B, driver):
    log(f"bf16 case {name} H={H} W={W} B={B} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    ref = oracle_model(cfg, w, table, bf16=True).decode(psi, sym)
    got = decode(cfg, w, table, psi, sym, driver)
    log(compare(got, ref, table, cfg["K"], tol=BF16_TOL))
    log({"max_abs_vs_fp32_oracle": vs_fp32(cfg, w, table, psi, sym, got)})
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    y = inputs.encoder_input(sym, u, ref["mean"])
    got_e, s = encode(cfg, w, table, psi, y, driver)
    assert np.array_equal(s, sym)
    log(compare(got_e, ref, table, cfg["K"], tol=BF16_TOL))


@pytest.mark.parametrize("driver", ["graph", "resident"])
def test_bf16_consecutive_calls_with_new_inputs(driver):
    # one plan, the same output buffers, decodes of two different symbol sets
    # in turn: no activation of an earlier call may be read as current data
    cfg, w, table, psi, sym = make_case("minnen-hr-4k-240x135-m320", H=9, W=20)
    sym2 = inputs.make_symbols(cfg["B"], cfg["H"], cfg["W"], cfg["M"], cfg["lap_b"], cfg["clip"], seed=7)
    model = oracle_model(cfg, w, table, bf16=True)
    refs = [model.decode(psi, s) for s in (sym, sym2)]
    plan = gpu_plan(cfg, w, table, driver, precision="bf16")
    out = plan.alloc_out()
    psi_d = torch.from_numpy(psi).cuda()
    for rep in range(2):
        for s, ref in zip((sym, sym2), refs):
            plan.decode(psi_d, torch.from_numpy(s).cuda(), out=out)
            plan.sync()
            log(compare(to_np(out), ref, table, cfg["K"], tol=BF16_TOL))
    plan.close()


@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
@pytest.mark.parametrize("name,H,W,B", [
    ("minnen-kodak-48x32-m192", 32, 48, 1),
    ("cheng-gmm3-1080p-120x68-m192", 14, 24, 1),
    ("minnen-relaxed-b8-120x68-m192", 9, 16, 8),
    ("minnen-hr-4k-240x135-m320", 9, 20, 1),
])
def test_bf16_reduced_global(name, H, W, B, driver):
    log(f"bf16 case {name} H={H} W={W} B={B} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    ref = oracle_model(cfg, w, table, bf16=True).decode(psi, sym)
    got = decode(cfg, w, table, psi, sym, driver)
    log(compare(got, ref, table, cfg["K"], tol=BF16_TOL))


@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
@pytest.mark.parametrize("name,H,W", WIDE)
def test_bf16_wide_global(name, H, W, driver):
    log(f"bf16 case {name} wide H={H} W={W} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W)
    assert max_rows_per_step(H, W, 3) == 40
    got = decode(cfg, w, table, psi, sym, driver)
    ref = oracle_refs.ref_decode(name, H, W, bf16=True).result()
    log(compare(got, ref, table, cfg["K"], tol=BF16_TOL))
    ref32 = oracle_refs.ref_decode(name, H, W).result()
    log({"max_abs_vs_fp32_oracle": vs_fp32(cfg, w, table, psi, sym, got, ref32)})
    if driver == "graph":
        u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
        y = inputs.encoder_input(sym, u, ref["mean"])
        got_e, s = encode(cfg, w, table, psi, y, driver)
        assert np.array_equal(s, sym)
        log(compare(got_e, ref, table, cfg["K"], tol=BF16_TOL))


@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
def test_bf16_4k_full_size(driver):
    # the 3840x2160 workload (240x135 latents, M = 320) at its full size: the
    # top rows against the bf16 oracle's decode of them, teacher-forced
    # sampled latents, and encode reproducing the symbols and y_hat
    name = "minnen-hr-4k-240x135-m320"
    log(f"bf16 case {name} full size driver={driver}")
    cfg, w, table, psi, sym = make_case(name)
    got = decode(cfg, w, table, psi, sym, driver)
    ref = oracle_refs.ref_decode(name, rows=ROWS_4K, bf16=True).result()
    log(top_rows_check(cfg, w, table, psi, sym, got, ROWS_4K, bf16=True, tol=BF16_TOL, ref=ref))
    model = oracle_model(cfg, w, table, bf16=True)
    log(teacher_forced(cfg, got, psi, sym, model, sample_latents(cfg, 300), table, tol=BF16_TOL))
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    y = inputs.encoder_input(sym, u, got["mean"])
    got_e, s = encode(cfg, w, table, psi, y, driver)
    mism = int((s != sym).sum())
    log({"encode_symbol_mismatches": mism})
    assert mism == 0
    assert np.array_equal(got_e["y_hat"], got["y_hat"])
