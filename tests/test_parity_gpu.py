"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle on the
same seeded inputs.

Global parity compares every output of a whole decode (and encode) with the
oracle's sequential raster decode.  The "wide" grids (40 x 120 latents) put 40
latents on a wavefront, three 16-row tiles, at K = 3 and at M = 320.  At the
full workload sizes the oracle decodes the top grid rows (an exact
sub-decode: every tap lies in the latent's row or above); for the 4K workload
65 rows, so that all five row tiles of its widest steps are compared element
by element.  In addition the oracle's per-latent function is evaluated on the
GPU's own final reconstruction at sampled latents (teacher-forced), which also
catches any tap read before it was written.  The oracle references are
computed on host threads while the GPU tests run (oracle_refs).
Bars: 1e-4 absolute on floats; symbols bit-exact; scale indices identical
except scales within 1e-4 relative of a table level (counted).
"""
import sys

import numpy as np
import pytest

from paper_2607_19082_amd import inputs, wf

import oracle_refs
from gpu_helpers import (compare, gpu_plan, make_case, max_rows_per_step, oracle_model, sample_latents,
                         teacher_forced, to_np, top_rows_check)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

WIDE = [
    # (workload, H, W): 40 latents per wavefront, three 16-row tiles per step
    ("cheng-gmm3-1080p-120x68-m192", 40, 120),
    ("minnen-hr-4k-240x135-m320", 40, 120),
]
TOP_ROWS = {"cheng-gmm3-1080p-120x68-m192": 20, "minnen-relaxed-b8-120x68-m192": 3,
            "minnen-hr-4k-240x135-m320": 65}

if torch.cuda.is_available():
    oracle_refs.prefetch([("minnen-hr-4k-240x135-m320", None, None, None, 65, False)]
                         + [(n, H, W, None, None, False) for n, H, W in WIDE]
                         + [(n, None, None, None, r, False) for n, r in TOP_ROWS.items()])


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


def run_decode(cfg, w, table, psi, sym, driver="stream", precision="fp32"):
    plan = gpu_plan(cfg, w, table, driver, precision)
    psi_d = torch.from_numpy(psi).cuda()
    sym_d = torch.from_numpy(sym).cuda()
    out = plan.decode(psi_d, sym_d)
    plan.sync()
    res = to_np(out)
    plan.close()
    return res


def run_encode(cfg, w, table, psi, y, driver="stream", precision="fp32"):
    plan = gpu_plan(cfg, w, table, driver, precision)
    out, s = plan.encode(torch.from_numpy(psi).cuda(), torch.from_numpy(y).cuda())
    plan.sync()
    res, s = to_np(out), s.cpu().numpy()
    plan.close()
    return res, s


SMALL = [
    # (workload, H, W, B): ragged grids, at most 16 latents per wavefront
    # (one row tile; the wide cases below span three)
    ("minnen-16x16-m192", 7, 9, 1),
    ("minnen-16x16-m192", 5, 3, 2),
    ("cheng-gmm3-1080p-120x68-m192", 6, 11, 1),
    ("minnen-relaxed-b8-120x68-m192", 5, 7, 3),
    ("minnen-hr-4k-240x135-m320", 4, 10, 1),
]


DRIVERS = ["stream", "graph", "persistent", "dataflow", "resident"]


@pytest.mark.parametrize("driver", DRIVERS)
@pytest.mark.parametrize("name,H,W,B", SMALL)
def test_small_decode_encode(name, H, W, B, driver):
    log(f"case {name} H={H} W={W} B={B} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    model = oracle_model(cfg, w, table)
    ref = model.decode(psi, sym)
    got = run_decode(cfg, w, table, psi, sym, driver)
    log(compare(got, ref, table, cfg["K"]))
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    y = inputs.encoder_input(sym, u, ref["mean"])
    got_e, s = run_encode(cfg, w, table, psi, y, driver)
    assert np.array_equal(s, sym)
    log(compare(got_e, ref, table, cfg["K"]))


@pytest.mark.parametrize("driver", DRIVERS)
@pytest.mark.parametrize("name", ["minnen-16x16-m192", "minnen-kodak-48x32-m192"])
def test_full_decode_encode(name, driver):
    log(f"case {name} full size driver={driver}")
    cfg, w, table, psi, sym = make_case(name)
    model = oracle_model(cfg, w, table)
    ref = model.decode(psi, sym)
    got = run_decode(cfg, w, table, psi, sym, driver)
    log(compare(got, ref, table, cfg["K"]))
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    y = inputs.encoder_input(sym, u, ref["mean"])
    got_e, s = run_encode(cfg, w, table, psi, y, driver)
    assert np.array_equal(s, sym)
    log(compare(got_e, ref, table, cfg["K"]))


@pytest.mark.parametrize("name,H,W,B", [
    ("cheng-gmm3-1080p-120x68-m192", 14, 24, 1),
    ("minnen-relaxed-b8-120x68-m192", 9, 16, 8),
    ("minnen-hr-4k-240x135-m320", 9, 20, 1),
])
@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
def test_reduced_global(name, H, W, B, driver):
    log(f"case {name} reduced H={H} W={W} B={B} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    ref = oracle_model(cfg, w, table).decode(psi, sym)
    got = run_decode(cfg, w, table, psi, sym, driver)
    log(compare(got, ref, table, cfg["K"]))


@pytest.mark.parametrize("name,H,W", WIDE)
@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
def test_wide_global(name, H, W, driver):
    # every output of a decode whose wavefronts span three row tiles
    log(f"case {name} wide H={H} W={W} driver={driver}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W)
    assert max_rows_per_step(H, W, 3) == 40
    got = run_decode(cfg, w, table, psi, sym, driver)
    ref = oracle_refs.ref_decode(name, H, W).result()
    log(compare(got, ref, table, cfg["K"]))
    if driver == "graph":
        u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
        y = inputs.encoder_input(sym, u, ref["mean"])
        got_e, s = run_encode(cfg, w, table, psi, y, driver)
        assert np.array_equal(s, sym)
        log(compare(got_e, ref, table, cfg["K"]))


@pytest.mark.parametrize("name,n", [
    ("cheng-gmm3-1080p-120x68-m192", 600),
    ("minnen-relaxed-b8-120x68-m192", 600),
    ("minnen-hr-4k-240x135-m320", 300),
])
@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
def test_full_size_teacher_forced(name, n, driver):
    rows = TOP_ROWS[name]
    log(f"case {name} full size, top {rows} rows + teacher-forced sample of {n}, driver={driver}")
    cfg, w, table, psi, sym = make_case(name)
    got = run_decode(cfg, w, table, psi, sym, driver)
    ref = oracle_refs.ref_decode(name, rows=rows).result()
    log(top_rows_check(cfg, w, table, psi, sym, got, rows, ref=ref))
    model = oracle_model(cfg, w, table)
    lats = sample_latents(cfg, n)
    log(teacher_forced(cfg, got, psi, sym, model, lats, table))


def test_graph_replays_match_and_reuse_plan():
    # one graph plan, several calls with different buffers and both
    # directions, with eager work and syncs in between: every replay must
    # match the oracle
    cfg, w, table, psi, sym = make_case("minnen-16x16-m192", H=6, W=8, B=1)
    model = oracle_model(cfg, w, table)
    ref = model.decode(psi, sym)
    plan = gpu_plan(cfg, w, table, "graph")
    psi_d = torch.from_numpy(psi).cuda()
    sym_d = torch.from_numpy(sym).cuda()
    u = inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    y_d = torch.from_numpy(inputs.encoder_input(sym, u, ref["mean"])).cuda()
    for it in range(3):
        out = plan.decode(psi_d, sym_d)
        plan.sync()
        compare(to_np(out), ref, table, cfg["K"])
        junk = torch.randn(1000, device="cuda").sum().item()  # eager work between replays
        assert np.isfinite(junk)
        out_e, s = plan.encode(psi_d, y_d)
        plan.sync()
        assert np.array_equal(s.cpu().numpy(), sym)
        compare(to_np(out_e), ref, table, cfg["K"])
    plan.close()


@pytest.mark.parametrize("driver", ["graph", "persistent", "dataflow", "resident"])
def test_consecutive_calls_with_new_inputs(driver):
    # one plan, the same output buffers, two decodes of different symbols
    # (and an encode in between): nothing of an earlier call may be read back
    # as current data by a later one
    cfg, w, table, psi, sym = make_case("minnen-hr-4k-240x135-m320", H=9, W=20)
    sym2 = inputs.make_symbols(cfg["B"], cfg["H"], cfg["W"], cfg["M"], cfg["lap_b"], cfg["clip"], seed=7)
    model = oracle_model(cfg, w, table)
    refs = [model.decode(psi, s) for s in (sym, sym2)]
    plan = gpu_plan(cfg, w, table, driver)
    out = plan.alloc_out()
    psi_d = torch.from_numpy(psi).cuda()
    for rep in range(2):
        for s, ref in zip((sym, sym2), refs):
            plan.decode(psi_d, torch.from_numpy(s).cuda(), out=out)
            plan.sync()
            log(compare(to_np(out), ref, table, cfg["K"]))
        y = inputs.encoder_input(sym, inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"]), refs[0]["mean"])
        _, s_out = plan.encode(psi_d, torch.from_numpy(y).cuda(), out=out)
        plan.sync()
        assert np.array_equal(s_out.cpu().numpy(), sym)
    plan.close()
