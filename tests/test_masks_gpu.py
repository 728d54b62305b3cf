"""GPU parity for causal masks of other radii (Appendix A, Def. 1): the 3x3
mask (R = 1, shear 2) and the 7x7 mask (R = 3, shear 4), through the C-ABI
against the oracle's decode with the same (2R+1)x(2R+1) weights; and grids
narrower than a mask's shear, which every mask decodes in raster order (the
earliest-possible schedule there).

Every driver runs the exact decode and encode; the stream and graph drivers
also run the context-approximation decode (Sec. III-D).  The resident driver
refuses the 7x7 mask at M = 320 (its context slices would need more k-parts
than its registers and workgroup slots allow), which is checked too.  Bars as
for the 5x5 mask: floats within 1e-4 (fp32) or 1e-3 (bf16, against the
oracle's bf16 mode), encode symbols bit-exact, scale indices identical except
counted boundary cases.  At the 3840x2160 size the oracle decodes the top grid rows
(an exact sub-decode: taps lie at or above their latent's row) and its
per-latent function is evaluated on the GPU's own reconstruction at sampled
latents.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_19082_amd import inputs, wf

from gpu_helpers import BF16_TOL, FP32_TOL, compare, sample_latents, teacher_forced, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

RADIUS = {"3x3": 1, "7x7": 3, "full": 2, "relaxed": 2}
SHEAR = {"3x3": 2, "7x7": 4, "full": 3, "relaxed": 2}


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


def case(name, mask, H=None, W=None, B=None):
    """A workload's shapes and distributions with weights of the mask's size."""
    cfg, _, table, psi, sym = inputs.make_inputs(name, H=H, W=W, B=B)
    w = inputs.make_weights(cfg["M"], cfg["K"], radius=RADIUS[mask])
    return cfg, w, table, psi, sym


def model(cfg, w, table, bf16=False, group=1, H=None, mask=None):
    return oracle.Model(w, table, H or cfg["H"], cfg["W"], cfg["B"], cfg["K"], relaxed=mask == "relaxed", bf16=bf16,
                        group=group)


def plan(cfg, w, table, mask, driver, precision, group=1):
    return wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask=mask, precision=precision,
                   driver=driver, group=group)


def check_schedule(p, cfg, mask, group):
    step, n = p.schedule()
    lam = min(SHEAR[mask], cfg["W"])
    T = cfg["W"] + lam * (cfg["H"] - 1)
    assert n == -(-T // group)
    ii, jj = np.meshgrid(np.arange(cfg["H"]), np.arange(cfg["W"]), indexing="ij")
    assert np.array_equal(step, (lam * ii + jj) // group)


def decode_encode(cfg, w, table, psi, sym, mask, driver, precision, group):
    bf = precision == "bf16"
    tol = BF16_TOL if bf else FP32_TOL
    ref = model(cfg, w, table, bf, group, mask=mask).decode(psi, sym)
    p = plan(cfg, w, table, mask, driver, precision, group)
    check_schedule(p, cfg, mask, group)
    out = p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    p.sync()
    log(compare(to_np(out), ref, table, cfg["K"], tol=tol))
    y = inputs.encoder_input(sym, inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"]), ref["mean"])
    out_e, s = p.encode(torch.from_numpy(psi).cuda(), torch.from_numpy(y).cuda())
    p.sync()
    assert np.array_equal(s.cpu().numpy(), sym)
    log(compare(to_np(out_e), ref, table, cfg["K"], tol=tol))
    p.close()


SMALL = [
    # (workload, H, W, B): ragged grids (at most 16 rows, one row tile, per step)
    ("minnen-16x16-m192", 7, 9, 1),
    ("cheng-gmm3-1080p-120x68-m192", 6, 11, 1),
    ("minnen-hr-4k-240x135-m320", 4, 10, 2),
]


def resident_refuses(cfg, mask):
    return mask == "7x7" and cfg["M"] == 320


@pytest.mark.parametrize("driver", ["stream", "graph", "persistent", "dataflow", "resident"])
@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("mask", ["3x3", "7x7"])
@pytest.mark.parametrize("name,H,W,B", SMALL)
def test_mask_small(name, H, W, B, mask, precision, driver):
    log(f"mask case {name} H={H} W={W} B={B} mask={mask} precision={precision} driver={driver}")
    cfg, w, table, psi, sym = case(name, mask, H, W, B)
    if driver == "resident" and resident_refuses(cfg, mask):
        with pytest.raises(wf.WfError) as e:
            plan(cfg, w, table, mask, driver, precision)
        assert e.value.code == wf.WF_E_UNSUPPORTED and "resident" in str(e.value)
        return
    decode_encode(cfg, w, table, psi, sym, mask, driver, precision, 1)


@pytest.mark.parametrize("N", [2, 3])
@pytest.mark.parametrize("driver", ["stream", "graph"])
@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("mask", ["3x3", "7x7"])
@pytest.mark.parametrize("name,H,W,B", SMALL[1:])
def test_mask_grouped_small(name, H, W, B, mask, precision, driver, N):
    log(f"mask grouped case {name} H={H} W={W} B={B} mask={mask} precision={precision} driver={driver} N={N}")
    cfg, w, table, psi, sym = case(name, mask, H, W, B)
    decode_encode(cfg, w, table, psi, sym, mask, driver, precision, N)


def test_mask_grid_as_wide_as_the_shear():
    for mask in ("3x3", "7x7"):
        lam = SHEAR[mask]
        log(f"mask case W={lam} mask={mask}")
        cfg, w, table, psi, sym = case("minnen-16x16-m192", mask, 6, lam, 2)
        decode_encode(cfg, w, table, psi, sym, mask, "graph", "fp32", 1)


@pytest.mark.parametrize("driver", ["stream", "graph", "persistent", "dataflow", "resident"])
@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("mask", ["full", "relaxed", "3x3", "7x7"])
def test_grid_narrower_than_the_shear(mask, precision, driver):
    """Every W below the shear: one latent per image and step, raster order."""
    for W in range(1, SHEAR[mask]):
        log(f"narrow case W={W} mask={mask} precision={precision} driver={driver}")
        cfg, w, table, psi, sym = case("cheng-gmm3-1080p-120x68-m192", mask, 5, W, 2)
        decode_encode(cfg, w, table, psi, sym, mask, driver, precision, 1)


@pytest.mark.parametrize("mask,precision,N", [("7x7", "fp32", 1), ("7x7", "bf16", 1), ("3x3", "fp32", 1),
                                              ("7x7", "fp32", 8)])
def test_mask_4k_full_size(mask, precision, N):
    name, rows, n = "minnen-hr-4k-240x135-m320", 5, 300
    log(f"mask case {name} full size mask={mask} precision={precision} N={N}: top {rows} rows + {n} teacher-forced")
    cfg, w, table, psi, sym = case(name, mask)
    bf = precision == "bf16"
    tol = BF16_TOL if bf else FP32_TOL
    p = plan(cfg, w, table, mask, "graph", precision, N)
    out = p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    p.sync()
    got = to_np(out)
    p.close()
    top = model(cfg, w, table, bf, N, H=rows).decode(psi[:, :rows].copy(), sym[:, :rows].copy())
    log(compare({k: v[:, :rows] for k, v in got.items()}, top, table, cfg["K"], tol=tol))
    lats = sample_latents(cfg, n)
    log(teacher_forced(cfg, got, psi, sym, model(cfg, w, table, bf, N), lats, table, tol=tol))
