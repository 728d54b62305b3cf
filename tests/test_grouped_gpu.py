"""GPU parity of the context-approximation decode (Sec. III-D, Fig. 3):
groups of N wavefronts decoded as one step, same-group taps filled with the
mean of the decoded taps, through the C-ABI against the oracle's grouped
decode on the same seeded inputs.

Bars as for the exact decode: floats within 1e-4 (fp32) or 1e-2 (bf16, against
the oracle's bf16 mode), encode symbols bit-exact, scale indices identical
except counted boundary cases.  At the 3840x2160 size the oracle decodes the
top grid rows (taps and groups depend only on rows at or above a latent, so
this is an exact sub-decode) and its per-latent function is evaluated on the
GPU's own reconstruction at sampled latents.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_19082_amd import inputs, wf

from gpu_helpers import BF16_TOL, FP32_TOL, compare, make_case, sample_latents, teacher_forced, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


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


def model(cfg, w, table, N, bf16=False, H=None):
    return oracle.Model(w, table, H or cfg["H"], cfg["W"], cfg["B"], cfg["K"], relaxed=cfg["relaxed"],
                        bf16=bf16, group=N)


def plan(cfg, w, table, N, driver, precision):
    return wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], mask="relaxed" if cfg["relaxed"] else "full",
                   precision=precision, driver=driver, group=N)


SMALL = [
    ("minnen-16x16-m192", 7, 9, 1),
    ("cheng-gmm3-1080p-120x68-m192", 6, 11, 1),
    ("minnen-relaxed-b8-120x68-m192", 5, 7, 3),
    ("minnen-hr-4k-240x135-m320", 4, 10, 1),
]


@pytest.mark.parametrize("N", [2, 3, 4])
@pytest.mark.parametrize("driver", ["stream", "graph"])
@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name,H,W,B", SMALL)
def test_grouped_small(name, H, W, B, driver, precision, N):
    log(f"grouped case {name} H={H} W={W} B={B} N={N} driver={driver} precision={precision}")
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    bf = precision == "bf16"
    tol = BF16_TOL if bf else FP32_TOL
    m = model(cfg, w, table, N, bf)
    ref = m.decode(psi, sym)
    p = plan(cfg, w, table, N, driver, precision)
    step, n = p.schedule()
    lam = 2 if cfg["relaxed"] else 3
    T = cfg["W"] + lam * (cfg["H"] - 1)
    assert n == -(-T // N)
    ii, jj = np.meshgrid(np.arange(cfg["H"]), np.arange(cfg["W"]), indexing="ij")
    assert np.array_equal(step, (lam * ii + jj) // N)
    out = p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    p.sync()
    got = to_np(out)
    log(compare(got, ref, table, cfg["K"], tol=tol))
    y = inputs.encoder_input(sym, inputs.make_noise(cfg["B"], cfg["H"], cfg["W"], cfg["M"]), ref["mean"])
    out_e, s = p.encode(torch.from_numpy(psi).cuda(), torch.from_numpy(y).cuda())
    p.sync()
    assert np.array_equal(s.cpu().numpy(), sym)
    log(compare(to_np(out_e), ref, table, cfg["K"], tol=tol))
    p.close()


@pytest.mark.parametrize("precision,N", [("fp32", 4), ("fp32", 8), ("bf16", 4)])
def test_grouped_4k_full_size(precision, N):
    name, rows, n = "minnen-hr-4k-240x135-m320", 5, 300
    log(f"grouped case {name} full size N={N} precision={precision}: top {rows} rows + {n} teacher-forced")
    cfg, w, table, psi, sym = make_case(name)
    bf = precision == "bf16"
    tol = BF16_TOL if bf else FP32_TOL
    p = plan(cfg, w, table, N, "graph", precision)
    out = p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    p.sync()
    got = to_np(out)
    p.close()
    top = model(cfg, w, table, N, bf, H=rows).decode(psi[:, :rows].copy(), sym[:, :rows].copy())
    log(compare({k: v[:, :rows] for k, v in got.items()}, top, table, cfg["K"], tol=tol))
    lats = sample_latents(cfg, n)
    log(teacher_forced(cfg, got, psi, sym, model(cfg, w, table, N, bf), lats, table, tol=tol))
