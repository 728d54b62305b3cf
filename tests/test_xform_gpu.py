"""GPU parity of the transforms around the autoregressive decode (hyper-decoder
h_s and synthesis g_s, the latent pipeline of Sec. II-A; layer list in
oracle/transforms.py), through the C-ABI, against the fp64 PyTorch oracle.

Bar: the largest absolute error over an output is at most 1e-4 (fp32) or
1e-2 (bf16: bf16 weights, activations as bf16 pairs) times max(1, the largest
output magnitude): the products here run over up to 4320 terms, so the bar is
taken relative to the output's scale.  Small grids are compared whole; at the
3840x2160 size the oracle recomputes crops of the input (with the receptive
field's margin, pinned in test_transforms) and the GPU output is compared
there.
"""
import sys

import numpy as np
import pytest

from oracle import transforms as T
from paper_2607_19082_amd import inputs, wf

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


TOL = {"fp32": 1e-4, "bf16": 1e-2}


def check(got, ref, precision, what):
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what
    err = float(np.abs(got.astype(np.float64) - ref).max())
    scale = max(1.0, float(np.abs(ref).max()))
    log(f"{what}: max abs err {err:.3e}, output scale {scale:.3e}")
    assert err <= TOL[precision] * scale, (what, err, scale)


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("B,H,W", [(2, 5, 7), (1, 8, 4), (1, 1, 1)])
def test_transforms_small(B, H, W, precision):
    N, M = 32, 64
    log(f"xform case N={N} M={M} B={B} H={H} W={W} precision={precision}")
    w = inputs.make_transform_weights(N, M)
    z = inputs.make_zhat(B, -(-H // 4), -(-W // 4), N)
    y = np.random.default_rng(7).normal(scale=2.0, size=(B, H, W, M)).astype(np.float32)
    x = wf.Xform(w, N, M, B, H, W, precision)
    psi = x.hyper_synthesis(torch.from_numpy(z).cuda())
    img = x.synthesis(torch.from_numpy(y).cuda())
    torch.cuda.synchronize()
    check(psi.cpu().numpy(), T.hyper_synthesis(z, w)[:, :H, :W], precision, "psi")
    check(img.cpu().numpy(), T.synthesis(y, w), precision, "image")
    x.close()


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
def test_transforms_4k_full_size(precision):
    name = "minnen-hr-4k-240x135-m320"
    cfg = inputs.workload(name)
    N, M, B, H, W = 192, cfg["M"], 1, cfg["H"], cfg["W"]
    log(f"xform case {name} full size N={N} M={M} precision={precision}")
    w = inputs.make_transform_weights(N, M)
    Hz, Wz = -(-H // 4), -(-W // 4)
    z = inputs.make_zhat(B, Hz, Wz, N)
    y = np.random.default_rng(8).normal(scale=2.0, size=(B, H, W, M)).astype(np.float32)
    x = wf.Xform(w, N, M, B, H, W, precision)
    psi = x.hyper_synthesis(torch.from_numpy(z).cuda()).cpu().numpy()
    img = x.synthesis(torch.from_numpy(y).cuda()).cpu().numpy()
    x.close()
    assert np.all(np.isfinite(psi)) and np.all(np.isfinite(img))
    # psi: crops of z at corners and inside; the pinned margin is 2 z pixels
    # (8 psi pixels) on each side, except at the grid's own edges
    for zy, zx in ((0, 0), (10, 27), (Hz - 6, Wz - 6), (0, Wz - 6), (Hz - 6, 0)):
        ref = T.hyper_synthesis(z[:, zy:zy + 6, zx:zx + 6], w)
        lo_y = 0 if zy == 0 else 8
        lo_x = 0 if zx == 0 else 8
        hi_y = 24 if zy + 6 >= Hz else 16
        hi_x = 24 if zx + 6 >= Wz else 16
        py, px = 4 * zy, 4 * zx
        hi_y = min(hi_y, H - py)
        hi_x = min(hi_x, W - px)
        check(psi[:, py + lo_y:py + hi_y, px + lo_x:px + hi_x], ref[:, lo_y:hi_y, lo_x:hi_x], precision,
              f"psi crop at z ({zy}, {zx})")
    # image: crops of y_hat, margins of one latent before and two after
    for ly, lx in ((0, 0), (60, 111), (H - 5, W - 5)):
        ref = T.synthesis(y[:, ly:ly + 5, lx:lx + 5], w)
        lo_y = 0 if ly == 0 else 16
        lo_x = 0 if lx == 0 else 16
        hi_y = 80 if ly + 5 >= H else 48
        hi_x = 80 if lx + 5 >= W else 48
        oy, ox = 16 * ly, 16 * lx
        check(img[:, oy + lo_y:oy + hi_y, ox + lo_x:ox + hi_x], ref[:, lo_y:hi_y, lo_x:hi_x], precision,
              f"image crop at y ({ly}, {lx})")
