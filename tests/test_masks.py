"""Pins of the oracle for causal masks of any radius (Appendix A, Def. 1:
(2R+1)x(2R+1), the R rows above within horizontal offset R and the R
latents to the left; shear lambda = R + 1, Sec. III-B).

* R = 1: the library fixed point with the 3x3 mask built from the context
  cells printed in Fig. 2(c); R = 3: the same with the 7x7 mask built from the
  schedule oracle's dependence vectors (pinned by Thm. 1 in test_schedule).
* The wavefront order t = (R+1)i + j gives the raster decode's bits, a
  column-major order does not.
* Weights at non-causal positions are ignored.
* Context approximation with the 3x3 mask reproduces Fig. 3(b), whose figure
  is drawn for exactly that mask.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import schedule as S
from paper_2607_19082_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def read_cells(name, keys):
    focus, cells = None, []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            parts = line.split()
            if not parts or parts[0].startswith("#"):
                continue
            if parts[0] == "focus":
                focus = (int(parts[1]), int(parts[2]))
            elif parts[0] in keys:
                cells.append((int(parts[1]), int(parts[2])))
    return focus, cells


def mask_from_cells(focus, cells, R):
    m = np.zeros((2 * R + 1, 2 * R + 1))
    for r, c in cells:
        m[r - focus[0] + R, c - focus[1] + R] = 1.0
    return m


def mask_from_vectors(R):
    m = np.zeros((2 * R + 1, 2 * R + 1))
    for di, dj in S.dependence_vectors(2 * R + 1):
        m[R - di, R - dj] = 1.0
    return m


def library_params(w, table, y_hat, psi, K, mask, R, slope=0.01):
    """Per-latent parameters from a fixed reconstruction with library routines
    in fp64: torch conv2d over the masked kernel, numpy matmuls, LeakyReLU."""
    B, H, W, M = y_hat.shape
    cw = w["ctx_w"].astype(np.float64) * mask[None, None]
    x = torch.from_numpy(y_hat.astype(np.float64)).permute(0, 3, 1, 2)
    ctx = torch.nn.functional.conv2d(x, torch.from_numpy(cw), torch.from_numpy(w["ctx_b"].astype(np.float64)),
                                     padding=R).permute(0, 2, 3, 1).numpy()
    h = np.concatenate([psi.astype(np.float64), ctx], axis=-1)
    for k in (1, 2):
        h = h @ w[f"w{k}"].astype(np.float64).T + w[f"b{k}"].astype(np.float64)
        h = np.where(h >= 0, h, slope * h)
    o = h @ w["w3"].astype(np.float64).T + w["b3"].astype(np.float64)
    assert K == 1
    mu, sig = o[..., :M], np.maximum(o[..., M:2 * M], table[0])
    idx = np.searchsorted(table[:-1].astype(np.float64), sig, side="left")
    return mu, sig, idx


def case(R, M=8, H=7, W=9, B=1, K=1):
    w = inputs.make_weights(M, K, radius=R)
    table = inputs.scale_table()
    psi = inputs.make_psi(B, H, W, M)
    sym = inputs.make_symbols(B, H, W, M, 2.0, 32)
    return w, table, psi, sym


@pytest.mark.parametrize("R", [1, 3])
def test_fixed_point_against_library(R):
    w, table, psi, sym = case(R)
    out = oracle.Model(w, table, 7, 9).decode(psi, sym)
    if R == 1:
        mask = mask_from_cells(*read_cells("fig2c_wavefront_3x3_lambda2_8x8.txt", ("context",)), R)
    else:
        mask = mask_from_vectors(R)
    assert mask.sum() == 2 * R * R + 2 * R
    mu, sig, idx = library_params(w, table, out["y_hat"], psi, 1, mask, R)
    np.testing.assert_allclose(out["mean"], mu, rtol=0, atol=2e-5)
    np.testing.assert_allclose(out["scale"][..., 0, :], sig, rtol=0, atol=2e-5)
    np.testing.assert_allclose(out["y_hat"] - mu, sym, rtol=0, atol=2e-5)
    t = table[:-1].astype(np.float64)
    s = out["scale"][..., 0, :].astype(np.float64)
    near = (np.abs(s[..., None] - t) <= 1e-5 * t).any(axis=-1) & (s != table[0])
    assert np.array_equal(out["idx"][..., 0, :][~near], idx[~near])
    assert np.abs(out["mean"]).max() > 0.1


@pytest.mark.parametrize("R", [1, 2, 3])
def test_wavefront_order_is_exact(R):
    H, W, B = 6, 9, 2
    w, table, psi, sym = case(R, H=H, W=W, B=B)
    m = oracle.Model(w, table, H, W, B)
    ref = m.decode(psi, sym)
    lam = R + 1
    wave = sorted(((lam * i + j, b, i, j) for b in range(B) for i in range(H) for j in range(W)))
    got = m.decode(psi, sym, order=np.array([b * H * W + i * W + j for _, b, i, j in wave], np.int64))
    assert all(np.array_equal(got[k], ref[k]) for k in ref)
    col = np.array([b * H * W + i * W + j for b in range(B) for j in range(W) for i in range(H)], np.int64)
    bad = m.decode(psi, sym, order=col)
    assert not all(np.array_equal(bad[k], ref[k]) for k in ref)


@pytest.mark.parametrize("R", [1, 3])
def test_non_causal_weights_ignored(R):
    w, table, psi, sym = case(R)
    ref = oracle.Model(w, table, 7, 9).decode(psi, sym)
    w2 = dict(w)
    noise = np.random.default_rng(9).normal(size=w["ctx_w"].shape).astype(np.float32)
    w2["ctx_w"] = np.where(mask_from_vectors(R)[None, None] > 0, w["ctx_w"], noise).astype(np.float32)
    got = oracle.Model(w2, table, 7, 9).decode(psi, sym)
    assert all(np.array_equal(got[k], ref[k]) for k in ref)


def test_fig3b_with_the_3x3_mask():
    focus, _ = read_cells("fig3b_grouped_lambda2_N2_8x8.txt", ())
    _, known = read_cells("fig3b_grouped_lambda2_N2_8x8.txt", ("known",))
    _, filled = read_cells("fig3b_grouped_lambda2_N2_8x8.txt", ("filled",))
    w, table, _, _ = case(1, H=8, W=8)
    m = oracle.Model(w, table, 8, 8, group=2)
    for cells, want in ((known, 1), (filled, 2)):
        for r, c in cells:
            assert m.tap_status(focus[0], focus[1], r - focus[0], c - focus[1]) == want
    # the figure's four context cells are exactly the 3x3 causal taps
    taps = {(r - focus[0], c - focus[1]) for r, c in known + filled}
    assert taps == {(-1 * di, -1 * dj) for di, dj in S.dependence_vectors(3)}
