"""Pins of the schedule oracle against the paper's closed forms and figures.

* Appendix A, Thm. 1: lambda = R + 1 is valid and its step count
  lambda*I + J - lambda equals the DAG's critical path (for J >= R + 1).
* Sec. III-B, Eq. 5-7: for the 5x5 mask the smallest valid integer shear is 3.
* Fig. 2(c)/(d): the printed 8x8 step grids and the shaded context cells.
"""
import os
import random

import pytest

from oracle import schedule as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def read_fig(name):
    grid, focus, ctx = [], None, []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("focus"):
                focus = tuple(int(v) for v in line.split()[1:])
            elif line.startswith("context"):
                ctx.append(tuple(int(v) for v in line.split()[1:]))
            else:
                grid.append([int(v) for v in line.split()])
    return grid, focus, ctx


@pytest.mark.parametrize("fname,kernel,lam", [
    ("fig2d_wavefront_5x5_lambda3_8x8.txt", 5, 3),
    ("fig2c_wavefront_3x3_lambda2_8x8.txt", 3, 2),
])
def test_figure_grids(fname, kernel, lam):
    grid, focus, ctx = read_fig(fname)
    ds = S.dependence_vectors(kernel)
    # the printed numbers are the linear schedule lambda*i + j
    assert S.linear_rank(8, 8, lam, 1) == grid
    # the shaded cells are exactly the mask's dependence vectors at the focus
    fi, fj = focus
    assert sorted((fi - di, fj - dj) for di, dj in ds) == sorted(ctx)
    # every context cell is decoded strictly earlier than the focus
    assert all(grid[r][c] < grid[fi][fj] for r, c in ctx)
    # step count: Thm. 1 closed form and the DAG's critical path
    assert S.n_steps(grid) == lam * 8 + 8 - lam
    assert S.critical_path_steps(8, 8, ds) == S.n_steps(grid)
    assert S.is_valid(grid, S.edges(8, 8, ds))


def test_shear_condition_eq7():
    # Eq. 6-7: pi . d > 0 for all d with pi = (lambda, 1); the critical vector
    # (1, -2) forces lambda > 2 for the 5x5 mask.
    ds = S.dependence_vectors(5)
    assert (1, -2) in ds
    ok = [lam for lam in range(0, 6) if all(lam * di + dj > 0 for di, dj in ds)]
    assert min(ok) == 3


@pytest.mark.parametrize("H", range(1, 13))
@pytest.mark.parametrize("W", range(1, 13))
def test_full_mask_optimal(H, W):
    ds = S.dependence_vectors(5)
    es = S.edges(H, W, ds)
    rank = S.linear_rank(H, W, 3, 1)
    assert S.is_valid(rank, es)
    cp = S.critical_path_steps(H, W, ds)
    if W >= 3:
        # Thm. 1 (J >= R + 1): optimal, and ASAP levels are 3i + j exactly
        assert cp == W + 3 * (H - 1) == S.n_steps(rank)
        assert S.asap_levels(H, W, ds) == rank
        best, arg = S.best_linear_schedules(H, W, ds)
        assert best == cp
        if H >= 2:
            assert arg == [(3, 1)]
    else:
        # narrow grids: still valid, but the DAG allows fewer steps
        assert cp <= S.n_steps(rank)
        if H >= 2:
            assert cp < S.n_steps(rank)


@pytest.mark.parametrize("H", range(1, 11))
@pytest.mark.parametrize("W", range(1, 11))
def test_relaxed_mask(H, W):
    ds = S.dependence_vectors(5, relaxed=True)
    assert len(ds) == 10 and (1, -2) not in ds and (2, -2) not in ds
    es = S.edges(H, W, ds)
    rank = S.linear_rank(H, W, 2, 1)
    assert S.is_valid(rank, es)
    # lambda = 3 is no longer needed; lambda = 2 is the least valid shear
    if W >= 2 and H >= 2:
        assert not S.is_valid(S.linear_rank(H, W, 1, 1), es)
    cp = S.critical_path_steps(H, W, ds)
    if W >= 2:
        assert cp == W + 2 * (H - 1) == S.n_steps(rank)
        assert S.asap_levels(H, W, ds) == rank
        best, arg = S.best_linear_schedules(H, W, ds)
        assert best == cp
        if H >= 2:
            assert arg == [(2, 1)]


@pytest.mark.parametrize("kernel", [3, 7])
def test_general_R(kernel):
    # Thm. 1 for R = 1 and R = 3: lambda = R + 1 valid and optimal for J >= R + 1
    R = kernel // 2
    ds = S.dependence_vectors(kernel)
    for H in range(1, 9):
        for W in range(R + 1, R + 6):
            rank = S.linear_rank(H, W, R + 1, 1)
            assert S.is_valid(rank, S.edges(H, W, ds))
            assert S.critical_path_steps(H, W, ds) == (R + 1) * H + W - (R + 1)


def test_wavefronts_are_independent():
    # no edge joins two latents of the same wavefront (Sec. III-A)
    H, W = 9, 11
    ds = S.dependence_vectors(5)
    rank = S.linear_rank(H, W, 3, 1)
    es = S.edges(H, W, ds)
    for s, d in es:
        assert rank[s[0]][s[1]] != rank[d[0]][d[1]]
    sets = S.wavefront_sets(rank)
    assert sum(len(v) for v in sets.values()) == H * W
    assert max(len(v) for v in sets.values()) == min(H, -(-W // 3))


def test_invalid_schedule_detected():
    # a plausible mistake (shear 2 for the 5x5 mask) must be rejected
    rng = random.Random(0)
    for _ in range(20):
        H, W = rng.randint(2, 9), rng.randint(3, 9)
        es = S.edges(H, W, S.dependence_vectors(5))
        assert not S.is_valid(S.linear_rank(H, W, 2, 1), es)
