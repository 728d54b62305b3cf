"""Schedule oracle: the dependency DAG of a causal mask, by brute force.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The DAG has one vertex per latent and an edge (i',j') -> (i,j) whenever the
offset (i-i', j-j') is one of the mask's dependence vectors and the source lies
inside the grid (Sec. III-A, Eq. 3; Appendix A, Def. 1).  A rank function is a
valid schedule when every edge goes from a smaller to a larger rank (Eq. 4).
The minimal number of parallel steps of any schedule is the number of vertices
on the longest path (Appendix A, Thm. 1, lower bound); ASAP levels reach it.
"""


def dependence_vectors(kernel=5, relaxed=False):
    """Dependence vectors d = (di, dj) of a (2R+1)x(2R+1) raster-causal mask:
    the R rows above within horizontal offset R, plus the R latents to the left
    (Appendix A, Def. 1).  ``relaxed`` drops the two upper-right vectors
    (1,-2) and (2,-2) of the 5x5 mask."""
    R = kernel // 2
    ds = [(r, q) for r in range(1, R + 1) for q in range(-R, R + 1)]
    ds += [(0, p) for p in range(1, R + 1)]
    if relaxed:
        if kernel != 5:
            raise ValueError("the relaxed mask is defined for the 5x5 kernel only")
        ds = [d for d in ds if d not in ((1, -2), (2, -2))]
    return ds


def edges(H, W, ds):
    """All edges (src, dst) of the DAG on an H x W grid; vertices are (i, j)."""
    out = []
    for i in range(H):
        for j in range(W):
            for di, dj in ds:
                si, sj = i - di, j - dj
                if 0 <= si < H and 0 <= sj < W:
                    out.append(((si, sj), (i, j)))
    return out


def asap_levels(H, W, ds):
    """Earliest step of every vertex: 0 without predecessors, else one more than
    the latest predecessor.  Raster order is a topological order (every d has
    di > 0, or di == 0 and dj > 0), so one raster pass suffices."""
    lev = [[0] * W for _ in range(H)]
    for i in range(H):
        for j in range(W):
            best = -1
            for di, dj in ds:
                si, sj = i - di, j - dj
                if 0 <= si < H and 0 <= sj < W:
                    best = max(best, lev[si][sj])
            lev[i][j] = best + 1
    return lev


def critical_path_steps(H, W, ds):
    """Number of vertices on the longest directed path = minimal step count."""
    return max(max(row) for row in asap_levels(H, W, ds)) + 1


def linear_rank(H, W, a, b):
    """Rank a*i + b*j of every vertex, as rows of a list."""
    return [[a * i + b * j for j in range(W)] for i in range(H)]


def is_valid(rank, es):
    """Eq. 4: every edge goes from a strictly smaller rank to a larger one."""
    return all(rank[s[0]][s[1]] < rank[d[0]][d[1]] for s, d in es)


def n_steps(rank):
    """Number of distinct parallel steps between the smallest and largest rank."""
    flat = [v for row in rank for v in row]
    return max(flat) - min(flat) + 1


def best_linear_schedules(H, W, ds, amax=8, bmax=8):
    """Brute force over linear schedules a*i + b*j with 0 <= a <= amax,
    1 <= b <= bmax: return (min_steps, [(a, b), ...]) among the valid ones."""
    es = edges(H, W, ds)
    best, arg = None, []
    for a in range(0, amax + 1):
        for b in range(1, bmax + 1):
            r = linear_rank(H, W, a, b)
            if not is_valid(r, es):
                continue
            s = n_steps(r)
            if best is None or s < best:
                best, arg = s, [(a, b)]
            elif s == best:
                arg.append((a, b))
    return best, arg


def wavefront_sets(rank):
    """Group the vertices by rank: {t: [(i, j), ...]} in row order."""
    sets = {}
    for i, row in enumerate(rank):
        for j, t in enumerate(row):
            sets.setdefault(t, []).append((i, j))
    return dict(sorted(sets.items()))


def group_of(i, j, lam, N):
    """Group of latent (i, j) when N consecutive wavefronts t = lam*i + j are
    decoded together (Sec. III-D, Fig. 3): floor(t / N)."""
    return (lam * i + j) // N
