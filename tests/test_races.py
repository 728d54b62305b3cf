"""Race checks of the two drivers that exchange data inside one launch (the
dataflow and the resident driver), on the CPU.

The causality of the wavefront decode (Sec. III-A, Eq. 3-4: a latent is
decoded only after every latent of its causal mask) holds on the GPU only if
every job waits for the jobs whose results it reads, and, where a buffer is
reused, for the readers of the previous contents before it overwrites them.
The waits come from the library itself (wf_plan_deps, computed by the same
functions the kernels call); what each job reads and writes is modelled here
from the data layout the drivers document, independently of the kernels:

* dataflow: y_hat written once per latent by the mean columns of layer 3
  (C0); layer 1 (A) reads the two new taps and the step's old-tap context;
  the context k-parts (CTX) and their sum (CTXL) read the old taps; h1 is one
  buffer by row tile, h2 and the context are double-buffered by step parity;
* resident: one output buffer per task (step, image, 16-row band) and role,
  so only read-after-write order matters; the context parts before the last
  (CTX) read the old taps (in raster order) before the first one of age 2,
  i.e. the eight of ages 3 to 8, and the last part (CTXL) the other two and
  the CTX parts; layer 1 also reads the hoisted part of its task, which the
  hoist workgroups compute inside the launch.

A simulation runs the jobs in orders the waits allow (random, "latest job
first", and orders that starve one kind of job), and asserts that every read
finds the data of the job that should have written it, and that no write
overwrites data that a reader still needs.  Every wait must point at jobs earlier in the
global order (then in-order processing cannot deadlock).  Planted omissions
-- a dropped or weakened wait -- must each be caught.
"""
import random

import pytest

from paper_2607_19082_amd import inputs, wf

CTX, CTXL, A, B, C0, C1, HOIST = range(7)
KINDS = 6        # dataflow job kinds
ROLES = 7        # resident roles (the six kinds and the in-launch hoist)
NEW_TAPS = [(-1, 2), (0, -1)]                                    # the 5x5 mask, lambda = 3
OLD_TAPS = [(-2, dx) for dx in range(-2, 3)] + [(-1, dx) for dx in range(-2, 2)] + [(0, -2)]
LAM = 3


def step_span(H, W, t):
    i0 = max(0, -(-(t - W + 1) // LAM))
    i1 = min(H - 1, t // LAM)
    return i0, max(0, i1 - i0 + 1)


def taps_in_grid(H, W, b, i, j, taps):
    return [(b, i + dy, j + dx) for dy, dx in taps if 0 <= i + dy < H and 0 <= j + dx < W]


# Scheduling policies of the simulations: "latest" runs the runnable job that
# comes last in the global order; "random" any runnable job; "starve K" the
# latest runnable job not of kind (role) K, and one of kind K only when
# nothing else can run -- the orders in which a missing wait shows.
POLICIES = ["latest", "random 1", "random 2"] + [f"starve {k}" for k in range(7)]


def pick(run, pos, kind, policy, rng):
    if policy.startswith("random"):
        return rng.choice(run)
    if policy.startswith("starve"):
        k = int(policy.split()[1])
        other = [q for q in run if kind(q) != k]
        return max(other or run, key=pos)
    return max(run, key=pos)


# ---------------------------------------------------------------------------
# dataflow driver


def dataflow_jobs(H, W, Bn, M):
    d, keep = wf.make_desc(inputs.make_weights(M, 1), inputs.scale_table(), H, W, B=Bn, driver="dataflow")
    v = wf.plan_deps(d)
    nrt_max = int(v[-1])
    rows = v[:-1].reshape(-1, 20)
    jobs = []
    for r in rows:
        t, kind, part, rt, ct, li, pos, nw = (int(x) for x in r[:8])
        waits = [tuple(int(x) for x in r[8 + 4 * i:12 + 4 * i]) for i in range(nw)]
        jobs.append(dict(t=t, kind=kind, part=part, rt=rt, ct=ct, li=li, pos=pos, waits=waits))
    return jobs, nrt_max


def group(nrt_max, t, kind, rt):
    return (t * KINDS + kind) * (nrt_max + 1) + rt


def cnt_range(lo, hi, x):
    return sum(1 for c in range(lo, hi) if c % 8 == x)


def step_rows(H, W, Bn, t):
    """Rows of step t: image-major, ascending grid row; row r -> (b, i, j)."""
    i0, n = step_span(H, W, t)
    return [(b, i0 + q, t - LAM * (i0 + q)) for b in range(Bn) for q in range(n)]


class DataflowSim:
    def __init__(self, H, W, Bn, jobs, nrt_max):
        self.H, self.W, self.Bn, self.jobs, self.nrt_max = H, W, Bn, jobs, nrt_max
        self.ncols = {}
        for j in jobs:
            self.ncols.setdefault((j["kind"], j["part"] if j["kind"] == CTX else 0), set()).add(j["ct"])
        has_ctx = any(j["kind"] == CTX for j in jobs)
        self.nparts = max(j["part"] for j in jobs if j["kind"] == CTX) + 2 if has_ctx else 1
        self.G = len(self.ncols[(C0, 0)])

    def rows_of(self, t, rt):
        return step_rows(self.H, self.W, self.Bn, t)[16 * rt:16 * rt + 16]

    def reads_writes(self, j):
        """(latents read, cells read as (cell, version), cells written as (cell, version, readers))."""
        t, kind, rt, ct, part = j["t"], j["kind"], j["rt"], j["ct"], j["part"]
        H, W = self.H, self.W
        lat, rd, wr = [], [], []
        par = t % 2
        nctx = sorted(self.ncols.get((CTXL, 0), []))
        if kind in (CTX, CTXL):
            for b, i, jj in self.rows_of(t, rt):
                lat += taps_in_grid(H, W, b, i, jj, OLD_TAPS)
            if kind == CTX:
                wr.append((("ctx", par, part, rt, ct), t, {("CTXL", t, rt, ct)}))
            else:
                rd += [(("ctx", par, p, rt, ct), t) for p in range(self.nparts - 1)]
                wr.append((("ctx", par, self.nparts - 1, rt, ct), t,
                           {("A", t, rt, c) for c in self.ncols[(A, 0)]}))
        elif kind == A:
            for b, i, jj in self.rows_of(t, rt):
                lat += taps_in_grid(H, W, b, i, jj, NEW_TAPS)
            rd += [(("ctx", par, self.nparts - 1, rt, c), t) for c in nctx]
            wr.append((("h1", rt, ct), t, {("B", t, rt, c) for c in self.ncols[(B, 0)]}))
        elif kind == B:
            rd += [(("h1", rt, c), t) for c in self.ncols[(A, 0)]]
            readers = ({("C0", t, rt, c) for c in self.ncols[(C0, 0)]}
                       | {("C1", t, rt, c) for c in self.ncols[(C1, 0)]})
            wr.append((("h2", par, rt, ct), t, readers))
        else:
            rd += [(("h2", par, rt, c), t) for c in self.ncols[(B, 0)]]
        return lat, rd, wr

    def run(self, waits_of, policy):
        """Execute every job in an order the waits allow; returns the hazards found."""
        rng = random.Random(policy)
        jobs = self.jobs
        cnt = {}
        done = [False] * len(jobs)
        lat_done = {}      # latent -> C0 column tiles written
        cells = {}         # cell -> [version, pending readers]
        name = {A: "A", B: "B", C0: "C0", C1: "C1", CTX: "CTX", CTXL: "CTXL"}
        hazards = []

        def ready(k):
            for g, lo, hi, mult in waits_of(jobs[k]):
                for x in range(8):
                    if cnt.get((g, x), 0) < mult * cnt_range(lo, hi, x):
                        return False
            return True

        pending = set(range(len(jobs)))
        while pending:
            run = [k for k in pending if ready(k)]
            if not run:
                hazards.append("deadlock")
                break
            k = pick(run, lambda q: jobs[q]["pos"], lambda q: jobs[q]["kind"], policy, rng)
            j = jobs[k]
            lat, rd, wr = self.reads_writes(j)
            me = (name[j["kind"]], j["t"], j["rt"], j["ct"])
            for L in lat:
                if lat_done.get(L, 0) < self.G:
                    hazards.append(("y_hat not written", me, L))
            for cell, ver in rd:
                c = cells.get(cell)
                if c is None or c[0] != ver:
                    hazards.append(("stale read", me, cell, None if c is None else c[0]))
                else:
                    c[1].discard(me)
            for cell, ver, readers in wr:
                c = cells.get(cell)
                if c is not None and c[1]:
                    hazards.append(("overwrite before read", me, cell, sorted(c[1])[:2]))
                cells[cell] = [ver, set(readers)]
            if j["kind"] == C0:
                for b, i, jj in self.rows_of(j["t"], j["rt"]):
                    lat_done[(b, i, jj)] = lat_done.get((b, i, jj), 0) + 1
            x = j["ct"] % 8
            cnt[(group(self.nrt_max, j["t"], j["kind"], j["rt"]), x)] = \
                cnt.get((group(self.nrt_max, j["t"], j["kind"], j["rt"]), x), 0) + 1
            if j["kind"] in (C0, C1):
                g = group(self.nrt_max, j["t"], j["kind"], self.nrt_max)
                cnt[(g, x)] = cnt.get((g, x), 0) + 1
            pending.discard(k)
            done[k] = True
            if len(hazards) > 20:
                break
        return hazards


DF_GEOMS = [(9, 20, 2, 32), (12, 14, 4, 32)]   # H, W, B, M: one and two row tiles per step


@pytest.mark.parametrize("H,W,Bn,M", DF_GEOMS)
def test_dataflow_waits_point_backwards(H, W, Bn, M):
    """Every wait is on jobs earlier in the global order, and on all the jobs
    its targets count (none missing, none extra): in-order processing of the
    lists then always has a runnable job."""
    jobs, nrt_max = dataflow_jobs(H, W, Bn, M)
    assert sorted(j["pos"] for j in jobs) == list(range(len(jobs)))
    bumpers = {}
    for j in jobs:
        x = j["ct"] % 8
        gs = [group(nrt_max, j["t"], j["kind"], j["rt"])]
        if j["kind"] in (C0, C1):
            gs.append(group(nrt_max, j["t"], j["kind"], nrt_max))
        for g in gs:
            bumpers.setdefault((g, x), []).append(j["pos"])
    for j in jobs:
        for g, lo, hi, mult in j["waits"]:
            for x in range(8):
                who = bumpers.get((g, x), [])
                assert len(who) == mult * cnt_range(lo, hi, x), (j, g, x)
                assert all(p < j["pos"] for p in who), (j, g, x)


@pytest.mark.parametrize("H,W,Bn,M", DF_GEOMS)
def test_dataflow_simulation_has_no_hazard(H, W, Bn, M):
    jobs, nrt_max = dataflow_jobs(H, W, Bn, M)
    sim = DataflowSim(H, W, Bn, jobs, nrt_max)
    for policy in POLICIES:
        assert sim.run(lambda j: j["waits"], policy) == [], policy


def _drop(kind, pred):
    """A waits function with the waits of `kind` jobs matching pred removed."""
    def waits(j):
        return [w for w in j["waits"] if not (j["kind"] == kind and pred(j, w))]
    return waits


def _weaken(kind, pred):
    """The same with those waits' multiplicity lowered to one."""
    def waits(j):
        return [(g, lo, hi, 1) if j["kind"] == kind and pred(j, (g, lo, hi, m)) else (g, lo, hi, m)
                for g, lo, hi, m in j["waits"]]
    return waits


def _is_kind(nrt_max, kind):
    return lambda j, w: (w[0] // (nrt_max + 1)) % KINDS == kind


DF_PLANTS = {
    # layer 1 without the previous step's y_hat (its two new taps)
    "A without C0(t-1)": lambda n: _drop(A, _is_kind(n, C0)),
    # layer 1 without its context sum
    "A without CTXL(t)": lambda n: _drop(A, _is_kind(n, CTXL)),
    # the context without the taps of step t-2
    "CTX without C0(t-2)": lambda n: _drop(CTX, _is_kind(n, C0)),
    # the context sum without the other parts
    "CTXL without CTX(t)": lambda n: _drop(CTXL, _is_kind(n, CTX)),
    # layer 2 overwriting h2 of step t-2 before its scale columns read it
    "B without C1(t-2)": lambda n: _drop(B, _is_kind(n, C1)),
    # the step total counted once instead of once per row tile
    "A with one row tile of C0(t-1)": lambda n: _weaken(A, _is_kind(n, C0)),
}


@pytest.mark.parametrize("plant", sorted(DF_PLANTS))
def test_dataflow_simulation_catches_planted_omissions(plant):
    H, W, Bn, M = 12, 14, 4, 32
    jobs, nrt_max = dataflow_jobs(H, W, Bn, M)
    sim = DataflowSim(H, W, Bn, jobs, nrt_max)
    waits = DF_PLANTS[plant](nrt_max)
    found = [h for policy in POLICIES for h in sim.run(waits, policy)]
    assert found, plant


# ---------------------------------------------------------------------------
# resident driver


def resident_tasks(H, W, Bn, M, precision="fp32"):
    d, keep = wf.make_desc(inputs.make_weights(M, 1), inputs.scale_table(), H, W, B=Bn, driver="resident",
                           precision=precision)
    v = wf.plan_deps(d).reshape(-1, 3 + ROLES * 6)
    tasks = [tuple(int(x) for x in r[:3]) for r in v]
    waits = {}
    for k, r in enumerate(v):
        for role in range(ROLES):
            q = r[3 + role * 6:3 + role * 6 + 6]
            waits[(role, k)] = [(int(q[2 * i]), int(q[2 * i + 1])) for i in range(3) if q[2 * i] >= 0]
    return tasks, waits


def resident_reads(H, W, tasks, hoist):
    """The data each (role, task) reads: latents of y_hat (written by the C0
    of the task holding them) and the outputs of other (role, task)."""
    index = {x: k for k, x in enumerate(tasks)}

    def producer(b, i, j):
        return (C0, index[(LAM * i + j, b, i // 16)])

    reads = {}
    for k, (t, b, beta) in enumerate(tasks):
        rows = [(b, i, t - LAM * i) for i in range(16 * beta, min(H, 16 * beta + 16)) if 0 <= t - LAM * i < W]
        part0 = {producer(*L) for (bb, i, j) in rows for L in taps_in_grid(H, W, bb, i, j, OLD_TAPS[:8])}
        part1 = {producer(*L) for (bb, i, j) in rows for L in taps_in_grid(H, W, bb, i, j, OLD_TAPS[8:])}
        new = {producer(*L) for (bb, i, j) in rows for L in taps_in_grid(H, W, bb, i, j, NEW_TAPS)}
        reads[(CTX, k)] = part0
        reads[(CTXL, k)] = part1 | {(CTX, k)}
        reads[(A, k)] = new | {(CTXL, k)} | ({(HOIST, k)} if hoist else set())
        reads[(HOIST, k)] = set()
        reads[(B, k)] = {(A, k)}
        reads[(C0, k)] = {(B, k)}
        reads[(C1, k)] = {(B, k)}
    return reads


def resident_run(tasks, waits_of, reads, policy):
    rng = random.Random(policy)
    nodes = [(role, k) for k in range(len(tasks)) for role in range(ROLES)]
    done = set()
    hazards = []
    pending = set(nodes)
    order = {n: (n[1], n[0]) for n in nodes}
    while pending:
        run = [n for n in pending if all(w in done for w in waits_of(n))]
        if not run:
            hazards.append("deadlock")
            break
        n = pick(run, lambda q: order[q], lambda q: q[0], policy, rng)
        missing = [p for p in reads[n] if p not in done]
        if missing:
            hazards.append(("read before write", n, missing[:2]))
        done.add(n)
        pending.discard(n)
        if len(hazards) > 20:
            break
    return hazards


# bands of 16 rows, several per step; bf16 plans compute the hoisted part of
# layer 1 inside the launch
RES_GEOMS = [(40, 30, 2, 32, "fp32"), (35, 12, 3, 32, "fp32"), (40, 30, 2, 32, "bf16")]


@pytest.mark.parametrize("H,W,Bn,M,prec", RES_GEOMS)
def test_resident_waits_point_backwards(H, W, Bn, M, prec):
    """A task waits only for earlier tasks, or for earlier roles of its own
    task (context, its sum, layers 1, 2, 3): each role's workgroups take
    their tasks in the global order, so the grid never deadlocks."""
    tasks, waits = resident_tasks(H, W, Bn, M, prec)
    # the global order: by step, image, band
    assert tasks == sorted(tasks)
    chain = {HOIST: -1, CTX: 0, CTXL: 1, A: 2, B: 3, C0: 4, C1: 4}
    for (role, k), ws in waits.items():
        for r2, k2 in ws:
            assert k2 < k or (k2 == k and chain[r2] < chain[role]), (role, k, r2, k2)


@pytest.mark.parametrize("H,W,Bn,M,prec", RES_GEOMS)
def test_resident_simulation_has_no_hazard(H, W, Bn, M, prec):
    tasks, waits = resident_tasks(H, W, Bn, M, prec)
    reads = resident_reads(H, W, tasks, prec == "bf16")
    for policy in POLICIES:
        assert resident_run(tasks, lambda n: waits[n], reads, policy) == [], policy


RES_PLANTS = {
    # layer 1 without the band above's task of step t-1 (the upper new tap of row 0)
    "A without the band above": lambda waits, tasks: {
        n: ([w for w in ws if not (n[0] == A and w[0] == C0 and tasks[w[1]][2] != tasks[n[1]][2])] if n[0] == A else ws)
        for n, ws in waits.items()},
    # the context without the band above's task of step t-2
    "CTX without the band above": lambda waits, tasks: {
        n: ([w for w in ws if not (w[0] == C0 and tasks[w[1]][2] != tasks[n[1]][2])] if n[0] == CTX else ws)
        for n, ws in waits.items()},
    # the context without the task's hoisted part (which layer 1 reads after it)
    "CTX without the hoist": lambda waits, tasks: {
        n: ([w for w in ws if w[0] != HOIST] if n[0] == CTX else ws) for n, ws in waits.items()},
    # the context sum without the other parts
    "CTXL without CTX": lambda waits, tasks: {
        n: ([w for w in ws if w[0] != CTX] if n[0] == CTXL else ws) for n, ws in waits.items()},
    # the parts before the last (taps of age >= 3) waiting for step t-4 instead of t-3
    "CTX one step short": lambda waits, tasks: {
        n: ([w for w in ws if w[0] != C0] + [(C0, w2) for w2 in
             [_task_at(tasks, tasks[n[1]][0] - 4, tasks[n[1]][1], tasks[n[1]][2] - d) for d in (0, 1)] if w2 >= 0]
            if n[0] == CTX else ws)
        for n, ws in waits.items()},
    # the last part (which holds the taps of age 2) waiting as long as the others
    "CTXL at the other parts' lag": lambda waits, tasks: {
        n: ([w for w in ws if w[0] != C0] + [(C0, w2) for w2 in
             [_task_at(tasks, tasks[n[1]][0] - 3, tasks[n[1]][1], tasks[n[1]][2] - d) for d in (0, 1)] if w2 >= 0]
            if n[0] == CTXL else ws)
        for n, ws in waits.items()},
}


def _task_at(tasks, t, b, beta):
    """The latest task of band beta (image b) at a step <= t, or -1."""
    best = -1
    for k, (t2, b2, beta2) in enumerate(tasks):
        if b2 == b and beta2 == beta and t2 <= t:
            best = k
    return best


@pytest.mark.parametrize("plant", sorted(RES_PLANTS))
def test_resident_simulation_catches_planted_omissions(plant):
    H, W, Bn, M = 40, 30, 2, 32
    tasks, waits = resident_tasks(H, W, Bn, M, "bf16")
    reads = resident_reads(H, W, tasks, True)
    planted = RES_PLANTS[plant](waits, tasks)
    found = [h for policy in POLICIES for h in resident_run(tasks, lambda n: planted[n], reads, policy)]
    assert found, plant
