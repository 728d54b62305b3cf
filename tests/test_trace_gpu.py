"""GPU checks of the measurement hooks behind the per-step latency figures:
wf_plan_trace (device wall-clock stamps of the persistent driver's barriers
and of the dataflow driver's jobs) and wf_measure_floor.

* recording changes no output bit;
* the persistent driver fills 2 + 3T rows of G + 1 entries, each workgroup's
  own stamps increase from barrier to barrier, workgroup 0 leaves a barrier
  no earlier than any workgroup reached it, and no workgroup reaches the next
  barrier before the last one reached this one;
* rows that do not fit the capacity are left untouched, and a NULL array
  turns recording off;
* the dataflow driver's triples (waiting, inputs complete, results landed)
  are ordered;
* the stream and graph drivers refuse the hook.
"""
import sys

import numpy as np
import pytest

from paper_2607_19082_amd import wf

from gpu_helpers import gpu_plan, make_case, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# the device wall clock runs at 100 MHz; stamps of different workgroups are
# compared with this slack (ticks) for clock skew between compute units
SKEW = 200


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


def decode(plan, psi, sym):
    out = plan.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
    plan.sync()
    return to_np(out)


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
def test_persistent_barrier_stamps(precision):
    cfg, w, table, psi, sym = make_case("minnen-16x16-m192", H=6, W=9, B=2)
    log(f"trace case persistent H=6 W=9 B=2 precision={precision}")
    T = 9 + 3 * 5
    plan = gpu_plan(cfg, w, table, "persistent", precision)
    plain = decode(plan, psi, sym)
    needed, G = plan.trace(None)
    assert needed == (2 + 3 * T) * (G + 1)
    st = torch.full((needed,), -1, dtype=torch.int64, device="cuda")
    plan.trace(st)
    traced = decode(plan, psi, sym)
    for k in plain:
        assert np.array_equal(traced[k], plain[k]), k
    a = st.cpu().numpy().reshape(2 + 3 * T, G + 1)
    assert (a > 0).all()
    arr, rel = a[:, :G], a[:, G]
    assert (np.diff(arr, axis=0) > 0).all()          # each workgroup's own stamps increase
    assert (np.diff(rel) > 0).all()
    assert (rel >= arr[:, 0]).all()                  # workgroup 0 arrives, then leaves
    assert (rel + SKEW >= arr.max(axis=1)).all()     # nobody reaches a barrier after it opened
    # nobody reaches the next barrier before the last one reached this one
    assert (arr[1:].min(axis=1) + SKEW >= arr[:-1].max(axis=1)).all()
    log(f"grid {G}, {T} steps, decode {(rel[-1] - arr[0].min()) / 100.0:.1f} us")

    # a capacity one short of a call's rows leaves the last row untouched
    st.fill_(-1)
    plan.trace(st[:needed - 1])
    decode(plan, psi, sym)
    b = st.cpu().numpy().reshape(2 + 3 * T, G + 1)
    assert (b[:-1] > 0).all() and (b[-1] == -1).all()
    # NULL turns recording off
    plan.trace(None)
    st.fill_(-1)
    decode(plan, psi, sym)
    assert int((st != -1).sum().item()) == 0
    plan.close()


def test_dataflow_job_stamps():
    cfg, w, table, psi, sym = make_case("minnen-16x16-m192", H=6, W=9, B=1)
    log("trace case dataflow H=6 W=9 B=1 fp32")
    plan = gpu_plan(cfg, w, table, "dataflow", "fp32")
    plain = decode(plan, psi, sym)
    needed, G = plan.trace(None)
    assert needed > 0 and needed % 3 == 0 and G > 0
    st = torch.full((needed,), -1, dtype=torch.int64, device="cuda")
    plan.trace(st)
    traced = decode(plan, psi, sym)
    plan.trace(None)
    plan.close()
    for k in plain:
        assert np.array_equal(traced[k], plain[k]), k
    t = st.cpu().numpy().reshape(-1, 3)
    assert (t > 0).all()
    assert (t[:, 0] <= t[:, 1]).all() and (t[:, 1] <= t[:, 2]).all()
    log(f"{t.shape[0]} jobs, span {(t[:, 2].max() - t[:, 0].min()) / 100.0:.1f} us")


@pytest.mark.parametrize("driver", ["stream", "graph"])
def test_trace_refused_by_launch_drivers(driver):
    cfg, w, table, psi, sym = make_case("minnen-16x16-m192", H=4, W=5, B=1)
    plan = gpu_plan(cfg, w, table, driver, "fp32")
    with pytest.raises(wf.WfError) as e:
        plan.trace(None)
    assert e.value.code == wf.WF_E_UNSUPPORTED
    plan.close()


def test_measure_floor():
    cfg, w, table, psi, sym = make_case("minnen-16x16-m192", H=4, W=5, B=1)
    plan = gpu_plan(cfg, w, table, "graph", "fp32")
    node, bar = plan.measure_floor()
    log(f"graph node {node:.2f} us, barrier round {bar:.2f} us")
    assert 0.0 < node < 1000.0
    assert bar == -1.0 or 0.0 < bar < 1000.0
    # the plan still decodes after the probes
    decode(plan, psi, sym)
    plan.close()
