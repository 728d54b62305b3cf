"""Failure paths of the in-launch drivers on the GPU, forced from the host
so that every kernel still exits normally:

* time-out drain: with every counter or barrier wait made unreachable
  (wf_plan_set_waits, stall = 1) and a 10 ms budget, a decode of the
  persistent, dataflow and resident drivers ends, and wf_plan_sync reports
  WF_E_TIMEOUT; the next call, with the waits restored, decodes exactly what
  a call before the stall decoded;
* residency: a plan limited to fewer compute units than its cooperative grid
  needs (wf_desc.cu_limit) is refused with WF_E_UNSUPPORTED;
* the resident driver's line-granularity conditions: M a multiple of 32, y_hat
  aligned to 128 bytes.
"""
import sys

import numpy as np
import pytest

from paper_2607_19082_amd import inputs, wf

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wf.lib()
    torch.cuda.set_device(0)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("driver", ["persistent", "dataflow", "resident"])
def test_timeout_drains_and_recovers(driver):
    cfg, w, table, psi, sym = inputs.make_inputs("minnen-16x16-m192")
    p = wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], driver=driver)
    psi_d, sym_d = torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda()
    log(f"timeout case driver={driver}: reference decode")
    ref = {k: v.clone() for k, v in p.decode(psi_d, sym_d).items()}
    p.sync()
    log(f"timeout case driver={driver}: stalled decode")
    p.set_waits(spin_budget_ticks=1_000_000, stall=1)   # 10 ms
    out = p.decode(psi_d, sym_d)
    with pytest.raises(wf.WfError) as e:
        p.sync()
    assert e.value.code == wf.WF_E_TIMEOUT
    log(f"timeout case driver={driver}: decode after the stall")
    p.set_waits(0, 0)
    out = p.decode(psi_d, sym_d)
    p.sync()
    for k in ref:
        assert torch.equal(out[k], ref[k]), k
    p.close()


@pytest.mark.parametrize("driver", ["persistent", "dataflow", "resident"])
def test_too_few_compute_units_are_refused(driver):
    cfg, w, table, psi, sym = inputs.make_inputs("minnen-16x16-m192")
    log(f"residency case driver={driver}")
    with pytest.raises(wf.WfError) as e:
        wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], driver=driver, cu_limit=4)
    assert e.value.code == wf.WF_E_UNSUPPORTED
    # all compute units: accepted
    wf.Plan(w, table, cfg["H"], cfg["W"], cfg["B"], cfg["K"], driver=driver).close()


def test_resident_refusals():
    """The resident driver reads y_hat with cached loads while it is being
    written, which needs every latent's row to be whole 128-byte lines: it
    refuses M = 16 plans and a y_hat that is not 128-byte aligned."""
    table = inputs.scale_table()
    log("resident refusal cases")
    with pytest.raises(wf.WfError) as e:
        wf.Plan(inputs.make_weights(16, 1), table, 4, 5, 1, 1, driver="resident")
    assert e.value.code == wf.WF_E_UNSUPPORTED
    cfg, w, tab, psi, sym = inputs.make_inputs("minnen-16x16-m192", H=4, W=6)
    p = wf.Plan(w, tab, cfg["H"], cfg["W"], cfg["B"], cfg["K"], driver="resident")
    out = p.alloc_out()
    shape = out["y_hat"].shape
    buf = torch.empty(out["y_hat"].numel() + 1, dtype=torch.float32, device="cuda")
    out["y_hat"] = buf[1:].view(shape)   # 4 bytes off
    with pytest.raises(wf.WfError) as e:
        p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda(), out=out)
    assert e.value.code == wf.WF_E_INVALID
    p.close()
