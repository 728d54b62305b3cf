"""wf_decode_noalloc (the decode whose working memory is the library's static
device array) against wf_decode on the same plans and inputs, through the
C-ABI: two calls in a row, the second on a smaller input, each compared with
the existing entry point's outputs to the parity bar (bit-identical where both
run the same per-step kernels), and a decode too large for the array rejected
with WF_E_UNSUPPORTED."""
import sys

import numpy as np
import pytest

from paper_2607_19082_amd import wf

from gpu_helpers import BF16_TOL, FP32_TOL, compare, gpu_plan, make_case, oracle_model, to_np

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


def both(cfg, w, table, psi, sym, driver, precision):
    plan = gpu_plan(cfg, w, table, driver, precision)
    psi_d, sym_d = torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda()
    ref = plan.decode(psi_d, sym_d)
    plan.sync()
    ref = to_np(ref)
    out = plan.alloc_out()
    for v in out.values():
        v.fill_(7)   # nothing of a previous call may show through
    plan.decode_noalloc(psi_d, sym_d, out)
    plan.sync()
    got = to_np(out)
    plan.close()
    return got, ref


@pytest.mark.parametrize("driver,precision", [("stream", "fp32"), ("graph", "fp32"), ("graph", "bf16"),
                                              ("dataflow", "fp32")])
def test_noalloc_matches_decode_twice(driver, precision):
    tol = BF16_TOL if precision == "bf16" else FP32_TOL
    # first call: the 16x16 workload; second: a smaller GMM grid
    for name, H, W in (("minnen-16x16-m192", None, None), ("cheng-gmm3-1080p-120x68-m192", 6, 11)):
        log(f"noalloc case {name} H={H} W={W} driver={driver} precision={precision}")
        cfg, w, table, psi, sym = make_case(name, H=H, W=W)
        got, ref = both(cfg, w, table, psi, sym, driver, precision)
        stats = compare(got, ref, table, cfg["K"], tol=tol)
        log(stats)
        if driver in ("stream", "graph"):
            # the same per-step kernels in the same order: the same bits
            for k in ref:
                assert np.array_equal(got[k], ref[k]), k
        oref = oracle_model(cfg, w, table, bf16=precision == "bf16").decode(psi, sym)
        log(compare(got, oref, table, cfg["K"], tol=tol))


def test_noalloc_rejects_too_large():
    cfg, w, table, psi, sym = make_case("minnen-hr-4k-240x135-m320")
    plan = gpu_plan(cfg, w, table, "graph", "fp32")
    out = plan.alloc_out()
    with pytest.raises(wf.WfError) as e:
        plan.decode_noalloc(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda(), out)
    assert e.value.code == wf.WF_E_UNSUPPORTED
    assert "bytes of working memory" in str(e.value)
    plan.close()
