"""GPU check of the scales-first parameter layout: a model whose last layer
emits its blocks as scale | mean (| weight) decodes, through the C-ABI with
param_order = scales_first, bit for bit like the same model given in the
native order, and matches the oracle within the usual bars."""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_19082_amd import inputs, wf

from gpu_helpers import BF16_TOL, FP32_TOL, compare, make_case, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wf.lib()  # fails loudly when the library is missing
    torch.cuda.set_device(0)
    return torch.device("cuda", 0)


def scales_first(w, K, M):
    """The same model with the last layer's row blocks reversed: native
    mean | scale (K = 1) or weight | mean | scale (K = 3, blocks of 3M)."""
    bs = M if K == 1 else 3 * M
    nb = 2 if K == 1 else 3
    order = [b * bs + r for b in reversed(range(nb)) for r in range(bs)]
    return dict(w, w3=np.ascontiguousarray(w["w3"][order]), b3=np.ascontiguousarray(w["b3"][order]))


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name,H,W,B", [("minnen-16x16-m192", 6, 9, 2), ("cheng-gmm3-1080p-120x68-m192", 5, 10, 1)])
def test_scales_first_layout(name, H, W, B, precision):
    print(f"param-order case {name} H={H} W={W} B={B} precision={precision}", flush=True)
    sys.stdout.flush()
    cfg, w, table, psi, sym = make_case(name, H=H, W=W, B=B)
    K, M = cfg["K"], cfg["M"]
    outs = []
    for weights, order in ((w, "native"), (scales_first(w, K, M), "scales_first")):
        p = wf.Plan(weights, table, H, W, B, K, precision=precision, driver="graph", param_order=order)
        out = p.decode(torch.from_numpy(psi).cuda(), torch.from_numpy(sym).cuda())
        p.sync()
        outs.append(to_np(out))
        p.close()
    assert all(np.array_equal(outs[0][k], outs[1][k]) for k in outs[0])
    bf = precision == "bf16"
    ref = oracle.Model(w, table, H, W, B, K, bf16=bf).decode(psi, sym)
    print(compare(outs[1], ref, table, K, tol=BF16_TOL if bf else FP32_TOL), flush=True)
