"""Coherence litmus test of the exchange inside one launch (wf_litmus), the
mechanism the persistent, dataflow and resident drivers use to pass y_hat
and the activations between workgroups on different XCDs (the causality of
Sec. III-A, Eq. 4 depends on it): agent-coherent stores, s_waitcnt, a relaxed
agent-scope counter; the consumer on another XCD polls, then reads with
agent-coherent loads (mode 0) or ordinary loads of addresses written once per
launch (mode 1); or, with the counter bumped before the stores land, reads
agent-coherent and reads again every word still holding the pre-launch fill
(mode 2, the fp32 layer-1/-2 hand-offs of the resident driver).  Every word
must read back as written."""
import sys

import pytest

from paper_2607_19082_amd import wf

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wf.lib()
    torch.cuda.set_device(0)


@pytest.mark.parametrize("mode", [0, 1, 2])
@pytest.mark.parametrize("pairs,rounds", [(8, 400), (128, 100)])
def test_litmus(mode, pairs, rounds):
    print(f"litmus mode={mode} pairs={pairs} rounds={rounds}", flush=True)
    sys.stdout.flush()
    bad = wf.litmus(mode, pairs, rounds)
    assert bad == 0, bad
