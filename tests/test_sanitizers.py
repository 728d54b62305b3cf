"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only: the sanitizers instrument the host side; the device code is built
as usual and never runs here).

A copy of the library is built with the host side instrumented, then a child
process (with the sanitizer runtime preloaded) drives every host entry point
that needs no device: the schedules of every mask on sizes from 1x1 up to the
4K grid, the validation of good and bad plan descriptions, the entropy
coders' tables (including the too-wide error), the dependency lists of the
in-launch drivers over several geometries, and a plan build that fails for
want of a device (its cleanup path).  Any sanitizer report fails the test.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

DRIVE = r'''
import sys
import numpy as np
sys.path.insert(0, ROOT)
from paper_2607_19082_amd import inputs, wf
wf.LIB_PATH = LIB
L = wf.lib()
t = inputs.scale_table()
for mask in ["full", "relaxed", "3x3", "7x7"]:
    for H, W in [(1, 1), (1, 7), (5, 1), (3, 2), (9, 20), (68, 120), (135, 240)]:
        step, T = wf.schedule(H, W, mask)[:2]
        assert step.shape == (H, W) and 0 < T <= H * W, (mask, H, W)
for K in (1, 3):
    w = inputs.make_weights(32, K)
    for kw in (dict(), dict(driver="graph"), dict(precision="bf16"), dict(group=3), dict(mask="7x7"),
               dict(entropy_coder="rans", driver="graph"), dict(driver="resident"), dict(driver="dataflow")):
        wk = inputs.make_weights(32, K, radius=3) if kw.get("mask") == "7x7" else w
        d, keep = wf.make_desc(wk, t, 6, 9, **kw)
        assert wf.validate(d) == wf.WF_OK, (K, kw)
        for bad in (dict(H=0), dict(M=15), dict(K=2), dict(L=1), dict(entropy_coder=9), dict(group=-1)):
            d2, keep2 = wf.make_desc(wk, t, 6, 9, **kw)
            for f, v in bad.items():
                setattr(d2, f, v)
            assert wf.validate(d2) != wf.WF_OK, (K, kw, bad)
            assert len(L.wf_last_error()) > 0
for tab in (t, inputs.scale_table(levels=17, lo=0.5, hi=40.0)):
    wf.ec_tables(tab)
    wf.mix_tables(tab)
for fn in (wf.ec_tables, wf.mix_tables):
    try:
        fn(np.array([1.0, 3000.0], np.float32))
        raise AssertionError("a too-wide level was accepted")
    except wf.WfError:
        pass
for drv in ("dataflow", "resident"):
    for M, H, W, B, mask in [(16, 1, 1, 1, "full"), (32, 12, 14, 3, "full"), (16, 40, 30, 2, "relaxed"),
                             (16, 9, 20, 1, "3x3"), (48, 20, 9, 2, "full")]:
        R = {"3x3": 1, "7x7": 3}.get(mask, 2)
        d, keep = wf.make_desc(inputs.make_weights(M, 1, radius=R), t, H, W, B=B, mask=mask, driver=drv)
        assert wf.plan_deps(d).size > 0
# a plan build without a device fails cleanly
d, keep = wf.make_desc(inputs.make_weights(16, 1), t, 4, 5)
try:
    wf.Plan(inputs.make_weights(16, 1), t, 4, 5, 1, 1)
    raise AssertionError("a plan was built without a device")
except Exception as e:
    assert "HIP" in str(e) or "device" in str(e).lower() or isinstance(e, wf.WfError), e
print("sanitized run ok", flush=True)
'''


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if not os.path.exists(HIPCC) or _asan_runtime() is None:
        pytest.skip("hipcc or the sanitizer runtime is missing")
    out = str(tmp_path_factory.mktemp("asan") / "libwf_asan.so")
    csrc = os.path.join(ROOT, "paper_2607_19082_amd", "csrc")
    # the sanitizers instrument the host code only (-Xarch_host before each)
    cmd = [HIPCC, "--offload-arch=gfx950", "-O0", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-g",
           "-I", os.path.join(ROOT, "include"), "-I", csrc] + sorted(glob.glob(os.path.join(csrc, "*.hip"))) + [
        "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return out


def test_host_code_under_sanitizers(sanitized_lib):
    env = dict(os.environ)
    env["LD_PRELOAD"] = _asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:exitcode=23"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1:exitcode=24"
    code = f"ROOT = {ROOT!r}\nLIB = {sanitized_lib!r}\n" + DRIVE
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    report = r.stdout[-2000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    assert "sanitized run ok" in r.stdout, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
