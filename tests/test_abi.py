"""Host-side checks of the C-ABI library (no GPU needed).

The library must load, export every function that include/wf.h declares,
produce the same schedule as the brute-force schedule oracle (bit-exact), and
reject bad descriptions with the documented status codes before touching the
GPU.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import schedule as S
from paper_2607_19082_amd import inputs, wf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(wf.LIB_PATH):
        from paper_2607_19082_amd import build
        build.build()
    return wf.lib()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "wf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\s*\*)\s*\*?\s*(wf_\w+)\s*\(", src, flags=re.M)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(wf.EXPORTS) == names


@pytest.mark.parametrize("mask,kernel,relaxed,lam", [("full", 5, False, 3), ("relaxed", 5, True, 2),
                                                     ("3x3", 3, False, 2), ("7x7", 7, False, 4)])
def test_schedule_matches_oracle(lib, mask, kernel, relaxed, lam):
    """The library's schedule is the earliest-possible one (ASAP levels of the
    brute-force DAG) on every grid, also those narrower than the shear, where
    it is the raster order."""
    ds = S.dependence_vectors(kernel, relaxed=relaxed)
    for H in range(1, 10):
        for W in range(1, 12):
            step, n, got_lam = wf.schedule(H, W, mask)
            assert got_lam == min(lam, W)
            asap = np.array(S.asap_levels(H, W, ds), np.int32)
            assert np.array_equal(step, asap), (H, W)
            assert n == S.critical_path_steps(H, W, ds) == W + got_lam * (H - 1)


@pytest.mark.parametrize("H,W,mask", [(135, 240, "full"), (68, 120, "relaxed"), (32, 48, "full")])
def test_schedule_workload_sizes(lib, H, W, mask):
    step, n, lam = wf.schedule(H, W, mask)
    assert n == W + lam * (H - 1)
    assert n == {(135, 240): 642, (68, 120): 254, (32, 48): 141}[(H, W)]
    # every edge of the DAG goes forward in time (vectorised Eq. 4 check)
    for di, dj in S.dependence_vectors(5, relaxed=(mask == "relaxed")):
        if dj > 0:
            a, b = step[di:, dj:], step[:H - di, :W - dj]
        elif dj < 0:
            a, b = step[di:, :W + dj], step[:H - di, -dj:]
        else:
            a, b = step[di:, :], step[:H - di, :]
        assert np.all(a > b)


def test_schedule_errors(lib):
    n = ctypes.c_int32()
    assert lib.wf_schedule(0, 5, 0, None, ctypes.byref(n), None) == wf.WF_E_INVALID
    assert lib.wf_schedule(5, 5, 7, None, ctypes.byref(n), None) == wf.WF_E_INVALID
    assert lib.wf_schedule(5, 5, 0, None, None, None) == wf.WF_E_INVALID
    assert lib.wf_schedule(5, 5, 4, None, ctypes.byref(n), None) == wf.WF_E_INVALID
    # grids narrower than the shear: the raster order, H*W steps
    lam = ctypes.c_int32()
    for mask, W in ((0, 2), (1, 1), (2, 1), (3, 3), (3, 1)):
        assert lib.wf_schedule(5, W, mask, None, ctypes.byref(n), ctypes.byref(lam)) == wf.WF_OK
        assert (n.value, lam.value) == (5 * W, W)


def _desc(**kw):
    M = kw.pop("M", 16)
    K = kw.get("K", 1)
    w = inputs.make_weights(M, K)
    base = dict(H=4, W=5, B=1, K=K)
    base.update(kw)
    return wf.make_desc(w, inputs.scale_table(), **base)


def test_validate(lib):
    d, keep = _desc()
    assert wf.validate(d) == wf.WF_OK
    # narrower than the shear: the exact decode runs in raster order, context
    # approximation (defined on the wavefronts t = lambda*i + j) is refused
    d, keep = _desc(W=2)
    assert wf.validate(d) == wf.WF_OK
    d.group = 2
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
    assert b"shear" in lib.wf_last_error()
    d, keep = _desc(M=8)
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
    # bf16 operands: a k-block of 32 channels must not straddle two taps
    d, keep = _desc(M=32, precision="bf16")
    assert wf.validate(d) == wf.WF_OK
    d, keep = _desc(M=48, precision="bf16")
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
    d, keep = _desc(M=48)
    assert wf.validate(d) == wf.WF_OK
    d, keep = _desc()
    d.K = 2
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc()
    d.w2 = None
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc()
    d.H = 0
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc()
    d.mask = 4
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc()
    d.driver = 9
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc(param_order="scales_first")
    assert wf.validate(d) == wf.WF_OK
    d.param_order = 2
    assert wf.validate(d) == wf.WF_E_INVALID
    # context approximation: group size >= 0; groups need a per-step-launch driver
    d, keep = _desc()
    d.group = -1
    assert wf.validate(d) == wf.WF_E_INVALID
    for drv, want in (("stream", wf.WF_OK), ("graph", wf.WF_OK), ("persistent", wf.WF_E_UNSUPPORTED),
                      ("dataflow", wf.WF_E_UNSUPPORTED)):
        d, keep = _desc()
        d.driver = wf.DRIVER[drv]
        d.group = 4
        assert wf.validate(d) == want, drv
    t = keep["table"]
    t[5] = t[4]
    assert wf.validate(d) == wf.WF_E_INVALID
    assert lib.wf_validate(None) == wf.WF_E_INVALID
    assert len(lib.wf_last_error()) > 0


def test_null_arguments_rejected(lib):
    out = wf.Out()
    assert lib.wf_decode(None, None, None, ctypes.byref(out), None) == wf.WF_E_INVALID
    assert lib.wf_encode(None, None, None, None, ctypes.byref(out), None) == wf.WF_E_INVALID
    assert lib.wf_decode_noalloc(None, None, None, ctypes.byref(out), None) == wf.WF_E_INVALID
    assert lib.wf_plan(None, None) == wf.WF_E_INVALID
    assert lib.wf_plan_sync(None, None) == wf.WF_E_INVALID
    assert lib.wf_plan_schedule(None, None, None) == wf.WF_E_INVALID
    lib.wf_plan_destroy(None)


@pytest.mark.parametrize("mask,R,W_min", [("3x3", 1, 2), ("full", 2, 3), ("7x7", 3, 4)])
def test_masks_of_any_radius(lib, mask, R, W_min):
    """The (2R+1)x(2R+1) masks validate with weights of their own kernel size;
    the binding refuses weights of another size before any pointer is read."""
    w = inputs.make_weights(16, 1, radius=R)
    d, keep = wf.make_desc(w, inputs.scale_table(), 4, W_min, mask=mask)
    assert wf.validate(d) == wf.WF_OK
    d.W = W_min - 1
    assert wf.validate(d) == wf.WF_OK
    d.group = 3
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
    other = inputs.make_weights(16, 1, radius=1 if R != 1 else 2)
    with pytest.raises(ValueError):
        wf.make_desc(other, inputs.scale_table(), 4, W_min, mask=mask)


def test_entropy_coder_validation(lib):
    d, keep = _desc(entropy_coder="rans", driver="graph")
    assert wf.validate(d) == wf.WF_OK
    d.entropy_coder = 2
    assert wf.validate(d) == wf.WF_E_INVALID
    d, keep = _desc(entropy_coder="rans", driver="graph", K=3)   # the mixture coder
    assert wf.validate(d) == wf.WF_OK
    for kw in (dict(group=2), dict(driver="persistent"), dict(driver="dataflow"), dict(driver="resident")):
        args = dict(entropy_coder="rans", driver="graph")
        args.update(kw)
        d, keep = _desc(**args)
        assert wf.validate(d) == wf.WF_E_UNSUPPORTED, kw
        assert b"entropy" in lib.wf_last_error()


def test_entropy_tables_match_the_oracle(lib):
    """The library builds its rANS tables itself; they must equal the
    oracle's, entry for entry (the coder's bits depend on every one)."""
    import oracle
    for table in (inputs.scale_table(), inputs.scale_table(levels=17, lo=0.5, hi=40.0)):
        n, base, cum = wf.ec_tables(table)
        on, obase, ocum = oracle.rans_tables(table)
        assert np.array_equal(n, on) and np.array_equal(base, obase) and np.array_equal(cum, ocum)
    with pytest.raises(wf.WfError) as e:
        wf.ec_tables(np.array([1.0, 3000.0], np.float32))
    assert e.value.code == wf.WF_E_UNSUPPORTED


def test_mixture_tables_match_the_oracle(lib):
    """The mixture coder's level CDFs (K = 3), built by the library itself,
    equal the oracle's entry for entry."""
    import oracle
    for table in (inputs.scale_table(), inputs.scale_table(levels=17, lo=0.5, hi=40.0)):
        X, base, G = wf.mix_tables(table)
        oX, obase, oG = oracle.mix_tables(table)
        assert np.array_equal(X, oX) and np.array_equal(base, obase) and np.array_equal(G, oG)
    with pytest.raises(wf.WfError) as e:
        wf.mix_tables(np.array([1.0, 3000.0], np.float32))
    assert e.value.code == wf.WF_E_UNSUPPORTED


def test_xform_validation(lib):
    """The transform plan refuses bad descriptions before touching the GPU."""
    w = inputs.make_transform_weights(32, 64)
    x = wf.XformDesc(32, 64, 1, 5, 7, 0)
    keep = {k: np.ascontiguousarray(v, np.float32) for k, v in w.items()}
    for k in range(3):
        x.hs_w[k] = keep[f"hs{k + 1}_w"].ctypes.data
        x.hs_b[k] = keep[f"hs{k + 1}_b"].ctypes.data
        x.gdn_beta[k] = keep[f"gdn{k + 1}_beta"].ctypes.data
        x.gdn_gamma[k] = keep[f"gdn{k + 1}_gamma"].ctypes.data
    for k in range(4):
        x.gs_w[k] = keep[f"gs{k + 1}_w"].ctypes.data
        x.gs_b[k] = keep[f"gs{k + 1}_b"].ctypes.data
    h = ctypes.c_void_p()
    for field, value, want in (("N", 24, wf.WF_E_UNSUPPORTED), ("precision", 5, wf.WF_E_INVALID),
                               ("H", 0, wf.WF_E_INVALID), ("W", 100000, wf.WF_E_UNSUPPORTED)):
        old = getattr(x, field)
        setattr(x, field, value)
        assert lib.wf_xform_plan(ctypes.byref(x), ctypes.byref(h)) == want, field
        setattr(x, field, old)
    x.precision = 1
    x.M = 48   # 3M/2 = 72 is not a multiple of the bf16 k-block
    assert lib.wf_xform_plan(ctypes.byref(x), ctypes.byref(h)) == wf.WF_E_UNSUPPORTED
    x.M, x.precision = 64, 0
    x.gs_w[2] = None
    assert lib.wf_xform_plan(ctypes.byref(x), ctypes.byref(h)) == wf.WF_E_INVALID
    assert lib.wf_xform_plan(None, ctypes.byref(h)) == wf.WF_E_INVALID


def test_size_limit(lib):
    """The largest problem a plan accepts: every array the kernels address
    through one raw-buffer window (0x7fff0000 bytes) must fit it; with M = 16
    the binding one is the layer-1 activations, B*H*W rows of d1 = 53 values
    padded to 64 fp32."""
    d, keep = _desc(H=1, W=0x7fff0000 // 256 - 1)
    assert wf.validate(d) == wf.WF_OK
    d, keep = _desc(H=1, W=0x7fff0000 // 256)
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
    assert b"too large" in lib.wf_last_error()
    d, keep = _desc(H=4096, W=4096, B=4)
    assert wf.validate(d) == wf.WF_E_UNSUPPORTED
