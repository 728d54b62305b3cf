"""Oracle references for the GPU parity tests, computed on host threads.

The oracle is C called through ctypes, which releases the GIL during a call,
so several whole oracle decodes run at once on the host cores while the GPU
tests run.  A test module names the references it will need when it is
imported on a machine with a GPU (`prefetch`); a test then waits for its
reference (`ref_decode(...).result()`).  Every reference is the oracle's own
decode of seeded inputs: nothing here reads the GPU path's outputs.
"""
import os
import threading
from concurrent.futures import ThreadPoolExecutor

import oracle
from paper_2607_19082_amd import inputs

_lock = threading.Lock()
_pool = None
_futs = {}


def _executor():
    global _pool
    if _pool is None:
        _pool = ThreadPoolExecutor(max_workers=max(1, min(6, (os.cpu_count() or 2) - 2)),
                                   thread_name_prefix="oracle")
    return _pool


def _decode(name, H, W, B, rows, bf16):
    cfg, w, table, psi, sym = inputs.make_inputs(name, H=H, W=W, B=B)
    if rows is not None:
        psi, sym = psi[:, :rows].copy(), sym[:, :rows].copy()
    Hr = cfg["H"] if rows is None else rows
    m = oracle.Model(w, table, Hr, cfg["W"], cfg["B"], cfg["K"], relaxed=cfg["relaxed"], bf16=bf16)
    return m.decode(psi, sym)


def ref_decode(name, H=None, W=None, B=None, rows=None, bf16=False):
    """Future of the oracle's decode of workload `name` (optionally resized to
    H x W x B), or of its top `rows` grid rows (an exact sub-decode: every tap
    lies in the latent's row or above)."""
    key = (name, H, W, B, rows, bool(bf16))
    with _lock:
        f = _futs.get(key)
        if f is None:
            f = _executor().submit(_decode, name, H, W, B, rows, bool(bf16))
            _futs[key] = f
    return f


def prefetch(cases):
    """Start the listed references now: tuples (name, H, W, B, rows, bf16)."""
    for c in cases:
        ref_decode(*c)


def shutdown():
    global _pool
    with _lock:
        if _pool is not None:
            _pool.shutdown(wait=False, cancel_futures=True)
            _pool = None
