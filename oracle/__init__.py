"""CPU oracle for wavefront decoding of a spatial autoregressive context model.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU product path never does,
and this package never imports the GPU path.

* ``wf_oracle.c`` -- plain sequential decode/encode of the latent grid in a
  given topological order (raster by default, Sec. III-A, Eq. 2), with the 5x5
  causal masked-conv context (Appendix A, Def. 1, R = 2) and the 1x1 entropy
  parameter network (Sec. II-B, Eq. 1); fp64 accumulation, fp32 storage.
  With ``group`` N > 1 it is the context-approximation decode of Sec. III-D
  (Fig. 3): groups of N wavefronts, same-group taps filled with the mean of
  the decoded taps.
* ``wf_rans.c`` -- rANS entropy coding of the symbols under the mean-scale
  Gaussian model (Sec. II-A; the coder the paper pairs with the wavefront
  decode, Sec. III-C): per-level frequency tables built from the scale
  table, one stream per (image, grid row, channel), and the model decode that
  takes its symbols from those streams; for the 3-component mixture model,
  the same streams with per-latent mixture frequencies built in integer
  arithmetic from quantised parameters.
* ``schedule.py`` -- the dependency DAG of the mask (Eq. 3, Def. 1), its ASAP
  levels and critical path, and a brute-force search over linear schedules
  (Sec. III-B, Eq. 5-7; Appendix A, Thm. 1).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wf_oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "wf_rans.c")]
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build():
    """Compile the C oracle with gcc (-O2, no fast-math, single thread)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fno-fast-math", "-ffp-contract=off", "-o", _LIB] + _SRCS + ["-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


class _Model(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("M", ctypes.c_int32),
        ("B", ctypes.c_int32), ("K", ctypes.c_int32),
        ("d1", ctypes.c_int32), ("d2", ctypes.c_int32),
        ("relaxed", ctypes.c_int32), ("bf16", ctypes.c_int32),
        ("slope", ctypes.c_float),
        ("ctx_w", ctypes.c_void_p), ("ctx_b", ctypes.c_void_p),
        ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
        ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p),
        ("w3", ctypes.c_void_p), ("b3", ctypes.c_void_p),
        ("table", ctypes.c_void_p), ("L", ctypes.c_int32),
        ("group", ctypes.c_int32), ("radius", ctypes.c_int32),
    ]


class _Out(ctypes.Structure):
    _fields_ = [
        ("y_hat", ctypes.c_void_p), ("mean", ctypes.c_void_p),
        ("scale", ctypes.c_void_p), ("idx", ctypes.c_void_p),
        ("weight", ctypes.c_void_p), ("comp_mean", ctypes.c_void_p),
    ]


def _load():
    global _lib
    if _lib is None:
        srcs = _SRCS + [os.path.join(_HERE, "wf_rans.h")]
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(os.path.getmtime(f) for f in srcs):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_run.argtypes = [ctypes.POINTER(_Model), ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.POINTER(_Out)]
        lib.oracle_run.restype = ctypes.c_int
        lib.oracle_eval.argtypes = [ctypes.POINTER(_Model), ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(_Out)]
        lib.oracle_eval.restype = ctypes.c_int
        lib.oracle_tap_status.argtypes = [ctypes.POINTER(_Model), ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, ctypes.c_int]
        lib.oracle_tap_status.restype = ctypes.c_int
        lib.oracle_run_bits.argtypes = [ctypes.POINTER(_Model), ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(_Out)]
        lib.oracle_run_bits.restype = ctypes.c_int
        lib.oracle_rans_tables.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int64]
        lib.oracle_rans_tables.restype = ctypes.c_int64
        lib.oracle_rans_encode.argtypes = [ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 4 + [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_rans_encode.restype = ctypes.c_int64
        lib.oracle_rans_decode.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 4 + [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
        lib.oracle_rans_decode.restype = ctypes.c_int
        lib.oracle_mix_tables.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_int64]
        lib.oracle_mix_tables.restype = ctypes.c_int64
        lib.oracle_mix_encode.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int] * 4 + [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_mix_encode.restype = ctypes.c_int64
        lib.oracle_mix_decode.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int] * 4 + [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
        lib.oracle_mix_decode.restype = ctypes.c_int
        lib.oracle_mix_latent.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        lib.oracle_mix_latent.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a):
    return None if a is None else a.ctypes.data


class Model:
    """Model description for the oracle.  ``weights`` is a dict with keys
    ctx_w [2M][M][5][5], ctx_b [2M], w1 [d1][4M], b1, w2 [d2][d1], b2,
    w3 [n3][d2], b3 (PyTorch layouts); ``table`` is the scale table.  ``group``
    N > 1 selects the context-approximation decode with groups of N
    wavefronts (N <= 1: the exact autoregressive decode).  The conv weight may
    be [2M][M][2R+1][2R+1] for any mask radius R (Def. 1); R = 2 is the 5x5
    mask."""

    def __init__(self, weights, table, H, W, B=1, K=1, relaxed=False, bf16=False,
                 slope=0.01, group=1):
        self.arrays = {k: _f32(v) for k, v in weights.items()}
        self.table = _f32(table)
        M = self.arrays["ctx_w"].shape[1]
        k = self.arrays["ctx_w"].shape[2]
        if k % 2 != 1 or self.arrays["ctx_w"].shape[3] != k:
            raise ValueError("ctx_w must be [2M][M][2R+1][2R+1]")
        self.radius = k // 2
        if relaxed and self.radius != 2:
            raise ValueError("the relaxed mask is defined for the 5x5 kernel only")
        d1 = self.arrays["w1"].shape[0]
        d2 = self.arrays["w2"].shape[0]
        n3 = self.arrays["w3"].shape[0]
        if n3 != (2 if K == 1 else 9) * M:
            raise ValueError("w3 rows do not match K and M")
        self.H, self.W, self.M, self.B, self.K = H, W, M, B, K
        self.d1, self.d2 = d1, d2
        a = self.arrays
        self._m = _Model(H, W, M, B, K, d1, d2, int(relaxed), int(bf16), slope,
                         _ptr(a["ctx_w"]), _ptr(a["ctx_b"]), _ptr(a["w1"]), _ptr(a["b1"]),
                         _ptr(a["w2"]), _ptr(a["b2"]), _ptr(a["w3"]), _ptr(a["b3"]),
                         _ptr(self.table), len(self.table), int(group), self.radius)
        self.group = int(group)

    def tap_status(self, i, j, dy, dx):
        """0: tap (dy,dx) of latent (i,j) lies outside the grid; 1: it was
        decoded in an earlier group (its value is used); 2: it belongs to the
        latent's own group (filled with the mean of the decoded taps)."""
        return _load().oracle_tap_status(ctypes.byref(self._m), i, j, dy, dx)

    def _alloc(self, n):
        M, K = self.M, self.K
        outs = {
            "y_hat": np.zeros((n, M), np.float32),
            "mean": np.zeros((n, M), np.float32),
            "scale": np.zeros((n, K, M), np.float32),
            "idx": np.zeros((n, K, M), np.int32),
            "weight": np.zeros((n, K, M), np.float32),
            "comp_mean": np.zeros((n, K, M), np.float32),
        }
        c = _Out(*(_ptr(outs[k]) for k in ("y_hat", "mean", "scale", "idx", "weight", "comp_mean")))
        return outs, c

    def _shape(self, outs):
        B, H, W = self.B, self.H, self.W
        return {k: v.reshape((B, H, W) + v.shape[1:]) for k, v in outs.items()}

    def decode(self, psi, sym, order=None):
        """Sequential decode from int32 symbols [B][H][W][M]; returns a dict of
        NHWC arrays y_hat, mean, scale, idx, weight, comp_mean (the last four
        with a component axis of length K before the channel axis)."""
        return self._run(psi, np.ascontiguousarray(sym, dtype=np.int32).copy(), None, order)[0]

    def encode(self, psi, y, order=None):
        """Sequential encode of y [B][H][W][M]; returns (outputs, symbols)."""
        sym = np.zeros((self.B, self.H, self.W, self.M), np.int32)
        return self._run(psi, sym, _f32(y), order)

    def _run(self, psi, sym, y, order):
        psi = _f32(psi)
        n = self.B * self.H * self.W
        if psi.size != n * 2 * self.M or sym.size != n * self.M:
            raise ValueError("psi / symbol shape mismatch")
        outs, c = self._alloc(n)
        ordp = None
        if order is not None:
            order = np.ascontiguousarray(order, dtype=np.int64)
            ordp = order.ctypes.data
        rc = _load().oracle_run(ctypes.byref(self._m), _ptr(psi), sym.ctypes.data,
                                _ptr(y), ordp, n if order is None else len(order),
                                ctypes.byref(c))
        if rc != 0:
            raise RuntimeError("oracle_run failed")
        return self._shape(outs), sym.reshape(self.B, self.H, self.W, self.M)

    def decode_bits(self, psi, bits, offsets):
        """Decode with the symbols read from rANS streams (``rans_encode``'s
        layout for K = 1, ``mix_encode``'s for K = 3).  Returns (outputs,
        decoded symbols)."""
        psi = _f32(psi)
        bits = np.ascontiguousarray(bits, dtype=np.uint32)
        offsets = np.ascontiguousarray(offsets, dtype=np.uint32)
        n = self.B * self.H * self.W
        if offsets.size != self.B * self.H * self.M + 1:
            raise ValueError("one offset per stream plus the total")
        sym = np.zeros((n, self.M), np.int32)
        outs, c = self._alloc(n)
        rc = _load().oracle_run_bits(ctypes.byref(self._m), _ptr(psi), bits.ctypes.data, offsets.ctypes.data,
                                     sym.ctypes.data, ctypes.byref(c))
        if rc != 0:
            raise RuntimeError("oracle_run_bits failed")
        return self._shape(outs), sym.reshape(self.B, self.H, self.W, self.M)

    def eval(self, y_hat, psi, lats=None):
        """Teacher-forced parameters from a given reconstruction, at the listed
        flat latent indices (all latents when None).  Returns flat arrays
        indexed like ``lats``."""
        y_hat = _f32(y_hat)
        psi = _f32(psi)
        latp = None
        n = self.B * self.H * self.W
        if lats is not None:
            lats = np.ascontiguousarray(lats, dtype=np.int64)
            latp = lats.ctypes.data
            n = len(lats)
        outs, c = self._alloc(n)
        rc = _load().oracle_eval(ctypes.byref(self._m), _ptr(y_hat), _ptr(psi), latp, n,
                                 ctypes.byref(c))
        if rc != 0:
            raise RuntimeError("oracle_eval failed")
        outs.pop("y_hat")
        return outs


def rans_tables(table):
    """Frequency tables of a scale table: (n [L], base [L+1], cum [base[L]])
    as built by the oracle's coder."""
    table = _f32(table)
    L = len(table)
    n = np.zeros(L, np.int32)
    base = np.zeros(L + 1, np.int64)
    total = _load().oracle_rans_tables(table.ctypes.data, L, n.ctypes.data, base.ctypes.data, None, 0)
    if total < 0:
        raise RuntimeError("oracle_rans_tables failed")
    cum = np.zeros(total, np.uint32)
    _load().oracle_rans_tables(table.ctypes.data, L, None, None, cum.ctypes.data, total)
    return n, base, cum


def rans_encode(sym, idx, table):
    """rANS streams of symbols sym [B][H][W][M] at scale indices idx (same
    shape): one stream per (image, grid row, channel).  Returns (bits uint32,
    offsets uint32 [B*H*M + 1])."""
    sym = np.ascontiguousarray(sym, dtype=np.int32)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    table = _f32(table)
    B, H, W, M = sym.shape
    offsets = np.zeros(B * H * M + 1, np.uint32)
    lib = _load()
    total = lib.oracle_rans_encode(sym.ctypes.data, idx.ctypes.data, B, H, W, M, table.ctypes.data, len(table),
                                   None, 0, offsets.ctypes.data)
    if total < 0:
        raise RuntimeError("oracle_rans_encode failed")
    bits = np.zeros(max(int(total), 1), np.uint32)
    if lib.oracle_rans_encode(sym.ctypes.data, idx.ctypes.data, B, H, W, M, table.ctypes.data, len(table),
                              bits.ctypes.data, len(bits), offsets.ctypes.data) != total:
        raise RuntimeError("oracle_rans_encode failed")
    return bits[:total], offsets


def rans_decode(bits, offsets, idx, table):
    """Symbols of rANS streams given the scale indices idx [B][H][W][M]."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    bits = np.ascontiguousarray(bits, dtype=np.uint32)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint32)
    table = _f32(table)
    B, H, W, M = idx.shape
    sym = np.zeros(idx.shape, np.int32)
    if _load().oracle_rans_decode(bits.ctypes.data, offsets.ctypes.data, idx.ctypes.data, B, H, W, M,
                                  table.ctypes.data, len(table), sym.ctypes.data) != 0:
        raise RuntimeError("oracle_rans_decode failed")
    return sym


def mix_tables(table):
    """The mixture coder's level tables: (X [L], base [L+1], G [base[L]]),
    G_l(x) for x = -X_l..X_l at base[l] + x + X_l."""
    table = _f32(table)
    L = len(table)
    X = np.zeros(L, np.int32)
    base = np.zeros(L + 1, np.int64)
    total = _load().oracle_mix_tables(table.ctypes.data, L, X.ctypes.data, base.ctypes.data, None, 0)
    if total < 0:
        raise RuntimeError("oracle_mix_tables failed")
    G = np.zeros(total, np.uint32)
    _load().oracle_mix_tables(table.ctypes.data, L, None, None, G.ctypes.data, total)
    return X, base, G


def mix_latent(table, w, cm, mu, lvl):
    """One latent channel's quantised mixture parameters and cumulative
    frequencies: dict(v, q, lo, hi, cum) with cum[u] = cum(lo + u), u = 0..S."""
    table = _f32(table)
    w = _f32(np.asarray(w).reshape(3))
    cm = _f32(np.asarray(cm).reshape(3))
    lvl = np.ascontiguousarray(np.asarray(lvl).reshape(3), dtype=np.int32)
    v = np.zeros(3, np.uint32)
    q = np.zeros(3, np.int32)
    lohi = np.zeros(2, np.int32)
    cap = 1 << 16
    cum = np.zeros(cap, np.uint32)
    S = _load().oracle_mix_latent(table.ctypes.data, len(table), w.ctypes.data, cm.ctypes.data, float(np.float32(mu)),
                                  lvl.ctypes.data, v.ctypes.data, q.ctypes.data, lohi.ctypes.data, cum.ctypes.data,
                                  cap)
    if S < 0:
        raise RuntimeError("oracle_mix_latent failed")
    return {"v": v, "q": q, "lo": int(lohi[0]), "hi": int(lohi[1]), "cum": cum[:S + 1].copy()}


def _mix_args(weight, cmean, mean, idx):
    weight = _f32(weight)
    cmean = _f32(cmean)
    mean = _f32(mean)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    B, H, W, K, M = weight.shape
    if K != 3 or cmean.shape != weight.shape or idx.shape != weight.shape or mean.shape != (B, H, W, M):
        raise ValueError("weight, comp_mean, idx: [B][H][W][3][M]; mean: [B][H][W][M]")
    return weight, cmean, mean, idx, (B, H, W, M)


def mix_encode(sym, weight, cmean, mean, idx, table):
    """rANS streams of symbols sym [B][H][W][M] under the 3-component mixture
    of weight, comp_mean, idx [B][H][W][3][M] and mixture mean [B][H][W][M]:
    one stream per (image, grid row, channel).  Returns (bits, offsets)."""
    weight, cmean, mean, idx, (B, H, W, M) = _mix_args(weight, cmean, mean, idx)
    sym = np.ascontiguousarray(sym, dtype=np.int32)
    table = _f32(table)
    offsets = np.zeros(B * H * M + 1, np.uint32)
    lib = _load()
    args = (sym.ctypes.data, weight.ctypes.data, cmean.ctypes.data, mean.ctypes.data, idx.ctypes.data, B, H, W, M,
            table.ctypes.data, len(table))
    total = lib.oracle_mix_encode(*args, None, 0, offsets.ctypes.data)
    if total < 0:
        raise RuntimeError("oracle_mix_encode failed")
    bits = np.zeros(max(int(total), 1), np.uint32)
    if lib.oracle_mix_encode(*args, bits.ctypes.data, len(bits), offsets.ctypes.data) != total:
        raise RuntimeError("oracle_mix_encode failed")
    return bits[:total], offsets


def mix_decode(bits, offsets, weight, cmean, mean, idx, table):
    """Symbols of mixture-coded streams given every latent's parameters."""
    weight, cmean, mean, idx, (B, H, W, M) = _mix_args(weight, cmean, mean, idx)
    bits = np.ascontiguousarray(bits, dtype=np.uint32)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint32)
    table = _f32(table)
    sym = np.zeros((B, H, W, M), np.int32)
    if _load().oracle_mix_decode(bits.ctypes.data, offsets.ctypes.data, weight.ctypes.data, cmean.ctypes.data,
                                 mean.ctypes.data, idx.ctypes.data, B, H, W, M, table.ctypes.data, len(table),
                                 sym.ctypes.data) != 0:
        raise RuntimeError("oracle_mix_decode failed")
    return sym
