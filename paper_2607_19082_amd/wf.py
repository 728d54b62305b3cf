"""Python binding of libwf (ctypes): argument marshalling only.

Every step of the decode/encode runs in the library's HIP kernels; this module
only checks tensor shapes/dtypes/devices and passes raw device pointers and the
current HIP stream.  It raises if the library is missing; there is no fallback.
"""
import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libwf.so")

WF_OK, WF_E_INVALID, WF_E_UNSUPPORTED, WF_E_HIP, WF_E_NOMEM, WF_E_TIMEOUT = 0, -1, -2, -3, -4, -5
WF_E_STREAM, WF_E_CAPACITY = -6, -7
ENTROPY_CODER = {None: 0, "none": 0, "rans": 1}
MASK = {"full": 0, "relaxed": 1, "3x3": 2, "7x7": 3}
PARAM_ORDER = {"native": 0, "scales_first": 1}
KERNEL = {"full": 5, "relaxed": 5, "3x3": 3, "7x7": 7}   # ctx_w's spatial size per mask
PRECISION = {"fp32": 0, "bf16": 1}
DRIVER = {"stream": 0, "graph": 1, "persistent": 2, "dataflow": 3, "resident": 4}

EXPORTS = ["wf_schedule", "wf_validate", "wf_plan", "wf_plan_schedule", "wf_plan_deps", "wf_plan_set_waits", "wf_litmus", "wf_decode",
           "wf_encode", "wf_ec_tables", "wf_mix_tables", "wf_encode_bits", "wf_decode_bits", "wf_plan_trace",
           "wf_measure_floor", "wf_plan_sync", "wf_xform_plan", "wf_hyper_synthesis", "wf_synthesis",
           "wf_decode_noalloc", "wf_xform_destroy", "wf_plan_destroy", "wf_last_error"]


class WfError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libwf error {code}: {msg}")
        self.code = code


class Desc(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("M", ctypes.c_int32),
        ("B", ctypes.c_int32), ("K", ctypes.c_int32),
        ("d1", ctypes.c_int32), ("d2", ctypes.c_int32),
        ("mask", ctypes.c_int32), ("precision", ctypes.c_int32), ("driver", ctypes.c_int32),
        ("lrelu_slope", ctypes.c_float),
        ("ctx_w", ctypes.c_void_p), ("ctx_b", ctypes.c_void_p),
        ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
        ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p),
        ("w3", ctypes.c_void_p), ("b3", ctypes.c_void_p),
        ("scale_table", ctypes.c_void_p), ("L", ctypes.c_int32),
        ("group", ctypes.c_int32), ("param_order", ctypes.c_int32),
        ("entropy_coder", ctypes.c_int32), ("cu_limit", ctypes.c_int32),
    ]


class XformDesc(ctypes.Structure):
    _fields_ = [
        ("N", ctypes.c_int32), ("M", ctypes.c_int32), ("B", ctypes.c_int32),
        ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("precision", ctypes.c_int32),
        ("hs_w", ctypes.c_void_p * 3), ("hs_b", ctypes.c_void_p * 3),
        ("gs_w", ctypes.c_void_p * 4), ("gs_b", ctypes.c_void_p * 4),
        ("gdn_beta", ctypes.c_void_p * 3), ("gdn_gamma", ctypes.c_void_p * 3),
    ]


class Out(ctypes.Structure):
    _fields_ = [
        ("y_hat", ctypes.c_void_p), ("mean", ctypes.c_void_p), ("scale", ctypes.c_void_p),
        ("idx", ctypes.c_void_p), ("weight", ctypes.c_void_p), ("comp_mean", ctypes.c_void_p),
    ]


_lib = None


def lib():
    """Load libwf.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2607_19082_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.wf_schedule.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P, P, P]
        L.wf_validate.argtypes = [ctypes.POINTER(Desc)]
        L.wf_plan.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(ctypes.c_void_p)]
        L.wf_plan_schedule.argtypes = [P, P, P]
        L.wf_plan_deps.argtypes = [ctypes.POINTER(Desc), P, ctypes.c_int64, P]
        L.wf_litmus.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P, P]
        L.wf_plan_set_waits.argtypes = [P, ctypes.c_int64, ctypes.c_int32]
        L.wf_decode.argtypes = [P, P, P, ctypes.POINTER(Out), P]
        L.wf_decode_noalloc.argtypes = [P, P, P, ctypes.POINTER(Out), P]
        L.wf_encode.argtypes = [P, P, P, P, ctypes.POINTER(Out), P]
        L.wf_ec_tables.argtypes = [P, ctypes.c_int32, P, P, P, ctypes.c_int64]
        L.wf_mix_tables.argtypes = [P, ctypes.c_int32, P, P, P, ctypes.c_int64]
        L.wf_encode_bits.argtypes = [P, P, P, P, ctypes.POINTER(Out), P, ctypes.c_int64, P, P]
        L.wf_decode_bits.argtypes = [P, P, P, ctypes.c_int64, P, P, ctypes.POINTER(Out), P]
        L.wf_xform_plan.argtypes = [ctypes.POINTER(XformDesc), ctypes.POINTER(ctypes.c_void_p)]
        L.wf_hyper_synthesis.argtypes = [P, P, P, P]
        L.wf_synthesis.argtypes = [P, P, P, P]
        L.wf_xform_destroy.argtypes = [P]
        L.wf_plan_trace.argtypes = [P, P, ctypes.c_int64, P, P]
        L.wf_measure_floor.argtypes = [P, P, P]
        L.wf_plan_sync.argtypes = [P, P]
        L.wf_plan_destroy.argtypes = [P]
        L.wf_plan_destroy.restype = None
        L.wf_last_error.restype = ctypes.c_char_p
        for name in EXPORTS[:-2]:
            getattr(L, name).restype = ctypes.c_int
        L.wf_xform_destroy.restype = None
        _lib = L
    return _lib


def _check(rc):
    if rc != WF_OK:
        raise WfError(rc, lib().wf_last_error().decode())


def schedule(H, W, mask="full"):
    """(step_of [H][W] int32, n_steps, lambda) from the library's host planner."""
    step = np.zeros((H, W), np.int32)
    n = ctypes.c_int32()
    lam = ctypes.c_int32()
    _check(lib().wf_schedule(H, W, MASK[mask], step.ctypes.data, ctypes.byref(n), ctypes.byref(lam)))
    return step, n.value, lam.value


def make_desc(weights, table, H, W, B=1, K=1, mask="full", precision="fp32", driver="stream",
              slope=0.01, group=1, param_order="native", entropy_coder=None, cu_limit=0):
    """Build a Desc plus the host arrays it points to (keep both alive)."""
    arrs = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in weights.items()}
    arrs["table"] = np.ascontiguousarray(table, dtype=np.float32)
    M = arrs["ctx_w"].shape[1]
    k = KERNEL[mask]
    if arrs["ctx_w"].shape != (2 * M, M, k, k):
        raise ValueError(f"ctx_w must have shape (2M, M, {k}, {k}) for the {mask} mask, got {arrs['ctx_w'].shape}")
    d = Desc(H, W, M, B, K, arrs["w1"].shape[0], arrs["w2"].shape[0], MASK[mask],
             PRECISION[precision], DRIVER[driver], slope,
             arrs["ctx_w"].ctypes.data, arrs["ctx_b"].ctypes.data,
             arrs["w1"].ctypes.data, arrs["b1"].ctypes.data,
             arrs["w2"].ctypes.data, arrs["b2"].ctypes.data,
             arrs["w3"].ctypes.data, arrs["b3"].ctypes.data,
             arrs["table"].ctypes.data, len(arrs["table"]), group, PARAM_ORDER[param_order],
             ENTROPY_CODER[entropy_coder], cu_limit)
    return d, arrs


def validate(desc):
    return lib().wf_validate(ctypes.byref(desc))


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Plan:
    """A plan for one model and grid shape.  Inputs/outputs are torch tensors
    on the current HIP device; calls are asynchronous on the given (default:
    current) torch stream."""

    def __init__(self, weights, table, H, W, B=1, K=1, mask="full", precision="fp32",
                 driver="stream", slope=0.01, group=1, param_order="native", entropy_coder=None, cu_limit=0):
        self.desc, self._arrs = make_desc(weights, table, H, W, B, K, mask, precision, driver, slope, group,
                                          param_order, entropy_coder, cu_limit)
        self.group = group
        self.H, self.W, self.B, self.K = H, W, B, K
        self.M = self.desc.M
        h = ctypes.c_void_p()
        _check(lib().wf_plan(ctypes.byref(self.desc), ctypes.byref(h)))
        self._h = h
        self._arrs = None  # the plan holds device copies

    def close(self):
        if getattr(self, "_h", None):
            lib().wf_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_waits(self, spin_budget_ticks=0, stall=0):
        """The in-launch drivers' wait budget (100 MHz ticks; 0: 1 s) and the
        stall test hook (wf_plan_set_waits), for the calls that follow."""
        _check(lib().wf_plan_set_waits(self._h, int(spin_budget_ticks), int(stall)))

    def schedule(self):
        step = np.zeros((self.H, self.W), np.int32)
        n = ctypes.c_int32()
        _check(lib().wf_plan_schedule(self._h, step.ctypes.data, ctypes.byref(n)))
        return step, n.value

    def alloc_out(self):
        import torch
        B, H, W, M, K = self.B, self.H, self.W, self.M, self.K
        dev = torch.device("cuda", torch.cuda.current_device())
        o = {
            "y_hat": torch.empty((B, H, W, M), dtype=torch.float32, device=dev),
            "mean": torch.empty((B, H, W, M), dtype=torch.float32, device=dev),
            "scale": torch.empty((B, H, W, K, M), dtype=torch.float32, device=dev),
            "idx": torch.empty((B, H, W, K, M), dtype=torch.int32, device=dev),
        }
        if K == 3:
            o["weight"] = torch.empty((B, H, W, K, M), dtype=torch.float32, device=dev)
            o["comp_mean"] = torch.empty((B, H, W, K, M), dtype=torch.float32, device=dev)
        return o

    def _check_tensor(self, t, shape, dtype, name):
        import torch
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError(f"{name} must be a CUDA (HIP) tensor")
        if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
        return ctypes.c_void_p(t.data_ptr())

    def _out_struct(self, out):
        import torch
        B, H, W, M, K = self.B, self.H, self.W, self.M, self.K
        f = torch.float32
        ptrs = [self._check_tensor(out["y_hat"], (B, H, W, M), f, "y_hat"),
                self._check_tensor(out["mean"], (B, H, W, M), f, "mean"),
                self._check_tensor(out["scale"], (B, H, W, K, M), f, "scale"),
                self._check_tensor(out["idx"], (B, H, W, K, M), torch.int32, "idx")]
        if K == 3:
            ptrs += [self._check_tensor(out["weight"], (B, H, W, K, M), f, "weight"),
                     self._check_tensor(out["comp_mean"], (B, H, W, K, M), f, "comp_mean")]
        else:
            ptrs += [None, None]
        return Out(*[p.value if p is not None else None for p in ptrs])

    def decode(self, psi, sym, out=None, stream=None):
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        out = out if out is not None else self.alloc_out()
        p_psi = self._check_tensor(psi, (B, H, W, 2 * M), torch.float32, "psi")
        p_sym = self._check_tensor(sym, (B, H, W, M), torch.int32, "sym")
        o = self._out_struct(out)
        _check(lib().wf_decode(self._h, p_psi, p_sym, ctypes.byref(o), _stream_handle(stream)))
        return out

    def decode_noalloc(self, psi, sym, out, stream=None):
        """wf_decode_noalloc: the same decode with the call's working memory in
        the library's static device array (the outputs must be given)."""
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        p_psi = self._check_tensor(psi, (B, H, W, 2 * M), torch.float32, "psi")
        p_sym = self._check_tensor(sym, (B, H, W, M), torch.int32, "sym")
        o = self._out_struct(out)
        _check(lib().wf_decode_noalloc(self._h, p_psi, p_sym, ctypes.byref(o), _stream_handle(stream)))
        return out

    def encode(self, psi, y, out=None, sym_out=None, stream=None):
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        out = out if out is not None else self.alloc_out()
        if sym_out is None:
            sym_out = torch.empty((B, H, W, M), dtype=torch.int32, device=y.device)
        p_psi = self._check_tensor(psi, (B, H, W, 2 * M), torch.float32, "psi")
        p_y = self._check_tensor(y, (B, H, W, M), torch.float32, "y")
        p_s = self._check_tensor(sym_out, (B, H, W, M), torch.int32, "sym_out")
        o = self._out_struct(out)
        _check(lib().wf_encode(self._h, p_psi, p_y, p_s, ctypes.byref(o), _stream_handle(stream)))
        return out, sym_out

    def encode_bits(self, psi, y, bits, out=None, sym_out=None, stream=None):
        """Encode and code the symbols into rANS streams: `bits` is a uint32
        (int32 view) CUDA tensor of any length; returns (out, sym_out,
        offsets) with offsets [B*H*M + 1] (int32 view of uint32; the last
        entry is the total word count, valid after sync)."""
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        out = out if out is not None else self.alloc_out()
        if sym_out is None:
            sym_out = torch.empty((B, H, W, M), dtype=torch.int32, device=y.device)
        offsets = torch.empty(B * H * M + 1, dtype=torch.int32, device=y.device)
        p_psi = self._check_tensor(psi, (B, H, W, 2 * M), torch.float32, "psi")
        p_y = self._check_tensor(y, (B, H, W, M), torch.float32, "y")
        p_s = self._check_tensor(sym_out, (B, H, W, M), torch.int32, "sym_out")
        p_b = self._check_tensor(bits, (bits.numel(),), torch.int32, "bits")
        p_o = self._check_tensor(offsets, (B * H * M + 1,), torch.int32, "offsets")
        o = self._out_struct(out)
        _check(lib().wf_encode_bits(self._h, p_psi, p_y, p_s, ctypes.byref(o), p_b, bits.numel(), p_o,
                                    _stream_handle(stream)))
        return out, sym_out, offsets

    def decode_bits(self, psi, bits, offsets, out=None, sym_out=None, n_words=None, stream=None):
        """Decode with the symbols read from rANS streams (`bits`, `offsets`
        as written by encode_bits, int32 views).  Returns (out, sym_out)."""
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        out = out if out is not None else self.alloc_out()
        if sym_out is None:
            sym_out = torch.empty((B, H, W, M), dtype=torch.int32, device=psi.device)
        p_psi = self._check_tensor(psi, (B, H, W, 2 * M), torch.float32, "psi")
        p_b = self._check_tensor(bits, (bits.numel(),), torch.int32, "bits")
        p_o = self._check_tensor(offsets, (B * H * M + 1,), torch.int32, "offsets")
        p_s = self._check_tensor(sym_out, (B, H, W, M), torch.int32, "sym_out")
        o = self._out_struct(out)
        n = bits.numel() if n_words is None else int(n_words)
        if not 0 <= n <= bits.numel():
            raise ValueError(f"n_words must lie in [0, bits.numel()] = [0, {bits.numel()}], got {n}")
        _check(lib().wf_decode_bits(self._h, p_psi, p_b, n, p_o, p_s, ctypes.byref(o), _stream_handle(stream)))
        return out, sym_out

    def trace(self, stamps=None):
        """Record barrier timestamps of later calls into the int64 CUDA tensor
        `stamps` (None: stop).  Returns (entries needed per call, grid)."""
        needed = ctypes.c_int64()
        grid = ctypes.c_int32()
        ptr = ctypes.c_void_p(stamps.data_ptr()) if stamps is not None else None
        cap = stamps.numel() if stamps is not None else 0
        _check(lib().wf_plan_trace(self._h, ptr, cap, ctypes.byref(needed), ctypes.byref(grid)))
        return needed.value, grid.value

    def measure_floor(self):
        """(graph node us, barrier round us) latency floors on this device."""
        node = ctypes.c_float()
        bar = ctypes.c_float()
        _check(lib().wf_measure_floor(self._h, ctypes.byref(node), ctypes.byref(bar)))
        return node.value, bar.value

    def sync(self, stream=None):
        _check(lib().wf_plan_sync(self._h, _stream_handle(stream)))


def ec_tables(table):
    """The library's rANS frequency tables of a scale table (host only):
    (n [L], base [L+1], cum [base[L]] uint32)."""
    table = np.ascontiguousarray(table, dtype=np.float32)
    L = len(table)
    n = np.zeros(L, np.int32)
    base = np.zeros(L + 1, np.int64)
    _check(lib().wf_ec_tables(table.ctypes.data, L, n.ctypes.data, base.ctypes.data, None, 0))
    cum = np.zeros(int(base[-1]), np.uint32)
    _check(lib().wf_ec_tables(table.ctypes.data, L, None, None, cum.ctypes.data, len(cum)))
    return n, base, cum


def plan_deps(desc):
    """The dependency lists of the dataflow or resident driver for a plan
    description (host only): the flat int32 array of wf_plan_deps."""
    n = ctypes.c_int64(0)
    _check(lib().wf_plan_deps(ctypes.byref(desc), None, 0, ctypes.byref(n)))
    out = np.zeros(n.value, np.int32)
    _check(lib().wf_plan_deps(ctypes.byref(desc), out.ctypes.data, len(out), ctypes.byref(n)))
    return out


def litmus(mode, pairs, rounds, stream=None):
    """The cross-XCD coherence litmus test (wf_litmus): the number of words
    a consumer read wrong."""
    n = ctypes.c_uint64(0)
    _check(lib().wf_litmus(mode, pairs, rounds, ctypes.byref(n), _stream_handle(stream)))
    return n.value


def mix_tables(table):
    """The library's mixture-coder level tables of a scale table (host only):
    (X [L], base [L+1], G [base[L]] uint32)."""
    table = np.ascontiguousarray(table, dtype=np.float32)
    L = len(table)
    X = np.zeros(L, np.int32)
    base = np.zeros(L + 1, np.int64)
    _check(lib().wf_mix_tables(table.ctypes.data, L, X.ctypes.data, base.ctypes.data, None, 0))
    G = np.zeros(int(base[-1]), np.uint32)
    _check(lib().wf_mix_tables(table.ctypes.data, L, None, None, G.ctypes.data, len(G)))
    return X, base, G


class Xform:
    """The hyper-decoder and synthesis transforms on the GPU (weights as drawn
    by inputs.make_transform_weights, PyTorch layouts).  Calls take and return
    torch tensors on the current HIP device, asynchronously on the stream."""

    def __init__(self, weights, N, M, B, H, W, precision="fp32"):
        a = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in weights.items()}
        M2 = M * 3 // 2
        shapes = {"hs1_w": (N, M, 5, 5), "hs2_w": (M, M2, 5, 5), "hs3_w": (2 * M, M2, 3, 3),
                  "gs1_w": (M, N, 5, 5), "gs2_w": (N, N, 5, 5), "gs3_w": (N, N, 5, 5), "gs4_w": (N, 3, 5, 5)}
        for k, shp in shapes.items():
            if a[k].shape != shp:
                raise ValueError(f"{k} must have shape {shp}, got {a[k].shape}")
        d = XformDesc(N, M, B, H, W, PRECISION[precision])
        for k in range(3):
            d.hs_w[k] = a[f"hs{k + 1}_w"].ctypes.data
            d.hs_b[k] = a[f"hs{k + 1}_b"].ctypes.data
            d.gdn_beta[k] = a[f"gdn{k + 1}_beta"].ctypes.data
            d.gdn_gamma[k] = a[f"gdn{k + 1}_gamma"].ctypes.data
        for k in range(4):
            d.gs_w[k] = a[f"gs{k + 1}_w"].ctypes.data
            d.gs_b[k] = a[f"gs{k + 1}_b"].ctypes.data
        h = ctypes.c_void_p()
        _check(lib().wf_xform_plan(ctypes.byref(d), ctypes.byref(h)))
        self._h = h
        self.N, self.M, self.B, self.H, self.W = N, M, B, H, W

    def close(self):
        if getattr(self, "_h", None):
            lib().wf_xform_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def _ptr(t, shape, name):
        import torch
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 or \
                tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError(f"{name}: expected a contiguous fp32 CUDA tensor {tuple(shape)}")
        return ctypes.c_void_p(t.data_ptr())

    def hyper_synthesis(self, z_hat, psi=None, stream=None):
        import torch
        B, H, W, N, M = self.B, self.H, self.W, self.N, self.M
        if psi is None:
            psi = torch.empty((B, H, W, 2 * M), dtype=torch.float32, device=z_hat.device)
        _check(lib().wf_hyper_synthesis(self._h, self._ptr(z_hat, (B, -(-H // 4), -(-W // 4), N), "z_hat"),
                                        self._ptr(psi, (B, H, W, 2 * M), "psi"), _stream_handle(stream)))
        return psi

    def synthesis(self, y_hat, image=None, stream=None):
        import torch
        B, H, W, M = self.B, self.H, self.W, self.M
        if image is None:
            image = torch.empty((B, 16 * H, 16 * W, 3), dtype=torch.float32, device=y_hat.device)
        _check(lib().wf_synthesis(self._h, self._ptr(y_hat, (B, H, W, M), "y_hat"),
                                  self._ptr(image, (B, 16 * H, 16 * W, 3), "image"), _stream_handle(stream)))
        return image
