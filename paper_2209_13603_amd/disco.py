"""ctypes binding of ``libdisco.so`` (the C ABI in ``include/disco.h``).

Argument marshalling only: every step of the forward and transposed ops runs
in the library's HIP kernels.  torch tensors supply device memory and the
current stream.  The library is loaded on first use; if it is missing the
call raises immediately (build it with ``python -m paper_2209_13603_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH

DISCO_OK = 0
DISCO_ERR_INVALID_ARGUMENT = 1
DISCO_ERR_UNSUPPORTED = 2
DISCO_ERR_SHAPE = 3
DISCO_ERR_DTYPE = 4
DISCO_ERR_OUT_OF_MEMORY = 5
DISCO_ERR_DEVICE = 6

DISCO_FLOAT32 = 0
DISCO_BFLOAT16 = 1

DISCO_BASIS_BILINEAR_3X3 = 0
DISCO_BASIS_AXISYMMETRIC_4 = 1
DISCO_BASIS_SEPARABLE_4X4 = 2
DISCO_QUAD_FEJER1 = 0
DISCO_QUAD_SAMPLING_THEOREM = 0
DISCO_QUAD_CELL_AREA = 1
DISCO_SAMPLING_CELL_CENTRED = 0
DISCO_SAMPLING_POLES = 1
BASES = {"bilinear3x3": DISCO_BASIS_BILINEAR_3X3, "axisym4": DISCO_BASIS_AXISYMMETRIC_4,
         "separable4x4": DISCO_BASIS_SEPARABLE_4X4}
BASIS_SIZE = {DISCO_BASIS_BILINEAR_3X3: 9, DISCO_BASIS_AXISYMMETRIC_4: 4, DISCO_BASIS_SEPARABLE_4X4: 16}
SAMPLINGS = {"cell_centred": DISCO_SAMPLING_CELL_CENTRED, "poles": DISCO_SAMPLING_POLES}
DISCO_PLAN_BACKWARD = 1
DISCO_PLAN_EAGER = 2

ALGO_AUTO = 0
ALGO_GATHER_THEN_CONTRACT = 1
ALGO_CONTRACT_THEN_GATHER = 2
ALGO_FUSED = 3
ALGO_FUSED_DIRECT = 4
ALGO_MATRIX_CORE = 5
ALGOS = {"auto": ALGO_AUTO, "gather_then_contract": ALGO_GATHER_THEN_CONTRACT,
         "contract_then_gather": ALGO_CONTRACT_THEN_GATHER, "fused": ALGO_FUSED,
         "fused_direct": ALGO_FUSED_DIRECT, "matrix_core": ALGO_MATRIX_CORE}

# Every exported symbol declared in include/disco.h.
EXPORTS = ("disco_plan_create", "disco_plan_destroy", "disco_plan_query", "disco_forward",
           "disco_transpose", "disco_forward_algo", "disco_transpose_algo", "disco_forward_backward",
           "disco_transpose_backward", "disco_forward_depthwise", "disco_transpose_depthwise",
           "disco_forward_depthwise_backward", "disco_transpose_depthwise_backward",
           "disco_psi_entries", "disco_forward_noalloc",
           "disco_kernel_timing_enable", "disco_kernel_timing_read", "disco_kernel_work",
           "disco_status_string", "disco_last_error", "disco_debug_bounds_violations")


def debug_bounds_violations() -> int:
    """Kernel files whose psi-index range checks failed since the last call
    (waits for the device; -1 for a library built without the checks)."""
    return int(library().disco_debug_bounds_violations())


class DiscoError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (_status_name(status), message))
        self.status = status
        self.message = message


class Basis(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("quadrature", ctypes.c_int32),
                ("node_spacing", ctypes.c_double), ("sampling", ctypes.c_int32),
                ("flags", ctypes.c_int32)]


class Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 4)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("nlat_in", ctypes.c_int32), ("nlon_in", ctypes.c_int32),
                ("nlat_out", ctypes.c_int32), ("nlon_out", ctypes.c_int32),
                ("phases_forward", ctypes.c_int32), ("phases_transpose", ctypes.c_int32),
                ("max_window", ctypes.c_int32), ("full_ring_windows", ctypes.c_int32),
                ("nnz_entries", ctypes.c_int64), ("nnz_entries_transpose", ctypes.c_int64),
                ("nnz_pairs_total", ctypes.c_int64), ("psi_bytes", ctypes.c_int64),
                ("h", ctypes.c_double), ("spectral_rings_forward", ctypes.c_int32),
                ("spectral_rings_transpose", ctypes.c_int32),
                ("sweep_patterns_forward", ctypes.c_int32),
                ("sweep_patterns_transpose", ctypes.c_int32),
                ("spectral_pairs_forward", ctypes.c_int32), ("spectral_pairs_transpose", ctypes.c_int32),
                ("spectral_slots_forward", ctypes.c_int32), ("spectral_slots_transpose", ctypes.c_int32),
                ("psi_compressed_bytes", ctypes.c_int64), ("bytes_entries", ctypes.c_int64),
                ("bytes_general", ctypes.c_int64), ("bytes_spectral", ctypes.c_int64),
                ("bytes_sweep", ctypes.c_int64), ("bytes_stencil", ctypes.c_int64),
                ("bytes_matrix_core", ctypes.c_int64), ("psi_bytes_all_layouts", ctypes.c_int64),
                ("spectral_tables_forward", ctypes.c_int32), ("spectral_tables_transpose", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def _status_name(s):
    names = {0: "DISCO_OK", 1: "DISCO_ERR_INVALID_ARGUMENT", 2: "DISCO_ERR_UNSUPPORTED",
             3: "DISCO_ERR_SHAPE", 4: "DISCO_ERR_DTYPE", 5: "DISCO_ERR_OUT_OF_MEMORY",
             6: "DISCO_ERR_DEVICE"}
    return names.get(s, "DISCO_ERR_%d" % s)


def library(path: str = None) -> ctypes.CDLL:
    """Load libdisco.so (once); raises if it has not been built.  The
    environment variable DISCO_LIBRARY names another build of it (for
    instance the range-checking libdisco_debug_bounds.so)."""
    global _lib
    if _lib is not None:
        return _lib
    if path is None:
        path = os.environ.get("DISCO_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise FileNotFoundError("libdisco.so not built at %s: run `python -m "
                                "paper_2209_13603_amd.build` (there is no CPU fallback)" % path)
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.disco_plan_create.argtypes = [ctypes.c_int] * 4 + [ctypes.c_double, P(Basis),
                                                           P(ctypes.c_void_p)]
    lib.disco_plan_destroy.argtypes = [ctypes.c_void_p]
    lib.disco_plan_query.argtypes = [ctypes.c_void_p, P(PlanInfo)]
    for name in ("disco_forward", "disco_transpose", "disco_forward_depthwise", "disco_transpose_depthwise",
                 "disco_forward_noalloc"):
        getattr(lib, name).argtypes = [ctypes.c_void_p, P(Tensor), P(Tensor), P(Tensor),
                                       ctypes.c_void_p]
    for name in ("disco_forward_algo", "disco_transpose_algo"):
        getattr(lib, name).argtypes = [ctypes.c_void_p, P(Tensor), P(Tensor), P(Tensor),
                                       ctypes.c_void_p, ctypes.c_int32]
    for name in ("disco_forward_backward", "disco_transpose_backward", "disco_forward_depthwise_backward",
                 "disco_transpose_depthwise_backward"):
        getattr(lib, name).argtypes = [ctypes.c_void_p, P(Tensor), P(Tensor), P(Tensor), P(Tensor),
                                       P(Tensor), ctypes.c_void_p]
        getattr(lib, name).restype = ctypes.c_int
    lib.disco_psi_entries.argtypes = ([ctypes.c_int] * 4 + [ctypes.c_double, P(Basis), ctypes.c_int32,
                                      ctypes.c_int64] + [P(ctypes.c_int32)] * 4
                                      + [P(ctypes.c_float), P(ctypes.c_int64), P(ctypes.c_int32),
                                         P(ctypes.c_int32)])
    for name in ("disco_plan_create", "disco_plan_destroy", "disco_plan_query", "disco_forward",
                 "disco_transpose", "disco_forward_algo", "disco_transpose_algo",
                 "disco_forward_depthwise", "disco_transpose_depthwise", "disco_psi_entries",
                 "disco_forward_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    lib.disco_kernel_timing_enable.argtypes = [ctypes.c_int32]
    lib.disco_kernel_timing_enable.restype = ctypes.c_int
    lib.disco_kernel_timing_read.argtypes = [ctypes.c_int32, ctypes.c_char_p, P(ctypes.c_int64),
                                             P(ctypes.c_double), P(ctypes.c_int32)]
    lib.disco_kernel_timing_read.restype = ctypes.c_int
    lib.disco_kernel_work.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_char_p,
                                      P(ctypes.c_int64), P(ctypes.c_int64), P(ctypes.c_int64),
                                      P(ctypes.c_int32)]
    lib.disco_kernel_work.restype = ctypes.c_int
    lib.disco_status_string.argtypes = [ctypes.c_int]
    lib.disco_status_string.restype = ctypes.c_char_p
    lib.disco_last_error.argtypes = []
    lib.disco_last_error.restype = ctypes.c_char_p
    lib.disco_debug_bounds_violations.argtypes = []
    lib.disco_debug_bounds_violations.restype = ctypes.c_int32
    _lib = lib
    return lib


def _check(status: int):
    if status != DISCO_OK:
        msg = library().disco_last_error().decode()
        raise DiscoError(status, msg)


def _basis(node_spacing=0.0, quadrature=DISCO_QUAD_FEJER1, kind=DISCO_BASIS_BILINEAR_3X3,
           sampling=DISCO_SAMPLING_CELL_CENTRED, flags=0):
    kind = BASES[kind] if isinstance(kind, str) else int(kind)
    sampling = SAMPLINGS[sampling] if isinstance(sampling, str) else int(sampling)
    return Basis(kind, quadrature, float(node_spacing), sampling, int(flags))


def _tensor(t) -> Tensor:
    import torch
    if t.dtype == torch.float32:
        dt = DISCO_FLOAT32
    elif t.dtype == torch.bfloat16:
        dt = DISCO_BFLOAT16
    else:
        dt = 99
    if not t.is_contiguous():
        raise ValueError("tensors passed to libdisco must be contiguous")
    shape = (ctypes.c_int64 * 4)(*(list(t.shape) + [0] * (4 - t.dim())))
    return Tensor(ctypes.c_void_p(t.data_ptr() if t.numel() else 0), dt, t.dim(), shape)


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Plan:
    """A DISCO plan for one (in-grid, out-grid) pair (``disco_plan_create``)."""

    def __init__(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, node_spacing=0.0,
                 quadrature=DISCO_QUAD_FEJER1, basis=DISCO_BASIS_BILINEAR_3X3,
                 sampling=DISCO_SAMPLING_CELL_CENTRED, backward=False, eager=False):
        lib = library()
        h = ctypes.c_void_p()
        b = _basis(node_spacing, quadrature, basis, sampling,
                   (DISCO_PLAN_BACKWARD if backward else 0) | (DISCO_PLAN_EAGER if eager else 0))
        _check(lib.disco_plan_create(nlat_in, nlon_in, nlat_out, nlon_out, float(theta_c),
                                     ctypes.byref(b), ctypes.byref(h)))
        self._h = h
        self.grid_in = (nlat_in, nlon_in)
        self.grid_out = (nlat_out, nlon_out)
        self.theta_c = float(theta_c)

    def close(self):
        if self._h is not None and self._h.value:
            _check(library().disco_plan_destroy(self._h))
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def info(self) -> dict:
        inf = PlanInfo()
        _check(library().disco_plan_query(self._h, ctypes.byref(inf)))
        return inf.as_dict()

    def kernel_work(self, transpose: bool, algo, c_in: int, c_out: int, dtype: str = "fp32",
                    capacity: int = 16) -> dict:
        """{kernel name: (out_pixels, in_pixels, pairs)} per batch item and channel
        for the kernels one call with these arguments launches."""
        algo = ALGOS[algo] if isinstance(algo, str) else int(algo)
        dt = DISCO_BFLOAT16 if dtype == "bf16" else DISCO_FLOAT32
        names = ctypes.create_string_buffer(64 * capacity)
        outp = (ctypes.c_int64 * capacity)()
        inp = (ctypes.c_int64 * capacity)()
        pairs = (ctypes.c_int64 * capacity)()
        count = ctypes.c_int32()
        _check(library().disco_kernel_work(self._h, int(bool(transpose)), algo, c_in, c_out, dt, capacity,
                                           names, outp, inp, pairs, ctypes.byref(count)))
        out = {}
        for i in range(min(count.value, capacity)):
            nm = names.raw[64 * i: 64 * i + 64].split(b"\0", 1)[0].decode()
            out[nm] = (int(outp[i]), int(inp[i]), int(pairs[i]))
        return out

    def _run(self, fn, x, w, y, algo, stream):
        algo = ALGOS[algo] if isinstance(algo, str) else int(algo)
        tx, tw, ty = _tensor(x), _tensor(w), _tensor(y)
        _check(getattr(library(), fn)(self._h, ctypes.byref(tx), ctypes.byref(tw),
                                      ctypes.byref(ty), _stream(stream), algo))
        return y

    def forward(self, x, w, y=None, algo="auto", stream=None):
        """y[B, Cout, nlat_out, nlon_out] = DISCO(x[B, Cin, nlat_in, nlon_in]; w[Cout, Cin, K])."""
        if y is None:
            import torch
            y = torch.empty((x.shape[0], w.shape[0]) + self.grid_out, dtype=x.dtype,
                            device=x.device)
        return self._run("disco_forward_algo", x, w, y, algo, stream)

    def forward_noalloc(self, x, w, y, stream=None):
        """disco_forward_noalloc: the forward op with its scratch memory in the
        library's fixed per-GPU array (nothing allocated; y must be given)."""
        tx, tw, ty = _tensor(x), _tensor(w), _tensor(y)
        _check(library().disco_forward_noalloc(self._h, ctypes.byref(tx), ctypes.byref(tw),
                                               ctypes.byref(ty), _stream(stream)))
        return y

    def transpose(self, x, w, y=None, algo="auto", stream=None):
        """y[B, CoutT, nlat_in, nlon_in] = DISCO^T(x[B, CinT, nlat_out, nlon_out]; w[CinT, CoutT, K])."""
        if y is None:
            import torch
            y = torch.empty((x.shape[0], w.shape[1]) + self.grid_in, dtype=x.dtype,
                            device=x.device)
        return self._run("disco_transpose_algo", x, w, y, algo, stream)

    def _run_dw(self, fn, x, w, y, stream):
        tx, tw, ty = _tensor(x), _tensor(w), _tensor(y)
        _check(getattr(library(), fn)(self._h, ctypes.byref(tx), ctypes.byref(tw), ctypes.byref(ty),
                                      _stream(stream)))
        return y

    def forward_depthwise(self, x, w, y=None, stream=None):
        """Depthwise forward op: y[B, C, out-grid], channel c = x[:, c] filtered by w[c] (w [C, K])."""
        if y is None:
            import torch
            y = torch.empty((x.shape[0], x.shape[1]) + self.grid_out, dtype=x.dtype, device=x.device)
        return self._run_dw("disco_forward_depthwise", x, w, y, stream)

    def transpose_depthwise(self, x, w, y=None, stream=None):
        """Depthwise transposed op: x[B, C, out-grid] -> y[B, C, in-grid], w [C, K]."""
        if y is None:
            import torch
            y = torch.empty((x.shape[0], x.shape[1]) + self.grid_in, dtype=x.dtype, device=x.device)
        return self._run_dw("disco_transpose_depthwise", x, w, y, stream)


def _backward(plan, fn, x, w, dy, dx, dw, stream):
    tx = _tensor(x) if x is not None else None
    tw = _tensor(w) if w is not None else None
    tdy = _tensor(dy)
    tdx = _tensor(dx) if dx is not None else None
    tdw = _tensor(dw) if dw is not None else None
    ref = lambda t: ctypes.byref(t) if t is not None else None
    _check(getattr(library(), fn)(plan._h, ref(tx), ref(tw), ref(tdy), ref(tdx), ref(tdw), _stream(stream)))
    return dx, dw


def forward_backward(plan, x, w, dy, want_dx=True, want_dw=True, stream=None):
    """Gradients of the forward op (``disco_forward_backward``): returns (dx, dw),
    None for the ones not asked for."""
    import torch
    dx = torch.empty((dy.shape[0], w.shape[1]) + plan.grid_in, dtype=dy.dtype, device=dy.device) \
        if want_dx else None
    dw = torch.empty_like(w) if want_dw else None
    return _backward(plan, "disco_forward_backward", x if want_dw else None, w if want_dx else None,
                     dy, dx, dw, stream)


def transpose_backward(plan, x, w, dy, want_dx=True, want_dw=True, stream=None):
    """Gradients of the transposed op (``disco_transpose_backward``): x[B, CinT,
    out-grid], w[CinT, CoutT, K], dy[B, CoutT, in-grid] -> (dx, dw)."""
    import torch
    dx = torch.empty((dy.shape[0], w.shape[0]) + plan.grid_out, dtype=dy.dtype, device=dy.device) \
        if want_dx else None
    dw = torch.empty_like(w) if want_dw else None
    return _backward(plan, "disco_transpose_backward", x if want_dw else None, w if want_dx else None,
                     dy, dx, dw, stream)


def forward_depthwise_backward(plan, x, w, dy, want_dx=True, want_dw=True, stream=None):
    """Gradients of the depthwise forward op (``disco_forward_depthwise_backward``):
    x[B, C, in-grid], w[C, K], dy[B, C, out-grid] -> (dx, dw)."""
    import torch
    dx = torch.empty((dy.shape[0], dy.shape[1]) + plan.grid_in, dtype=dy.dtype, device=dy.device) \
        if want_dx else None
    dw = torch.empty_like(w) if want_dw else None
    return _backward(plan, "disco_forward_depthwise_backward", x if want_dw else None, w if want_dx else None,
                     dy, dx, dw, stream)


def transpose_depthwise_backward(plan, x, w, dy, want_dx=True, want_dw=True, stream=None):
    """Gradients of the depthwise transposed op (``disco_transpose_depthwise_backward``):
    x[B, C, out-grid], w[C, K], dy[B, C, in-grid] -> (dx, dw)."""
    import torch
    dx = torch.empty((dy.shape[0], dy.shape[1]) + plan.grid_out, dtype=dy.dtype, device=dy.device) \
        if want_dx else None
    dw = torch.empty_like(w) if want_dw else None
    return _backward(plan, "disco_transpose_depthwise_backward", x if want_dw else None, w if want_dx else None,
                     dy, dx, dw, stream)


def kernel_timing(on: bool):
    """Enable or disable per-kernel event timing inside the library."""
    _check(library().disco_kernel_timing_enable(1 if on else 0))


def kernel_timing_read(capacity: int = 16) -> dict:
    """{kernel name: (launches, total milliseconds)} since the last read."""
    names = ctypes.create_string_buffer(64 * capacity)
    launches = (ctypes.c_int64 * capacity)()
    total = (ctypes.c_double * capacity)()
    count = ctypes.c_int32()
    _check(library().disco_kernel_timing_read(capacity, names, launches, total,
                                              ctypes.byref(count)))
    out = {}
    for i in range(min(count.value, capacity)):
        nm = names.raw[64 * i: 64 * i + 64].split(b"\0", 1)[0].decode()
        out[nm] = (int(launches[i]), float(total[i]))
    return out


def psi_entries(nlat_in, nlon_in, nlat_out, nlon_out, theta_c, transpose=False, node_spacing=0.0,
                quadrature=DISCO_QUAD_FEJER1, basis=DISCO_BASIS_BILINEAR_3X3,
                sampling=DISCO_SAMPLING_CELL_CENTRED) -> dict:
    """Host-only export of the stored psi entries of the forward (or transposed) op."""
    lib = library()
    b = _basis(node_spacing, quadrature, basis, sampling)
    count = ctypes.c_int64()
    phases = ctypes.c_int32()
    stride = ctypes.c_int32()
    null_i = ctypes.POINTER(ctypes.c_int32)()
    null_f = ctypes.POINTER(ctypes.c_float)()
    _check(lib.disco_psi_entries(nlat_in, nlon_in, nlat_out, nlon_out, float(theta_c),
                                 ctypes.byref(b), int(transpose), 0, null_i, null_i, null_i,
                                 null_i, null_f, ctypes.byref(count), ctypes.byref(phases),
                                 ctypes.byref(stride)))
    n = count.value
    arrs = {k: np.zeros(n, dtype=np.int32) for k in ("out_ring", "phase", "in_ring", "offset")}
    vals = np.zeros((n, 16 if basis == DISCO_BASIS_SEPARABLE_4X4 else 9), dtype=np.float32)
    ip = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    _check(lib.disco_psi_entries(nlat_in, nlon_in, nlat_out, nlon_out, float(theta_c),
                                 ctypes.byref(b), int(transpose), n, ip(arrs["out_ring"]),
                                 ip(arrs["phase"]), ip(arrs["in_ring"]), ip(arrs["offset"]),
                                 vals.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                 ctypes.byref(count), ctypes.byref(phases), ctypes.byref(stride)))
    arrs["values"] = vals
    arrs["phases"] = phases.value
    arrs["stride"] = stride.value
    return arrs
