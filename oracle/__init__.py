"""Brute-force fp64 CPU oracle for DISCO spherical convolution.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never imports, links or calls it, and it shares no code with the GPU library.

The arithmetic lives in ``disco_oracle.c`` (plain C99, fp64, OpenMP): the
finite DISCO sum of Ocampo, Price & McEwen (ICLR 2023), Sec. 3.2 eq. 4 for the
forward op and Sec. 3.5 eq. 6 for the transposed op, over every (output, input)
pixel pair.  This module only compiles it and marshals numpy arrays.

Parity pins (tests/test_oracle_pins.py) check it against closed forms, the
paper's worked node example (App. E.2), exact invariants and brute force.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "disco_oracle.c")
LIB_PATH = os.path.join(_HERE, "_build", "libdisco_oracle.so")

QUAD_FEJER1 = 0
QUAD_CELL_AREA = 1
SAMPLING_CELL_CENTRED = 0
SAMPLING_MW = 1        # pole-including (L + 1) x 2L grid of Sec. 4.2 / App. A
BASIS_BILINEAR = 0     # 3x3 node grid, K = 9
BASIS_AXISYM = 1       # 4 nodes along theta, K = 4
BASIS_SEPARABLE = 2    # 4 nodes along theta x 4 along phi, K = 16


def build(out: str = LIB_PATH, source: str = SOURCE, extra_flags=()) -> str:
    """Compile the oracle with gcc into a shared library; returns its path."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           *extra_flags, source, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


_P = ctypes.POINTER
_dp = _P(ctypes.c_double)
_i64p = _P(ctypes.c_int64)


def _ptr(a: np.ndarray, typ=_dp):
    return a.ctypes.data_as(typ)


class Oracle:
    """ctypes view of one compiled oracle library (the default, or a variant)."""

    def __init__(self, path: str = LIB_PATH):
        if not os.path.exists(path) and path == LIB_PATH:
            build(path)
        self.path = path
        lib = ctypes.CDLL(path)
        lib.oracle_colatitude.restype = ctypes.c_double
        lib.oracle_colatitude.argtypes = [ctypes.c_int, ctypes.c_int]
        lib.oracle_colatitude_s.restype = ctypes.c_double
        lib.oracle_colatitude_s.argtypes = [ctypes.c_int] * 3
        lib.oracle_quadrature_s.restype = ctypes.c_int
        lib.oracle_quadrature_s.argtypes = [ctypes.c_int] * 4 + [_dp]
        lib.oracle_basis_axisym.restype = None
        lib.oracle_basis_axisym.argtypes = [ctypes.c_double] * 2 + [_dp]
        lib.oracle_basis_separable.restype = None
        lib.oracle_basis_separable.argtypes = [ctypes.c_double] * 3 + [_dp]
        lib.oracle_psi_dense_ex.restype = ctypes.c_int
        lib.oracle_psi_dense_ex.argtypes = [ctypes.c_int] * 6 + [ctypes.c_double] * 2 + [_dp]
        lib.oracle_longitude.restype = ctypes.c_double
        lib.oracle_longitude.argtypes = [ctypes.c_int, ctypes.c_int]
        lib.oracle_quadrature.restype = ctypes.c_int
        lib.oracle_quadrature.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _dp]
        lib.oracle_frame_coords.restype = None
        lib.oracle_frame_coords.argtypes = [ctypes.c_double] * 4 + [_dp] * 3
        lib.oracle_basis.restype = None
        lib.oracle_basis.argtypes = [ctypes.c_double] * 3 + [_dp]
        lib.oracle_psi_dense.restype = ctypes.c_int
        lib.oracle_psi_dense.argtypes = [ctypes.c_int] * 4 + [ctypes.c_double] * 2 + [_dp]
        sig = ([ctypes.c_int] * 4 + [ctypes.c_double] * 2 + [ctypes.c_int] * 4 + [_dp] * 3
               + [ctypes.c_int, ctypes.c_int64, _i64p])
        for name in ("oracle_forward", "oracle_transpose"):
            f = getattr(lib, name)
            f.restype = ctypes.c_int
            f.argtypes = sig
        sig_ex = ([ctypes.c_int] * 6 + [ctypes.c_double] * 2 + [ctypes.c_int] * 4 + [_dp] * 3
                  + [ctypes.c_int, ctypes.c_int64, _i64p])
        for name in ("oracle_forward_ex", "oracle_transpose_ex"):
            f = getattr(lib, name)
            f.restype = ctypes.c_int
            f.argtypes = sig_ex
        for name in ("oracle_forward_adjoint_ex", "oracle_transpose_adjoint_ex"):
            f = getattr(lib, name)
            f.restype = ctypes.c_int
            f.argtypes = sig_ex
        lib.oracle_weight_grad_ex.restype = ctypes.c_int
        lib.oracle_weight_grad_ex.argtypes = ([ctypes.c_int] * 7 + [ctypes.c_double] * 2
                                              + [ctypes.c_int] * 4 + [_dp] * 3)
        lib.oracle_max_threads.restype = ctypes.c_int
        self.lib = lib

    # -- grid / quadrature ---------------------------------------------------
    def colatitudes(self, nlat: int, sampling: int = SAMPLING_CELL_CENTRED) -> np.ndarray:
        if sampling == SAMPLING_CELL_CENTRED:
            return np.array([self.lib.oracle_colatitude(t, nlat) for t in range(nlat)])
        return np.array([self.lib.oracle_colatitude_s(t, nlat, sampling) for t in range(nlat)])

    def longitudes(self, nlon: int) -> np.ndarray:
        return np.array([self.lib.oracle_longitude(p, nlon) for p in range(nlon)])

    def quadrature(self, nlat: int, nlon: int, kind: int = QUAD_FEJER1,
                   sampling: int = SAMPLING_CELL_CENTRED) -> np.ndarray:
        q = np.zeros(nlat)
        if sampling == SAMPLING_CELL_CENTRED:
            rc = self.lib.oracle_quadrature(nlat, nlon, kind, _ptr(q))
        else:
            rc = self.lib.oracle_quadrature_s(nlat, nlon, sampling, kind, _ptr(q))
        if rc:
            raise ValueError("oracle_quadrature failed (%d)" % rc)
        return q

    # -- geometry / basis ------------------------------------------------------
    def frame_coords(self, theta_j, phi_j, theta_i, phi_i):
        th, u, v = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        self.lib.oracle_frame_coords(theta_j, phi_j, theta_i, phi_i,
                                     ctypes.byref(th), ctypes.byref(u), ctypes.byref(v))
        return th.value, u.value, v.value

    def basis(self, u: float, v: float, h: float) -> np.ndarray:
        out = np.zeros(9)
        self.lib.oracle_basis(u, v, h, _ptr(out))
        return out

    def basis_axisym(self, Theta: float, h: float) -> np.ndarray:
        out = np.zeros(4)
        self.lib.oracle_basis_axisym(Theta, h, _ptr(out))
        return out

    def basis_separable(self, Theta: float, Phi: float, h: float) -> np.ndarray:
        out = np.zeros(16)
        self.lib.oracle_basis_separable(Theta, Phi, h, _ptr(out))
        return out

    def psi_dense(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, h=None, *,
                  sampling=SAMPLING_CELL_CENTRED, basis=BASIS_BILINEAR) -> np.ndarray:
        h = default_h(theta_c, basis) if not h else h
        n_in, n_out = nlat_in * nlon_in, nlat_out * nlon_out
        psi = np.zeros((n_out, n_in, basis_size(basis)))
        if sampling == SAMPLING_CELL_CENTRED and basis == BASIS_BILINEAR:
            rc = self.lib.oracle_psi_dense(nlat_in, nlon_in, nlat_out, nlon_out, theta_c, h, _ptr(psi))
        else:
            rc = self.lib.oracle_psi_dense_ex(nlat_in, nlon_in, nlat_out, nlon_out, sampling, basis,
                                              theta_c, h, _ptr(psi))
        if rc:
            raise ValueError("oracle_psi_dense failed (%d)" % rc)
        return psi

    # -- convolutions --------------------------------------------------------------
    def _run(self, fn, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, w, h, quad, window,
             pix, out_grid, sampling=SAMPLING_CELL_CENTRED, basis=BASIS_BILINEAR):
        x = np.ascontiguousarray(x, dtype=np.float64)
        w = np.ascontiguousarray(w, dtype=np.float64)
        B, C_x = x.shape[0], x.shape[1]
        C_y = w.shape[0] if fn == "oracle_forward" else w.shape[1]
        if w.shape[2] != basis_size(basis):
            raise ValueError("w last extent must be %d" % basis_size(basis))
        if (w.shape[1] if fn == "oracle_forward" else w.shape[0]) != C_x:
            raise ValueError("w does not match the input channels")
        if pix is None:
            pix = np.arange(out_grid[0] * out_grid[1], dtype=np.int64)
        pix = np.ascontiguousarray(pix, dtype=np.int64)
        y = np.zeros((B, C_y, pix.size))
        h = default_h(theta_c, basis) if not h else h
        if sampling == SAMPLING_CELL_CENTRED and basis == BASIS_BILINEAR:
            rc = getattr(self.lib, fn)(nlat_in, nlon_in, nlat_out, nlon_out, theta_c, h, quad,
                                       B, C_x, C_y, _ptr(x), _ptr(w), _ptr(y), int(window),
                                       pix.size, _ptr(pix, _i64p))
        else:
            rc = getattr(self.lib, fn + "_ex")(nlat_in, nlon_in, nlat_out, nlon_out, sampling,
                                               basis, theta_c, h, quad, B, C_x, C_y, _ptr(x),
                                               _ptr(w), _ptr(y), int(window), pix.size,
                                               _ptr(pix, _i64p))
        if rc:
            raise ValueError("%s failed (%d)" % (fn, rc))
        return y

    def forward(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, w, *, h=None,
                quad=QUAD_FEJER1, window=True, pix=None, sampling=SAMPLING_CELL_CENTRED,
                basis=BASIS_BILINEAR):
        """y[B, Cout, n] for x[B, Cin, nlat_in, nlon_in], w[Cout, Cin, K].

        ``pix`` selects flat out-grid pixels (default: all, returned reshaped
        to [B, Cout, nlat_out, nlon_out])."""
        y = self._run("oracle_forward", nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, w, h,
                      quad, window, pix, (nlat_out, nlon_out), sampling, basis)
        if pix is None:
            y = y.reshape(y.shape[0], y.shape[1], nlat_out, nlon_out)
        return y

    def transpose(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, w, *, h=None,
                  quad=QUAD_FEJER1, window=True, pix=None, sampling=SAMPLING_CELL_CENTRED,
                  basis=BASIS_BILINEAR):
        """Transposed op of plan (in-grid, out-grid): x[B, CinT, nlat_out, nlon_out],
        w[CinT, CoutT, K] -> y[B, CoutT, nlat_in, nlon_in] (or [B, CoutT, n])."""
        y = self._run("oracle_transpose", nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, w, h,
                      quad, window, pix, (nlat_in, nlon_in), sampling, basis)
        if pix is None:
            y = y.reshape(y.shape[0], y.shape[1], nlat_in, nlon_in)
        return y

    # -- gradients (App. C) ------------------------------------------------------
    def input_grad(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, dy, w, *, transpose=False,
                   h=None, quad=QUAD_FEJER1, window=True, pix=None, sampling=SAMPLING_CELL_CENTRED,
                   basis=BASIS_BILINEAR):
        """A^T dy for the forward op (dy[B, Cout, out-grid], w[Cout, Cin, K] ->
        dx[B, Cin, in-grid]) or, with transpose=True, for the transposed op
        (dyT[B, CoutT, in-grid], w[CinT, CoutT, K] -> dxT[B, CinT, out-grid])."""
        dy = np.ascontiguousarray(dy, dtype=np.float64)
        w = np.ascontiguousarray(w, dtype=np.float64)
        if w.shape[2] != basis_size(basis):
            raise ValueError("w last extent must be %d" % basis_size(basis))
        B, C_dy = dy.shape[0], dy.shape[1]
        C_dx = w.shape[1] if not transpose else w.shape[0]
        if (w.shape[0] if not transpose else w.shape[1]) != C_dy:
            raise ValueError("w does not match the channels of dy")
        grid = (nlat_out, nlon_out) if transpose else (nlat_in, nlon_in)
        full = pix is None
        if full:
            pix = np.arange(grid[0] * grid[1], dtype=np.int64)
        pix = np.ascontiguousarray(pix, dtype=np.int64)
        dx = np.zeros((B, C_dx, pix.size))
        h = default_h(theta_c, basis) if not h else h
        fn = self.lib.oracle_transpose_adjoint_ex if transpose else self.lib.oracle_forward_adjoint_ex
        rc = fn(nlat_in, nlon_in, nlat_out, nlon_out, sampling, basis, theta_c, h, quad, B, C_dy, C_dx,
                _ptr(dy), _ptr(w), _ptr(dx), int(window), pix.size, _ptr(pix, _i64p))
        if rc:
            raise ValueError("input_grad failed (%d)" % rc)
        return dx.reshape(B, C_dx, grid[0], grid[1]) if full else dx

    def weight_grad(self, nlat_in, nlon_in, nlat_out, nlon_out, theta_c, x, dy, *, transpose=False,
                    h=None, quad=QUAD_FEJER1, sampling=SAMPLING_CELL_CENTRED, basis=BASIS_BILINEAR):
        """dW of the forward op (x[B, Cin, in-grid], dy[B, Cout, out-grid] ->
        [Cout, Cin, K]) or of the transposed op (xT[B, CinT, out-grid],
        dyT[B, CoutT, in-grid] -> [CinT, CoutT, K])."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        dy = np.ascontiguousarray(dy, dtype=np.float64)
        B, C_x, C_dy = x.shape[0], x.shape[1], dy.shape[1]
        K = basis_size(basis)
        dw = np.zeros((C_x, C_dy, K) if transpose else (C_dy, C_x, K))
        h = default_h(theta_c, basis) if not h else h
        rc = self.lib.oracle_weight_grad_ex(int(transpose), nlat_in, nlon_in, nlat_out, nlon_out, sampling,
                                            basis, theta_c, h, quad, B, C_x, C_dy, _ptr(x), _ptr(dy),
                                            _ptr(dw))
        if rc:
            raise ValueError("weight_grad failed (%d)" % rc)
        return dw

    def max_threads(self) -> int:
        return int(self.lib.oracle_max_threads())


_default = None


def default() -> Oracle:
    """The oracle built from ``disco_oracle.c`` (compiled on first use)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            build()
        _default = Oracle(LIB_PATH)
    return _default


def default_h(theta_c: float, basis: int = BASIS_BILINEAR) -> float:
    """Node spacing.  3x3 grid: theta_c / 3 (App. E.2 puts the edge nodes at
    pi/L with a cutoff of 3 pi/L).  Axisymmetric: theta_c / 4, four nodes at
    0, h, 2h, 3h whose last hat vanishes at the cutoff."""
    return theta_c / 4.0 if basis in (BASIS_AXISYM, BASIS_SEPARABLE) else theta_c / 3.0


def basis_size(basis: int) -> int:
    return {BASIS_AXISYM: 4, BASIS_SEPARABLE: 16}.get(basis, 9)


def depthwise_weights(w_dw: np.ndarray) -> np.ndarray:
    """Depthwise channels (each channel filtered by its own filter, Sec. 4.2's
    depthwise-separable layers): the op with W[c][c'][k] = delta(c, c') w[c][k]."""
    C, K = w_dw.shape
    w = np.zeros((C, C, K))
    for c in range(C):
        w[c, c] = w_dw[c]
    return w


__all__ = ["Oracle", "build", "default", "default_h", "basis_size", "QUAD_FEJER1",
           "QUAD_CELL_AREA", "SAMPLING_CELL_CENTRED", "SAMPLING_MW", "BASIS_BILINEAR",
           "BASIS_AXISYM", "BASIS_SEPARABLE", "depthwise_weights"]
