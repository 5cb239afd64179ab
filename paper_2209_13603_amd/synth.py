"""Seeded synthetic inputs for the DISCO workloads.

This module holds the workload definitions (grid sizes, cutoff, batch,
channels, storage dtype) and the seeded input generators.  It holds none of the
convolution's arithmetic, and both the GPU path's tests and the oracle's tests
draw their inputs from it.

Recipe (per workload, one ``numpy.random.default_rng(seed)`` stream, PCG64):
  * x first, in C order [B, C, nlat, nlon], then w in C order [.., .., 9];
  * values are drawn in float64 and rounded to the storage dtype with
    round-to-nearest-even (fp32 or bf16); the oracle consumes exactly the
    rounded values;
  * x ~ N(0, 1) and w ~ N(0, 1 / (C_in * 9)), where C_in counts the channels
    the op reads;
  * the 2048 x 4096 workload replaces x by a smooth band-limited field: per
    channel, 64 real spherical harmonics (l, m) drawn without replacement from
    1 <= l <= 16, 0 <= m <= l, random phases and N(0, 1) amplitudes,
    normalised to unit area-weighted RMS, plus N(0, 0.1^2) white noise;
  * the paper's own timed layer (one channel, batch 1, the axisymmetric
    four-node basis, theta_c = 3 pi / L on the pole-including (L + 1) x 2L
    grid, L = 1024, 2048, 4096) takes the same field evaluated on that grid,
    and w ~ N(0, 1 / 4);
  * depthwise workloads (each channel filtered by its own w[c], the
    depthwise half of a depthwise-separable layer) draw w [C, K] ~ N(0, 1 / K).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

K_BASIS = 9
BASIS_K = {"bilinear3x3": 9, "axisym4": 4, "separable4x4": 16}
BASIS_CODE = {"bilinear3x3": 0, "axisym4": 1, "separable4x4": 2}


@dataclass(frozen=True)
class Workload:
    """One benchmark / parity configuration.

    The plan is always (in-grid -> out-grid) of the forward op; for
    ``op == "transpose"`` the op maps the plan's out-grid back to its in-grid.
    """
    name: str
    nlat_in: int
    nlon_in: int
    nlat_out: int
    nlon_out: int
    theta_c: float
    batch: int
    c_in: int           # channels the op reads
    c_out: int          # channels the op writes
    dtype: str          # storage dtype of x, w, y: "fp32" or "bf16"
    op: str             # "forward" or "transpose"
    seed: int
    field: str = "normal"  # "normal" or "sh_field"
    basis: str = "bilinear3x3"     # "bilinear3x3" (K = 9), "axisym4" (K = 4) or "separable4x4" (K = 16)
    sampling: str = "cell_centred"  # "cell_centred" or "poles" ((L + 1) x 2L with both poles)
    channels: str = "full"         # "full" (W [Cout, Cin, K]) or "depthwise" (w [C, K], Cin = Cout = C)

    @property
    def K(self) -> int:
        return BASIS_K[self.basis]

    def plan_kwargs(self) -> dict:
        """Keyword arguments of ``disco.Plan`` beyond the grid and cutoff."""
        return {"basis": self.basis, "sampling": self.sampling}

    def oracle_kwargs(self) -> dict:
        """The same choice in the oracle's integer codes."""
        return {"basis": BASIS_CODE[self.basis],
                "sampling": 1 if self.sampling == "poles" else 0}

    @property
    def depthwise(self) -> bool:
        return self.channels == "depthwise"

    @property
    def x_shape(self):
        if self.op == "forward":
            return (self.batch, self.c_in, self.nlat_in, self.nlon_in)
        return (self.batch, self.c_in, self.nlat_out, self.nlon_out)

    @property
    def y_shape(self):
        if self.op == "forward":
            return (self.batch, self.c_out, self.nlat_out, self.nlon_out)
        return (self.batch, self.c_out, self.nlat_in, self.nlon_in)

    @property
    def w_shape(self):
        # forward: W[Cout][Cin][K]; transpose: W[CinT][CoutT][K] (the adjoint
        # pair shares one buffer); depthwise: w[C][K].
        if self.depthwise:
            return (self.c_in, self.K)
        if self.op == "forward":
            return (self.c_out, self.c_in, self.K)
        return (self.c_in, self.c_out, self.K)

    @property
    def out_pix_chan(self) -> int:
        b, c, a, n = self.y_shape
        return b * c * a * n

    def plan_args(self):
        return (self.nlat_in, self.nlon_in, self.nlat_out, self.nlon_out, self.theta_c)


WORKLOADS = {
    "sphere32x64": Workload("sphere32x64", 32, 64, 32, 64, 3 * math.pi / 32, 1, 4, 4, "fp32",
                            "forward", 0),
    "down128x256_to_64x128": Workload("down128x256_to_64x128", 128, 256, 64, 128,
                                      3 * math.pi / 64, 4, 16, 16, "fp32", "forward", 1),
    "sphere512x1024": Workload("sphere512x1024", 512, 1024, 512, 1024, 3 * math.pi / 512, 2,
                               32, 32, "fp32", "forward", 2),
    "up256x512_to_512x1024_bf16": Workload("up256x512_to_512x1024_bf16", 512, 1024, 256, 512,
                                           3 * math.pi / 256, 4, 64, 32, "bf16", "transpose",
                                           3),
    "sphere2048x4096": Workload("sphere2048x4096", 2048, 4096, 2048, 4096, 3 * math.pi / 2048,
                                1, 8, 8, "fp32", "forward", 4, "sh_field"),
}
# The paper's own timed layer (App. B), L = 1024, 2048, 4096.
for _i, _L in enumerate((1024, 2048, 4096)):
    _n = "poles_axisym_L%d" % _L
    WORKLOADS[_n] = Workload(_n, _L + 1, 2 * _L, _L + 1, 2 * _L, 3 * math.pi / _L, 1, 1, 1, "fp32",
                             "forward", 5 + _i, "sh_field", "axisym4", "poles")
# The separable four-by-four basis with depthwise channels (the filtering half
# of the paper's depthwise-separable DISCO layers) on the 2048 x 4096 sphere,
# eight channels, and its transpose on the 2x upsampling of the 256 x 512 grid.
WORKLOADS["sphere2048x4096_separable_dw"] = Workload(
    "sphere2048x4096_separable_dw", 2048, 4096, 2048, 4096, 3 * math.pi / 2048, 1, 8, 8, "fp32",
    "forward", 8, "sh_field", "separable4x4", "cell_centred", "depthwise")
WORKLOADS["up256x512_to_512x1024_separable_dw"] = Workload(
    "up256x512_to_512x1024_separable_dw", 512, 1024, 256, 512, 3 * math.pi / 256, 4, 32, 32, "fp32",
    "transpose", 9, "normal", "separable4x4", "cell_centred", "depthwise")

# The headline workload: forward on the 2048 x 4096 sphere.
HEADLINE = "sphere2048x4096"


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float64/float32 values to bfloat16 (nearest-even), returned as float32."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    out = u.astype(np.uint32).view(np.float32)
    # NaN stays NaN (inputs here are finite; kept for completeness).
    return np.where(np.isnan(f), f, out)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage precision (returned as float32 holding exact values)."""
    if dtype == "fp32":
        return np.asarray(a, dtype=np.float32)
    if dtype == "bf16":
        return round_to_bf16(a)
    raise ValueError(dtype)


def _assoc_legendre(lmax: int, x: np.ndarray) -> dict:
    """P_l^m(x) for 0 <= m <= l <= lmax (no Condon-Shortley phase), by the
    standard three-term recurrence in l at fixed m."""
    s = np.sqrt(np.maximum(0.0, 1.0 - x * x))
    P = {}
    pmm = np.ones_like(x)
    for m in range(lmax + 1):
        if m > 0:
            pmm = pmm * (2 * m - 1) * s
        P[(m, m)] = pmm
        if m + 1 <= lmax:
            P[(m + 1, m)] = x * (2 * m + 1) * pmm
        for l in range(m + 2, lmax + 1):
            P[(l, m)] = ((2 * l - 1) * x * P[(l - 1, m)] - (l + m - 1) * P[(l - 2, m)]) / (l - m)
    return P


def colatitudes(nlat: int, sampling: str = "cell_centred") -> np.ndarray:
    """Ring colatitudes of either grid (cell-centred, or both poles included)."""
    if sampling == "poles":
        return np.arange(nlat) * math.pi / (nlat - 1)
    return (np.arange(nlat) + 0.5) * math.pi / nlat


def sh_field(rng: np.random.Generator, nlat: int, nlon: int, n_terms: int = 64,
             lmax: int = 16, noise: float = 0.1, sampling: str = "cell_centred") -> np.ndarray:
    """One channel of the smooth random field (see module docstring)."""
    pairs = [(l, m) for l in range(1, lmax + 1) for m in range(0, l + 1)]
    pick = rng.choice(len(pairs), size=n_terms, replace=False)
    alpha = rng.uniform(0.0, 2.0 * math.pi, size=n_terms)
    amp = rng.standard_normal(n_terms)
    theta = colatitudes(nlat, sampling)
    phi = 2.0 * math.pi * np.arange(nlon) / nlon
    P = _assoc_legendre(lmax, np.cos(theta))
    # f = sum_m A_m(theta) cos(m phi) + B_m(theta) sin(m phi)
    A = np.zeros((nlat, lmax + 1))
    Bm = np.zeros((nlat, lmax + 1))
    for n, idx in enumerate(pick):
        l, m = pairs[idx]
        norm = math.sqrt((2 * l + 1) / (4 * math.pi) * math.factorial(l - m) / math.factorial(l + m))
        if m > 0:
            norm *= math.sqrt(2.0)
        col = amp[n] * norm * P[(l, m)]
        A[:, m] += col * math.cos(alpha[n])
        Bm[:, m] -= col * math.sin(alpha[n])
    ms = np.arange(lmax + 1)
    f = A @ np.cos(np.outer(ms, phi)) + Bm @ np.sin(np.outer(ms, phi))
    area = np.sin(theta)[:, None]
    rms = math.sqrt(float((area * f * f).sum() / (area.sum() * nlon)))
    f = f / rms
    return f + noise * rng.standard_normal((nlat, nlon))


def make_inputs(wl: Workload, batch: int | None = None):
    """Seeded (x, w) for a workload, as float32 arrays holding storage-exact values."""
    rng = np.random.default_rng(wl.seed)
    xs = list(wl.x_shape)
    if batch is not None:
        xs[0] = batch
    if wl.field == "sh_field":
        x = np.empty(xs)
        for b in range(xs[0]):
            for c in range(xs[1]):
                x[b, c] = sh_field(rng, xs[2], xs[3], sampling=wl.sampling)
    else:
        x = rng.standard_normal(xs)
    fan_in = wl.K if wl.depthwise else wl.c_in * wl.K
    w = rng.standard_normal(wl.w_shape) * math.sqrt(1.0 / fan_in)
    return to_storage(x, wl.dtype), to_storage(w, wl.dtype)


def random_inputs(seed: int, x_shape, w_shape, dtype: str = "fp32", c_in: int | None = None):
    """Generic seeded N(0,1) x and N(0, 1/(C_in*K)) w for ad-hoc test shapes
    (K = the last extent of w)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(x_shape)
    c_in = x_shape[1] if c_in is None else c_in
    w = rng.standard_normal(w_shape) * math.sqrt(1.0 / (c_in * w_shape[-1]))
    return to_storage(x, dtype), to_storage(w, dtype)
