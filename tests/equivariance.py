"""Equivariance harness (App. D): the mean relative error between rotating a
signal before and after a DISCO convolution, measured the way the paper
measures it for Table 5, on the pole-including (L + 1) x 2L grid.

Test infrastructure: the convolution is passed in as a black box (the oracle
on the CPU, the library on the GPU); nothing here is on the product path.

Pieces:
  * orthonormal associated Legendre functions Pbar_lm(cos theta) by the
    standard three-term recurrence in l at fixed m (no Condon-Shortley phase;
    analysis and synthesis use the same functions, so the sign convention
    cancels), Y_lm = Pbar_lm e^{i m phi};
  * a real signal band-limited at L is f = sum_{l < L} sum_{0 <= m <= l}
    s_m Pbar_lm Re(b_lm e^{i m phi}), s_0 = 1, s_m = 2 (the complex expansion
    with b_{l,-m} = conj(b_lm)); random signals draw Re b, Im b ~ N(0, 1/2)
    and b_l0 ~ N(0, 1);
  * analysis on the grid: an FFT along each ring (2L longitudes resolve
    |m| < L), then per m a least-squares fit over the L + 1 rings of the
    degrees |m| <= l < L, rows weighted by the square roots of the ring
    quadrature weights.  Exact for band-limited signals; for others (the
    convolution's output, which the paper does not band-limit either) it is
    the projection onto degrees below L in the grid's quadrature norm;
  * rotation: (Q f)(w) = f(Q^{-1} w), evaluated exactly from the expansion at
    the rotated grid points; Q = Z(alpha) Y(beta) Z(gamma), active,
    right-handed;
  * rotation in harmonic space (the fast path): Wigner D matrices
    D_{m'm} = e^{-i m' alpha} d_{m'm}(beta) e^{-i m gamma}, d(beta) =
    exp(-i beta J_y) from the eigenvectors of J_y in the |l m> basis
    (computed once per degree), in this basis (no Condon-Shortley phase, so
    conjugated by (-1)^m for m > 0); pinned against the point evaluation
    above;
  * the error (App. D): mean over signals and rotations of
    ||P D(Q f) - Q P D(f)|| / ||P D(Q f)||, norms from the grid's quadrature,
    with P the projection onto degrees below L (analysis then synthesis) on
    both sides: the grid holds a signal band-limited at L exactly, and what
    the convolution puts at higher degrees is not a rotation error (with
    both sides projected a rotation about z is exact at any angle, because
    the op commutes with whole-pixel longitude shifts and so keeps each
    longitudinal frequency below L).
Filters (App. D): cutoff 5 pi / L, four nodes along theta (and four along
phi for the directional, separable filter); best case the smooth
psi_S(theta) = exp(-c^2 / (c^2 - theta^2)) at the nodes (times cos(phi) for
the directional filter), worst case random node values.
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------- #
# Spherical harmonics
# --------------------------------------------------------------------------- #
def legendre_table(L: int, x: np.ndarray) -> np.ndarray:
    """Pbar[l, m, i] for 0 <= m <= l < L at points x = cos(theta) (zero for m > l),
    normalised so that Y_lm(theta, phi) = Pbar_lm(cos theta) e^{i m phi} is
    orthonormal on the sphere."""
    x = np.asarray(x, dtype=np.float64)
    s = np.sqrt(np.maximum(0.0, 1.0 - x * x))
    P = np.zeros((L, L) + x.shape)
    pmm = np.full(x.shape, 1.0 / math.sqrt(4.0 * math.pi))
    for m in range(L):
        if m > 0:
            pmm = pmm * math.sqrt((2.0 * m + 1.0) / (2.0 * m)) * s
        P[m, m] = pmm
        if m + 1 < L:
            P[m + 1, m] = math.sqrt(2.0 * m + 3.0) * x * pmm
        for l in range(m + 2, L):
            a = math.sqrt((4.0 * l * l - 1.0) / (l * l - m * m))
            b = math.sqrt(((l - 1.0) ** 2 - m * m) / (4.0 * (l - 1.0) ** 2 - 1.0))
            P[l, m] = a * (x * P[l - 1, m] - b * P[l - 2, m])
    return P


def pole_grid(L: int):
    """Colatitudes pi t / L (t = 0..L, both poles) and longitudes pi p / L (p < 2L)."""
    return np.arange(L + 1) * math.pi / L, np.arange(2 * L) * math.pi / L


def synthesize(b: np.ndarray, theta: np.ndarray, phi: np.ndarray) -> np.ndarray:
    """f at arbitrary points (theta, phi of one shape) from b[l, m] (m <= l < L),
    the recurrence run per m with only two rows kept (memory O(points))."""
    L = b.shape[0]
    x = np.cos(theta)
    s = np.sqrt(np.maximum(0.0, 1.0 - x * x))
    out = np.zeros(theta.shape)
    pmm = np.full(theta.shape, 1.0 / math.sqrt(4.0 * math.pi))
    for m in range(L):
        if m > 0:
            pmm = pmm * math.sqrt((2.0 * m + 1.0) / (2.0 * m)) * s
        gr = b[m, m].real * pmm
        gi = b[m, m].imag * pmm
        p2, p1 = pmm, None
        if m + 1 < L:
            p1 = math.sqrt(2.0 * m + 3.0) * x * pmm
            gr = gr + b[m + 1, m].real * p1
            gi = gi + b[m + 1, m].imag * p1
        for l in range(m + 2, L):
            a = math.sqrt((4.0 * l * l - 1.0) / (l * l - m * m))
            c = math.sqrt(((l - 1.0) ** 2 - m * m) / (4.0 * (l - 1.0) ** 2 - 1.0))
            p = a * (x * p1 - c * p2)
            gr = gr + b[l, m].real * p
            gi = gi + b[l, m].imag * p
            p2, p1 = p1, p
        term = gr * np.cos(m * phi) - gi * np.sin(m * phi)
        out += term if m == 0 else 2.0 * term
    return out


def synthesize_grid(b: np.ndarray, L: int) -> np.ndarray:
    th, ph = pole_grid(L)
    T, Ph = np.meshgrid(th, ph, indexing="ij")
    return synthesize(b, T, Ph)


def analyse_grid(f: np.ndarray, L: int, q: np.ndarray | None = None) -> np.ndarray:
    """b[l, m] (0 <= m <= l < L) of a real signal on the (L + 1) x 2L grid
    (q: ring quadrature weights for the fit, default uniform)."""
    th, _ = pole_grid(L)
    F = np.fft.fft(f, axis=1) / (2 * L)       # F[t, m] = mean_p f e^{-i m phi_p}
    P = legendre_table(L, np.cos(th))          # [l, m, t]
    sq = np.ones(L + 1) if q is None else np.sqrt(np.asarray(q, dtype=np.float64))
    b = np.zeros((L, L), dtype=np.complex128)
    for m in range(L):
        A = P[m:, m].T * sq[:, None]           # [t, l]
        rhs = F[:, m] * sq
        if m == 0:
            rhs = rhs.real
        sol, *_ = np.linalg.lstsq(A, rhs, rcond=None)
        b[m:, m] = sol
    b[:, 0] = b[:, 0].real
    return b


def random_coefficients(L: int, rng: np.random.Generator) -> np.ndarray:
    b = (rng.standard_normal((L, L)) + 1j * rng.standard_normal((L, L))) / math.sqrt(2.0)
    b[:, 0] = rng.standard_normal(L)
    return np.tril(b)


# --------------------------------------------------------------------------- #
# Rotations
# --------------------------------------------------------------------------- #
def rot_z(a: float) -> np.ndarray:
    c, s = math.cos(a), math.sin(a)
    return np.array([[c, -s, 0.0], [s, c, 0.0], [0.0, 0.0, 1.0]])


def rot_y(a: float) -> np.ndarray:
    c, s = math.cos(a), math.sin(a)
    return np.array([[c, 0.0, s], [0.0, 1.0, 0.0], [-s, 0.0, c]])


def euler_zyz(alpha: float, beta: float, gamma: float) -> np.ndarray:
    return rot_z(alpha) @ rot_y(beta) @ rot_z(gamma)


def rotated_points(Q: np.ndarray, theta: np.ndarray, phi: np.ndarray):
    """(theta', phi') of Q^{-1} w for every point w."""
    v = np.stack([np.sin(theta) * np.cos(phi), np.sin(theta) * np.sin(phi), np.cos(theta)])
    r = np.tensordot(Q.T, v, axes=(1, 0))
    return np.arccos(np.clip(r[2], -1.0, 1.0)), np.arctan2(r[1], r[0])


def rotate_grid(b: np.ndarray, Q: np.ndarray, L: int) -> np.ndarray:
    """(Q f) on the grid: f(Q^{-1} w_i) from f's expansion."""
    th, ph = pole_grid(L)
    T, Ph = np.meshgrid(th, ph, indexing="ij")
    tr, pr = rotated_points(Q, T, Ph)
    return synthesize(b, tr, pr)


# --------------------------------------------------------------------------- #
# Batched synthesis, analysis and rotation in harmonic space (fast path)
# --------------------------------------------------------------------------- #
_JY = {}


def jy_eigen(l: int):
    """Eigenvalues and eigenvectors of J_y on the degree-l space (basis
    m = -l..l): J_y = (J_+ - J_-) / 2i with <m+1|J_+|m> = sqrt(l(l+1) - m(m+1))."""
    if l not in _JY:
        n = 2 * l + 1
        m = np.arange(-l, l)
        Jp = np.zeros((n, n))
        Jp[np.arange(1, n), np.arange(n - 1)] = np.sqrt(l * (l + 1) - m * (m + 1.0))
        _JY[l] = np.linalg.eigh((Jp - Jp.T) / 2j)
    return _JY[l]


class Harmonics:
    """Degrees below L on the (L + 1) x 2L pole-including grid, for batches of
    S signals held as coefficients b[l, m, s] (0 <= m <= l < L, the
    convention above): synthesis by a Legendre table and an FFT along
    longitude, analysis by per-m weighted least squares (pseudo-inverses
    computed once), rotation by Wigner D matrices."""

    def __init__(self, L: int, q: np.ndarray):
        self.L = L
        th, _ = pole_grid(L)
        P = legendre_table(L, np.cos(th))                  # [l, m, t]
        sq = np.sqrt(np.asarray(q, dtype=np.float64))
        self.Pt = [np.ascontiguousarray(P[m:, m].T) for m in range(L)]            # [t, l]
        self.pinv = [np.linalg.pinv(self.Pt[m] * sq[:, None]) * sq[None, :] for m in range(L)]

    def synth(self, b: np.ndarray) -> np.ndarray:
        """f[s, t, p] from b[l, m, s]: per m the ring values of the m-th
        longitudinal frequency, then a real inverse FFT along longitude."""
        from scipy import fft
        L = self.L
        X = np.zeros((L + 1, L + 1, b.shape[2]), dtype=np.complex128)   # [m, t, s]
        for m in range(L):
            X[m] = self.Pt[m] @ b[m:, m]
        f = fft.irfft(X, n=2 * L, axis=0, workers=-1) * (2 * L)         # [p, t, s]
        return np.ascontiguousarray(f.transpose(2, 1, 0))

    def analyse(self, f: np.ndarray) -> np.ndarray:
        """b[l, m, s] of real signals f[s, t, p] (the quadrature-weighted
        least-squares projection onto degrees below L)."""
        from scipy import fft
        L = self.L
        F = fft.rfft(np.ascontiguousarray(f.transpose(2, 1, 0)), axis=0, workers=-1) / (2 * L)  # [m, t, s]
        b = np.zeros((L, L, f.shape[0]), dtype=np.complex128)
        for m in range(L):
            b[m:, m] = self.pinv[m] @ (F[m].real if m == 0 else F[m])
        return b

    def rotate(self, b: np.ndarray, alpha: float, beta: float, gamma: float) -> np.ndarray:
        """Coefficients of (Q f)(w) = f(Q^{-1} w), Q = Z(alpha) Y(beta) Z(gamma)."""
        out = np.zeros_like(b)
        for l in range(self.L):
            lam, V = jy_eigen(l)
            m = np.arange(-l, l + 1)
            eps = np.where(m > 0, (-1.0) ** m, 1.0)
            c = np.concatenate([np.conj(b[l, 1:l + 1][::-1]), b[l, :l + 1]], axis=0)   # m = -l..l
            c = c * (eps * np.exp(-1j * m * gamma))[:, None]
            c = V @ (np.exp(-1j * beta * lam)[:, None] * (V.conj().T @ c))
            c = c * (eps * np.exp(-1j * m * alpha))[:, None]
            out[l, :l + 1] = c[l:]
        return out


def random_coefficients_batch(L: int, S: int, rng: np.random.Generator) -> np.ndarray:
    return np.stack([random_coefficients(L, rng) for _ in range(S)], axis=2)


# --------------------------------------------------------------------------- #
# Filters and the error
# --------------------------------------------------------------------------- #
def smooth_profile(theta: np.ndarray, cutoff: float) -> np.ndarray:
    theta = np.asarray(theta, dtype=np.float64)
    out = np.zeros_like(theta)
    inside = theta < cutoff
    out[inside] = np.exp(-cutoff ** 2 / (cutoff ** 2 - theta[inside] ** 2))
    return out


def filter_weights(kind: str, case: str, cutoff: float, rng: np.random.Generator) -> np.ndarray:
    """W [1, 1, K]: kind "axisym" (K = 4, nodes at a h, h = cutoff / 4) or
    "directional" (the separable basis, K = 16, W[4a + b] = theta-part(a h)
    phi-part(b pi / 2)); case "best" (smooth) or "worst" (random)."""
    h = cutoff / 4.0
    t = smooth_profile(np.arange(4) * h, cutoff)
    if kind == "axisym":
        w = t if case == "best" else rng.standard_normal(4)
    else:
        w = np.outer(t, np.cos(np.arange(4) * math.pi / 2)).ravel() if case == "best" \
            else rng.standard_normal(16)
    return w.reshape(1, 1, -1)


def norm_q(g: np.ndarray, q: np.ndarray) -> float:
    return math.sqrt(float((q[:, None] * g * g).sum()))


def equivariance_errors(op, L: int, q: np.ndarray, angles, n_signals: int, seed: int, H=None) -> np.ndarray:
    """The relative equivariance error of `op` (a callable f[S, L+1, 2L] ->
    y[S, L+1, 2L] applied to a batch of signals) for every signal and
    rotation Z(a) Y(b) Z(g) given as (a, b, g) triples; q the grid's ring
    quadrature weights.  Both sides are projected onto degrees below L:
    ||P op(Q f) - Q P op(f)|| / ||P op(Q f)||."""
    H = H or Harmonics(L, q)
    rng = np.random.default_rng(seed)
    b = random_coefficients_batch(L, n_signals, rng)
    bd = H.analyse(op(H.synth(b)))
    errs = []
    for ang in angles:
        lhs = H.synth(H.analyse(op(H.synth(H.rotate(b, *ang)))))
        rhs = H.synth(H.rotate(bd, *ang))
        for s in range(n_signals):
            errs.append(norm_q(lhs[s] - rhs[s], q) / norm_q(lhs[s], q))
    return np.array(errs)


def equivariance_error(op, L: int, q: np.ndarray, angles, n_signals: int, seed: int, H=None):
    """Mean and standard deviation over signals x rotations of the errors above."""
    e = equivariance_errors(op, L, q, angles, n_signals, seed, H)
    return float(e.mean()), float(e.std())


def rotation_angles(kind: str, beta_deg, n: int, seed: int):
    """App. D's rotations as Euler triples (alpha, beta, gamma) of
    Z(alpha) Y(beta) Z(gamma): for the axisymmetric filter uniform on
    SO(3)/SO(2) (gamma = 0, cos(beta) uniform); for the directional one
    random alpha, gamma and a fixed beta."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        a, g = rng.uniform(0.0, 2.0 * math.pi, 2)
        if kind == "axisym":
            out.append((a, math.acos(rng.uniform(-1.0, 1.0)), 0.0))
        else:
            out.append((a, math.radians(beta_deg), g))
    return out


def rotations(kind: str, beta_deg, n: int, seed: int):
    """The same rotations as 3 x 3 matrices."""
    return [euler_zyz(*t) for t in rotation_angles(kind, beta_deg, n, seed)]


def table(op_factory, Ls, n_signals: int = 5, n_rotations: int = 5, seed: int = 0, on_row=None):
    """Rows (L, filter, case, beta, mean %, std %, sq mean %, sq std %) of a
    Table-5-shaped run; the last two are the same statistics of the squared
    ratio (||P op(Q f) - Q P op(f)||^2 / ||P op(Q f)||^2), reported beside
    the ratio of norms because the printed table's magnitudes and its
    quadratic growth with beta are those of the squared ratio.
    op_factory(L, cutoff, kind, w) returns the one-channel convolution on the
    (L + 1) x 2L grid with the axisymmetric ("axisym") or separable
    ("directional") basis and weights w [1, 1, K]; op_factory.quadrature(L)
    gives the grid's ring weights; on_row, if given, is called with each row
    as it is finished."""
    rows = []
    for L in Ls:
        cutoff = 5.0 * math.pi / L
        q = op_factory.quadrature(L)
        H = Harmonics(L, q)
        for kind, betas in (("axisym", [None]), ("directional", [0.0, 5.0, 10.0])):
            for case in ("best", "worst"):
                w = filter_weights(kind, case, cutoff, np.random.default_rng(seed + 1))
                op = op_factory(L, cutoff, kind, w)
                for beta in betas:
                    R = rotation_angles(kind, beta, n_rotations, seed + 2)
                    e = equivariance_errors(op, L, q, R, n_signals, seed + 3, H)
                    e2 = e * e
                    rows.append((L, kind, case, beta, 100.0 * float(e.mean()), 100.0 * float(e.std()),
                                 100.0 * float(e2.mean()), 100.0 * float(e2.std())))
                    if on_row:
                        on_row(rows[-1])
    return rows


class GpuOps:
    """The library's one-channel op on cuda:0 (plans cached per L and basis)."""

    def __init__(self):
        import oracle
        from paper_2209_13603_amd import disco
        self._disco = disco
        self._o = oracle.default()
        self._plans = {}

    def quadrature(self, L):
        return self._o.quadrature(L + 1, 2 * L, sampling=1)

    def __call__(self, L, cutoff, kind, w):
        import torch
        key = (L, kind)
        if key not in self._plans:
            self._plans[key] = self._disco.Plan(L + 1, 2 * L, L + 1, 2 * L, cutoff,
                                                basis="axisym4" if kind == "axisym" else "separable4x4",
                                                sampling="poles")
        plan = self._plans[key]
        wt = torch.from_numpy(np.asarray(w, dtype=np.float32)).to("cuda:0")

        def op(f):
            x = torch.from_numpy(np.asarray(f, dtype=np.float32)[:, None]).to("cuda:0")
            y = plan.forward(x, wt)
            return y[:, 0].double().cpu().numpy()
        return op


class OracleOps:
    """The oracle's one-channel op (fp64, CPU)."""

    def __init__(self):
        import oracle
        self._o = oracle.default()

    def quadrature(self, L):
        return self._o.quadrature(L + 1, 2 * L, sampling=1)

    def __call__(self, L, cutoff, kind, w):
        basis = 1 if kind == "axisym" else 2
        o = self._o

        def op(f):
            return o.forward(L + 1, 2 * L, L + 1, 2 * L, cutoff, np.asarray(f)[:, None], w,
                             sampling=1, basis=basis)[:, 0]
        return op


def format_rows(rows) -> str:
    out = ["| L | filter | case | beta | error % (mean +- std) | squared ratio % (mean +- std) |",
           "|---|---|---|---|---|---|"]
    for L, kind, case, beta, m, s, m2, s2 in rows:
        b = "-" if beta is None else "%g deg" % beta
        out.append("| %d | %s | %s | %s | %.3f +- %.3f | %.3f +- %.3f |" % (L, kind, case, b, m, s, m2, s2))
    return "\n".join(out)


if __name__ == "__main__":
    import argparse
    import os
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    ap = argparse.ArgumentParser(description="Table-5-shaped equivariance errors of the DISCO op")
    ap.add_argument("--L", type=int, nargs="+", default=[32, 64, 128])
    ap.add_argument("--device", choices=["gpu", "oracle"], default="gpu")
    ap.add_argument("--signals", type=int, default=5)
    ap.add_argument("--rotations", type=int, default=5)
    a = ap.parse_args()
    ops = GpuOps() if a.device == "gpu" else OracleOps()
    print("N_f = %d signals, N_Q = %d rotations, device %s" % (a.signals, a.rotations, a.device), flush=True)
    rows = table(ops, a.L, a.signals, a.rotations,
                 on_row=lambda r: print("  " + format_rows([r]).splitlines()[-1], flush=True))
    print(format_rows(rows), flush=True)
