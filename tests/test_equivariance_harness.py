"""Pins of the equivariance harness (App. D) and its Table-5-shaped run on the
oracle.  The harness's pieces are checked against a library routine and
closed forms: the Legendre functions against scipy's spherical harmonics,
analysis against synthesis for band-limited signals, rotation of the degree-1
harmonic cos(theta) against the rotated z coordinate, whole-pixel z rotations
against rolls of the grid, composition of rotations, the harmonic-space
(Wigner D) rotation against the point evaluation, an exactly equivariant
(harmonic-space) filter measuring zero error, and the oracle's op under
rotations about z by angles that are not whole pixels (exact once both sides
are projected onto degrees below L)."""
import math

import numpy as np
import pytest
from scipy import special

import equivariance as E
import oracle


def _sph(l, m, th, ph):
    if hasattr(special, "sph_harm_y"):
        return special.sph_harm_y(l, m, th, ph)
    return special.sph_harm(m, l, ph, th)


def test_legendre_matches_scipy_spherical_harmonics():
    L = 20
    r = np.random.default_rng(0)
    th, ph = r.uniform(0, math.pi, 64), r.uniform(0, 2 * math.pi, 64)
    P = E.legendre_table(L, np.cos(th))
    for l in range(L):
        for m in range(l + 1):
            # scipy carries the Condon-Shortley phase (-1)^m
            ref = _sph(l, m, th, ph) * (-1) ** m
            assert np.abs(P[l, m] * np.exp(1j * m * ph) - ref).max() <= 1e-12


@pytest.mark.parametrize("L", [8, 17, 32])
def test_bandlimited_roundtrip(L):
    r = np.random.default_rng(L)
    b = E.random_coefficients(L, r)
    f = E.synthesize_grid(b, L)
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)
    for qq in (None, q):
        assert np.abs(E.analyse_grid(f, L, qq) - b).max() <= 1e-11 * np.abs(b).max()


def test_rotation_of_cos_theta_is_the_rotated_z_coordinate():
    L = 6
    b = np.zeros((L, L), dtype=complex)
    b[1, 0] = math.sqrt(4 * math.pi / 3)          # cos(theta) = sqrt(4 pi / 3) Y_10
    th, ph = E.pole_grid(L)
    T, Ph = np.meshgrid(th, ph, indexing="ij")
    v = np.stack([np.sin(T) * np.cos(Ph), np.sin(T) * np.sin(Ph), np.cos(T)])
    for Q in E.rotations("directional", 37.0, 4, 1) + E.rotations("axisym", None, 4, 2):
        got = E.rotate_grid(b, Q, L)
        ref = np.tensordot(Q.T, v, axes=(1, 0))[2]   # (Q f)(x) = f(Q^T x) = (Q^T x)_z
        assert np.abs(got - ref).max() <= 1e-12


def test_whole_pixel_z_rotation_is_a_roll():
    L = 16
    b = E.random_coefficients(L, np.random.default_rng(3))
    f = E.synthesize_grid(b, L)
    for k in (1, 5, 2 * L - 3):
        got = E.rotate_grid(b, E.rot_z(math.pi * k / L), L)
        assert np.abs(got - np.roll(f, k, axis=1)).max() <= 1e-10 * np.abs(f).max()


def test_rotations_compose():
    L = 12
    b = E.random_coefficients(L, np.random.default_rng(4))
    Q1, Q2 = E.rotations("directional", 23.0, 2, 5)
    f1 = E.rotate_grid(b, Q1, L)
    twice = E.rotate_grid(E.analyse_grid(f1, L), Q2, L)
    once = E.rotate_grid(b, Q2 @ Q1, L)
    assert np.abs(twice - once).max() <= 1e-10 * np.abs(once).max()


@pytest.mark.parametrize("L", [8, 21])
def test_harmonic_rotation_matches_point_evaluation(L):
    """Wigner D rotation of the coefficients, then synthesis, equals the
    expansion evaluated at the rotated grid points, for every Euler triple
    kind the runs use (including beta = 0 and beta near pi)."""
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)
    H = E.Harmonics(L, q)
    b = E.random_coefficients_batch(L, 2, np.random.default_rng(L))
    angles = E.rotation_angles("axisym", None, 3, 8) + E.rotation_angles("directional", 10.0, 2, 9) \
        + [(0.3, 0.0, 1.1), (2.0, math.pi - 1e-3, 0.4)]
    for ang in angles:
        got = H.synth(H.rotate(b, *ang))
        for s in range(2):
            ref = E.rotate_grid(b[:, :, s], E.euler_zyz(*ang), L)
            assert np.abs(got[s] - ref).max() <= 1e-11 * np.abs(ref).max()


def test_batched_analysis_matches_the_per_signal_fit():
    L = 13
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)
    H = E.Harmonics(L, q)
    b = E.random_coefficients_batch(L, 3, np.random.default_rng(5))
    f = H.synth(b)
    for s in range(3):
        assert np.abs(f[s] - E.synthesize_grid(b[:, :, s], L)).max() <= 1e-12 * np.abs(f[s]).max()
    assert np.abs(H.analyse(f) - b).max() <= 1e-11 * np.abs(b).max()
    # a signal with degrees above L is projected as the per-signal fit projects it
    g = np.random.default_rng(6).standard_normal((2, L + 1, 2 * L))
    for s in range(2):
        assert np.abs(H.analyse(g)[:, :, s] - E.analyse_grid(g[s], L, q)).max() <= 1e-10


def test_oracle_z_rotation_by_a_fraction_of_a_pixel_is_exact_after_projection():
    """The op commutes with whole-pixel longitude shifts, so it keeps each
    longitudinal frequency; with both sides projected onto degrees below L a
    rotation about z by any angle gives rounding-level error."""
    L = 12
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)
    ops = E.OracleOps()
    cutoff = 5.0 * math.pi / L
    for kind in ("axisym", "directional"):
        w = E.filter_weights(kind, "worst", cutoff, np.random.default_rng(1))
        op = ops(L, cutoff, kind, w)
        angles = [(0.37 * math.pi / L, 0.0, 0.0), (1.234, 0.0, 2.71)]
        m, _ = E.equivariance_error(op, L, q, angles, 2, 3)
        assert m <= 1e-10


def test_exactly_equivariant_filter_measures_zero():
    """A convolution applied in harmonic space (degree-wise gains) commutes with
    every rotation: the harness must report rounding-level error."""
    L = 16
    g = np.exp(-0.2 * np.arange(L))
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)

    def op(f):
        return E.synthesize_grid(E.analyse_grid(f, L, q) * g[:, None], L)

    def op_batch(fs):
        return np.stack([op(f) for f in fs])
    for kind, beta in (("axisym", None), ("directional", 10.0)):
        m, _ = E.equivariance_error(op_batch, L, q, E.rotation_angles(kind, beta, 3, 6), 2, 7)
        assert m <= 1e-12


def test_table_shape_on_the_oracle():
    """The shape of Table 5 at L = 16: random (worst) filters err more than
    smooth (best) ones; directional errors grow with the latitudinal angle
    beta, starting from rounding level at beta = 0; the smooth axisymmetric
    filter errs less than the directional one at beta > 0."""
    rows = E.table(E.OracleOps(), [16], n_signals=3, n_rotations=3)
    err = {(k, c, b): m for (_, k, c, b, m, *_) in rows}
    assert err[("axisym", "best", None)] < err[("axisym", "worst", None)]
    for c in ("best", "worst"):
        assert err[("directional", c, 0.0)] < err[("directional", c, 5.0)] < err[("directional", c, 10.0)]
        assert err[("directional", c, 0.0)] <= 1e-8           # percent
    assert err[("axisym", "best", None)] < err[("directional", "best", 5.0)]
