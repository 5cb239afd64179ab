"""Pins of the equivariance harness (App. D) and its Table-5-shaped run on the
oracle.  The harness's pieces are checked against a library routine and
closed forms: the Legendre functions against scipy's spherical harmonics,
analysis against synthesis for band-limited signals, rotation of the degree-1
harmonic cos(theta) against the rotated z coordinate, whole-pixel z rotations
against rolls of the grid, composition of rotations, and an exactly
equivariant (harmonic-space) filter measuring zero error."""
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


def test_exactly_equivariant_filter_measures_zero():
    """A convolution applied in harmonic space (degree-wise gains) commutes with
    every rotation: the harness must report rounding-level error."""
    L = 16
    g = np.exp(-0.2 * np.arange(L))
    q = oracle.default().quadrature(L + 1, 2 * L, sampling=1)

    def op(f):
        return E.synthesize_grid(E.analyse_grid(f, L, q) * g[:, None], L)
    for kind, beta in (("axisym", None), ("directional", 10.0)):
        m, _ = E.equivariance_error(op, L, q, E.rotations(kind, beta, 3, 6), 2, 7)
        assert m <= 1e-12


def test_table_shape_on_the_oracle():
    """The shape of Table 5 at L = 16: random (worst) filters err more than
    smooth (best) ones; directional errors grow with the latitudinal angle
    beta; the smooth axisymmetric filter errs less than the directional one
    at beta > 0."""
    rows = E.table(E.OracleOps(), [16], n_signals=3, n_rotations=3)
    err = {(k, c, b): m for (_, k, c, b, m, _) in rows}
    assert err[("axisym", "best", None)] < err[("axisym", "worst", None)]
    for c in ("best", "worst"):
        assert err[("directional", c, 0.0)] < err[("directional", c, 5.0)] < err[("directional", c, 10.0)]
    assert err[("axisym", "best", None)] < err[("directional", "best", 5.0)]
