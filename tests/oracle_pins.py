"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with an independent fact: a closed form, a library
routine (scipy's Legendre polynomials, numpy's Gauss-Legendre rule and linear
solver), the paper's worked node example (App. E.2), an exact invariant of the
method, or brute force on tiny inputs.  ``test_oracle_pins.py`` runs them on
the real oracle; ``test_oracle_mutants.py`` runs them on copies of the oracle
with planted mistakes and requires every mistake to fail at least one pin.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
from scipy.special import eval_legendre

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _xw(seed, B, Cin, nlat, nlon, Cout):
    r = _rng(seed)
    return r.standard_normal((B, Cin, nlat, nlon)), r.standard_normal((Cout, Cin, 9)) / 6.0


def _select_w(nk=9):
    """W with Cin = 1, Cout = 9 and W[k, 0, k'] = delta(k, k'): y then equals Z."""
    w = np.zeros((nk, 1, 9))
    for k in range(9):
        w[k, 0, k] = 1.0
    return w


def _haversine_dist(th1, ph1, th2, ph2):
    """Great-circle distance between colatitude/longitude points (haversine)."""
    h = np.sin((th1 - th2) / 2) ** 2 + np.sin(th1) * np.sin(th2) * np.sin((ph1 - ph2) / 2) ** 2
    return 2 * np.arcsin(np.sqrt(np.clip(h, 0.0, 1.0)))


# --------------------------------------------------------------------------- #
# Quadrature (Sec. 3.2 / 4.1 adopt sampling-theorem quadrature; App. A)
# --------------------------------------------------------------------------- #
def pin_quadrature_total(o):
    """Weights sum to the area of the unit sphere, 4 pi."""
    for n in (1, 2, 3, 7, 32, 64, 128, 2048):
        for nlon in (2, 64, 4096):
            tot = o.quadrature(n, nlon).sum() * nlon
            assert abs(tot - 4 * math.pi) <= 1e-13 * 4 * math.pi, (n, nlon, tot)


def pin_quadrature_legendre_exact(o):
    """The rule integrates P_l(cos theta) exactly for l < nlat: the integral over
    the sphere is 4 pi for l = 0 and 0 otherwise (orthogonality)."""
    for n in (4, 7, 32, 64, 129, 512):
        nlon = 8
        q = o.quadrature(n, nlon)
        x = np.cos(o.colatitudes(n))
        for l in range(n):
            val = nlon * float(np.dot(q, eval_legendre(l, x)))
            expect = 4 * math.pi if l == 0 else 0.0
            assert abs(val - expect) <= 1e-12, (n, l, val)


def pin_quadrature_unique(o):
    """n weights that integrate P_0..P_{n-1} exactly on n distinct nodes are
    unique: solve that linear system with numpy and compare."""
    for n in (5, 8, 16, 33):
        x = np.cos(o.colatitudes(n))
        V = np.stack([eval_legendre(l, x) for l in range(n)])
        rhs = np.zeros(n)
        rhs[0] = 2.0
        w = np.linalg.solve(V, rhs)
        nlon = 6
        q = o.quadrature(n, nlon) * nlon / (2 * math.pi)
        assert np.allclose(q, w, rtol=0, atol=1e-12), (n, np.abs(q - w).max())


def _cell_area_weights(n, nlon):
    """Area of the cell of ring t of the cell-centred grid divided among the
    ring's nlon pixels: the spherical band between colatitudes t pi / n and
    (t + 1) pi / n has area 2 pi (cos(t pi / n) - cos((t + 1) pi / n))."""
    t = np.arange(n)
    return (2 * math.pi / nlon) * (np.cos(t * math.pi / n) - np.cos((t + 1) * math.pi / n))


def pin_quadrature_cell_area(o):
    """Cell-area quadrature (the alternative rule the plan can select on the
    cell-centred grid): each ring's weight is the area of its latitude band
    divided by nlon (a difference of cosines, computed here independently),
    the weights total 4 pi, and the forward and transposed ops apply exactly
    these weights (dense products with Psi against the looped sums, and the
    centre value of a delta input)."""
    for n in (1, 2, 3, 7, 32, 129, 2048):
        for nlon in (2, 64, 4096):
            q = o.quadrature(n, nlon, kind=1)
            ref = _cell_area_weights(n, nlon)
            # the cosine difference cancels: its error is a few ulps of 2 pi / nlon
            assert np.abs(q - ref).max() <= 8 * np.finfo(float).eps * 2 * math.pi / nlon, (n, nlon)
            assert abs(q.sum() * nlon - 4 * math.pi) <= 1e-13 * 4 * math.pi, (n, nlon)
    for (a, b, c, d) in _DENSE_CASES:
        tc = 3 * math.pi / min(a, c)
        psi = o.psi_dense(a, b, c, d, tc)                  # [Nout, Nin, 9]
        qi = np.repeat(_cell_area_weights(a, b), b)
        qo = np.repeat(_cell_area_weights(c, d), d)
        x, w = _xw(40, 2, 3, a, b, 4)
        Z = np.einsum("jik,bci->bckj", psi, x.reshape(2, 3, -1) * qi)
        y_dense = np.einsum("ock,bckj->boj", w, Z).reshape(2, 4, c, d)
        y = o.forward(a, b, c, d, tc, x, w, quad=1)
        assert np.abs(y - y_dense).max() <= 1e-13 * np.abs(y_dense).max()
        xT, wT = _xw(41, 2, 4, c, d, 4)
        wT = wT.reshape(4, 4, 9)[:, :3]
        ZT = np.einsum("jik,bcj->bcki", psi, xT.reshape(2, 4, -1) * qo)
        yT_dense = np.einsum("cok,bcki->boi", wT, ZT).reshape(2, 3, a, b)
        yT = o.transpose(a, b, c, d, tc, xT, wT, quad=1)
        assert np.abs(yT - yT_dense).max() <= 1e-13 * np.abs(yT_dense).max()
    a, b = 16, 32
    x = np.zeros((1, 1, a, b))
    x[0, 0, 3, 7] = 1.0
    Z = o.forward(a, b, a, b, 3 * math.pi / a, x, _select_w(), quad=1)[0]
    assert abs(Z[4, 3, 7] - _cell_area_weights(a, b)[3]) <= 1e-14 * _cell_area_weights(a, b)[3]


def pin_node_spacing_override(o):
    """A node spacing h other than the default moves the hats' nodes (Sec. 3.4:
    equally spaced nodes, linear interpolation): with a delta input one ring
    south of the output point, on the same meridian, the tangent-plane point
    is (u, v) = (d, 0) with d the ring step, so the 3x3 basis gives
    psi_4 = 1 - d / h and psi_7 = d / h for h >= d (closed form), and the
    axisymmetric basis psi_1 = 2 - d / h, psi_2 = d / h - 1 for h <= d < 2 h,
    all times the input ring's quadrature weight."""
    a, b = 16, 32
    tc = 3 * math.pi / a
    d = math.pi / a
    q = o.quadrature(a, b)
    x = np.zeros((1, 1, a, b))
    x[0, 0, 7, 5] = 1.0
    for h in (tc / 2, 0.4 * tc):
        Z = o.forward(a, b, a, b, tc, x, _select_w(), h=h)[0]
        e = np.zeros(9)
        e[4] = (1 - d / h) * q[7]
        e[7] = d / h * q[7]
        assert np.abs(Z[:, 6, 5] - e).max() <= 1e-14 * q[7], (h, Z[:, 6, 5], e)
    h = 0.6 * d
    Z = o.forward(a, b, a, b, tc, x, np.eye(4).reshape(4, 1, 4), h=h, basis=1)[0]
    e = np.array([0.0, 2 - d / h, d / h - 1, 0.0]) * q[7]
    assert np.abs(Z[:, 6, 5] - e).max() <= 1e-14 * q[7], (Z[:, 6, 5], e)


def pin_grid(o):
    """Cell-centred equiangular grid: colatitude (t + 1/2) pi / nlat,
    longitude 2 pi p / nlon."""
    th = o.colatitudes(8)
    assert np.allclose(th, (np.arange(8) + 0.5) * math.pi / 8, atol=1e-15)
    ph = o.longitudes(16)
    assert np.allclose(ph, np.arange(16) * 2 * math.pi / 16, atol=1e-15)


# --------------------------------------------------------------------------- #
# Geometry of R_j^{-1} w_i (Sec. 3.2, Sec. 4.1 rotated coordinates)
# --------------------------------------------------------------------------- #
def pin_geometry_worked_example(o):
    """App. E.2: with the filter centred on the pole, the 9 node positions map
    onto the square 3x3 grid {-h, 0, h}^2, and each basis function is 1 at its
    own node and 0 at the other eight."""
    with open(os.path.join(GOLDEN, "nodes_3x3.json")) as f:
        g = json.load(f)
    for L in (32, 256, 2048):
        h = math.pi / L
        seen = set()
        for node in g["nodes"]:
            th = node["theta"] * math.pi / L
            ph = node["phi"] * math.pi
            Th, u, v = o.frame_coords(0.0, 0.0, th, ph)
            assert abs(Th - th) <= 1e-15, (node, Th)
            eu, ev = node["uv"]
            assert abs(u / h - eu) <= 1e-12 and abs(v / h - ev) <= 1e-12, (node, u / h, v / h)
            psi = o.basis(u, v, h)
            k = int(np.argmax(psi))
            assert abs(psi[k] - 1.0) <= 1e-12 and np.abs(np.delete(psi, k)).max() <= 1e-12
            seen.add(k)
        assert seen == set(range(9))


def pin_geometry_identity_and_meridian(o):
    """Filter centred on the input point: Theta = 0.  Same meridian:
    Theta = |theta_i - theta_j|, u = theta_i - theta_j (south positive), v = 0."""
    r = _rng(1)
    for _ in range(200):
        thj = r.uniform(0.01, math.pi - 0.01)
        phj = r.uniform(0, 2 * math.pi)
        Th, u, v = o.frame_coords(thj, phj, thj, phj)
        assert Th <= 1e-15 and abs(u) <= 1e-15 and abs(v) <= 1e-15
        d = r.uniform(-0.05, 0.05)
        thi = min(max(thj + d, 1e-3), math.pi - 1e-3)
        Th, u, v = o.frame_coords(thj, phj, thi, phj)
        assert abs(Th - abs(thi - thj)) <= 2e-15, (Th, thi - thj)
        assert abs(u - (thi - thj)) <= 2e-15 and abs(v) <= 2e-15


def pin_geometry_general(o):
    """Random pairs: Theta equals the haversine great-circle distance; the
    direction Phi = atan2(v, u) equals pi minus the initial bearing from the
    centre to the point (bearing clockwise from north, the navigation formula),
    i.e. Phi = 0 is south and Phi = pi/2 is east."""
    r = _rng(2)
    for _ in range(500):
        thj = r.uniform(0.02, math.pi - 0.02)
        phj = r.uniform(0, 2 * math.pi)
        thi = thj + r.uniform(-0.3, 0.3)
        thi = min(max(thi, 1e-3), math.pi - 1e-3)
        phi = phj + r.uniform(-0.4, 0.4)
        Th, u, v = o.frame_coords(thj, phj, thi, phi)
        d = float(_haversine_dist(thi, phi, thj, phj))
        assert abs(Th - d) <= 1e-13, (Th, d)
        assert abs(math.hypot(u, v) - Th) <= 1e-13
        if d < 1e-4:
            continue
        latj, lati = math.pi / 2 - thj, math.pi / 2 - thi
        dl = phi - phj
        bearing = math.atan2(math.sin(dl) * math.cos(lati),
                             math.cos(latj) * math.sin(lati)
                             - math.sin(latj) * math.cos(lati) * math.cos(dl))
        Phi = math.atan2(v, u)
        diff = (Phi - (math.pi - bearing) + math.pi) % (2 * math.pi) - math.pi
        assert abs(diff) <= 1e-9, (Phi, bearing)


def pin_geometry_same_ring(o):
    """Two points on one ring: sin(Theta/2) = sin(theta) |sin(dphi/2)| and
    v has the sign of sin(dphi) (east positive)."""
    r = _rng(3)
    for _ in range(200):
        th = r.uniform(0.01, math.pi - 0.01)
        ph = r.uniform(0, 2 * math.pi)
        dp = r.uniform(-0.5, 0.5)
        Th, u, v = o.frame_coords(th, ph, th, ph + dp)
        assert abs(math.sin(Th / 2) - math.sin(th) * abs(math.sin(dp / 2))) <= 1e-15
        if abs(dp) > 1e-6:
            assert np.sign(v) == np.sign(math.sin(dp))


# --------------------------------------------------------------------------- #
# Basis (Sec. 3.4, App. E.2: bilinear interpolation on the 3x3 node grid)
# --------------------------------------------------------------------------- #
def pin_basis(o):
    h = 0.0123
    # Kronecker delta at the nodes, node k = 3a + b at ((a-1)h, (b-1)h).
    for a in range(3):
        for b in range(3):
            psi = o.basis((a - 1) * h, (b - 1) * h, h)
            e = np.zeros(9)
            e[3 * a + b] = 1.0
            assert np.allclose(psi, e, atol=1e-15), (a, b, psi)
    r = _rng(4)
    for _ in range(500):
        u, v = r.uniform(-h, h, 2)
        psi = o.basis(u, v, h)
        # Partition of unity inside the node square.
        assert abs(psi.sum() - 1.0) <= 1e-14
        # Bilinear interpolation reproduces any bilinear function exactly.
        c = r.standard_normal(4)
        f = lambda uu, vv: c[0] + c[1] * uu / h + c[2] * vv / h + c[3] * uu * vv / h ** 2
        nodes = [f((k // 3 - 1) * h, (k % 3 - 1) * h) for k in range(9)]
        assert abs(float(np.dot(psi, nodes)) - f(u, v)) <= 1e-12
    for _ in range(500):
        u, v = r.uniform(-3 * h, 3 * h, 2)
        psi = o.basis(u, v, h)
        assert (psi >= 0).all() and (psi <= 1).all()
        assert np.count_nonzero(psi) <= 4
        if max(abs(u), abs(v)) >= 2 * h:
            assert not psi.any()
    # Linear profile along the u axis: the south node's weight at u = s h.
    for s in (0.0, 0.25, 0.5, 1.0, 1.5, 2.0):
        psi = o.basis(s * h, 0.0, h)
        assert abs(psi[7] - max(0.0, 1 - abs(s - 1))) <= 1e-15


# --------------------------------------------------------------------------- #
# The sums (Sec. 3.2 eq. 4, Sec. 3.5 eq. 6, Sec. 4.1-4.2)
# --------------------------------------------------------------------------- #
_DENSE_CASES = [(8, 16, 8, 16), (16, 32, 8, 16), (12, 24, 6, 12)]


def pin_compressed_tensor_identity(o):
    """Sec. 4.2: Psi[t',p',t,p] = Psi[t',0,t,p - s p'] (longitude shift)."""
    for (a, b, c, d) in _DENSE_CASES:
        tc = 3 * math.pi / min(a, c)
        psi = o.psi_dense(a, b, c, d, tc).reshape(c, d, a, b, 9)
        s = b // d
        assert np.abs(psi).max() > 0.5
        for pp in range(d):
            ref = np.roll(psi[:, 0], s * pp, axis=2)
            assert np.abs(psi[:, pp] - ref).max() <= 1e-13, (a, b, c, d, pp)


def pin_dense_vs_loop(o):
    """The looped forward and transposed sums equal dense products
    y = W . (Psi diag(q) x) and yT = W^T . (Psi^T diag(q_out) xT)."""
    for (a, b, c, d) in _DENSE_CASES:
        tc = 3 * math.pi / min(a, c)
        psi = o.psi_dense(a, b, c, d, tc)                  # [Nout, Nin, 9]
        qi = np.repeat(o.quadrature(a, b), b)
        qo = np.repeat(o.quadrature(c, d), d)
        x, w = _xw(10, 2, 3, a, b, 4)
        Z = np.einsum("jik,bci->bckj", psi, x.reshape(2, 3, -1) * qi)
        y_dense = np.einsum("ock,bckj->boj", w, Z).reshape(2, 4, c, d)
        y = o.forward(a, b, c, d, tc, x, w)
        assert np.abs(y - y_dense).max() <= 1e-13 * np.abs(y_dense).max()
        xT, wT = _xw(11, 2, 4, c, d, 4)
        wT = wT.reshape(4, 4, 9)[:, :3]                    # [CinT=4, CoutT=3, 9]
        ZT = np.einsum("jik,bcj->bcki", psi, xT.reshape(2, 4, -1) * qo)
        yT_dense = np.einsum("cok,bcki->boi", wT, ZT).reshape(2, 3, a, b)
        yT = o.transpose(a, b, c, d, tc, xT, wT)
        assert np.abs(yT - yT_dense).max() <= 1e-13 * np.abs(yT_dense).max()


def pin_shift_equivariance(o):
    """Sec. 3.3: rotations about the z axis commute with the convolution; on
    the grid a shift by whole output pixels is exact (Sec. 4.2)."""
    for (a, b, c, d) in [(16, 32, 16, 32), (16, 32, 8, 16)]:
        tc = 3 * math.pi / min(a, c)
        s = b // d
        x, w = _xw(12, 1, 2, a, b, 3)
        y = o.forward(a, b, c, d, tc, x, w)
        for m in (1, 3):
            ys = o.forward(a, b, c, d, tc, np.roll(x, s * m, axis=-1), w)
            assert np.abs(ys - np.roll(y, m, axis=-1)).max() <= 1e-13 * np.abs(y).max()
        xT, wT = _xw(13, 1, 3, c, d, 2)
        wT = wT.reshape(2, 3, 9).transpose(1, 0, 2).copy()  # [CinT=3, CoutT=2, 9]
        yT = o.transpose(a, b, c, d, tc, xT, wT)
        ysT = o.transpose(a, b, c, d, tc, np.roll(xT, 2, axis=-1), wT)
        assert np.abs(ysT - np.roll(yT, 2 * s, axis=-1)).max() <= 1e-13 * np.abs(yT).max()


def pin_mirror_symmetry(o):
    """Mirror phi -> -phi swaps east and west (node column b <-> 2 - b); the
    flip theta -> pi - theta swaps north and south (node row a <-> 2 - a)."""
    a, b, c, d = 16, 32, 8, 16
    tc = 3 * math.pi / c
    x, w = _xw(14, 1, 2, a, b, 2)
    y = o.forward(a, b, c, d, tc, x, w)
    perm_b = [3 * (k // 3) + (2 - k % 3) for k in range(9)]
    perm_a = [3 * (2 - k // 3) + (k % 3) for k in range(9)]
    xm = x[..., (-np.arange(b)) % b]
    ym = o.forward(a, b, c, d, tc, xm, w[:, :, perm_b])
    assert np.abs(ym - y[..., (-np.arange(d)) % d]).max() <= 1e-13 * np.abs(y).max()
    xf = x[:, :, ::-1, :]
    yf = o.forward(a, b, c, d, tc, xf, w[:, :, perm_a])
    assert np.abs(yf - y[:, :, ::-1, :]).max() <= 1e-12 * np.abs(y).max()


def pin_compact_support_and_delta(o):
    """A delta input at pixel i0 reaches only outputs within the basis support
    radius 2 sqrt(2) h (< theta_c); at the centre only the central node fires
    with value q(t0), one ring north of it only the south node (u = +h)."""
    a, b = 16, 32
    tc = 3 * math.pi / a
    h = tc / 3
    q = o.quadrature(a, b)
    th = o.colatitudes(a)
    ph = o.longitudes(b)
    for (t0, p0) in [(7, 5), (0, 3), (15, 30), (2, 0)]:
        x = np.zeros((1, 1, a, b))
        x[0, 0, t0, p0] = 1.0
        Z = o.forward(a, b, a, b, tc, x, _select_w())[0]   # [9, a, b]
        dist = _haversine_dist(th[:, None], ph[None, :], th[t0], ph[p0])
        far = dist > 2 * math.sqrt(2) * h + 1e-12
        assert not Z[:, far].any()
        assert np.count_nonzero(Z.any(axis=0)) > 1
        e = np.zeros(9)
        e[4] = q[t0]
        assert np.abs(Z[:, t0, p0] - e).max() <= 1e-15
        if t0 > 0:
            e = np.zeros(9)
            e[7] = q[t0]
            assert np.abs(Z[:, t0 - 1, p0] - e).max() <= 1e-14, Z[:, t0 - 1, p0]


def pin_adjoint(o):
    """Sec. 3.5 with R11: the transposed op is the adjoint of the forward op in
    the quadrature-weighted inner products, <A x, g>_q_out = <x, B g>_q_in."""
    for (a, b, c, d) in [(16, 32, 16, 32), (16, 32, 8, 16), (12, 24, 6, 12)]:
        tc = 3 * math.pi / min(a, c)
        r = _rng(15)
        Cin, Cout = 3, 2
        x = r.standard_normal((2, Cin, a, b))
        g = r.standard_normal((2, Cout, c, d))
        w = r.standard_normal((Cout, Cin, 9))
        Ax = o.forward(a, b, c, d, tc, x, w)
        Bg = o.transpose(a, b, c, d, tc, g, w)
        qo = o.quadrature(c, d)[None, None, :, None]
        qi = o.quadrature(a, b)[None, None, :, None]
        lhs = float((Ax * g * qo).sum())
        rhs = float((x * Bg * qi).sum())
        assert abs(lhs - rhs) <= 1e-12 * max(abs(lhs), 1.0), (lhs, rhs)


def filter_integrals(h, n=24):
    """S_k = integral over the sphere of psi_k, computed in the filter frame:
    with the azimuthal equidistant map dmu = (sin r / r) du dv, r = |(u, v)|,
    by Gauss-Legendre on each hat cell."""
    xg, wg = np.polynomial.legendre.leggauss(n)
    S = np.zeros(9)
    for a in range(3):
        for b in range(3):
            tot = 0.0
            for cu in (a - 2, a - 1):
                for cv in (b - 2, b - 1):
                    u = (cu + (xg + 1) / 2) * h
                    v = (cv + (xg + 1) / 2) * h
                    U, Vv = np.meshgrid(u, v, indexing="ij")
                    Wt = np.outer(wg, wg) * (h / 2) ** 2
                    val = np.maximum(0, 1 - np.abs(U / h - (a - 1))) * \
                        np.maximum(0, 1 - np.abs(Vv / h - (b - 1)))
                    rr = np.hypot(U, Vv)
                    tot += float((Wt * val * np.sinc(rr / math.pi)).sum())
            S[3 * a + b] = tot
    return S


def pin_constant_input(o):
    """x = 1 everywhere: each Z_k is exactly constant along an output ring
    (shift invariance) and approximates the filter integral S_k (Sec. 3.2: the
    only error is quadrature).  With a hat one pixel wide the sampling error
    is O((pixel / h)^2): at fixed theta_c it must fall by at least 2.5x per
    doubling of the grid (second order) and be below 2e-3 at 512 x 1024."""
    tc = 3 * math.pi / 32
    h = tc / 3
    S = filter_integrals(h)
    a, b = 32, 64
    Z = o.forward(a, b, a, b, tc, np.ones((1, 1, a, b)), _select_w())[0]   # [9, a, b]
    spread = np.abs(Z - Z[:, :, :1]).max()
    assert spread <= 1e-14 * np.abs(Z).max(), spread
    errs = []
    for a in (32, 64, 128, 256, 512):
        b = 2 * a
        pix = np.arange(a) * b            # one pixel per ring: rings are constant
        Zr = o.forward(a, b, a, b, tc, np.ones((1, 1, a, b)), _select_w(), pix=pix)[0]
        errs.append(float(np.abs(Zr / S[:, None] - 1).max()))
    assert errs[0] <= 0.15, errs
    for e0, e1 in zip(errs, errs[1:]):
        assert e1 * 2.5 <= e0, errs
    assert errs[-1] <= 2e-3, errs


def pin_window_equals_all_pairs(o):
    """Skipping rings farther than theta_c in colatitude changes nothing (the
    geodesic distance is at least the colatitude difference): bitwise."""
    for (a, b, c, d) in [(32, 64, 32, 64), (32, 64, 16, 32)]:
        tc = 3 * math.pi / min(a, c)
        x, w = _xw(16, 1, 2, a, b, 2)
        y_all = o.forward(a, b, c, d, tc, x, w, window=False)
        y_win = o.forward(a, b, c, d, tc, x, w, window=True)
        assert np.array_equal(y_all, y_win)
        xT, wT = _xw(17, 1, 2, c, d, 2)
        yT_all = o.transpose(a, b, c, d, tc, xT, wT, window=False)
        yT_win = o.transpose(a, b, c, d, tc, xT, wT, window=True)
        assert np.array_equal(yT_all, yT_win)


def pin_pixel_subset(o):
    """Computing a subset of output pixels gives the same values as the full run."""
    a, b, c, d = 16, 32, 8, 16
    tc = 3 * math.pi / c
    x, w = _xw(18, 2, 2, a, b, 3)
    y = o.forward(a, b, c, d, tc, x, w)
    pix = np.array([0, 5, 17, 100, c * d - 1])
    ys = o.forward(a, b, c, d, tc, x, w, pix=pix)
    assert np.array_equal(ys, y.reshape(2, 3, -1)[:, :, pix])


# --------------------------------------------------------------------------- #
# The paper's own timed configuration: the pole-including grid of Sec. 4.2
# with App. A's quadrature, and the axisymmetric basis of Sec. 3.4 / App. B.
# --------------------------------------------------------------------------- #
_MW, _AX = 1, 1


def _select_w4():
    """W with Cin = 1, Cout = 4 and W[k, 0, k'] = delta(k, k'): y then equals Z."""
    w = np.zeros((4, 1, 4))
    for k in range(4):
        w[k, 0, k] = 1.0
    return w


def pin_mw_grid(o):
    """(theta_t, phi_p) = (pi t / L, pi p / L), 0 <= t <= L, 0 <= p < 2L."""
    for L in (1, 4, 8, 33):
        th = o.colatitudes(L + 1, sampling=_MW)
        assert np.allclose(th, np.arange(L + 1) * math.pi / L, rtol=0, atol=1e-15)
        assert th[0] == 0.0 and abs(th[-1] - math.pi) <= 1e-15
        assert np.allclose(o.longitudes(2 * L), np.arange(2 * L) * math.pi / L, rtol=0, atol=1e-15)


def pin_mw_quadrature_total_and_symmetry(o):
    """App. A weights: total 4 pi, antipodally symmetric (q_t = q_{L-t}), positive."""
    for L in (1, 2, 3, 8, 9, 64, 1024, 2048):
        q = o.quadrature(L + 1, 2 * L, sampling=_MW)
        assert abs(q.sum() * 2 * L - 4 * math.pi) <= 1e-12 * 4 * math.pi, (L, q.sum())
        assert np.abs(q - q[::-1]).max() <= 1e-13 * q.max(), L
        assert (q > 0).all(), L


def pin_mw_quadrature_interpolatory(o):
    """On the L + 1 distinct nodes x_t = cos(theta_t) exactly one rule
    integrates every polynomial of degree <= L.  The Chebyshev moments
    int_{-1}^{1} T_n dx = 2 / (1 - n^2) (n even), 0 (n odd) fix it (numpy's
    Chebyshev Vandermonde matrix and linear solver); App. A's weights, folded
    from the band-limited transform of sin(theta), must be that rule times the
    longitude step 2 pi / (2L)."""
    for L in (2, 3, 4, 8, 15, 16, 33, 64):
        x = np.cos(np.arange(L + 1) * math.pi / L)
        V = np.polynomial.chebyshev.chebvander(x, L).T
        mom = np.array([2.0 / (1 - n * n) if n % 2 == 0 else 0.0 for n in range(L + 1)])
        w = np.linalg.solve(V, mom)
        q = o.quadrature(L + 1, 2 * L, sampling=_MW) * (2 * L) / (2 * math.pi)
        assert np.abs(q - w).max() <= 1e-13, (L, np.abs(q - w).max())


def pin_mw_quadrature_legendre_exact(o):
    """Band-limited signals integrate exactly (the sampling theorem the grid
    comes with): P_l(cos theta) over the sphere is 4 pi for l = 0, else 0,
    for every l < L."""
    for L in (4, 7, 32, 65, 256):
        q = o.quadrature(L + 1, 2 * L, sampling=_MW)
        x = np.cos(o.colatitudes(L + 1, sampling=_MW))
        for l in range(L):
            val = 2 * L * float(np.dot(q, eval_legendre(l, x)))
            expect = 4 * math.pi if l == 0 else 0.0
            assert abs(val - expect) <= 1e-12, (L, l, val)


def pin_axisym_basis(o):
    """Four hats along Theta at nodes 0, h, 2h, 3h (Sec. 3.4, linear
    interpolation): Kronecker delta at the nodes, partition of unity on
    [0, 3h], linear functions reproduced there, only the last hat (falling to
    zero at 4h) on [3h, 4h], nothing beyond."""
    h = 0.0123
    for j in range(4):
        e = np.zeros(4)
        e[j] = 1.0
        assert np.abs(o.basis_axisym(j * h, h) - e).max() <= 1e-15, j
    assert np.abs(o.basis_axisym(1.5 * h, h) - [0, 0.5, 0.5, 0]).max() <= 1e-15
    assert np.abs(o.basis_axisym(3.5 * h, h) - [0, 0, 0, 0.5]).max() <= 1e-15
    assert not o.basis_axisym(4 * h, h).any() and not o.basis_axisym(5.2 * h, h).any()
    r = _rng(40)
    for _ in range(300):
        t = r.uniform(0, 3 * h)
        psi = o.basis_axisym(t, h)
        assert abs(psi.sum() - 1.0) <= 1e-14
        c0, c1 = r.standard_normal(2)
        assert abs(float(np.dot(psi, c0 + c1 * np.arange(4))) - (c0 + c1 * t / h)) <= 1e-12
        assert np.count_nonzero(psi) <= 2
        t = r.uniform(3 * h, 4 * h)
        psi = o.basis_axisym(t, h)
        assert np.abs(psi[:3]).max() == 0.0 and abs(psi[3] - (4 - t / h)) <= 1e-14


def pin_axisym_pole_closed_form(o):
    """At a pole every input point of ring t lies at geodesic distance theta_t
    (north) or pi - theta_t (south), so the 2-D sum collapses to a 1-D sum over
    rings: Z_k(pole) = sum_t psi_k(dist_t) q_t sum_p x[t, p], the same at every
    longitude of the pole ring (the ring is one point)."""
    for L, tc_pix in ((16, 3), (12, 5)):
        tc = tc_pix * math.pi / L
        h = tc / 4
        x = _rng(41).standard_normal((1, 1, L + 1, 2 * L))
        Z = o.forward(L + 1, 2 * L, L + 1, 2 * L, tc, x, _select_w4(), sampling=_MW, basis=_AX)[0]
        q = o.quadrature(L + 1, 2 * L, sampling=_MW)
        th = np.arange(L + 1) * math.pi / L
        rows = x[0, 0].sum(axis=1)
        for tp, dist in ((0, th), (L, math.pi - th)):
            expect = np.zeros(4)
            for t in range(L + 1):
                if dist[t] <= tc:
                    expect += o.basis_axisym(float(dist[t]), h) * q[t] * rows[t]
            got = Z[:, tp, :]
            scale = np.abs(expect).max()
            assert np.abs(got - expect[:, None]).max() <= 1e-13 * scale, (L, tp, got[:, 0], expect)


def pin_axisym_grid_isometries(o):
    """An axisymmetric filter sees only the geodesic distance, so the op
    commutes with every isometry that maps the grid onto itself: whole-pixel
    longitude shifts, the mirror phi -> -phi and the flip theta -> pi - theta
    (all exact up to rounding), for the forward and the transposed op, with
    and without 2x downsampling."""
    for (L, Lo) in ((12, 12), (12, 6)):
        a, b, c, d = L + 1, 2 * L, Lo + 1, 2 * Lo
        tc = 3 * math.pi / Lo
        s = b // d
        r = _rng(42)
        x = r.standard_normal((1, 2, a, b))
        w = r.standard_normal((2, 2, 4))
        kw = dict(sampling=_MW, basis=_AX)
        y = o.forward(a, b, c, d, tc, x, w, **kw)
        sc = np.abs(y).max()
        ys = o.forward(a, b, c, d, tc, np.roll(x, s, axis=-1), w, **kw)
        assert np.abs(ys - np.roll(y, 1, axis=-1)).max() <= 1e-13 * sc
        ym = o.forward(a, b, c, d, tc, x[..., (-np.arange(b)) % b], w, **kw)
        assert np.abs(ym - y[..., (-np.arange(d)) % d]).max() <= 1e-13 * sc
        yf = o.forward(a, b, c, d, tc, x[:, :, ::-1, :], w, **kw)
        assert np.abs(yf - y[:, :, ::-1, :]).max() <= 1e-12 * sc
        for tp in (0, c - 1):
            assert np.abs(y[:, :, tp, :] - y[:, :, tp, :1]).max() <= 1e-13 * sc
        xT = r.standard_normal((1, 2, c, d))
        yT = o.transpose(a, b, c, d, tc, xT, w, **kw)
        scT = np.abs(yT).max()
        yTf = o.transpose(a, b, c, d, tc, xT[:, :, ::-1, :], w, **kw)
        assert np.abs(yTf - yT[:, :, ::-1, :]).max() <= 1e-12 * scT
        yTm = o.transpose(a, b, c, d, tc, xT[..., (-np.arange(d)) % d], w, **kw)
        assert np.abs(yTm - yT[..., (-np.arange(b)) % b]).max() <= 1e-13 * scT


def pin_axisym_adjoint(o):
    """The transposed op is the adjoint of the forward op in the
    quadrature-weighted inner products, on the pole-including grid too."""
    for (L, Lo) in ((12, 12), (16, 8)):
        a, b, c, d = L + 1, 2 * L, Lo + 1, 2 * Lo
        tc = 3 * math.pi / Lo
        r = _rng(43)
        x = r.standard_normal((2, 3, a, b))
        g = r.standard_normal((2, 2, c, d))
        w = r.standard_normal((2, 3, 4))
        kw = dict(sampling=_MW, basis=_AX)
        Ax = o.forward(a, b, c, d, tc, x, w, **kw)
        Bg = o.transpose(a, b, c, d, tc, g, w, **kw)
        qo = o.quadrature(c, d, sampling=_MW)[None, None, :, None]
        qi = o.quadrature(a, b, sampling=_MW)[None, None, :, None]
        lhs = float((Ax * g * qo).sum())
        rhs = float((x * Bg * qi).sum())
        assert abs(lhs - rhs) <= 1e-12 * max(abs(lhs), 1.0), (lhs, rhs)


def axisym_filter_integrals(h, n=24):
    """S_k = integral over the sphere of psi_k(Theta) = 2 pi int psi_k(t) sin t dt,
    Gauss-Legendre on each side of the hat."""
    xg, wg = np.polynomial.legendre.leggauss(n)
    S = np.zeros(4)
    for k in range(4):
        for lo, hi in (((k - 1) * h, k * h), (k * h, (k + 1) * h)):
            lo = max(lo, 0.0)
            if hi <= lo:
                continue
            t = lo + (xg + 1) / 2 * (hi - lo)
            f = np.maximum(0.0, 1 - np.abs(t / h - k)) * np.sin(t)
            S[k] += 2 * math.pi * float(((hi - lo) / 2 * wg * f).sum())
    return S


def pin_axisym_constant_input(o):
    """x = 1 on the pole-including grid: every Z_k approximates the filter
    integral S_k (the only error is quadrature, Sec. 3.2), at second order in
    the pixel size at fixed theta_c: from L = 128 on the error falls at least
    3x per doubling and is below 4e-3 at L = 512."""
    tc = 3 * math.pi / 32
    S = axisym_filter_integrals(tc / 4)
    errs = []
    for L in (128, 256, 512):
        pix = np.arange(L + 1) * 2 * L        # one pixel per ring: rings are constant
        Z = o.forward(L + 1, 2 * L, L + 1, 2 * L, tc, np.ones((1, 1, L + 1, 2 * L)), _select_w4(),
                      pix=pix, sampling=_MW, basis=_AX)[0]
        errs.append(float(np.abs(Z / S[:, None] - 1).max()))
    for e0, e1 in zip(errs, errs[1:]):
        assert e1 * 3 <= e0, errs
    assert errs[-1] <= 4e-3, errs


# --------------------------------------------------------------------------- #
# Gradients (App. C): the input gradient is the product with Psi transposed,
# the weight gradient the chain rule through the sparse values.
# --------------------------------------------------------------------------- #
_GRAD_CASES = [
    # (nlat_in, nlon_in, nlat_out, nlon_out, sampling, basis)
    (16, 32, 8, 16, 0, 0),
    (8, 16, 16, 32, 0, 0),
    (9, 16, 9, 16, 1, 1),
    (17, 32, 9, 16, 1, 0),
    (12, 24, 6, 12, 0, 1),
    (16, 32, 8, 16, 0, 2),
    (9, 16, 9, 16, 1, 2),
]


def _grad_tc(a, c, smp):
    return 3 * math.pi / (min(a, c) - (1 if smp == 1 else 0))


def pin_gradients_match_dense_autograd(o):
    """As the paper validated its sparse gradients: the same op written as a
    dense product, y = W . (Psi diag(q) x) (forward) or W^T . (Psi^T diag(q_out)
    xT) (transpose), differentiated by torch's autograd in fp64, gives the
    input and weight gradients to machine precision."""
    import torch
    for (a, b, c, d, smp, bas) in _GRAD_CASES:
        tc = _grad_tc(a, c, smp)
        K = {1: 4, 2: 16}.get(bas, 9)
        kw = dict(sampling=smp, basis=bas)
        psi = torch.tensor(o.psi_dense(a, b, c, d, tc, **kw))            # [Nout, Nin, K]
        qi = torch.tensor(np.repeat(o.quadrature(a, b, sampling=smp), b))
        qo = torch.tensor(np.repeat(o.quadrature(c, d, sampling=smp), d))
        r = _rng(50)
        B, C1, C2 = 2, 3, 4
        # forward: x[B, C1, in], w[C2, C1, K], y[B, C2, out]
        x = torch.tensor(r.standard_normal((B, C1, a * b)), requires_grad=True)
        w = torch.tensor(r.standard_normal((C2, C1, K)), requires_grad=True)
        dy = torch.tensor(r.standard_normal((B, C2, c * d)))
        Z = torch.einsum("jik,bci->bckj", psi, x * qi)
        (torch.einsum("ock,bckj->boj", w, Z) * dy).sum().backward()
        dx = o.input_grad(a, b, c, d, tc, dy.numpy().reshape(B, C2, c, d), w.detach().numpy(), **kw)
        dw = o.weight_grad(a, b, c, d, tc, x.detach().numpy().reshape(B, C1, a, b),
                           dy.numpy().reshape(B, C2, c, d), **kw)
        gx, gw = x.grad.numpy().reshape(dx.shape), w.grad.numpy()
        assert np.abs(dx - gx).max() <= 1e-13 * np.abs(gx).max(), (a, c, smp, bas)
        assert np.abs(dw - gw).max() <= 1e-13 * np.abs(gw).max(), (a, c, smp, bas)
        # transpose: xT[B, C1, out], w[C1, C2, K], yT[B, C2, in]
        xT = torch.tensor(r.standard_normal((B, C1, c * d)), requires_grad=True)
        wT = torch.tensor(r.standard_normal((C1, C2, K)), requires_grad=True)
        dyT = torch.tensor(r.standard_normal((B, C2, a * b)))
        ZT = torch.einsum("jik,bcj->bcki", psi, xT * qo)
        (torch.einsum("cok,bcki->boi", wT, ZT) * dyT).sum().backward()
        dxT = o.input_grad(a, b, c, d, tc, dyT.numpy().reshape(B, C2, a, b), wT.detach().numpy(),
                           transpose=True, **kw)
        dwT = o.weight_grad(a, b, c, d, tc, xT.detach().numpy().reshape(B, C1, c, d),
                            dyT.numpy().reshape(B, C2, a, b), transpose=True, **kw)
        gxT, gwT = xT.grad.numpy().reshape(dxT.shape), wT.grad.numpy()
        assert np.abs(dxT - gxT).max() <= 1e-13 * np.abs(gxT).max(), (a, c, smp, bas)
        assert np.abs(dwT - gwT).max() <= 1e-13 * np.abs(gwT).max(), (a, c, smp, bas)


def pin_input_gradient_is_plain_adjoint(o):
    """<A x, dy> = <x, A^T dy> in the plain (unweighted) inner product, for
    the forward and the transposed op."""
    for (a, b, c, d, smp, bas) in _GRAD_CASES:
        tc = _grad_tc(a, c, smp)
        K = {1: 4, 2: 16}.get(bas, 9)
        kw = dict(sampling=smp, basis=bas)
        r = _rng(51)
        x = r.standard_normal((2, 3, a, b))
        w = r.standard_normal((2, 3, K))
        dy = r.standard_normal((2, 2, c, d))
        lhs = float((o.forward(a, b, c, d, tc, x, w, **kw) * dy).sum())
        rhs = float((x * o.input_grad(a, b, c, d, tc, dy, w, **kw)).sum())
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (lhs, rhs)
        xT = r.standard_normal((2, 3, c, d))
        dyT = r.standard_normal((2, 2, a, b))
        wT = r.standard_normal((3, 2, K))
        lhs = float((o.transpose(a, b, c, d, tc, xT, wT, **kw) * dyT).sum())
        rhs = float((xT * o.input_grad(a, b, c, d, tc, dyT, wT, transpose=True, **kw)).sum())
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (lhs, rhs)


def pin_weight_gradient_by_linearity(o):
    """y is linear in W, so dW[co, ci, k] = <y(x; E_{co,ci,k}), dy> with E the
    unit weight tensor: every element through the op itself."""
    for (a, b, c, d, smp, bas) in _GRAD_CASES[:3]:
        tc = _grad_tc(a, c, smp)
        K = {1: 4, 2: 16}.get(bas, 9)
        kw = dict(sampling=smp, basis=bas)
        r = _rng(52)
        x = r.standard_normal((2, 2, a, b))
        dy = r.standard_normal((2, 3, c, d))
        dw = o.weight_grad(a, b, c, d, tc, x, dy, **kw)
        for (co, ci, k) in [(0, 0, 0), (2, 1, K - 1), (1, 0, K // 2)]:
            E = np.zeros((3, 2, K))
            E[co, ci, k] = 1.0
            ref = float((o.forward(a, b, c, d, tc, x, E, **kw) * dy).sum())
            assert abs(dw[co, ci, k] - ref) <= 1e-12 * max(1.0, abs(ref)), (co, ci, k, dw[co, ci, k], ref)
        xT = r.standard_normal((2, 2, c, d))
        dyT = r.standard_normal((2, 3, a, b))
        dwT = o.weight_grad(a, b, c, d, tc, xT, dyT, transpose=True, **kw)
        for (cp, cc, k) in [(0, 0, 0), (1, 2, K - 1)]:
            E = np.zeros((2, 3, K))
            E[cp, cc, k] = 1.0
            ref = float((o.transpose(a, b, c, d, tc, xT, E, **kw) * dyT).sum())
            assert abs(dwT[cp, cc, k] - ref) <= 1e-12 * max(1.0, abs(ref)), (cp, cc, k)


def pin_forward_adjoint_from_transpose(o):
    """The forward op's adjoint and the transposed op share the filter pairs
    and differ only in where the quadrature sits: A^T dy = diag(q_in) T diag(1 / q_out) dy."""
    for (a, b, c, d, smp, bas) in _GRAD_CASES:
        tc = _grad_tc(a, c, smp)
        K = {1: 4, 2: 16}.get(bas, 9)
        kw = dict(sampling=smp, basis=bas)
        r = _rng(53)
        w = r.standard_normal((3, 2, K))
        dy = r.standard_normal((1, 3, c, d))
        qi = o.quadrature(a, b, sampling=smp)[None, None, :, None]
        qo = o.quadrature(c, d, sampling=smp)[None, None, :, None]
        got = o.input_grad(a, b, c, d, tc, dy, w, **kw)
        ref = qi * o.transpose(a, b, c, d, tc, dy / qo, w, **kw)
        assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()


# --------------------------------------------------------------------------- #
# Separable basis (Sec. 3.4, App. E: four nodes along theta and along phi) and
# depthwise channels (Sec. 4.2).
# --------------------------------------------------------------------------- #
_SEP = 2


def pin_separable_basis(o):
    """psi_{4a+b}(Theta, Phi) = L(Theta/h - a) mu_b(Phi): the theta factor is the
    axisymmetric hat (pinned above); along Phi four periodic hats at b pi/2 with
    the Kronecker property, a partition of unity at every direction, linear
    reproduction between neighbouring nodes and period 2 pi.  At the centre
    only node (0, 0) fires (direction taken as 0)."""
    h = 0.0123
    r = _rng(70)
    for _ in range(300):
        t = r.uniform(0, 4.2 * h)
        ph = r.uniform(-3 * math.pi, 3 * math.pi)
        psi = o.basis_separable(t, ph, h).reshape(4, 4)
        lam = o.basis_axisym(t, h)
        mu = psi.sum(axis=0) / max(lam.sum(), 1e-300) if lam.sum() > 0 else None
        if lam.sum() > 0:
            assert np.abs(psi - np.outer(lam, mu)).max() <= 1e-14
            assert abs(mu.sum() - 1.0) <= 1e-13
            assert np.count_nonzero(mu > 1e-15) <= 2
            # linear between the two nodes around ph
            base = math.floor((ph % (2 * math.pi)) / (math.pi / 2))
            frac = (ph % (2 * math.pi)) / (math.pi / 2) - base
            assert abs(mu[base % 4] - (1 - frac)) <= 1e-12 and abs(mu[(base + 1) % 4] - frac) <= 1e-12
        psi2 = o.basis_separable(t, ph + 2 * math.pi, h)
        assert np.abs(psi2 - psi.ravel()).max() <= 1e-12
    for b in range(4):
        e = np.zeros(4)
        e[b] = 1.0
        psi = o.basis_separable(h, b * math.pi / 2, h).reshape(4, 4)
        assert np.abs(psi[1] - e).max() <= 1e-15 and np.abs(np.delete(psi, 1, axis=0)).max() == 0.0
    c = o.basis_separable(0.0, 1.234, h)
    e = np.zeros(16)
    e[0] = 1.0
    assert np.array_equal(c, e)


def pin_separable_reduces_to_axisymmetric(o):
    """With phi node values all equal the separable filter is the axisymmetric
    one (the phi hats sum to one in every direction): W_sep[.,.,4a+b] = W_ax[.,.,a]
    gives the axisymmetric op's output, forward and transposed, on both grids."""
    for (a, b, c, d, smp) in ((16, 32, 8, 16, 0), (9, 16, 9, 16, 1), (17, 32, 9, 16, 1)):
        tc = 3 * math.pi / (min(a, c) - (1 if smp == 1 else 0))
        r = _rng(71)
        x = r.standard_normal((2, 2, a, b))
        w4 = r.standard_normal((3, 2, 4))
        w16 = np.repeat(w4, 4, axis=2)
        y4 = o.forward(a, b, c, d, tc, x, w4, sampling=smp, basis=_AX)
        y16 = o.forward(a, b, c, d, tc, x, w16, sampling=smp, basis=_SEP)
        assert np.abs(y16 - y4).max() <= 1e-13 * np.abs(y4).max()
        xT = r.standard_normal((2, 3, c, d))
        yT4 = o.transpose(a, b, c, d, tc, xT, w4, sampling=smp, basis=_AX)
        yT16 = o.transpose(a, b, c, d, tc, xT, w16, sampling=smp, basis=_SEP)
        assert np.abs(yT16 - yT4).max() <= 1e-13 * np.abs(yT4).max()


def pin_separable_mirror_symmetry(o):
    """phi -> -phi maps the phi node b to -b (1 <-> 3); theta -> pi - theta maps
    b to 2 - b (0 <-> 2).  The flip is checked where no output meets an input
    point (2x downsampling: the centre's direction convention is not
    flip-symmetric)."""
    a, b, c, d = 16, 32, 8, 16
    tc = 3 * math.pi / c
    r = _rng(72)
    x = r.standard_normal((1, 2, a, b))
    w = r.standard_normal((2, 2, 16))
    y = o.forward(a, b, c, d, tc, x, w, basis=_SEP)
    perm_m = [4 * (k // 4) + (-(k % 4)) % 4 for k in range(16)]
    perm_f = [4 * (k // 4) + (2 - k % 4) % 4 for k in range(16)]
    ym = o.forward(a, b, c, d, tc, x[..., (-np.arange(b)) % b], w[:, :, perm_m], basis=_SEP)
    assert np.abs(ym - y[..., (-np.arange(d)) % d]).max() <= 1e-13 * np.abs(y).max()
    yf = o.forward(a, b, c, d, tc, x[:, :, ::-1, :], w[:, :, perm_f], basis=_SEP)
    assert np.abs(yf - y[:, :, ::-1, :]).max() <= 1e-12 * np.abs(y).max()
    # same grid (outputs on input points): the mirror still holds exactly
    y = o.forward(a, b, a, b, tc, x, w, basis=_SEP)
    ym = o.forward(a, b, a, b, tc, x[..., (-np.arange(b)) % b], w[:, :, perm_m], basis=_SEP)
    assert np.abs(ym - y[..., (-np.arange(b)) % b]).max() <= 1e-13 * np.abs(y).max()


def pin_depthwise_is_per_channel(o):
    """Depthwise channels: channel c of the output is channel c of the input
    filtered by w[c] alone, i.e. each channel run as its own one-channel op."""
    import oracle as _orc
    a, b = 9, 16
    tc = 3 * math.pi / 8
    r = _rng(73)
    for bas, K in ((_AX, 4), (_SEP, 16), (0, 9)):
        x = r.standard_normal((2, 3, a, b))
        wd = r.standard_normal((3, K))
        y = o.forward(a, b, a, b, tc, x, _orc.depthwise_weights(wd), sampling=1, basis=bas)
        for c in range(3):
            yc = o.forward(a, b, a, b, tc, x[:, c:c + 1], wd[c][None, None, :], sampling=1, basis=bas)
            assert np.abs(y[:, c:c + 1] - yc).max() <= 1e-13 * np.abs(y).max()


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
