/*
 * disco_oracle.c -- brute-force fp64 reference for DISCO spherical convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that the GPU library is
 * checked against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load it.  It shares no code, header, table or constant with
 * the GPU library and includes nothing from it.
 *
 * What it computes (Ocampo, Price & McEwen, "Scalable and Equivariant
 * Spherical CNNs by Discrete-Continuous (DISCO) Convolutions", ICLR 2023):
 *
 *   forward   (Sec. 3.2, eq. 4 restricted to SO(3)/SO(2); Sec. 4.1 sparse form)
 *     Z[b,ci,k](j) = sum_i psi_k(R_j^{-1} w_i) q_in(i) x[b,ci,i]
 *     y[b,co,j]    = sum_{ci,k} W[co,ci,k] Z[b,ci,k](j)
 *   transpose (Sec. 3.5, eq. 6: the filter is centred at the transposed op's
 *              input points w_j and weighted by their quadrature)
 *     Z'[b,c',k](i) = sum_j psi_k(R_j^{-1} w_i) q_out(j) xT[b,c',j]
 *     yT[b,c,i]     = sum_{c',k} W[c',c,k] Z'[b,c',k](i)
 *
 * with R_j = Z(phi_j) Y(theta_j) (Sec. 3.2, zyz Euler angles without gamma).
 *
 * It is the plain finite sum over every (output, input) pixel pair: the sparse
 * form (Sec. 4.1) and the longitude-shift compression (Sec. 4.2) are exact
 * rewrites of this sum, so none of them appear here.  Geometry goes through
 * explicit 3x3 rotation matrices in Cartesian coordinates (a different route
 * from the GPU library's plan).  Everything is double precision.
 *
 * Two grids (the cell-centred equiangular grid, and the paper's own
 * pole-including grid of Sec. 4.2 with App. A's quadrature) and two bases
 * (the 3x3 node grid of App. E.2, K = 9, and the axisymmetric filter with four
 * nodes along theta that App. B times, K = 4) are offered.
 *
 * Readings of points the paper leaves open (grid, quadrature rule, rotation
 * handedness, tangent-plane map, node spacing, basis ordering) are stated at
 * each function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

/* ------------------------------------------------------------------------- */
/* Grid.  Equiangular, cell-centred: colatitude (t + 1/2) pi / nlat, longitude
 * 2 pi p / nlon; longitude is the fastest index.  (The paper's own grid keeps
 * both poles, Sec. 4.2 "Explicit sampling"; this workload's grid does not.)  */
/* ------------------------------------------------------------------------- */
double oracle_colatitude(int t, int nlat) { return (t + 0.5) * M_PI / (double)nlat; }
double oracle_longitude(int p, int nlon) { return 2.0 * M_PI * (double)p / (double)nlon; }

/* The paper's own grid (Sec. 4.2, "Explicit sampling"; the antipodal variant
 * of the McEwen-Wiaux sampling, App. A): with L = nlat - 1, colatitude
 * pi t / L for t = 0..L, both poles included, and longitude pi p / L for
 * p = 0..2L-1, i.e. nlon = 2L.  Each pole ring holds 2L samples of one point.
 * sampling 0 = cell-centred (above), 1 = this grid. */
double oracle_colatitude_s(int t, int nlat, int sampling)
{
    if (sampling == 1) return M_PI * (double)t / (double)(nlat - 1);
    return oracle_colatitude(t, nlat);
}

/* ------------------------------------------------------------------------- */
/* Quadrature weights q(theta_t), one per ring; a pixel's weight is its ring's.
 * The paper adopts sampling-theorem quadrature without upsampling (Sec. 3.2,
 * Sec. 4.1, App. A).  App. A gives weights only for its pole-including grid;
 * on the cell-centred grid the analogous rule that integrates band-limited
 * signals exactly is Fejer's first rule in x = cos(theta), times 2 pi / nlon
 * for the longitude sum:
 *   w_t = (2/n) [ 1 - 2 sum_{m=1}^{floor(n/2)} cos(2 m theta_t) / (4 m^2 - 1) ]
 * kind 0 = that rule; kind 1 = exact cell areas 2 sin(theta_t) sin(dtheta/2). */
/* ------------------------------------------------------------------------- */
int oracle_quadrature(int nlat, int nlon, int kind, double* q)
{
    if (nlat < 1 || nlon < 1 || !q) return 1;
    for (int t = 0; t < nlat; ++t) {
        double th = oracle_colatitude(t, nlat);
        double w;
        if (kind == 0) {
            double s = 0.0;
            for (int m = 1; m <= nlat / 2; ++m)
                s += cos(2.0 * m * th) / (4.0 * (double)m * (double)m - 1.0);
            w = (2.0 / nlat) * (1.0 - 2.0 * s);
        } else if (kind == 1) {
            w = 2.0 * sin(th) * sin(0.5 * M_PI / nlat);
        } else {
            return 2;
        }
        q[t] = (2.0 * M_PI / nlon) * w;
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Quadrature of the pole-including grid (App. A), taken in the appendix's
 * steps.  The colatitude integral of a band-limited signal is extended to the
 * torus: sin(theta) on [0, pi], zero on (pi, 2 pi), has the Fourier
 * coefficients
 *   w(m) = int_0^pi sin(t) e^{i m t} dt = +-i pi/2 (m = +-1), 0 (other odd m),
 *          2 / (1 - m^2) (even m);
 * its band-limited version is w_r(t) = sum_{m=-L}^{L-1} w(m) e^{i m t}; the
 * torus sample at colatitude theta_{2L-t} = 2 pi - theta_t is the sphere's
 * sample at (theta_t, phi + pi), so its weight folds back onto ring t (not for
 * the poles, t = 0 and t = L, which are their own images):
 *   q(theta_t) = 2 pi / (2L)^2 [ w_r(theta_t) + (1 - d_{t0})(1 - d_{tL}) w_r(theta_{2L-t}) ]
 * (spin s = 0).  The first factor 2 pi / (2L) is the longitude step of the
 * 2L samples per ring, the second 1 / (2L) the normalisation of the 2L-point
 * transform along the extended colatitude; the rule is stated for nlon = 2L
 * and is only offered there.  w_r is real at the sample points (conjugate
 * pairs m, -m; e^{-i L theta_t} = (-1)^t), its real part is taken.          */
/* ------------------------------------------------------------------------- */
static void sin_fourier(int m, double* re, double* im)
{
    *re = 0.0;
    *im = 0.0;
    if (m == 1) {
        *im = 0.5 * M_PI;
    } else if (m == -1) {
        *im = -0.5 * M_PI;
    } else if (m % 2 == 0) {
        *re = 2.0 / (1.0 - (double)m * (double)m);
    }
}

static double band_limited_sin(int L, double theta)
{
    double acc = 0.0;
    for (int m = -L; m <= L - 1; ++m) {
        double re, im;
        sin_fourier(m, &re, &im);
        /* Re(w(m) e^{i m theta}) */
        acc += re * cos(m * theta) - im * sin(m * theta);
    }
    return acc;
}

static int quadrature_mw(int nlat, int nlon, double* q)
{
    int L = nlat - 1;
    if (L < 1 || nlon != 2 * L) return 1;
    for (int t = 0; t <= L; ++t) {
        double s = band_limited_sin(L, M_PI * (double)t / (double)L);
        if (t != 0 && t != L) s += band_limited_sin(L, M_PI * (double)(2 * L - t) / (double)L);
        q[t] = 2.0 * M_PI / ((2.0 * L) * (2.0 * L)) * s;
    }
    return 0;
}

/* Weights of either grid: sampling 1 takes App. A's rule (kind must be 0). */
int oracle_quadrature_s(int nlat, int nlon, int sampling, int kind, double* q)
{
    if (sampling == 0) return oracle_quadrature(nlat, nlon, kind, q);
    if (sampling != 1 || kind != 0 || !q) return 2;
    return quadrature_mw(nlat, nlon, q);
}

/* ------------------------------------------------------------------------- */
/* Rotations.  Active, right-handed:
 *   Z(a) = [[cos a, -sin a, 0], [sin a, cos a, 0], [0, 0, 1]]
 *   Y(b) = [[cos b, 0, sin b], [0, 1, 0], [-sin b, 0, cos b]]
 * R_j^{-1} = Y(-theta_j) Z(-phi_j) maps the output point to the north pole.  */
/* ------------------------------------------------------------------------- */
static void mat_z(double a, double m[9])
{
    double c = cos(a), s = sin(a);
    m[0] = c;   m[1] = -s;  m[2] = 0.0;
    m[3] = s;   m[4] = c;   m[5] = 0.0;
    m[6] = 0.0; m[7] = 0.0; m[8] = 1.0;
}
static void mat_y(double b, double m[9])
{
    double c = cos(b), s = sin(b);
    m[0] = c;   m[1] = 0.0; m[2] = s;
    m[3] = 0.0; m[4] = 1.0; m[5] = 0.0;
    m[6] = -s;  m[7] = 0.0; m[8] = c;
}
static void mat_mul(const double a[9], const double b[9], double c[9])
{
    for (int r = 0; r < 3; ++r)
        for (int col = 0; col < 3; ++col) {
            double s = 0.0;
            for (int k = 0; k < 3; ++k) s += a[3 * r + k] * b[3 * k + col];
            c[3 * r + col] = s;
        }
}
/* M = R^{-1} for R = Z(phi) Y(theta). */
static void inverse_rotation(double theta, double phi, double m[9])
{
    double my[9], mz[9];
    mat_y(-theta, my);
    mat_z(-phi, mz);
    mat_mul(my, mz, m);
}
static void unit_vector(double theta, double phi, double e[3])
{
    e[0] = sin(theta) * cos(phi);
    e[1] = sin(theta) * sin(phi);
    e[2] = cos(theta);
}

/* Filter-frame coordinates of R_j^{-1} w_i.  Theta is the geodesic distance
 * from the filter centre, taken with atan2 (never acos).  The tangent-plane
 * map is azimuthal equidistant, (u, v) = Theta (cos Phi, sin Phi): it is the
 * azimuthal projection that puts the 3x3 grid's edge nodes at Theta = h and
 * its corner nodes at Theta = sqrt(2) h, as App. E.2 places them.  Phi = 0
 * points to increasing colatitude (south), Phi = pi/2 to increasing
 * longitude (east). */
static void frame_coords_m(const double m[9], const double e[3],
                           double* Theta, double* u, double* v)
{
    double xr = m[0] * e[0] + m[1] * e[1] + m[2] * e[2];
    double yr = m[3] * e[0] + m[4] * e[1] + m[5] * e[2];
    double zr = m[6] * e[0] + m[7] * e[1] + m[8] * e[2];
    double rho = hypot(xr, yr);
    double th = atan2(rho, zr);
    *Theta = th;
    if (rho > 0.0) {
        *u = th * xr / rho;
        *v = th * yr / rho;
    } else {
        *u = 0.0;
        *v = 0.0;
    }
}

void oracle_frame_coords(double theta_j, double phi_j, double theta_i, double phi_i,
                         double* Theta, double* u, double* v)
{
    double m[9], e[3];
    inverse_rotation(theta_j, phi_j, m);
    unit_vector(theta_i, phi_i, e);
    frame_coords_m(m, e, Theta, u, v);
}

/* ------------------------------------------------------------------------- */
/* Filter basis (Sec. 3.4 and App. E.2): a square 3x3 node grid with spacing h
 * in the tangent plane, nodes at ((a-1) h, (b-1) h), a, b in {0,1,2}, node
 * index k = 3a + b (a along u = south, b along v = east).  Values between
 * nodes by bilinear interpolation of a zero-padded node grid, i.e. the tensor
 * product of hat functions L(s) = max(0, 1 - |s|):
 *   psi_k(u, v) = L(u/h - (a-1)) L(v/h - (b-1)).
 * The filter is zero beyond the cutoff Theta > theta_c (Sec. 3.4).           */
/* ------------------------------------------------------------------------- */
static double hat(double s)
{
    double a = fabs(s);
    return a < 1.0 ? 1.0 - a : 0.0;
}

void oracle_basis(double u, double v, double h, double psi[9])
{
    for (int a = 0; a < 3; ++a)
        for (int b = 0; b < 3; ++b)
            psi[3 * a + b] = hat(u / h - (a - 1)) * hat(v / h - (b - 1));
}

/* Axisymmetric basis (Sec. 3.4: filters psi(theta) with equally spaced nodes
 * along theta and linear interpolation, zero above the cutoff), the one the
 * paper times (App. B: 4 nodes, cutoff 3 pi / L).  Nodes at k h, k = 0..3,
 * with h = theta_c / 4 by default, so that the last hat reaches zero exactly
 * at the cutoff and the filter is continuous:
 *   psi_k(Theta) = L(Theta / h - k).                                          */
void oracle_basis_axisym(double Theta, double h, double psi[4])
{
    for (int k = 0; k < 4; ++k) psi[k] = hat(Theta / h - k);
}

/* Separable basis (Sec. 3.4: psi(theta, phi) = theta-part(theta) phi-part(phi),
 * equally spaced nodes along both, linear interpolation; App. E uses four
 * nodes along theta and along phi).  Along Theta the four hats of the
 * axisymmetric basis; along the direction Phi = atan2(v, u) of the filter
 * frame (0 south, pi/2 east) four periodic hats at Phi = b pi / 2,
 *   mu_b(Phi) = max(0, 1 - |Phi - b pi/2|_{mod 2 pi} / (pi / 2)),
 * and psi_{4a+b} = L(Theta / h - a) mu_b(Phi), K = 16.  The separable filter
 * with node values t_a and p_b is W_{4a+b} = t_a p_b.  At the centre
 * (Theta = 0) the direction is undefined; Phi = 0 is taken there (the value of
 * atan2 at the origin), and any point within 1e-12 rad of the centre counts
 * as the centre. */
void oracle_basis_separable(double Theta, double Phi, double h, double psi[16])
{
    if (Theta <= 1e-12) Phi = 0.0;
    for (int a = 0; a < 4; ++a) {
        double la = hat(Theta / h - a);
        for (int b = 0; b < 4; ++b) {
            double d = fmod(fabs(Phi - b * 0.5 * M_PI), 2.0 * M_PI);
            if (d > M_PI) d = 2.0 * M_PI - d;
            psi[4 * a + b] = la * hat(d / (0.5 * M_PI));
        }
    }
}

/* basis 0 = the 3x3 grid (K = 9), 1 = axisymmetric (K = 4), 2 = separable (K = 16). */
static int basis_size(int basis) { return basis == 1 ? 4 : basis == 2 ? 16 : 9; }

/* Evaluate the K basis functions of the filter centred at (theta_j, phi_j)
 * at the input point e; returns 0 if the point is beyond the cutoff or all
 * values vanish, 1 otherwise. */
static int filter_values(int basis, const double m[9], const double e[3], double theta_c,
                         double h, double psi[16])
{
    double Th, u, v;
    frame_coords_m(m, e, &Th, &u, &v);
    if (Th > theta_c) return 0;
    if (basis == 1)
        oracle_basis_axisym(Th, h, psi);
    else if (basis == 2)
        oracle_basis_separable(Th, atan2(v, u), h, psi);
    else
        oracle_basis(u, v, h, psi);
    for (int k = 0; k < basis_size(basis); ++k)
        if (psi[k] != 0.0) return 1;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Dense Psi tensor psi[j][i][k] = psi_k(R_j^{-1} w_i) (no quadrature),
 * j over out-grid pixels, i over in-grid pixels (Sec. 4.1).  Tiny grids only. */
/* ------------------------------------------------------------------------- */
int oracle_psi_dense_ex(int nlat_in, int nlon_in, int nlat_out, int nlon_out, int sampling,
                        int basis, double theta_c, double h, double* psi)
{
    if (!psi) return 1;
    int K = basis_size(basis);
    int64_t n_in = (int64_t)nlat_in * nlon_in, n_out = (int64_t)nlat_out * nlon_out;
    memset(psi, 0, sizeof(double) * (size_t)(n_out * n_in * K));
#pragma omp parallel for schedule(dynamic)
    for (int64_t j = 0; j < n_out; ++j) {
        double m[9];
        inverse_rotation(oracle_colatitude_s((int)(j / nlon_out), nlat_out, sampling),
                         oracle_longitude((int)(j % nlon_out), nlon_out), m);
        for (int64_t i = 0; i < n_in; ++i) {
            double e[3], val[16];
            unit_vector(oracle_colatitude_s((int)(i / nlon_in), nlat_in, sampling),
                        oracle_longitude((int)(i % nlon_in), nlon_in), e);
            if (filter_values(basis, m, e, theta_c, h, val))
                for (int k = 0; k < K; ++k) psi[(j * n_in + i) * K + k] = val[k];
        }
    }
    return 0;
}

int oracle_psi_dense(int nlat_in, int nlon_in, int nlat_out, int nlon_out,
                     double theta_c, double h, double* psi)
{
    return oracle_psi_dense_ex(nlat_in, nlon_in, nlat_out, nlon_out, 0, 0, theta_c, h, psi);
}

/* ------------------------------------------------------------------------- */
/* The convolution sums.
 *
 * `window` = 0 visits every input ring; `window` = 1 visits only rings whose
 * colatitude is within theta_c of the output point's.  The second is exact:
 * by the spherical law of cosines the geodesic distance between two points is
 * at least the difference of their colatitudes, so every skipped ring lies
 * entirely beyond the cutoff.  Inside a visited ring every longitude is
 * visited.
 *
 * `pix` lists the flat output-pixel indices to compute (t * nlon + p); y is
 * written as y[b][c][n] for n over that list.                                */
/* ------------------------------------------------------------------------- */
typedef struct {
    int nlat, nlon;
} grid_t;

typedef struct {
    int sampling;  /* 0 cell-centred, 1 pole-including */
    int basis;     /* 0 the 3x3 grid, 1 axisymmetric */
    int quad_kind; /* 0 the grid's sampling-theorem rule, 1 cell areas */
} config_t;

/* Shared body: the filter is centred at points of grid `ctr`, evaluated at
 * points of grid `ev`.  forward: centre = output pixel, sum over input pixels
 * (the evaluation points), quadrature of the evaluation points' grid.
 * transpose: centre = each input pixel of the transposed op, evaluation at the
 * output pixel, quadrature of the centres' grid. */
static int disco_sum(int transpose, grid_t g_in, grid_t g_out, double theta_c, double h,
                     config_t cfg, int B, int Cin, int Cout, const double* x,
                     const double* w, double* y, int window, int64_t n_pix,
                     const int64_t* pix)
{
    if (!x || !w || !y || !pix || B < 0 || Cin < 1 || Cout < 1) return 1;
    const int K = basis_size(cfg.basis);
    const int smp = cfg.sampling;
    double* q_in = (double*)malloc(sizeof(double) * (size_t)g_in.nlat);
    if (!q_in) return 3;
    if (oracle_quadrature_s(g_in.nlat, g_in.nlon, smp, cfg.quad_kind, q_in)) {
        free(q_in);
        return 2;
    }
    int64_t n_in = (int64_t)g_in.nlat * g_in.nlon;
    int64_t n_out_total = (int64_t)g_out.nlat * g_out.nlon;
    int bad = 0;
#pragma omp parallel
    {
        double* Z = (double*)malloc(sizeof(double) * (size_t)B * Cin * 16);
#pragma omp for schedule(dynamic)
        for (int64_t n = 0; n < n_pix; ++n) {
            int64_t o = pix[n];
            if (o < 0 || o >= n_out_total || !Z) {
#pragma omp atomic write
                bad = 1;
                continue;
            }
            int to = (int)(o / g_out.nlon), po = (int)(o % g_out.nlon);
            double th_o = oracle_colatitude_s(to, g_out.nlat, smp), ph_o = oracle_longitude(po, g_out.nlon);
            memset(Z, 0, sizeof(double) * (size_t)B * Cin * 16);
            double m_o[9], e_o[3];
            inverse_rotation(th_o, ph_o, m_o);
            unit_vector(th_o, ph_o, e_o);
            for (int t = 0; t < g_in.nlat; ++t) {
                double th_i = oracle_colatitude_s(t, g_in.nlat, smp);
                if (window && fabs(th_i - th_o) > theta_c) continue;
                for (int p = 0; p < g_in.nlon; ++p) {
                    double ph_i = oracle_longitude(p, g_in.nlon);
                    double val[16];
                    int nz;
                    if (!transpose) {
                        double e_i[3];
                        unit_vector(th_i, ph_i, e_i);
                        nz = filter_values(cfg.basis, m_o, e_i, theta_c, h, val);
                    } else {
                        double m_i[9];
                        inverse_rotation(th_i, ph_i, m_i);
                        nz = filter_values(cfg.basis, m_i, e_o, theta_c, h, val);
                    }
                    if (!nz) continue;
                    double qw = q_in[t];
                    for (int b = 0; b < B; ++b)
                        for (int c = 0; c < Cin; ++c) {
                            double xv = x[((int64_t)b * Cin + c) * n_in + (int64_t)t * g_in.nlon + p];
                            double* zc = Z + ((size_t)b * Cin + c) * 16;
                            for (int k = 0; k < K; ++k) zc[k] += val[k] * qw * xv;
                        }
                }
            }
            for (int b = 0; b < B; ++b)
                for (int co = 0; co < Cout; ++co) {
                    double s = 0.0;
                    for (int ci = 0; ci < Cin; ++ci)
                        for (int k = 0; k < K; ++k) {
                            /* forward: W[co][ci][k]; transpose: W[ci][co][k]. */
                            double wv = transpose ? w[((int64_t)ci * Cout + co) * K + k]
                                                  : w[((int64_t)co * Cin + ci) * K + k];
                            s += wv * Z[((size_t)b * Cin + ci) * 16 + k];
                        }
                    y[((int64_t)b * Cout + co) * n_pix + n] = s;
                }
        }
        free(Z);
    }
    free(q_in);
    return bad ? 4 : 0;
}

/* Forward op from the in-grid to the out-grid.
 * x[B][Cin][nlat_in][nlon_in], w[Cout][Cin][K], y[B][Cout][n_pix]. */
int oracle_forward_ex(int nlat_in, int nlon_in, int nlat_out, int nlon_out, int sampling,
                      int basis, double theta_c, double h, int quad_kind, int B, int Cin,
                      int Cout, const double* x, const double* w, double* y, int window,
                      int64_t n_pix, const int64_t* pix)
{
    grid_t gi = {nlat_in, nlon_in}, go = {nlat_out, nlon_out};
    config_t cfg = {sampling, basis, quad_kind};
    return disco_sum(0, gi, go, theta_c, h, cfg, B, Cin, Cout, x, w, y, window, n_pix, pix);
}

/* Transposed op of the same plan, from the out-grid back to the in-grid.
 * xT[B][CinT][nlat_out][nlon_out], w[CinT][CoutT][K], yT[B][CoutT][n_pix]
 * with pix indexing the in-grid. */
int oracle_transpose_ex(int nlat_in, int nlon_in, int nlat_out, int nlon_out, int sampling,
                        int basis, double theta_c, double h, int quad_kind, int B, int CinT,
                        int CoutT, const double* xT, const double* w, double* yT, int window,
                        int64_t n_pix, const int64_t* pix)
{
    /* The transposed op reads the plan's out-grid and writes its in-grid. */
    grid_t gi = {nlat_out, nlon_out}, go = {nlat_in, nlon_in};
    config_t cfg = {sampling, basis, quad_kind};
    return disco_sum(1, gi, go, theta_c, h, cfg, B, CinT, CoutT, xT, w, yT, window, n_pix, pix);
}

/* The cell-centred grid with the 3x3 basis. */
int oracle_forward(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double theta_c,
                   double h, int quad_kind, int B, int Cin, int Cout, const double* x,
                   const double* w, double* y, int window, int64_t n_pix, const int64_t* pix)
{
    return oracle_forward_ex(nlat_in, nlon_in, nlat_out, nlon_out, 0, 0, theta_c, h, quad_kind,
                             B, Cin, Cout, x, w, y, window, n_pix, pix);
}

int oracle_transpose(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double theta_c,
                     double h, int quad_kind, int B, int CinT, int CoutT, const double* xT,
                     const double* w, double* yT, int window, int64_t n_pix, const int64_t* pix)
{
    return oracle_transpose_ex(nlat_in, nlon_in, nlat_out, nlon_out, 0, 0, theta_c, h, quad_kind,
                               B, CinT, CoutT, xT, w, yT, window, n_pix, pix);
}

/* ------------------------------------------------------------------------- */
/* Gradients (App. C).  Both ops are linear in x and in W.  For a scalar loss
 * with upstream gradient dy = d loss / dy:
 *   input gradient   dx = A^T dy, the product with Psi transposed in input
 *                    and output coordinates (App. C, activation gradient);
 *   weight gradient  dW = d <dy, y> / dW: the chain rule through the sparse
 *                    values (App. C, kernel-tensor gradient) to the weights
 *                    of the basis functions,
 *     forward   dW[co][ci][k] = sum_{b,j} dy[b,co,j]  Z[b,ci,k](j)
 *     transpose dW[c'][c][k]  = sum_{b,i} dyT[b,c,i]  Z'[b,c',k](i).
 * Written out per pair of points: the filter is always centred at the
 * plan's out-grid point j and evaluated at its in-grid point i; the forward
 * op carries the quadrature weight q_in(i), the transposed op q_out(j), and
 * each op's adjoint carries the same factor, so that
 *   forward adjoint    dx[b,ci,i]  = sum_{co,k} W[co][ci][k] sum_j psi_k(R_j^{-1} w_i) q_in(i)  dy[b,co,j]
 *   transpose adjoint  dxT[b,c',j] = sum_{c,k}  W[c'][c][k]  sum_i psi_k(R_j^{-1} w_i) q_out(j) dyT[b,c,i]
 */
/* ------------------------------------------------------------------------- */
static int adjoint_sum(int of_transpose, grid_t g_in, grid_t g_out, double theta_c, double h,
                       config_t cfg, int B, int C_dy, int C_dx, const double* dy,
                       const double* w, double* dx, int window, int64_t n_pix, const int64_t* pix)
{
    if (!dy || !w || !dx || !pix || B < 0 || C_dy < 1 || C_dx < 1) return 1;
    const int K = basis_size(cfg.basis);
    const int smp = cfg.sampling;
    /* Outputs: the in-grid for the forward op's adjoint, the out-grid for the
     * transposed op's; the sum runs over the other grid. */
    grid_t g_dst = of_transpose ? g_out : g_in;
    grid_t g_src = of_transpose ? g_in : g_out;
    double* q = (double*)malloc(sizeof(double) * (size_t)(of_transpose ? g_out.nlat : g_in.nlat));
    if (!q) return 3;
    if (oracle_quadrature_s(of_transpose ? g_out.nlat : g_in.nlat, of_transpose ? g_out.nlon : g_in.nlon,
                            smp, cfg.quad_kind, q)) {
        free(q);
        return 2;
    }
    int64_t n_src = (int64_t)g_src.nlat * g_src.nlon, n_dst = (int64_t)g_dst.nlat * g_dst.nlon;
    int bad = 0;
#pragma omp parallel
    {
        double* Z = (double*)malloc(sizeof(double) * (size_t)B * C_dy * 16);
#pragma omp for schedule(dynamic)
        for (int64_t n = 0; n < n_pix; ++n) {
            int64_t o = pix[n];
            if (o < 0 || o >= n_dst || !Z) {
#pragma omp atomic write
                bad = 1;
                continue;
            }
            int td = (int)(o / g_dst.nlon), pd = (int)(o % g_dst.nlon);
            double th_d = oracle_colatitude_s(td, g_dst.nlat, smp), ph_d = oracle_longitude(pd, g_dst.nlon);
            memset(Z, 0, sizeof(double) * (size_t)B * C_dy * 16);
            double m_d[9], e_d[3];
            inverse_rotation(th_d, ph_d, m_d);
            unit_vector(th_d, ph_d, e_d);
            for (int t = 0; t < g_src.nlat; ++t) {
                double th_s = oracle_colatitude_s(t, g_src.nlat, smp);
                if (window && fabs(th_s - th_d) > theta_c) continue;
                for (int p = 0; p < g_src.nlon; ++p) {
                    double ph_s = oracle_longitude(p, g_src.nlon);
                    double val[16];
                    int nz;
                    if (!of_transpose) {
                        /* centre at the source point j (out-grid), evaluate at the output i */
                        double m_s[9];
                        inverse_rotation(th_s, ph_s, m_s);
                        nz = filter_values(cfg.basis, m_s, e_d, theta_c, h, val);
                    } else {
                        /* centre at the output j (out-grid), evaluate at the source i */
                        double e_s[3];
                        unit_vector(th_s, ph_s, e_s);
                        nz = filter_values(cfg.basis, m_d, e_s, theta_c, h, val);
                    }
                    if (!nz) continue;
                    for (int b = 0; b < B; ++b)
                        for (int c = 0; c < C_dy; ++c) {
                            double v = dy[((int64_t)b * C_dy + c) * n_src + (int64_t)t * g_src.nlon + p];
                            double* zc = Z + ((size_t)b * C_dy + c) * 16;
                            for (int k = 0; k < K; ++k) zc[k] += val[k] * v;
                        }
                }
            }
            double qw = q[td];
            for (int b = 0; b < B; ++b)
                for (int cx = 0; cx < C_dx; ++cx) {
                    double s = 0.0;
                    for (int cy = 0; cy < C_dy; ++cy)
                        for (int k = 0; k < K; ++k) {
                            /* forward op: W[co = cy][ci = cx][k]; transposed op: W[c' = cx][c = cy][k]. */
                            double wv = of_transpose ? w[((int64_t)cx * C_dy + cy) * K + k]
                                                     : w[((int64_t)cy * C_dx + cx) * K + k];
                            s += wv * Z[((size_t)b * C_dy + cy) * 16 + k];
                        }
                    dx[((int64_t)b * C_dx + cx) * n_pix + n] = qw * s;
                }
        }
        free(Z);
    }
    free(q);
    return bad ? 4 : 0;
}

/* Forward op's input gradient: dy[B][Cout][nlat_out][nlon_out], w[Cout][Cin][K]
 * -> dx[B][Cin][n_pix], pix over the in-grid. */
int oracle_forward_adjoint_ex(int nlat_in, int nlon_in, int nlat_out, int nlon_out, int sampling,
                              int basis, double theta_c, double h, int quad_kind, int B, int Cout,
                              int Cin, const double* dy, const double* w, double* dx, int window,
                              int64_t n_pix, const int64_t* pix)
{
    grid_t gi = {nlat_in, nlon_in}, go = {nlat_out, nlon_out};
    config_t cfg = {sampling, basis, quad_kind};
    return adjoint_sum(0, gi, go, theta_c, h, cfg, B, Cout, Cin, dy, w, dx, window, n_pix, pix);
}

/* Transposed op's input gradient: dyT[B][CoutT][nlat_in][nlon_in],
 * w[CinT][CoutT][K] -> dxT[B][CinT][n_pix], pix over the out-grid. */
int oracle_transpose_adjoint_ex(int nlat_in, int nlon_in, int nlat_out, int nlon_out, int sampling,
                                int basis, double theta_c, double h, int quad_kind, int B, int CoutT,
                                int CinT, const double* dyT, const double* w, double* dxT, int window,
                                int64_t n_pix, const int64_t* pix)
{
    grid_t gi = {nlat_in, nlon_in}, go = {nlat_out, nlon_out};
    config_t cfg = {sampling, basis, quad_kind};
    return adjoint_sum(1, gi, go, theta_c, h, cfg, B, CoutT, CinT, dyT, w, dxT, window, n_pix, pix);
}

/* Weight gradient of either op: Z of every output pixel from the same sum as
 * the op (disco_sum with the selection W[k'][0][k] = delta(k, k') per input
 * channel would give it too; here it is accumulated directly), then
 * dW += dy (x) Z over batch and output pixels.
 *   forward:   x[B][Cin][in-grid],  dy[B][Cout][out-grid], dw[Cout][Cin][K]
 *   transpose: xT[B][CinT][out-grid], dyT[B][CoutT][in-grid], dw[CinT][CoutT][K] */
int oracle_weight_grad_ex(int transpose, int nlat_in, int nlon_in, int nlat_out, int nlon_out,
                          int sampling, int basis, double theta_c, double h, int quad_kind, int B,
                          int C_x, int C_dy, const double* x, const double* dy, double* dw)
{
    if (!x || !dy || !dw || B < 0 || C_x < 1 || C_dy < 1) return 1;
    const int K = basis_size(basis);
    grid_t gi = transpose ? (grid_t){nlat_out, nlon_out} : (grid_t){nlat_in, nlon_in};
    grid_t go = transpose ? (grid_t){nlat_in, nlon_in} : (grid_t){nlat_out, nlon_out};
    config_t cfg = {sampling, basis, quad_kind};
    int64_t n_out = (int64_t)go.nlat * go.nlon;
    int64_t* pix = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_out);
    /* Z for every (b, ci, k) through the op's own sum with a selection W:
     * input channel c of batch item b becomes item b * C_x + c with one
     * channel, and output channel k' of W_sel[k'][0][k] = delta picks Z_k. */
    double* wsel = (double*)calloc((size_t)K * K, sizeof(double));
    double* Z = (double*)malloc(sizeof(double) * (size_t)B * C_x * K * n_out);
    if (!pix || !wsel || !Z) {
        free(pix); free(wsel); free(Z);
        return 3;
    }
    for (int64_t n = 0; n < n_out; ++n) pix[n] = n;
    for (int k = 0; k < K; ++k) wsel[k * K + k] = 1.0;
    int rc = disco_sum(transpose, gi, go, theta_c, h, cfg, B * C_x, 1, K, x, wsel, Z, 1, n_out, pix);
    if (rc == 0) {
        memset(dw, 0, sizeof(double) * (size_t)C_x * C_dy * K);
        for (int b = 0; b < B; ++b)
            for (int cx = 0; cx < C_x; ++cx)
                for (int cy = 0; cy < C_dy; ++cy)
                    for (int k = 0; k < K; ++k) {
                        const double* zr = Z + (((int64_t)b * C_x + cx) * K + k) * n_out;
                        const double* dr = dy + ((int64_t)b * C_dy + cy) * n_out;
                        double s = 0.0;
                        for (int64_t n = 0; n < n_out; ++n) s += dr[n] * zr[n];
                        /* forward: dW[co = cy][ci = cx][k]; transpose: dW[c' = cx][c = cy][k] */
                        int64_t at = transpose ? ((int64_t)cx * C_dy + cy) * K + k : ((int64_t)cy * C_x + cx) * K + k;
                        dw[at] += s;
                    }
    }
    free(pix); free(wsel); free(Z);
    return rc;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
