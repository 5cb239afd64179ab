// disco_plan.cpp -- host construction of the sparse psi tensor (fp64).
//
// Sec. 4.1: Psi_ji = psi(R_j^{-1} w_i) is evaluated only where it can be
// non-zero, using the cutoff theta_c to limit the rotated coordinates that are
// computed.  Sec. 4.2: on an equiangular grid a rotation about z is a cyclic
// longitude shift, so the pattern of one output ring (per longitude phase) is
// stored once and reused at every output longitude.
//
// Per output ring the builder visits only input rings whose colatitude is
// within the search radius (the geodesic distance is at least the colatitude
// difference) and, on each, only the closed-form longitude window where the
// distance can be within the radius (spherical law of cosines), plus one
// pixel of margin.  Each candidate pair is evaluated in fp64 with the
// half-angle form of R_j^{-1} w_i, which keeps full relative precision for
// nearby points (the colatitude difference comes from integer ring indices,
// the longitude difference from an integer residue):
//   x' = sin(ti - tj) - 2 sin(ti) cos(tj) sin^2(dphi/2)
//   y' = sin(ti) sin(dphi)
//   z' = cos(ti - tj) - 2 sin(ti) sin(tj) sin^2(dphi/2)
// Theta = atan2(|(x', y')|, z'), (u, v) = Theta (x', y') / |(x', y')|
// (azimuthal equidistant tangent plane: u south, v east); the axisymmetric
// basis needs Theta only, the separable one Theta and the direction
// Phi = atan2(v, u) (0 south, pi / 2 east; 0 at the centre itself).  Basis values below 1e-12 (rounding noise where a
// hat is evaluated at its own zero) are set to zero, and entries whose basis
// values are all zero are dropped.  Values absorb the quadrature weight of the
// op's input ring (Sec. 4.1: quadrature absorbed into f) and are then rounded
// to fp32.
//
// On the pole-including grid (Sec. 4.2 explicit sampling) a pole ring is one
// point: its sine is taken as exactly zero, which makes every window that
// touches it a whole ring, and the distance to it is the colatitude
// difference alone.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <numeric>

#include "disco.h"
#include "disco_internal.h"

namespace disco {

namespace {

constexpr double kPi = 3.14159265358979323846;
// Basis values below this (the hats are at most 1) are treated as zero.
constexpr double kPsiFloor = 1e-12;

bool poles(int sampling) { return sampling == DISCO_SAMPLING_POLES; }

// Colatitude of ring t: cell-centred (t + 1/2) pi / nlat, or pi t / (nlat - 1)
// on the pole-including grid.
double colat(int t, int nlat, int sampling) {
    return poles(sampling) ? kPi * t / (nlat - 1) : (t + 0.5) * kPi / nlat;
}

// sin and cos of ring t's colatitude, exactly (0, +-1) at the poles.
void ring_trig(int t, int nlat, int sampling, double* s, double* c) {
    if (poles(sampling) && (t == 0 || t == nlat - 1)) {
        *s = 0.0;
        *c = t == 0 ? 1.0 : -1.0;
        return;
    }
    const double th = colat(t, nlat, sampling);
    *s = std::sin(th);
    *c = std::cos(th);
}

// theta(ti on the op's input grid) - theta(to on its output grid), from
// integers.
double colat_diff(int ti, int nlat_i, int to, int nlat_o, int sampling) {
    if (poles(sampling)) {
        const int64_t num = (int64_t)ti * (nlat_o - 1) - (int64_t)to * (nlat_i - 1);
        return kPi * (double)num / ((double)(nlat_i - 1) * (nlat_o - 1));
    }
    const int64_t num = (int64_t)(2 * ti + 1) * nlat_o - (int64_t)(2 * to + 1) * nlat_i;
    return kPi * (double)num / (2.0 * (double)nlat_i * nlat_o);
}

// App. A weights of the pole-including grid (L = nlat - 1, nlon = 2L):
// q(theta_t) = 2 pi / (2L)^2 [w_r(theta_t) + w_r(theta_{2L-t})] inside and
// 2 pi / (2L)^2 w_r(theta_t) at the poles, w_r the band-limited (|m| <= L,
// m = -L included) Fourier series of sin(theta) on [0, pi], zero on
// (pi, 2 pi).  Taken in real form: the coefficients of m and -m are complex
// conjugates, the odd ones vanish except m = +-1, whose sine terms cancel in
// the fold and vanish at the poles, and e^{-i L theta_t} = cos(L theta_t), so
//   w_r + fold = c_t [2 + sum_{even 2 <= m < L} 4 cos(m theta_t) / (1 - m^2)
//                + (L even) 2 cos(L theta_t) / (1 - L^2)],
// c_t = 2 inside and 1 at the poles.
std::vector<double> weights_poles(int nlat) {
    const int L = nlat - 1;
    std::vector<double> q((size_t)nlat);
    for (int t = 0; t <= L; ++t) {
        const double th = kPi * t / L;
        double acc = 2.0;
        for (int m = 2; m < L; m += 2) acc += 4.0 * std::cos(m * th) / (1.0 - (double)m * m);
        if (L % 2 == 0) acc += 2.0 * std::cos(L * th) / (1.0 - (double)L * L);
        const double ct = (t == 0 || t == L) ? 1.0 : 2.0;
        q[(size_t)t] = 2.0 * kPi / (4.0 * (double)L * L) * ct * acc;
    }
    return q;
}

// Quadrature weight per ring (a pixel's weight is its ring's).  Fejer's first
// rule in cos(theta) on the cell-centred colatitudes, times 2 pi / nlon, is
// exact for band-limited signals on this grid (the sampling-theorem
// quadrature the paper adopts, Sec. 3.2 and App. A); cell areas are offered as
// the alternative.  The pole-including grid takes App. A's own weights.
std::vector<double> ring_weights(int nlat, int nlon, int kind, int sampling) {
    if (poles(sampling)) return weights_poles(nlat);
    std::vector<double> q(nlat);
    const double dphi = 2.0 * kPi / nlon;
    for (int t = 0; t < nlat; ++t) {
        const double th = colat(t, nlat, sampling);
        double w;
        if (kind == DISCO_QUAD_CELL_AREA) {
            const double half = 0.5 * kPi / nlat;
            w = std::cos(th - half) - std::cos(th + half);
        } else {
            double acc = 0.0;
            for (int m = 1; 2 * m <= nlat; ++m)
                acc += std::cos(2.0 * m * th) / ((2.0 * m - 1.0) * (2.0 * m + 1.0));
            w = 2.0 / nlat * (1.0 - 2.0 * acc);
        }
        q[t] = w * dphi;
    }
    return q;
}

double hat(double s) {
    const double a = std::fabs(s);
    return a < 1.0 ? 1.0 - a : 0.0;
}

}  // namespace

int make_op_geom(const PlanParams& p, bool transpose, OpGeom* g, std::string* err) {
    OpGeom o{};
    o.centre_at_input = transpose;
    if (!transpose) {
        o.nlat_o = p.nlat_out; o.nlon_o = p.nlon_out;
        o.nlat_i = p.nlat_in;  o.nlon_i = p.nlon_in;
    } else {
        o.nlat_o = p.nlat_in;  o.nlon_o = p.nlon_in;
        o.nlat_i = p.nlat_out; o.nlon_i = p.nlon_out;
    }
    if (o.nlon_i % o.nlon_o == 0) {
        o.P = 1;
        o.stride = o.nlon_i / o.nlon_o;
    } else if (o.nlon_o % o.nlon_i == 0) {
        o.P = o.nlon_o / o.nlon_i;
        o.stride = 1;
    } else {
        if (err) *err = "longitude counts must divide one another (nlon_in=" +
                        std::to_string(p.nlon_in) + ", nlon_out=" + std::to_string(p.nlon_out) + ")";
        return DISCO_ERR_UNSUPPORTED;
    }
    o.nq = o.nlon_o / o.P;
    *g = o;
    return DISCO_OK;
}

int build_host_op(const PlanParams& p, bool transpose, HostOp* op, std::string* err, bool quad_at_output) {
    OpGeom g;
    int rc = make_op_geom(p, transpose, &g, err);
    if (rc) return rc;
    op->g = g;
    op->basis = p.basis;
    const bool axisym = p.basis == DISCO_BASIS_AXISYMMETRIC_4;
    const bool separable = p.basis == DISCO_BASIS_SEPARABLE_4X4;
    // Quadrature of the op's input grid: the forward op sums over plan
    // in-grid points; the transposed op over plan out-grid points, its centres.
    const std::vector<double> q = ring_weights(g.nlat_i, g.nlon_i, p.quadrature, p.sampling);
    // The adjoint ops weight by their output ring instead (App. C).
    const std::vector<double> q_o =
        quad_at_output ? ring_weights(g.nlat_o, g.nlon_o, p.quadrature, p.sampling) : std::vector<double>();
    const double h = p.h;
    // Basis support radius: the 3x3 hats vanish for max(|u|, |v|) >= 2h, the
    // axisymmetric and separable ones for Theta >= 4h.
    const double radius = std::min(p.theta_c, (axisym || separable) ? 4.0 * h : 2.0 * std::sqrt(2.0) * h);
    const int64_t M = (int64_t)g.nlon_i * g.nlon_o;  // longitude residues per 2 pi

    std::vector<double> sin_o(g.nlat_o), cos_o(g.nlat_o), sin_i(g.nlat_i), cos_i(g.nlat_i);
    for (int t = 0; t < g.nlat_o; ++t) ring_trig(t, g.nlat_o, p.sampling, &sin_o[t], &cos_o[t]);
    for (int t = 0; t < g.nlat_i; ++t) ring_trig(t, g.nlat_i, p.sampling, &sin_i[t], &cos_i[t]);

    op->pat_ptr.assign(1, 0);
    op->t_in.clear(); op->d.clear(); op->d_raw.clear(); op->cell.clear(); op->val.clear(); op->val64.clear();
    op->max_window = 0; op->full_ring_windows = 0; op->nnz_pairs = 0;

    for (int to = 0; to < g.nlat_o; ++to) {
        for (int r = 0; r < g.P; ++r) {
            for (int ti = 0; ti < g.nlat_i; ++ti) {
                const double qw = quad_at_output ? q_o[to] : q[ti];
                // Colatitude difference (input - output) from integers.
                const double dth_io = colat_diff(ti, g.nlat_i, to, g.nlat_o, p.sampling);
                if (std::fabs(dth_io) > radius * (1.0 + 1e-12)) continue;
                // Centre ring c and evaluation ring e of the filter.
                double sc, cc, se, ce, dth;  // dth = theta_e - theta_c
                if (!g.centre_at_input) {
                    sc = sin_o[to]; cc = cos_o[to]; se = sin_i[ti]; ce = cos_i[ti]; dth = dth_io;
                } else {
                    sc = sin_i[ti]; cc = cos_i[ti]; se = sin_o[to]; ce = cos_o[to]; dth = -dth_io;
                }
                // Longitude window: distance <= radius  <=>  |dphi| <= dphi_max.
                const double den = sc * se;
                const double cmax = den > 0 ? (std::cos(radius) - cc * ce) / den : -2.0;
                // Residue n = d * nlon_o - r * nlon_i of phi_i - phi_o = 2 pi n / M.
                int64_t d_lo, d_hi;
                bool full = false;
                if (cmax <= -1.0) {
                    full = true;
                } else {
                    const double dphi_max = std::acos(std::min(1.0, cmax));
                    const double nmax = dphi_max * (double)M / (2.0 * kPi);
                    d_lo = (int64_t)std::floor(((double)r * g.nlon_i - nmax) / g.nlon_o) - 1;
                    d_hi = (int64_t)std::ceil(((double)r * g.nlon_i + nmax) / g.nlon_o) + 1;
                    if (d_hi - d_lo + 1 >= g.nlon_i) full = true;
                }
                if (full) {
                    // Exactly one full turn, centred on the output longitude.
                    d_lo = (int64_t)std::ceil(((double)r * g.nlon_i - 0.5 * (double)M) / g.nlon_o);
                    d_hi = d_lo + g.nlon_i - 1;
                }
                int32_t kept = 0;
                for (int64_t dd = d_lo; dd <= d_hi; ++dd) {
                    int64_t n = dd * g.nlon_o - (int64_t)r * g.nlon_i;
                    n %= M;
                    if (n > M / 2) n -= M;
                    if (n < -M / 2) n += M;
                    // phi_e - phi_c: input minus output for the forward op.
                    const double dphi = 2.0 * kPi * (double)n / (double)M * (g.centre_at_input ? -1.0 : 1.0);
                    const double s2 = std::sin(0.5 * dphi);
                    const double xs = std::sin(dth) - 2.0 * se * cc * s2 * s2;
                    const double ys = se * std::sin(dphi);
                    const double zs = std::cos(dth) - 2.0 * se * sc * s2 * s2;
                    const double rho = std::hypot(xs, ys);
                    const double Th = std::atan2(rho, zs);
                    if (Th > p.theta_c) continue;
                    float vals[kBasis];
                    double vals64[kBasis];
                    bool any = false;
                    int nzk = 0;
                    if (axisym) {
                        // psi_k(Theta) = hat(Theta / h - k), k = 0..3 (Sec. 3.4).
                        for (int k = 0; k < kBasis; ++k) {
                            double psi = k < kAxisymBasis ? hat(Th / h - k) : 0.0;
                            if (psi < kPsiFloor) psi = 0.0;
                            vals64[k] = psi * qw;
                            vals[k] = (float)vals64[k];
                            if (psi != 0.0) { any = true; ++nzk; }
                        }
                        if (!any) continue;
                        int64_t dnorm = dd % g.nlon_i;
                        if (dnorm < 0) dnorm += g.nlon_i;
                        op->t_in.push_back(ti);
                        op->d.push_back((int32_t)dnorm);
                        op->d_raw.push_back((int32_t)dd);
                        op->cell.push_back(0);
                        op->val.insert(op->val.end(), vals, vals + kBasis);
                        op->val64.insert(op->val64.end(), vals64, vals64 + kBasis);
                        op->nnz_pairs += (int64_t)nzk * g.nq;
                        ++kept;
                        continue;
                    }
                    if (separable) {
                        // psi_{4a+b} = hat(Theta / h - a) mu_b(Phi), mu_b the
                        // periodic hat of width pi / 2 at node b pi / 2 (Sec. 3.4
                        // with four nodes along theta and phi).  On the cell
                        // (a, b) with a = floor(Theta / h), b the quadrant of Phi,
                        // only a, a + 1 (if <= 3) and b, b + 1 (mod 4) fire;
                        // their four products are stored in that order.
                        double Phi = 0.0;
                        if (Th > 1e-12) {
                            Phi = std::atan2(ys, xs);
                            if (Phi < 0.0) Phi += 2.0 * kPi;
                        }
                        const double sp = Phi / (0.5 * kPi);
                        const int b = std::min(3, std::max(0, (int)std::floor(sp)));
                        const int a = std::min(3, std::max(0, (int)std::floor(Th / h)));
                        const double ta[2] = {hat(Th / h - a), a + 1 <= 3 ? hat(Th / h - (a + 1)) : 0.0};
                        const double pb[2] = {hat(sp - b), hat(sp - (b + 1))};
                        for (int k = 0; k < kBasis; ++k) { vals[k] = 0.0f; vals64[k] = 0.0; }
                        for (int i = 0; i < 2; ++i)
                            for (int j = 0; j < 2; ++j) {
                                double psi = ta[i] * pb[j];
                                if (psi < kPsiFloor) psi = 0.0;
                                vals64[2 * i + j] = psi * qw;
                                vals[2 * i + j] = (float)vals64[2 * i + j];
                                if (psi != 0.0) { any = true; ++nzk; }
                            }
                        if (!any) continue;
                        int64_t dnorm = dd % g.nlon_i;
                        if (dnorm < 0) dnorm += g.nlon_i;
                        op->t_in.push_back(ti);
                        op->d.push_back((int32_t)dnorm);
                        op->d_raw.push_back((int32_t)dd);
                        op->cell.push_back((uint8_t)(4 * a + b));
                        op->val.insert(op->val.end(), vals, vals + kBasis);
                        op->val64.insert(op->val64.end(), vals64, vals64 + kBasis);
                        op->nnz_pairs += (int64_t)nzk * g.nq;
                        ++kept;
                        continue;
                    }
                    double u = 0.0, v = 0.0;
                    if (rho > 0.0) { u = Th * xs / rho; v = Th * ys / rho; }
                    for (int a = 0; a < 3; ++a) {
                        const double ha = hat(u / h - (a - 1));
                        for (int b = 0; b < 3; ++b) {
                            double psi = ha * hat(v / h - (b - 1));
                            // A hat evaluated at its own zero (e.g. a point exactly
                            // two node spacings away) comes out as rounding noise of
                            // the fp64 geometry (~1e-16); such values are exact zeros.
                            if (psi < kPsiFloor) psi = 0.0;
                            vals64[3 * a + b] = psi * qw;
                            vals[3 * a + b] = (float)vals64[3 * a + b];
                            if (psi != 0.0) { any = true; ++nzk; }
                        }
                    }
                    if (!any) continue;
                    int64_t dnorm = dd % g.nlon_i;
                    if (dnorm < 0) dnorm += g.nlon_i;
                    // Hat cell containing (u, v): cell c spans [(c-2) h, (c-1) h);
                    // only the nodes on its corners can be non-zero there.
                    const int cu = std::min(3, std::max(0, (int)std::floor(u / h) + 2));
                    const int cv = std::min(3, std::max(0, (int)std::floor(v / h) + 2));
                    op->t_in.push_back(ti);
                    op->d.push_back((int32_t)dnorm);
                    op->d_raw.push_back((int32_t)dd);
                    op->cell.push_back((uint8_t)(4 * cu + cv));
                    op->val.insert(op->val.end(), vals, vals + kBasis);
                    op->val64.insert(op->val64.end(), vals64, vals64 + kBasis);
                    op->nnz_pairs += (int64_t)nzk * g.nq;
                    ++kept;
                }
                if (kept > 0 && full) ++op->full_ring_windows;
                op->max_window = std::max(op->max_window, kept);
            }
            op->pat_ptr.push_back((int32_t)op->t_in.size());
        }
    }
    return DISCO_OK;
}

Work pattern_work(const HostOp& op, const std::vector<uint8_t>& include) {
    const OpGeom& g = op.g;
    Work w;
    // Output step q reads input longitude (stride * q + d) mod nlon_i, so an
    // entry of offset d touches the nq longitudes congruent to d modulo the
    // stride: distinct input pixels per ring = residues seen * nq.
    std::vector<std::vector<uint8_t>> residues((size_t)g.nlat_i);
    for (int pat = 0; pat < g.n_patterns(); ++pat) {
        if (!include.empty() && !include[(size_t)pat]) continue;
        w.out_pixels += g.nq;
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e) {
            int nz = 0;
            for (int k = 0; k < kBasis; ++k) nz += op.val[(size_t)e * kBasis + k] != 0.0f;
            w.pairs += (int64_t)nz * g.nq;
            std::vector<uint8_t>& r = residues[(size_t)op.t_in[(size_t)e]];
            if (r.empty()) r.assign((size_t)g.stride, 0);
            r[(size_t)(op.d[(size_t)e] % g.stride)] = 1;
        }
    }
    for (const std::vector<uint8_t>& r : residues)
        for (uint8_t v : r) w.in_pixels += v ? g.nq : 0;
    return w;
}

}  // namespace disco
