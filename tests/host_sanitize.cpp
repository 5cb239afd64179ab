// host_sanitize.cpp -- drives every host-side step of a plan (grid and
// quadrature, neighbour search, basis evaluation, the packed, sweep,
// spectral and stencil layouts, the work figures) on the CPU, for a build
// with AddressSanitizer and UndefinedBehaviorSanitizer.  No device call is
// made: the layouts are built exactly as plan creation builds them before
// uploading.  Exits non-zero on the first step that fails; a sanitizer
// finding aborts the process.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "disco.h"
#include "disco_internal.h"

using namespace disco;

namespace {

int failures = 0;

void check(int rc, const std::string& what, const std::string& err) {
    if (rc != DISCO_OK) {
        std::printf("FAIL %s: status %d (%s)\n", what.c_str(), rc, err.c_str());
        ++failures;
    }
}

uint16_t bf16_of(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Spectral tables: every pair's frequency-domain psi rows, read as the
// product kernel reads them (its table, rows a = 0 and a = 2 exchanged for an
// equator mirror), equal the DFT of the pair's own entries at a few
// frequencies, evaluated directly in fp64; and when the spectral rings are
// symmetric about the equator, every pair of the southern half reads a
// northern table.
void check_spectral(const HostOp& op, const SpectralHost& sp, const std::string& what) {
    if (sp.rings.empty()) return;
    const int N = sp.N, M = sp.M;
    const double pi = 3.14159265358979323846;
    size_t p = 0;
    int south = 0;
    std::vector<uint8_t> is_heavy((size_t)op.g.nlat_o, 0);
    for (int32_t to : sp.rings) is_heavy[(size_t)to] = 1;
    bool symmetric = true;
    for (int t = 0; t < op.g.nlat_o; ++t) symmetric &= is_heavy[(size_t)t] == is_heavy[(size_t)(op.g.nlat_o - 1 - t)];
    for (int32_t to : sp.rings) {
        const int32_t e1 = op.pat_ptr[(size_t)to + 1];
        for (int32_t e = op.pat_ptr[(size_t)to]; e < e1; ++p) {
            const int32_t ti = op.t_in[(size_t)e];
            int32_t eend = e;
            while (eend < e1 && op.t_in[(size_t)eend] == ti) ++eend;
            if (p >= sp.pair_tab.size()) {
                std::printf("FAIL %s: spectral pair table too short\n", what.c_str());
                ++failures;
                return;
            }
            const int32_t tb = sp.pair_tab[p];
            const int32_t tab = tb & 0x7fffffff, r0 = tb < 0 ? 6 : 0;
            if (tab >= sp.n_tables || (size_t)(tab + 1) * 9 * (M + 1) > sp.vs.size()) {
                std::printf("FAIL %s: pair %zu reads table %d of %d\n", what.c_str(), p, tab, sp.n_tables);
                ++failures;
                return;
            }
            if (to > op.g.nlat_o - 1 - to) south += tb < 0;
            double scale = 0.0;
            for (int32_t k = e; k < eend; ++k)
                for (int kk = 0; kk < kBasis; ++kk) scale += std::fabs(op.val64[(size_t)k * kBasis + kk]);
            scale /= N;
            for (int m : {0, 1, M / 3, M}) {
                for (int a = 0; a < 3; ++a) {
                    double re0 = 0, im0 = 0, re1 = 0;
                    for (int32_t k = e; k < eend; ++k) {
                        const double ang = -2.0 * pi * (double)m * op.d[(size_t)k] / N;
                        re0 += op.val64[(size_t)k * kBasis + 3 * a] * std::cos(ang);
                        im0 += op.val64[(size_t)k * kBasis + 3 * a] * std::sin(ang);
                        re1 += op.val64[(size_t)k * kBasis + 3 * a + 1] * std::cos(ang);
                    }
                    const int row = a == 0 ? r0 : a == 2 ? 6 - r0 : 3;
                    const float* v = &sp.vs[(size_t)tab * 9 * (M + 1)];
                    const double got[3] = {v[(size_t)(row + 0) * (M + 1) + m], v[(size_t)(row + 1) * (M + 1) + m],
                                           v[(size_t)(row + 2) * (M + 1) + m]};
                    const double want[3] = {re0 / N, im0 / N, re1 / N};
                    for (int j = 0; j < 3; ++j)
                        if (std::fabs(got[j] - want[j]) > 1e-6 * scale + 1e-30) {
                            std::printf("FAIL %s: pair %zu (rings %d, %d) row %d freq %d: table %.9g, DFT %.9g\n",
                                        what.c_str(), p, to, ti, 3 * a + j, m, got[j], want[j]);
                            ++failures;
                            return;
                        }
                }
            }
            e = eend;
        }
    }
    if (p != sp.pair_tab.size()) {
        std::printf("FAIL %s: %zu pairs, table of %zu\n", what.c_str(), p, sp.pair_tab.size());
        ++failures;
    }
    int south_pairs = 0;
    for (size_t r = 0; r < sp.rings.size(); ++r)
        if (sp.rings[r] > op.g.nlat_o - 1 - sp.rings[r]) south_pairs += sp.pair_ptr[r + 1] - sp.pair_ptr[r];
    if (symmetric && south != south_pairs) {
        std::printf("FAIL %s: %d of %d southern spectral pairs share a northern table\n", what.c_str(), south,
                    south_pairs);
        ++failures;
    }
}

// The matrix-core layout holds every entry's nine values (rounded to bf16)
// exactly once, at its (output ring, phase, input ring, offset), and nothing
// else; every staged element a lane reads lies inside its segment.
// The sweep layout holds every non-zero value of the patterns it covers
// exactly once, at the input column and basis function of the op's entry:
// entries are mapped back through the spans resident in the run's LDS slots
// and decoded by their group (hat cell or single-value group); no entry is
// without a non-zero value.
void check_sweep(const HostOp& op, const SweepHost& sw, const std::string& what) {
    const OpGeom& g = op.g;
    std::map<std::tuple<int, int, int, int>, float> want, got;
    for (int pat = 0; pat < g.n_patterns(); ++pat) {
        if (!sw.covered[(size_t)pat]) continue;
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e)
            for (int k = 0; k < kBasis; ++k) {
                const float v = op.val[(size_t)e * kBasis + k];
                if (v != 0.0f) want[{pat, op.t_in[(size_t)e], op.d_raw[(size_t)e], k}] = v;
            }
    }
    auto fail = [&](const char* m) {
        std::printf("FAIL %s: sweep layout: %s\n", what.c_str(), m);
        ++failures;
    };
    for (const SRun& R : sw.runs) {
        std::map<int, PSpan> resident;  // by lds_base
        for (int32_t pi = R.pat_begin; pi < R.pat_end; ++pi) {
            const SPat& P = sw.pats[(size_t)pi];
            for (int a = P.act_begin; a < P.act_begin + spat_nact(P); ++a) resident[sw.acts[(size_t)a].lds_base] = sw.acts[(size_t)a];
            int e = P.ent, n_groups = 0;
            for (int pos = 0; pos < kSweepGroups; ++pos) {
                int grp = -1;
                for (int q = 0; q < kSweepGroups; ++q)
                    if (sweep_group_pos(q) == pos) grp = q;
                const int n = grp < 16 ? (int)((P.ncell[grp / 4] >> (8 * (grp % 4))) & 255u) : spat_single(P, grp - 16);
                const int a0 = grp < 16 ? (grp / 4 == 0 ? 0 : grp / 4 - 1) : (grp - 16) / 3;
                const int na = grp < 16 ? ((grp / 4 == 0 || grp / 4 == 3) ? 1 : 2) : 1;
                const int b0 = grp < 16 ? (grp % 4 == 0 ? 0 : grp % 4 - 1) : (grp - 16) % 3;
                const int nb = grp < 16 ? ((grp % 4 == 0 || grp % 4 == 3) ? 1 : 2) : 1;
                for (int i = 0; i < n; ++i, ++e) {
                    const PEntry& E = sw.entries[(size_t)e];
                    auto it = resident.upper_bound(E.off);
                    if (it == resident.begin()) return fail("an entry before every slot");
                    --it;
                    const PSpan& S = it->second;
                    if (E.off >= S.lds_base + S.len) return fail("an entry outside its slot's span");
                    const int ti = S.row / g.nlon_i, d_raw = S.dstart + (E.off - S.lds_base);
                    bool any = false;
                    for (int ia = 0; ia < na; ++ia)
                        for (int ib = 0; ib < nb; ++ib) {
                            const float v = E.v[ia * nb + ib];
                            if (v == 0.0f) continue;
                            any = true;
                            auto key = std::make_tuple(P.pattern, ti, d_raw, 3 * (a0 + ia) + b0 + ib);
                            if (got.count(key)) return fail("a value stored twice");
                            got[key] = v;
                        }
                    for (int j = na * nb; j < 4; ++j)
                        if (E.v[j] != 0.0f) return fail("a value past the group's basis functions");
                    if (!any) return fail("an entry without a non-zero value");
                }
                n_groups += n;
            }
            if (n_groups != spat_nent(P)) return fail("group counts do not add up to the pattern's entries");
        }
    }
    if (got != want) fail("values differ from the op's");
}

void check_mfma(const HostOp& op, const std::string& what) {
    MfmaHost M;
    std::string err;
    const int rc = pack_mfma(op, &M, &err);
    if (!mfma_supported(op.g, op.basis)) {
        if (rc != DISCO_ERR_UNSUPPORTED) {
            std::printf("FAIL %s: pack_mfma accepted an uncovered op\n", what.c_str());
            ++failures;
        }
        return;
    }
    check(rc, what + " pack_mfma", err);
    if (rc != DISCO_OK) return;
    const OpGeom& g = op.g;
    const int N = g.nlon_i, P = g.P;
    std::map<std::tuple<int, int, int, int, int>, uint16_t> want, got;
    for (int pat = 0; pat < g.n_patterns(); ++pat)
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e)
            for (int k = 0; k < kBasis; ++k) {
                const uint16_t v = bf16_of(op.val[(size_t)e * kBasis + k]);
                if (v != 0) want[{pat / P, pat % P, op.t_in[(size_t)e], op.d[(size_t)e], k}] = v;
            }
    std::vector<int> ring_segs((size_t)g.nlat_o, 0);
    for (const MSeg& S : M.segs) {
        ring_segs[(size_t)S.ring]++;
        if (S.chunk_end - S.chunk_begin > kMfmaMaxChunks || S.n_elems > kMfmaMaxElems ||
            S.span_end - S.span_begin > 4 * kMfmaMaxChunks) {
            std::printf("FAIL %s: segment over its budgets\n", what.c_str());
            ++failures;
            return;
        }
        for (int c = S.chunk_begin; c < S.chunk_end; ++c)
            for (int gq = 0; gq < 4; ++gq) {
                const int ge = M.chunks[(size_t)c].grp[gq];
                // largest element a lane reads: ge + stride * (tile - 1) + 6
                if (ge < 0 || ge + g.stride * (kMfmaTile - 1) + 6 >= S.n_elems) {
                    std::printf("FAIL %s: group reads outside its segment\n", what.c_str());
                    ++failures;
                    return;
                }
                int sp = S.span_begin;
                while (sp + 1 < S.span_end && M.spans[(size_t)sp + 1].lds_base <= ge) ++sp;
                const PSpan& SP = M.spans[(size_t)sp];
                if (SP.dstart % 8 != 0 || SP.len % 8 != 0 || ge + g.stride * (kMfmaTile - 1) + 6 >= SP.lds_base + SP.len) {
                    std::printf("FAIL %s: span misaligned or too short\n", what.c_str());
                    ++failures;
                    return;
                }
                const int ti = SP.row / N, d0 = ge - SP.lds_base + SP.dstart;
                for (int r = 0; r < P; ++r)
                    for (int k = 0; k < 16; ++k)
                        for (int u = 0; u < 8; ++u) {
                            const size_t idx = (((size_t)c * P + r) * 64 + (size_t)(k + 16 * gq)) * 8 + (size_t)u;
                            const uint16_t v = M.aop[idx];
                            if (v == 0) continue;
                            if (k >= kBasis) {
                                std::printf("FAIL %s: value in a padding row\n", what.c_str());
                                ++failures;
                                return;
                            }
                            auto key = std::make_tuple(S.ring, r, ti, (d0 + u) % N, k);
                            if (got.count(key)) {
                                std::printf("FAIL %s: value stored twice\n", what.c_str());
                                ++failures;
                                return;
                            }
                            got[key] = v;
                        }
            }
    }
    // The dispatch order lists every (segment, longitude tile) exactly once.
    const size_t n_items = M.segs.size() * (size_t)M.n_qtiles;
    std::vector<int> seen(n_items, 0);
    if (M.order.size() % 8 != 0 || M.n_qtiles != (g.nq + kMfmaTile - 1) / kMfmaTile) {
        std::printf("FAIL %s: dispatch order shape\n", what.c_str());
        ++failures;
        return;
    }
    for (int32_t it : M.order)
        if (it >= 0) {
            if ((size_t)it >= n_items || seen[(size_t)it]++) {
                std::printf("FAIL %s: dispatch order repeats or overruns an item\n", what.c_str());
                ++failures;
                return;
            }
        }
    for (int v : seen)
        if (v != 1) {
            std::printf("FAIL %s: dispatch order misses an item\n", what.c_str());
            ++failures;
            return;
        }
    for (int t = 0; t < g.nlat_o; ++t)
        if (ring_segs[(size_t)t] == 0) {
            std::printf("FAIL %s: output ring %d has no segment\n", what.c_str(), t);
            ++failures;
            return;
        }
    if (got != want) {
        std::printf("FAIL %s: matrix-core values differ from the entries (%zu against %zu)\n", what.c_str(),
                    got.size(), want.size());
        ++failures;
    }
}

void run_op(const PlanParams& p, bool transpose, bool quad_at_output, const char* tag) {
    HostOp op;
    std::string err;
    const std::string what = std::string(tag) + (transpose ? " transpose" : " forward") +
                             (quad_at_output ? " adjoint" : "");
    int rc = build_host_op(p, transpose, &op, &err, quad_at_output);
    check(rc, what + " build_host_op", err);
    if (rc != DISCO_OK) return;
    (void)pattern_work(op, {});
    const CellMap cm = cell_map(op.basis);
    (void)cm;
    for (int64_t e = 0; e < (int64_t)op.t_in.size(); ++e) {
        int cell = 0;
        float v[4];
        if (!entry_cell_values(op, e, &cell, v)) {
            std::printf("FAIL %s: entry %lld has a value outside its cell\n", what.c_str(), (long long)e);
            ++failures;
            break;
        }
    }
    for (int tile : {64, 128, kTileQ}) {
        for (int target : {64, 512}) {
            PackedHost P;
            check(pack_op(op, target, {}, &P, &err, tile), what + " pack_op", err);
        }
    }
    if (op.g.stride == 1) {
        for (int tile : {kStencilSmallTile, kStencilTile}) {
            StencilHost S;
            check(pack_stencil(op, 256, tile, &S, &err), what + " pack_stencil", err);
        }
    }
    if (op.basis != DISCO_BASIS_BILINEAR_3X3) return;
    check_mfma(op, what);
    SpectralHost sp;
    std::vector<uint8_t> heavy;
    check(build_spectral(op, 128, &sp, &heavy, &err), what + " build_spectral", err);
    check_spectral(op, sp, what);
    {
        // Most rings of a small grid on the spectral path.
        SpectralHost sp8;
        std::vector<uint8_t> heavy8;
        check(build_spectral(op, 8, &sp8, &heavy8, &err), what + " build_spectral (8)", err);
        check_spectral(op, sp8, what + " (8 entries)");
    }
    std::vector<uint8_t> light(heavy.size());
    for (size_t i = 0; i < heavy.size(); ++i) light[i] = !heavy[i];
    (void)pattern_work(op, heavy);
    (void)pattern_work(op, light);
    PackedHost PL;
    check(pack_op(op, 512, heavy, &PL, &err), what + " pack_op (light)", err);
    SweepHost sw;
    check(pack_sweep(op, 768, heavy, &sw, &err), what + " pack_sweep", err);
    check_sweep(op, sw, what);
    std::vector<uint8_t> rest(sw.covered);
    for (size_t i = 0; i < rest.size() && i < heavy.size(); ++i) rest[i] |= heavy[i];
    PackedHost PR;
    check(pack_op(op, 512, rest, &PR, &err), what + " pack_op (rest)", err);
}

void run_plan(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double tc, int basis, int quad, int sampling,
              double h) {
    PlanParams p{};
    p.nlat_in = nlat_in; p.nlon_in = nlon_in; p.nlat_out = nlat_out; p.nlon_out = nlon_out;
    p.theta_c = tc;
    p.h = h > 0 ? h : (basis == DISCO_BASIS_BILINEAR_3X3 ? tc / 3.0 : tc / 4.0);
    p.quadrature = quad;
    p.basis = basis;
    p.sampling = sampling;
    p.flags = DISCO_PLAN_BACKWARD;
    char tag[160];
    std::snprintf(tag, sizeof(tag), "%dx%d->%dx%d basis %d quad %d sampling %d h %.4g", nlat_in, nlon_in, nlat_out,
                  nlon_out, basis, quad, sampling, p.h);
    for (bool tr : {false, true})
        for (bool adj : {false, true}) run_op(p, tr, adj, tag);
}

// The C ABI's host-side paths: argument validation of plan creation (every
// rejected case returns before any device call), the host-only export of the
// stored entries, and the status strings.  Plan creation with valid
// arguments builds every op on the host and then needs a device; without one
// it must fail cleanly with DISCO_ERR_DEVICE.
void run_abi() {
    const double pi = 3.14159265358979323846;
    disco_plan_t plan = nullptr;
    struct Bad { int a, b, c, d; double tc; int expect; } bad[] = {
        {0, 16, 8, 16, 0.5, DISCO_ERR_INVALID_ARGUMENT}, {8, 1, 8, 16, 0.5, DISCO_ERR_INVALID_ARGUMENT},
        {8, 16, 8, 16, 0.0, DISCO_ERR_INVALID_ARGUMENT}, {8, 16, 8, 16, 4.0, DISCO_ERR_INVALID_ARGUMENT},
        {8, 16, 8, 24, 0.5, DISCO_ERR_UNSUPPORTED}};
    for (auto& c : bad) {
        const disco_status_t s = disco_plan_create(c.a, c.b, c.c, c.d, c.tc, nullptr, &plan);
        if (s != c.expect) {
            std::printf("FAIL plan_create(%d,%d,%d,%d,%g): %d, expected %d\n", c.a, c.b, c.c, c.d, c.tc, (int)s,
                        c.expect);
            ++failures;
        }
        (void)disco_last_error();
    }
    disco_basis_t b{DISCO_BASIS_BILINEAR_3X3, 7, 0.0, 0, 0};
    if (disco_plan_create(8, 16, 8, 16, 0.5, &b, &plan) != DISCO_ERR_UNSUPPORTED) ++failures;
    b = disco_basis_t{DISCO_BASIS_BILINEAR_3X3, 0, -1.0, 0, 0};
    if (disco_plan_create(8, 16, 8, 16, 0.5, &b, &plan) != DISCO_ERR_INVALID_ARGUMENT) ++failures;
    if (disco_plan_create(8, 16, 8, 16, 0.5, nullptr, nullptr) != DISCO_ERR_INVALID_ARGUMENT) ++failures;
    // Valid arguments: host build of all four ops, then no device.
    b = disco_basis_t{DISCO_BASIS_BILINEAR_3X3, 0, 0.0, 0, DISCO_PLAN_BACKWARD};
    const disco_status_t sv = disco_plan_create(32, 64, 16, 32, 3 * pi / 16, &b, &plan);
    if (sv == DISCO_OK) (void)disco_plan_destroy(plan);
    (void)disco_plan_destroy(nullptr);
    // Entry export on several grids and bases, sized then filled.
    const int cases[][4] = {{16, 32, 8, 16}, {8, 16, 16, 32}, {33, 300, 33, 300}};
    for (auto& c : cases)
        for (int basis : {0, 1, 2})
            for (int tr : {0, 1}) {
                disco_basis_t bb{basis, 0, 0.0, 0, 0};
                int64_t n = 0;
                int32_t P = 0, S = 0;
                const double tc = 3 * pi / std::min(c[0], c[2]);
                disco_status_t s = disco_psi_entries(c[0], c[1], c[2], c[3], tc, &bb, tr, 0, nullptr, nullptr, nullptr,
                                                     nullptr, nullptr, &n, &P, &S);
                if (s != DISCO_OK || n <= 0) { ++failures; continue; }
                std::vector<int32_t> r((size_t)n), ph((size_t)n), ri((size_t)n), off((size_t)n);
                std::vector<float> v((size_t)n * 16);
                s = disco_psi_entries(c[0], c[1], c[2], c[3], tc, &bb, tr, n, r.data(), ph.data(), ri.data(), off.data(),
                                      v.data(), &n, &P, &S);
                if (s != DISCO_OK) ++failures;
            }
    for (int s = 0; s <= 7; ++s) (void)disco_status_string((disco_status_t)s);
}

}  // namespace

int main(int argc, char** argv) {
    const bool big = argc > 1 && std::string(argv[1]) == "--big";
    const double pi = 3.14159265358979323846;
    // Cell-centred grids: same grid, downsampling, upsampling, odd sizes,
    // latitude-only change, several tiles with a ragged tail.
    const int cases[][4] = {{8, 16, 8, 16},   {16, 32, 8, 16},  {12, 24, 6, 12},   {8, 16, 16, 32},
                            {32, 64, 32, 64}, {10, 20, 5, 20},  {33, 300, 33, 300}, {128, 256, 64, 128},
                            {64, 128, 64, 128}, {256, 512, 512, 1024}};
    for (auto& c : cases) {
        const double tc = 3 * pi / std::min(c[0], c[2]);
        for (int basis : {0, 1, 2}) run_plan(c[0], c[1], c[2], c[3], tc, basis, 0, 0, 0.0);
        run_plan(c[0], c[1], c[2], c[3], tc, 0, 1, 0, 0.0);
        run_plan(c[0], c[1], c[2], c[3], tc, 0, 0, 0, tc / 2);
    }
    // The pole-including grid (App. A).
    const int poles[][4] = {{9, 16, 9, 16}, {17, 32, 9, 16}, {9, 16, 17, 32}, {41, 80, 41, 80}};
    for (auto& c : poles) {
        const double tc = 3 * pi / (std::min(c[0], c[2]) - 1);
        for (int basis : {0, 1, 2}) run_plan(c[0], c[1], c[2], c[3], tc, basis, 0, 1, 0.0);
    }
    if (big) run_plan(2048, 4096, 2048, 4096, 3 * pi / 2048, 0, 0, 0, 0.0);
    run_abi();
    std::printf("%s (%d failures)\n", failures ? "FAILED" : "OK", failures);
    return failures ? 1 : 0;
}
