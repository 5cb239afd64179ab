// disco_spectral_plan.cpp -- host construction of the spectral data of heavy rings.
//
// For an output ring t_o of an op with one longitude phase and unit stride
// (nlon_in == nlon_out == N), the stored entries (t_i, d, v_k) of one input
// ring form, along longitude, the N-periodic sequences v_k[n] (zero outside
// the window), and the op's sum over that ring is the circular
// cross-correlation  Z_k[q] = sum_n v_k[n] x_{t_i}[(q + n) mod N]  whose DFT is
// Xhat[m] conj(Vhat_k[m]) (Sec. 4.2: the compressed pattern is reused at
// every output longitude by a shift).  This file computes Vhat_k in fp64 with
// its own radix-2 FFT, checks the east-west mirror symmetry that lets 9 floats
// per frequency describe all nine basis functions, and rounds to fp32.
//
// The grids are symmetric about the equator: reflecting both rings of a pair
// (t_o -> nlat_o - 1 - t_o, t_i -> nlat_i - 1 - t_i) flips the sign of the
// local coordinate along the meridian and keeps the one along the parallel and
// the longitude offsets, so the reflected pair's psi rows are this pair's with
// the radial index a of psi_{3a+b} replaced by 2 - a.  A pair whose stored
// entries show exactly that relation to an earlier pair reads that pair's
// table with its rows a = 0 and a = 2 exchanged instead of holding its own.
#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdlib>

#include "disco.h"
#include "disco_internal.h"

namespace disco {

namespace {

using cd = std::complex<double>;

bool is_pow2(int n) { return n > 0 && (n & (n - 1)) == 0; }

// In-place iterative radix-2 DFT, X[m] = sum_n x[n] exp(-2 pi i m n / N);
// w[t] = exp(-2 pi i t / N) for t < N / 2.
void fft(std::vector<cd>& a, const std::vector<cd>& w) {
    const size_t n = a.size();
    for (size_t i = 1, j = 0; i < n; ++i) {
        size_t bit = n >> 1;
        for (; j & bit; bit >>= 1) j ^= bit;
        j ^= bit;
        if (i < j) std::swap(a[i], a[j]);
    }
    for (size_t len = 2; len <= n; len <<= 1) {
        const size_t step = n / len;
        for (size_t i = 0; i < n; i += len)
            for (size_t k = 0; k < len / 2; ++k) {
                const cd u = a[i + k], v = a[i + k + len / 2] * w[k * step];
                a[i + k] = u + v;
                a[i + k + len / 2] = u - v;
            }
    }
}

}  // namespace

int build_spectral(const HostOp& op, int min_entries, SpectralHost* sp, std::vector<uint8_t>* heavy,
                   std::string* err) {
    (void)err;
    const OpGeom& g = op.g;
    heavy->assign((size_t)g.n_patterns(), 0);
    *sp = SpectralHost{};
    const int N = g.nlon_i;
    // N <= 8192: the device FFTs keep two M-point buffers and two short
    // twiddle tables in LDS (about 16 M bytes, 65 KB at M = 4096).
    if (g.P != 1 || g.stride != 1 || g.nlon_o != N || !is_pow2(N) || N < 64 || N > 8192) return DISCO_OK;
    const int M = N / 2;

    std::vector<int32_t> rings;
    for (int to = 0; to < g.nlat_o; ++to)
        if (op.pat_ptr[(size_t)to + 1] - op.pat_ptr[(size_t)to] >= min_entries) rings.push_back(to);
    if (rings.empty()) return DISCO_OK;

    // Mirror symmetry: entry at offset d with values v_{3a+b} must match the
    // entry at -d with v_{3a+2-b}.  If the stored pattern does not have it
    // (it always should), the spectral path is not used for this op.
    std::vector<int32_t> at((size_t)N, -1);
    for (int32_t to : rings) {
        const int32_t e0 = op.pat_ptr[(size_t)to], e1 = op.pat_ptr[(size_t)to + 1];
        double vmax = 0.0;
        for (int32_t e = e0; e < e1; ++e)
            for (int k = 0; k < kBasis; ++k) vmax = std::max(vmax, std::fabs(op.val64[(size_t)e * kBasis + k]));
        int32_t e = e0;
        while (e < e1) {  // one input ring at a time (entries are grouped by ring)
            const int32_t ti = op.t_in[(size_t)e];
            int32_t eend = e;
            while (eend < e1 && op.t_in[(size_t)eend] == ti) ++eend;
            for (int32_t k = e; k < eend; ++k) at[(size_t)op.d[(size_t)k]] = k;
            for (int32_t k = e; k < eend; ++k) {
                const int32_t f = at[(size_t)((N - op.d[(size_t)k]) % N)];
                for (int a = 0; a < 3; ++a)
                    for (int b = 0; b < 3; ++b) {
                        const double v = op.val64[(size_t)k * kBasis + 3 * a + b];
                        const double vm = f < 0 ? 0.0 : op.val64[(size_t)f * kBasis + 3 * a + (2 - b)];
                        if (std::fabs(v - vm) > 1e-12 * vmax) return DISCO_OK;
                    }
            }
            for (int32_t k = e; k < eend; ++k) at[(size_t)op.d[(size_t)k]] = -1;
            e = eend;
        }
    }

    // Input-ring slots and pairs.
    std::vector<int32_t> slot_of(g.nlat_i, -1);
    sp->N = N;
    sp->M = M;
    sp->rings = rings;
    sp->pair_ptr.assign(1, 0);
    for (int32_t to : rings) {
        std::vector<int32_t> tis;
        for (int32_t e = op.pat_ptr[(size_t)to]; e < op.pat_ptr[(size_t)to + 1]; ++e)
            if (tis.empty() || tis.back() != op.t_in[(size_t)e]) tis.push_back(op.t_in[(size_t)e]);
        for (int32_t ti : tis) {
            if (slot_of[(size_t)ti] < 0) {
                slot_of[(size_t)ti] = (int32_t)sp->slot_ring.size();
                sp->slot_ring.push_back(ti);
            }
            sp->pair_slot.push_back(slot_of[(size_t)ti]);
        }
        sp->pair_ptr.push_back((int32_t)sp->pair_slot.size());
        (*heavy)[(size_t)to] = 1;
    }
    // Entry range of every pair, and the table each pair reads: its own, or
    // (bit 31) the equator mirror's with rows a = 0 and a = 2 exchanged.
    struct PairEnt { int32_t to, ti, e0, e1; };
    std::vector<PairEnt> pe;
    for (int32_t to : rings) {
        const int32_t e1 = op.pat_ptr[(size_t)to + 1];
        for (int32_t e = op.pat_ptr[(size_t)to]; e < e1;) {
            const int32_t ti = op.t_in[(size_t)e];
            int32_t eend = e;
            while (eend < e1 && op.t_in[(size_t)eend] == ti) ++eend;
            pe.push_back({to, ti, e, eend});
            e = eend;
        }
    }
    const size_t n_pairs = pe.size();
    std::vector<int32_t> ring_first((size_t)g.nlat_o, -1);  // first pair of each spectral ring
    for (size_t p = n_pairs; p-- > 0;) ring_first[(size_t)pe[p].to] = (int32_t)p;
    sp->pair_tab.assign(n_pairs, -1);
    std::vector<int32_t> owners;  // pair whose entries make each table
    auto mirrors = [&](const PairEnt& p, const PairEnt& q) {
        if (p.e1 - p.e0 != q.e1 - q.e0) return false;
        double vmax = 0.0;
        for (const PairEnt* r : {&p, &q})
            for (int32_t e = r->e0; e < r->e1; ++e)
                for (int k = 0; k < kBasis; ++k) vmax = std::max(vmax, std::fabs(op.val64[(size_t)e * kBasis + k]));
        for (int32_t e = q.e0; e < q.e1; ++e) at[(size_t)op.d[(size_t)e]] = e;
        bool same = true;
        for (int32_t e = p.e0; e < p.e1 && same; ++e) {
            const int32_t f = at[(size_t)op.d[(size_t)e]];
            if (f < 0) { same = false; break; }
            for (int a = 0; a < 3 && same; ++a)
                for (int b = 0; b < 3; ++b)
                    if (std::fabs(op.val64[(size_t)e * kBasis + 3 * a + b] -
                                  op.val64[(size_t)f * kBasis + 3 * (2 - a) + b]) > 1e-12 * vmax) {
                        same = false;
                        break;
                    }
        }
        for (int32_t e = q.e0; e < q.e1; ++e) at[(size_t)op.d[(size_t)e]] = -1;
        return same;
    };
    for (size_t p = 0; p < n_pairs; ++p) {
        const PairEnt& P = pe[p];
        // The mirror pair, if it is an earlier one with a table of its own.
        int32_t mq = -1;
        const int32_t mto = g.nlat_o - 1 - P.to, mti = g.nlat_i - 1 - P.ti;
        for (int32_t q = ring_first[(size_t)mto]; q >= 0 && q < (int32_t)p && pe[(size_t)q].to == mto; ++q)
            if (pe[(size_t)q].ti == mti) mq = q;
        if (mq >= 0 && sp->pair_tab[(size_t)mq] >= 0 && mirrors(P, pe[(size_t)mq])) {
            sp->pair_tab[p] = sp->pair_tab[(size_t)mq] | (int32_t)0x80000000u;
        } else {
            sp->pair_tab[p] = (int32_t)owners.size();
            owners.push_back((int32_t)p);
        }
    }
    // Vhat per table: b = 0 (complex) and b = 1 (real) columns, scaled by 1/N
    // (the inverse transform on the device is unnormalised).
    sp->n_tables = (int32_t)owners.size();
    sp->vs.assign(owners.size() * 9 * (size_t)(M + 1), 0.0f);
    std::vector<cd> buf((size_t)N), wtab((size_t)M);
    for (int t = 0; t < M; ++t) {
        const double ang = -2.0 * 3.14159265358979323846 * (double)t / (double)N;
        wtab[(size_t)t] = cd(std::cos(ang), std::sin(ang));
    }
    for (size_t tb = 0; tb < owners.size(); ++tb) {
        {
            const int32_t e = pe[(size_t)owners[tb]].e0, eend = pe[(size_t)owners[tb]].e1;
            float* dst = &sp->vs[tb * 9 * (size_t)(M + 1)];
            for (int a = 0; a < 3; ++a) {
                // Two real sequences in one complex FFT: v_{3a} + i v_{3a+1}.
                std::fill(buf.begin(), buf.end(), cd(0.0, 0.0));
                for (int32_t k = e; k < eend; ++k) {
                    const int32_t dn = op.d[(size_t)k];
                    buf[(size_t)dn] += cd(op.val64[(size_t)k * kBasis + 3 * a], op.val64[(size_t)k * kBasis + 3 * a + 1]);
                }
                fft(buf, wtab);
                for (int m = 0; m <= M; ++m) {
                    const cd zm = buf[(size_t)m], zc = std::conj(buf[(size_t)((N - m) % N)]);
                    const cd v0 = 0.5 * (zm + zc);                // DFT of v_{3a}
                    const cd v1 = cd(0.0, -0.5) * (zm - zc);      // DFT of v_{3a+1} (real)
                    dst[(size_t)(3 * a + 0) * (M + 1) + m] = (float)(v0.real() / N);
                    dst[(size_t)(3 * a + 1) * (M + 1) + m] = (float)(v0.imag() / N);
                    dst[(size_t)(3 * a + 2) * (M + 1) + m] = (float)(v1.real() / N);
                }
            }
        }
    }
    sp->tw.resize((size_t)N);
    for (int t = 0; t < M; ++t) {
        const double ang = -2.0 * 3.14159265358979323846 * (double)t / (double)N;
        sp->tw[(size_t)2 * t] = (float)std::cos(ang);
        sp->tw[(size_t)2 * t + 1] = (float)std::sin(ang);
    }
    return DISCO_OK;
}

}  // namespace disco
