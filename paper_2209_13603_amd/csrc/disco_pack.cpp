// disco_pack.cpp -- host packing of one op's psi entries for the LDS-staged
// fused kernel (layout described in disco_internal.h).
#include <algorithm>
#include <cstdio>
#include <cstring>

#include "disco.h"
#include "disco_internal.h"

namespace disco {

namespace {

// Nodes of hat cell c (0..3) along one axis: the cell spans [(c-2) h, (c-1) h)
// and only nodes (c-1) and c (inside 0..2) can be non-zero there.
int cell_first(int c) { return c == 0 ? 0 : c - 1; }
int cell_count(int c) { return (c == 0 || c == 3) ? 1 : 2; }

struct Piece {
    int32_t ti, d_first, d_last;
    int32_t e_begin, e_end;  // entries (indices into the op) of this piece
    int32_t n() const { return e_end - e_begin; }
};

}  // namespace

CellMap cell_map(int basis) {
    CellMap m;
    for (int c = 0; c < kCells; ++c)
        for (int j = 0; j < 4; ++j) m.k[c][j] = -1;
    if (basis == DISCO_BASIS_AXISYMMETRIC_4) {
        for (int j = 0; j < kAxisymBasis; ++j) m.k[0][j] = (int8_t)j;
    } else if (basis == DISCO_BASIS_SEPARABLE_4X4) {
        for (int a = 0; a < 4; ++a)
            for (int b = 0; b < 4; ++b)
                for (int i = 0; i < 2; ++i)
                    for (int j = 0; j < 2; ++j)
                        if (a + i <= 3) m.k[4 * a + b][2 * i + j] = (int8_t)(4 * (a + i) + (b + j) % 4);
    } else {
        for (int cu = 0; cu < 4; ++cu)
            for (int cv = 0; cv < 4; ++cv) {
                int n = 0;
                for (int a = cell_first(cu); a < cell_first(cu) + cell_count(cu); ++a)
                    for (int b = cell_first(cv); b < cell_first(cv) + cell_count(cv); ++b)
                        m.k[4 * cu + cv][n++] = (int8_t)(3 * a + b);
            }
    }
    return m;
}

bool entry_cell_values(const HostOp& op, int64_t e, int* cell, float v[4]) {
    const float* v9 = &op.val[(size_t)e * kBasis];
    for (int j = 0; j < 4; ++j) v[j] = 0.0f;
    if (op.basis == DISCO_BASIS_AXISYMMETRIC_4) {
        *cell = 0;
        for (int j = 0; j < kAxisymBasis; ++j) v[j] = v9[j];
        return true;
    }
    *cell = op.cell[(size_t)e];
    if (op.basis == DISCO_BASIS_SEPARABLE_4X4) {
        for (int j = 0; j < 4; ++j) v[j] = v9[j];
        for (int j = 4; j < kBasis; ++j)
            if (v9[j] != 0.0f) return false;
        return true;
    }
    const CellMap m = cell_map(op.basis);
    float rest[kBasis];
    for (int k = 0; k < kBasis; ++k) rest[k] = v9[k];
    for (int j = 0; j < 4; ++j) {
        const int k = m.k[*cell][j];
        if (k >= 0) {
            v[j] = v9[k];
            rest[k] = 0.0f;
        }
    }
    for (int k = 0; k < kBasis; ++k)
        if (rest[k] != 0.0f) return false;
    return true;
}

int pack_op(const HostOp& op, int target_entries, const std::vector<uint8_t>& skip, PackedHost* out,
            std::string* err, int tile) {
    const OpGeom& g = op.g;
    const int s = g.stride;
    if (tile != 64 && tile != 128 && tile != kTileQ) {
        if (err) *err = "internal: unknown tile width";
        return DISCO_ERR_DEVICE;
    }
    const int halo = s * (tile - 1);  // extra columns a tile reads beyond one entry
    if (halo + 1 > kLdsCols) {
        if (err) *err = "longitude stride too large for the staged kernel";
        return DISCO_ERR_UNSUPPORTED;
    }
    const int max_extent = kLdsCols - halo;  // max (d_last - d_first + 1) of one piece
    // Entries of one chunk: the work-item target times the lane groups that
    // share a chunk (tiles narrower than a workgroup), at most kChunkEntries,
    // so that no chunk outweighs the work items by more than that.
    const int chunk_cap = std::max(1, std::min(kChunkEntries, target_entries * (kTileQ / tile)));
    PackedHost P;
    P.tile = tile;
    std::vector<int32_t> pattern_seg_count(g.n_patterns(), 0);

    for (int pat = 0; pat < g.n_patterns(); ++pat) {
        if (!skip.empty() && skip[(size_t)pat]) continue;
        const int32_t e0 = op.pat_ptr[(size_t)pat], e1 = op.pat_ptr[(size_t)pat + 1];
        // 1. Pieces: runs of one input ring with a bounded offset extent.
        std::vector<Piece> pieces;
        for (int32_t e = e0; e < e1; ++e) {
            const int32_t ti = op.t_in[(size_t)e], dr = op.d_raw[(size_t)e];
            if (!pieces.empty() && pieces.back().ti == ti && dr - pieces.back().d_first + 1 <= max_extent &&
                dr > pieces.back().d_last && pieces.back().n() < chunk_cap) {
                pieces.back().d_last = dr;
                pieces.back().e_end = e + 1;
            } else {
                pieces.push_back(Piece{ti, dr, dr, e, e + 1});
            }
        }
        // 2. Chunks: pieces packed greedily under the LDS column and entry budgets.
        std::vector<std::pair<int, int>> chunk_pieces;  // [begin, end) into pieces
        int used = 0, used_e = 0;
        for (int i = 0; i < (int)pieces.size(); ++i) {
            const int len = halo + pieces[(size_t)i].d_last - pieces[(size_t)i].d_first + 1;
            const int ne = pieces[(size_t)i].n();
            if (chunk_pieces.empty() || used + len > kLdsCols || used_e + ne > chunk_cap) {
                chunk_pieces.push_back({i, i + 1});
                used = len;
                used_e = ne;
            } else {
                chunk_pieces.back().second = i + 1;
                used += len;
                used_e += ne;
            }
        }
        // 3. Emit chunks; entries sorted by cell; then segments.
        const int32_t chunk_first = (int32_t)P.chunks.size();
        std::vector<int32_t> chunk_entries;
        for (auto& cp : chunk_pieces) {
            PChunk C{};
            C.span_begin = (int32_t)P.spans.size();
            int lds = 0;
            std::vector<std::pair<int, PEntry>> ents;  // (cell, entry)
            for (int i = cp.first; i < cp.second; ++i) {
                const Piece& pc = pieces[(size_t)i];
                PSpan sp{pc.ti * g.nlon_i, pc.d_first, halo + pc.d_last - pc.d_first + 1, lds};
                for (int32_t e = pc.e_begin; e < pc.e_end; ++e) {
                    PEntry E{};
                    E.off = lds + (op.d_raw[(size_t)e] - pc.d_first);
                    int cell = 0;
                    if (!entry_cell_values(op, e, &cell, E.v)) {
                        if (err) *err = "internal: basis value outside its hat cell";
                        return DISCO_ERR_DEVICE;
                    }
                    ents.push_back({cell, E});
                }
                lds += sp.len;
                P.spans.push_back(sp);
            }
            C.span_end = (int32_t)P.spans.size();
            std::stable_sort(ents.begin(), ents.end(),
                             [](const std::pair<int, PEntry>& a, const std::pair<int, PEntry>& b) {
                                 return a.first < b.first;
                             });
            int32_t base = (int32_t)P.entries.size();
            int k = 0;
            for (int c = 0; c <= kCells; ++c) {
                while (k < (int)ents.size() && ents[(size_t)k].first < c) ++k;
                C.cls[c] = base + k;
            }
            for (auto& pe : ents) P.entries.push_back(pe.second);
            chunk_entries.push_back((int32_t)ents.size());
            P.chunks.push_back(C);
        }
        // Segments: consecutive chunks with at most target_entries entries
        // (a chunk above the target forms a segment on its own).
        const int32_t nch = (int32_t)chunk_pieces.size();
        std::vector<std::pair<int32_t, int32_t>> segs;
        if (nch == 0) {
            segs.push_back({chunk_first, chunk_first});  // empty pattern: writes zeros
        } else {
            int acc = 0;
            for (int32_t c = 0; c < nch; ++c) {
                if (segs.empty() || acc + chunk_entries[(size_t)c] > target_entries) {
                    segs.push_back({chunk_first + c, chunk_first + c + 1});
                    acc = chunk_entries[(size_t)c];
                } else {
                    segs.back().second = chunk_first + c + 1;
                    acc += chunk_entries[(size_t)c];
                }
            }
        }
        if (segs.size() > 1) {
            P.red_pattern.push_back(pat);
            if (P.red_ptr.empty()) P.red_ptr.push_back(0);
        }
        for (auto& sg : segs) {
            int32_t slot = -1;
            if (segs.size() > 1) {
                slot = P.n_slots++;
                P.red_slots.push_back(slot);
            }
            P.segs.push_back(PSeg{pat, sg.first, sg.second, slot});
        }
        if (segs.size() > 1) P.red_ptr.push_back((int32_t)P.red_slots.size());
        pattern_seg_count[(size_t)pat] = (int32_t)segs.size();
    }
    // Work items: runs of consecutive segments with at most target_entries
    // entries in total (and at most 64 segments).
    int acc = 0;
    for (int32_t i = 0; i < (int32_t)P.segs.size(); ++i) {
        const PSeg& sg = P.segs[(size_t)i];
        // Cost model in entry units: entries, staged columns, fixed per-segment work.
        int n = 8;
        for (int32_t c = sg.chunk_begin; c < sg.chunk_end; ++c) {
            const PChunk& C = P.chunks[(size_t)c];
            n += C.cls[kCells] - C.cls[0];
            for (int32_t sp = C.span_begin; sp < C.span_end; ++sp) n += P.spans[(size_t)sp].len / 16;
        }
        if (P.items.empty() || acc + n > target_entries || P.items.back().seg_end - P.items.back().seg_begin >= 64) {
            P.items.push_back(PItem{i, i + 1});
            acc = n;
        } else {
            P.items.back().seg_end = i + 1;
            acc += n;
        }
    }
    *out = std::move(P);
    return DISCO_OK;
}

}  // namespace disco

namespace disco {

int pack_sweep(const HostOp& op, int target_cost, const std::vector<uint8_t>& skip, SweepHost* out,
               std::string* err) {
    (void)err;
    const OpGeom& g = op.g;
    const int s = g.stride;
    const int halo = s * (kSweepTile - 1);
    SweepHost H;
    H.covered.assign((size_t)g.n_patterns(), 0);

    // Per pattern: the input rings it reads with their raw offset ranges.
    struct RingUse { int32_t ti, dmin, dmax; };
    auto ring_uses = [&](int pat) {
        std::vector<RingUse> u;
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e) {
            const int32_t ti = op.t_in[(size_t)e], dr = op.d_raw[(size_t)e];
            if (!u.empty() && u.back().ti == ti) {
                u.back().dmin = std::min(u.back().dmin, dr);
                u.back().dmax = std::max(u.back().dmax, dr);
            } else {
                u.push_back(RingUse{ti, dr, dr});
            }
        }
        return u;
    };
    // A pattern's entries in walk order: each entry goes to its hat cell with
    // the cell's 1, 2 or 4 values, or, when only one of those values is not
    // zero and that basis function's single-value group is still empty, to
    // that group with that value alone; entries without a non-zero value are
    // left out.
    struct GEnt { int grp; int32_t e; float v[4]; };
    auto group_entries = [&](int pat) {
        std::vector<GEnt> out;
        int count[kSweepGroups] = {0};
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e) {
            const int cell = op.cell[(size_t)e];
            const int cu = cell / 4, cv = cell % 4;
            const int fa = cu == 0 ? 0 : cu - 1, na = (cu == 0 || cu == 3) ? 1 : 2;
            const int fb = cv == 0 ? 0 : cv - 1, nb = (cv == 0 || cv == 3) ? 1 : 2;
            const float* v9 = &op.val[(size_t)e * kBasis];
            GEnt G{cell, e, {0.0f, 0.0f, 0.0f, 0.0f}};
            int k = 0, nz = 0, kz = 0;
            for (int a = fa; a < fa + na; ++a)
                for (int b = fb; b < fb + nb; ++b) {
                    G.v[k++] = v9[3 * a + b];
                    if (v9[3 * a + b] != 0.0f) { ++nz; kz = 3 * a + b; }
                }
            if (nz == 0) continue;
            if (nz == 1 && k > 1 && count[16 + kz] == 0) G = GEnt{16 + kz, e, {v9[kz], 0.0f, 0.0f, 0.0f}};
            ++count[G.grp];
            out.push_back(G);
        }
        std::stable_sort(out.begin(), out.end(), [](const GEnt& x, const GEnt& y) {
            return sweep_group_pos(x.grp) < sweep_group_pos(y.grp);
        });
        return out;
    };
    std::vector<int32_t> n_grouped((size_t)g.n_patterns(), -1);
    auto n_entries = [&](int pat) {
        int32_t& n = n_grouped[(size_t)pat];
        if (n < 0) n = (int32_t)group_entries(pat).size();
        return (int)n;
    };
    auto eligible = [&](int pat) {
        if (!skip.empty() && skip[(size_t)pat]) return false;
        const int n = n_entries(pat);
        return n > 0 && n <= kSweepEntries;
    };

    int pat = 0;
    const int np = g.n_patterns();
    while (pat < np) {
        if (!eligible(pat)) { ++pat; continue; }
        // Grow a run [pat, end) while its slots fit in kSweepCols and its cost
        // stays under the target.
        std::vector<std::vector<RingUse>> uses;
        int end = pat, cost = 0;
        for (; end < np && eligible(end); ++end) {
            std::vector<RingUse> u = ring_uses(end);
            uses.push_back(u);
            // Ring ranges over the run so far and live intervals.
            std::vector<int32_t> first(g.nlat_i, -1), last(g.nlat_i, -1), dmin(g.nlat_i, 0), dmax(g.nlat_i, 0);
            for (size_t i = 0; i < uses.size(); ++i)
                for (auto& r : uses[i]) {
                    if (first[(size_t)r.ti] < 0) { first[(size_t)r.ti] = (int)i; dmin[(size_t)r.ti] = r.dmin; dmax[(size_t)r.ti] = r.dmax; }
                    last[(size_t)r.ti] = (int)i;
                    dmin[(size_t)r.ti] = std::min(dmin[(size_t)r.ti], r.dmin);
                    dmax[(size_t)r.ti] = std::max(dmax[(size_t)r.ti], r.dmax);
                }
            int cap = 0, live_max = 0;
            for (int t = 0; t < g.nlat_i; ++t)
                if (first[(size_t)t] >= 0) cap = std::max(cap, halo + dmax[(size_t)t] - dmin[(size_t)t] + 1);
            for (size_t i = 0; i < uses.size(); ++i) {
                int live = 0;
                for (int t = 0; t < g.nlat_i; ++t)
                    if (first[(size_t)t] >= 0 && first[(size_t)t] <= (int)i && last[(size_t)t] >= (int)i) ++live;
                live_max = std::max(live_max, live);
            }
            const int c = n_entries(end) + 24 + (int)u.size() * 2;
            if (end > pat && ((int64_t)live_max * cap > kSweepCols || cost + c > target_cost)) {
                uses.pop_back();
                break;
            }
            if ((int64_t)live_max * cap > kSweepCols) {  // a lone pattern that does not fit
                uses.pop_back();
                break;
            }
            cost += c;
        }
        if (end == pat) { ++pat; continue; }  // not even one pattern fits: left to the general kernel
        // Final slot layout of the run [pat, end).
        const int n = end - pat;
        std::vector<int32_t> first(g.nlat_i, -1), last(g.nlat_i, -1), dmin(g.nlat_i, 0), dmax(g.nlat_i, 0);
        for (int i = 0; i < n; ++i)
            for (auto& r : uses[(size_t)i]) {
                if (first[(size_t)r.ti] < 0) { first[(size_t)r.ti] = i; dmin[(size_t)r.ti] = r.dmin; dmax[(size_t)r.ti] = r.dmax; }
                last[(size_t)r.ti] = i;
                dmin[(size_t)r.ti] = std::min(dmin[(size_t)r.ti], r.dmin);
                dmax[(size_t)r.ti] = std::max(dmax[(size_t)r.ti], r.dmax);
            }
        int cap = 0;
        for (int t = 0; t < g.nlat_i; ++t)
            if (first[(size_t)t] >= 0) cap = std::max(cap, halo + dmax[(size_t)t] - dmin[(size_t)t] + 1);
        std::vector<int32_t> slot(g.nlat_i, -1);
        std::vector<int32_t> slot_ring;  // ring currently in each slot (-1: free)
        SRun R{(int32_t)H.pats.size(), 0};
        for (int i = 0; i < n; ++i) {
            const int p = pat + i;
            // Free slots whose ring is no longer read.
            for (auto& sr : slot_ring)
                if (sr >= 0 && last[(size_t)sr] < i) sr = -1;
            SPat SP{};
            SP.pattern = p;
            SP.act_begin = (int32_t)H.acts.size();
            for (auto& r : uses[(size_t)i]) {
                if (first[(size_t)r.ti] != i) continue;
                int sl = -1;
                for (size_t k = 0; k < slot_ring.size(); ++k)
                    if (slot_ring[k] < 0) { sl = (int)k; break; }
                if (sl < 0) { sl = (int)slot_ring.size(); slot_ring.push_back(-1); }
                slot_ring[(size_t)sl] = r.ti;
                slot[(size_t)r.ti] = sl;
                H.acts.push_back(PSpan{r.ti * g.nlon_i, dmin[(size_t)r.ti], halo + dmax[(size_t)r.ti] - dmin[(size_t)r.ti] + 1, sl * cap});
            }
            const int nact = (int)H.acts.size() - SP.act_begin;
            if (nact > 255) {
                if (err) *err = "internal: more than 255 new spans in one sweep pattern";
                return DISCO_ERR_DEVICE;
            }
            if (nact > 0) SP.first = H.acts[(size_t)SP.act_begin];
            // Entries in walk order.
            const std::vector<GEnt> ents = group_entries(p);
            SP.ent = (int32_t)H.entries.size();
            SP.nact_nent = nact | ((int32_t)ents.size() << 8);
            for (const GEnt& G : ents) {
                const int32_t ti = op.t_in[(size_t)G.e];
                if (G.grp < 16)
                    SP.ncell[G.grp / 4] += 1u << (8 * (G.grp % 4));
                else
                    SP.nact_nent |= 1 << G.grp;  // bit 16 + K
                H.entries.push_back(PEntry{slot[(size_t)ti] * cap + (op.d_raw[(size_t)G.e] - dmin[(size_t)ti]),
                                           {G.v[0], G.v[1], G.v[2], G.v[3]}});
            }
            H.pats.push_back(SP);
            H.covered[(size_t)p] = 1;
        }
        R.pat_end = (int32_t)H.pats.size();
        if ((int64_t)slot_ring.size() * cap > kSweepCols) {
            if (err) *err = "internal: sweep slots exceed the LDS budget";
            return DISCO_ERR_DEVICE;
        }
        H.runs.push_back(R);
        pat = end;
    }
    // Longest runs first: workgroups start roughly in grid order, so the
    // tail of the launch is made of the short runs.
    std::vector<int64_t> cost(H.runs.size(), 0);
    for (size_t r = 0; r < H.runs.size(); ++r)
        for (int32_t p = H.runs[r].pat_begin; p < H.runs[r].pat_end; ++p) {
            const SPat& P = H.pats[(size_t)p];
            cost[r] += spat_nent(P) + 24 + 2 * spat_nact(P);
        }
    std::vector<size_t> order(H.runs.size());
    for (size_t r = 0; r < order.size(); ++r) order[r] = r;
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return cost[a] > cost[b]; });
    std::vector<SRun> sorted;
    for (size_t r : order) sorted.push_back(H.runs[r]);
    H.runs.swap(sorted);
    *out = std::move(H);
    return DISCO_OK;
}

}  // namespace disco

namespace disco {

int pack_stencil(const HostOp& op, int target_entries, int tile, StencilHost* out, std::string* err) {
    const OpGeom& g = op.g;
    if (g.stride != 1) {
        if (err) *err = "the blocked stencil layout needs longitude stride 1";
        return DISCO_ERR_UNSUPPORTED;
    }
    if (tile != kStencilTile && tile != kStencilSmallTile) {
        if (err) *err = "internal: unknown stencil tile";
        return DISCO_ERR_DEVICE;
    }
    const int cols = stencil_cols(tile), max_entries = stencil_entries(tile), max_run = stencil_max_run(tile);
    StencilHost H;
    H.tile = tile;
    struct Run {
        int32_t ti, d_first, d_last;
        std::vector<PVal> v;
        std::vector<uint8_t> c;
    };
    for (int pat = 0; pat < g.n_patterns(); ++pat) {
        const int32_t e0 = op.pat_ptr[(size_t)pat], e1 = op.pat_ptr[(size_t)pat + 1];
        // 1. Runs of consecutive offsets on one input ring (gaps of up to
        //    three offsets filled with zero entries), padded to whole blocks.
        std::vector<Run> runs;
        for (int32_t e = e0; e < e1; ++e) {
            const int32_t ti = op.t_in[(size_t)e], dr = op.d_raw[(size_t)e];
            PVal pv{};
            int cell = 0;
            if (!entry_cell_values(op, e, &cell, pv.v)) {
                if (err) *err = "internal: basis value outside its hat cell";
                return DISCO_ERR_DEVICE;
            }
            if (!runs.empty() && runs.back().ti == ti && dr > runs.back().d_last &&
                dr - runs.back().d_last <= 4 && dr - runs.back().d_first + 1 <= max_run) {
                Run& r = runs.back();
                for (int32_t gap = r.d_last + 1; gap < dr; ++gap) {
                    r.v.push_back(PVal{});
                    r.c.push_back(0);
                }
                r.v.push_back(pv);
                r.c.push_back((uint8_t)cell);
                r.d_last = dr;
            } else {
                runs.push_back(Run{ti, dr, dr, {pv}, {(uint8_t)cell}});
            }
        }
        for (Run& r : runs)
            while (r.v.size() % 4) {
                r.v.push_back(PVal{});
                r.c.push_back(0);
            }
        // 2. Chunks: runs packed greedily under the LDS column and entry budgets.
        const int32_t chunk_first = (int32_t)H.chunks.size();
        std::vector<int32_t> chunk_entries;
        int used = 0, used_e = 0;
        for (size_t i = 0; i < runs.size(); ++i) {
            const int ne = (int)runs[i].v.size();
            const int len = stencil_span(tile, ne / 4);  // staged columns, a multiple of 4
            if (H.chunks.size() == (size_t)chunk_first || used + len > cols || used_e + ne > max_entries) {
                const int32_t pb = (int32_t)H.pieces.size(), eb = (int32_t)H.vals.size();
                H.chunks.push_back(SChunk{pb, pb, eb, eb});
                chunk_entries.push_back(0);
                used = 0;
                used_e = 0;
            }
            SChunk& C = H.chunks.back();
            H.pieces.push_back(SPiece{runs[i].ti * g.nlon_i, runs[i].d_first, used, ne / 4});
            H.vals.insert(H.vals.end(), runs[i].v.begin(), runs[i].v.end());
            H.cells.insert(H.cells.end(), runs[i].c.begin(), runs[i].c.end());
            C.piece_end = (int32_t)H.pieces.size();
            C.ent_end = (int32_t)H.vals.size();
            chunk_entries.back() += ne;
            used += len;
            used_e += ne;
        }
        // 3. Segments of consecutive chunks with at most target_entries entries.
        const int32_t nch = (int32_t)H.chunks.size() - chunk_first;
        std::vector<std::pair<int32_t, int32_t>> segs;
        if (nch == 0) {
            segs.push_back({chunk_first, chunk_first});  // empty pattern: writes zeros
        } else {
            int acc = 0;
            for (int32_t c = 0; c < nch; ++c) {
                if (segs.empty() || acc + chunk_entries[(size_t)c] > target_entries) {
                    segs.push_back({chunk_first + c, chunk_first + c + 1});
                    acc = chunk_entries[(size_t)c];
                } else {
                    segs.back().second = chunk_first + c + 1;
                    acc += chunk_entries[(size_t)c];
                }
            }
        }
        if (segs.size() > 1) {
            H.red_pattern.push_back(pat);
            if (H.red_ptr.empty()) H.red_ptr.push_back(0);
        }
        for (auto& sg : segs) {
            int32_t slot = -1;
            if (segs.size() > 1) {
                slot = H.n_slots++;
                H.red_slots.push_back(slot);
            }
            H.segs.push_back(PSeg{pat, sg.first, sg.second, slot});
        }
        if (segs.size() > 1) H.red_ptr.push_back((int32_t)H.red_slots.size());
    }
    // Work items: runs of consecutive segments with a bounded cost (entries,
    // staged columns, fixed per-segment work) and at most 64 segments.
    int acc = 0;
    for (int32_t i = 0; i < (int32_t)H.segs.size(); ++i) {
        const PSeg& sg = H.segs[(size_t)i];
        int n = 16;
        for (int32_t c = sg.chunk_begin; c < sg.chunk_end; ++c) {
            const SChunk& C = H.chunks[(size_t)c];
            n += C.ent_end - C.ent_begin;
            n += (C.piece_end - C.piece_begin) * tile / 32;
        }
        if (H.items.empty() || acc + n > target_entries || H.items.back().seg_end - H.items.back().seg_begin >= 64) {
            H.items.push_back(PItem{i, i + 1});
            acc = n;
        } else {
            H.items.back().seg_end = i + 1;
            acc += n;
        }
    }
    *out = std::move(H);
    return DISCO_OK;
}

}  // namespace disco

namespace disco {

namespace {

// fp32 -> bf16, round to nearest even (NaN kept quiet).
uint16_t bf16_rne(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// One group: eight consecutive offsets d0 .. d0 + 7 of input ring ti, with the
// values of every phase (zero where a phase has no entry).
struct MGroup {
    int32_t ti, d0;
    float v[2][kBasis][8];
};

}  // namespace

int pack_mfma(const HostOp& op, MfmaHost* out, std::string* err) {
    const OpGeom& g = op.g;
    const int s = g.stride, P = g.P, N = g.nlon_i;
    if (!mfma_supported(g, op.basis)) {
        if (err) *err = "the matrix-core layout needs the 3x3 basis, at most two longitude phases, stride <= 4 "
                        "and nlon_in a multiple of 8";
        return DISCO_ERR_UNSUPPORTED;
    }
    const int halo = s * (kMfmaTile - 1);
    MfmaHost H;
    H.P = P;
    for (int to = 0; to < g.nlat_o; ++to) {
        // 1. Offsets (mod nlon_i) of every input ring, over all phases.
        std::vector<std::vector<int32_t>> ring_d((size_t)g.nlat_i);
        for (int r = 0; r < P; ++r) {
            const int pat = to * P + r;
            for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e)
                ring_d[(size_t)op.t_in[(size_t)e]].push_back(op.d[(size_t)e]);
        }
        // 2. Per input ring, the shortest arc of offsets covering them all,
        // cut into groups of eight; each entry lands in exactly one slot.
        std::vector<MGroup> groups;
        std::vector<int32_t> arc_start((size_t)g.nlat_i, -1), first_group((size_t)g.nlat_i, -1);
        for (int ti = 0; ti < g.nlat_i; ++ti) {
            std::vector<int32_t>& ds = ring_d[(size_t)ti];
            if (ds.empty()) continue;
            std::sort(ds.begin(), ds.end());
            ds.erase(std::unique(ds.begin(), ds.end()), ds.end());
            int32_t a0 = ds[0], gap = N - ds.back() + ds[0];  // gap across the seam
            for (size_t i = 1; i < ds.size(); ++i)
                if (ds[i] - ds[i - 1] > gap) {
                    gap = ds[i] - ds[i - 1];
                    a0 = ds[i];
                }
            const int32_t width = N - gap + 1;
            const int ng = (width + 7) / 8;
            arc_start[(size_t)ti] = a0;
            first_group[(size_t)ti] = (int32_t)groups.size();
            for (int j = 0; j < ng; ++j) {
                MGroup G{};
                G.ti = ti;
                G.d0 = a0 + 8 * j;
                groups.push_back(G);
            }
        }
        for (int r = 0; r < P; ++r) {
            const int pat = to * P + r;
            for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e) {
                const int ti = op.t_in[(size_t)e];
                const int32_t pos = ((op.d[(size_t)e] - arc_start[(size_t)ti]) % N + N) % N;
                MGroup& G = groups[(size_t)(first_group[(size_t)ti] + pos / 8)];
                for (int k = 0; k < kBasis; ++k) G.v[r][k][pos % 8] = op.val[(size_t)e * kBasis + k];
            }
        }
        // 3. Segments: runs of groups under the chunk and staged-element
        // budgets; spans = per input ring, the offsets its groups read.
        struct Seg { size_t g0, g1; };
        std::vector<Seg> segs;
        // Elements staged for groups d0 in [dmin, dmax]: a lane reads elements
        // up to (dmax - dstart) + halo + 6, each holding two inputs.
        auto span_len = [&](int32_t dmin, int32_t dmax) {
            const int32_t dstart = dmin & ~7;
            return (halo + (dmax - dstart) + 7 + 7) & ~7;
        };
        auto seg_elems = [&](size_t g0, size_t g1) {
            int32_t total = 0;
            for (size_t i = g0; i < g1;) {
                size_t j = i;
                while (j < g1 && groups[j].ti == groups[i].ti) ++j;
                total += span_len(groups[i].d0, groups[j - 1].d0);
                i = j;
            }
            return total;
        };
        for (size_t i = 0; i < groups.size(); ++i) {
            if (!segs.empty() && (int)(i - segs.back().g0) < 4 * kMfmaMaxChunks &&
                seg_elems(segs.back().g0, i + 1) <= kMfmaMaxElems) {
                segs.back().g1 = i + 1;
            } else {
                segs.push_back(Seg{i, i + 1});
            }
        }
        if (segs.empty()) segs.push_back(Seg{0, 0});  // no entries: the ring's outputs are zero
        const bool split = segs.size() > 1;
        int32_t slot0 = -1;
        if (split) {
            slot0 = H.n_slots;
            H.n_slots += (int32_t)segs.size() * P;
            for (int r = 0; r < P; ++r) {
                H.red_pattern.push_back(to * P + r);
                for (size_t k = 0; k < segs.size(); ++k) H.red_slots.push_back(slot0 + (int32_t)k * P + r);
                H.red_ptr.push_back((int32_t)H.red_slots.size());
            }
        }
        // 4. Emit spans, chunk headers and the A operands.
        for (size_t si = 0; si < segs.size(); ++si) {
            const Seg& sg = segs[si];
            MSeg M{};
            M.ring = to;
            M.span_begin = (int32_t)H.spans.size();
            M.chunk_begin = (int32_t)H.chunks.size();
            M.slot = split ? slot0 + (int32_t)si * P : -1;
            std::vector<int32_t> grp_elem;
            int32_t lds = 0;
            for (size_t i = sg.g0; i < sg.g1;) {
                size_t j = i;
                while (j < sg.g1 && groups[j].ti == groups[i].ti) ++j;
                const int32_t dstart = groups[i].d0 & ~7;
                const int32_t len = span_len(groups[i].d0, groups[j - 1].d0);
                H.spans.push_back(PSpan{groups[i].ti * N, dstart, len, lds});
                for (size_t k = i; k < j; ++k) grp_elem.push_back(lds + groups[k].d0 - dstart);
                lds += len;
                i = j;
            }
            M.span_end = (int32_t)H.spans.size();
            M.n_elems = lds;
            const size_t ng = sg.g1 - sg.g0;
            const size_t nch = (ng + 3) / 4;
            for (size_t c = 0; c < nch; ++c) {
                MChunkHdr hd{};
                for (int gq = 0; gq < 4; ++gq) {
                    const size_t gi = 4 * c + gq;
                    hd.grp[gq] = gi < ng ? grp_elem[gi] : 0;  // padding group: any staged element, values zero
                }
                H.chunks.push_back(hd);
                for (int r = 0; r < P; ++r)
                    for (int lane = 0; lane < 64; ++lane) {
                        const int row = lane % 16, gq = lane / 16;
                        const size_t gi = 4 * c + gq;
                        for (int u = 0; u < 8; ++u) {
                            const float v = (gi < ng && row < kBasis) ? groups[sg.g0 + gi].v[r][row][u] : 0.0f;
                            H.aop.push_back(bf16_rne(v));
                        }
                    }
            }
            M.chunk_end = (int32_t)H.chunks.size();
            H.segs.push_back(M);
        }
    }
    H.red_ptr.insert(H.red_ptr.begin(), 0);
    // 5. Dispatch order.  Work of an item ~ its chunks plus a fixed share
    // (staging and the contraction); contiguous runs of items cut at equal
    // shares of the total, each run sorted heaviest first.
    const int nqt = (g.nq + kMfmaTile - 1) / kMfmaTile;
    H.n_qtiles = nqt;
    std::vector<int64_t> cost;
    for (const MSeg& S : H.segs)
        for (int t = 0; t < nqt; ++t) cost.push_back(S.chunk_end - S.chunk_begin + 2);
    int64_t total = 0;
    for (int64_t c : cost) total += c;
    std::vector<std::vector<int32_t>> runs(8);
    int64_t acc = 0;
    for (size_t i = 0; i < cost.size(); ++i) {
        const int x = (int)std::min<int64_t>(7, (acc + cost[i] / 2) * 8 / std::max<int64_t>(total, 1));
        runs[(size_t)x].push_back((int32_t)i);
        acc += cost[i];
    }
    size_t longest = 0;
    for (auto& r : runs) {
        std::stable_sort(r.begin(), r.end(), [&](int32_t a, int32_t b) { return cost[(size_t)a] > cost[(size_t)b]; });
        longest = std::max(longest, r.size());
    }
    H.order.assign(8 * longest, -1);
    for (int x = 0; x < 8; ++x)
        for (size_t j = 0; j < runs[(size_t)x].size(); ++j) H.order[8 * j + (size_t)x] = runs[(size_t)x][j];
    *out = std::move(H);
    return DISCO_OK;
}

}  // namespace disco
