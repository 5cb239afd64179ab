// disco_pack.cpp -- host packing of one op's psi entries for the LDS-staged
// fused kernel (layout described in disco_internal.h).
#include <algorithm>
#include <cstdio>

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

int pack_op(const HostOp& op, int target_entries, const std::vector<uint8_t>& skip, PackedHost* out,
            std::string* err) {
    const OpGeom& g = op.g;
    const int s = g.stride;
    const int halo = s * (kTileQ - 1);  // extra columns a tile reads beyond one entry
    if (halo + 1 > kLdsCols) {
        if (err) *err = "longitude stride too large for the staged kernel";
        return DISCO_ERR_UNSUPPORTED;
    }
    const int max_extent = kLdsCols - halo;  // max (d_last - d_first + 1) of one piece
    PackedHost P;
    std::vector<int32_t> pattern_seg_count(g.n_patterns(), 0);

    for (int pat = 0; pat < g.n_patterns(); ++pat) {
        if (!skip.empty() && skip[(size_t)pat]) continue;
        const int32_t e0 = op.pat_ptr[(size_t)pat], e1 = op.pat_ptr[(size_t)pat + 1];
        // 1. Pieces: runs of one input ring with a bounded offset extent.
        std::vector<Piece> pieces;
        for (int32_t e = e0; e < e1; ++e) {
            const int32_t ti = op.t_in[(size_t)e], dr = op.d_raw[(size_t)e];
            if (!pieces.empty() && pieces.back().ti == ti && dr - pieces.back().d_first + 1 <= max_extent &&
                dr > pieces.back().d_last && pieces.back().n() < kChunkEntries) {
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
            if (chunk_pieces.empty() || used + len > kLdsCols || used_e + ne > kChunkEntries) {
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
                    const int cell = op.cell[(size_t)e];
                    const int cu = cell / 4, cv = cell % 4;
                    PEntry E{};
                    E.off = lds + (op.d_raw[(size_t)e] - pc.d_first);
                    int n = 0;
                    const float* v9 = &op.val[(size_t)e * kBasis];
                    for (int a = 0; a < 3; ++a)
                        for (int b = 0; b < 3; ++b) {
                            const bool in_cell = a >= cell_first(cu) && a < cell_first(cu) + cell_count(cu) &&
                                                 b >= cell_first(cv) && b < cell_first(cv) + cell_count(cv);
                            if (in_cell) {
                                E.v[n++] = v9[3 * a + b];
                            } else if (v9[3 * a + b] != 0.0f) {
                                if (err) *err = "internal: basis value outside its hat cell";
                                return DISCO_ERR_DEVICE;
                            }
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
