// disco_stencil.hip -- the DISCO convolution with W folded into psi per call:
// every call of the axisymmetric and separable bases (Sec. 3.4), and depthwise
// channels (Sec. 4.2) with any basis.
//
// The paper writes the op as one sparse-dense product with
// Psi_ji = psi(R_j^{-1} w_i) (Sec. 4.1 eq. 7), psi the interpolated filter
// itself; with learnable node values p_k, psi = sum_k p_k psi_k, so for each
// (output channel, input channel) pair the stored per-entry basis values fold
// into one weight, c = sum_k W[co, ci, k] psi_k q.  With few channels (App. B
// times one channel; depthwise layers filter each channel alone) that costs
// one FMA per stored entry and output channel instead of a gather per basis
// function and a contraction.
//
// An entry stores the (at most four) basis values of its hat cell; the op's
// cell map names the basis function of each.  Per input channel the kernels
// stage a table T[j][cell][m] = W[co0 + j, ci, map[cell][m]] (0 where the map
// has no function) in LDS, and fold c = sum_m T[j][cell][m] v[m] while an
// entry is staged.
//
// Layout and walk are the packed one of the fused kernel (disco_fused.hip):
// one workgroup = 256 consecutive output longitudes of one pattern (output
// ring, phase) of a work item, for one batch element and a tile of COT output
// channels.  For each input channel and each chunk of the pattern:
//   1. the chunk's spans of input-ring longitudes are copied into LDS
//      (coalesced along longitude, wrapping at the 0 / 2 pi seam, bf16 widened
//      to fp32), and each entry's offset and its COT folded weights;
//   2. lane q reads its input at (stride * q + offset) for every entry and
//      accumulates weight * x into its COT outputs.
// The accumulation order of a lane depends only on the pattern, never on q,
// so whole-pixel longitude shifts commute with the op bitwise.  Patterns cut
// into several segments write partial outputs that k_reduce_partials sums in
// a fixed order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

DISCO_BOUNDS_FLAG

constexpr int kBlock = kTileQ;

__device__ __forceinline__ float load_val(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_val(const uint16_t* p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}
__device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ void store_val(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_val(uint16_t* p, int64_t i, float v) { p[i] = to_bf16(v); }

// Consecutive blocks go to the 8 XCDs in turn; remap so that each XCD walks a
// contiguous range of work items (neighbouring rings share input rings).
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int xcd = bid & 7, local = bid >> 3;
    const int per = nb >> 3, rem = nb & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Fills T[j][cell][m] (64 floats per output channel j of the tile) for input
// channel ci.  dw_c > 0: depthwise, item b takes row b mod dw_c of a [C][K]
// W (Ci = Co = 1).
template <typename T, int COT, int NT>
__device__ __forceinline__ void fill_fold_table(float* wt, const int8_t* __restrict__ cmap,
                                                const T* __restrict__ w, int K, int b, int ci, int co0,
                                                int Ci, int Co, bool w_trans, int dw_c) {
    for (int idx = threadIdx.x; idx < COT * kCells * 4; idx += NT) {
        const int j = idx / (kCells * 4), cm = idx - j * (kCells * 4);
        const int k = cmap[cm];
        const int co = co0 + j;
        float v = 0.0f;
        if (k >= 0 && co < Co) {
            const int64_t base = dw_c > 0 ? (int64_t)(b % dw_c) * K
                                 : w_trans ? ((int64_t)ci * Co + co) * K
                                           : ((int64_t)co * Ci + ci) * K;
            v = load_val(w, base + k);
        }
        wt[idx] = v;
    }
}

// TQ: output longitudes (lanes) per workgroup, the width the op's spans were
// packed for (PackedDev::tile).
template <typename T, int COT, int TQ>
__global__ __launch_bounds__(TQ) void k_stencil(const PItem* __restrict__ items,
                                                    const PSeg* __restrict__ segs,
                                                    const PChunk* __restrict__ chunks,
                                                    const PSpan* __restrict__ spans,
                                                    const int32_t* __restrict__ offs,
                                                    const PVal* __restrict__ vals,
                                                    const int8_t* __restrict__ cmap, OpGeom g,
                                                    const T* __restrict__ x, const T* __restrict__ w,
                                                    T* __restrict__ y, float* __restrict__ partial,
                                                    int Ci, int Co, int K, int n_qtiles, int n_cotiles,
                                                    bool w_trans, int dw_c) {
    __shared__ float xs[kLdsCols];
    __shared__ __align__(16) int eoffs[kChunkEntries];
    __shared__ __align__(16) float ew[kChunkEntries * COT];  // [entry][j]
    __shared__ __align__(16) float wt[COT * kCells * 4];     // [j][cell][m]

    const int tid = threadIdx.x;
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int item = bid / n_qtiles;
    const int qt = bid - item * n_qtiles;
    const int b = blockIdx.y / n_cotiles;
    const int co0 = (blockIdx.y - b * n_cotiles) * COT;
    const int q0 = qt * TQ;
    const int q = q0 + tid;
    const int lane_col = g.stride * tid;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const PItem it = items[item];

    for (int si = it.seg_begin; si < it.seg_end; ++si) {
        const PSeg sg = segs[si];
        float acc[COT];
#pragma unroll
        for (int j = 0; j < COT; ++j) acc[j] = 0.0f;
        for (int ci = 0; ci < Ci; ++ci) {
            // W[co0 + j][ci][.] (forward) or W[ci][co0 + j][.] (transposed op)
            // through the cell map.  The previous readers of the table (the
            // last chunk's staging) are behind that chunk's second barrier;
            // the next chunk's first barrier orders these writes before use.
            fill_fold_table<T, COT, TQ>(wt, cmap, w, K, b, ci, co0, Ci, Co, w_trans, dw_c);
            const T* xc = x + ((int64_t)b * Ci + ci) * n_in;
            for (int ch = sg.chunk_begin; ch < sg.chunk_end; ++ch) {
                const PChunk C = chunks[ch];
                __syncthreads();  // readers of the previous chunk (or channel) are done
                for (int sp = C.span_begin; sp < C.span_end; ++sp) {
                    const PSpan S = spans[sp];
                    int start = (g.stride * q0 + S.dstart) % g.nlon_i;
                    if (start < 0) start += g.nlon_i;
                    for (int j = tid; j < S.len; j += TQ) {
                        int idx = start + j;
                        if (idx >= g.nlon_i) idx = idx % g.nlon_i;
                        DISCO_CHECK(S.lds_base + j >= 0 && S.lds_base + j < kLdsCols);
                        xs[S.lds_base + j] = load_val(xc, (int64_t)S.row + idx);
                    }
                }
                const int ebase = C.cls[0], ne = C.cls[kCells] - C.cls[0];
                for (int i = tid; i < ne; i += TQ) {
                    eoffs[i] = offs[ebase + i];
                    const PVal pv = vals[ebase + i];
                    // Entries are sorted by cell: cls[c] is the first of cell c.
                    int cell = 0;
#pragma unroll
                    for (int c = 1; c < kCells; ++c) cell += ebase + i >= C.cls[c] ? 1 : 0;
#pragma unroll
                    for (int j = 0; j < COT; ++j) {
                        const float4 t = *(const float4*)(wt + (j * kCells + cell) * 4);
                        ew[i * COT + j] = t.x * pv.v[0] + t.y * pv.v[1] + t.z * pv.v[2] + t.w * pv.v[3];
                    }
                }
                __syncthreads();
                int e = 0;
                for (; e + 4 <= ne; e += 4) {
                    const int4 o = *(const int4*)(eoffs + e);
                    DISCO_CHECK(lane_col + o.x >= 0 && lane_col + o.x < kLdsCols && lane_col + o.y >= 0 && lane_col + o.y < kLdsCols &&
                                lane_col + o.z >= 0 && lane_col + o.z < kLdsCols && lane_col + o.w >= 0 && lane_col + o.w < kLdsCols);
                    const float x0 = xs[lane_col + o.x], x1 = xs[lane_col + o.y];
                    const float x2 = xs[lane_col + o.z], x3 = xs[lane_col + o.w];
#pragma unroll
                    for (int j = 0; j < COT; ++j) {
                        acc[j] = fmaf(ew[(e + 0) * COT + j], x0, acc[j]);
                        acc[j] = fmaf(ew[(e + 1) * COT + j], x1, acc[j]);
                        acc[j] = fmaf(ew[(e + 2) * COT + j], x2, acc[j]);
                        acc[j] = fmaf(ew[(e + 3) * COT + j], x3, acc[j]);
                    }
                }
                for (; e < ne; ++e) {
                    DISCO_CHECK(lane_col + eoffs[e] >= 0 && lane_col + eoffs[e] < kLdsCols);
                    const float xv = xs[lane_col + eoffs[e]];
#pragma unroll
                    for (int j = 0; j < COT; ++j) acc[j] = fmaf(ew[e * COT + j], xv, acc[j]);
                }
            }
        }
        if (q < g.nq) {
            const int to = sg.pattern / g.P, r = sg.pattern - (sg.pattern / g.P) * g.P;
            if (sg.slot < 0) {
                const int64_t pix = (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
#pragma unroll
                for (int j = 0; j < COT; ++j)
                    if (co0 + j < Co) store_val(y, ((int64_t)b * Co + co0 + j) * n_out + pix, acc[j]);
            } else {
                const int B = gridDim.y / n_cotiles;
#pragma unroll
                for (int j = 0; j < COT; ++j)
                    if (co0 + j < Co)
                        partial[(((int64_t)sg.slot * B + b) * Co + co0 + j) * g.nq + q] = acc[j];
            }
        }
    }
}

template <typename T, int COT, int TQ>
hipError_t stencil_launch_tq(const ExecArgs& a, const PackedDev& P, float* partial) {
    const OpGeom& g = a.op->g;
    const int n_qtiles = (g.nq + TQ - 1) / TQ;
    const int n_cot = (a.Co + COT - 1) / COT;
    dim3 grid((unsigned)(P.n_items * n_qtiles), (unsigned)(a.B * n_cot));
    const int tk = timing_begin("stencil", a.stream);
    hipLaunchKernelGGL((k_stencil<T, COT, TQ>), grid, dim3(TQ), 0, a.stream, P.items, P.segs, P.chunks,
                       P.spans, P.offs, P.vals, a.op->cmap_dev, g, (const T*)a.x, (const T*)a.w, (T*)a.y,
                       partial, a.Ci, a.Co, basis_size(a.op->basis), n_qtiles, n_cot, a.w_trans, a.dw_c);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

template <typename T, int COT>
hipError_t stencil_launch(const ExecArgs& a, const PackedDev& P, float* partial) {
    if (P.n_items == 0) return hipSuccess;
    hipError_t e = P.tile == 64    ? stencil_launch_tq<T, COT, 64>(a, P, partial)
                   : P.tile == 128 ? stencil_launch_tq<T, COT, 128>(a, P, partial)
                                   : stencil_launch_tq<T, COT, kTileQ>(a, P, partial);
    if (e != hipSuccess) return e;
    return launch_reduce_partials(a, P, partial);
}

template <typename T>
hipError_t stencil_dispatch(const ExecArgs& a, const PackedDev& P, float* partial) {
    if (a.Co == 1) return stencil_launch<T, 1>(a, P, partial);
    if (a.Co <= 4) return stencil_launch<T, 4>(a, P, partial);
    return stencil_launch<T, 8>(a, P, partial);
}

// The blocked form for one output channel and longitude stride 1: lane l of
// a workgroup owns outputs q0 + 4l .. q0 + 4l + 3.  Entry i of a piece
// (offset dstart + i) adds c_i x[q + dstart + i] to output q, so for the
// block of entries 4b .. 4b + 3 the lane's four outputs need inputs
// x[q0 + 4l + dstart + 4b + m], m = 0..6: the aligned float4 V0 (m < 4) and
// V1 (m >= 4) at LDS columns 4l + 4b and 4l + 4b + 4 of the piece's span;
// V1 is the next block's V0.  Per block: one float4 of x and one float4 of
// folded weights (the same for every lane) from LDS for 16 FMAs.  TILE
// output longitudes per workgroup of TILE / 4 lanes; the chunk budgets scale
// with it, so every tile stages 16 columns and 2 entries per lane.
template <typename T, int TILE>
__global__ __launch_bounds__(TILE / 4) void k_stencil_blocked(const PItem* __restrict__ items,
                                                            const PSeg* __restrict__ segs,
                                                            const SChunk* __restrict__ chunks,
                                                            const SPiece* __restrict__ pieces,
                                                            const PVal* __restrict__ vals,
                                                            const uint8_t* __restrict__ cells,
                                                            const int8_t* __restrict__ cmap, OpGeom g,
                                                            const T* __restrict__ x,
                                                            const T* __restrict__ w, T* __restrict__ y,
                                                            float* __restrict__ partial, int Ci, int K,
                                                            int n_qtiles, int dw_c) {
    constexpr int NT = TILE / 4;
    constexpr int kCols = stencil_cols(TILE);
    constexpr int kEntries = stencil_entries(TILE);
    constexpr int kMaxPieces = kCols / TILE;  // every span is >= one tile
    constexpr int kColsPerThread = kCols / NT;
    constexpr int kEntriesPerThread = kEntries / NT;
    __shared__ float4 xs4[kCols / 4];
    __shared__ float4 ew4[kEntries / 4 + 1];
    __shared__ float4 wt4[kCells];  // [cell][m]
    float* xs = (float*)xs4;
    float* ew = (float*)ew4;

    const int tid = threadIdx.x;
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int item = bid / n_qtiles;
    const int qt = bid - item * n_qtiles;
    const int b = blockIdx.y;
    const int q0 = qt * TILE;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const PItem it = items[item];

    for (int si = it.seg_begin; si < it.seg_end; ++si) {
        const PSeg sg = segs[si];
        float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, a3 = 0.0f;
        for (int ci = 0; ci < Ci; ++ci) {
            // One output channel: W[0][ci][.] and the transposed op's
            // W[ci][0][.] are the same row (ordered as k_stencil's table).
            fill_fold_table<T, 1, NT>((float*)wt4, cmap, w, K, b, ci, 0, Ci, 1, false, dw_c);
            const T* xc = x + ((int64_t)b * Ci + ci) * n_in;
            for (int ch = sg.chunk_begin; ch < sg.chunk_end; ++ch) {
                const SChunk C = chunks[ch];
                // The chunk's spans fill LDS columns [0, used) back to back
                // (at most kCols / TILE pieces).  Every thread
                // first issues the loads of all its columns and entries, then
                // stores them, so that a chunk costs one memory latency.
                const int np = C.piece_end - C.piece_begin;
                int pbase[kMaxPieces], prow[kMaxPieces], pstart[kMaxPieces];
                int used = 0;
#pragma unroll
                for (int pp = 0; pp < kMaxPieces; ++pp) {
                    pbase[pp] = kCols;
                    prow[pp] = 0;
                    pstart[pp] = 0;
                    if (pp < np) {
                        const SPiece S = pieces[C.piece_begin + pp];
                        int st = (q0 + S.dstart) % g.nlon_i;
                        if (st < 0) st += g.nlon_i;
                        pbase[pp] = S.lds_base;
                        prow[pp] = S.row;
                        pstart[pp] = st;
                        used = S.lds_base + stencil_span(TILE, S.nblk);
                    }
                }
                float v[kColsPerThread];
#pragma unroll
                for (int u = 0; u < kColsPerThread; ++u) {
                    const int c = tid + u * NT;
                    v[u] = 0.0f;
                    if (c < used) {
                        int base = pbase[0], row = prow[0], st = pstart[0];
#pragma unroll
                        for (int pp = 1; pp < kMaxPieces; ++pp)
                            if (c >= pbase[pp]) { base = pbase[pp]; row = prow[pp]; st = pstart[pp]; }
                        int idx = st + (c - base);
                        while (idx >= g.nlon_i) idx -= g.nlon_i;
                        v[u] = load_val(xc, (int64_t)row + idx);
                    }
                }
                const int ne = C.ent_end - C.ent_begin;
                PVal pv[kEntriesPerThread];
                int pc[kEntriesPerThread];
#pragma unroll
                for (int u = 0; u < kEntriesPerThread; ++u) {
                    const int i = tid + u * NT;
                    pc[u] = 0;
                    if (i < ne) {
                        pv[u] = vals[C.ent_begin + i];
                        pc[u] = cells[C.ent_begin + i];
                    }
                }
                __syncthreads();  // readers of the previous chunk (or channel) are done
#pragma unroll
                for (int u = 0; u < kColsPerThread; ++u) {
                    const int c = tid + u * NT;
                    if (c < used) xs[c] = v[u];
                }
#pragma unroll
                for (int u = 0; u < kEntriesPerThread; ++u) {
                    const int i = tid + u * NT;
                    if (i < ne) {
                        const float4 t = wt4[pc[u]];
                        ew[i] = t.x * pv[u].v[0] + t.y * pv[u].v[1] + t.z * pv[u].v[2] + t.w * pv[u].v[3];
                    }
                }
                __syncthreads();
                int cb = 0;  // the piece's first weight block
                for (int p = C.piece_begin; p < C.piece_end; ++p) {
                    const SPiece S = pieces[p];
                    // lds_base is a multiple of 4, so the lane's blocks are
                    // float4 elements (16-byte aligned, conflict-free rows).
                    // The next block's x and weights are read one block
                    // ahead (the span and the weight table carry one spare
                    // block for the last).
                    const int xb = (S.lds_base >> 2) + tid;
                    DISCO_CHECK(xb >= 0 && xb + S.nblk + 1 < kCols / 4 && cb + S.nblk < kEntries / 4 + 1);
                    float4 V0 = xs4[xb], V1 = xs4[xb + 1];
                    float4 c = ew4[cb];
#pragma unroll 2
                    for (int bb = 0; bb < S.nblk; ++bb) {
                        const float4 V2 = xs4[xb + bb + 2];
                        const float4 cn = ew4[cb + bb + 1];
                        a0 = fmaf(c.x, V0.x, a0); a0 = fmaf(c.y, V0.y, a0); a0 = fmaf(c.z, V0.z, a0); a0 = fmaf(c.w, V0.w, a0);
                        a1 = fmaf(c.x, V0.y, a1); a1 = fmaf(c.y, V0.z, a1); a1 = fmaf(c.z, V0.w, a1); a1 = fmaf(c.w, V1.x, a1);
                        a2 = fmaf(c.x, V0.z, a2); a2 = fmaf(c.y, V0.w, a2); a2 = fmaf(c.z, V1.x, a2); a2 = fmaf(c.w, V1.y, a2);
                        a3 = fmaf(c.x, V0.w, a3); a3 = fmaf(c.y, V1.x, a3); a3 = fmaf(c.z, V1.y, a3); a3 = fmaf(c.w, V1.z, a3);
                        V0 = V1;
                        V1 = V2;
                        c = cn;
                    }
                    cb += S.nblk;
                }
            }
        }
        const int to = sg.pattern / g.P, r = sg.pattern - (sg.pattern / g.P) * g.P;
        const float av[4] = {a0, a1, a2, a3};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int q = q0 + 4 * tid + j;
            if (q >= g.nq) continue;
            if (sg.slot < 0)
                store_val(y, (int64_t)b * n_out + (int64_t)to * g.nlon_o + (int64_t)q * g.P + r, av[j]);
            else
                partial[((int64_t)sg.slot * gridDim.y + b) * g.nq + q] = av[j];
        }
    }
}

template <typename T, int TILE>
hipError_t stencil_blocked_launch(const ExecArgs& a, const StencilDev& S, float* partial) {
    const OpGeom& g = a.op->g;
    if (S.P.n_items == 0) return hipSuccess;
    const int n_qtiles = (g.nq + TILE - 1) / TILE;
    dim3 grid((unsigned)(S.P.n_items * n_qtiles), (unsigned)a.B);
    const int tk = timing_begin("stencil_blocked", a.stream);
    hipLaunchKernelGGL((k_stencil_blocked<T, TILE>), grid, dim3(TILE / 4), 0, a.stream, S.P.items, S.P.segs,
                       S.chunks, S.pieces, S.vals, S.cells, a.op->cmap_dev, g, (const T*)a.x, (const T*)a.w,
                       (T*)a.y, partial, a.Ci, basis_size(a.op->basis), n_qtiles, a.dw_c);
    timing_end(tk, a.stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_reduce_partials(a, S.P, partial);
}

}  // namespace

DISCO_BOUNDS_READER(bounds_flag_stencil)

hipError_t launch_stencil_blocked(const ExecArgs& a, const StencilDev& S, float* partial_ws) {
    if (S.tile == kStencilSmallTile)
        return a.dtype == 1 ? stencil_blocked_launch<uint16_t, kStencilSmallTile>(a, S, partial_ws)
                            : stencil_blocked_launch<float, kStencilSmallTile>(a, S, partial_ws);
    if (S.tile != kStencilTile) return hipErrorInvalidValue;
    return a.dtype == 1 ? stencil_blocked_launch<uint16_t, kStencilTile>(a, S, partial_ws)
                        : stencil_blocked_launch<float, kStencilTile>(a, S, partial_ws);
}

hipError_t launch_stencil(const ExecArgs& a, const PackedDev& P, float* partial_ws) {
    return a.dtype == 1 ? stencil_dispatch<uint16_t>(a, P, partial_ws) : stencil_dispatch<float>(a, P, partial_ws);
}

}  // namespace disco
