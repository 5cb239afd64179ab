// disco_fused.hip -- the LDS-staged sparse gather of Sec. 4.2's compressed
// product (eq. 9) fused with the channel contraction.
//
// One workgroup = 256 lanes = 256 consecutive output longitudes q of one
// pattern (output ring, phase) of a work item, for one batch element and one
// tile of output channels.  For each pass over kCIC input channels and each
// chunk of the pattern:
//   1. the chunk's spans of input-ring longitudes are copied from HBM into LDS
//      as float4 groups of 4 channels (coalesced along longitude, wrapping at
//      the 0 / 2 pi seam once per span, bf16 widened to fp32);
//   2. entries are visited in hat-cell order; an entry's offset and its (at
//      most four) non-zero basis values are wave-uniform, so each lane reads
//      its input with ds_read_b128 at (stride * lane + offset) and does
//      exactly the FMAs of the basis functions that can be non-zero in that
//      cell, into Z[c][k] registers;
//   3. after the pass, Z is contracted with W (staged in LDS) into the output
//      channel accumulators.
// The accumulation order of a lane depends only on the pattern, never on q, so
// whole-pixel longitude shifts commute with the op bitwise, and runs are
// deterministic.  Patterns cut into several segments write partial outputs
// to workspace slots; k_reduce_partials sums them in slot order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

DISCO_BOUNDS_FLAG

constexpr int kBlock = kTileQ;
constexpr int kNCQ = kCIC / 4;  // float4 channel groups per pass
typedef float v4f __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
constexpr int kKK = kCIC * kBasis;  // contraction length of one channel pass (72)
static_assert(kKK % 4 == 0, "bf16 contraction takes four kk per instruction");

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

__host__ __device__ constexpr int cell_first(int c) { return c == 0 ? 0 : c - 1; }
__host__ __device__ constexpr int cell_count(int c) { return (c == 0 || c == 3) ? 1 : 2; }

// Blocks are dispatched round-robin over the 8 XCDs; remap so that each XCD
// walks a contiguous range of work items (neighbouring output rings share
// input rings, which then stay in that XCD's L2).
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int xcd = bid & 7, local = bid >> 3;
    const int per = nb >> 3, rem = nb & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// FMAs of one entry of hat cell CELL: z[c][k] += v_n * x[c] for the cell's
// (at most four) nodes k, all indices compile-time.
template <int CELL>
__device__ __forceinline__ void fma_cell(const float4& v, const float4 (&xv)[kNCQ],
                                         float (&z)[kCIC][kBasis]) {
    constexpr int CU = CELL / 4, CV = CELL % 4;
    constexpr int A0 = cell_first(CU), NA = cell_count(CU);
    constexpr int B0 = cell_first(CV), NB = cell_count(CV);
    const float vn[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int ia = 0; ia < NA; ++ia)
#pragma unroll
        for (int ib = 0; ib < NB; ++ib) {
            const float vv = vn[ia * NB + ib];
            const int k = 3 * (A0 + ia) + (B0 + ib);
#pragma unroll
            for (int g = 0; g < kNCQ; ++g) {
                z[4 * g + 0][k] = fmaf(vv, xv[g].x, z[4 * g + 0][k]);
                z[4 * g + 1][k] = fmaf(vv, xv[g].y, z[4 * g + 1][k]);
                z[4 * g + 2][k] = fmaf(vv, xv[g].z, z[4 * g + 2][k]);
                z[4 * g + 3][k] = fmaf(vv, xv[g].w, z[4 * g + 3][k]);
            }
        }
}

constexpr int kEntryPad = 3;  // padding entries after a chunk's entries (lookahead reads)

// Entries [e, ee) of one cell, with the input and values of the next entry
// already in flight while an entry's FMAs run.  On entry (and on return) x0
// and v0 hold the input and values of entry e and o1 the LDS column offset of
// entry e + 1; entries are taken in pairs so that the two register sets swap
// roles statically instead of being copied.  A lane group's entries are
// contiguous across cells, so the lookahead runs across cell boundaries (and
// into the next group's entries or the kEntryPad padding entries after the
// chunk, which are read but never used).  The scheduling barriers keep the
// next entry's LDS reads above the current entry's FMAs.
template <int CELL>
__device__ __forceinline__ void run_cell(int& e, int ee, float4 (&x0)[kNCQ], float4& v0, int& o1,
                                         const int* __restrict__ eoffs, const float4* __restrict__ evs,
                                         const float4* __restrict__ xs, int lane_col, float (&z)[kCIC][kBasis]) {
    for (; e + 1 < ee; e += 2) {
        float4 x1[kNCQ];
        DISCO_CHECK(lane_col + o1 >= 0 && lane_col + o1 < kLdsCols && e + 3 < kChunkEntries + kEntryPad);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x1[g] = xs[g * kLdsCols + lane_col + o1];
        const float4 v1 = evs[e + 1];
        const int o2 = eoffs[e + 2];
        __builtin_amdgcn_sched_barrier(0);
        fma_cell<CELL>(v0, x0, z);
        __builtin_amdgcn_sched_barrier(0);
        DISCO_CHECK(lane_col + o2 >= 0 && lane_col + o2 < kLdsCols);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x0[g] = xs[g * kLdsCols + lane_col + o2];
        v0 = evs[e + 2];
        o1 = eoffs[e + 3];
        __builtin_amdgcn_sched_barrier(0);
        fma_cell<CELL>(v1, x1, z);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (e < ee) {
        fma_cell<CELL>(v0, x0, z);
        DISCO_CHECK(lane_col + o1 >= 0 && lane_col + o1 < kLdsCols && e + 2 < kChunkEntries + kEntryPad);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x0[g] = xs[g * kLdsCols + lane_col + o1];
        v0 = evs[e + 1];
        o1 = eoffs[e + 2];
        ++e;
    }
}

// TQ: output longitudes per workgroup, the width the op's spans were packed
// for (PackedDev::tile).  A workgroup always has kBlock threads: with TQ <
// kBlock they form kParts = kBlock / TQ groups of TQ lanes over the same
// longitudes, each group gathering an equal share of every chunk's entries
// (in entry order, so within whole cells or parts of one), and the groups'
// contracted outputs are summed in group order at the end of a segment.
template <typename T, int COT, int TQ>
__global__ __launch_bounds__(kBlock) void k_fused(const PItem* __restrict__ items,
                                                  const PSeg* __restrict__ segs,
                                                  const PChunk* __restrict__ chunks,
                                                  const PSpan* __restrict__ spans,
                                                  const int32_t* __restrict__ offs,
                                                  const PVal* __restrict__ vals, OpGeom g,
                                                  const T* __restrict__ x, const T* __restrict__ w,
                                                  T* __restrict__ y, float* __restrict__ partial,
                                                  int Ci, int Co, int n_qtiles, int n_cotiles,
                                                  bool w_trans) {
    __shared__ float4 xs[kNCQ * kLdsCols];
    __shared__ float4 evs[kChunkEntries + kEntryPad];
    __shared__ int eoffs[kChunkEntries + kEntryPad];
    __shared__ float ws[kCIC * kBasis * COT];
    constexpr bool kBf16 = sizeof(T) == 2;

    constexpr int kParts = kBlock / TQ;
    static_assert(kParts * TQ == kBlock && TQ >= 64, "tiles of 64, 128 or 256 longitudes");
    const int tid = threadIdx.x;
    const int lane = tid & (TQ - 1);  // output longitude within the tile
    const int part = tid / TQ;        // share of the entries
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int item = bid / n_qtiles;
    const int qt = bid - item * n_qtiles;
    const int b = blockIdx.y / n_cotiles;
    const int co0 = (blockIdx.y - b * n_cotiles) * COT;
    const int q0 = qt * TQ;
    const int q = q0 + lane;
    const int lane_col = g.stride * lane;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const PItem it = items[item];

    for (int si = it.seg_begin; si < it.seg_end; ++si) {
        const PSeg sg = segs[si];
        v4f yacc[COT / 4];
#pragma unroll
        for (int j = 0; j < COT / 4; ++j) yacc[j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
        for (int ci0 = 0; ci0 < Ci; ci0 += kCIC) {
            float z[kCIC][kBasis];
#pragma unroll
            for (int c = 0; c < kCIC; ++c)
#pragma unroll
                for (int k = 0; k < kBasis; ++k) z[c][k] = 0.0f;
            __syncthreads();  // previous users of ws / xs are done
            for (int i = tid; i < kCIC * kBasis * COT; i += kBlock) {
                // ws[j][c][k]: output channel j of the tile, pass channel c, basis k
                // (bf16 storage: the raw bf16 values, packed two per word).
                const int j = i / (kCIC * kBasis), ck = i % (kCIC * kBasis), c = ck / kBasis, k = ck % kBasis;
                const int co = co0 + j, ci = ci0 + c;
                const bool in = co < Co && ci < Ci;
                const int64_t idx = w_trans ? ((int64_t)ci * Co + co) * kBasis + k : ((int64_t)co * Ci + ci) * kBasis + k;
                if constexpr (kBf16) {
                    ((uint16_t*)ws)[i] = in ? w[idx] : (uint16_t)0;
                } else {
                    ws[i] = in ? load_val(w, idx) : 0.0f;
                }
            }
            for (int ch = sg.chunk_begin; ch < sg.chunk_end; ++ch) {
                const PChunk C = chunks[ch];
                if (ch != sg.chunk_begin) __syncthreads();  // readers of the previous chunk
                for (int sp = C.span_begin; sp < C.span_end; ++sp) {
                    const PSpan S = spans[sp];
                    int start = (g.stride * q0 + S.dstart) % g.nlon_i;
                    if (start < 0) start += g.nlon_i;
                    for (int j = tid; j < S.len; j += kBlock) {
                        int idx = start + j;
                        if (idx >= g.nlon_i) idx = idx % g.nlon_i;
#pragma unroll
                        for (int gq = 0; gq < kNCQ; ++gq) {
                            float4 v;
                            const int c = ci0 + 4 * gq;
                            const T* xp = x + ((int64_t)b * Ci) * n_in + S.row + idx;
                            v.x = c + 0 < Ci ? load_val(xp, (int64_t)(c + 0) * n_in) : 0.0f;
                            v.y = c + 1 < Ci ? load_val(xp, (int64_t)(c + 1) * n_in) : 0.0f;
                            v.z = c + 2 < Ci ? load_val(xp, (int64_t)(c + 2) * n_in) : 0.0f;
                            v.w = c + 3 < Ci ? load_val(xp, (int64_t)(c + 3) * n_in) : 0.0f;
                            DISCO_CHECK(S.lds_base + j >= 0 && S.lds_base + j < kLdsCols);
                            xs[gq * kLdsCols + S.lds_base + j] = v;
                        }
                    }
                }
                {
                    const int ebase = C.cls[0], ne = C.cls[kCells] - C.cls[0];
                    for (int i = tid; i < ne; i += kBlock) {
                        DISCO_CHECK(i < kChunkEntries);
                        eoffs[i] = offs[ebase + i];
                        const PVal pv = vals[ebase + i];
                        evs[i] = make_float4(pv.v[0], pv.v[1], pv.v[2], pv.v[3]);
                    }
                    if (tid < kEntryPad) {
                        eoffs[ne + tid] = 0;
                        evs[ne + tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                    }
                }
                __syncthreads();
                // Waves whose output longitudes all lie past the ring's end
                // stage but do not gather.
                if (q0 + (lane & ~63) >= g.nq) continue;
                const int ne = C.cls[kCells] - C.cls[0];
                const int lo = ne * part / kParts, hi = ne * (part + 1) / kParts;
                auto share = [&](int c) { return C.cls[c] - C.cls[0] < lo ? lo : C.cls[c] - C.cls[0] > hi ? hi : C.cls[c] - C.cls[0]; };
                // Prime: entry lo in (x0, v0), the offset of entry lo + 1 in o1.
                int e = lo;
                float4 x0[kNCQ];
                const int o0 = eoffs[e];
                DISCO_CHECK(lane_col + o0 >= 0 && lane_col + o0 < kLdsCols);
#pragma unroll
                for (int gq = 0; gq < kNCQ; ++gq) x0[gq] = xs[gq * kLdsCols + lane_col + o0];
                float4 v0 = evs[e];
                int o1 = eoffs[e + 1];
                run_cell<0>(e, share(1), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<1>(e, share(2), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<2>(e, share(3), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<3>(e, share(4), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<4>(e, share(5), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<5>(e, share(6), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<6>(e, share(7), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<7>(e, share(8), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<8>(e, share(9), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<9>(e, share(10), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<10>(e, share(11), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<11>(e, share(12), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<12>(e, share(13), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<13>(e, share(14), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<14>(e, share(15), x0, v0, o1, eoffs, evs, xs, lane_col, z);
                run_cell<15>(e, share(16), x0, v0, o1, eoffs, evs, xs, lane_col, z);
            }
            if (sg.chunk_begin == sg.chunk_end) __syncthreads();  // ws visible
            // Contraction of this pass on the matrix cores:
            //   y[co][q] += sum_{c,k} W(co, ci0 + c, k) Z[c][k][q].
            // v_mfma_f32_4x4x1_16b_f32 treats the wave as 16 blocks of 4
            // lanes; block b computes D[i][j] += A[i] B[j] with lane 4b + i
            // supplying A[i] and lane 4b + j supplying B[j].  With A[i] =
            // W(co0 + 4 quad + i, kk) and B[j] = Z[kk] of lane 4b + j's own
            // pixel, lane l ends with y[co0 + 4 quad + r][its pixel] in
            // register r: one instruction per (kk, 4 output channels).
            // With bf16 storage, v_mfma_f32_4x4x4_16b_bf16 takes four kk per
            // instruction (block b: D[i][j] += sum_kk A[i][kk] B[kk][j], lane
            // 4b + i holding A[i][.], lane 4b + j holding B[.][j]); W is
            // exact in bf16 and Z is rounded to bf16 for it (fp32
            // accumulation), an error of the order of the bf16 output's own.
            const int li = tid & 3;
            if constexpr (kBf16) {
                const uint16_t* ws16 = (const uint16_t*)ws;
#pragma unroll
                for (int g4 = 0; g4 < kKK / 4; ++g4) {
                    v4s zb;
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int kk = 4 * g4 + u;
                        zb[u] = (short)to_bf16(z[kk / kBasis][kk % kBasis]);
                    }
#pragma unroll
                    for (int qd = 0; qd < COT / 4; ++qd) {
                        const v4s wa = *(const v4s*)(ws16 + (4 * qd + li) * kKK + 4 * g4);
                        yacc[qd] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(wa, zb, yacc[qd], 0, 0, 0);
                    }
                }
            } else {
#pragma unroll
                for (int qd = 0; qd < COT / 4; ++qd) {
                    const float* wrow = ws + (4 * qd + li) * (kCIC * kBasis);
#pragma unroll
                    for (int c = 0; c < kCIC; ++c)
#pragma unroll
                        for (int k = 0; k < kBasis; ++k)
                            yacc[qd] = __builtin_amdgcn_mfma_f32_4x4x1f32(wrow[c * kBasis + k], z[c][k],
                                                                         yacc[qd], 0, 0, 0);
                }
            }
        }
        if constexpr (kParts > 1) {
            // The groups' outputs, summed in group order through LDS (the
            // staging buffer, free until the next segment's first barrier).
            float* red = (float*)xs;
            static_assert((kParts - 1) * COT * TQ <= kNCQ * kLdsCols * 4, "reduction fits the staging buffer");
            __syncthreads();  // the contraction's reads of ws and the gather's of xs are done
            if (part > 0) {
#pragma unroll
                for (int j = 0; j < COT; ++j) red[((part - 1) * COT + j) * TQ + lane] = yacc[j / 4][j % 4];
            }
            __syncthreads();
            if (part == 0) {
#pragma unroll
                for (int p = 1; p < kParts; ++p)
#pragma unroll
                    for (int j = 0; j < COT; ++j) yacc[j / 4][j % 4] += red[((p - 1) * COT + j) * TQ + lane];
            }
        }
        if (part == 0 && q < g.nq) {
            const int to = sg.pattern / g.P, r = sg.pattern - (sg.pattern / g.P) * g.P;
            if (sg.slot < 0) {
                const int64_t pix = (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
#pragma unroll
                for (int j = 0; j < COT; ++j)
                    if (co0 + j < Co) store_val(y, ((int64_t)b * Co + co0 + j) * n_out + pix, yacc[j / 4][j % 4]);
            } else {
                const int B = gridDim.y / n_cotiles;
#pragma unroll
                for (int j = 0; j < COT; ++j)
                    if (co0 + j < Co)
                        partial[(((int64_t)sg.slot * B + b) * Co + co0 + j) * g.nq + q] = yacc[j / 4][j % 4];
            }
        }
    }
}

// y of split patterns = sum of their partial slots, in slot order.
// grid: (ceil(nq / 256), n_split, B * Co)
template <typename T>
__global__ __launch_bounds__(kBlock) void k_reduce_partials(const int32_t* __restrict__ red_pattern,
                                                            const int32_t* __restrict__ red_ptr,
                                                            const int32_t* __restrict__ red_slots,
                                                            const float* __restrict__ partial,
                                                            OpGeom g, T* __restrict__ y, int B, int Co) {
    const int q = blockIdx.x * kBlock + threadIdx.x;
    const int sp = blockIdx.y;
    const int b = blockIdx.z / Co, co = blockIdx.z - (blockIdx.z / Co) * Co;
    if (q >= g.nq) return;
    const int pat = red_pattern[sp];
    const int to = pat / g.P, r = pat - (pat / g.P) * g.P;
    const int s0 = red_ptr[sp], s1 = red_ptr[sp + 1];
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const int64_t pix = (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
    // Loads of four slots issued together, then added in slot order.
    const float* pq = partial + ((int64_t)b * Co + co) * g.nq + q;
    const int64_t slot_stride = (int64_t)B * Co * g.nq;
    float acc = 0.0f;
    int s = s0;
    for (; s + 4 <= s1; s += 4) {
        float v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = pq[red_slots[s + u] * slot_stride];
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += v[u];
    }
    for (; s < s1; ++s) acc += pq[red_slots[s] * slot_stride];
    store_val(y, ((int64_t)b * Co + co) * n_out + pix, acc);
}

template <typename T, int COT, int TQ>
hipError_t fused_launch_tq(const ExecArgs& a, const PackedDev& P, float* partial) {
    const OpGeom& g = a.op->g;
    const int n_qtiles = (g.nq + TQ - 1) / TQ;
    const int n_cot = (a.Co + COT - 1) / COT;
    dim3 grid((unsigned)(P.n_items * n_qtiles), (unsigned)(a.B * n_cot));
    int tk = timing_begin("fused_gather_contract", a.stream);
    hipLaunchKernelGGL((k_fused<T, COT, TQ>), grid, dim3(kBlock), 0, a.stream, P.items, P.segs, P.chunks,
                       P.spans, P.offs, P.vals, g, (const T*)a.x, (const T*)a.w, (T*)a.y, partial, a.Ci,
                       a.Co, n_qtiles, n_cot, a.w_trans);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

template <typename T, int COT>
hipError_t fused_launch(const ExecArgs& a, const PackedDev& P, float* partial) {
    if (P.n_items == 0) return hipSuccess;
    hipError_t e = P.tile == 64    ? fused_launch_tq<T, COT, 64>(a, P, partial)
                   : P.tile == 128 ? fused_launch_tq<T, COT, 128>(a, P, partial)
                                   : fused_launch_tq<T, COT, kTileQ>(a, P, partial);
    if (e != hipSuccess) return e;
    return launch_reduce_partials(a, P, partial);
}

template <typename T>
hipError_t fused_dispatch(const ExecArgs& a, const PackedDev& P, float* partial) {
    if (a.Co <= 4) return fused_launch<T, 4>(a, P, partial);
    if (a.Co <= 8) return fused_launch<T, 8>(a, P, partial);
    if (a.Co <= 16) return fused_launch<T, 16>(a, P, partial);
    return fused_launch<T, 32>(a, P, partial);
}

}  // namespace

DISCO_BOUNDS_READER(bounds_flag_fused)

hipError_t launch_reduce_partials(const ExecArgs& a, const PackedDev& P, const float* partial) {
    const OpGeom& g = a.op->g;
    if (P.n_items == 0 || P.n_split == 0) return hipSuccess;
    dim3 grid((unsigned)((g.nq + kBlock - 1) / kBlock), (unsigned)P.n_split, (unsigned)(a.B * a.Co));
    const int tk = timing_begin("reduce_partials", a.stream);
    if (a.dtype == 1)
        hipLaunchKernelGGL((k_reduce_partials<uint16_t>), grid, dim3(kBlock), 0, a.stream, P.red_pattern,
                           P.red_ptr, P.red_slots, partial, g, (uint16_t*)a.y, a.B, a.Co);
    else
        hipLaunchKernelGGL((k_reduce_partials<float>), grid, dim3(kBlock), 0, a.stream, P.red_pattern,
                           P.red_ptr, P.red_slots, partial, g, (float*)a.y, a.B, a.Co);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

size_t workspace_bytes_fused(const ExecArgs& a, const PackedDev& P) {
    return sizeof(float) * (size_t)P.n_slots * a.B * a.Co * a.op->g.nq;
}

hipError_t launch_fused(const ExecArgs& a, const PackedDev& P, float* partial_ws) {
    return a.dtype == 1 ? fused_dispatch<uint16_t>(a, P, partial_ws) : fused_dispatch<float>(a, P, partial_ws);
}

}  // namespace disco
