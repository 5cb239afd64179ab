// disco_sweep.hip -- the fused gather + contraction walking runs of output
// rings with the input-ring spans kept resident in LDS.
//
// Same arithmetic as disco_fused.hip (Sec. 4.2's compressed product, hat-cell
// sorted entries, MFMA 4x4x1 channel contraction), organised for light rings:
// a workgroup owns kSweepTile consecutive output longitudes of every pattern of one
// run; each input ring the run reads is staged once, into an LDS slot chosen
// at plan time, and stays there while consecutive patterns read it.  Before
// each pattern only the rings it reads first are loaded, so an output ring
// costs one new input-ring span instead of the ~7 its window covers.  All
// input channels are resident (Ci <= kCIC), so a pattern needs one pass.
//
// With ZOUT the same walk writes the gathered sums Z[b, c, k, pixel] (fp32)
// instead of contracting them: the gather half of the gather-then-contract
// schedule, one launch per group of kCIC input channels.
//
// More than kCIC input channels run one contracting launch per group of kCIC
// channels: the first launch stores y, the later ones add their partial sums
// with fp32 atomic adds (no return value, one add per element and launch, so
// the order of the additions is the launch order and the result does not
// vary between runs).  bf16 outputs accumulate in an fp32 workspace that a
// last kernel rounds into y for the patterns the runs cover.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "disco_internal.h"

namespace disco {

namespace {

DISCO_BOUNDS_FLAG

constexpr int kBlock = kSweepTile;
constexpr int kNCQ = kCIC / 4;
constexpr int kPF = (kBlock + 8 + kBlock - 1) / kBlock;  // prefetched span columns per lane
constexpr int kPFE = (kSweepEntries + kBlock - 1) / kBlock;  // prefetched entries per lane
typedef float v4f __attribute__((ext_vector_type(4)));

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
// Raw buffer access (word 3 of the descriptor for gfx9 raw dword access): an
// offset at or past num_records reads 0 and drops a store, which replaces the
// bounds tests of the channel loads and output stores, and the channel
// stride rides in the scalar offset instead of a 64-bit VALU address add.
constexpr int kRawBufferFlags = 0x00020000;
constexpr int kBufferOutOfRange = (int)0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* p, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, kRawBufferFlags);
}
__device__ __forceinline__ float buffer_load_val(const float*, __amdgpu_buffer_rsrc_t r, int off, int soff) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, soff, 0));
}
__device__ __forceinline__ float buffer_load_val(const uint16_t*, __amdgpu_buffer_rsrc_t r, int off, int soff) {
    return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, soff, 0) << 16);
}
__device__ __forceinline__ void buffer_store_val(float*, __amdgpu_buffer_rsrc_t r, int off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, 0);
}
__device__ __forceinline__ void buffer_store_val(uint16_t*, __amdgpu_buffer_rsrc_t r, int off, float v) {
    __builtin_amdgcn_raw_buffer_store_b16(to_bf16(v), r, off, 0, 0);
}
// Output modes of the contracting sweep: store T into y, store fp32 into the
// partial-sum buffer, or add fp32 into it.
enum { kStoreY = 0, kStoreF32 = 1, kAddF32 = 2 };

__host__ __device__ constexpr int cell_first(int c) { return c == 0 ? 0 : c - 1; }
__host__ __device__ constexpr int cell_count(int c) { return (c == 0 || c == 3) ? 1 : 2; }

__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int xcd = bid & 7, local = bid >> 3;
    const int per = nb >> 3, rem = nb & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

constexpr int kEntryPad = 3;  // padding entries after a pattern's entries (lookahead reads)

// Workgroup barrier that orders LDS only: global loads in flight (the next
// pattern's prefetch) and stores stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The entry group at position pos of the walk, and the walk itself: f is
// called with each position in order, as a compile-time constant.
constexpr int sweep_group_at(int pos) {
    for (int g = 0; g < kSweepGroups; ++g)
        if (sweep_group_pos(g) == pos) return g;
    return -1;
}
constexpr bool sweep_walk_is_a_permutation() {
    for (int p = 0; p < kSweepGroups; ++p)
        if (sweep_group_at(p) < 0) return false;
    return true;
}
static_assert(sweep_walk_is_a_permutation(), "every walk position holds one group");
template <int POS, class F>
__device__ __forceinline__ void walk_groups(F& f) {
    if constexpr (POS < kSweepGroups) {
        f(std::integral_constant<int, POS>{});
        walk_groups<POS + 1>(f);
    }
}

// Basis functions touched by entry group G (a hat cell, or a basis
// function's single-value group): rows A0 .. A0 + NA - 1, columns B0 .. B0 +
// NB - 1 of the 3 x 3 grid, the entry's values in row-major order.
constexpr int grp_a0(int G) { return G < 16 ? cell_first(G / 4) : (G - 16) / 3; }
constexpr int grp_na(int G) { return G < 16 ? cell_count(G / 4) : 1; }
constexpr int grp_b0(int G) { return G < 16 ? cell_first(G % 4) : (G - 16) % 3; }
constexpr int grp_nb(int G) { return G < 16 ? cell_count(G % 4) : 1; }

template <int G>
__device__ __forceinline__ void fma_cell(const float4& v, const float4 (&xv)[kNCQ], float (&z)[kCIC][kBasis]) {
    constexpr int A0 = grp_a0(G), NA = grp_na(G), B0 = grp_b0(G), NB = grp_nb(G);
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

// Entries [e, ee) of one group, with the input and values of the next entry
// already in flight while an entry's FMAs run.  On entry (and on return) x0
// and v0 hold the input and values of entry e and o1 the LDS column offset of
// entry e + 1; entries are taken in pairs so that the two register sets swap
// roles statically instead of being copied.  Groups are contiguous in the
// entry array, so the lookahead runs across group boundaries; the array ends
// with kEntryPad padding entries (offset 0, values 0), so the lookahead reads need
// no bounds test.  The scheduling barriers keep the compiler from sinking
// the next entry's LDS reads below the current entry's FMAs (which it does to
// save registers, leaving the read latency exposed).
template <int G>
__device__ __forceinline__ void entry_one(int e, float4 (&x0)[kNCQ], float4& v0, int& o1,
                                          const int* __restrict__ eoffs, const float4* __restrict__ evs,
                                          const float4* __restrict__ xs, int lane_col, float (&z)[kCIC][kBasis]) {
    fma_cell<G>(v0, x0, z);
    DISCO_CHECK(lane_col + o1 >= 0 && lane_col + o1 < kSweepCols && e + 2 < kSweepEntries + kEntryPad);
#pragma unroll
    for (int g = 0; g < kNCQ; ++g) x0[g] = xs[g * kSweepCols + lane_col + o1];
    v0 = evs[e + 1];
    o1 = eoffs[e + 2];
}

template <int G>
__device__ __forceinline__ void run_cell(int& e, int ee, float4 (&x0)[kNCQ], float4& v0, int& o1,
                                         const int* __restrict__ eoffs, const float4* __restrict__ evs,
                                         const float4* __restrict__ xs, int lane_col, float (&z)[kCIC][kBasis]) {
    for (; e + 1 < ee; e += 2) {
        float4 x1[kNCQ];
        DISCO_CHECK(lane_col + o1 >= 0 && lane_col + o1 < kSweepCols && e + 3 < kSweepEntries + kEntryPad);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x1[g] = xs[g * kSweepCols + lane_col + o1];
        const float4 v1 = evs[e + 1];
        const int o2 = eoffs[e + 2];
        __builtin_amdgcn_sched_barrier(0);
        fma_cell<G>(v0, x0, z);
        __builtin_amdgcn_sched_barrier(0);
        DISCO_CHECK(lane_col + o2 >= 0 && lane_col + o2 < kSweepCols);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x0[g] = xs[g * kSweepCols + lane_col + o2];
        v0 = evs[e + 2];
        o1 = eoffs[e + 3];
        __builtin_amdgcn_sched_barrier(0);
        fma_cell<G>(v1, x1, z);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (e < ee) {
        entry_one<G>(e, x0, v0, o1, eoffs, evs, xs, lane_col, z);
        ++e;
    }
}

constexpr int kKK = kCIC * kBasis;    // contraction length of one pass (72)
constexpr int kWG = (kKK + 15) / 16;  // W registers per 4 output channels

// y[co][pixel] += sum_ci W(co, ci, K) Z[ci][K][pixel] for one basis function
// K: one v_mfma_f32_4x4x1_16b_f32 per (ci, 4 output channels); A is
// broadcast from block kk % 16 (CBSZ = 4, ABID = kk % 16, kk = 9 ci + K) of
// register wv[qd][kk / 16].  Called as soon as the gather has finished every
// cell that touches K, so the matrix cores work while the VALU gathers the
// remaining cells and the registers of Z[.][K] are free again.
// Z[.][K] of the lane's pixel for the kCIC channels of this launch: channels
// 4 h .. 4 h + 3 go through buffer zr[h] (9 planes per channel, plane bytes
// zplane), channel c at scalar offset (9 (c % 4) + K) zplane.
template <int K>
__device__ __forceinline__ void store_z_k(const __amdgpu_buffer_rsrc_t (&zr)[kNCQ], int off, int zplane,
                                          const float (&z)[kCIC][kBasis]) {
#pragma unroll
    for (int c = 0; c < kCIC; ++c)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(z[c][K]), zr[c / 4], off, (kBasis * (c % 4) + K) * zplane,
                                              0);
}

template <int K, int CI, int NQ>
__device__ __forceinline__ void mfma_contract_k(v4f (&yacc)[NQ], const float (&wv)[NQ][kWG],
                                                const float (&z)[kCIC][kBasis]) {
    if constexpr (CI < kCIC) {
        constexpr int KK = CI * kBasis + K;
#pragma unroll
        for (int qd = 0; qd < NQ; ++qd)
            yacc[qd] = __builtin_amdgcn_mfma_f32_4x4x1f32(wv[qd][KK / 16], z[CI][K], yacc[qd], 4, KK % 16, 0);
        mfma_contract_k<K, CI + 1, NQ>(yacc, wv, z);
    }
}

// bf16 storage: the same contraction on the bf16 matrix cores
// (v_mfma_f32_4x4x4_16b_bf16, four products per instruction, fp32
// accumulation), with the gathered sums rounded to bf16 (round to nearest
// even, v_cvt_pk_bf16_f32) like the general kernel does for bf16 storage.
// The contraction index is kk' = 8 K + ci here, so that one basis function's
// eight channels are two groups of four: group G = 2 K + (ci / 4) takes A
// from block G % 16 (CBSZ = 4) of wb[qd][G / 16], where lane 4 b + i holds
// W(co0 + 4 qd + i, kk' = 4 (16 h + b) + u) for u = 0..3 in register h.
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __bf16 bf4 __attribute__((ext_vector_type(4)));

template <int G, int NQ>
__device__ __forceinline__ void mfma_bf16_group(v4f (&yacc)[NQ], const v4s (&wb)[NQ][2], v4s zb) {
#pragma unroll
    for (int qd = 0; qd < NQ; ++qd)
        yacc[qd] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(wb[qd][G / 16], zb, yacc[qd], 4, G % 16, 0);
}

template <int K, int NQ>
__device__ __forceinline__ void mfma_contract_k_bf16(v4f (&yacc)[NQ], const v4s (&wb)[NQ][2],
                                                     const float (&z)[kCIC][kBasis]) {
    static_assert(kCIC == 8, "two groups of four channels per basis function");
    const v4f lo = {z[0][K], z[1][K], z[2][K], z[3][K]};
    const v4f hi = {z[4][K], z[5][K], z[6][K], z[7][K]};
    mfma_bf16_group<2 * K, NQ>(yacc, wb, __builtin_bit_cast(v4s, __builtin_convertvector(lo, bf4)));
    mfma_bf16_group<2 * K + 1, NQ>(yacc, wb, __builtin_bit_cast(v4s, __builtin_convertvector(hi, bf4)));
}

// grid: (n_runs * n_qtiles, B * n_cotiles); the launch reads input channels
// cg0 .. cg0 + kCIC - 1 (those below Ci; cg0 is 0 with YMODE kStoreY) and
// writes y by YMODE (y32: the fp32 [B][Co][pixels] partial sums of kStoreF32
// and kAddF32).  With ZOUT
// the second grid dimension runs over (batch item, group of kCIC input
// channels) instead (n_cotiles = number of channel groups) and z receives
// Z[b, c, k, pixel] for the group's channels; w and y are not used.
// Up to 8 output channels per launch the registers are held to 128 VGPRs, so
// that the four workgroups the LDS admits per CU are all resident.
template <typename T, int COT, bool ZOUT, int YMODE>
__global__ __launch_bounds__(kBlock, COT <= 8 ? 4 : 1) void k_sweep(const SRun* __restrict__ runs, const SPat* __restrict__ pats,
                                                  const PSpan* __restrict__ acts, const int32_t* __restrict__ offs,
                                                  const PVal* __restrict__ vals, OpGeom g,
                                                  const T* __restrict__ x, const T* __restrict__ w,
                                                  T* __restrict__ y, float* __restrict__ zout, int Ci, int Co,
                                                  int n_qtiles, int n_cotiles, bool w_trans, int cg0,
                                                  float* __restrict__ y32) {
    __shared__ float4 xs[kNCQ * kSweepCols];
    __shared__ float4 evs[kSweepEntries + kEntryPad];
    __shared__ int eoffs[kSweepEntries + kEntryPad];

    const int tid = threadIdx.x;
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    // Work item = (longitude tile, run), runs fastest: the workgroups in
    // flight on one XCD cover consecutive runs of the same tile, which share
    // the input rings at their boundaries in that XCD's L2.
    const int n_runs = gridDim.x / n_qtiles;
    const int qt = bid / n_runs;
    const int run = bid - qt * n_runs;
    const int b = blockIdx.y / n_cotiles;
    const int co0 = (blockIdx.y - b * n_cotiles) * COT;          // output channel tile
    const int c0 = ZOUT ? (blockIdx.y - b * n_cotiles) * kCIC : (YMODE == kStoreY ? 0 : cg0);  // input channel group
    const int q0 = qt * kBlock;
    const int q = q0 + tid;
    const int lane_col = g.stride * tid;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    // The input channels c0 .. c0 + kCIC - 1 of batch item b as one buffer of
    // channel planes: channel c0 + c of a column is read at scalar offset
    // c * plane, and channels past Ci read 0 (the host keeps kCIC * n_in *
    // sizeof(T) below 2^31).
    const int plane = (int)(n_in * (int64_t)sizeof(T));
    const int nch = Ci - c0 < kCIC ? Ci - c0 : kCIC;
    const __amdgpu_buffer_rsrc_t xr = buffer_of(x + ((int64_t)b * Ci + c0) * n_in, nch * plane);
    const int out_plane = (int)(n_out * (int64_t)sizeof(T));  // bytes of one output channel plane
    // Z output (ZOUT): channels c0 + 4 h .. c0 + 4 h + 3 as buffer zr[h]; a
    // buffer ends after its last existing channel (the host keeps 36 planes
    // below 2^31 bytes).
    const int zplane = (int)(n_out * (int64_t)sizeof(float));
    __amdgpu_buffer_rsrc_t zr[kNCQ];
    if constexpr (ZOUT) {
#pragma unroll
        for (int h = 0; h < kNCQ; ++h) {
            const int nv = nch - 4 * h < 0 ? 0 : (nch - 4 * h < 4 ? nch - 4 * h : 4);
            zr[h] = buffer_of(zout + ((int64_t)b * Ci + c0 + 4 * h) * kBasis * n_out, nv * kBasis * zplane);
        }
    }
    const SRun R = runs[run];

    // W in registers for the MFMA contraction: with CBSZ = 4 the A operand of
    // v_mfma_f32_4x4x1_16b_f32 is taken from block ABID and broadcast to all
    // 16 blocks, so wv[qd][g] at lane 4b + i holds W(co0 + 4 qd + i, kk =
    // 16 g + b) and one register serves 16 values of kk.
    constexpr bool kMM16 = sizeof(T) == 2 && !ZOUT;  // bf16 matrix-core contraction
    float wv[kMM16 ? 1 : COT / 4][kMM16 ? 1 : kWG];
    v4s wb[kMM16 ? COT / 4 : 1][2];
    if constexpr (kMM16) {
        const int li = tid & 3, blk = (tid & 63) >> 2;
#pragma unroll
        for (int qd = 0; qd < COT / 4; ++qd)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                v4s r;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int kk = 4 * (16 * h + blk) + u, co = co0 + 4 * qd + li;
                    const int c = c0 + kk % kCIC, k = kk / kCIC;
                    short v = 0;
                    if (kk < kKK && co < Co && c < Ci) {
                        const int64_t idx = w_trans ? ((int64_t)c * Co + co) * kBasis + k : ((int64_t)co * Ci + c) * kBasis + k;
                        v = (short)((const uint16_t*)w)[idx];
                    }
                    r[u] = v;
                }
                wb[qd][h] = r;
            }
    } else if constexpr (!ZOUT) {
        const int li = tid & 3, blk = (tid & 63) >> 2;
#pragma unroll
        for (int qd = 0; qd < COT / 4; ++qd)
#pragma unroll
            for (int gg = 0; gg < kWG; ++gg) {
                const int kk = 16 * gg + blk, co = co0 + 4 * qd + li;
                const int c = c0 + kk / kBasis, k = kk % kBasis;
                float v = 0.0f;
                if (kk < kKK && co < Co && c < Ci) {
                    const int64_t idx = w_trans ? ((int64_t)c * Co + co) * kBasis + k : ((int64_t)co * Ci + c) * kBasis + k;
                    v = load_val(w, idx);
                }
                wv[qd][gg] = v;
            }
    }
    // Let the W loads land before the pattern loop (s_waitcnt vmcnt(0)):
    // otherwise the compiler waits for them inside the loop, before every
    // contraction, and that wait also drains the next pattern's prefetch.
    __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));

    // Staging of pattern pi's new spans and entries.  Columns j = tid + 256 i
    // for i < kPF of the first span of the next pattern, and its entries, are
    // loaded into registers while the current pattern computes; anything
    // beyond that (the first pattern of a run, or a second new span) is
    // loaded directly.
    float4 pf[kPF][kNCQ];
    int pf_off[kPFE];
    float4 pf_val[kPFE];
    auto load_col = [&](const PSpan& S, int start, int j, float4 (&v)[kNCQ]) {
        int idx = start + j;
        if (idx >= g.nlon_i) idx = idx % g.nlon_i;
        const int off = (S.row + idx) * (int)sizeof(T);
#pragma unroll
        for (int gq = 0; gq < kNCQ; ++gq) {
            const int c = 4 * gq;
            v[gq].x = buffer_load_val(x, xr, off, (c + 0) * plane);
            v[gq].y = buffer_load_val(x, xr, off, (c + 1) * plane);
            v[gq].z = buffer_load_val(x, xr, off, (c + 2) * plane);
            v[gq].w = buffer_load_val(x, xr, off, (c + 3) * plane);
        }
    };
    auto span_start = [&](const PSpan& S) {
        int start = (g.stride * q0 + S.dstart) % g.nlon_i;
        return start < 0 ? start + g.nlon_i : start;
    };
    auto prefetch = [&](const SPat& P) {
        if (spat_nact(P) > 0) {
            const PSpan S = P.first;
            const int start = span_start(S);
#pragma unroll
            for (int i = 0; i < kPF; ++i) {
                const int j = tid + i * kBlock;
                if (j < S.len) load_col(S, start, j, pf[i]);
            }
        }
        const int ne = spat_nent(P);
#pragma unroll
        for (int i = 0; i < kPFE; ++i) {
            const int k = tid + i * kBlock;
            if (k < ne) {
                pf_off[i] = offs[P.ent + k];
                const PVal pv = vals[P.ent + k];
                pf_val[i] = make_float4(pv.v[0], pv.v[1], pv.v[2], pv.v[3]);
            }
        }
    };
    // Pattern descriptors are read one pattern ahead (SPn), and each carries
    // its first new span inline, so the scalar loads on the way from one
    // pattern to the next are a single request issued before the previous
    // pattern's last contraction rather than a chain of dependent ones.
    SPat SP = pats[R.pat_begin];
    SPat SPn = pats[R.pat_begin + 1 < R.pat_end ? R.pat_begin + 1 : R.pat_begin];
    bool have_pf = false;
    for (int pi = R.pat_begin; pi < R.pat_end; ++pi) {
        lds_barrier();  // the previous pattern's reads of LDS are done
        const int ne = spat_nent(SP);
        const int act_end = SP.act_begin + spat_nact(SP);
        int ai0 = SP.act_begin;
        if (have_pf) {
            // The prefetched columns of the first new span and the entries go
            // in first, in straight-line code, so that their wait counts only
            // the loads before the stores of the previous pattern.  (A pattern
            // may read no new ring: the other phases of an output ring.)
            if (act_end > SP.act_begin) {
                const PSpan S = SP.first;
#pragma unroll
                for (int i = 0; i < kPF; ++i) {
                    const int j = tid + i * kBlock;
                    if (j < S.len) {
                        DISCO_CHECK(S.lds_base + j >= 0 && S.lds_base + j < kSweepCols);
#pragma unroll
                        for (int gq = 0; gq < kNCQ; ++gq) xs[gq * kSweepCols + S.lds_base + j] = pf[i][gq];
                    }
                }
                // Columns of the first span past the prefetch, if any.
                const int start = span_start(S);
                for (int j = kPF * kBlock + tid; j < S.len; j += kBlock) {
                    float4 v[kNCQ];
                    load_col(S, start, j, v);
                    DISCO_CHECK(S.lds_base + j >= 0 && S.lds_base + j < kSweepCols);
#pragma unroll
                    for (int gq = 0; gq < kNCQ; ++gq) xs[gq * kSweepCols + S.lds_base + j] = v[gq];
                }
                ai0 = SP.act_begin + 1;
            }
#pragma unroll
            for (int i = 0; i < kPFE; ++i) {
                const int k = tid + i * kBlock;
                if (k < ne) {
                    DISCO_CHECK(k < kSweepEntries);
                    eoffs[k] = pf_off[i];
                    evs[k] = pf_val[i];
                }
            }
        }
        // Spans and entries the prefetch did not cover are loaded directly.
        for (int ai = ai0; ai < act_end; ++ai) {
            const PSpan S = acts[ai];
            const int start = span_start(S);
            for (int j = tid; j < S.len; j += kBlock) {
                float4 v[kNCQ];
                load_col(S, start, j, v);
                DISCO_CHECK(S.lds_base + j >= 0 && S.lds_base + j < kSweepCols);
#pragma unroll
                for (int gq = 0; gq < kNCQ; ++gq) xs[gq * kSweepCols + S.lds_base + j] = v[gq];
            }
        }
        for (int k = (have_pf ? kPFE * kBlock : 0) + tid; k < ne; k += kBlock) {
            DISCO_CHECK(k < kSweepEntries);
            eoffs[k] = offs[SP.ent + k];
            const PVal pv = vals[SP.ent + k];
            evs[k] = make_float4(pv.v[0], pv.v[1], pv.v[2], pv.v[3]);
        }
        if (tid < kEntryPad) {
            eoffs[ne + tid] = 0;
            evs[ne + tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        lds_barrier();
        have_pf = pi + 1 < R.pat_end;
        if (have_pf) prefetch(SPn);
        float z[kCIC][kBasis];
#pragma unroll
        for (int c = 0; c < kCIC; ++c)
#pragma unroll
            for (int k = 0; k < kBasis; ++k) z[c][k] = 0.0f;
        // Prime: entry 0 in (x0, v0), the offset of entry 1 in o1 (padding
        // entries when the pattern has fewer).
        float4 x0[kNCQ];
        const int o0 = eoffs[0];
        DISCO_CHECK(lane_col + o0 >= 0 && lane_col + o0 < kSweepCols);
#pragma unroll
        for (int g = 0; g < kNCQ; ++g) x0[g] = xs[g * kSweepCols + lane_col + o0];
        float4 v0 = evs[0];
        int o1 = eoffs[1];
        int e = 0;
        int zoff = 0;
        if constexpr (ZOUT) {
            const int pt = SP.pattern, tz = pt / g.P, pz = pt - tz * g.P;
            zoff = q < g.nq ? (tz * g.nlon_o + q * g.P + pz) * (int)sizeof(float) : kBufferOutOfRange;
        }
        // Contraction on the matrix cores: lane l ends with y[co0 + 4 quad +
        // r][its pixel] in register r of yacc[quad].
        v4f yacc[COT / 4];
#pragma unroll
        for (int j = 0; j < COT / 4; ++j) yacc[j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
        // The entry groups in walk order; after basis function K's
        // single-value group its sums are complete and are contracted (or
        // stored) right there.  The next pattern's descriptor is requested
        // before the last contraction.
        const int pattern = SP.pattern;
        auto step = [&](auto pos_c) {
            constexpr int grp = sweep_group_at(decltype(pos_c)::value);
            if constexpr (grp < 16) {
                run_cell<grp>(e, e + (int)((SP.ncell[grp / 4] >> (8 * (grp % 4))) & 255u), x0, v0, o1, eoffs, evs, xs,
                              lane_col, z);
            } else {
                constexpr int K = grp - 16;
                if (spat_single(SP, K)) {
                    entry_one<grp>(e, x0, v0, o1, eoffs, evs, xs, lane_col, z);
                    ++e;
                }
                if constexpr (K == kBasis - 1) {
                    SP = SPn;
                    SPn = pats[pi + 2 < R.pat_end ? pi + 2 : pi];
                }
                if constexpr (ZOUT) store_z_k<K>(zr, zoff, zplane, z);
                else if constexpr (kMM16) mfma_contract_k_bf16<K, COT / 4>(yacc, wb, z);
                else mfma_contract_k<K, 0, COT / 4>(yacc, wv, z);
            }
        };
        walk_groups<0>(step);
        // Every lane issues the same COT stores (outputs that do not exist are
        // dropped by the buffer range check: an out-of-range offset for
        // longitudes past the ring, an empty buffer for channels past Cout),
        // so the number of memory operations after the prefetch is fixed and
        // its wait does not cover the stores.
        if constexpr (ZOUT) continue;
        const int to = pattern / g.P, r = pattern - (pattern / g.P) * g.P;
        const int pix = to * g.nlon_o + q * g.P + r;
        if constexpr (YMODE == kStoreY) {
            const int pix_off = q < g.nq ? pix * (int)sizeof(T) : kBufferOutOfRange;
#pragma unroll
            for (int j = 0; j < COT; ++j) {
                const __amdgpu_buffer_rsrc_t yr =
                    buffer_of(y + ((int64_t)b * Co + co0 + j) * n_out, co0 + j < Co ? out_plane : 0);
                buffer_store_val(y, yr, pix_off, yacc[j / 4][j % 4]);
            }
        } else {
            const int off32 = q < g.nq ? pix * (int)sizeof(float) : kBufferOutOfRange;
            const int plane32 = (int)(n_out * (int64_t)sizeof(float));
#pragma unroll
            for (int j = 0; j < COT; ++j) {
                const __amdgpu_buffer_rsrc_t yr =
                    buffer_of(y32 + ((int64_t)b * Co + co0 + j) * n_out, co0 + j < Co ? plane32 : 0);
                if constexpr (YMODE == kAddF32)
                    (void)__builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(yacc[j / 4][j % 4], yr, off32, 0, 0);
                else
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(yacc[j / 4][j % 4]), yr, off32, 0, 0);
            }
        }
    }
}

// y32[b][co][pixel] rounded to bf16 into y for the covered patterns.
// grid: (ceil(nq / 256), n_cov, B * Co).
__global__ __launch_bounds__(kBlock) void k_convert_y(const int32_t* __restrict__ pats, const float* __restrict__ y32,
                                                     uint16_t* __restrict__ y, OpGeom g) {
    const int q = blockIdx.x * kBlock + threadIdx.x;
    if (q >= g.nq) return;
    const int pattern = pats[blockIdx.y];
    const int to = pattern / g.P, r = pattern - to * g.P;
    const int64_t i = (int64_t)blockIdx.z * g.nlat_o * g.nlon_o + (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
    y[i] = to_bf16(y32[i]);
}

template <typename T, int COT>
hipError_t sweep_launch(const ExecArgs& a, float* y32) {
    const OpGeom& g = a.op->g;
    const SweepDev& S = a.op->sweep;
    if (S.n_runs == 0) return hipSuccess;
    const int n_qtiles = (g.nq + kBlock - 1) / kBlock;
    const int n_cot = (a.Co + COT - 1) / COT;
    const int n_grp = (a.Ci + kCIC - 1) / kCIC;
    // fp32 outputs accumulate in y itself; bf16 ones in y32.
    const bool f32 = a.dtype != 1;
    float* acc = f32 ? (float*)a.y : y32;
    if (n_grp > 1 && !acc) return hipErrorInvalidValue;
    dim3 grid((unsigned)(S.n_runs * n_qtiles), (unsigned)(a.B * n_cot));
    for (int grp = 0; grp < n_grp; ++grp) {
        const int ymode = grp > 0 ? kAddF32 : (n_grp > 1 && !f32 ? kStoreF32 : kStoreY);
        const int tk = timing_begin("sweep_gather_contract", a.stream);
        if (ymode == kStoreY)
            hipLaunchKernelGGL((k_sweep<T, COT, false, kStoreY>), grid, dim3(kBlock), 0, a.stream, S.runs, S.pats,
                               S.acts, S.offs, S.vals, g, (const T*)a.x, (const T*)a.w, (T*)a.y, (float*)nullptr, a.Ci,
                               a.Co, n_qtiles, n_cot, a.w_trans, 0, (float*)nullptr);
        else if (ymode == kStoreF32)
            hipLaunchKernelGGL((k_sweep<T, COT, false, kStoreF32>), grid, dim3(kBlock), 0, a.stream, S.runs, S.pats,
                               S.acts, S.offs, S.vals, g, (const T*)a.x, (const T*)a.w, (T*)a.y, (float*)nullptr, a.Ci,
                               a.Co, n_qtiles, n_cot, a.w_trans, grp * kCIC, acc);
        else
            hipLaunchKernelGGL((k_sweep<T, COT, false, kAddF32>), grid, dim3(kBlock), 0, a.stream, S.runs, S.pats,
                               S.acts, S.offs, S.vals, g, (const T*)a.x, (const T*)a.w, (T*)a.y, (float*)nullptr, a.Ci,
                               a.Co, n_qtiles, n_cot, a.w_trans, grp * kCIC, acc);
        timing_end(tk, a.stream);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_grp > 1 && !f32 && S.n_cov > 0) {
        dim3 g2((unsigned)((g.nq + kBlock - 1) / kBlock), (unsigned)S.n_cov, (unsigned)(a.B * a.Co));
        const int tk = timing_begin("convert_y", a.stream);
        hipLaunchKernelGGL(k_convert_y, g2, dim3(kBlock), 0, a.stream, S.cov_pats, (const float*)y32,
                           (uint16_t*)a.y, g);
        timing_end(tk, a.stream);
    }
    return hipGetLastError();
}

template <typename T>
hipError_t sweep_dispatch(const ExecArgs& a, float* y32) {
    if (a.Co <= 4) return sweep_launch<T, 4>(a, y32);
    if (a.Co <= 8) return sweep_launch<T, 8>(a, y32);
    if (a.Co <= 16) return sweep_launch<T, 16>(a, y32);
    return sweep_launch<T, 32>(a, y32);
}

}  // namespace

DISCO_BOUNDS_READER(bounds_flag_sweep)

size_t workspace_bytes_sweep(const ExecArgs& a) {
    if (a.dtype != 1 || a.Ci <= kCIC || a.op->sweep.n_runs == 0) return 0;
    const OpGeom& g = a.op->g;
    return sizeof(float) * (size_t)a.B * a.Co * (size_t)g.nlat_o * g.nlon_o;
}

hipError_t launch_sweep(const ExecArgs& a, float* y32_ws) {
    return a.dtype == 1 ? sweep_dispatch<uint16_t>(a, y32_ws) : sweep_dispatch<float>(a, y32_ws);
}

hipError_t launch_sweep_z(const ExecArgs& a, float* z) {
    const OpGeom& g = a.op->g;
    const SweepDev& S = a.op->sweep_z.n_runs > 0 ? a.op->sweep_z : a.op->sweep;
    if (S.n_runs == 0) return hipSuccess;
    const int n_qtiles = (g.nq + kBlock - 1) / kBlock;
    const int n_cg = (a.Ci + kCIC - 1) / kCIC;
    dim3 grid((unsigned)(S.n_runs * n_qtiles), (unsigned)(a.B * n_cg));
    const int tk = timing_begin("sweep_gather_z", a.stream);
    if (a.dtype == 1)
        hipLaunchKernelGGL((k_sweep<uint16_t, 4, true, kStoreY>), grid, dim3(kBlock), 0, a.stream, S.runs, S.pats,
                           S.acts, S.offs, S.vals, g, (const uint16_t*)a.x, (const uint16_t*)nullptr,
                           (uint16_t*)nullptr, z, a.Ci, a.Co, n_qtiles, n_cg, a.w_trans, 0, (float*)nullptr);
    else
        hipLaunchKernelGGL((k_sweep<float, 4, true, kStoreY>), grid, dim3(kBlock), 0, a.stream, S.runs, S.pats, S.acts,
                           S.offs, S.vals, g, (const float*)a.x, (const float*)nullptr, (float*)nullptr, z, a.Ci, a.Co,
                           n_qtiles, n_cg, a.w_trans, 0, (float*)nullptr);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

}  // namespace disco
