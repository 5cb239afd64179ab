// disco_mfma.hip -- Sec. 4.2's compressed product (eq. 9) for bf16 storage
// with both of its steps on bf16 matrix cores (layout and notation in
// disco_internal.h, "Matrix-core layout").
//
// Per workgroup: one segment of an output ring (all longitude phases), one
// tile of kMfmaTile output longitudes, one batch item, up to 32 output
// channels.  For every pass over kMfmaCis input channels:
//   1. the segment's spans are staged into LDS, each staged element holding
//      two consecutive inputs (4 bytes), so that the eight inputs a lane
//      needs for one instruction (x[s q + d0 .. s q + d0 + 7]) are the four
//      elements e, e + 2, e + 4, e + 6: two ds_read2_b32 at any longitude
//      alignment;
//   2. per input channel and chunk, v_mfma_f32_16x16x32_bf16 accumulates
//      Z[phase][k][16 longitudes] (A = the chunk's values, B = the inputs);
//   3. per pair of input channels, Z of both (rounded to bf16) is the B
//      operand of the contraction with W (A), into y[phase][co][longitude]
//      in fp32.
// The values are rounded to bf16 for the matrix cores (the stored x and W
// are bf16 already); accumulation is fp32 throughout.  The accumulation
// order of an output depends only on its ring and phase, not on its
// longitude.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

DISCO_BOUNDS_FLAG

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));

constexpr int kNB = 4;                          // 16-longitude blocks per wave
constexpr int kWaves = kMfmaTile / (16 * kNB);  // waves per workgroup
static_assert(kWaves * 64 == kMfmaTile, "one lane per output longitude of a block row");
static_assert(kMfmaCis % 2 == 0, "the contraction takes input channels in pairs");

__device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// W operand table: for input-channel pair cp and 16-channel output block cb,
// lane i + 16 g holds the 8 bf16 W[co = 16 cb + i][ci = 2 cp + j / 4][k =
// 4 g + j % 4], j = 0..7, zero outside the tensor and for k >= 9.  The
// contraction's reduction index 8 g + j thus pairs with row 4 g + j % 4 of
// the Z of channel 2 cp + j / 4, which is where the first product leaves it.
// w: [Co][Ci][9], or [Ci][Co][9] when w_trans.  grid: ceil(n_pairs * n_cb * 64 / 256).
__global__ __launch_bounds__(256) void k_mfma_wop(const uint16_t* __restrict__ w, uint4* __restrict__ wop, int Ci,
                                                  int Co, int n_pairs, int n_cb, bool w_trans) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n_pairs * n_cb * 64) return;
    const int lane = i & 63, cb = (i >> 6) % n_cb, cp = (i >> 6) / n_cb;
    const int co = 16 * cb + (lane & 15), g = lane >> 4;
    uint32_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int ci = 2 * cp + j / 4, k = 4 * g + j % 4;
        const bool in = co < Co && ci < Ci && k < kBasis;
        const int64_t idx = w_trans ? ((int64_t)ci * Co + co) * kBasis + k : ((int64_t)co * Ci + ci) * kBasis + k;
        v[j] = in ? w[idx] : 0u;
    }
    wop[i] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
}

// Most spans one segment can have: one per group.
constexpr int kMfmaMaxSpans = 4 * kMfmaMaxChunks;

// Staging of one pass (kMfmaCis input channels): thread item it is (channel
// cl, block blk of 8 staged elements), fixed for the workgroup (code
// cl << 8 | blk, or -1); one aligned 16-byte and one 4-byte load give the 9
// inputs the block's elements hold, from the block's ring offset in the
// table sb (row + longitude of the block at q0, bit 31: the next 8 inputs
// wrap past the seam).  Loads for the next pass are issued before the
// current pass computes and written to LDS after it.
constexpr int kStageItems = (kMfmaCis * kMfmaMaxElems / 8 + kMfmaTile - 1) / kMfmaTile;
constexpr int kWopItems = kMfmaCis / 2 * 2 * 64 / kMfmaTile;  // W operands per thread (two output blocks)
static_assert(kMfmaCis / 2 * 2 * 64 % kMfmaTile == 0, "W operands spread evenly over the threads");
static_assert(kMfmaMaxElems / 8 <= 256 && kMfmaCis <= 128, "item codes pack the block into 8 bits");
struct Stage {
    uint4 a[kStageItems];
    uint32_t c[kStageItems];
    uint4 w[kWopItems];
};

__device__ __forceinline__ void stage_load(Stage& st, const int (&code)[kStageItems], const int* sb, int ci0, int Ci,
                                           const uint16_t* __restrict__ xb, int64_t n_in, int N,
                                           const uint4* __restrict__ wop, const int (&widx)[kWopItems]) {
    // Every item loads (items without data read the first staged block of
    // channel 0, which exists) and zeroes what it must not use: no branches.
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int cl = code[it] >> 8;
        const bool ok = code[it] >= 0 && ci0 + cl < Ci;
        const int v = sb[ok ? code[it] & 255 : 0];
        const uint16_t* xp = xb + (ok ? (int64_t)(ci0 + cl) * n_in : 0) + (v & 0x7fffffff);
        const uint4 a = *(const uint4*)xp;
        const uint32_t c = *(const uint32_t*)(xp + (v < 0 ? 8 - N : 8));
        st.a[it] = ok ? a : make_uint4(0u, 0u, 0u, 0u);
        st.c[it] = ok ? c : 0u;
    }
#pragma unroll
    for (int j = 0; j < kWopItems; ++j) {
        const uint4 wv = wop[widx[j] >= 0 ? widx[j] : 0];
        st.w[j] = widx[j] >= 0 ? wv : make_uint4(0u, 0u, 0u, 0u);
    }
}

__device__ __forceinline__ void stage_store(const Stage& st, const int (&code)[kStageItems], uint32_t* xs, uint4* ws,
                                            int nw, int tid) {
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        if (code[it] < 0) continue;
        const uint32_t wd[5] = {st.a[it].x, st.a[it].y, st.a[it].z, st.a[it].w, st.c[it]};
        uint4* dst = (uint4*)(xs + (code[it] >> 8) * kMfmaMaxElems + 8 * (code[it] & 255));
#pragma unroll
        for (int u = 0; u < 2; ++u)
            dst[u] = make_uint4(wd[2 * u], __builtin_amdgcn_alignbyte(wd[2 * u + 1], wd[2 * u], 2), wd[2 * u + 1],
                                __builtin_amdgcn_alignbyte(wd[2 * u + 2], wd[2 * u + 1], 2));
    }
#pragma unroll
    for (int j = 0; j < kWopItems; ++j)
        if (tid + j * kMfmaTile < nw) ws[tid + j * kMfmaTile] = st.w[j];
}

// NPH: longitude phases of the op (1 or 2); COB: 16-channel output blocks per
// workgroup (1 or 2).  grid: (the dispatch order's length, B * n_cot); the
// order maps a workgroup to its work item (see MfmaHost::order).
template <int NPH, int COB>
__global__ __launch_bounds__(kMfmaTile, 2) void k_mfma(const MSeg* __restrict__ segs, const PSpan* __restrict__ spans,
                                                    const MChunkHdr* __restrict__ chunks,
                                                    const uint4* __restrict__ aop, const uint4* __restrict__ wop,
                                                    const int32_t* __restrict__ order, OpGeom g,
                                                    const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                    float* __restrict__ partial, int Ci, int Co, int n_qtiles,
                                                    int n_cot) {
    __shared__ uint32_t xs[kMfmaCis * kMfmaMaxElems];
    __shared__ uint4 as[kMfmaMaxChunks * NPH * 64];
    __shared__ uint4 ws[kMfmaCis / 2 * COB * 64];
    __shared__ int hs[kMfmaMaxChunks * 4];
    __shared__ PSpan ss[kMfmaMaxSpans];
    __shared__ int sb[kMfmaMaxElems / 8];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 15, gq = lane >> 4;
    const int item = order[blockIdx.x];
    if (item < 0) return;
    const int segi = item / n_qtiles, qt = item - segi * n_qtiles;
    const int b = blockIdx.y / n_cot, cot = blockIdx.y - b * n_cot;
    const int n_cb = n_cot * COB;
    const MSeg S = segs[segi];
    const int nch = S.chunk_end - S.chunk_begin, nsp = S.span_end - S.span_begin;
    const int q0 = qt * kMfmaTile;
    const int s = g.stride, N = g.nlon_i;
    const int64_t n_in = (int64_t)g.nlat_i * N;
    const int lq = wave * 16 * kNB + n;  // tile-relative output longitude of this lane in block 0
    const int nblk = S.n_elems >> 3;     // 8-element blocks per staged channel
    constexpr int nw = kMfmaCis / 2 * COB * 64;

    for (int i = tid; i < nch * NPH * 64; i += kMfmaTile) as[i] = aop[(int64_t)S.chunk_begin * NPH * 64 + i];
    if (tid < nch * 4) hs[tid] = chunks[S.chunk_begin + tid / 4].grp[tid % 4];
    if (tid < nsp) ss[tid] = spans[S.span_begin + tid];
    __syncthreads();
    // Ring offset of every staged block at this tile (see stage_load).
    for (int blk = tid; blk < nblk; blk += kMfmaTile) {
        int sp = 0;
        while (sp + 1 < nsp && ss[sp + 1].lds_base <= 8 * blk) ++sp;
        const int lon = (s * q0 + ss[sp].dstart + 8 * blk - ss[sp].lds_base) % N;
        sb[blk] = (ss[sp].row + lon) | (lon + 8 >= N ? (int)0x80000000u : 0);
    }
    int code[kStageItems];
#pragma unroll
    for (int it = 0; it < kStageItems; ++it) {
        const int i = tid + it * kMfmaTile;
        const int cl = nblk > 0 ? i / nblk : kMfmaCis;
        code[it] = cl < kMfmaCis ? (cl << 8 | (i - cl * nblk)) : -1;
    }
    __syncthreads();
    const uint16_t* xb = x + (int64_t)b * Ci * n_in;
    // The first chunk's values stay in registers for the whole workgroup.
    bf8 A0[NPH];
#pragma unroll
    for (int r = 0; r < NPH; ++r) A0[r] = __builtin_bit_cast(bf8, as[r * 64 + lane]);

    // W operands of pass ci0: item i = tid + j kMfmaTile = (pair p, block
    // cb, lane l) < nw stages those of input-channel pair ci0 / 2 + p for
    // this workgroup's output block cb.
    auto widx = [&](int ci0, int (&wi)[kWopItems]) {
#pragma unroll
        for (int j = 0; j < kWopItems; ++j) {
            const int i = tid + j * kMfmaTile;
            const int wpl = i / (COB * 64), wcb = (i / 64) % COB, wln = i & 63;
            wi[j] = i < nw ? (((ci0 >> 1) + wpl) * n_cb + cot * COB + wcb) * 64 + wln : -1;
        }
    };
    Stage st;
    int wi[kWopItems];
    widx(0, wi);
    stage_load(st, code, sb, 0, Ci, xb, n_in, N, wop, wi);

    f4 Y[NPH][kNB][COB];
#pragma unroll
    for (int r = 0; r < NPH; ++r)
#pragma unroll
        for (int qb = 0; qb < kNB; ++qb)
#pragma unroll
            for (int cb = 0; cb < COB; ++cb) Y[r][qb][cb] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    for (int ci0 = 0; ci0 < Ci; ci0 += kMfmaCis) {
        __syncthreads();  // the previous pass's readers are done
        stage_store(st, code, xs, ws, nw, tid);
        __syncthreads();
        if (ci0 + kMfmaCis < Ci) {
            widx(ci0 + kMfmaCis, wi);
            stage_load(st, code, sb, ci0 + kMfmaCis, Ci, xb, n_in, N, wop, wi);
        }
        // Per pair of input channels: Z on the matrix cores, then the
        // contraction with W.
        // A segment without chunks (an output ring with no entries) leaves y
        // at zero.
#pragma unroll 1
        for (int cp = 0; cp < (nch > 0 ? kMfmaCis / 2 : 0); ++cp) {
            f4 Z[2][NPH][kNB];
            const uint32_t* xc = xs + 2 * cp * kMfmaMaxElems + s * lq;
            // One chunk: its LDS reads, then its products (the first chunk
            // starts the accumulators from zero).
            auto chunk = [&](int c, bool first) {
                DISCO_CHECK(hs[4 * c + gq] >= 0 && s * lq + hs[4 * c + gq] + 16 * s * (kNB - 1) + 6 < kMfmaMaxElems);
                const uint32_t* xb = xc + hs[4 * c + gq];
                bf8 A[NPH];
#pragma unroll
                for (int r = 0; r < NPH; ++r) A[r] = first ? A0[r] : __builtin_bit_cast(bf8, as[(c * NPH + r) * 64 + lane]);
                bf8 Bv[2][kNB];
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int qb = 0; qb < kNB; ++qb) {
                        const uint32_t* e = xb + h * kMfmaMaxElems + 16 * s * qb;
                        Bv[h][qb] = __builtin_bit_cast(bf8, make_uint4(e[0], e[2], e[4], e[6]));
                    }
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int qb = 0; qb < kNB; ++qb)
#pragma unroll
                        for (int r = 0; r < NPH; ++r)
                            Z[h][r][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                A[r], Bv[h][qb], first ? f4{0.0f, 0.0f, 0.0f, 0.0f} : Z[h][r][qb], 0, 0, 0);
                // All of the chunk's LDS reads first, then its products, so
                // that one wait covers them (the scheduler otherwise reuses one
                // register set and waits before every product pair).
                __builtin_amdgcn_sched_group_barrier(0x100, 4 * kNB, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 2 * kNB * NPH, 0);
            };
            chunk(0, true);
#pragma unroll 1
            for (int c = 1; c < nch; ++c) chunk(c, false);
            bf8 Wm[COB];
#pragma unroll
            for (int cb = 0; cb < COB; ++cb) Wm[cb] = __builtin_bit_cast(bf8, ws[(cp * COB + cb) * 64 + lane]);
#pragma unroll
            for (int r = 0; r < NPH; ++r)
#pragma unroll
                for (int qb = 0; qb < kNB; ++qb) {
                    const f8 zz = {Z[0][r][qb][0], Z[0][r][qb][1], Z[0][r][qb][2], Z[0][r][qb][3],
                                   Z[1][r][qb][0], Z[1][r][qb][1], Z[1][r][qb][2], Z[1][r][qb][3]};
                    const bf8 zb = __builtin_convertvector(zz, bf8);
#pragma unroll
                    for (int cb = 0; cb < COB; ++cb)
                        Y[r][qb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Wm[cb], zb, Y[r][qb][cb], 0, 0, 0);
                }
        }
    }

    // Lane n + 16 g holds y[co = 16 cb + 4 g + j][q] in register j of each block.
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const int B = gridDim.y / n_cot;
#pragma unroll
    for (int qb = 0; qb < kNB; ++qb) {
        const int q = q0 + lq + 16 * qb;
        if (q >= g.nq) continue;
#pragma unroll
        for (int cb = 0; cb < COB; ++cb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int co = 16 * (cot * COB + cb) + 4 * gq + j;
                if (co >= Co) continue;
                if (S.slot < 0) {
                    const int64_t pix = (int64_t)S.ring * g.nlon_o + (int64_t)q * NPH;
                    uint16_t* yp = y + ((int64_t)b * Co + co) * n_out + pix;
                    if constexpr (NPH == 2) {
                        *(uint32_t*)yp = (uint32_t)to_bf16(Y[0][qb][cb][j]) | ((uint32_t)to_bf16(Y[1][qb][cb][j]) << 16);
                    } else {
                        *yp = to_bf16(Y[0][qb][cb][j]);
                    }
                } else {
#pragma unroll
                    for (int r = 0; r < NPH; ++r)
                        partial[(((int64_t)(S.slot + r) * B + b) * Co + co) * g.nq + q] = Y[r][qb][cb][j];
                }
            }
    }
}

int mfma_cob(int Co) { return Co <= 16 ? 1 : 2; }
int mfma_pairs(int Ci) { return (Ci + kMfmaCis - 1) / kMfmaCis * (kMfmaCis / 2); }
size_t mfma_wop_bytes(const ExecArgs& a) {
    const int cob = mfma_cob(a.Co), n_cot = (a.Co + 16 * cob - 1) / (16 * cob);
    return ((size_t)mfma_pairs(a.Ci) * n_cot * cob * 64 * 16 + 255) / 256 * 256;
}

template <int NPH, int COB>
hipError_t mfma_launch(const ExecArgs& a, const uint4* wop, float* partial) {
    const MfmaDev& M = a.op->mfma;
    const OpGeom& g = a.op->g;
    const int n_cot = (a.Co + 16 * COB - 1) / (16 * COB);
    dim3 grid((unsigned)M.n_order, (unsigned)(a.B * n_cot));
    const int tk = timing_begin("mfma_gather_contract", a.stream);
    hipLaunchKernelGGL((k_mfma<NPH, COB>), grid, dim3(kMfmaTile), 0, a.stream, M.segs, M.spans, M.chunks,
                       (const uint4*)M.aop, wop, M.order, g, (const uint16_t*)a.x, (uint16_t*)a.y, partial, a.Ci,
                       a.Co, M.n_qtiles, n_cot);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

}  // namespace

DISCO_BOUNDS_READER(bounds_flag_mfma)

size_t workspace_bytes_mfma(const ExecArgs& a) {
    return mfma_wop_bytes(a) + sizeof(float) * (size_t)a.op->mfma.P.n_slots * a.B * a.Co * a.op->g.nq;
}

hipError_t launch_mfma(const ExecArgs& a, void* ws) {
    const MfmaDev& M = a.op->mfma;
    if (M.n_segs == 0) return hipSuccess;
    const int cob = mfma_cob(a.Co), n_cot = (a.Co + 16 * cob - 1) / (16 * cob);
    const int n_pairs = mfma_pairs(a.Ci), n_cb = n_cot * cob;
    uint4* wop = (uint4*)ws;
    float* partial = (float*)((char*)ws + mfma_wop_bytes(a));
    const int n_w = n_pairs * n_cb * 64;
    int tk = timing_begin("mfma_weights", a.stream);
    hipLaunchKernelGGL(k_mfma_wop, dim3((unsigned)((n_w + 255) / 256)), dim3(256), 0, a.stream,
                       (const uint16_t*)a.w, wop, a.Ci, a.Co, n_pairs, n_cb, a.w_trans);
    timing_end(tk, a.stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const bool two = a.op->g.P == 2;
    if (two) e = cob == 1 ? mfma_launch<2, 1>(a, wop, partial) : mfma_launch<2, 2>(a, wop, partial);
    else e = cob == 1 ? mfma_launch<1, 1>(a, wop, partial) : mfma_launch<1, 2>(a, wop, partial);
    if (e != hipSuccess) return e;
    return launch_reduce_partials(a, M.P, partial);
}

}  // namespace disco
