// disco_grad.hip -- the weight gradient's reduction over pixels (App. C).
//
// With the gathered sums Zs[b][(c_x, k)][p] of an op (computed by the op's
// own kernels with a selection W) and the upstream gradient dy[b][m][p],
//   G[m][n] = sum_b sum_p dy[b][m][p] Zs[b][n][p],   n = c_x K + k,
// is a product of two short, very wide matrices.  k_weight_grad_mfma gives
// each workgroup one batch item, one range of pixels and a tile of G of 16
// rows of dy by up to 128 rows of Zs (so that, for N <= 128, every input
// element is read from HBM once): steps of 64 pixels of all the tile's rows
// are staged in LDS with coalesced loads (the next step's loads in flight
// while the current one computes), and v_mfma_f32_16x16x4_f32 reduces four
// pixels per instruction, the four waves taking alternate groups of four;
// the waves' tiles are summed in LDS and the workgroup writes its partial
// tile.  k_weight_grad_reduce sums the partials of each element over (batch
// item, pixel range) in a fixed order, so the result is deterministic, and
// writes dW in the op's layout.
//
// Depthwise channels need only the diagonal blocks, dW[c][k] = sum_b sum_p
// dy[b][c][p] Zs[b][c][k][p]: k_weight_grad (every lane accumulates a 1 x K
// tile over its pixels, the lanes' tiles summed with lane shuffles and the
// waves' in LDS) runs on B x C one-row items (M = 1, N = K) and
// k_weight_grad_reduce_dw sums each channel's partials over (batch item,
// pixel range) in a fixed order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

constexpr int kBlock = 256;
constexpr int kTileM = 8;   // rows of dy per workgroup
constexpr int kTileN = 16;  // rows of Zs per workgroup (dy is read N / kTileN times)

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

// grid: (n_chunks * n_mt * n_nt, 1, B), the pixel chunk fastest in x (grid x
// has no 16-bit limit, so any number of tiles fits).  partial:
// [B][n_chunks][M][N].
template <typename T>
__global__ __launch_bounds__(kBlock) void k_weight_grad(const T* __restrict__ dy, const T* __restrict__ zs,
                                                        float* __restrict__ partial, int M, int N, int64_t P,
                                                        int64_t chunk_len, int n_nt, int n_chunks) {
    __shared__ float red[kBlock / 64][kTileM * kTileN];
    const int tid = threadIdx.x;
    const int chunk = (int)(blockIdx.x % (unsigned)n_chunks);
    const int tile = (int)(blockIdx.x / (unsigned)n_chunks);
    const int m0 = (tile / n_nt) * kTileM, n0 = (tile % n_nt) * kTileN;
    const int b = blockIdx.z;
    const int64_t p0 = (int64_t)chunk * chunk_len;
    const int64_t p1 = p0 + chunk_len < P ? p0 + chunk_len : P;
    float acc[kTileM][kTileN];
#pragma unroll
    for (int i = 0; i < kTileM; ++i)
#pragma unroll
        for (int j = 0; j < kTileN; ++j) acc[i][j] = 0.0f;
    const T* dyb = dy + (int64_t)b * M * P;
    const T* zb = zs + (int64_t)b * N * P;
    for (int64_t p = p0 + tid; p < p1; p += kBlock) {
        float a[kTileM], z[kTileN];
#pragma unroll
        for (int i = 0; i < kTileM; ++i) a[i] = m0 + i < M ? load_val(dyb, (int64_t)(m0 + i) * P + p) : 0.0f;
#pragma unroll
        for (int j = 0; j < kTileN; ++j) z[j] = n0 + j < N ? load_val(zb, (int64_t)(n0 + j) * P + p) : 0.0f;
#pragma unroll
        for (int i = 0; i < kTileM; ++i)
#pragma unroll
            for (int j = 0; j < kTileN; ++j) acc[i][j] = fmaf(a[i], z[j], acc[i][j]);
    }
    // Sum over the 64 lanes of each wave, then over the waves.
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < kTileM; ++i)
#pragma unroll
        for (int j = 0; j < kTileN; ++j) {
            float v = acc[i][j];
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[wave][i * kTileN + j] = v;
        }
    __syncthreads();
    if (tid < kTileM * kTileN) {
        const int i = tid / kTileN, j = tid % kTileN;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) v += red[w][tid];
        if (m0 + i < M && n0 + j < N)
            partial[(((int64_t)b * n_chunks + chunk) * M + m0 + i) * N + n0 + j] = v;
    }
}

typedef float f4v __attribute__((ext_vector_type(4)));
constexpr int kMT = 16;          // rows of dy per workgroup (the instruction's 16 rows)
constexpr int kPix = 64;         // pixels staged per step (one per lane and row)
constexpr int kLd = kPix + 2;    // LDS row stride in floats: operand reads free of bank conflicts

// grid: (n_chunks * n_mt * n_nt, 1, B), n_mt = ceil(M / 16), n_nt = ceil(N /
// (16 NB)).  Row r of batch item b starts at (b rows + r) * stride and P of
// its values are summed (P <= stride).  LDS rows 0..15 hold dy rows m0..,
// rows 16.. the Zs rows n0..; rows past M or N hold zeros.  partial:
// [B][n_chunks][M][N].
template <typename T, int NB>
__global__ __launch_bounds__(kBlock) void k_weight_grad_mfma(const T* __restrict__ dy, const T* __restrict__ zs,
                                                             float* __restrict__ partial, int M, int N, int64_t P,
                                                             int64_t stride, int64_t chunk_len, int n_nt,
                                                             int n_chunks) {
    constexpr int kRows = kMT + 16 * NB;
    constexpr int kIt = kRows / (kBlock / 64);  // staged rows per wave and step
    static_assert(kRows % (kBlock / 64) == 0, "the waves stage whole rows");
    static_assert(kRows * kLd >= 4 * NB * 256, "the wave reduction fits the staging buffer");
    __shared__ float st[kRows * kLd];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int chunk = (int)(blockIdx.x % (unsigned)n_chunks);
    const int tile = (int)(blockIdx.x / (unsigned)n_chunks);
    const int m0 = (tile / n_nt) * kMT, n0 = (tile % n_nt) * (16 * NB);
    const int mr = M - m0 < kMT ? M - m0 : kMT, nr = N - n0 < 16 * NB ? N - n0 : 16 * NB;
    const int b = blockIdx.z;
    const int64_t p0 = (int64_t)chunk * chunk_len;
    const int64_t p1 = p0 + chunk_len < P ? p0 + chunk_len : P;
    const T* dyb = dy + (int64_t)b * M * stride;
    const T* zb = zs + (int64_t)b * N * stride;
    // Staged row r = wave + 4 it of this lane: its source row (wave-uniform),
    // or none.
    auto row_src = [&](int r) -> const T* {
        if (r < kMT) return r < mr ? dyb + (int64_t)(m0 + r) * stride : nullptr;
        return r - kMT < nr ? zb + (int64_t)(n0 + r - kMT) * stride : nullptr;
    };
    auto load_step = [&](int64_t ps, float (&v)[kIt]) {
        const int64_t p = ps + lane;
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const T* src = row_src(wave + 4 * it);
            v[it] = src && p < p1 ? load_val(src, p) : 0.0f;
        }
    };
    f4v C[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) C[nb] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
    float v[kIt];
    if (p0 < p1) load_step(p0, v);
    for (int64_t ps = p0; ps < p1; ps += kPix) {
        __syncthreads();  // the previous step's operand reads are done
#pragma unroll
        for (int it = 0; it < kIt; ++it) st[(wave + 4 * it) * kLd + lane] = v[it];
        __syncthreads();
        if (ps + kPix < p1) load_step(ps + kPix, v);
        // Instruction kk of wave w reduces pixels 4 (w + 4 kk) .. + 3 of the
        // step: lane (row i, k) supplies dy[i][4 (w + 4 kk) + k] and, for
        // block nb, Zs[16 nb + i][same pixel].
        const int row = lane & 15;
#pragma unroll
        for (int kk = 0; kk < kPix / 16; ++kk) {
            const int pc = 4 * (wave + 4 * kk) + (lane >> 4);
            const float a = st[row * kLd + pc];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                C[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, st[(kMT + 16 * nb + row) * kLd + pc], C[nb], 0, 0, 0);
        }
    }
    // Lane (g, j) of block nb holds G[m0 + 4 g + r][n0 + 16 nb + j] in
    // register r; the waves' tiles are summed in LDS in wave order.
    __syncthreads();
    float* red = st;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((wave * NB + nb) * 4 + r) * 64 + lane] = C[nb][r];
    __syncthreads();
    for (int i = tid; i < NB * 256; i += kBlock) {
        const int nb = i >> 8, r = (i >> 6) & 3, l = i & 63;
        float acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) acc += red[((w * NB + nb) * 4 + r) * 64 + l];
        const int mi = 4 * (l >> 4) + r, nj = 16 * nb + (l & 15);
        if (mi < mr && nj < nr) partial[(((int64_t)b * n_chunks + chunk) * M + m0 + mi) * N + n0 + nj] = acc;
    }
}

// One workgroup per dW element e = (m, n): lane t sums the partials
// t, t + 256, ... of e over (b, chunk), then a fixed tree over the lanes.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_weight_grad_reduce(const float* __restrict__ partial, T* __restrict__ dw,
                                                               int B, int n_chunks, int M, int C_x, int K,
                                                               bool transposed_layout) {
    __shared__ float red[kBlock];
    const int N = C_x * K;
    const int e = blockIdx.x;
    const int tid = threadIdx.x;
    float v = 0.0f;
    for (int s = tid; s < B * n_chunks; s += kBlock) v += partial[(int64_t)s * M * N + e];
    red[tid] = v;
    __syncthreads();
    for (int half = kBlock / 2; half > 0; half >>= 1) {
        if (tid < half) red[tid] += red[tid + half];
        __syncthreads();
    }
    if (tid == 0) {
        const int m = e / N, n = e - (e / N) * N;
        const int cx = n / K, k = n - (n / K) * K;
        const int64_t at = transposed_layout ? ((int64_t)cx * M + m) * K + k : ((int64_t)m * C_x + cx) * K + k;
        store_val(dw, at, red[0]);
    }
}

// One workgroup per dW element e = (c, k) of a depthwise [C][K] dW: lane t
// sums the partials of items b C + c over (b, chunk) pairs t, t + 256, ...,
// then a fixed tree over the lanes.  partial: [B C][n_chunks][K].
template <typename T>
__global__ __launch_bounds__(kBlock) void k_weight_grad_reduce_dw(const float* __restrict__ partial,
                                                                  T* __restrict__ dw, int B, int C, int n_chunks,
                                                                  int K) {
    __shared__ float red[kBlock];
    const int e = blockIdx.x;
    const int c = e / K, k = e - (e / K) * K;
    const int tid = threadIdx.x;
    float v = 0.0f;
    for (int s = tid; s < B * n_chunks; s += kBlock) {
        const int b = s / n_chunks, chunk = s - (s / n_chunks) * n_chunks;
        v += partial[(((int64_t)b * C + c) * n_chunks + chunk) * K + k];
    }
    red[tid] = v;
    __syncthreads();
    for (int half = kBlock / 2; half > 0; half >>= 1) {
        if (tid < half) red[tid] += red[tid + half];
        __syncthreads();
    }
    if (tid == 0) store_val(dw, e, red[0]);
}

int64_t chunk_len_for(int B, int M, int N, int64_t P) {
    const int tiles = ((M + kTileM - 1) / kTileM) * ((N + kTileN - 1) / kTileN) * B;
    const int64_t want = std::max<int64_t>(1, 2048 / std::max(1, tiles));  // chunks per tile
    int64_t len = (P + want - 1) / want;
    len = std::max<int64_t>(len, 16 * kBlock);
    return (len + kBlock - 1) / kBlock * kBlock;
}

// Zs blocks of 16 rows per workgroup: all of N up to 128.
int mfma_nb(int N) { return std::min(8, std::max(1, (N + 15) / 16)); }

// Pixels per workgroup of the matrix-core kernel: about 2048 workgroups in
// all, at least 16 steps each.
int64_t chunk_len_mfma(int B, int M, int N, int64_t P) {
    const int nb = mfma_nb(N);
    const int tiles = ((M + kMT - 1) / kMT) * ((N + 16 * nb - 1) / (16 * nb)) * B;
    const int64_t want = std::max<int64_t>(1, 2048 / std::max(1, tiles));
    int64_t len = (P + want - 1) / want;
    len = std::max<int64_t>(len, 16 * kPix);
    return (len + kPix - 1) / kPix * kPix;
}

template <typename T, int NB>
void launch_wg_mfma(dim3 grid, hipStream_t s, const T* dy, const T* zs, float* ws, int M, int N, int64_t P,
                    int64_t stride, int64_t len, int n_nt, int n_chunks) {
    hipLaunchKernelGGL((k_weight_grad_mfma<T, NB>), grid, dim3(kBlock), 0, s, dy, zs, ws, M, N, P, stride, len, n_nt,
                       n_chunks);
}

// Partial slabs ([M][N] each) one launch of k_weight_grad_mfma writes.
int64_t wg_slabs(int B, int M, int N, int64_t P) {
    const int64_t len = chunk_len_mfma(B, M, N, P);
    return (int64_t)B * std::max<int64_t>(1, (P + len - 1) / len);
}

// The partial tiles of G over B batch items of rows with P summed values
// each (row stride `stride`), into wg_slabs(B, M, N, P) slabs at ws.
template <typename T>
hipError_t weight_grad_part(const T* dy, const T* zs, float* ws, int B, int M, int N, int64_t P, int64_t stride,
                            hipStream_t s) {
    const int64_t len = chunk_len_mfma(B, M, N, P);
    const int n_chunks = (int)std::max<int64_t>(1, (P + len - 1) / len);
    const int nb = mfma_nb(N);
    const int n_mt = (M + kMT - 1) / kMT, n_nt = (N + 16 * nb - 1) / (16 * nb);
    dim3 grid((unsigned)((int64_t)n_chunks * n_mt * n_nt), 1u, (unsigned)B);
    switch (nb) {
        case 1: launch_wg_mfma<T, 1>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 2: launch_wg_mfma<T, 2>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 3: launch_wg_mfma<T, 3>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 4: launch_wg_mfma<T, 4>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 5: launch_wg_mfma<T, 5>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 6: launch_wg_mfma<T, 6>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        case 7: launch_wg_mfma<T, 7>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
        default: launch_wg_mfma<T, 8>(grid, s, dy, zs, ws, M, N, P, stride, len, n_nt, n_chunks); break;
    }
    return hipGetLastError();
}

template <typename T>
hipError_t weight_grad_reduce(const float* ws, T* dw, int64_t slabs, int M, int C_x, int K, bool transposed_layout,
                              hipStream_t s) {
    const int tk = timing_begin("weight_grad_reduce", s);
    hipLaunchKernelGGL((k_weight_grad_reduce<T>), dim3((unsigned)(M * C_x * K)), dim3(kBlock), 0, s, ws, dw, 1,
                       (int)slabs, M, C_x, K, transposed_layout);
    timing_end(tk, s);
    return hipGetLastError();
}

template <typename T>
hipError_t weight_grad(const T* dy, const T* zs, T* dw, float* ws, int B, int M, int C_x, int K, int64_t P,
                       bool transposed_layout, hipStream_t s) {
    const int N = C_x * K;
    const int tk = timing_begin("weight_grad", s);
    hipError_t e = weight_grad_part(dy, zs, ws, B, M, N, P, P, s);
    timing_end(tk, s);
    if (e != hipSuccess) return e;
    return weight_grad_reduce(ws, dw, wg_slabs(B, M, N, P), M, C_x, K, transposed_layout, s);
}

template <typename T>
hipError_t weight_grad_dw(const T* dy, const T* zs, T* dw, float* ws, int B, int C, int K, int64_t P, hipStream_t s) {
    const int items = B * C;
    const int64_t len = chunk_len_for(items, 1, K, P);
    const int n_chunks = (int)std::max<int64_t>(1, (P + len - 1) / len);
    dim3 grid((unsigned)n_chunks, 1u, (unsigned)items);
    int tk = timing_begin("weight_grad", s);
    hipLaunchKernelGGL((k_weight_grad<T>), grid, dim3(kBlock), 0, s, dy, zs, ws, 1, K, P, len, 1, n_chunks);
    timing_end(tk, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    tk = timing_begin("weight_grad_reduce", s);
    hipLaunchKernelGGL((k_weight_grad_reduce_dw<T>), dim3((unsigned)(C * K)), dim3(kBlock), 0, s, ws, dw, B, C,
                       n_chunks, K);
    timing_end(tk, s);
    return hipGetLastError();
}

}  // namespace

namespace {
__global__ __launch_bounds__(kBlock) void k_zero_fill(uint16_t* __restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) p[i] = 0;
}
}  // namespace

hipError_t launch_zero_fill(void* p, size_t bytes, hipStream_t s) {
    const int64_t n = (int64_t)(bytes / 2);
    if (n == 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<int64_t>(1024, (n + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(k_zero_fill, dim3(blocks), dim3(kBlock), 0, s, (uint16_t*)p, n);
    return hipGetLastError();
}

size_t weight_grad_ws_bytes_dw(int B, int C, int K, int64_t P) {
    const int items = B * C;
    const int64_t len = chunk_len_for(items, 1, K, P);
    const int64_t n_chunks = std::max<int64_t>(1, (P + len - 1) / len);
    return sizeof(float) * (size_t)items * (size_t)n_chunks * (size_t)K;
}

hipError_t launch_weight_grad_dw(const void* dy, const void* zs, void* dw, float* ws, int dtype, int B, int C, int K,
                                 int64_t P, hipStream_t s) {
    if (K > kTileN) return hipErrorInvalidValue;
    if (dtype == 1)
        return weight_grad_dw<uint16_t>((const uint16_t*)dy, (const uint16_t*)zs, (uint16_t*)dw, ws, B, C, K, P, s);
    return weight_grad_dw<float>((const float*)dy, (const float*)zs, (float*)dw, ws, B, C, K, P, s);
}

size_t weight_grad_ws_bytes(int B, int M, int N, int64_t P) {
    return sizeof(float) * (size_t)wg_slabs(B, M, N, P) * (size_t)M * (size_t)N;
}

size_t weight_grad_split_ws_bytes(int B, int M, int N, int64_t P_light, int B_heavy, int64_t P_heavy) {
    return sizeof(float) * (size_t)(wg_slabs(B, M, N, P_light) + wg_slabs(B_heavy, M, N, P_heavy)) * (size_t)M *
           (size_t)N;
}

hipError_t launch_weight_grad_split(const float* dy, const float* zs, int B, int64_t P_light, int64_t stride,
                                    const float* dyh, const float* zh, int B_heavy, int64_t P_heavy, float* dw,
                                    float* ws, int M, int C_x, int K, bool transposed_layout, hipStream_t s) {
    const int N = C_x * K;
    const int64_t s1 = wg_slabs(B, M, N, P_light);
    const int tk = timing_begin("weight_grad", s);
    hipError_t e = weight_grad_part(dy, zs, ws, B, M, N, P_light, stride, s);
    if (e == hipSuccess) e = weight_grad_part(dyh, zh, ws + s1 * M * N, B_heavy, M, N, P_heavy, P_heavy, s);
    timing_end(tk, s);
    if (e != hipSuccess) return e;
    return weight_grad_reduce(ws, dw, s1 + wg_slabs(B_heavy, M, N, P_heavy), M, C_x, K, transposed_layout, s);
}

hipError_t launch_weight_grad(const void* dy, const void* zs, void* dw, float* ws, int dtype, int B, int M,
                              int C_x, int K, int64_t P, bool transposed_layout, hipStream_t s) {
    if (dtype == 1)
        return weight_grad<uint16_t>((const uint16_t*)dy, (const uint16_t*)zs, (uint16_t*)dw, ws, B, M, C_x, K, P,
                                     transposed_layout, s);
    return weight_grad<float>((const float*)dy, (const float*)zs, (float*)dw, ws, B, M, C_x, K, P, transposed_layout,
                              s);
}

}  // namespace disco
