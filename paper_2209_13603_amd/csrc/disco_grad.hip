// disco_grad.hip -- the weight gradient's reduction over pixels (App. C).
//
// With the gathered sums Zs[b][(c_x, k)][p] of an op (computed by the op's
// own kernels with a selection W) and the upstream gradient dy[b][m][p],
//   G[m][n] = sum_b sum_p dy[b][m][p] Zs[b][n][p],   n = c_x K + k,
// is a product of two short, very wide matrices.  k_weight_grad gives each
// workgroup one batch item, one range of pixels and an 8 x 16 tile of G: every
// lane accumulates the tile over its pixels (24 coalesced loads and 128 FMAs
// per pixel), the lanes' tiles are summed across the wave with lane shuffles
// and across the four waves in LDS, and the workgroup writes its partial tile.
// k_weight_grad_reduce sums the partials of each element over (batch item,
// pixel range) in a fixed order, so the result is deterministic, and writes
// dW in the op's layout.
//
// Depthwise channels need only the diagonal blocks, dW[c][k] = sum_b sum_p
// dy[b][c][p] Zs[b][c][k][p]: k_weight_grad runs on B x C one-row items
// (M = 1, N = K) and k_weight_grad_reduce_dw sums each channel's partials over
// (batch item, pixel range) in a fixed order.
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

template <typename T>
hipError_t weight_grad(const T* dy, const T* zs, T* dw, float* ws, int B, int M, int C_x, int K, int64_t P,
                       bool transposed_layout, hipStream_t s) {
    const int N = C_x * K;
    const int64_t len = chunk_len_for(B, M, N, P);
    const int n_chunks = (int)std::max<int64_t>(1, (P + len - 1) / len);
    const int n_mt = (M + kTileM - 1) / kTileM, n_nt = (N + kTileN - 1) / kTileN;
    dim3 grid((unsigned)((int64_t)n_chunks * n_mt * n_nt), 1u, (unsigned)B);
    int tk = timing_begin("weight_grad", s);
    hipLaunchKernelGGL((k_weight_grad<T>), grid, dim3(kBlock), 0, s, dy, zs, ws, M, N, P, len, n_nt, n_chunks);
    timing_end(tk, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int ne = M * N;
    tk = timing_begin("weight_grad_reduce", s);
    hipLaunchKernelGGL((k_weight_grad_reduce<T>), dim3((unsigned)ne), dim3(kBlock), 0, s, ws, dw, B, n_chunks, M, C_x,
                       K, transposed_layout);
    timing_end(tk, s);
    return hipGetLastError();
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
    return weight_grad_ws_bytes(B * C, 1, K, P);
}

hipError_t launch_weight_grad_dw(const void* dy, const void* zs, void* dw, float* ws, int dtype, int B, int C, int K,
                                 int64_t P, hipStream_t s) {
    if (K > kTileN) return hipErrorInvalidValue;
    if (dtype == 1)
        return weight_grad_dw<uint16_t>((const uint16_t*)dy, (const uint16_t*)zs, (uint16_t*)dw, ws, B, C, K, P, s);
    return weight_grad_dw<float>((const float*)dy, (const float*)zs, (float*)dw, ws, B, C, K, P, s);
}

size_t weight_grad_ws_bytes(int B, int M, int N, int64_t P) {
    const int64_t len = chunk_len_for(B, M, N, P);
    const int64_t n_chunks = std::max<int64_t>(1, (P + len - 1) / len);
    return sizeof(float) * (size_t)B * (size_t)n_chunks * (size_t)M * (size_t)N;
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
