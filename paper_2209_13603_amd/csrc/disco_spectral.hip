// disco_spectral.hip -- the spectral path for heavy output rings.
//
// Near the poles an output ring's windows span whole input rings, so its sum
// over one input ring is a circular cross-correlation along longitude
// (Sec. 4.2: one pattern reused at every output longitude).  Three kernels
// evaluate it exactly through the DFT (N = nlon, M = N / 2, power of two):
//   k_rfft_rings : Xhat of every input ring a heavy ring reads (real N-point
//                  DFT as an M-point complex Stockham FFT in LDS + split),
//   k_spectral   : Yhat[co][m] = sum_{t_i, ci} Xhat[t_i][ci][m] sum_k W[co][ci][k]
//                  conj(Vhat_k[m]), using Vhat_{3a+2} = conj(Vhat_{3a}) and
//                  real Vhat_{3a+1} (9 stored floats per pair and frequency),
//   k_irfft_rings: y of each heavy ring from Yhat (inverse real DFT).
// Vhat is precomputed on the host in fp64 and scaled by 1 / N; the device
// transforms are unnormalised.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

constexpr int kFftBlock = 256;
constexpr int kFftBatch = 8;  // global loads per thread in flight while staging a ring

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

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
    return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
__device__ __forceinline__ float2 conjf2(float2 a) { return make_float2(a.x, -a.y); }

// Twiddles in LDS as two short tables, hi[t >> 6] = tw[64 (t >> 6)] and
// lo[t & 63] = tw[t & 63], whose product is tw[t] = exp(-2 pi i t / (2M))
// (t < M) to a few ulp: 33.5 KB of LDS per FFT workgroup at M = 2048
// instead of 48 KB with the whole table, so four workgroups share a CU.
constexpr int kTwLo = 64;
__host__ __device__ constexpr int tw_hi_len(int M) { return M > kTwLo ? M / kTwLo : 1; }

// Fills the two tables from the global table tw (t < M); all threads.
__device__ __forceinline__ void load_twiddles(const float2* __restrict__ tw, float2* __restrict__ thi,
                                              float2* __restrict__ tlo, int M) {
    for (int i = threadIdx.x; i < kTwLo + tw_hi_len(M); i += blockDim.x) {
        if (i < kTwLo) {
            if (i < M) tlo[i] = tw[i];
        } else {
            thi[i - kTwLo] = tw[kTwLo * (i - kTwLo)];
        }
    }
}

// exp(-/+ 2 pi i t / (2M)) for t in [0, 2M) (the upper half is the negative
// of the lower).
__device__ __forceinline__ float2 tw_at(const float2* __restrict__ thi, const float2* __restrict__ tlo, int t,
                                        int M, bool inverse) {
    const bool upper = t >= M;
    const int tt = upper ? t - M : t;
    float2 w = cmul(thi[tt >> 6], tlo[tt & (kTwLo - 1)]);
    if (upper) w = make_float2(-w.x, -w.y);
    if (inverse) w.y = -w.y;
    return w;
}

// M-point complex FFT (M a power of two) in LDS, Stockham autosort between
// buffers a and b: radix-4 stages, then one radix-2 stage if log2 M is odd;
// sign -1 (forward) or +1 (inverse, unnormalised).  A stage combining
// sub-transforms of length Ls reads a[j + r M / R] (r < R), twiddles input
// r by exp(-/+ 2 pi i r k / (R Ls)) with k = j mod Ls, takes the R-point DFT
// and writes output s to b[R (j - k) + k + s Ls].  Returns the buffer with
// the result.
__device__ __forceinline__ float2* fft_lds(float2* a, float2* b, int M, const float2* __restrict__ thi,
                                          const float2* __restrict__ tlo, bool inverse) {
    int Ls = 1;
    const int q = M >> 2;
    for (; 4 * Ls <= M; Ls <<= 2) {
        const int tstep = M / (2 * Ls);
        for (int j = threadIdx.x; j < q; j += blockDim.x) {
            const int k = j & (Ls - 1);
            const int t = k * tstep;
            const float2 v0 = a[j];
            const float2 v1 = cmul(a[j + q], tw_at(thi, tlo, t, M, inverse));
            const float2 v2 = cmul(a[j + 2 * q], tw_at(thi, tlo, 2 * t, M, inverse));
            const float2 v3 = cmul(a[j + 3 * q], tw_at(thi, tlo, 3 * t, M, inverse));
            const float2 s02 = cadd(v0, v2), d02 = csub(v0, v2);
            const float2 s13 = cadd(v1, v3), d13 = csub(v1, v3);
            // -i d13 (forward) or +i d13 (inverse)
            const float2 jd13 = inverse ? make_float2(-d13.y, d13.x) : make_float2(d13.y, -d13.x);
            const int o = ((j - k) << 2) + k;
            b[o] = cadd(s02, s13);
            b[o + Ls] = cadd(d02, jd13);
            b[o + 2 * Ls] = csub(s02, s13);
            b[o + 3 * Ls] = csub(d02, jd13);
        }
        __syncthreads();
        float2* tmp = a;
        a = b;
        b = tmp;
    }
    if (2 * Ls == M) {
        const int half = M >> 1, tstep = M / Ls;
        for (int j = threadIdx.x; j < half; j += blockDim.x) {
            const int k = j & (Ls - 1);
            const float2 c0 = a[j];
            const float2 c1 = cmul(a[j + half], tw_at(thi, tlo, k * tstep, M, inverse));
            const int o = ((j - k) << 1) + k;
            b[o] = cadd(c0, c1);
            b[o + Ls] = csub(c0, c1);
        }
        __syncthreads();
        float2* tmp = a;
        a = b;
        b = tmp;
    }
    return a;
}

// Xhat[slot][b][ci][m], m in [0, M]: real DFT of ring slot_ring[slot] of x,
// the bins 0 < m < M multiplied by `interior` (2 gives the weights of a sum
// over the whole spectrum of a real signal, for Parseval's identity).
// grid: (n_slots, B * Ci)
template <typename T>
__global__ __launch_bounds__(kFftBlock) void k_rfft_rings(const int32_t* __restrict__ slot_ring,
                                                         const T* __restrict__ x, const float2* __restrict__ tw,
                                                         float2* __restrict__ xh, int B, int Ci, int nlat, int M,
                                                         float interior) {
    extern __shared__ float2 sm[];
    float2* a = sm;
    float2* bb = sm + M;
    float2* tlo = sm + 2 * M;
    float2* thi = tlo + kTwLo;
    const int slot = blockIdx.x;
    const int b = blockIdx.y / Ci, ci = blockIdx.y - (blockIdx.y / Ci) * Ci;
    const int N = 2 * M;
    const T* row = x + (((int64_t)b * Ci + ci) * nlat + slot_ring[slot]) * N;
    // Loads in batches of kFftBatch per thread, all issued before the LDS
    // writes (a loop with a run-time trip count would otherwise wait for
    // each load in turn).
    load_twiddles(tw, thi, tlo, M);
    for (int j0 = threadIdx.x; j0 < M; j0 += kFftBatch * kFftBlock) {
        float2 v[kFftBatch];
#pragma unroll
        for (int u = 0; u < kFftBatch; ++u) {
            const int j = j0 + u * kFftBlock;
            if (j < M) v[u] = make_float2(load_val(row, 2 * j), load_val(row, 2 * j + 1));
        }
#pragma unroll
        for (int u = 0; u < kFftBatch; ++u) {
            const int j = j0 + u * kFftBlock;
            if (j < M) a[j] = v[u];
        }
    }
    __syncthreads();
    const float2* Z = fft_lds(a, bb, M, thi, tlo, false);
    float2* out = xh + (((int64_t)slot * B + b) * Ci + ci) * (M + 1);
    for (int m = threadIdx.x; m <= M; m += blockDim.x) {
        const float2 zm = Z[m & (M - 1)];
        const float2 zc = conjf2(Z[(M - m) & (M - 1)]);
        const float2 e = make_float2(0.5f * (zm.x + zc.x), 0.5f * (zm.y + zc.y));
        const float2 dif = csub(zm, zc);
        const float2 o = make_float2(0.5f * dif.y, -0.5f * dif.x);  // (zm - zc) / (2i)
        const float2 w = tw_at(thi, tlo, m, M, false);  // m = M gives -1
        const float2 v = cadd(e, cmul(w, o));
        const float sc = m == 0 || m == M ? 1.0f : interior;
        out[m] = make_float2(sc * v.x, sc * v.y);
    }
}

// Yhat[h][b][co][m] for heavy ring h.  grid: (ceil((M+1)/BLK), n_rings, B * n_cotiles)
template <typename T, int COT, int BLK>
__global__ __launch_bounds__(BLK) void k_spectral(const int32_t* __restrict__ pair_ptr,
                                                       const int32_t* __restrict__ pair_slot,
                                                       const int32_t* __restrict__ pair_tab,
                                                       const float* __restrict__ vs,
                                                       const float2* __restrict__ xh,
                                                       const T* __restrict__ w, float2* __restrict__ yh,
                                                       int B, int Ci, int Co, int M, int n_cotiles,
                                                       bool w_trans) {
    // Input channels per accumulation pass.
    static_assert(COT <= 32, "output tiles of at most 32 channels");
    constexpr int SC = 4;
    // This pass's weights as (W_3a + W_3a+2, W_3a+2 - W_3a, W_3a+1) for each
    // (input channel, output channel, a), staged in LDS and read back by
    // broadcast (as uniform scalar loads they would need more SGPRs than
    // there are and spill).
    __shared__ float wsd[SC * COT * 9];
    const int m = blockIdx.x * BLK + threadIdx.x;
    const int h = blockIdx.y;
    const int b = blockIdx.z / n_cotiles;
    const int co0 = (blockIdx.z - b * n_cotiles) * COT;
    const bool active = m <= M;  // lanes past M still take part in the barriers
    const int p0 = pair_ptr[h], p1 = pair_ptr[h + 1];
    const int64_t vstride = (int64_t)(M + 1);
    float2 Y[COT];
#pragma unroll
    for (int j = 0; j < COT; ++j) Y[j] = make_float2(0.0f, 0.0f);
    for (int ci0 = 0; ci0 < Ci; ci0 += SC) {
        __syncthreads();  // the previous pass's reads of wsd are done
        for (int idx = threadIdx.x; idx < SC * COT * 3; idx += BLK) {
            const int c = idx / (COT * 3), r = idx - c * (COT * 3), j = r / 3, a = r - j * 3;
            const int ci = ci0 + c < Ci ? ci0 + c : Ci - 1;  // E, F, G are zero past Ci
            const int co = co0 + j < Co ? co0 + j : Co - 1;
            const int64_t base = w_trans ? ((int64_t)ci * Co + co) * kBasis : ((int64_t)co * Ci + ci) * kBasis;
            const float w0 = load_val(w, base + 3 * a), w1 = load_val(w, base + 3 * a + 1),
                        w2 = load_val(w, base + 3 * a + 2);
            wsd[3 * idx + 0] = w0 + w2;
            wsd[3 * idx + 1] = w2 - w0;
            wsd[3 * idx + 2] = w1;
        }
        __syncthreads();
        if (!active) continue;
        float2 E[SC][3], F[SC][3], G[SC][3];
#pragma unroll
        for (int c = 0; c < SC; ++c)
#pragma unroll
            for (int a = 0; a < 3; ++a) {
                E[c][a] = make_float2(0.0f, 0.0f);
                F[c][a] = make_float2(0.0f, 0.0f);
                G[c][a] = make_float2(0.0f, 0.0f);
            }
        for (int p = p0; p < p1; ++p) {
            // The pair's table; an equator mirror reads its rows a = 0 and
            // a = 2 exchanged.
            const int32_t tb = pair_tab[p];
            const int r0 = tb < 0 ? 6 : 0;
            const float* v = vs + (int64_t)(tb & 0x7fffffff) * 9 * vstride + m;
            float V[9];
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                V[j] = v[(r0 + j) * vstride];
                V[3 + j] = v[(3 + j) * vstride];
                V[6 + j] = v[(6 - r0 + j) * vstride];
            }
            const float2* xr = xh + (((int64_t)pair_slot[p] * B + b) * Ci) * vstride + m;
#pragma unroll
            for (int c = 0; c < SC; ++c) {
                const float2 X = ci0 + c < Ci ? xr[(int64_t)(ci0 + c) * vstride] : make_float2(0.0f, 0.0f);
#pragma unroll
                for (int a = 0; a < 3; ++a) {
                    E[c][a].x = fmaf(V[3 * a + 0], X.x, E[c][a].x);
                    E[c][a].y = fmaf(V[3 * a + 0], X.y, E[c][a].y);
                    F[c][a].x = fmaf(V[3 * a + 1], X.x, F[c][a].x);
                    F[c][a].y = fmaf(V[3 * a + 1], X.y, F[c][a].y);
                    G[c][a].x = fmaf(V[3 * a + 2], X.x, G[c][a].x);
                    G[c][a].y = fmaf(V[3 * a + 2], X.y, G[c][a].y);
                }
            }
        }
        // Yhat[co] += sum_{c,a} (W_3a + W_3a+2) E + i (W_3a+2 - W_3a) F + W_3a+1 G
#pragma unroll
        for (int j = 0; j < COT; ++j) {
#pragma unroll
            for (int c = 0; c < SC; ++c) {
#pragma unroll
                for (int a = 0; a < 3; ++a) {
                    const float* wd = wsd + 3 * ((c * COT + j) * 3 + a);
                    const float S = wd[0], D = wd[1], w1 = wd[2];
                    Y[j].x = fmaf(S, E[c][a].x, fmaf(-D, F[c][a].y, fmaf(w1, G[c][a].x, Y[j].x)));
                    Y[j].y = fmaf(S, E[c][a].y, fmaf(D, F[c][a].x, fmaf(w1, G[c][a].y, Y[j].y)));
                }
            }
        }
    }
    if (!active) return;
#pragma unroll
    for (int j = 0; j < COT; ++j)
        if (co0 + j < Co) yh[(((int64_t)h * B + b) * Co + co0 + j) * vstride + m] = Y[j];
}

// The gathered sums of the heavy rings in the frequency domain: the products
// of k_spectral without the channel contraction, Zhat[h][b][ci * 9 + k][m] =
// sum over the ring's pairs of Xhat[slot][ci][m] conj(Vhat_k[pair][m]), the
// nine planes of each input channel from the same E, F, G sums (k = 3a:
// E - iF, 3a + 1: G, 3a + 2: E + iF in the conjugate convention of
// k_spectral).  grid: (ceil((M+1)/256), n_rings, B * ceil(Ci / 4))
__global__ __launch_bounds__(kFftBlock) void k_spectral_z(const int32_t* __restrict__ pair_ptr,
                                                         const int32_t* __restrict__ pair_slot,
                                                         const int32_t* __restrict__ pair_tab,
                                                         const float* __restrict__ vs,
                                                         const float2* __restrict__ xh, float2* __restrict__ zh,
                                                         int B, int Ci, int M, int n_cg) {
    constexpr int SC = 4;
    const int m = blockIdx.x * kFftBlock + threadIdx.x;
    if (m > M) return;  // no barriers below
    const int h = blockIdx.y;
    const int b = blockIdx.z / n_cg;
    const int ci0 = (blockIdx.z - b * n_cg) * SC;
    const int p0 = pair_ptr[h], p1 = pair_ptr[h + 1];
    const int64_t vstride = (int64_t)(M + 1);
    float2 E[SC][3], F[SC][3], G[SC][3];
#pragma unroll
    for (int c = 0; c < SC; ++c)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            E[c][a] = make_float2(0.0f, 0.0f);
            F[c][a] = make_float2(0.0f, 0.0f);
            G[c][a] = make_float2(0.0f, 0.0f);
        }
    for (int p = p0; p < p1; ++p) {
        const int32_t tb = pair_tab[p];
        const int r0 = tb < 0 ? 6 : 0;
        const float* v = vs + (int64_t)(tb & 0x7fffffff) * 9 * vstride + m;
        float V[9];
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            V[j] = v[(r0 + j) * vstride];
            V[3 + j] = v[(3 + j) * vstride];
            V[6 + j] = v[(6 - r0 + j) * vstride];
        }
        const float2* xr = xh + (((int64_t)pair_slot[p] * B + b) * Ci) * vstride + m;
#pragma unroll
        for (int c = 0; c < SC; ++c) {
            const float2 X = ci0 + c < Ci ? xr[(int64_t)(ci0 + c) * vstride] : make_float2(0.0f, 0.0f);
#pragma unroll
            for (int a = 0; a < 3; ++a) {
                E[c][a].x = fmaf(V[3 * a + 0], X.x, E[c][a].x);
                E[c][a].y = fmaf(V[3 * a + 0], X.y, E[c][a].y);
                F[c][a].x = fmaf(V[3 * a + 1], X.x, F[c][a].x);
                F[c][a].y = fmaf(V[3 * a + 1], X.y, F[c][a].y);
                G[c][a].x = fmaf(V[3 * a + 2], X.x, G[c][a].x);
                G[c][a].y = fmaf(V[3 * a + 2], X.y, G[c][a].y);
            }
        }
    }
    const int Co = Ci * kBasis;
#pragma unroll
    for (int c = 0; c < SC; ++c) {
        if (ci0 + c >= Ci) continue;
        float2* zr = zh + (((int64_t)h * B + b) * Co + (int64_t)(ci0 + c) * kBasis) * vstride + m;
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            zr[(3 * a + 0) * vstride] = make_float2(E[c][a].x + F[c][a].y, E[c][a].y - F[c][a].x);
            zr[(3 * a + 1) * vstride] = G[c][a];
            zr[(3 * a + 2) * vstride] = make_float2(E[c][a].x - F[c][a].y, E[c][a].y + F[c][a].x);
        }
    }
}

// y[b][co][ring][:] = inverse real DFT of Yhat[h][b][co][:].  grid: (n_rings, B * Co)
template <typename T>
__global__ __launch_bounds__(kFftBlock) void k_irfft_rings(const int32_t* __restrict__ rings,
                                                          const float2* __restrict__ yh,
                                                          const float2* __restrict__ tw, T* __restrict__ y,
                                                          int B, int Co, int nlat_o, int M) {
    extern __shared__ float2 sm[];
    float2* a = sm;
    float2* bb = sm + M;
    float2* tlo = sm + 2 * M;
    float2* thi = tlo + kTwLo;
    const int h = blockIdx.x;
    const int b = blockIdx.y / Co, co = blockIdx.y - (blockIdx.y / Co) * Co;
    const float2* Y = yh + (((int64_t)h * B + b) * Co + co) * (M + 1);
    load_twiddles(tw, thi, tlo, M);
    for (int m0 = threadIdx.x; m0 < M; m0 += kFftBatch * kFftBlock) {
        float2 xm[kFftBatch], xc[kFftBatch], twm[kFftBatch];
#pragma unroll
        for (int u = 0; u < kFftBatch; ++u) {
            const int m = m0 + u * kFftBlock;
            if (m < M) {
                xm[u] = Y[m];
                xc[u] = conjf2(Y[M - m]);
                twm[u] = tw[m];
            }
        }
#pragma unroll
        for (int u = 0; u < kFftBatch; ++u) {
            const int m = m0 + u * kFftBlock;
            if (m < M) {
                const float2 e = cadd(xm[u], xc[u]);
                const float2 o = cmul(csub(xm[u], xc[u]), conjf2(twm[u]));
                a[m] = make_float2(e.x - o.y, e.y + o.x);  // e + i o
            }
        }
    }
    __syncthreads();
    const float2* z = fft_lds(a, bb, M, thi, tlo, true);
    const int N = 2 * M;
    const int64_t base = (((int64_t)b * Co + co) * nlat_o + rings[h]) * N;
    for (int j = threadIdx.x; j < M; j += blockDim.x) {
        const float2 v = z[j];
        store_val(y, base + 2 * j, v.x);
        store_val(y, base + 2 * j + 1, v.y);
    }
}

template <typename T, int COT, int BLK = kFftBlock>
hipError_t spectral_launch(const ExecArgs& a, float* ws, int stages) {
    const SpectralDev& S = a.op->spectral;
    const OpGeom& g = a.op->g;
    const int M = S.M;
    float2* xh = (float2*)ws;
    float2* yh = xh + (size_t)S.n_slots * a.B * a.Ci * (M + 1);
    const size_t lds = sizeof(float2) * (2 * (size_t)M + kTwLo + tw_hi_len(M));  // two FFT buffers, twiddle tables
    if (stages & 1) {
        const int tk = timing_begin("spectral_rfft", a.stream);
        hipLaunchKernelGGL((k_rfft_rings<T>), dim3(S.n_slots, a.B * a.Ci), dim3(kFftBlock), lds, a.stream,
                           S.slot_ring, (const T*)a.x, (const float2*)S.tw, xh, a.B, a.Ci, g.nlat_i, M, 1.0f);
        timing_end(tk, a.stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if ((stages & 2) && (stages & kSpectralZ)) {
        // a.Co = a.Ci * 9: the planes of every input channel, no W.
        const int n_cg = (a.Ci + 3) / 4;
        const int tk = timing_begin("spectral_mac", a.stream);
        hipLaunchKernelGGL(k_spectral_z, dim3((M + 1 + kFftBlock - 1) / kFftBlock, S.n_rings, a.B * n_cg),
                           dim3(kFftBlock), 0, a.stream, S.pair_ptr, S.pair_slot, S.pair_tab, S.vs, xh, yh, a.B, a.Ci,
                           M, n_cg);
        timing_end(tk, a.stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    } else if (stages & 2) {
        const int n_cot = (a.Co + COT - 1) / COT;
        const int tk = timing_begin("spectral_mac", a.stream);
        hipLaunchKernelGGL((k_spectral<T, COT, BLK>), dim3((M + 1 + BLK - 1) / BLK, S.n_rings, a.B * n_cot),
                           dim3(BLK), 0, a.stream, S.pair_ptr, S.pair_slot, S.pair_tab, S.vs, xh, (const T*)a.w, yh,
                           a.B, a.Ci, a.Co, M, n_cot, a.w_trans);
        timing_end(tk, a.stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (stages & 4) {
        const int tk = timing_begin("spectral_irfft", a.stream);
        hipLaunchKernelGGL((k_irfft_rings<T>), dim3(S.n_rings, a.B * a.Co), dim3(kFftBlock), lds, a.stream,
                           S.rings, yh, (const float2*)S.tw, (T*)a.y, a.B, a.Co, g.nlat_o, M);
        timing_end(tk, a.stream);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <typename T>
hipError_t spectral_dispatch(const ExecArgs& a, float* ws, int stages) {
    // Output channels in tiles of at most 8: wider tiles leave too few
    // workgroups (512 x 1024, 32 -> 32 channels: 240 with tiles of 32, the
    // products 207 -> 136 us with tiles of 8, where each tile redoes the
    // cheap per-pair sums).
    if (a.Co <= 4) return spectral_launch<T, 4>(a, ws, stages);
    if (a.Co <= 8 || (stages & kSpectralZ)) return spectral_launch<T, 8>(a, ws, stages);
    // More output channels: one tile of up to 32 (the per-pair sums done
    // once), the frequencies in workgroups of 64 so that they still fill
    // the chip.
    if (a.Co <= 32) return spectral_launch<T, 32, 64>(a, ws, stages);
    return spectral_launch<T, 8>(a, ws, stages);
}

}  // namespace

size_t workspace_bytes_spectral(const ExecArgs& a) {
    const SpectralDev& S = a.op->spectral;
    if (S.n_rings == 0) return 0;
    return sizeof(float2) * (size_t)(S.M + 1) * a.B * ((size_t)S.n_slots * a.Ci + (size_t)S.n_rings * a.Co);
}

float2* spectral_yhat(const ExecArgs& a, float* ws) {
    const SpectralDev& S = a.op->spectral;
    return (float2*)ws + (size_t)S.n_slots * a.B * a.Ci * (S.M + 1);
}

size_t spectral_dyhat_bytes(const ExecArgs& a, int C) {
    const SpectralDev& S = a.op->spectral;
    return sizeof(float2) * (size_t)S.n_rings * a.B * C * (S.M + 1);
}

hipError_t launch_spectral_dyhat(const ExecArgs& a, const float* dy, int C, float2* dyh) {
    const SpectralDev& S = a.op->spectral;
    if (S.n_rings == 0) return hipSuccess;
    const int M = S.M;
    const size_t lds = sizeof(float2) * (2 * (size_t)M + kTwLo + tw_hi_len(M));
    const int tk = timing_begin("spectral_rfft_dy", a.stream);
    hipLaunchKernelGGL((k_rfft_rings<float>), dim3(S.n_rings, a.B * C), dim3(kFftBlock), lds, a.stream, S.rings, dy,
                       (const float2*)S.tw, dyh, a.B, C, a.op->g.nlat_o, M, 2.0f);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

hipError_t launch_spectral(const ExecArgs& a, float* ws, int stages) {
    if (a.op->spectral.n_rings == 0) return hipSuccess;
    return a.dtype == 1 ? spectral_dispatch<uint16_t>(a, ws, stages) : spectral_dispatch<float>(a, ws, stages);
}

}  // namespace disco
