// disco_kernels.hip -- gfx950 kernels of the DISCO forward and transposed ops.
//
// The sparse-dense product of Sec. 4.1, in the compressed form of Sec. 4.2
// (eq. 9): each output ring r_o (and longitude phase) owns
// one list of (input ring, longitude offset, 9 values) entries; the output at
// longitude q reads the input at (stride * q + offset) mod nlon.  Lanes of a
// wavefront own consecutive output longitudes, so every entry is one
// wave-uniform set of 9 scalars applied to a contiguous, coalesced row
// segment of the input; the reduction order over entries is the same for
// every output longitude, which makes whole-pixel longitude shifts commute
// with the op bitwise.
//
// Two orderings of the channel contraction:
//   gather-then-contract:  Z[b,ci,k,n_o] = sum_e v_k x[b,ci,pix_e]
//                          y[b,co,n_o]   = sum_{ci,k} W[co,ci,k] Z[b,ci,k,n_o]
//   contract-then-gather:  X[b,co,k,n_i] = sum_ci W[co,ci,k] x[b,ci,n_i]
//                          y[b,co,n_o]   = sum_e sum_k v_k X[b,co,k,pix_e]
// The second moves the channel mixing to the coarser grid when the op
// upsamples.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "disco_internal.h"

namespace disco {

namespace {

constexpr int kBlock = 256;

// Storage types: fp32, or bf16 held as raw uint16.
__device__ __forceinline__ float load_val(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_val(const uint16_t* p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

// fp32 -> bf16 with round-to-nearest-even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ void store_val(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_val(uint16_t* p, int64_t i, float v) { p[i] = to_bf16(v); }

// W element for (op output channel co, op input channel ci, basis k):
// [Co][Ci][9] for the forward op, [Ci][Co][9] for the transposed op.
template <typename T>
__device__ __forceinline__ float w_at(const T* w, int co, int ci, int k, int Ci, int Co, bool w_trans) {
    const int64_t idx = w_trans ? ((int64_t)ci * Co + co) * kBasis + k : ((int64_t)co * Ci + ci) * kBasis + k;
    return load_val(w, idx);
}

// ---------------------------------------------------------------------------
// Gather of x into Z (9 planes per input channel).
// grid: (ceil(nq / 256), number of patterns, B * ceil(C / CG)); one lane per
// output longitude q of the pattern's ring and phase; the patterns are all of
// them, or the list pat_list when it is given.
template <typename T, int CG>
__global__ __launch_bounds__(kBlock) void k_gather_z(const int32_t* __restrict__ pat_ptr,
                                                     const DevEntry* __restrict__ ent, OpGeom g,
                                                     const T* __restrict__ x, float* __restrict__ z,
                                                     int C, int n_cgroups, const int32_t* __restrict__ pat_list) {
    const int q = blockIdx.x * kBlock + threadIdx.x;
    const int pat = pat_list ? pat_list[blockIdx.y] : (int)blockIdx.y;
    const int b = blockIdx.z / n_cgroups;
    const int c0 = (blockIdx.z % n_cgroups) * CG;
    if (q >= g.nq) return;
    const int to = pat / g.P, r = pat - to * g.P;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const int base = g.stride * q;
    float acc[CG][kBasis];
#pragma unroll
    for (int c = 0; c < CG; ++c)
#pragma unroll
        for (int k = 0; k < kBasis; ++k) acc[c][k] = 0.0f;
    const int e0 = pat_ptr[pat], e1 = pat_ptr[pat + 1];
    for (int e = e0; e < e1; ++e) {
        const DevEntry E = ent[e];
        int idx = base + E.d;
        if (idx >= g.nlon_i) idx -= g.nlon_i;
#pragma unroll
        for (int c = 0; c < CG; ++c) {
            const int cc = c0 + c < C ? c0 + c : C - 1;
            const float xv = load_val(x, ((int64_t)b * C + cc) * n_in + E.row + idx);
#pragma unroll
            for (int k = 0; k < kBasis; ++k) acc[c][k] = fmaf(E.v[k], xv, acc[c][k]);
        }
    }
    const int64_t pix = (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
#pragma unroll
    for (int c = 0; c < CG; ++c) {
        if (c0 + c < C) {
#pragma unroll
            for (int k = 0; k < kBasis; ++k)
                z[(((int64_t)b * C + c0 + c) * kBasis + k) * n_out + pix] = acc[c][k];
        }
    }
}

// Channel contraction of Z: y[b,co,n] = sum_{ci,k} W(co,ci,k) Z[b,ci,k,n],
// except on the output rings flagged in skip_ring (when given), whose y
// another kernel writes.  grid: (ceil(N / 256), B, ceil(Co / COT)).
template <typename T, int COT>
__global__ __launch_bounds__(kBlock) void k_contract_z(const float* __restrict__ z,
                                                       const T* __restrict__ w, T* __restrict__ y,
                                                       int Ci, int Co, int64_t N, bool w_trans,
                                                       const uint8_t* __restrict__ skip_ring, int nlon_o) {
    const int64_t n = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int b = blockIdx.y;
    const int co0 = blockIdx.z * COT;
    if (n >= N) return;
    if (skip_ring && skip_ring[n / nlon_o]) return;
    float acc[COT];
#pragma unroll
    for (int j = 0; j < COT; ++j) acc[j] = 0.0f;
    for (int ci = 0; ci < Ci; ++ci) {
#pragma unroll
        for (int k = 0; k < kBasis; ++k) {
            const float zv = z[(((int64_t)b * Ci + ci) * kBasis + k) * N + n];
#pragma unroll
            for (int j = 0; j < COT; ++j) {
                const int co = co0 + j < Co ? co0 + j : Co - 1;
                acc[j] = fmaf(w_at(w, co, ci, k, Ci, Co, w_trans), zv, acc[j]);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < COT; ++j) {
        if (co0 + j < Co) store_val(y, ((int64_t)b * Co + co0 + j) * N + n, acc[j]);
    }
}

// Channel contraction on the input grid: X[b,co,k,n] = sum_ci W(co,ci,k) x[b,ci,n].
// grid: (ceil(N / 256), B, ceil(Co * 9 / MT)).
template <typename T, int MT>
__global__ __launch_bounds__(kBlock) void k_contract_x(const T* __restrict__ x,
                                                       const T* __restrict__ w,
                                                       float* __restrict__ xc, int Ci, int Co,
                                                       int64_t N, bool w_trans) {
    const int64_t n = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int b = blockIdx.y;
    const int m0 = blockIdx.z * MT;
    const int M = Co * kBasis;
    if (n >= N) return;
    float acc[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) acc[j] = 0.0f;
    for (int ci = 0; ci < Ci; ++ci) {
        const float xv = load_val(x, ((int64_t)b * Ci + ci) * N + n);
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int m = m0 + j < M ? m0 + j : M - 1;
            acc[j] = fmaf(w_at(w, m / kBasis, ci, m % kBasis, Ci, Co, w_trans), xv, acc[j]);
        }
    }
#pragma unroll
    for (int j = 0; j < MT; ++j) {
        if (m0 + j < M) xc[((int64_t)b * M + m0 + j) * N + n] = acc[j];
    }
}

// Gather of the contracted planes: y[b,co,n_o] = sum_e sum_k v_k X[b,co,k,pix_e].
// grid: (ceil(nq / 256), n_patterns, B * ceil(Co / CG)).
template <typename T, int CG>
__global__ __launch_bounds__(kBlock) void k_gather_y(const int32_t* __restrict__ pat_ptr,
                                                     const DevEntry* __restrict__ ent, OpGeom g,
                                                     const float* __restrict__ xc,
                                                     T* __restrict__ y, int Co, int n_cgroups) {
    const int q = blockIdx.x * kBlock + threadIdx.x;
    const int pat = blockIdx.y;
    const int b = blockIdx.z / n_cgroups;
    const int c0 = (blockIdx.z % n_cgroups) * CG;
    if (q >= g.nq) return;
    const int to = pat / g.P, r = pat - to * g.P;
    const int64_t n_in = (int64_t)g.nlat_i * g.nlon_i;
    const int64_t n_out = (int64_t)g.nlat_o * g.nlon_o;
    const int base = g.stride * q;
    float acc[CG];
#pragma unroll
    for (int c = 0; c < CG; ++c) acc[c] = 0.0f;
    const int e0 = pat_ptr[pat], e1 = pat_ptr[pat + 1];
    for (int e = e0; e < e1; ++e) {
        const DevEntry E = ent[e];
        int idx = base + E.d;
        if (idx >= g.nlon_i) idx -= g.nlon_i;
#pragma unroll
        for (int c = 0; c < CG; ++c) {
            const int cc = c0 + c < Co ? c0 + c : Co - 1;
            const float* plane = xc + ((int64_t)b * Co + cc) * kBasis * n_in + E.row + idx;
#pragma unroll
            for (int k = 0; k < kBasis; ++k) acc[c] = fmaf(E.v[k], plane[k * n_in], acc[c]);
        }
    }
    const int64_t pix = (int64_t)to * g.nlon_o + (int64_t)q * g.P + r;
#pragma unroll
    for (int c = 0; c < CG; ++c) {
        if (c0 + c < Co) store_val(y, ((int64_t)b * Co + c0 + c) * n_out + pix, acc[c]);
    }
}

// The gather writes Z for every pattern the contraction then reads.  When
// the op has sweep runs (gather_z_split), the sweep kernel's Z mode gathers
// the patterns it covers, k_gather_z the light ones it does not, and the
// heavy polar rings, whose windows are whole rings (a Z there would take nine
// inverse FFTs per input channel and ring), keep the spectral path, which
// writes their y; the contraction skips those rings.
template <typename T>
hipError_t gather_then_contract(const ExecArgs& a, float* z, float* spec_ws) {
    const OpGeom& g = a.op->g;
    const DeviceOp& op = *a.op;
    const bool split = gather_z_split(a);
    constexpr int CG = 4;
    const int ncg = (a.Ci + CG - 1) / CG;
    hipError_t e = hipSuccess;
    if (split) {
        e = launch_sweep_z(a, z);
        if (e != hipSuccess) return e;
        if (op.n_rest_pats > 0) {
            dim3 grid1((g.nq + kBlock - 1) / kBlock, op.n_rest_pats, a.B * ncg);
            const int tk = timing_begin("gather_z", a.stream);
            hipLaunchKernelGGL((k_gather_z<T, CG>), grid1, dim3(kBlock), 0, a.stream, op.pat_ptr, op.entries, g,
                               (const T*)a.x, z, a.Ci, ncg, (const int32_t*)op.rest_pats);
            timing_end(tk, a.stream);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    } else {
        dim3 grid1((g.nq + kBlock - 1) / kBlock, g.n_patterns(), a.B * ncg);
        const int tk = timing_begin("gather_z", a.stream);
        hipLaunchKernelGGL((k_gather_z<T, CG>), grid1, dim3(kBlock), 0, a.stream, op.pat_ptr, op.entries, g,
                           (const T*)a.x, z, a.Ci, ncg, (const int32_t*)nullptr);
        timing_end(tk, a.stream);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t N = (int64_t)g.nlat_o * g.nlon_o;
    constexpr int COT = 8;
    dim3 grid2((unsigned)((N + kBlock - 1) / kBlock), a.B, (a.Co + COT - 1) / COT);
    const int tk = timing_begin("contract_z", a.stream);
    const uint8_t* skip = split && op.spectral.n_rings > 0 ? op.spectral_ring : nullptr;
    hipLaunchKernelGGL((k_contract_z<T, COT>), grid2, dim3(kBlock), 0, a.stream, z,
                       (const T*)a.w, (T*)a.y, a.Ci, a.Co, N, a.w_trans, skip, g.nlon_o);
    timing_end(tk, a.stream);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (skip) e = launch_spectral(a, spec_ws);
    return e;
}

template <typename T>
hipError_t contract_then_gather(const ExecArgs& a, float* xc) {
    const OpGeom& g = a.op->g;
    const int64_t N = (int64_t)g.nlat_i * g.nlon_i;
    constexpr int MT = 9;
    dim3 grid1((unsigned)((N + kBlock - 1) / kBlock), a.B, (a.Co * kBasis + MT - 1) / MT);
    int tk = timing_begin("contract_x", a.stream);
    hipLaunchKernelGGL((k_contract_x<T, MT>), grid1, dim3(kBlock), 0, a.stream, (const T*)a.x,
                       (const T*)a.w, xc, a.Ci, a.Co, N, a.w_trans);
    timing_end(tk, a.stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int CG = 4;
    const int ncg = (a.Co + CG - 1) / CG;
    dim3 grid2((g.nq + kBlock - 1) / kBlock, g.n_patterns(), a.B * ncg);
    tk = timing_begin("gather_y", a.stream);
    hipLaunchKernelGGL((k_gather_y<T, CG>), grid2, dim3(kBlock), 0, a.stream, a.op->pat_ptr,
                       a.op->entries, g, xc, (T*)a.y, a.Co, ncg);
    timing_end(tk, a.stream);
    return hipGetLastError();
}

}  // namespace

static size_t z_bytes(const ExecArgs& a) {
    const OpGeom& g = a.op->g;
    const size_t b = sizeof(float) * (size_t)a.B * a.Ci * kBasis * (size_t)g.nlat_o * g.nlon_o;
    return (b + 255) & ~(size_t)255;
}

bool gather_z_split(const ExecArgs& a) {
    // Z mode of the sweep: x channel groups and 36 Z planes addressed with
    // 32-bit buffer offsets.
    const OpGeom& g = a.op->g;
    const int64_t es = a.dtype == 1 ? 2 : 4;
    return a.op->sweep.n_runs > 0 && (int64_t)kCIC * g.nlat_i * g.nlon_i * es < ((int64_t)1 << 31) &&
           (int64_t)4 * kBasis * g.nlat_o * g.nlon_o * 4 < ((int64_t)1 << 31);
}

size_t workspace_bytes_gather_then_contract(const ExecArgs& a) {
    size_t b = z_bytes(a);
    if (gather_z_split(a) && a.op->spectral.n_rings > 0) b += workspace_bytes_spectral(a);
    return b;
}

size_t workspace_bytes_contract_then_gather(const ExecArgs& a) {
    const OpGeom& g = a.op->g;
    return sizeof(float) * (size_t)a.B * a.Co * kBasis * (size_t)g.nlat_i * g.nlon_i;
}

// The spectral rings' share of the gathered sums: the op's spectral kernels
// with Co = Ci * 9 output channels write the planes of Z directly (their
// products without the contraction).
static ExecArgs z_as_output(const ExecArgs& a, float* z) {
    ExecArgs s = a;
    s.w = nullptr;
    s.y = z;
    s.Co = a.Ci * kBasis;
    s.w_trans = false;
    return s;
}

size_t workspace_bytes_gather_z_all(const ExecArgs& a) {
    size_t b = 0;
    if (gather_z_split(a) && a.op->spectral.n_rings > 0) b = workspace_bytes_spectral(z_as_output(a, nullptr));
    return b;
}

static hipError_t gather_z_all(const ExecArgs& a, float* z, float* ws, int spectral_stages) {
    const OpGeom& g = a.op->g;
    const DeviceOp& op = *a.op;
    constexpr int CG = 4;
    const int ncg = (a.Ci + CG - 1) / CG;
    hipError_t e = hipSuccess;
    if (!gather_z_split(a)) {
        dim3 grid1((g.nq + kBlock - 1) / kBlock, g.n_patterns(), a.B * ncg);
        const int tk = timing_begin("gather_z", a.stream);
        hipLaunchKernelGGL((k_gather_z<float, CG>), grid1, dim3(kBlock), 0, a.stream, op.pat_ptr, op.entries, g,
                           (const float*)a.x, z, a.Ci, ncg, (const int32_t*)nullptr);
        timing_end(tk, a.stream);
        return hipGetLastError();
    }
    e = launch_sweep_z(a, z);
    if (e != hipSuccess) return e;
    if (op.n_rest_pats > 0) {
        dim3 grid1((g.nq + kBlock - 1) / kBlock, op.n_rest_pats, a.B * ncg);
        const int tk = timing_begin("gather_z", a.stream);
        hipLaunchKernelGGL((k_gather_z<float, CG>), grid1, dim3(kBlock), 0, a.stream, op.pat_ptr, op.entries, g,
                           (const float*)a.x, z, a.Ci, ncg, (const int32_t*)op.rest_pats);
        timing_end(tk, a.stream);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (op.spectral.n_rings == 0) return hipSuccess;
    return launch_spectral(z_as_output(a, z), ws, spectral_stages);
}

hipError_t launch_gather_z_all(const ExecArgs& a, float* z, float* ws) {
    return gather_z_all(a, z, ws, kSpectralAll | kSpectralZ);
}

hipError_t launch_gather_z_light(const ExecArgs& a, float* z, float* ws, float2** zhat) {
    *zhat = spectral_yhat(z_as_output(a, z), ws);
    return gather_z_all(a, z, ws, 1 | 2 | kSpectralZ);
}

hipError_t launch_gather_then_contract(const ExecArgs& a, float* z_ws) {
    float* spec_ws = (float*)((char*)z_ws + z_bytes(a));
    return a.dtype == 1 ? gather_then_contract<uint16_t>(a, z_ws, spec_ws) : gather_then_contract<float>(a, z_ws, spec_ws);
}

hipError_t launch_contract_then_gather(const ExecArgs& a, float* xc_ws) {
    return a.dtype == 1 ? contract_then_gather<uint16_t>(a, xc_ws) : contract_then_gather<float>(a, xc_ws);
}

}  // namespace disco
