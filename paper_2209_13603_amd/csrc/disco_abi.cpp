// disco_abi.cpp -- the C ABI of libdisco.so (declared in include/disco.h):
// argument validation, plan construction and upload, workspace management
// and dispatch to the kernels.  Validation is synchronous and happens before
// anything is enqueued; a failed call enqueues nothing.
#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>

#include "disco.h"
#include "disco_internal.h"

using namespace disco;

namespace {

// A roctx range around a library call (plan creation, an op, a gradient),
// seen by rocprofv3 --marker-trace; without a profiler it costs a call.
struct TraceRange {
    explicit TraceRange(const char* name) { roctxRangePushA(name); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange&) = delete;
    TraceRange& operator=(const TraceRange&) = delete;
};

// DISCO_LOG=1 in the environment: plan statistics on stderr.
bool log_enabled() {
    static const bool on = [] {
        const char* v = std::getenv("DISCO_LOG");
        return v && v[0] && std::strcmp(v, "0") != 0;
    }();
    return on;
}

void log_host_op(const char* name, const HostOp& h) {
    const OpGeom& g = h.g;
    const int K = basis_size(h.basis);
    const double compressed = (double)h.t_in.size() * (8 + 4 * K) + 4.0 * (double)h.pat_ptr.size();
    std::fprintf(stderr,
                 "disco: %s op %dx%d -> %dx%d: %d patterns (%d rings x %d phases, stride %d), %lld stored entries, "
                 "%lld non-zero (pixel pair, k) triples, largest window %d entries, %d full-ring windows, "
                 "compressed psi %.2f MB\n",
                 name, g.nlat_i, g.nlon_i, g.nlat_o, g.nlon_o, g.n_patterns(), g.nlat_o, g.P, g.stride,
                 (long long)h.t_in.size(), (long long)h.nnz_pairs, h.max_window, h.full_ring_windows,
                 compressed / 1e6);
}

}  // namespace

struct disco_plan {
    int device = 0;
    PlanParams params{};
    disco_plan_info_t info{};
    DeviceOp fwd, tr;
    // DISCO_PLAN_BACKWARD: the adjoint of each op (the other op's filter pairs
    // weighted by the quadrature of the adjoint's output points, App. C) and
    // K x K identity weights in fp32 and bf16 (the selection W that makes an
    // op's kernels write its gathered sums Z).
    DeviceOp fwd_adj, tr_adj;
    void* wsel32 = nullptr;
    void* wsel16 = nullptr;
    hipStream_t aux = nullptr;  // runs the spectral rings beside the direct kernels
    hipStream_t aux_dw = nullptr;  // runs the weight gradient's pass beside the input gradient's
    std::mutex lazy_mu;         // serialises the uploads of layouts on first use
};

namespace {

thread_local std::string g_last_error;

disco_status_t fail(disco_status_t s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

disco_status_t ok() {
    g_last_error.clear();
    return DISCO_OK;
}

bool fault_inject_alloc() {
    const char* v = std::getenv("DISCO_FAULT_INJECT");
    return v && std::strcmp(v, "alloc") == 0;
}

disco_status_t hip_fail(hipError_t e, const char* what) {
    if (e == hipErrorOutOfMemory) return fail(DISCO_ERR_OUT_OF_MEMORY, std::string(what) + ": " + hipGetErrorString(e));
    return fail(DISCO_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

disco_status_t resolve_params(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double theta_c,
                              const disco_basis_t* basis, PlanParams* p) {
    if (nlat_in < 1 || nlat_out < 1 || nlon_in < 2 || nlon_out < 2)
        return fail(DISCO_ERR_INVALID_ARGUMENT, "grid sizes need nlat >= 1 and nlon >= 2");
    if ((int64_t)nlat_in * nlon_in > (1LL << 30) || (int64_t)nlat_out * nlon_out > (1LL << 30))
        return fail(DISCO_ERR_INVALID_ARGUMENT, "grid larger than 2^30 pixels");
    if (!(theta_c > 0.0) || !(theta_c <= 3.14159265358979323846) || !std::isfinite(theta_c))
        return fail(DISCO_ERR_INVALID_ARGUMENT, "theta_c must lie in (0, pi]");
    disco_basis_t b{DISCO_BASIS_BILINEAR_3X3, DISCO_QUAD_SAMPLING_THEOREM, 0.0, DISCO_SAMPLING_CELL_CENTRED, 0};
    if (basis) b = *basis;
    if ((b.flags & ~(DISCO_PLAN_BACKWARD | DISCO_PLAN_EAGER)) != 0)
        return fail(DISCO_ERR_INVALID_ARGUMENT, "unknown basis.flags bits");
    if (b.kind != DISCO_BASIS_BILINEAR_3X3 && b.kind != DISCO_BASIS_AXISYMMETRIC_4 &&
        b.kind != DISCO_BASIS_SEPARABLE_4X4)
        return fail(DISCO_ERR_UNSUPPORTED, "unknown basis kind");
    if (b.sampling != DISCO_SAMPLING_CELL_CENTRED && b.sampling != DISCO_SAMPLING_POLES)
        return fail(DISCO_ERR_UNSUPPORTED, "unknown sampling");
    if (b.quadrature != DISCO_QUAD_SAMPLING_THEOREM && b.quadrature != DISCO_QUAD_CELL_AREA)
        return fail(DISCO_ERR_UNSUPPORTED, "unknown quadrature");
    if (b.sampling == DISCO_SAMPLING_POLES) {
        if (b.quadrature != DISCO_QUAD_SAMPLING_THEOREM)
            return fail(DISCO_ERR_UNSUPPORTED, "the pole-including grid takes its sampling-theorem weights only");
        if (nlat_in < 2 || nlat_out < 2 || nlon_in != 2 * (nlat_in - 1) || nlon_out != 2 * (nlat_out - 1))
            return fail(DISCO_ERR_INVALID_ARGUMENT, "the pole-including grid needs nlat >= 2 and nlon = 2 (nlat - 1)");
    }
    if (!(b.node_spacing >= 0.0) || !std::isfinite(b.node_spacing))
        return fail(DISCO_ERR_INVALID_ARGUMENT, "node_spacing must be >= 0");
    if (nlon_in % nlon_out != 0 && nlon_out % nlon_in != 0)
        return fail(DISCO_ERR_UNSUPPORTED, "nlon_in / nlon_out or nlon_out / nlon_in must be an integer");
    // One pattern per (output ring, longitude phase) of each op; kernels put
    // patterns in a 16-bit grid dimension.
    const int64_t pat_fwd = (int64_t)nlat_out * (nlon_out % nlon_in == 0 ? nlon_out / nlon_in : 1);
    const int64_t pat_tr = (int64_t)nlat_in * (nlon_in % nlon_out == 0 ? nlon_in / nlon_out : 1);
    if (pat_fwd > 65535 || pat_tr > 65535)
        return fail(DISCO_ERR_UNSUPPORTED, "more than 65535 latitude rings x longitude phases in one op");
    p->nlat_in = nlat_in; p->nlon_in = nlon_in; p->nlat_out = nlat_out; p->nlon_out = nlon_out;
    p->theta_c = theta_c;
    const double h_default = b.kind == DISCO_BASIS_BILINEAR_3X3 ? theta_c / 3.0 : theta_c / 4.0;
    p->h = b.node_spacing > 0.0 ? b.node_spacing : h_default;
    p->quadrature = b.quadrature;
    p->basis = b.kind;
    p->sampling = b.sampling;
    p->flags = b.flags;
    return DISCO_OK;
}

template <typename V>
disco_status_t upload_vec(const std::vector<V>& v, V** dst, int64_t* bytes, const char* what) {
    const size_t n = sizeof(V) * std::max<size_t>(v.size(), 1);
    hipError_t e = hipMalloc((void**)dst, n);
    if (e != hipSuccess) { *dst = nullptr; return hip_fail(e, what); }
    if (!v.empty()) {
        e = hipMemcpy(*dst, v.data(), sizeof(V) * v.size(), hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(e, what);
    }
    *bytes += (int64_t)n;
    return DISCO_OK;
}

// Entries per work item of the fused kernel (balances workgroups): 512,
// and fewer on small ops, where the launch is a handful of workgroups and
// the longest one's serial chain of staging and gathering is the time
// (measured: 32 x 64, 4 -> 4 channels: 41.5 us at 512, 17.6 us at 64 with the
// 64-lane tile; 128 x 256 -> 64 x 128, 16 -> 16 channels: 112 us at 512, 71 us
// at 128).  Environment DISCO_FUSED_TARGET_ENTRIES overrides, for tuning.
constexpr int kTargetEntries = 512;
int fused_target_entries(const HostOp& h, int tile) {
    const char* v = std::getenv("DISCO_FUSED_TARGET_ENTRIES");
    if (v && *v) return std::max(16, std::atoi(v));
    if (tile == 64) return 64;
    const int64_t tiles = (h.g.nq + tile - 1) / tile;
    if ((int64_t)h.t_in.size() * tiles < 65536) return 128;
    return kTargetEntries;
}

// Output rings with at least this many entries take the spectral path
// (environment DISCO_SPECTRAL_MIN_ENTRIES overrides, for tuning).
int spectral_min_entries() {
    const char* v = std::getenv("DISCO_SPECTRAL_MIN_ENTRIES");
    if (v && *v) return std::max(1, std::atoi(v));
    return 128;
}

disco_status_t upload_spectral(const SpectralHost& S, SpectralDev* d) {
    disco_status_t s;
    if ((s = upload_vec(S.rings, &d->rings, &d->bytes, "hipMalloc(spectral rings)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.pair_ptr, &d->pair_ptr, &d->bytes, "hipMalloc(spectral pairs)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.pair_slot, &d->pair_slot, &d->bytes, "hipMalloc(spectral pairs)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.pair_tab, &d->pair_tab, &d->bytes, "hipMalloc(spectral pairs)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.slot_ring, &d->slot_ring, &d->bytes, "hipMalloc(spectral slots)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.vs, &d->vs, &d->bytes, "hipMalloc(spectral psi)")) != DISCO_OK) return s;
    if ((s = upload_vec(S.tw, &d->tw, &d->bytes, "hipMalloc(twiddles)")) != DISCO_OK) return s;
    d->N = S.N;
    d->M = S.M;
    d->n_rings = (int)S.rings.size();
    d->n_pairs = (int)S.pair_slot.size();
    d->n_slots = (int)S.slot_ring.size();
    d->n_tables = S.n_tables;
    return DISCO_OK;
}

void free_spectral(SpectralDev* d) {
    void* ptrs[] = {d->rings, d->pair_ptr, d->pair_slot, d->pair_tab, d->slot_ring, d->vs, d->tw};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    *d = SpectralDev{};
}

disco_status_t pack_general(const HostOp& h, const std::vector<uint8_t>& skip, PackedHost* P) {
    std::string err;
    // The narrowest tile that covers a pattern's output longitudes (64, 128
    // or 256): the general kernel's 256 threads then split each chunk's
    // entries between 4, 2 or 1 groups of lanes instead of idling.
    const int tile = h.g.nq <= 64 ? 64 : h.g.nq <= 128 ? 128 : kTileQ;
    int rc = pack_op(h, fused_target_entries(h, tile), skip, P, &err, tile);
    if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    return DISCO_OK;
}

disco_status_t upload_packed(const PackedHost& P, PackedDev* d) {
    disco_status_t s;
    if ((s = upload_vec(P.spans, &d->spans, &d->bytes, "hipMalloc(spans)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.chunks, &d->chunks, &d->bytes, "hipMalloc(chunks)")) != DISCO_OK) return s;
    std::vector<int32_t> offs(P.entries.size());
    std::vector<PVal> vals(P.entries.size());
    for (size_t i = 0; i < P.entries.size(); ++i) {
        offs[i] = P.entries[i].off;
        for (int k = 0; k < 4; ++k) vals[i].v[k] = P.entries[i].v[k];
    }
    if ((s = upload_vec(offs, &d->offs, &d->bytes, "hipMalloc(entry offsets)")) != DISCO_OK) return s;
    if ((s = upload_vec(vals, &d->vals, &d->bytes, "hipMalloc(entry values)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.segs, &d->segs, &d->bytes, "hipMalloc(segments)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.items, &d->items, &d->bytes, "hipMalloc(items)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.red_pattern, &d->red_pattern, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.red_ptr, &d->red_ptr, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(P.red_slots, &d->red_slots, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    d->n_items = (int32_t)P.items.size();
    d->n_split = (int32_t)P.red_pattern.size();
    d->n_slots = P.n_slots;
    d->tile = P.tile;
    return DISCO_OK;
}

// Device bytes upload_packed would allocate (each table at least one element).
template <typename V>
int64_t vec_bytes(const std::vector<V>& v) { return (int64_t)(sizeof(V) * std::max<size_t>(v.size(), 1)); }
int64_t packed_bytes(const PackedHost& P) {
    const int64_t ne = (int64_t)std::max<size_t>(P.entries.size(), 1);
    return vec_bytes(P.spans) + vec_bytes(P.chunks) + ne * (int64_t)(sizeof(int32_t) + sizeof(PVal)) +
           vec_bytes(P.segs) + vec_bytes(P.items) + vec_bytes(P.red_pattern) + vec_bytes(P.red_ptr) +
           vec_bytes(P.red_slots);
}

// Cost of one sweep run (entries plus fixed per-pattern work).  The Z mode
// (all-HBM schedule) runs shorter runs: more workgroups keep more stores in
// flight (2048 x 4096, 8 channels: 520 us at 768, 502 us at 256), where the
// contracting sweep loses (357 -> 363 us at 512).
constexpr int kSweepTarget = 768;
constexpr int kSweepZTarget = 256;

disco_status_t upload_sweep(const SweepHost& H, SweepDev* d) {
    disco_status_t s;
    std::vector<int32_t> offs(H.entries.size());
    std::vector<PVal> vals(H.entries.size());
    for (size_t i = 0; i < H.entries.size(); ++i) {
        offs[i] = H.entries[i].off;
        for (int k = 0; k < 4; ++k) vals[i].v[k] = H.entries[i].v[k];
    }
    if ((s = upload_vec(H.runs, &d->runs, &d->bytes, "hipMalloc(sweep runs)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.pats, &d->pats, &d->bytes, "hipMalloc(sweep patterns)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.acts, &d->acts, &d->bytes, "hipMalloc(sweep spans)")) != DISCO_OK) return s;
    if ((s = upload_vec(offs, &d->offs, &d->bytes, "hipMalloc(sweep offsets)")) != DISCO_OK) return s;
    if ((s = upload_vec(vals, &d->vals, &d->bytes, "hipMalloc(sweep values)")) != DISCO_OK) return s;
    std::vector<int32_t> cov;
    for (size_t i = 0; i < H.covered.size(); ++i)
        if (H.covered[i]) cov.push_back((int32_t)i);
    if ((s = upload_vec(cov, &d->cov_pats, &d->bytes, "hipMalloc(sweep patterns)")) != DISCO_OK) return s;
    d->n_runs = (int32_t)H.runs.size();
    d->n_pats = (int32_t)H.pats.size();
    d->n_cov = (int32_t)cov.size();
    return DISCO_OK;
}

void free_sweep(SweepDev* d) {
    void* ptrs[] = {d->runs, d->pats, d->acts, d->offs, d->vals, d->cov_pats};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    *d = SweepDev{};
}

disco_status_t pack_stencil_host(const HostOp& h, StencilHost* H) {
    // Entries per work item: enough workgroups (items x longitude tiles) to
    // fill the chip several times over, within [128, 1024].
    // The tile: 512 output longitudes when a pattern has no more (two-phase
    // ops, small grids), so that no lanes idle; 1024 otherwise.
    const int tile = h.g.nq <= kStencilSmallTile ? kStencilSmallTile : kStencilTile;
    const int64_t n_qt = (h.g.nq + tile - 1) / tile;
    const int target = (int)std::min<int64_t>(1024, std::max<int64_t>(128, (int64_t)h.t_in.size() * n_qt / 4096));
    std::string err;
    int rc = pack_stencil(h, target, tile, H, &err);
    if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    return DISCO_OK;
}

disco_status_t upload_stencil(const StencilHost& H, StencilDev* d) {
    disco_status_t s;
    if ((s = upload_vec(H.pieces, &d->pieces, &d->bytes, "hipMalloc(stencil pieces)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.chunks, &d->chunks, &d->bytes, "hipMalloc(stencil chunks)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.vals, &d->vals, &d->bytes, "hipMalloc(stencil values)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.cells, &d->cells, &d->bytes, "hipMalloc(stencil cells)")) != DISCO_OK) return s;
    PackedDev& P = d->P;
    if ((s = upload_vec(H.segs, &P.segs, &d->bytes, "hipMalloc(segments)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.items, &P.items, &d->bytes, "hipMalloc(items)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.red_pattern, &P.red_pattern, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.red_ptr, &P.red_ptr, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.red_slots, &P.red_slots, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    P.n_items = (int32_t)H.items.size();
    P.n_split = (int32_t)H.red_pattern.size();
    P.n_slots = H.n_slots;
    d->tile = H.tile;
    d->n_padded = (int64_t)H.vals.size();
    return DISCO_OK;
}

int64_t stencil_bytes(const StencilHost& H) {
    return vec_bytes(H.pieces) + vec_bytes(H.chunks) + vec_bytes(H.vals) + vec_bytes(H.cells) + vec_bytes(H.segs) +
           vec_bytes(H.items) + vec_bytes(H.red_pattern) + vec_bytes(H.red_ptr) + vec_bytes(H.red_slots);
}

disco_status_t upload_mfma(const MfmaHost& H, MfmaDev* d) {
    disco_status_t s;
    if ((s = upload_vec(H.spans, &d->spans, &d->bytes, "hipMalloc(matrix-core spans)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.segs, &d->segs, &d->bytes, "hipMalloc(matrix-core segments)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.chunks, &d->chunks, &d->bytes, "hipMalloc(matrix-core chunks)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.aop, &d->aop, &d->bytes, "hipMalloc(matrix-core values)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.order, &d->order, &d->bytes, "hipMalloc(matrix-core order)")) != DISCO_OK) return s;
    PackedDev& P = d->P;
    if ((s = upload_vec(H.red_pattern, &P.red_pattern, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.red_ptr, &P.red_ptr, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    if ((s = upload_vec(H.red_slots, &P.red_slots, &d->bytes, "hipMalloc(reduce)")) != DISCO_OK) return s;
    d->n_segs = (int32_t)H.segs.size();
    d->n_order = (int32_t)H.order.size();
    d->n_qtiles = H.n_qtiles;
    P.n_items = d->n_segs;
    P.n_split = (int32_t)H.red_pattern.size();
    P.n_slots = H.n_slots;
    return DISCO_OK;
}

void free_mfma(MfmaDev* d) {
    void* ptrs[] = {d->spans, d->segs, d->chunks, d->aop, d->order, d->P.red_pattern, d->P.red_ptr, d->P.red_slots};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    *d = MfmaDev{};
}

void free_packed(PackedDev* d) {
    void* ptrs[] = {d->spans, d->chunks, d->offs, d->vals, d->segs, d->items, d->red_pattern, d->red_ptr, d->red_slots};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    *d = PackedDev{};
}

}  // namespace

namespace disco {

// Host tables of one op's layout groups (see kPart*), packed at plan
// creation and uploaded on first use.
struct OpTables {
    // kPartEntries: the plain entry tables.
    std::vector<int32_t> pat_ptr;
    std::vector<DevEntry> ent;
    // kPartDirect: the general kernel over every pattern.
    PackedHost packed;
    // kPartStencil (longitude stride 1): the blocked stencil layout.
    bool has_stencil = false;
    StencilHost stencil;
    // kPartCore (3x3 basis): spectral rings, their flags, the general kernel
    // for the light rings, the sweep and the general kernel for the rest.
    SpectralHost sp;
    std::vector<uint8_t> spectral_flag;
    bool has_light = false, has_sweep = false;
    PackedHost light, rest;
    SweepHost sw;
    SweepHost sw_z;  // kPartEntries: the Z mode's shorter runs (when there is a sweep)
    std::vector<int32_t> rest_pats;
    int64_t bytes[4] = {0, 0, 0, 0};  // device bytes of each group (core, direct, entries, stencil)
};

}  // namespace disco

namespace {

int part_index(int part) { return part == kPartCore ? 0 : part == kPartDirect ? 1 : part == kPartEntries ? 2 : 3; }

// Host side of one op: every group's tables packed, the op's metadata and
// work figures set, the cell map uploaded (64 bytes).  Nothing else on the
// device yet.
disco_status_t prepare_op(const HostOp& h, DeviceOp* d) {
    if (fault_inject_alloc()) return fail(DISCO_ERR_OUT_OF_MEMORY, "allocation failure injected (DISCO_FAULT_INJECT=alloc)");
    d->g = h.g;
    d->basis = h.basis;
    d->n_entries = (int64_t)h.t_in.size();
    d->nnz_pairs = h.nnz_pairs;
    d->work_all = pattern_work(h, {});
    auto T = std::make_shared<OpTables>();
    T->pat_ptr = h.pat_ptr;
    T->ent.resize((size_t)d->n_entries);
    for (int64_t e = 0; e < d->n_entries; ++e) {
        DevEntry& E = T->ent[(size_t)e];
        E.row = h.t_in[(size_t)e] * h.g.nlon_i;
        E.d = h.d[(size_t)e];
        for (int k = 0; k < kBasis; ++k) E.v[k] = h.val[(size_t)e * kBasis + k];
        E.pad = 0;
    }
    T->bytes[2] = vec_bytes(T->pat_ptr) + vec_bytes(T->ent);
    disco_status_t s;
    if ((s = pack_general(h, {}, &T->packed)) != DISCO_OK) return s;
    T->bytes[1] = packed_bytes(T->packed);
    // Every basis has the folded-weight stencil kernels (all calls of the
    // axisymmetric and separable bases, depthwise calls of any basis): the
    // general one on the packed layout, the blocked one when the longitude
    // stride is 1.  The spectral and sweep layouts are built for the 3x3 basis.
    if (h.g.stride == 1) {
        if ((s = pack_stencil_host(h, &T->stencil)) != DISCO_OK) return s;
        T->has_stencil = true;
        T->bytes[3] = stencil_bytes(T->stencil);
    }
    const CellMap cm = cell_map(h.basis);
    std::vector<int8_t> cmv(&cm.k[0][0], &cm.k[0][0] + sizeof(cm.k));
    if ((s = upload_vec(cmv, &d->cmap_dev, &d->bytes, "hipMalloc(cell map)")) != DISCO_OK) return s;
    if (h.basis != DISCO_BASIS_BILINEAR_3X3) {
        d->work_light = d->work_all;
        d->tables = T;
        d->built.store(kPartCore);  // nothing in the group for these bases
        return DISCO_OK;
    }
    std::vector<uint8_t> heavy;
    std::string err;
    int rc = build_spectral(h, spectral_min_entries(), &T->sp, &heavy, &err);
    if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    int64_t core = 0;
    if (!T->sp.rings.empty()) {
        T->spectral_flag.assign((size_t)h.g.nlat_o, 0);
        for (int32_t r : T->sp.rings) T->spectral_flag[(size_t)r] = 1;
        int32_t lo = 0, hi = h.g.nlat_o;
        while (lo < h.g.nlat_o && T->spectral_flag[(size_t)lo]) ++lo;
        while (hi > lo && T->spectral_flag[(size_t)hi - 1]) --hi;
        if (lo < hi && lo + (h.g.nlat_o - hi) == (int32_t)T->sp.rings.size()) {
            d->cap_lo = lo;
            d->cap_hi = hi;
        }
        if ((s = pack_general(h, heavy, &T->light)) != DISCO_OK) return s;
        T->has_light = true;
        core += vec_bytes(T->sp.rings) + vec_bytes(T->sp.pair_ptr) + vec_bytes(T->sp.pair_slot) +
                vec_bytes(T->sp.pair_tab) + vec_bytes(T->sp.slot_ring) + vec_bytes(T->sp.vs) + vec_bytes(T->sp.tw) + h.g.nlat_o +
                packed_bytes(T->light);
        std::vector<uint8_t> light(heavy.size());
        for (size_t i = 0; i < heavy.size(); ++i) light[i] = !heavy[i];
        d->work_spectral = pattern_work(h, heavy);
        d->work_light = pattern_work(h, light);
    } else {
        d->work_light = d->work_all;
    }
    // Sweep runs over the light patterns; the rest go to the general kernel.
    rc = pack_sweep(h, kSweepTarget, heavy, &T->sw, &err);
    if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    if (!T->sw.runs.empty()) {
        std::vector<uint8_t> rest_skip(T->sw.covered);
        for (size_t i = 0; i < rest_skip.size() && i < heavy.size(); ++i) rest_skip[i] |= heavy[i];
        if ((s = pack_general(h, rest_skip, &T->rest)) != DISCO_OK) return s;
        T->has_sweep = true;
        for (size_t i = 0; i < rest_skip.size(); ++i) rest_skip[i] = !rest_skip[i];
        d->work_sweep = pattern_work(h, T->sw.covered);
        d->work_rest = pattern_work(h, rest_skip);
        for (size_t i = 0; i < rest_skip.size(); ++i)
            if (rest_skip[i]) T->rest_pats.push_back((int32_t)i);
        int64_t cov = 0;
        for (uint8_t c : T->sw.covered) cov += c;
        auto sweep_bytes = [cov](const SweepHost& W) {
            const int64_t ne = (int64_t)std::max<size_t>(W.entries.size(), 1);
            return vec_bytes(W.runs) + vec_bytes(W.pats) + vec_bytes(W.acts) +
                   ne * (int64_t)(sizeof(int32_t) + sizeof(PVal)) + (int64_t)sizeof(int32_t) * std::max<int64_t>(cov, 1);
        };
        core += sweep_bytes(T->sw) + packed_bytes(T->rest) + (T->rest_pats.empty() ? 0 : vec_bytes(T->rest_pats));
        rc = pack_sweep(h, kSweepZTarget, heavy, &T->sw_z, &err);
        if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
        if (T->sw_z.covered != T->sw.covered) return fail(DISCO_ERR_DEVICE, "internal: sweep layouts cover different rings");
        T->bytes[2] += sweep_bytes(T->sw_z);
    }
    T->bytes[0] = core;
    d->tables = T;
    return DISCO_OK;
}

// Uploads the groups in `parts` that are not on the device yet (the caller
// holds the plan's lock, with the plan's device current).
disco_status_t upload_parts(DeviceOp* d, int parts) {
    const int todo = parts & ~d->built;
    if (!todo) return DISCO_OK;
    if (fault_inject_alloc()) return fail(DISCO_ERR_OUT_OF_MEMORY, "allocation failure injected (DISCO_FAULT_INJECT=alloc)");
    const OpTables* T = d->tables.get();
    if (!T) return fail(DISCO_ERR_DEVICE, "internal: layout tables released before upload");
    disco_status_t s;
    if (todo & kPartEntries) {
        if ((s = upload_vec(T->pat_ptr, &d->pat_ptr, &d->bytes_entries, "hipMalloc(pattern table)")) != DISCO_OK) return s;
        if ((s = upload_vec(T->ent, &d->entries, &d->bytes_entries, "hipMalloc(psi entries)")) != DISCO_OK) return s;
        if (T->has_sweep && (s = upload_sweep(T->sw_z, &d->sweep_z)) != DISCO_OK) return s;
        d->built.fetch_or(kPartEntries);
    }
    if (todo & kPartDirect) {
        if ((s = upload_packed(T->packed, &d->packed)) != DISCO_OK) return s;
        d->built.fetch_or(kPartDirect);
    }
    if (todo & kPartStencil) {
        if (T->has_stencil && (s = upload_stencil(T->stencil, &d->stencil)) != DISCO_OK) return s;
        d->built.fetch_or(kPartStencil);
    }
    if (todo & kPartCore) {
        if (!T->sp.rings.empty()) {
            if ((s = upload_spectral(T->sp, &d->spectral)) != DISCO_OK) return s;
            int64_t b = 0;
            if ((s = upload_vec(T->spectral_flag, &d->spectral_ring, &b, "hipMalloc(spectral ring flags)")) != DISCO_OK)
                return s;
            d->spectral.bytes += b;
        }
        if (T->has_light && (s = upload_packed(T->light, &d->packed_light)) != DISCO_OK) return s;
        if (T->has_sweep) {
            if ((s = upload_sweep(T->sw, &d->sweep)) != DISCO_OK) return s;
            if ((s = upload_packed(T->rest, &d->packed_rest)) != DISCO_OK) return s;
            if (!T->rest_pats.empty()) {
                int64_t b = 0;
                if ((s = upload_vec(T->rest_pats, &d->rest_pats, &b, "hipMalloc(rest patterns)")) != DISCO_OK) return s;
                d->packed_rest.bytes += b;
                d->n_rest_pats = (int32_t)T->rest_pats.size();
            }
        }
        d->built.fetch_or(kPartCore);
    }
    d->bytes = d->bytes_entries + d->packed.bytes + d->stencil.bytes + d->spectral.bytes + d->packed_light.bytes +
               d->sweep.bytes + d->sweep_z.bytes + d->packed_rest.bytes + 64;
    if (d->built == kPartAll) d->tables.reset();
    return DISCO_OK;
}

void free_op(DeviceOp* d) {
    if (d->pat_ptr) (void)hipFree(d->pat_ptr);
    if (d->entries) (void)hipFree(d->entries);
    if (d->rest_pats) (void)hipFree(d->rest_pats);
    if (d->spectral_ring) (void)hipFree(d->spectral_ring);
    if (d->cmap_dev) (void)hipFree(d->cmap_dev);
    d->spectral_ring = nullptr;
    d->cmap_dev = nullptr;
    d->pat_ptr = nullptr;
    d->entries = nullptr;
    d->rest_pats = nullptr;
    d->n_rest_pats = 0;
    free_packed(&d->packed);
    free_packed(&d->packed_light);
    free_packed(&d->packed_rest);
    free_spectral(&d->spectral);
    free_sweep(&d->sweep);
    free_sweep(&d->sweep_z);
    free_mfma(&d->mfma);
    d->mfma_state = 0;
    void* sp[] = {d->stencil.pieces, d->stencil.chunks, d->stencil.vals, d->stencil.cells};
    for (void* p : sp)
        if (p) (void)hipFree(p);
    free_packed(&d->stencil.P);
    d->stencil = StencilDev{};
    d->built.store(0);
    d->bytes = d->bytes_entries = 0;
    d->tables.reset();
}

int64_t numel(const disco_tensor_t* t) {
    int64_t n = 1;
    for (int i = 0; i < t->ndim; ++i) n *= t->shape[i];
    return n;
}

size_t elem_bytes(int dtype) { return dtype == DISCO_BFLOAT16 ? 2 : 4; }

bool overlaps(const disco_tensor_t* a, const disco_tensor_t* b) {
    const uintptr_t a0 = (uintptr_t)a->data, a1 = a0 + (uintptr_t)numel(a) * elem_bytes(a->dtype);
    const uintptr_t b0 = (uintptr_t)b->data, b1 = b0 + (uintptr_t)numel(b) * elem_bytes(b->dtype);
    return a0 < b1 && b0 < a1 && a1 > a0 && b1 > b0;
}

disco_status_t check_device_ptr(const void* p, int device, const char* name) {
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof(attr));
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(DISCO_ERR_DEVICE, std::string(name) + " is not a device pointer known to HIP");
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
        return fail(DISCO_ERR_DEVICE, std::string(name) + " is not device memory");
    if (attr.device != device)
        return fail(DISCO_ERR_DEVICE, std::string(name) + " lives on device " + std::to_string(attr.device) +
                                          ", the plan on device " + std::to_string(device));
    return DISCO_OK;
}

// Shared entry of forward and transpose.
// Which kernels one call runs, given the requested algorithm and channels.
struct Dispatch {
    int32_t algo;
    bool spectral, sweep;
    const PackedDev* packed;  // pattern set of the general fused kernel
    const Work* packed_work;
};

// The small-op rule of AUTO: below 2^18 output pixel-channels one launch of
// the general kernel over every ring (launch latency dominates), else the
// fused schedule.
int32_t resolve_auto(const DeviceOp& op, int32_t algo, int64_t Co) {
    if (algo != DISCO_ALGO_AUTO) return algo;
    const double out_pix_chan = (double)Co * op.g.nlat_o * op.g.nlon_o;
    return out_pix_chan < (double)(1 << 18) ? DISCO_ALGO_FUSED_DIRECT : DISCO_ALGO_FUSED;
}

Dispatch dispatch(const DeviceOp& op, int32_t algo, int Ci, int Co, int32_t dtype) {
    const OpGeom& g = op.g;
    // Small ops are bound by launch latency: one direct fused kernel.
    // Otherwise the fused schedule (spectral polar rings, ring sweep, general
    // kernel for the rest).
    algo = resolve_auto(op, algo, Co);
    Dispatch d{algo, false, false, &op.packed, &op.work_all};
    if (op.basis != DISCO_BASIS_BILINEAR_3X3) return d;
    d.spectral = algo == DISCO_ALGO_FUSED && op.spectral.n_rings > 0;
    // The sweep kernel addresses x and y through 32-bit buffer offsets: the
    // kCIC input channel planes of one launch and one output plane (fp32 when
    // partial sums accumulate) must stay below 2^31 bytes (2048 x 4096 fp32:
    // 268 MB and 34 MB); larger grids take the general kernel.  More than
    // kCIC input channels take one sweep launch per channel group.
    const int64_t es = (int64_t)elem_bytes(dtype);
    const bool sweep_offsets_fit = (int64_t)kCIC * g.nlat_i * g.nlon_i * es < ((int64_t)1 << 31) &&
                                   (int64_t)g.nlat_o * g.nlon_o * 4 < ((int64_t)1 << 31);
    // Several channel groups pay off on single-phase ops (measured: 512 x
    // 1024, 32 -> 32 channels, 0.76 -> 0.65 ms); on ops with longitude
    // phases (the transposed upsampling op, 64 -> 32 channels in bf16) the
    // groups' fp32 atomic merges dominate (eight launches of 0.5 ms against
    // the general kernel's 3.2 ms for the whole op), so groups lose.
    d.sweep = algo == DISCO_ALGO_FUSED && op.sweep.n_runs > 0 && sweep_offsets_fit && (Ci <= kCIC || g.P == 1);
    if (d.sweep) {
        d.packed = &op.packed_rest;
        d.packed_work = &op.work_rest;
    } else if (d.spectral) {
        d.packed = &op.packed_light;
        d.packed_work = &op.work_light;
    }
    return d;
}

// Validates one application of `op` (x -> y with weights w, W laid out
// [op Ci][op Co][K] when transpose, else [op Co][op Ci][K]) without launching.
disco_status_t check_op_args(disco_plan_t plan, const DeviceOp& op, bool transpose, const disco_tensor_t* x,
                             const disco_tensor_t* w, const disco_tensor_t* y, int32_t algo);

// Scratch memory the caller provides (the non-allocating entry point): the
// kernels' workspace is taken from it and nothing is allocated; the spectral
// rings then run on the caller's stream (no helper stream, no events).
struct ExtScratch {
    void* ptr;
    size_t bytes;
};

// depthwise: x [B, C, ...], w [C, K], y [B, C, ...] (channel c filtered by
// w[c] alone); algo is then ignored.
disco_status_t run_op(disco_plan_t plan, const DeviceOp& op, bool transpose, const disco_tensor_t* x,
                      const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream, int32_t algo,
                      bool depthwise = false, const ExtScratch* ext = nullptr);

disco_status_t run(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                   disco_tensor_t* y, hipStream_t stream, int32_t algo, bool transpose, bool depthwise = false) {
    TraceRange range(transpose ? (depthwise ? "disco_transpose_depthwise" : "disco_transpose")
                               : (depthwise ? "disco_forward_depthwise" : "disco_forward"));
    if (!plan) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan is NULL");
    return run_op(plan, transpose ? plan->tr : plan->fwd, transpose, x, w, y, stream, algo, depthwise);
}

disco_status_t check_common(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                            const disco_tensor_t* y);

// Depthwise application of `op`: x [B, C, op input grid], w [C, K],
// y [B, C, op output grid].
disco_status_t check_dw_args(disco_plan_t plan, const DeviceOp& op, const disco_tensor_t* x,
                             const disco_tensor_t* w, const disco_tensor_t* y) {
    if (!x || !w || !y) return fail(DISCO_ERR_INVALID_ARGUMENT, "tensor descriptor is NULL");
    const OpGeom& g = op.g;
    if (x->ndim != 4 || y->ndim != 4 || w->ndim != 2)
        return fail(DISCO_ERR_SHAPE, "x and y must be 4-D [B, C, nlat, nlon], depthwise w 2-D [C, K]");
    for (int i = 0; i < 4; ++i)
        if (x->shape[i] < 0 || y->shape[i] < 0 || (i < 2 && w->shape[i] < 0))
            return fail(DISCO_ERR_SHAPE, "negative extent");
    const int64_t B = x->shape[0], C = x->shape[1];
    if (x->shape[2] != g.nlat_i || x->shape[3] != g.nlon_i)
        return fail(DISCO_ERR_SHAPE, "x grid must be [" + std::to_string(g.nlat_i) + ", " + std::to_string(g.nlon_i) + "]");
    if (y->shape[2] != g.nlat_o || y->shape[3] != g.nlon_o)
        return fail(DISCO_ERR_SHAPE, "y grid must be [" + std::to_string(g.nlat_o) + ", " + std::to_string(g.nlon_o) + "]");
    if (y->shape[0] != B || y->shape[1] != C) return fail(DISCO_ERR_SHAPE, "depthwise x and y must have the same [B, C]");
    const int K = basis_size(op.basis);
    if (w->shape[0] != C || w->shape[1] != K)
        return fail(DISCO_ERR_SHAPE, "depthwise w must be [C, " + std::to_string(K) + "]");
    if (C < 1) return fail(DISCO_ERR_SHAPE, "channel count must be >= 1");
    if (B * C > 65535) return fail(DISCO_ERR_SHAPE, "batch x channels too large for a depthwise call");
    return check_common(plan, x, w, y);
}

disco_status_t check_op_args(disco_plan_t plan, const DeviceOp& op, bool transpose, const disco_tensor_t* x,
                             const disco_tensor_t* w, const disco_tensor_t* y, int32_t algo) {
    if (!x || !w || !y) return fail(DISCO_ERR_INVALID_ARGUMENT, "tensor descriptor is NULL");
    if (algo < DISCO_ALGO_AUTO || algo > DISCO_ALGO_MATRIX_CORE) return fail(DISCO_ERR_INVALID_ARGUMENT, "unknown algo");
    const OpGeom& g = op.g;
    if (x->ndim != 4 || y->ndim != 4 || w->ndim != 3)
        return fail(DISCO_ERR_SHAPE, "x and y must be 4-D [B, C, nlat, nlon], w 3-D");
    for (int i = 0; i < 4; ++i)
        if (x->shape[i] < 0 || y->shape[i] < 0 || (i < 3 && w->shape[i] < 0))
            return fail(DISCO_ERR_SHAPE, "negative extent");
    const int64_t B = x->shape[0], Ci = x->shape[1], Co = y->shape[1];
    if (x->shape[2] != g.nlat_i || x->shape[3] != g.nlon_i)
        return fail(DISCO_ERR_SHAPE, "x grid must be [" + std::to_string(g.nlat_i) + ", " + std::to_string(g.nlon_i) + "]");
    if (y->shape[2] != g.nlat_o || y->shape[3] != g.nlon_o)
        return fail(DISCO_ERR_SHAPE, "y grid must be [" + std::to_string(g.nlat_o) + ", " + std::to_string(g.nlon_o) + "]");
    if (y->shape[0] != B) return fail(DISCO_ERR_SHAPE, "x and y batch differ");
    const int K = basis_size(op.basis);
    const std::string ks = std::to_string(K);
    if (w->shape[2] != K) return fail(DISCO_ERR_SHAPE, "w last extent must be " + ks);
    if (!transpose && (w->shape[0] != Co || w->shape[1] != Ci))
        return fail(DISCO_ERR_SHAPE, "forward w must be [Cout, Cin, " + ks + "]");
    if (transpose && (w->shape[0] != Ci || w->shape[1] != Co))
        return fail(DISCO_ERR_SHAPE, "transpose w must be [CinT, CoutT, " + ks + "]");
    const bool folded = op.basis != DISCO_BASIS_BILINEAR_3X3;
    if (folded && (algo == DISCO_ALGO_GATHER_THEN_CONTRACT || algo == DISCO_ALGO_CONTRACT_THEN_GATHER ||
                   algo == DISCO_ALGO_MATRIX_CORE))
        return fail(DISCO_ERR_UNSUPPORTED, "only the 3x3 basis has the two-kernel and matrix-core schedules");
    if (Ci < 1 || Co < 1) return fail(DISCO_ERR_SHAPE, "channel counts must be >= 1");
    if (B > 65535 || Ci > 4096 || Co > 4096) return fail(DISCO_ERR_SHAPE, "batch or channels too large");
    return check_common(plan, x, w, y);
}

// dtype, device residency and overlap checks shared by every application.
disco_status_t check_common(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                            const disco_tensor_t* y) {
    const int64_t B = x->shape[0];
    // Kernels put (batch item, channel) pairs in a 16-bit grid dimension.
    if (B * std::max(x->shape[1], y->shape[1]) > 65535)
        return fail(DISCO_ERR_SHAPE, "batch x channels above 65535");
    if (x->dtype != y->dtype || w->dtype != x->dtype)
        return fail(DISCO_ERR_DTYPE, "x, w and y must share one dtype");
    if (x->dtype != DISCO_FLOAT32 && x->dtype != DISCO_BFLOAT16)
        return fail(DISCO_ERR_DTYPE, "dtype must be DISCO_FLOAT32 or DISCO_BFLOAT16");
    if (B == 0) return DISCO_OK;
    if (!x->data || !w->data || !y->data) return fail(DISCO_ERR_INVALID_ARGUMENT, "NULL data pointer");
    if (overlaps(y, x) || overlaps(y, w)) return fail(DISCO_ERR_INVALID_ARGUMENT, "y overlaps x or w");
    // Index arithmetic inside the kernels keeps per-plane offsets in 64 bits;
    // the grid itself is bounded by 2^30 pixels at plan creation.
    disco_status_t s;
    if ((s = check_device_ptr(x->data, plan->device, "x")) != DISCO_OK) return s;
    if ((s = check_device_ptr(w->data, plan->device, "w")) != DISCO_OK) return s;
    if ((s = check_device_ptr(y->data, plan->device, "y")) != DISCO_OK) return s;
    return DISCO_OK;
}

// Builds the op's bf16 matrix-core tables on first use (once per op; the
// host op is rebuilt from the plan's parameters).  An op the layout does not
// cover is marked so and left to the other kernels.
disco_status_t ensure_mfma(disco_plan_t plan, const DeviceOp& cop) {
    DeviceOp& op = const_cast<DeviceOp&>(cop);
    std::lock_guard<std::mutex> lock(plan->lazy_mu);
    if (op.mfma_state != 0) return DISCO_OK;
    HostOp h;
    MfmaHost H;
    std::string err;
    try {
        int rc = build_host_op(plan->params, op.src_transpose, &h, &err, op.src_adjoint);
        if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
        rc = pack_mfma(h, &H, &err);
        if (rc == DISCO_ERR_UNSUPPORTED) {
            op.mfma_state = -1;
            return DISCO_OK;
        }
        if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    } catch (const std::bad_alloc&) {
        return fail(DISCO_ERR_OUT_OF_MEMORY, "host allocation failed while packing the matrix-core tables");
    }
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return fail(DISCO_ERR_DEVICE, "hipGetDevice failed");
    if (cur != plan->device && hipSetDevice(plan->device) != hipSuccess)
        return fail(DISCO_ERR_DEVICE, "hipSetDevice failed");
    disco_status_t s = upload_mfma(H, &op.mfma);
    if (cur != plan->device) (void)hipSetDevice(cur);
    if (s != DISCO_OK) {
        free_mfma(&op.mfma);
        return s;
    }
    op.mfma_state = 1;
    return DISCO_OK;
}

// Uploads the op's layout groups in `parts` that are not on the device yet
// (host tables packed at plan creation; synchronous copies).
disco_status_t ensure_parts(disco_plan_t plan, const DeviceOp& cop, int parts) {
    DeviceOp& op = const_cast<DeviceOp&>(cop);
    std::lock_guard<std::mutex> lock(plan->lazy_mu);
    if (!(parts & ~op.built)) return DISCO_OK;
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return fail(DISCO_ERR_DEVICE, "hipGetDevice failed");
    if (cur != plan->device && hipSetDevice(plan->device) != hipSuccess)
        return fail(DISCO_ERR_DEVICE, "hipSetDevice failed");
    const disco_status_t s = upload_parts(&op, parts);
    if (cur != plan->device) (void)hipSetDevice(cur);
    return s;
}

// Layout groups a call runs on (3x3 basis unless `folded`).
int needed_parts(const DeviceOp& op, int32_t algo, bool folded) {
    if (folded) return kPartDirect | (op.g.stride == 1 ? kPartStencil : 0);
    switch (algo) {
        case DISCO_ALGO_GATHER_THEN_CONTRACT: return kPartEntries | kPartCore;
        case DISCO_ALGO_CONTRACT_THEN_GATHER: return kPartEntries;
        case DISCO_ALGO_FUSED_DIRECT: return kPartDirect;
        default: return kPartCore;
    }
}

disco_status_t run_op(disco_plan_t plan, const DeviceOp& op, bool transpose, const disco_tensor_t* x,
                      const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream, int32_t algo,
                      bool depthwise, const ExtScratch* ext) {
    disco_status_t s = depthwise ? check_dw_args(plan, op, x, w, y) : check_op_args(plan, op, transpose, x, w, y, algo);
    if (s != DISCO_OK) return s;
    int64_t B = x->shape[0], Ci = x->shape[1], Co = y->shape[1];
    if (B == 0) return ok();
    // Folded-weight stencil kernels: every basis but the 3x3 grid, and
    // depthwise calls (B * C one-channel items, item i filtered by w[i mod C]).
    const bool axisym = op.basis != DISCO_BASIS_BILINEAR_3X3 || depthwise;

    ExecArgs a{};
    a.op = &op; a.x = x->data; a.w = w->data; a.y = y->data; a.dtype = x->dtype;
    if (depthwise) {
        a.dw_c = (int)Ci;
        B *= Ci;
        Ci = Co = 1;
        algo = DISCO_ALGO_AUTO;
    }
    a.B = (int)B; a.Ci = (int)Ci; a.Co = (int)Co; a.w_trans = transpose; a.stream = stream;

    // bf16 storage with the 3x3 basis: the matrix-core kernel where the op
    // has its layout (built here on the first such call, never by the
    // non-allocating entry point) and x and y are aligned for its vector
    // accesses.
    bool mfma = false;
    if (!axisym && x->dtype == DISCO_BFLOAT16 &&
        (algo == DISCO_ALGO_AUTO || algo == DISCO_ALGO_FUSED || algo == DISCO_ALGO_MATRIX_CORE)) {
        if (!ext && op.mfma_state == 0 && (s = ensure_mfma(plan, op)) != DISCO_OK) return s;
        mfma = op.mfma_state == 1 && ((uintptr_t)x->data % 16) == 0 && ((uintptr_t)y->data % 4) == 0;
    }
    if (algo == DISCO_ALGO_MATRIX_CORE && !mfma)
        return fail(DISCO_ERR_UNSUPPORTED, "the matrix-core kernel needs bf16 storage, the 3x3 basis, at most two "
                                           "longitude phases, stride <= 4, nlon_in a multiple of 8 and aligned x "
                                           "(16 bytes) and y (4 bytes)");
    if (mfma) algo = DISCO_ALGO_MATRIX_CORE;
    if (!mfma) {
        algo = resolve_auto(op, algo, Co);
        const int parts = needed_parts(op, algo, axisym);
        if (parts & ~op.built) {
            if (ext)
                return fail(DISCO_ERR_UNSUPPORTED, "the tables this call runs on are not on the device yet and the "
                                                   "non-allocating entry point does not build them: make one "
                                                   "ordinary call with the same shapes first");
            if ((s = ensure_parts(plan, op, parts)) != DISCO_OK) return s;
        }
    }
    const Dispatch dp = dispatch(op, mfma ? DISCO_ALGO_FUSED_DIRECT : algo, (int)Ci, (int)Co, x->dtype);
    if (!mfma) algo = dp.algo;
    // The fused schedule of an op with neither spectral rings nor a sweep for
    // these channels runs the general kernel over every ring.
    if (!mfma && !axisym && dp.packed == &op.packed && !(op.built & kPartDirect)) {
        if (ext)
            return fail(DISCO_ERR_UNSUPPORTED, "the tables this call runs on are not on the device yet and the "
                                               "non-allocating entry point does not build them: make one ordinary "
                                               "call with the same shapes first");
        if ((s = ensure_parts(plan, op, kPartDirect)) != DISCO_OK) return s;
    }
    const bool spectral = dp.spectral, sweep = dp.sweep;
    const PackedDev& packed = axisym ? op.packed : *dp.packed;
    // One output channel on a stride-1 op takes the blocked stencil kernel.
    const bool blocked = axisym && op.stencil.P.n_items > 0 && Co == 1;
    size_t ws_spec = 0, ws_sweep = 0, ws = 0;
    if (blocked) {
        ws = workspace_bytes_fused(a, op.stencil.P);
    } else if (axisym) {
        ws = workspace_bytes_fused(a, packed);
    } else if (mfma) {
        ws = workspace_bytes_mfma(a);
    } else if (algo == DISCO_ALGO_CONTRACT_THEN_GATHER) {
        ws = workspace_bytes_contract_then_gather(a);
    } else if (algo == DISCO_ALGO_GATHER_THEN_CONTRACT) {
        ws = workspace_bytes_gather_then_contract(a);
    } else {
        ws_spec = spectral ? (workspace_bytes_spectral(a) + 255) / 256 * 256 : 0;
        ws_sweep = sweep ? (workspace_bytes_sweep(a) + 255) / 256 * 256 : 0;
        ws = ws_spec + ws_sweep + workspace_bytes_fused(a, packed);
    }
    if (ext && ws > ext->bytes)
        return fail(DISCO_ERR_UNSUPPORTED, "this call needs " + std::to_string(ws) + " bytes of scratch memory; the "
                    "non-allocating entry point has " + std::to_string(ext->bytes));
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return fail(DISCO_ERR_DEVICE, "hipGetDevice failed");
    if (cur != plan->device && hipSetDevice(plan->device) != hipSuccess)
        return fail(DISCO_ERR_DEVICE, "hipSetDevice failed");
    struct Restore { int d; bool on; ~Restore() { if (on) (void)hipSetDevice(d); } } restore{cur, cur != plan->device};

    if (!ext && fault_inject_alloc())
        return fail(DISCO_ERR_OUT_OF_MEMORY, "allocation failure injected (DISCO_FAULT_INJECT=alloc)");
    float* ws_ptr = ext ? (float*)ext->ptr : nullptr;
    hipError_t e = hipSuccess;
    if (ws > 0 && !ext) {
        e = hipMallocAsync((void**)&ws_ptr, ws, stream);
        if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(workspace)");
    }
    if (blocked) {
        e = launch_stencil_blocked(a, op.stencil, ws_ptr);
    } else if (axisym) {
        e = launch_stencil(a, packed, ws_ptr);
    } else if (mfma) {
        e = launch_mfma(a, ws_ptr);
    } else if (algo == DISCO_ALGO_CONTRACT_THEN_GATHER) {
        e = launch_contract_then_gather(a, ws_ptr);
    } else if (algo == DISCO_ALGO_GATHER_THEN_CONTRACT) {
        e = launch_gather_then_contract(a, ws_ptr);
    } else {
        // The spectral rings (input transforms, products, inverse
        // transforms) run on the plan's helper stream, forked from and joined
        // back into the caller's stream, beside the direct kernels on the
        // caller's stream; when the sweep kernel takes the light rings, the
        // general kernel's remaining rings follow the spectral ones there.
        hipEvent_t fork = nullptr, join = nullptr;
        const bool fork_aux = spectral && plan->aux && !ext;
        ExecArgs as = a;
        if (fork_aux) {
            as.stream = plan->aux;
            e = hipEventCreateWithFlags(&fork, hipEventDisableTiming);
            if (e == hipSuccess) e = hipEventCreateWithFlags(&join, hipEventDisableTiming);
            if (e == hipSuccess) e = hipEventRecord(fork, stream);
            if (e == hipSuccess) e = hipStreamWaitEvent(plan->aux, fork, 0);
            if (e == hipSuccess) e = launch_spectral(as, ws_ptr, kSpectralAll);
            if (e == hipSuccess && sweep) e = launch_fused(as, packed, (float*)((char*)ws_ptr + ws_spec + ws_sweep));
            if (e == hipSuccess) e = hipEventRecord(join, plan->aux);
        } else if (spectral) {
            e = launch_spectral(a, ws_ptr);
        }
        if (e == hipSuccess && sweep) e = launch_sweep(a, ws_sweep ? (float*)((char*)ws_ptr + ws_spec) : nullptr);
        if (e == hipSuccess && !(fork_aux && sweep))
            e = launch_fused(a, packed, (float*)((char*)ws_ptr + ws_spec + ws_sweep));
        if (join) {
            hipError_t ej = hipStreamWaitEvent(stream, join, 0);
            if (e == hipSuccess) e = ej;
        }
        if (fork) (void)hipEventDestroy(fork);
        if (join) (void)hipEventDestroy(join);
    }
    hipError_t e2 = ws_ptr && !ext ? hipFreeAsync(ws_ptr, stream) : hipSuccess;
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    if (e2 != hipSuccess) return hip_fail(e2, "hipFreeAsync(workspace)");
    return ok();
}

// Gradients of the forward (transpose = false) or transposed op, App. C.
// The input gradient is one application of the adjoint op (built at plan
// creation with DISCO_PLAN_BACKWARD; W is read in the other op's layout).
// The weight gradient first runs the op's own kernels on x viewed as B * C_x
// one-channel items with the K x K identity as W, which writes the gathered
// sums Z [B * C_x][K][pixels] to a workspace, then reduces dy (x) Z over
// pixels (disco_grad.hip).  Everything is validated before anything is
// enqueued.
// depthwise: w and dw are [C, K] and every channel is its own one-channel op
// (dx through the adjoint op run depthwise, dW the diagonal blocks only).
disco_status_t backward(disco_plan_t plan, bool transpose, const disco_tensor_t* x, const disco_tensor_t* w,
                        const disco_tensor_t* dy, disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream,
                        bool depthwise = false) {
    TraceRange range(transpose ? "disco_transpose_backward" : "disco_forward_backward");
    if (!plan) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!(plan->params.flags & DISCO_PLAN_BACKWARD))
        return fail(DISCO_ERR_UNSUPPORTED, "plan was created without DISCO_PLAN_BACKWARD");
    if (!dy) return fail(DISCO_ERR_INVALID_ARGUMENT, "dy is NULL");
    if (!dx && !dw) return ok();
    const DeviceOp& op = transpose ? plan->tr : plan->fwd;
    const DeviceOp& adj = transpose ? plan->tr_adj : plan->fwd_adj;
    const int K = basis_size(op.basis);
    disco_status_t s;
    // Input gradient: dy -> dx through the adjoint op, whose W layout is the
    // other op's.
    if (dx) {
        s = depthwise ? check_dw_args(plan, adj, dy, w, dx) : check_op_args(plan, adj, !transpose, dy, w, dx, DISCO_ALGO_AUTO);
        if (s != DISCO_OK) return s;
    }
    // Weight gradient: shapes, then the Z pass's own arguments.
    disco_tensor_t xz{}, wsel{}, zt{};
    int64_t B = 0, C_x = 0, C_dy = 0, P = 0;
    if (dw) {
        if (!x) return fail(DISCO_ERR_INVALID_ARGUMENT, "x is NULL (needed for dw)");
        if (x->ndim != 4 || dw->ndim != (depthwise ? 2 : 3) || dy->ndim != 4)
            return fail(DISCO_ERR_SHAPE, depthwise ? "x and dy must be 4-D, depthwise dw 2-D" : "x and dy must be 4-D, dw 3-D");
        B = x->shape[0]; C_x = x->shape[1]; C_dy = dy->shape[1];
        if (dy->shape[0] != B) return fail(DISCO_ERR_SHAPE, "x and dy batch differ");
        if (dy->shape[2] != op.g.nlat_o || dy->shape[3] != op.g.nlon_o)
            return fail(DISCO_ERR_SHAPE, "dy grid must be the op's output grid");
        if (depthwise) {
            if (C_dy != C_x) return fail(DISCO_ERR_SHAPE, "depthwise x and dy must have the same channels");
            if (dw->shape[0] != C_x || dw->shape[1] != K) return fail(DISCO_ERR_SHAPE, "depthwise dw must be [C, K]");
        } else {
            const int64_t want0 = transpose ? C_x : C_dy, want1 = transpose ? C_dy : C_x;
            if (dw->shape[0] != want0 || dw->shape[1] != want1 || dw->shape[2] != K)
                return fail(DISCO_ERR_SHAPE, std::string("dw must be ") + (transpose ? "[CinT, CoutT, K]" : "[Cout, Cin, K]"));
        }
        if (dw->dtype != x->dtype || dy->dtype != x->dtype) return fail(DISCO_ERR_DTYPE, "x, dy and dw must share one dtype");
        if (B * C_x * K > 65535)
            return fail(DISCO_ERR_SHAPE, "batch x channels x basis functions too large for the weight gradient");
        P = (int64_t)op.g.nlat_o * op.g.nlon_o;
        // dw is written even for an empty batch (a sum over nothing: zeros).
        if (!dw->data) return fail(DISCO_ERR_INVALID_ARGUMENT, "NULL data pointer");
        if ((s = check_device_ptr(dw->data, plan->device, "dw")) != DISCO_OK) return s;
        if (B > 0) {
            if (!dy->data) return fail(DISCO_ERR_INVALID_ARGUMENT, "NULL data pointer");
            if ((s = check_device_ptr(dy->data, plan->device, "dy")) != DISCO_OK) return s;
            if (overlaps(dw, x) || overlaps(dw, dy) || (dx && overlaps(dw, dx)))
                return fail(DISCO_ERR_INVALID_ARGUMENT, "dw overlaps another tensor");
            // dx may be written while the weight gradient's pass reads x.
            if (dx && dx->data && overlaps(dx, x))
                return fail(DISCO_ERR_INVALID_ARGUMENT, "dx overlaps x (x is read for dw while dx is written)");
        }
        xz = *x;
        xz.shape[0] = B * C_x;
        xz.shape[1] = 1;
        wsel.data = x->dtype == DISCO_BFLOAT16 ? plan->wsel16 : plan->wsel32;
        wsel.dtype = x->dtype;
        wsel.ndim = 3;
        wsel.shape[0] = transpose ? 1 : K;
        wsel.shape[1] = transpose ? K : 1;
        wsel.shape[2] = K;
        zt.dtype = x->dtype;
        zt.ndim = 4;
        zt.shape[0] = B * C_x;
        zt.shape[1] = K;
        zt.shape[2] = op.g.nlat_o;
        zt.shape[3] = op.g.nlon_o;
        if (x->shape[2] != op.g.nlat_i || x->shape[3] != op.g.nlon_i)
            return fail(DISCO_ERR_SHAPE, "x grid must be the op's input grid");
        if (C_x < 1 || C_dy < 1 || C_dy > 4096) return fail(DISCO_ERR_SHAPE, "channel counts out of range");
        if (x->dtype != DISCO_FLOAT32 && x->dtype != DISCO_BFLOAT16)
            return fail(DISCO_ERR_DTYPE, "dtype must be DISCO_FLOAT32 or DISCO_BFLOAT16");
        if (B > 0) {
            if (!x->data) return fail(DISCO_ERR_INVALID_ARGUMENT, "NULL data pointer");
            if ((s = check_device_ptr(x->data, plan->device, "x")) != DISCO_OK) return s;
        }
    }
    // With both gradients asked for, the weight gradient's pass (bound by
    // HBM: Z written, then reduced with dy) runs on the plan's second helper
    // stream beside the input gradient (the adjoint op, bound by arithmetic),
    // forked from the caller's stream and joined back into it on every return
    // below.
    hipStream_t ds = stream;
    struct Join {
        hipStream_t from = nullptr, to = nullptr;
        hipEvent_t ev = nullptr;
        ~Join() {
            if (!ev) return;
            (void)hipEventRecord(ev, from);
            (void)hipStreamWaitEvent(to, ev, 0);
            (void)hipEventDestroy(ev);
        }
    } join;
    if (dx && dw && B > 0 && plan->aux_dw) {
        int dev0 = 0;
        (void)hipGetDevice(&dev0);
        if (dev0 != plan->device) (void)hipSetDevice(plan->device);
        hipEvent_t fork = nullptr, jev = nullptr;
        hipError_t e = hipEventCreateWithFlags(&fork, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&jev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventRecord(fork, stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(plan->aux_dw, fork, 0);
        if (fork) (void)hipEventDestroy(fork);
        if (dev0 != plan->device) (void)hipSetDevice(dev0);
        if (e != hipSuccess) {
            if (jev) (void)hipEventDestroy(jev);
            return hip_fail(e, "stream fork");
        }
        join.from = plan->aux_dw;
        join.to = stream;
        join.ev = jev;
        ds = plan->aux_dw;
    }
    if (dx && (s = run_op(plan, adj, !transpose, dy, w, dx, stream, DISCO_ALGO_AUTO, depthwise)) != DISCO_OK) return s;
    if (!dw) return ok();
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return fail(DISCO_ERR_DEVICE, "hipGetDevice failed");
    if (cur != plan->device && hipSetDevice(plan->device) != hipSuccess)
        return fail(DISCO_ERR_DEVICE, "hipSetDevice failed");
    if (B == 0) {
        struct Restore0 { int d; bool on; ~Restore0() { if (on) (void)hipSetDevice(d); } } r0{cur, cur != plan->device};
        const hipError_t ez = launch_zero_fill(dw->data, (size_t)numel(dw) * elem_bytes(dw->dtype), ds);
        return ez == hipSuccess ? ok() : hip_fail(ez, "kernel launch");
    }
    struct Restore { int d; bool on; ~Restore() { if (on) (void)hipSetDevice(d); } } restore{cur, cur != plan->device};
    // fp32 with the 3x3 basis: Z of all channels in one pass (sweep Z mode,
    // spectral rings' products without the contraction); otherwise the op's own kernels
    // once per input channel (items of B * C_x).
    const bool onepass = x->dtype == DISCO_FLOAT32 && op.basis == DISCO_BASIS_BILINEAR_3X3;
    if (onepass && (s = ensure_parts(plan, op, kPartCore | kPartEntries)) != DISCO_OK) return s;
    ExecArgs za{};
    za.op = &op; za.x = x->data; za.dtype = 0; za.B = (int)B; za.Ci = (int)C_x; za.Co = (int)C_x * K;
    za.w_trans = transpose; za.stream = ds;
    const size_t zbytes = ((size_t)(B * C_x) * K * (size_t)P * elem_bytes(x->dtype) + 255) & ~(size_t)255;
    const size_t zws = onepass ? workspace_bytes_gather_z_all(za) : 0;
    // With the heavy rings forming the two polar caps, their share of dW is
    // summed in the frequency domain (Parseval: per ring, sum_q dy Z = sum_m
    // Re(conj(DYhat) Zhat) with the interior bins counted twice), so their Z
    // needs no inverse transforms and is not written to HBM.
    const bool split = onepass && !depthwise && gather_z_split(za) && op.spectral.n_rings > 0 && op.cap_lo < op.cap_hi;
    const int64_t off_light = split ? (int64_t)op.cap_lo * op.g.nlon_o : 0;
    const int64_t p_light = split ? (int64_t)(op.cap_hi - op.cap_lo) * op.g.nlon_o : P;
    const int b_heavy = split ? op.spectral.n_rings * (int)B : 0;
    const int64_t p_heavy = split ? 2 * (int64_t)(op.spectral.M + 1) : 0;
    const size_t dyh_bytes = split ? (spectral_dyhat_bytes(za, (int)C_dy) + 255) / 256 * 256 : 0;
    const size_t gbytes = depthwise ? weight_grad_ws_bytes_dw((int)B, (int)C_x, K, P)
                          : split   ? weight_grad_split_ws_bytes((int)B, (int)C_dy, (int)(C_x * K), p_light, b_heavy, p_heavy)
                                    : weight_grad_ws_bytes((int)B, (int)C_dy, (int)(C_x * K), P);
    void* zbuf = nullptr;
    float* gws = nullptr;
    hipError_t e = hipMallocAsync(&zbuf, zbytes + zws + dyh_bytes, ds);
    if (e != hipSuccess) return hip_fail(e, "hipMallocAsync(gathered sums)");
    e = hipMallocAsync((void**)&gws, gbytes, ds);
    if (e != hipSuccess) {
        (void)hipFreeAsync(zbuf, ds);
        return hip_fail(e, "hipMallocAsync(weight gradient partials)");
    }
    zt.data = zbuf;
    if (split) {
        float2* zhat = nullptr;
        float2* dyh = (float2*)((char*)zbuf + zbytes + zws);
        const float* dy32 = (const float*)dy->data;
        e = launch_gather_z_light(za, (float*)zbuf, (float*)((char*)zbuf + zbytes), &zhat);
        if (e == hipSuccess) e = launch_spectral_dyhat(za, dy32, (int)C_dy, dyh);
        if (e == hipSuccess)
            e = launch_weight_grad_split(dy32 + off_light, (const float*)zbuf + off_light, (int)B, p_light, P,
                                         (const float*)dyh, (const float*)zhat, b_heavy, p_heavy, (float*)dw->data,
                                         gws, (int)C_dy, (int)C_x, K, transpose, ds);
        s = e == hipSuccess ? DISCO_OK : hip_fail(e, "kernel launch");
        (void)hipFreeAsync(gws, ds);
        (void)hipFreeAsync(zbuf, ds);
        return s == DISCO_OK ? ok() : s;
    }
    if (onepass) {
        e = launch_gather_z_all(za, (float*)zbuf, (float*)((char*)zbuf + zbytes));
        s = e == hipSuccess ? DISCO_OK : hip_fail(e, "kernel launch");
    } else {
        s = run_op(plan, op, transpose, &xz, &wsel, &zt, ds, DISCO_ALGO_AUTO);
    }
    if (s == DISCO_OK) {
        e = depthwise ? launch_weight_grad_dw(dy->data, zbuf, dw->data, gws, x->dtype, (int)B, (int)C_x, K, P, ds)
                      : launch_weight_grad(dy->data, zbuf, dw->data, gws, x->dtype, (int)B, (int)C_dy, (int)C_x, K, P,
                                           transpose, ds);
        if (e != hipSuccess) s = hip_fail(e, "kernel launch");
    }
    (void)hipFreeAsync(gws, ds);
    (void)hipFreeAsync(zbuf, ds);
    return s == DISCO_OK ? ok() : s;
}

// ---- kernel timing (measurement tools only) --------------------------------
struct TimedLaunch {
    std::string name;
    hipEvent_t start = nullptr, stop = nullptr;
};
std::atomic<bool> g_timing_on{false};
std::mutex g_timing_mu;
std::vector<TimedLaunch> g_timed;

}  // namespace

namespace disco {

int plan_device(const disco_plan* plan) { return plan->device; }

disco_status_t set_last_error(disco_status_t s, const char* msg) { return fail(s, msg); }

disco_status_t forward_with_scratch(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                    disco_tensor_t* y, hipStream_t stream, void* scratch, size_t bytes) {
    if (!plan) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan is NULL");
    const ExtScratch ext{scratch, bytes};
    return run_op(plan, plan->fwd, false, x, w, y, stream, DISCO_ALGO_AUTO, false, &ext);
}

int timing_begin(const char* name, hipStream_t s) {
    if (!g_timing_on.load(std::memory_order_relaxed)) return -1;
    TimedLaunch t;
    t.name = name;
    if (hipEventCreate(&t.start) != hipSuccess || hipEventCreate(&t.stop) != hipSuccess) return -1;
    (void)hipEventRecord(t.start, s);
    std::lock_guard<std::mutex> lk(g_timing_mu);
    g_timed.push_back(t);
    return (int)g_timed.size() - 1;
}

void timing_end(int token, hipStream_t s) {
    if (token < 0) return;
    std::lock_guard<std::mutex> lk(g_timing_mu);
    if (token < (int)g_timed.size()) (void)hipEventRecord(g_timed[(size_t)token].stop, s);
}

}  // namespace disco

extern "C" {

int32_t disco_debug_bounds_violations(void) {
#ifdef DISCO_DEBUG_BOUNDS
    (void)hipDeviceSynchronize();
    int32_t n = 0;
    for (unsigned int f : {bounds_flag_sweep(), bounds_flag_fused(), bounds_flag_mfma(), bounds_flag_stencil()})
        n += f != 0u;
    return n;
#else
    return -1;
#endif
}

disco_status_t disco_kernel_timing_enable(int32_t on) {
    g_timing_on.store(on != 0);
    return ok();
}

disco_status_t disco_kernel_timing_read(int32_t capacity, char* names, int64_t* launches,
                                        double* total_ms, int32_t* count) {
    if (!count) return fail(DISCO_ERR_INVALID_ARGUMENT, "count is NULL");
    std::vector<TimedLaunch> rec;
    {
        std::lock_guard<std::mutex> lk(g_timing_mu);
        rec.swap(g_timed);
    }
    std::map<std::string, std::pair<int64_t, double>> agg;
    std::vector<std::string> order;
    disco_status_t st = DISCO_OK;
    for (auto& t : rec) {
        float ms = 0.0f;
        if (hipEventSynchronize(t.stop) != hipSuccess || hipEventElapsedTime(&ms, t.start, t.stop) != hipSuccess)
            st = DISCO_ERR_DEVICE;
        if (!agg.count(t.name)) order.push_back(t.name);
        auto& a = agg[t.name];
        a.first += 1;
        a.second += ms;
        (void)hipEventDestroy(t.start);
        (void)hipEventDestroy(t.stop);
    }
    *count = (int32_t)order.size();
    for (int32_t i = 0; i < capacity && i < (int32_t)order.size(); ++i) {
        if (names) {
            std::strncpy(names + 64 * (size_t)i, order[(size_t)i].c_str(), 63);
            names[64 * (size_t)i + 63] = 0;
        }
        if (launches) launches[i] = agg[order[(size_t)i]].first;
        if (total_ms) total_ms[i] = agg[order[(size_t)i]].second;
    }
    if (st != DISCO_OK) return fail(st, "event timing failed");
    return ok();
}

disco_status_t disco_plan_create(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double theta_c,
                                 const disco_basis_t* basis, disco_plan_t* plan_out) {
    if (!plan_out) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan_out is NULL");
    *plan_out = nullptr;
    TraceRange range("disco_plan_create");
    const auto t0 = std::chrono::steady_clock::now();
    PlanParams p{};
    disco_status_t s = resolve_params(nlat_in, nlon_in, nlat_out, nlon_out, theta_c, basis, &p);
    if (s != DISCO_OK) return s;
    HostOp hf, ht, hfa, hta;
    const bool with_backward = (p.flags & DISCO_PLAN_BACKWARD) != 0;
    std::string err;
    try {
        int rc = build_host_op(p, false, &hf, &err);
        if (rc == DISCO_OK) rc = build_host_op(p, true, &ht, &err);
        // Adjoints: the other op's filter pairs, weighted at their output points.
        if (rc == DISCO_OK && with_backward) rc = build_host_op(p, true, &hfa, &err, true);
        if (rc == DISCO_OK && with_backward) rc = build_host_op(p, false, &hta, &err, true);
        if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    } catch (const std::bad_alloc&) {
        return fail(DISCO_ERR_OUT_OF_MEMORY, "host allocation failed while building psi");
    }
    if (log_enabled()) {
        std::fprintf(stderr, "disco: plan theta_c %.6g, basis %d, quadrature %d, sampling %d, node spacing %.6g\n",
                     p.theta_c, p.basis, p.quadrature, p.sampling, p.h);
        log_host_op("forward", hf);
        log_host_op("transpose", ht);
        if (with_backward) {
            log_host_op("forward adjoint", hfa);
            log_host_op("transpose adjoint", hta);
        }
    }
    disco_plan* plan = new (std::nothrow) disco_plan();
    if (!plan) return fail(DISCO_ERR_OUT_OF_MEMORY, "host allocation failed");
    if (hipGetDevice(&plan->device) != hipSuccess) {
        (void)hipGetLastError();
        delete plan;
        return fail(DISCO_ERR_DEVICE, "no HIP device available");
    }
    plan->params = p;
    plan->tr.src_transpose = plan->fwd_adj.src_transpose = true;
    plan->fwd_adj.src_adjoint = plan->tr_adj.src_adjoint = true;
    try {
        s = prepare_op(hf, &plan->fwd);
        if (s == DISCO_OK) s = prepare_op(ht, &plan->tr);
        if (s == DISCO_OK && with_backward) s = prepare_op(hfa, &plan->fwd_adj);
        if (s == DISCO_OK && with_backward) s = prepare_op(hta, &plan->tr_adj);
    } catch (const std::bad_alloc&) {
        s = fail(DISCO_ERR_OUT_OF_MEMORY, "host allocation failed while packing psi");
    }
    // On the device now: what a forward call with AUTO runs on (the fused
    // schedule's groups; the general kernel over every ring as well when some
    // channel count makes the op small; the folded-weight layouts for the
    // other bases), or every group with DISCO_PLAN_EAGER.  The rest is
    // uploaded by the first call that runs on it.
    const bool eager = (p.flags & DISCO_PLAN_EAGER) != 0;
    auto eager_parts = [&](const DeviceOp& d) {
        if (eager) return (int)kPartAll;
        if (&d != &plan->fwd) return 0;
        // The general kernel over every ring as well: for small grids (AUTO
        // takes it below 2^18 output pixel-channels) and for ops whose fused
        // schedule has no spectral rings and, for some channel counts, no
        // sweep (two longitude phases and more than 8 input channels).
        const bool small = (double)d.g.nlat_o * d.g.nlon_o < (double)(1 << 18);
        const OpTables* T = d.tables.get();
        const bool bare = T && T->sp.rings.empty() && (!T->has_sweep || d.g.P > 1);
        return d.basis != DISCO_BASIS_BILINEAR_3X3 ? needed_parts(d, DISCO_ALGO_AUTO, true)
                                                   : (kPartCore | (small || bare ? kPartDirect : 0));
    };
    for (DeviceOp* d : {&plan->fwd, &plan->tr, &plan->fwd_adj, &plan->tr_adj})
        if (s == DISCO_OK && d->tables) s = upload_parts(d, eager_parts(*d));
    if (s == DISCO_OK && with_backward) {
        const int K = basis_size(p.basis);
        std::vector<float> id32((size_t)K * K, 0.0f);
        std::vector<uint16_t> id16((size_t)K * K, 0);
        for (int k = 0; k < K; ++k) {
            id32[(size_t)k * K + k] = 1.0f;
            id16[(size_t)k * K + k] = 0x3f80;  // 1.0 in bf16
        }
        int64_t dummy = 0;
        s = upload_vec(id32, (float**)&plan->wsel32, &dummy, "hipMalloc(selection weights)");
        if (s == DISCO_OK) s = upload_vec(id16, (uint16_t**)&plan->wsel16, &dummy, "hipMalloc(selection weights)");
    }
    if (s != DISCO_OK) {
        free_op(&plan->fwd);
        free_op(&plan->tr);
        free_op(&plan->fwd_adj);
        free_op(&plan->tr_adj);
        if (plan->wsel32) (void)hipFree(plan->wsel32);
        if (plan->wsel16) (void)hipFree(plan->wsel16);
        delete plan;
        return s;
    }
    bool any_spectral = false;
    for (const DeviceOp* d : {&plan->fwd, &plan->tr, &plan->fwd_adj, &plan->tr_adj})
        any_spectral |= d->spectral.n_rings > 0 || (d->tables && !d->tables->sp.rings.empty());
    if (any_spectral && hipStreamCreateWithFlags(&plan->aux, hipStreamNonBlocking) != hipSuccess) plan->aux = nullptr;
    if ((p.flags & DISCO_PLAN_BACKWARD) && hipStreamCreateWithFlags(&plan->aux_dw, hipStreamNonBlocking) != hipSuccess)
        plan->aux_dw = nullptr;
    // Keep freed workspace in the device's pool rather than returning it to
    // the driver at every synchronisation.
    hipMemPool_t pool;
    if (hipDeviceGetDefaultMemPool(&pool, plan->device) == hipSuccess) {
        uint64_t thr = UINT64_MAX;
        (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
    }
    (void)hipGetLastError();
    disco_plan_info_t& I = plan->info;
    I.K = basis_size(p.basis);
    I.nlat_in = nlat_in; I.nlon_in = nlon_in; I.nlat_out = nlat_out; I.nlon_out = nlon_out;
    I.phases_forward = hf.g.P;
    I.phases_transpose = ht.g.P;
    I.max_window = std::max(hf.max_window, ht.max_window);
    I.full_ring_windows = hf.full_ring_windows;
    I.nnz_entries = (int64_t)hf.t_in.size();
    I.nnz_entries_transpose = (int64_t)ht.t_in.size();
    I.nnz_pairs_total = hf.nnz_pairs;
    I.h = p.h;
    // Structure counts from the host tables (every op's are packed).
    auto structure = [](const DeviceOp& d, int32_t* rings, int32_t* pats, int32_t* pairs, int32_t* slots,
                        int32_t* tables) {
        const OpTables* T = d.tables.get();
        *rings = T ? (int32_t)T->sp.rings.size() : d.spectral.n_rings;
        *pats = T ? (int32_t)T->sw.pats.size() : d.sweep.n_pats;
        *pairs = T ? (int32_t)T->sp.pair_slot.size() : d.spectral.n_pairs;
        *slots = T ? (int32_t)T->sp.slot_ring.size() : d.spectral.n_slots;
        *tables = T ? T->sp.n_tables : d.spectral.n_tables;
    };
    structure(plan->fwd, &I.spectral_rings_forward, &I.sweep_patterns_forward, &I.spectral_pairs_forward,
              &I.spectral_slots_forward, &I.spectral_tables_forward);
    structure(plan->tr, &I.spectral_rings_transpose, &I.sweep_patterns_transpose, &I.spectral_pairs_transpose,
              &I.spectral_slots_transpose, &I.spectral_tables_transpose);
    I.psi_compressed_bytes = (int64_t)hf.t_in.size() * (8 + 4 * I.K) + 4 * (int64_t)hf.pat_ptr.size();
    for (const DeviceOp* d : {&plan->fwd, &plan->tr, &plan->fwd_adj, &plan->tr_adj}) {
        const OpTables* T = d->tables.get();
        if (!T && d->bytes == 0) continue;  // an adjoint the plan does not have
        I.psi_bytes_all_layouts += T ? 64 + T->bytes[0] + T->bytes[1] + T->bytes[2] + T->bytes[3] : d->bytes;
    }
    if (log_enabled()) {
        int64_t live = 0;
        for (const DeviceOp* d : {&plan->fwd, &plan->tr, &plan->fwd_adj, &plan->tr_adj}) live += d->bytes;
        const double sec = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        std::fprintf(stderr,
                     "disco: plan built in %.3f s: forward op %d spectral rings, %d sweep patterns; transpose op %d "
                     "spectral rings, %d sweep patterns; device tables %.2f MB now (%s), %.2f MB with every layout\n",
                     sec, I.spectral_rings_forward, I.sweep_patterns_forward, I.spectral_rings_transpose,
                     I.sweep_patterns_transpose, live / 1e6, eager ? "all layouts" : "the rest on first use",
                     I.psi_bytes_all_layouts / 1e6);
    }
    *plan_out = plan;
    return ok();
}

disco_status_t disco_plan_destroy(disco_plan_t plan) {
    if (!plan) return ok();
    int cur = 0;
    (void)hipGetDevice(&cur);
    if (cur != plan->device) (void)hipSetDevice(plan->device);
    if (plan->aux) {
        (void)hipStreamSynchronize(plan->aux);
        (void)hipStreamDestroy(plan->aux);
    }
    if (plan->aux_dw) {
        (void)hipStreamSynchronize(plan->aux_dw);
        (void)hipStreamDestroy(plan->aux_dw);
    }
    free_op(&plan->fwd);
    free_op(&plan->tr);
    free_op(&plan->fwd_adj);
    free_op(&plan->tr_adj);
    if (plan->wsel32) (void)hipFree(plan->wsel32);
    if (plan->wsel16) (void)hipFree(plan->wsel16);
    if (cur != plan->device) (void)hipSetDevice(cur);
    delete plan;
    return ok();
}

disco_status_t disco_plan_query(disco_plan_t plan, disco_plan_info_t* info) {
    if (!plan || !info) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan or info is NULL");
    std::lock_guard<std::mutex> lock(plan->lazy_mu);
    disco_plan_info_t I = plan->info;
    // Device memory as it stands (groups and matrix-core tables built since
    // creation included).
    I.psi_bytes = I.bytes_entries = I.bytes_general = I.bytes_spectral = I.bytes_sweep = I.bytes_stencil = 0;
    I.bytes_matrix_core = 0;
    for (const DeviceOp* d : {&plan->fwd, &plan->tr, &plan->fwd_adj, &plan->tr_adj}) {
        I.bytes_entries += d->bytes_entries;
        I.bytes_general += d->packed.bytes + d->packed_light.bytes + d->packed_rest.bytes;
        I.bytes_spectral += d->spectral.bytes;
        I.bytes_sweep += d->sweep.bytes + d->sweep_z.bytes;
        I.bytes_stencil += d->stencil.bytes;
        I.bytes_matrix_core += d->mfma.bytes;
        I.psi_bytes += d->bytes + d->mfma.bytes;
    }
    *info = I;
    return ok();
}

disco_status_t disco_kernel_work(disco_plan_t plan, int32_t transpose, int32_t algo, int32_t c_in,
                                 int32_t c_out, int32_t dtype, int32_t capacity, char* names,
                                 int64_t* out_pixels, int64_t* in_pixels, int64_t* pairs, int32_t* count) {
    if (!plan || !count) return fail(DISCO_ERR_INVALID_ARGUMENT, "plan or count is NULL");
    if (algo < DISCO_ALGO_AUTO || algo > DISCO_ALGO_MATRIX_CORE) return fail(DISCO_ERR_INVALID_ARGUMENT, "unknown algo");
    if (c_in < 1 || c_out < 1) return fail(DISCO_ERR_SHAPE, "channel counts must be >= 1");
    if (dtype != DISCO_FLOAT32 && dtype != DISCO_BFLOAT16) return fail(DISCO_ERR_DTYPE, "unknown dtype");
    const DeviceOp& op = transpose ? plan->tr : plan->fwd;
    // The matrix-core kernel: what a bf16 call with this algo runs (its
    // tables are not built by this query).
    const bool mfma = dtype == DISCO_BFLOAT16 && mfma_supported(op.g, op.basis) && op.mfma_state >= 0 &&
                      (algo == DISCO_ALGO_AUTO || algo == DISCO_ALGO_FUSED || algo == DISCO_ALGO_MATRIX_CORE);
    if (algo == DISCO_ALGO_MATRIX_CORE && !mfma)
        return fail(DISCO_ERR_UNSUPPORTED, "no matrix-core kernel for this op and dtype");
    if (!mfma) {
        // The figures need the groups the call would run on (uploaded here
        // if a call has not done so yet).
        const disco_status_t s = ensure_parts(plan, op, needed_parts(op, resolve_auto(op, algo, c_out),
                                                                     op.basis != DISCO_BASIS_BILINEAR_3X3));
        if (s != DISCO_OK) return s;
    }
    const Dispatch dp = dispatch(op, mfma ? DISCO_ALGO_FUSED_DIRECT : algo, c_in, c_out, dtype);
    if (!mfma && dp.packed == &op.packed) {
        const disco_status_t s = ensure_parts(plan, op, kPartDirect);
        if (s != DISCO_OK) return s;
    }
    struct Row { const char* name; Work w; };
    std::vector<Row> rows;
    auto spectral_rows = [&op](const SpectralDev&, std::vector<Row>* r) {
        const Work& sw = op.work_spectral;
        r->push_back({"spectral_rfft", Work{0, sw.in_pixels, 0}});
        r->push_back({"spectral_mac", Work{0, 0, sw.pairs}});
        r->push_back({"spectral_irfft", Work{sw.out_pixels, 0, 0}});
    };
    const Work& all = op.work_all;
    ExecArgs ea{};
    ea.op = &op;
    ea.dtype = dtype;
    ea.B = 1;
    ea.Ci = c_in;
    ea.Co = c_out;
    if (mfma) {
        rows.push_back({"mfma_weights", Work{0, 0, 0}});
        rows.push_back({"mfma_gather_contract", all});
        if (op.mfma.P.n_split > 0) rows.push_back({"reduce_partials", Work{0, 0, 0}});
    } else if (op.basis != DISCO_BASIS_BILINEAR_3X3) {
        if (dp.algo != DISCO_ALGO_GATHER_THEN_CONTRACT && dp.algo != DISCO_ALGO_CONTRACT_THEN_GATHER) {
            // Folded psi: one value per (output pixel, input pixel) pair.
            const Work fw{all.out_pixels, all.in_pixels, op.n_entries * op.g.nq};
            const bool blocked = op.stencil.P.n_items > 0 && c_out == 1;
            rows.push_back({blocked ? "stencil_blocked" : "stencil", fw});
            if ((blocked ? op.stencil.P.n_split : op.packed.n_split) > 0)
                rows.push_back({"reduce_partials", Work{0, 0, 0}});
        }
    } else if (dp.algo == DISCO_ALGO_GATHER_THEN_CONTRACT && gather_z_split(ea)) {
        rows.push_back({"sweep_gather_z", op.work_sweep});
        if (op.n_rest_pats > 0) rows.push_back({"gather_z", op.work_rest});
        rows.push_back({"contract_z", Work{all.out_pixels - op.work_spectral.out_pixels, 0, 0}});
        if (op.spectral.n_rings > 0) spectral_rows(op.spectral, &rows);
    } else if (dp.algo == DISCO_ALGO_GATHER_THEN_CONTRACT) {
        rows.push_back({"gather_z", all});
        rows.push_back({"contract_z", Work{all.out_pixels, 0, 0}});
    } else if (dp.algo == DISCO_ALGO_CONTRACT_THEN_GATHER) {
        rows.push_back({"contract_x", Work{0, all.in_pixels, 0}});
        rows.push_back({"gather_y", all});
    } else {
        if (dp.spectral) spectral_rows(op.spectral, &rows);
        if (dp.sweep) rows.push_back({"sweep_gather_contract", op.work_sweep});
        if (dp.sweep && workspace_bytes_sweep(ea) > 0)
            rows.push_back({"convert_y", Work{op.work_sweep.out_pixels, 0, 0}});
        if (dp.packed->n_items > 0) rows.push_back({"fused_gather_contract", *dp.packed_work});
        if (dp.packed->n_items > 0 && dp.packed->n_split > 0)
            rows.push_back({"reduce_partials", Work{0, 0, 0}});
    }
    *count = (int32_t)rows.size();
    for (int32_t i = 0; i < capacity && i < (int32_t)rows.size(); ++i) {
        if (names) {
            std::strncpy(names + 64 * (size_t)i, rows[(size_t)i].name, 63);
            names[64 * (size_t)i + 63] = 0;
        }
        if (out_pixels) out_pixels[i] = rows[(size_t)i].w.out_pixels;
        if (in_pixels) in_pixels[i] = rows[(size_t)i].w.in_pixels;
        if (pairs) pairs[i] = rows[(size_t)i].w.pairs;
    }
    return ok();
}

disco_status_t disco_forward(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                             disco_tensor_t* y, hipStream_t stream) {
    return run(plan, x, w, y, stream, DISCO_ALGO_AUTO, false);
}

disco_status_t disco_transpose(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                               disco_tensor_t* y, hipStream_t stream) {
    return run(plan, x, w, y, stream, DISCO_ALGO_AUTO, true);
}

disco_status_t disco_forward_backward(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                      const disco_tensor_t* dy, disco_tensor_t* dx, disco_tensor_t* dw,
                                      hipStream_t stream) {
    return backward(plan, false, x, w, dy, dx, dw, stream);
}

disco_status_t disco_transpose_backward(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                        const disco_tensor_t* dy, disco_tensor_t* dx, disco_tensor_t* dw,
                                        hipStream_t stream) {
    return backward(plan, true, x, w, dy, dx, dw, stream);
}

disco_status_t disco_forward_depthwise(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                       disco_tensor_t* y, hipStream_t stream) {
    return run(plan, x, w, y, stream, DISCO_ALGO_AUTO, false, true);
}

disco_status_t disco_transpose_depthwise(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                         disco_tensor_t* y, hipStream_t stream) {
    return run(plan, x, w, y, stream, DISCO_ALGO_AUTO, true, true);
}

disco_status_t disco_forward_depthwise_backward(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                                const disco_tensor_t* dy, disco_tensor_t* dx, disco_tensor_t* dw,
                                                hipStream_t stream) {
    return backward(plan, false, x, w, dy, dx, dw, stream, true);
}

disco_status_t disco_transpose_depthwise_backward(disco_plan_t plan, const disco_tensor_t* x,
                                                  const disco_tensor_t* w, const disco_tensor_t* dy,
                                                  disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream) {
    return backward(plan, true, x, w, dy, dx, dw, stream, true);
}

disco_status_t disco_forward_algo(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                  disco_tensor_t* y, hipStream_t stream, int32_t algo) {
    return run(plan, x, w, y, stream, algo, false);
}

disco_status_t disco_transpose_algo(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                    disco_tensor_t* y, hipStream_t stream, int32_t algo) {
    return run(plan, x, w, y, stream, algo, true);
}

disco_status_t disco_psi_entries(int nlat_in, int nlon_in, int nlat_out, int nlon_out, double theta_c,
                                 const disco_basis_t* basis, int32_t transpose, int64_t capacity,
                                 int32_t* out_ring, int32_t* phase, int32_t* in_ring, int32_t* offset,
                                 float* values, int64_t* count, int32_t* phases, int32_t* stride) {
    if (!count) return fail(DISCO_ERR_INVALID_ARGUMENT, "count is NULL");
    PlanParams p{};
    disco_status_t s = resolve_params(nlat_in, nlon_in, nlat_out, nlon_out, theta_c, basis, &p);
    if (s != DISCO_OK) return s;
    HostOp op;
    std::string err;
    try {
        int rc = build_host_op(p, transpose != 0, &op, &err);
        if (rc != DISCO_OK) return fail((disco_status_t)rc, err);
    } catch (const std::bad_alloc&) {
        return fail(DISCO_ERR_OUT_OF_MEMORY, "host allocation failed while building psi");
    }
    const int64_t n = (int64_t)op.t_in.size();
    *count = n;
    if (phases) *phases = op.g.P;
    if (stride) *stride = op.g.stride;
    if (capacity < n) return ok();
    if (!out_ring || !phase || !in_ring || !offset || !values)
        return fail(DISCO_ERR_INVALID_ARGUMENT, "output array is NULL");
    const bool sep = p.basis == DISCO_BASIS_SEPARABLE_4X4;
    const int row = sep ? kSeparableBasis : kBasis;
    const CellMap cm = cell_map(p.basis);
    for (int pat = 0; pat < op.g.n_patterns(); ++pat)
        for (int32_t e = op.pat_ptr[(size_t)pat]; e < op.pat_ptr[(size_t)pat + 1]; ++e) {
            out_ring[e] = pat / op.g.P;
            phase[e] = pat % op.g.P;
            in_ring[e] = op.t_in[(size_t)e];
            offset[e] = op.d[(size_t)e];
            float* out = values + (size_t)e * row;
            if (!sep) {
                std::memcpy(out, &op.val[(size_t)e * kBasis], sizeof(float) * kBasis);
                continue;
            }
            // The separable op stores its cell's four values: spread them.
            for (int k = 0; k < row; ++k) out[k] = 0.0f;
            const int c = op.cell[(size_t)e];
            for (int m = 0; m < 4; ++m)
                if (cm.k[c][m] >= 0) out[cm.k[c][m]] = op.val[(size_t)e * kBasis + m];
        }
    return ok();
}

const char* disco_status_string(disco_status_t status) {
    switch (status) {
        case DISCO_OK: return "DISCO_OK";
        case DISCO_ERR_INVALID_ARGUMENT: return "DISCO_ERR_INVALID_ARGUMENT";
        case DISCO_ERR_UNSUPPORTED: return "DISCO_ERR_UNSUPPORTED";
        case DISCO_ERR_SHAPE: return "DISCO_ERR_SHAPE";
        case DISCO_ERR_DTYPE: return "DISCO_ERR_DTYPE";
        case DISCO_ERR_OUT_OF_MEMORY: return "DISCO_ERR_OUT_OF_MEMORY";
        case DISCO_ERR_DEVICE: return "DISCO_ERR_DEVICE";
    }
    return "DISCO_ERR_UNKNOWN";
}

const char* disco_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
