// disco_internal.h -- shared declarations of libdisco's plan builder, kernels
// and C ABI layer.  Not installed; the public interface is include/disco.h.
#pragma once

#include <atomic>
#include <cstdint>
#include <memory>
#include <string>
#include <vector>

#include <hip/hip_runtime.h>

#include "disco.h"

// Device-side range checks of the psi indices against the buffers they
// index (a build with -DDISCO_DEBUG_BOUNDS; the default build has none).
// Each kernel file keeps a flag that a failed check sets; the flags are read
// and cleared through disco_debug_bounds_violations().  A check reports, it
// does not skip the access: the accesses it covers are LDS reads and writes
// inside the workgroup's allocation by the layouts' construction, which is
// what the check verifies.
#ifdef DISCO_DEBUG_BOUNDS
#define DISCO_BOUNDS_FLAG static __device__ unsigned int disco_bounds_flag = 0u;
#define DISCO_CHECK(cond)                                        \
    do {                                                         \
        if (!(cond)) atomicOr(&disco_bounds_flag, 1u);           \
    } while (0)
#define DISCO_BOUNDS_READER(fn)                                                              \
    unsigned int fn() {                                                                      \
        unsigned int v = 0u, z = 0u;                                                         \
        if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(disco_bounds_flag), sizeof(v)) != hipSuccess) \
            v = 1u;                                                                          \
        (void)hipMemcpyToSymbol(HIP_SYMBOL(disco_bounds_flag), &z, sizeof(z));              \
        return v;                                                                            \
    }
#else
#define DISCO_BOUNDS_FLAG
#define DISCO_CHECK(cond) \
    do {                  \
    } while (0)
#define DISCO_BOUNDS_READER(fn) \
    unsigned int fn() { return 0u; }
#endif

namespace disco {

// Values stored per psi entry: the nine functions of the 3x3 basis, the four
// of the axisymmetric basis followed by zeros, or, for the separable basis,
// the (at most four) functions of the entry's cell (CellMap order) followed
// by zeros.
constexpr int kBasis = 9;
constexpr int kAxisymBasis = 4;
constexpr int kSeparableBasis = 16;

// Parameters of a plan: the forward op maps the in-grid to the out-grid.
struct PlanParams {
    int nlat_in, nlon_in, nlat_out, nlon_out;
    double theta_c;  // filter cutoff (radians)
    double h;        // node spacing (radians)
    int quadrature;  // DISCO_QUAD_*
    int basis;       // DISCO_BASIS_*
    int sampling;    // DISCO_SAMPLING_*
    int flags;       // DISCO_PLAN_*
};

// Basis size K of a DISCO_BASIS_* kind.
inline int basis_size(int basis) { return basis == 1 ? kAxisymBasis : basis == 2 ? kSeparableBasis : kBasis; }

// Longitude structure of one op (forward or transposed) as a gather:
// output pixel p_o = P * q + r (q in [0, nq), phase r in [0, P)) reads input
// pixel (stride * q + d) mod nlon_i for each stored entry (t_i, d) of the
// pattern of (output ring, r).  One of nlon_i / nlon_o and nlon_o / nlon_i is
// an integer s: then (P, stride) = (1, s) or (s, 1).
struct OpGeom {
    int nlat_o, nlon_o;  // op output grid
    int nlat_i, nlon_i;  // op input grid
    int P, stride, nq;
    bool centre_at_input;  // transposed op: the filter sits on the op's input points
    int n_patterns() const { return nlat_o * P; }
};

// Host-built sparse psi of one op, patterns in (output ring, phase) order,
// entries of a pattern ordered by input ring then by longitude offset.
struct HostOp {
    OpGeom g{};
    int basis = 0;                 // DISCO_BASIS_*
    std::vector<int32_t> pat_ptr;  // n_patterns + 1
    std::vector<int32_t> t_in;     // per entry: input ring
    std::vector<int32_t> d;        // per entry: offset in [0, nlon_i)
    std::vector<int32_t> d_raw;    // per entry: unwrapped offset (contiguous along a window)
    std::vector<uint8_t> cell;     // per entry: hat cell (CellMap), 0 for the axisymmetric basis
    std::vector<float> val;        // per entry: 9 values times q(input ring): psi_0..8 (3x3), psi_0..3 then
                                   // zeros (axisymmetric), the cell's values then zeros (separable)
    std::vector<double> val64;     // the same values before rounding to fp32
    int32_t max_window = 0;
    int32_t full_ring_windows = 0;
    int64_t nnz_pairs = 0;  // non-zero (output pixel, input pixel, k) triples
};

// Hat cells.  Every basis is a sum of products of hats, so the support
// splits into cells on which at most four basis functions are non-zero:
//   3x3 grid: cell 4 cu + cv covers [(cu - 2) h, (cu - 1) h) x [(cv - 2) h,
//     (cv - 1) h) of the tangent plane, with nodes a in {cu - 1, cu} and b in
//     {cv - 1, cv} (those inside 0..2), listed a-major;
//   axisymmetric: one cell holding all four functions;
//   separable: cell 4 a + b is Theta in [a h, (a + 1) h) and direction in
//     [b pi / 2, (b + 1) pi / 2), with functions 4 a' + b' for a' in {a, a + 1}
//     (a' <= 3) and b' in {b, (b + 1) mod 4}, listed a'-major.
// k[c][m] is the basis function of value m of an entry in cell c (-1: none).
struct CellMap { int8_t k[16][4]; };
CellMap cell_map(int basis);
// The cell of entry e and its values in CellMap order (zeros where k < 0).
// Returns false if the entry has a non-zero value outside its cell.
bool entry_cell_values(const HostOp& op, int64_t e, int* cell, float v[4]);

// Algorithmic work of a set of an op's patterns, per batch item and channel:
// output pixels written, distinct input pixels read, non-zero (output pixel,
// input pixel, k) triples of psi.  `include` empty selects every pattern.
struct Work {
    int64_t out_pixels = 0, in_pixels = 0, pairs = 0;
};
Work pattern_work(const HostOp& op, const std::vector<uint8_t>& include);

// Returns 0 on success, otherwise a disco_status_t with *err set.
int make_op_geom(const PlanParams& p, bool transpose, OpGeom* g, std::string* err);
// quad_at_output: weight each value with the quadrature of the op's output
// ring instead of its input ring (the adjoint of the other op, App. C).
int build_host_op(const PlanParams& p, bool transpose, HostOp* op, std::string* err,
                  bool quad_at_output = false);

// ---------------------------------------------------------------------------
// Packed layout for the LDS-staged fused kernel (disco_fused.hip).
//
// A workgroup owns kTileQ consecutive output longitudes q of one pattern
// (output ring, phase), one lane per q.  The pattern's entries are cut into
// chunks; a chunk lists spans of input-ring longitudes that are staged into
// LDS together (channel-interleaved), and its entries are sorted by hat cell
// so that each entry touches exactly the basis functions that can be non-zero
// there.  Consecutive chunks of a pattern form a segment; a pattern with
// several segments ("split") accumulates partial outputs in a workspace slot
// per segment that a second kernel sums in a fixed order.  Work items are runs
// of consecutive segments with a bounded number of entries.
constexpr int kTileQ = 256;    // output longitudes per workgroup
constexpr int kCIC = 8;        // input channels per staging pass
constexpr int kLdsCols = 1024; // staged input longitudes per chunk (per channel)
constexpr int kChunkEntries = 512;  // entries staged in LDS per chunk
constexpr int kCells = 16;

struct PSpan { int32_t row, dstart, len, lds_base; };            // row = ring * nlon_i
struct PChunk { int32_t span_begin, span_end, cls[kCells + 1], pad; };
struct PEntry { int32_t off; float v[4]; };                       // off: LDS column at lane 0
struct PVal { float v[4]; };                                      // device: values, SoA with offsets
struct PSeg { int32_t pattern, chunk_begin, chunk_end, slot; };   // slot -1: writes y
struct PItem { int32_t seg_begin, seg_end; };
static_assert(sizeof(PChunk) == 80, "PChunk layout");
static_assert(sizeof(PEntry) == 20, "PEntry layout");

struct PackedHost {
    int32_t tile = kTileQ;              // output longitudes (lanes) per workgroup: 64, 128 or 256
    std::vector<PSpan> spans;
    std::vector<PChunk> chunks;
    std::vector<PEntry> entries;
    std::vector<PSeg> segs;
    std::vector<PItem> items;
    std::vector<int32_t> red_pattern;   // split patterns
    std::vector<int32_t> red_ptr;       // CSR over red_slots, size red_pattern + 1
    std::vector<int32_t> red_slots;     // slots of each split pattern, in summation order
    int32_t n_slots = 0;
};
// skip[pattern] != 0 leaves the pattern out of the segments and work items
// (its output is produced elsewhere); skip may be empty.
// tile: output longitudes (lanes) per workgroup, 64, 128 or kTileQ; the
// spans carry the halo of that width.
int pack_op(const HostOp& op, int target_entries, const std::vector<uint8_t>& skip, PackedHost* out,
            std::string* err, int tile = kTileQ);

// ---------------------------------------------------------------------------
// Blocked layout of the folded-weight stencil kernel for ops with longitude
// stride 1 and one output channel (disco_stencil.hip): a workgroup owns
// `tile` consecutive output longitudes (four per lane) of one pattern.
// A pattern's entries on one input ring form runs of consecutive offsets
// (the filter's disc meets a ring in one arc); each run ("piece") is padded
// with zero entries to whole blocks of four, so a lane's four outputs take
// the block's four weights against seven consecutive inputs read as two
// aligned float4 (one of them kept from the previous block).  A chunk's
// pieces are staged in LDS together (each span tile + 4 nblk
// floats, 16-byte aligned); chunks form segments and work items as in the
// fused layout (PSeg / PItem, split patterns summed by k_reduce_partials).
// Each span carries one more block of columns than its entries read, and
// the weight table four more entries, for the kernel's one-block-ahead reads.
constexpr int kStencilTile = 1024;      // output longitudes per workgroup (ops with nq > 512)
constexpr int kStencilSmallTile = 512;  // ... for ops with at most 512 output longitudes per pattern
// Chunk budgets scale with the tile (lanes = tile / 4) and are set for
// occupancy: 4 tile staged floats and tile / 2 entries per chunk keep the
// kernel at 91 VGPRs and five waves per SIMD for the 1024-longitude tile
// (8192 and 1024 gave 148 VGPRs, three waves, and 1.7x the time at L = 2048).
constexpr int stencil_cols(int tile) { return 4 * tile; }         // LDS floats staged per chunk
constexpr int stencil_entries(int tile) { return tile / 2; }      // padded entries (weights) per chunk
constexpr int stencil_max_run(int tile) { return tile / 2; }      // entries of one piece
constexpr int stencil_span(int tile, int nblk) { return tile + 4 * nblk + 4; }
struct SPiece { int32_t row, dstart, lds_base, nblk; };           // row = ring * nlon_i; stencil_span(tile, nblk) columns
struct SChunk { int32_t piece_begin, piece_end, ent_begin, ent_end; };

struct StencilHost {
    int32_t tile = kStencilTile;        // output longitudes per workgroup
    std::vector<SPiece> pieces;
    std::vector<SChunk> chunks;
    std::vector<PVal> vals;             // per padded entry: its cell's values times q (zeros for padding)
    std::vector<uint8_t> cells;         // per padded entry: its cell (CellMap)
    std::vector<PSeg> segs;             // chunk_begin / chunk_end index chunks
    std::vector<PItem> items;
    std::vector<int32_t> red_pattern, red_ptr, red_slots;
    int32_t n_slots = 0;
};
int pack_stencil(const HostOp& op, int target_entries, int tile, StencilHost* out, std::string* err);

// ---------------------------------------------------------------------------
// Sweep layout (disco_sweep.hip): a workgroup walks a run of consecutive
// patterns for one 256-longitude tile, keeping the spans of the input rings
// the run reads resident in LDS slots; before each pattern it stages only the
// rings first needed there (into slots whose previous ring is no longer
// read).  Used for patterns with at most kSweepEntries entries when every
// input channel fits one staging pass (Ci <= kCIC).
constexpr int kSweepTile = 256;   // output longitudes (lanes) of a sweep workgroup
// LDS of a sweep workgroup: 2 x kSweepCols float4 of input plus the entry
// table, 39.5 KB, so that four workgroups (one wave per SIMD each) share a
// CU's 160 KB.  Rings with 128 entries or more are the spectral path's.
constexpr int kSweepCols = 1152;  // LDS columns (per channel) of all slots of a run
constexpr int kSweepEntries = 128;  // entries of one pattern on the sweep path

struct SRun { int32_t pat_begin, pat_end; };             // [begin, end) into SPat
// Entry groups of a sweep pattern, in the order the kernel walks them: the 16
// hat cells row by row, and after cell (a + 1, b + 1), the last cell that
// touches basis function K = 3 a + b, the group of entries whose only
// non-zero value is K's (a single product per channel instead of the 2 or 4
// of their cell).  Group ids: cell c is c, K's group is 16 + K.
constexpr int kSweepGroups = 25;
constexpr int sweep_last_cell(int K) { return 4 * (K / 3 + 1) + K % 3 + 1; }
constexpr int sweep_group_pos(int grp) {
    return grp >= 16 ? sweep_last_cell(grp - 16) + (grp - 16) + 1
                     : grp + (grp > 5) + (grp > 6) + (grp > 7) + (grp > 9) + (grp > 10) + (grp > 11) +
                           (grp > 13) + (grp > 14) + (grp > 15);
}
// One pattern of a run, 12 dwords (the kernel keeps two in scalar registers):
// the entries are [ent, ent + nent) in walk order; byte c % 4 of ncell[c / 4]
// = entries in hat cell c, bit 16 + K of nact_nent = one entry in basis
// function K's single-value group (a second one stays in its cell); the
// spans first read here are acts[act_begin, act_begin + nact), the first of
// them copied inline.
struct SPat {
    int32_t pattern;
    int32_t act_begin;
    int32_t nact_nent;           // nact in bits 0..7, nent in bits 8..15, singles in bits 16..24
    int32_t ent;
    uint32_t ncell[4];
    PSpan first;                 // acts[act_begin] (zeros when nact == 0)
};
static_assert(sizeof(SPat) == 48, "SPat layout");
static_assert(kSweepEntries <= 255, "per-cell and per-pattern entry counts are bytes");
constexpr int spat_nact(const SPat& P) { return P.nact_nent & 255; }
constexpr int spat_nent(const SPat& P) { return (P.nact_nent >> 8) & 255; }
constexpr int spat_single(const SPat& P, int K) { return (P.nact_nent >> (16 + K)) & 1; }

struct SweepHost {
    std::vector<SRun> runs;
    std::vector<SPat> pats;
    std::vector<PSpan> acts;
    std::vector<PEntry> entries;
    std::vector<uint8_t> covered;  // per pattern: handled by a run
};
int pack_sweep(const HostOp& op, int target_cost, const std::vector<uint8_t>& skip, SweepHost* out,
               std::string* err);

struct SweepDev {
    SRun* runs = nullptr;
    SPat* pats = nullptr;
    PSpan* acts = nullptr;
    int32_t* offs = nullptr;
    PVal* vals = nullptr;
    int32_t* cov_pats = nullptr;  // patterns the runs cover (fp32 partial sums converted to bf16)
    int32_t n_runs = 0;
    int32_t n_pats = 0;
    int32_t n_cov = 0;
    int64_t bytes = 0;
};

// ---------------------------------------------------------------------------
// Spectral path for heavy output rings (disco_spectral_plan.cpp, disco_spectral.hip).
//
// When an output ring's windows wrap whole input rings, its sum over one
// input ring is a circular cross-correlation along longitude (Sec. 4.2: the
// pattern is shift invariant), computed exactly through the discrete Fourier
// transform:  Yhat[co][m] = sum_{t_i, ci} Xhat[t_i][ci][m]
//   * sum_k W[co][ci][k] conj(Vhat_k[t_o, t_i][m]).
// East-west mirror symmetry of the 3x3 basis gives Vhat_{3a+2} =
// conj(Vhat_{3a}) and a real Vhat_{3a+1}, so each (ring pair, frequency)
// stores 9 floats: Re/Im Vhat_{3a} and Re Vhat_{3a+1} for a = 0, 1, 2.
// Pairs mirrored about the equator share one table (rows a = 0 and a = 2
// exchanged), which halves the tables of an op with both polar caps.
struct SpectralHost {
    int N = 0, M = 0;                 // ring length and M = N / 2
    std::vector<int32_t> rings;       // heavy output rings
    std::vector<int32_t> pair_ptr;    // CSR over pairs, size rings + 1
    std::vector<int32_t> pair_slot;   // input-ring slot of each pair
    std::vector<int32_t> pair_tab;    // table of each pair in vs; bit 31: read with rows a = 0, 2 exchanged
    int32_t n_tables = 0;             // tables in vs (pairs that are no equator mirror of an earlier one)
    std::vector<int32_t> slot_ring;   // input ring of each slot
    std::vector<float> vs;            // [table][9][M + 1], scaled by 1 / N
    std::vector<float> tw;            // [N / 2][2]: exp(-2 pi i t / N)
};
// Fills *sp (possibly with no rings) and marks heavy patterns in *heavy.
int build_spectral(const HostOp& op, int min_entries, SpectralHost* sp, std::vector<uint8_t>* heavy,
                   std::string* err);

struct SpectralDev {
    int N = 0, M = 0, n_rings = 0, n_pairs = 0, n_slots = 0, n_tables = 0;
    int32_t* rings = nullptr;
    int32_t* pair_ptr = nullptr;
    int32_t* pair_slot = nullptr;
    int32_t* pair_tab = nullptr;
    int32_t* slot_ring = nullptr;
    float* vs = nullptr;
    float* tw = nullptr;
    int64_t bytes = 0;
};

// ---------------------------------------------------------------------------
// Matrix-core layout (disco_mfma.hip) for bf16 storage: the 3x3 basis, at
// most two longitude phases, stride <= 4, nlon_in a multiple of 8.
//
// Both steps of the gather-then-contract product run on bf16 matrix cores.
// For one output ring, the entries of all its phases on one input ring are
// laid on the shortest arc of offsets that covers them, cut into groups of
// eight consecutive offsets (d0 .. d0 + 7); four groups make a chunk, the
// 32-long reduction of one v_mfma_f32_16x16x32_bf16:
//   Z[phase][k][q] += sum_{group, u} V[phase][k][group][u] x[ring][s q + d0 + u]
// with the values V (rows k = 0..8, rows 9..15 zero) as the A operand and the
// staged input as the B operand.  The second product
//   y[co][q] += sum_{ci, k} W[co][ci][k] Z[ci][k][q]
// takes two input channels per instruction.  A workgroup (4 waves, 16 output
// longitudes per block, four blocks per wave) runs one segment of an output
// ring (consecutive groups within the chunk and staged-element budgets) for
// kMfmaTile output longitudes; rings cut into several segments write fp32
// partial outputs to a slot per (segment, phase), summed by
// k_reduce_partials.
constexpr int kMfmaTile = 256;       // output longitudes per workgroup
constexpr int kMfmaCis = 8;          // input channels staged per pass
constexpr int kMfmaMaxChunks = 8;    // chunks (32 offsets each) of one segment
constexpr int kMfmaMaxElems = 1280;  // staged elements per channel of one segment
// Spans use PSpan: row = ring * nlon_i, dstart (a multiple of 8), len and
// lds_base in staged elements (element e of a span holds the two inputs at
// longitudes s q0 + dstart + e and + 1, q0 the tile's first output longitude).
struct MSeg { int32_t ring, chunk_begin, chunk_end, span_begin, span_end, n_elems, slot, pad; };
struct MChunkHdr { int32_t grp[4]; };  // staged element of each group's offset d0 at q = q0
struct MfmaHost {
    int32_t P = 1;
    std::vector<PSpan> spans;
    std::vector<MSeg> segs;
    std::vector<MChunkHdr> chunks;
    std::vector<uint16_t> aop;  // per chunk and phase: 64 lanes x 8 bf16 (lane i + 16 g: row i, group g)
    std::vector<int32_t> red_pattern, red_ptr, red_slots;
    int32_t n_slots = 0;
    // Dispatch order: workgroup index -> work item (segment * n_qtiles +
    // longitude tile) or -1 (nothing to do).  Workgroups go round-robin to
    // the 8 XCDs, so entry x + 8 j is the j-th item of XCD x: each XCD gets a
    // contiguous run of output rings (which share input rings in its L2) of
    // about an eighth of the total work, heaviest items first.
    std::vector<int32_t> order;
    int32_t n_qtiles = 0;
};
// Whether pack_mfma covers an op of this geometry and basis.
inline bool mfma_supported(const OpGeom& g, int basis) {
    return basis == DISCO_BASIS_BILINEAR_3X3 && g.P <= 2 && g.stride <= 4 && g.nlon_i % 8 == 0;
}
int pack_mfma(const HostOp& op, MfmaHost* out, std::string* err);

struct PackedDev {
    int32_t tile = kTileQ;       // lanes per workgroup the spans were cut for
    PSpan* spans = nullptr;
    PChunk* chunks = nullptr;
    int32_t* offs = nullptr;     // per entry: LDS column at lane 0
    PVal* vals = nullptr;        // per entry: non-zero basis values of its cell
    PSeg* segs = nullptr;
    PItem* items = nullptr;
    int32_t* red_pattern = nullptr;
    int32_t* red_ptr = nullptr;
    int32_t* red_slots = nullptr;
    int32_t n_items = 0, n_split = 0, n_slots = 0;
    int64_t bytes = 0;
};

struct MfmaDev {
    PSpan* spans = nullptr;
    MSeg* segs = nullptr;
    MChunkHdr* chunks = nullptr;
    uint16_t* aop = nullptr;
    int32_t* order = nullptr;
    PackedDev P;                 // the reduction tables (red_*, n_split, n_slots)
    int32_t n_segs = 0, n_order = 0, n_qtiles = 0;
    int64_t bytes = 0;
};

struct StencilDev {
    SPiece* pieces = nullptr;
    SChunk* chunks = nullptr;
    PVal* vals = nullptr;
    uint8_t* cells = nullptr;
    PackedDev P;                        // segs, items and the reduction tables (no spans)
    int32_t tile = kStencilTile;
    int64_t n_padded = 0;
    int64_t bytes = 0;
};

// Host-side tables of one op's layouts, kept until uploaded (disco_abi.cpp).
struct OpTables;
// Layout groups of an op, uploaded on first use: the fused schedule's
// (spectral rings, ring sweep, general kernel for the rest), the general
// kernel over every pattern, the plain entry tables, the stencil layout.
enum : int { kPartCore = 1, kPartDirect = 2, kPartEntries = 4, kPartStencil = 8, kPartAll = 15 };

// Device-side layout of one op (see disco_kernels.hip).
struct DevEntry {
    int32_t row;  // input ring * nlon_i
    int32_t d;    // longitude offset in [0, nlon_i)
    float v[kBasis];
    int32_t pad;
};
static_assert(sizeof(DevEntry) == 48, "DevEntry is 12 dwords");

struct DeviceOp {
    OpGeom g{};
    int basis = 0;           // DISCO_BASIS_*: bases other than the 3x3 grid run only the stencil kernels
    int8_t* cmap_dev = nullptr;  // device copy of cell_map(basis), 64 bytes
    PackedDev packed;        // every pattern through the direct kernel
    PackedDev packed_light;  // patterns not handled by the spectral path
    SpectralDev spectral;
    SweepDev sweep;          // light patterns walked by the sweep kernel (Ci <= kCIC)
    SweepDev sweep_z;        // the same patterns in shorter runs, for the sweep's Z mode
    StencilDev stencil;      // longitude stride 1: the blocked layout of the stencil kernels
    MfmaDev mfma;            // bf16 matrix-core layout, built at the op's first bf16 call
    int8_t mfma_state = 0;   // 0 not built yet, 1 built, -1 the op has no such layout
    bool src_transpose = false, src_adjoint = false;  // build_host_op arguments of this op
    std::atomic<int> built{0};  // kPart* groups on the device (set after their upload completes)
    std::shared_ptr<OpTables> tables;  // host tables of the groups not uploaded yet
    PackedDev packed_rest;   // light patterns the sweep runs do not cover
    int32_t* rest_pats = nullptr;  // device: those patterns' indices (gather-then-contract schedule)
    int32_t n_rest_pats = 0;
    uint8_t* spectral_ring = nullptr;  // device, nlat_o: 1 for output rings the spectral path writes
    // The spectral rings are exactly the polar caps [0, cap_lo) and [cap_hi,
    // nlat_o) (cap_lo < cap_hi), or cap_lo = cap_hi = 0.
    int32_t cap_lo = 0, cap_hi = 0;
    int32_t* pat_ptr = nullptr;  // device, n_patterns + 1
    DevEntry* entries = nullptr;  // device
    int64_t n_entries = 0;
    int64_t nnz_pairs = 0;
    int64_t bytes = 0;
    int64_t bytes_entries = 0;  // pat_ptr + entries (+ the cell map)
    // Work of the pattern sets above: all, spectral rings, the rest of them,
    // sweep-walked, and what the general kernel keeps beside the sweep.
    Work work_all, work_spectral, work_light, work_sweep, work_rest;
};

// Kernel launchers (disco_kernels.hip).  All return a hipError_t.
// dtype: 0 = fp32, 1 = bf16 (raw uint16 storage).
struct ExecArgs {
    const DeviceOp* op;
    const void* x;
    const void* w;
    void* y;
    int dtype;
    int B, Ci, Co;   // op's input / output channels
    bool w_trans;    // W is [Ci][Co][9] (transposed op) instead of [Co][Ci][9]
    hipStream_t stream;
    // Depthwise channels (stencil kernels only): x and y are viewed as B * C
    // one-channel items (B above is then B * C, Ci = Co = 1) and item i takes
    // the filter W[i mod dw_c][.] of a [C][K] weight tensor; 0 = full W.
    int dw_c = 0;
};

// The plan's device (the one that created it).
int plan_device(const disco_plan* plan);
// Records msg as this thread's last error and returns s.
disco_status_t set_last_error(disco_status_t s, const char* msg);
// disco_forward with every kernel's workspace taken from `scratch` (`bytes`
// bytes of device memory on the plan's device) instead of the stream-ordered
// pool: nothing is allocated and the spectral rings run on `stream` itself.
// A call that needs more than `bytes` fails with DISCO_ERR_UNSUPPORTED before
// anything is enqueued.
disco_status_t forward_with_scratch(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                    disco_tensor_t* y, hipStream_t stream, void* scratch, size_t bytes);

// Kernel timing hook: when enabled, brackets a launch with events on `s`.
// Returns the token to pass to timing_end (or -1 when disabled).
int timing_begin(const char* name, hipStream_t s);
void timing_end(int token, hipStream_t s);

hipError_t launch_gather_then_contract(const ExecArgs& a, float* z_ws);
hipError_t launch_sweep_z(const ExecArgs& a, float* z);   // disco_sweep.hip
bool gather_z_split(const ExecArgs& a);                   // sweep + spectral Z schedule usable
hipError_t launch_contract_then_gather(const ExecArgs& a, float* xc_ws);
// Gathered sums Z[b][ci][k][pixel] (fp32 storage, 3x3 basis) of every output
// ring into z (B * Ci * 9 * pixels floats): the sweep's Z mode, k_gather_z
// for the other light rings, the spectral kernels' transforms and their
// products without the contraction (kSpectralZ) for the heavy ones.  ws:
// workspace_bytes_gather_z_all bytes.
size_t workspace_bytes_gather_z_all(const ExecArgs& a);
hipError_t launch_gather_z_all(const ExecArgs& a, float* z, float* ws);
// The same without the heavy rings' inverse transforms: their Z stays in
// the frequency domain (spectral_yhat of the Z-as-output arguments, Ci * 9
// channels) and z is not written on the spectral rings.
hipError_t launch_gather_z_light(const ExecArgs& a, float* z, float* ws, float2** zhat);
size_t workspace_bytes_gather_then_contract(const ExecArgs& a);
size_t workspace_bytes_contract_then_gather(const ExecArgs& a);
hipError_t launch_fused(const ExecArgs& a, const PackedDev& P, float* partial_ws);
// The matrix-core kernel (bf16 storage): workspace = the W operand table
// (workspace_bytes_mfma_w) followed by the partial slots of split rings.
size_t workspace_bytes_mfma(const ExecArgs& a);
hipError_t launch_mfma(const ExecArgs& a, void* ws);
size_t workspace_bytes_fused(const ExecArgs& a, const PackedDev& P);
// stages: bit 0 the input-ring transforms, bit 1 the frequency-domain
// products, bit 2 the inverse transforms (in that order on one stream);
// with kSpectralZ the products write the nine gathered planes of every input
// channel (a.Co = a.Ci * 9, a.w unused) instead of contracting with W.
constexpr int kSpectralAll = 7;
constexpr int kSpectralZ = 8;
hipError_t launch_spectral(const ExecArgs& a, float* ws, int stages = kSpectralAll);
// Where the products' output Yhat[h][b][co][m] (M + 1 bins) lies in the
// spectral workspace ws of launch_spectral(a, ws, ...).
float2* spectral_yhat(const ExecArgs& a, float* ws);
// DYhat[h][b][c][m]: the real DFT of dy (fp32 [B][C][nlat_o][nlon_o]) on the
// op's spectral output rings, bins 0 < m < M doubled, so that the sum over a
// ring of dy times a signal with Yhat (as the products write it) is
// sum_m Re(DYhat[m]) Re(Yhat[m]) + Im(DYhat[m]) Im(Yhat[m]).
size_t spectral_dyhat_bytes(const ExecArgs& a, int C);
hipError_t launch_spectral_dyhat(const ExecArgs& a, const float* dy, int C, float2* dyh);
// The sweep takes kCIC input channels per launch: more input channels run
// one launch per group, the first storing y and the others adding their
// partial sums into it (fp32 atomic adds, one per element and launch, in
// launch order).  bf16 outputs accumulate in y32_ws (workspace_bytes_sweep
// bytes, fp32 [B][Co][pixels]) and are converted for the covered patterns at
// the end.
size_t workspace_bytes_sweep(const ExecArgs& a);
hipError_t launch_sweep(const ExecArgs& a, float* y32_ws);
size_t workspace_bytes_spectral(const ExecArgs& a);
// Sums the partial outputs of split patterns (the fused and stencil kernels' slots).
hipError_t launch_reduce_partials(const ExecArgs& a, const PackedDev& P, const float* partial);
// Folded-weight kernels (disco_stencil.hip), every basis: W folded into the
// packed psi values per call (through the op's CellMap), one scalar weight per
// entry and channel pair, gathered directly into y.  Workspace as
// launch_fused.
hipError_t launch_stencil(const ExecArgs& a, const PackedDev& P, float* partial_ws);
// The blocked kernel (one output channel, longitude stride 1); workspace
// sizeof(float) * n_slots * B * nq.
hipError_t launch_stencil_blocked(const ExecArgs& a, const StencilDev& S, float* partial_ws);

// Weight gradient reduction (disco_grad.hip): G[m][n] = sum_{b,p} A[b][m][p]
// Zs[b][n][p] over P pixels, A = dy [B][M][P] and Zs = the gathered sums
// [B][N][P] (N = C_x * K, rows (c_x, k)), written as dW[m][c_x][k] (forward
// layout) or dW[c_x][m][k] (transposed op's layout).  dtype 0 fp32, 1 bf16
// (inputs and dW); partials in ws (weight_grad_ws_bytes).
size_t weight_grad_ws_bytes(int B, int M, int N, int64_t P);
// fp32 only: G summed over two parts into one set of partials, the light
// rings' pixels (B items, rows of P_light values at row stride `stride`) and
// the heavy rings' frequency-domain rows (B_heavy = rings x B items, rows of
// P_heavy values, e.g. spectral_dyhat against the spectral Zhat as floats).
size_t weight_grad_split_ws_bytes(int B, int M, int N, int64_t P_light, int B_heavy, int64_t P_heavy);
hipError_t launch_weight_grad_split(const float* dy, const float* zs, int B, int64_t P_light, int64_t stride,
                                    const float* dyh, const float* zh, int B_heavy, int64_t P_heavy, float* dw,
                                    float* ws, int M, int C_x, int K, bool transposed_layout, hipStream_t s);
// Zeros `bytes` (a multiple of 2) of device memory with a kernel (no memset
// node when the caller captures a graph).
hipError_t launch_zero_fill(void* p, size_t bytes, hipStream_t s);
// The range-check flags of the kernel files (0 without DISCO_DEBUG_BOUNDS);
// each call reads and clears its file's flag.
unsigned int bounds_flag_sweep();
unsigned int bounds_flag_fused();
unsigned int bounds_flag_mfma();
unsigned int bounds_flag_stencil();
// Depthwise dW[c][k] = sum_{b,p} dy[b][c][p] Zs[b][c][k][p] (K <= 16), partials
// in ws (weight_grad_ws_bytes_dw), reduced in a fixed order.
size_t weight_grad_ws_bytes_dw(int B, int C, int K, int64_t P);
hipError_t launch_weight_grad_dw(const void* dy, const void* zs, void* dw, float* ws, int dtype, int B, int C, int K,
                                 int64_t P, hipStream_t s);
hipError_t launch_weight_grad(const void* dy, const void* zs, void* dw, float* ws, int dtype, int B, int M,
                              int C_x, int K, int64_t P, bool transposed_layout, hipStream_t s);

}  // namespace disco
