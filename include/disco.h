/*
 * disco.h -- C ABI of libdisco.so: DISCO spherical convolution on one
 * MI355X (gfx950) GPU.
 *
 * The operation is the DISCO spherical convolution of Ocampo, Price & McEwen,
 * "Scalable and Equivariant Spherical CNNs by Discrete-Continuous (DISCO)
 * Convolutions" (ICLR 2023), restricted to rotations R = Z(phi) Y(theta) in
 * SO(3)/SO(2) (Sec. 3.2), written as a sparse-dense product (Sec. 4.1):
 *
 *   forward    y[b,co,j] = sum_{ci,k} W[co,ci,k] sum_i psi_k(R_j^{-1} w_i) q_in(i) x[b,ci,i]
 *   transpose  y[b,c,i]  = sum_{c',k} W[c',c,k] sum_j psi_k(R_j^{-1} w_i) q_out(j) x[b,c',j]
 *              (Sec. 3.5, eq. 6: the filter is centred at the transposed
 *               op's input points and weighted by their quadrature)
 *
 * Grids are equiangular, longitude fastest in memory, longitude 2 pi p / nlon,
 * in one of two samplings: cell-centred, colatitude (t + 1/2) pi / nlat (the
 * default), or the paper's own pole-including grid (Sec. 4.2 "Explicit
 * sampling", the antipodal McEwen-Wiaux variant of App. A): with
 * L = nlat - 1, colatitude pi t / L for t = 0..L and nlon = 2L, each pole ring
 * holding 2L samples of one point.  A plan fixes one
 * (in-grid, out-grid) pair: the forward op maps in -> out, the transposed op
 * maps out -> in with the same filter pairs.  The longitude compression of
 * Sec. 4.2 (one psi pattern per output latitude ring, reused at every output
 * longitude by a cyclic shift) requires nlon_in / nlon_out or nlon_out /
 * nlon_in to be an integer.
 *
 * Bases (Sec. 3.4: equally spaced nodes, linear interpolation, zero beyond
 * theta_c):
 *   DISCO_BASIS_BILINEAR_3X3 (K = 9): the 3x3 node grid of App. E.2,
 *     projected onto the sphere with the azimuthal equidistant map (edge nodes
 *     at geodesic distance h, corner nodes at sqrt(2) h), bilinear
 *     interpolation between nodes, node index k = 3a + b with a along
 *     increasing colatitude (south) and b along increasing longitude (east);
 *   DISCO_BASIS_AXISYMMETRIC_4 (K = 4): the axisymmetric filter psi(theta)
 *     that App. B times, four nodes at geodesic distance k h, k = 0..3,
 *     psi_k(Theta) = max(0, 1 - |Theta / h - k|); the default h = theta_c / 4
 *     makes the last hat vanish at the cutoff;
 *   DISCO_BASIS_SEPARABLE_4X4 (K = 16): the separable filter
 *     psi(theta, phi) = theta-part(theta) phi-part(phi) of Sec. 3.4 with four
 *     nodes along each (App. E), as products of hats,
 *     psi_{4a+b}(Theta, Phi) = max(0, 1 - |Theta / h - a|) mu_b(Phi),
 *     mu_b(Phi) = max(0, 1 - |Phi - b pi / 2|_{mod 2 pi} / (pi / 2)),
 *     Phi = atan2(v, u) the direction in the filter's tangent plane (0 south,
 *     pi / 2 east; taken as 0 at the filter centre itself), default
 *     h = theta_c / 4.  A separable filter with node values t_a and p_b is
 *     W[., ., 4a+b] = t_a p_b.
 *
 * Channels: W[Cout][Cin][K] mixes every input channel into every output
 * channel; the depthwise calls filter each channel by its own W[c][K]
 * (the depthwise half of the paper's depthwise-separable layers, Sec. 4.2).
 *
 * Conventions for every call:
 *   - every call returns a disco_status_t; on failure nothing is enqueued on
 *     the stream and no output is written; disco_last_error() then holds a
 *     human-readable reason (thread-local, valid until the next call on the
 *     same thread);
 *   - tensors are dense, contiguous, row-major, on the device that created the
 *     plan; x, w and y must share one dtype (fp32, or bf16 storage with fp32
 *     accumulation); y must not overlap x or w and is fully overwritten;
 *   - the caller owns x, w and y and keeps them alive until the work enqueued
 *     on `stream` has completed; execution errors surface at the caller's next
 *     synchronisation, as usual in HIP;
 *   - a plan is immutable after creation and may be used from several host
 *     threads and streams at once.
 */
#ifndef DISCO_H
#define DISCO_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct disco_plan* disco_plan_t; /* opaque; owns the device psi tensors */

typedef enum {
    DISCO_OK = 0,
    DISCO_ERR_INVALID_ARGUMENT = 1, /* bad sizes, cutoff, null pointer, overlap */
    DISCO_ERR_UNSUPPORTED = 2,      /* valid but not implemented (longitude ratio, basis) */
    DISCO_ERR_SHAPE = 3,            /* tensor rank or shape does not match the plan */
    DISCO_ERR_DTYPE = 4,            /* mixed or unknown dtypes */
    DISCO_ERR_OUT_OF_MEMORY = 5,    /* device or host allocation failed */
    DISCO_ERR_DEVICE = 6            /* HIP runtime error, or tensor on another device */
} disco_status_t;

typedef enum { DISCO_FLOAT32 = 0, DISCO_BFLOAT16 = 1 } disco_dtype_t;

enum { DISCO_BASIS_BILINEAR_3X3 = 0,                /* K = 9 (App. E.2) */
       DISCO_BASIS_AXISYMMETRIC_4 = 1,               /* K = 4 (Sec. 3.4, App. B) */
       DISCO_BASIS_SEPARABLE_4X4 = 2 };              /* K = 16 (Sec. 3.4, App. E) */
/* Quadrature: 0 = the sampling-theorem weights of the grid (Sec. 4.1): Fejer's
 * first rule in cos(theta) on the cell-centred grid, App. A's weights on the
 * pole-including grid; 1 = cell areas (cell-centred grid only). */
enum { DISCO_QUAD_FEJER1 = 0, DISCO_QUAD_SAMPLING_THEOREM = 0, DISCO_QUAD_CELL_AREA = 1 };
enum { DISCO_SAMPLING_CELL_CENTRED = 0, DISCO_SAMPLING_POLES = 1 };

/* Execution variants.  AUTO picks the fastest path for the plan and shapes;
 * the others force one path (all give the same result up to fp32 rounding). */
typedef enum {
    DISCO_ALGO_AUTO = 0,
    DISCO_ALGO_GATHER_THEN_CONTRACT = 1, /* psi gather -> Z workspace -> W contraction */
    DISCO_ALGO_CONTRACT_THEN_GATHER = 2, /* W contraction on the input grid -> psi gather */
    DISCO_ALGO_FUSED = 3,       /* gather and contraction in one kernel; rings whose windows
                                   wrap whole input rings take the exact spectral (DFT) form */
    DISCO_ALGO_FUSED_DIRECT = 4, /* the fused kernel for every ring (no spectral form) */
    DISCO_ALGO_MATRIX_CORE = 5   /* bf16 storage, 3x3 basis: the gather and the contraction both on
                                    bf16 matrix cores, the values rounded to bf16 (Sec. 4.2, eq. 9);
                                    AUTO takes it for bf16 storage where the op allows it (at most two
                                    longitude phases, stride <= 4, nlon_in a multiple of 8, x 16-byte
                                    and y 4-byte aligned).  The first bf16 call of an op builds its
                                    tables (host packing and a synchronous upload, once per op); a
                                    caller that captures graphs makes one such call first.  The
                                    non-allocating entry point uses the tables only once built. */
} disco_algo_t;

typedef struct {
    int32_t kind;        /* DISCO_BASIS_BILINEAR_3X3, _AXISYMMETRIC_4 or _SEPARABLE_4X4 */
    int32_t quadrature;  /* DISCO_QUAD_SAMPLING_THEOREM (default) or DISCO_QUAD_CELL_AREA */
    double node_spacing; /* h in radians; 0 selects theta_c / 3 (3x3) or theta_c / 4 (the others) */
    int32_t sampling;    /* DISCO_SAMPLING_CELL_CENTRED (default) or DISCO_SAMPLING_POLES */
    int32_t flags;       /* 0, DISCO_PLAN_BACKWARD, DISCO_PLAN_EAGER or both */
} disco_basis_t;

/* Plan flags.  DISCO_PLAN_BACKWARD: also prepare the adjoint ops that
 * disco_forward_backward and disco_transpose_backward need.
 * Layouts: plan creation packs every layout of every op on the host but puts
 * on the device only what disco_forward with DISCO_ALGO_AUTO runs on; the
 * first call that runs on another layout (the transposed op, the adjoints,
 * another algo, depthwise calls of the 3x3 basis) uploads it, with
 * synchronous copies, once per plan.  DISCO_PLAN_EAGER uploads everything
 * at creation (for callers that capture graphs or must not see the first
 * call's upload); the bf16 matrix-core tables are built by the first bf16
 * call in either case. */
enum { DISCO_PLAN_BACKWARD = 1, DISCO_PLAN_EAGER = 2 };

typedef struct {
    void* data;       /* device pointer (may be NULL only when the tensor is empty) */
    int32_t dtype;    /* disco_dtype_t */
    int32_t ndim;     /* x, y: 4 ([B, C, nlat, nlon]); w: 3 ([C0, C1, K]), or 2 ([C, K]) depthwise */
    int64_t shape[4];
} disco_tensor_t;

typedef struct {
    int32_t K;                 /* basis size (9, 4 or 16) */
    int32_t nlat_in, nlon_in, nlat_out, nlon_out;
    int32_t phases_forward;    /* longitude phases of the forward op's patterns */
    int32_t phases_transpose;  /* ... and of the transposed op's */
    int32_t max_window;        /* widest stored longitude window, in input pixels */
    int32_t full_ring_windows; /* (pattern, input ring) pairs whose window is a whole ring */
    int64_t nnz_entries;       /* stored (pattern, input pixel) entries, forward op */
    int64_t nnz_entries_transpose;
    int64_t nnz_pairs_total;   /* non-zero (output pixel, input pixel, k) triples, forward */
    int64_t psi_bytes;         /* device bytes the plan holds now (see DISCO_PLAN_EAGER) */
    double h;                  /* node spacing actually used */
    int32_t spectral_rings_forward;   /* output rings of the forward op on the spectral path */
    int32_t spectral_rings_transpose; /* ... of the transposed op */
    int32_t sweep_patterns_forward;   /* (ring, phase) patterns of the forward op walked by the
                                         ring-sweep kernel (used when Cin <= 8) */
    int32_t sweep_patterns_transpose; /* ... of the transposed op */
    int32_t spectral_pairs_forward;   /* (spectral output ring, input ring) pairs of the forward op:
                                         one frequency-domain product per pair and frequency */
    int32_t spectral_pairs_transpose; /* ... of the transposed op */
    int32_t spectral_slots_forward;   /* input rings the forward op's spectral rings transform */
    int32_t spectral_slots_transpose; /* ... of the transposed op */
    /* Memory (App. B counts the non-zeros of Psi): the compressed psi of the
     * forward op in its plain form (per stored entry an input ring, a
     * longitude offset and K fp32 values, plus one pointer per pattern), and
     * the device bytes of each kernel layout the plan holds, summed over its
     * ops (psi_bytes is their total). */
    int64_t psi_compressed_bytes;
    int64_t bytes_entries;     /* the plain entry tables (two-kernel and contract-first schedules) */
    int64_t bytes_general;     /* the general fused kernel's chunked layouts */
    int64_t bytes_spectral;    /* the polar rings' frequency-domain psi rows and twiddles */
    int64_t bytes_sweep;       /* the ring sweep's runs, spans and entries */
    int64_t bytes_stencil;     /* the folded-weight stencil layouts */
    int64_t bytes_matrix_core; /* the bf16 matrix-core tables (built by the first bf16 call) */
    int64_t psi_bytes_all_layouts; /* device bytes once every layout of every op is built
                                      (matrix-core tables excluded) */
    int32_t spectral_tables_forward;   /* frequency-domain psi tables of the forward op's pairs:
                                          a pair mirrored about the equator from an earlier one
                                          shares that pair's table */
    int32_t spectral_tables_transpose; /* ... of the transposed op */
} disco_plan_info_t;

/* Builds the sparse psi tensors of the forward and transposed ops on the host
 * in fp64 (per output ring: neighbour search over input rings within theta_c,
 * closed-form longitude window, rotation, basis, quadrature; Sec. 4.1 and
 * 4.2), rounds them to fp32 and uploads them to the current device.
 *   nlat_* >= 1, nlon_* >= 2, 0 < theta_c <= pi; basis may be NULL (defaults);
 *   each op has at most 65535 (output ring, longitude phase) patterns.
 *   The pole-including sampling needs nlat >= 2 and nlon = 2 (nlat - 1) on
 *   both grids.
 * Errors: INVALID_ARGUMENT (sizes, cutoff, negative node spacing, unknown
 * flags, NULL plan_out), UNSUPPORTED (longitude ratio not an
 * integer, unknown basis, sampling or quadrature, cell areas on the
 * pole-including grid), OUT_OF_MEMORY, DEVICE.  On success *plan_out owns the device
 * memory until disco_plan_destroy.
 * With DISCO_LOG=1 in the environment the plan's statistics go to stderr
 * (per op: patterns, stored entries, non-zero triples, the largest window,
 * full-ring windows, compressed psi; then the schedule's structure, device
 * bytes and build time).  This call, the ops and the gradients each run
 * inside a roctx range named after them (rocprofv3 --marker-trace). */
disco_status_t disco_plan_create(int nlat_in, int nlon_in, int nlat_out, int nlon_out,
                                 double theta_c, const disco_basis_t* basis,
                                 disco_plan_t* plan_out);

/* Frees the plan and its device memory (NULL is accepted).  The caller
 * must ensure no enqueued work still uses the plan. */
disco_status_t disco_plan_destroy(disco_plan_t plan);

/* Fills *info with the plan's sizes and counts (App. B counts the non-zeros
 * of Psi as the memory figure). */
disco_status_t disco_plan_query(disco_plan_t plan, disco_plan_info_t* info);

/* Forward op (Sec. 3.2 eq. 4 on SO(3)/SO(2), Sec. 4.2 compressed product):
 *   x [B, Cin, nlat_in, nlon_in], w [Cout, Cin, K], y [B, Cout, nlat_out, nlon_out].
 * B may be 0 (nothing is enqueued); B * max(Cin, Cout) <= 65535, channels
 * <= 4096.  Errors: INVALID_ARGUMENT, SHAPE, DTYPE, OUT_OF_MEMORY
 * (workspace), DEVICE. */
disco_status_t disco_forward(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                             disco_tensor_t* y, hipStream_t stream);

/* Transposed op (Sec. 3.5 eq. 6), used for upsampling:
 *   x [B, CinT, nlat_out, nlon_out], w [CinT, CoutT, K] (the same buffer as
 *   the forward op's W of the adjoint pair), y [B, CoutT, nlat_in, nlon_in].
 * With quadrature-weighted inner products it is the adjoint of the forward
 * op.  Errors as disco_forward. */
disco_status_t disco_transpose(disco_plan_t plan, const disco_tensor_t* x,
                               const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream);

/* Depthwise forward and transposed ops (Sec. 4.2, the depthwise half of a
 * depthwise-separable layer): each channel is filtered by its own filter,
 *   forward    y[b,c,j] = sum_k W[c,k] sum_i psi_k(R_j^{-1} w_i) q_in(i) x[b,c,i]
 *   transpose  y[b,c,i] = sum_k W[c,k] sum_j psi_k(R_j^{-1} w_i) q_out(j) x[b,c,j]
 * i.e. disco_forward / disco_transpose with W'[c][c'][k] = (c == c') W[c][k].
 *   x [B, C, op input grid], w [C, K], y [B, C, op output grid]; any basis;
 *   B * C <= 65535.
 * W is folded into psi per call (one FMA per stored entry and channel).
 * Errors as disco_forward (SHAPE for a w that is not [C, K]). */
disco_status_t disco_forward_depthwise(disco_plan_t plan, const disco_tensor_t* x,
                                       const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream);
disco_status_t disco_transpose_depthwise(disco_plan_t plan, const disco_tensor_t* x,
                                         const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream);

/* disco_forward / disco_transpose with an explicit execution variant
 * (disco_algo_t).  Same arguments, errors and results.  With the
 * axisymmetric and separable bases every variant runs the one schedule those
 * bases have (W folded into psi per call, see disco_kernel_work's "stencil"
 * row) except GATHER_THEN_CONTRACT and CONTRACT_THEN_GATHER, which return
 * UNSUPPORTED. */
disco_status_t disco_forward_algo(disco_plan_t plan, const disco_tensor_t* x,
                                  const disco_tensor_t* w, disco_tensor_t* y, hipStream_t stream,
                                  int32_t algo);
disco_status_t disco_transpose_algo(disco_plan_t plan, const disco_tensor_t* x,
                                    const disco_tensor_t* w, disco_tensor_t* y,
                                    hipStream_t stream, int32_t algo);

/* Gradients of the forward op (App. C) for a scalar loss with upstream
 * gradient dy = d loss / dy [B, Cout, nlat_out, nlon_out]:
 *   dx [B, Cin, nlat_in, nlon_in] = A^T dy, the product with Psi transposed
 *      in input and output coordinates:
 *      dx[b,ci,i] = sum_{co,k} W[co,ci,k] sum_j psi_k(R_j^{-1} w_i) q_in(i) dy[b,co,j];
 *   dw [Cout, Cin, K] = sum_{b,j} dy[b,co,j] Z[b,ci,k](j), Z the gathered
 *      sums of the forward op (the chain rule through the sparse values to
 *      the basis weights).
 * x [B, Cin, nlat_in, nlon_in] is the forward input (read for dw only), w the
 * forward weights (read for dx only).  dx or dw may be NULL (not computed);
 * dx is overwritten, dw is overwritten (not accumulated; zeros for B = 0).
 * dx must not overlap dy or w, dw none of x, dy and dx, and when dw is asked
 * for dx must not overlap x either (dx may be written while x is read for
 * dw: with both asked for, dw's pass runs on a plan-owned helper stream
 * beside dx's, forked from stream and joined back into it, so the call's
 * work is complete when stream's is).  The plan must have
 * been created with DISCO_PLAN_BACKWARD.  dw is reduced over pixels in a fixed
 * order (deterministic); with bf16 storage the gathered sums are rounded to
 * bf16 before the reduction, which accumulates in fp32; dw needs
 * B * Cin * K <= 65535 (the input channels of dw's layout).  Errors as
 * disco_forward, and UNSUPPORTED for a plan without DISCO_PLAN_BACKWARD. */
disco_status_t disco_forward_backward(disco_plan_t plan, const disco_tensor_t* x,
                                      const disco_tensor_t* w, const disco_tensor_t* dy,
                                      disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream);

/* Gradients of the transposed op: dy [B, CoutT, nlat_in, nlon_in],
 * xT [B, CinT, nlat_out, nlon_out], w [CinT, CoutT, K];
 *   dx [B, CinT, nlat_out, nlon_out]:
 *      dx[b,c',j] = sum_{c,k} W[c',c,k] sum_i psi_k(R_j^{-1} w_i) q_out(j) dy[b,c,i];
 *   dw [CinT, CoutT, K] = sum_{b,i} dy[b,c,i] Z'[b,c',k](i).
 * Same conventions and errors as disco_forward_backward. */
disco_status_t disco_transpose_backward(disco_plan_t plan, const disco_tensor_t* x,
                                        const disco_tensor_t* w, const disco_tensor_t* dy,
                                        disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream);

/* Gradients of the depthwise ops (disco_forward_depthwise and
 * disco_transpose_depthwise; App. C applied to each channel's one-channel op):
 *   dx [B, C, op input grid]: dx[b,c] = A_c^T dy[b,c] with A_c the one-channel op of filter W[c],
 *      the adjoint of the depthwise op (the same as disco_forward_backward's
 *      dx with the diagonal W'[c][c'][k] = (c == c') W[c][k]);
 *   dw [C, K]:  dw[c,k] = sum_{b,j} dy[b,c,j] Z[b,c,k](j), Z the gathered sums
 *      of channel c (the diagonal blocks of the full weight gradient).
 * x [B, C, op input grid] is the depthwise op's input (read for dw only), w
 * [C, K] its weights (read for dx only), dy [B, C, op output grid]; dx or dw
 * may be NULL.  Same conventions as disco_forward_backward (plan created with
 * DISCO_PLAN_BACKWARD, dw reduced in a fixed order, overwritten, bf16 sums
 * rounded before the fp32 reduction); B * C * K <= 65535 when dw is asked
 * for.  Errors as disco_forward_backward. */
disco_status_t disco_forward_depthwise_backward(disco_plan_t plan, const disco_tensor_t* x,
                                                const disco_tensor_t* w, const disco_tensor_t* dy,
                                                disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream);
disco_status_t disco_transpose_depthwise_backward(disco_plan_t plan, const disco_tensor_t* x,
                                                  const disco_tensor_t* w, const disco_tensor_t* dy,
                                                  disco_tensor_t* dx, disco_tensor_t* dw, hipStream_t stream);

/* disco_forward for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, result and errors as disco_forward, except that the
 * kernels' scratch memory (the spectral rings' transforms, the fp32 partial
 * outputs of channel groups and of split patterns) comes from one fixed
 * device array of 64 MiB (67108864 bytes) per GPU, which the library holds
 * from the first call on that GPU until the process ends, and that the
 * spectral rings run on `stream` itself instead of beside it.  The call
 * allocates nothing (no hipMalloc, hipMallocAsync, hipFree or event).  A call
 * that needs more scratch than that (2048 x 4096 with 8 -> 8 channels and
 * batch 1 needs about 43 MB) fails with DISCO_ERR_UNSUPPORTED, naming both
 * sizes, before anything is enqueued.  Every call on one GPU shares that
 * GPU's array: calls that overlap in time on one GPU (several streams or
 * host threads) race and must be serialised by the caller.  Every kernel
 * writes the part of the array it reads before reading it, so nothing needs
 * clearing between calls. */
disco_status_t disco_forward_noalloc(disco_plan_t plan, const disco_tensor_t* x, const disco_tensor_t* w,
                                     disco_tensor_t* y, hipStream_t stream);

/* Host-only export of the stored psi entries of one op, without any device
 * (Sec. 4.1: Psi is constructed explicitly, only where it is non-zero).
 * transpose = 0 selects the forward op, 1 the transposed op.  Each entry is
 * (output ring, phase, input ring, longitude offset d, and a row of values:
 * 9 for the 3x3 basis, psi_0..8; 9 for the axisymmetric one, psi_0..3 then
 * five zeros; 16 for the separable one, psi_0..15); an output
 * pixel p_out = P * q + phase reads input pixel (stride * q + d) mod nlon of
 * the op's input grid, with P = phases and stride = nlon_in_op * P /
 * nlon_out_op.  Values are psi_k times the quadrature weight of the op's
 * input ring, rounded to fp32.  If capacity < *count the arrays are left
 * untouched and only *count, *phases and *stride are written (call with
 * capacity 0 to size the buffers).  Errors as disco_plan_create except
 * DEVICE, which cannot occur. */
disco_status_t disco_psi_entries(int nlat_in, int nlon_in, int nlat_out, int nlon_out,
                                 double theta_c, const disco_basis_t* basis, int32_t transpose,
                                 int64_t capacity, int32_t* out_ring, int32_t* phase,
                                 int32_t* in_ring, int32_t* offset, float* values,
                                 int64_t* count, int32_t* phases, int32_t* stride);

/* Kernel timing for measurement tools.  While enabled (on != 0), every
 * kernel the library launches from this process is bracketed by HIP events
 * recorded on the call's stream; disco_kernel_timing_read waits for the
 * recorded events, returns per-kernel totals (kernel name, launches,
 * milliseconds) for up to `capacity` kernels, writes the number of distinct
 * kernels to *count and clears the record.  names receives capacity rows of
 * 64 chars.  Enabling adds two event records per launch; disable it for
 * production use.  Errors: INVALID_ARGUMENT (NULL count), DEVICE. */
disco_status_t disco_kernel_timing_enable(int32_t on);
disco_status_t disco_kernel_timing_read(int32_t capacity, char* names, int64_t* launches,
                                        double* total_ms, int32_t* count);

/* Range checks of the psi indices, for a library built with
 * DISCO_DEBUG_BOUNDS (python -m paper_2209_13603_amd.build --debug-bounds
 * writes libdisco_debug_bounds.so): the kernels check every LDS index they
 * derive from the stored entries (input columns, entry slots, staged
 * elements) against the buffer it indexes and record a failure.  Waits for
 * the current device, then returns the number of kernel files (sweep,
 * general, matrix-core, stencil) that recorded one since the last call and
 * clears them; -1 for a library built without the checks. */
int32_t disco_debug_bounds_violations(void);

/* Algorithmic work of the kernels that one call of disco_forward_algo
 * (transpose == 0) or disco_transpose_algo (transpose != 0) with `algo`,
 * c_in input and c_out output channels and element type `dtype` launches on
 * this plan, for measurement tools (the dispatch is the one those calls
 * make).  Row i names the kernel as disco_kernel_timing_read does (64 chars
 * per row in `names`) and gives, per batch item and per channel:
 * out_pixels[i], the output pixels the kernel writes; in_pixels[i], the
 * distinct input pixels it reads; pairs[i], the non-zero (output pixel,
 * input pixel, k) triples of the sparse tensor (Sec. 4.1 eq. 7, of the
 * forward or the transposed op) whose products it accounts for (for the
 * "stencil" and "stencil_blocked" rows of the axisymmetric and separable
 * bases, whose psi has W folded in, the (output pixel, input pixel) pairs
 * instead; with these two bases a depthwise call runs the rows of
 * c_in = c_out = 1 once per channel).  A kernel
 * that only moves intermediate data reports zeros where it touches neither
 * x nor y.  Up to `capacity` rows are written (any output pointer may be
 * NULL) and *count receives the number of kernels.  Host only, no device
 * call.  Errors: INVALID_ARGUMENT (NULL plan or count, unknown algo), SHAPE
 * (channel count < 1), DTYPE (unknown dtype). */
disco_status_t disco_kernel_work(disco_plan_t plan, int32_t transpose, int32_t algo, int32_t c_in,
                                 int32_t c_out, int32_t dtype, int32_t capacity, char* names,
                                 int64_t* out_pixels, int64_t* in_pixels, int64_t* pairs, int32_t* count);

/* Static text for a status code (never NULL). */
const char* disco_status_string(disco_status_t status);

/* Detail of the last failed call on this thread ("" if none). */
const char* disco_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DISCO_H */
