/*
 * costa.h -- C ABI of the MI355X (gfx950) layout-transform library.
 *
 * The library computes the COSTA operation (Section 5, equation eq:costa)
 *
 *     A <- alpha * op(B) + beta * A,      op in {N (identity), T (transpose),
 *                                                C (conjugate transpose)}
 *
 * between two arbitrary grid layouts of the same P processes (Section 5,
 * "Matrix Layout"; Section 6, Figure 1).  On one GPU the P processes are
 * P virtual ranks: each rank's local matrix is a separate device buffer.
 * The exchange of packages between ranks (Algorithm 3) becomes a pack of the
 * remote blocks into per-(sender, receiver) message buffers in HBM and an
 * unpack-transform out of them; blocks whose sender is also their (relabeled)
 * receiver take a direct path without a message buffer (Section 6,
 * "Overlap of Communication and Computation").
 *
 * Conventions used throughout:
 *   - Every call returns a costa_status; nothing throws across the boundary.
 *     A detail string for the last error of the calling thread is available
 *     from costa_last_error().
 *   - Matrices and grids are described by global indices; element counts and
 *     offsets are int64, in elements (not bytes).
 *   - Sender of an element = its owner in the layout of B; receiver = its
 *     owner (its "label") in the layout of A.
 *   - A relabeling sigma (Section 4.1) is an int32 array of P entries:
 *     sigma[t] = physical rank that takes target label t.  NULL = identity.
 *   - Device pointers are HIP device addresses on the current device.  The
 *     caller owns every A/B buffer; the library owns its plans, work lists
 *     and message buffers (released by costa_finalize()).
 *   - Scalars alpha and beta are read on the host at call time, with the
 *     element type of the transform (double, double[2] for complex128,
 *     float, float[2] for complex64).
 *
 * Element arithmetic (the same reading as the test oracle):
 *   beta == 0           : A is not read (a NaN in A does not propagate);
 *   alpha == 1, beta == 0 : A = op(B) exactly (nothing to scale);
 *   otherwise           : t1 = alpha*op(b); t2 = beta*a; A = t1 + t2, each
 *                         product and sum rounded on its own (no FMA);
 *                         complex x*y = (xr*yr - xi*yi, xr*yi + xi*yr).
 *   conjugation flips the sign bit of the imaginary part (exact).
 */
#ifndef COSTA_H
#define COSTA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COSTA_SUCCESS = 0,
  COSTA_ERROR_INVALID_VALUE = 1,  /* bad argument: null pointer, bad splits/owners/op/dtype */
  COSTA_ERROR_SHAPE_MISMATCH = 2, /* A is not the shape of op(B), or the process counts differ */
  COSTA_ERROR_OUT_OF_MEMORY = 3,  /* not even one wave of message buffers fits on the device */
  COSTA_ERROR_DEVICE = 4,         /* a HIP call failed */
  COSTA_ERROR_NOT_SUPPORTED = 5   /* a valid request the library does not handle */
} costa_status;

/* op of equation (eq:costa); for real types C equals T. */
/* The enumerations a caller passes in end with an *_INT32 member that no call
 * accepts: it makes every int32 value a value of the type, so an unknown value
 * passed through the ABI is reported as COSTA_ERROR_INVALID_VALUE rather than
 * being undefined. */
typedef enum { COSTA_OP_N = 0, COSTA_OP_T = 1, COSTA_OP_C = 2, COSTA_OP_INT32 = 0x7fffffff } costa_op;

/* Storage order of blocks (Figure 1 "ordering"), or rank order of a process grid. */
typedef enum { COSTA_COL_MAJOR = 0, COSTA_ROW_MAJOR = 1, COSTA_ORDER_INT32 = 0x7fffffff } costa_order;

/* Element type (Section 6: arbitrary types through templates). */
typedef enum { COSTA_R64 = 0, COSTA_C128 = 1, COSTA_R32 = 2, COSTA_C64 = 3, COSTA_DTYPE_INT32 = 0x7fffffff } costa_dtype;

/* Opaque, immutable layout L(A) = (Grid_A, P, Owners_A) plus the local view. */
typedef struct costa_layout_s* costa_layout;

/* ---------------------------------------------------------------------------
 * Layouts (Section 5 "Matrix Layout"; Section 6 Figure 1)
 * ------------------------------------------------------------------------- */

/* General grid layout of an nrows x ncols matrix over nranks processes.
 *   row_splits : nbr+1 strictly increasing values, row_splits[0] = 0,
 *                row_splits[nbr] = nrows; block row bi = [rs[bi], rs[bi+1]).
 *                (nbr = 0 is allowed only when nrows = 0.)  Same for columns.
 *   owners     : nbr*nbc ranks in [0, nranks), row-major over (bi, bj).
 *   block_order: storage order of every block in its owner's buffer.
 *   block_offset, block_ld : nbr*nbc values each (row-major over blocks): the
 *                element offset of the block's first element inside its
 *                owner's buffer and its leading dimension (>= the block's
 *                extent along the contiguous direction).  Both NULL: default
 *                packing -- each rank stores its blocks one after another in
 *                row-major order of (bi, bj), each block packed with its own
 *                extent as leading dimension.  Blocks of one rank must not
 *                overlap in memory (not checked).
 * The arrays are copied; the caller keeps ownership.  *out is set on success
 * and must be released with costa_layout_destroy(). */
costa_status costa_layout_create(int64_t nrows, int64_t ncols, int32_t nbr, const int64_t* row_splits,
                                 int32_t nbc, const int64_t* col_splits, const int32_t* owners,
                                 int32_t nranks, costa_order block_order, const int64_t* block_offset,
                                 const int64_t* block_ld, costa_layout* out);

/* Block-cyclic (ScaLAPACK) layout: mb x nb blocks dealt cyclically over a
 * prow x pcol process grid, first process row/column 0 (for other first
 * processes and leading dimensions, costa_layout_create_scalapack()).  rank_order gives
 * rank = pr*pcol + pc (ROW_MAJOR) or pr + pc*prow (COL_MAJOR).  Local storage
 * is the ScaLAPACK local matrix of each rank, stored in block_order with
 * leading dimension max(1, local rows) (COL_MAJOR) or max(1, local cols)
 * (ROW_MAJOR).  Section 5 "Matrix Layout" with the splits at multiples of the
 * block size. */
costa_status costa_layout_create_block_cyclic(int64_t nrows, int64_t ncols, int64_t mb, int64_t nb,
                                              int32_t prow, int32_t pcol, costa_order rank_order,
                                              costa_order block_order, costa_layout* out);

/* A BLACS-style process grid: nprow x npcol processes out of `nranks`
 * ranks in all (0: exactly nprow*npcol).  Without a map the process at grid
 * position (pr, pc) is rank pr*npcol + pc (rank_order ROW_MAJOR, BLACS
 * "Row") or pr + pc*nprow (COL_MAJOR).  rank_map (may be NULL): nprow*npcol
 * distinct ranks in [0, nranks), column-major over the grid like a BLACS user
 * map: the process at (pr, pc) is rank_map[pr + pc*nprow]; rank_order is then
 * not read.  Ranks outside the grid hold nothing of the matrix.  The map is
 * copied by the calls that take a grid. */
typedef struct {
  int32_t nprow;
  int32_t npcol;
  costa_order rank_order;
  int32_t nranks;
  const int32_t* rank_map;
} costa_grid;

/* Layout of the matrix a ScaLAPACK array descriptor describes on `grid`:
 * desc[9] = {DTYPE_, CTXT_, M_, N_, MB_, NB_, RSRC_, CSRC_, LLD_}.  MB_ x NB_
 * blocks dealt cyclically, the first block row to process row RSRC_ and the
 * first block column to process column CSRC_; each rank stores its local
 * matrix column-major with leading dimension LLD_ (Section 5 "Matrix Layout"
 * with the splits at multiples of the block size; the local view of
 * Figure 1).  CTXT_ is not read: `grid` takes the place of the BLACS context.
 * One LLD_ serves every rank, so it must be >= max(1, local rows) of every
 * process row.  The layout has the grid's nranks ranks.  Errors:
 * NOT_SUPPORTED for DTYPE_ != 1; INVALID_VALUE for negative M_/N_, MB_/NB_ < 1,
 * RSRC_/CSRC_ outside the grid, LLD_ too small, nranks below nprow*npcol, a
 * rank map with entries out of range or repeated. */
costa_status costa_layout_create_scalapack(const int32_t* desc, const costa_grid* grid, costa_layout* out);

/* The m x n submatrix of `parent` whose first element is the parent's
 * element (i0, j0), 0-based (Section 5, "Scale and Transpose/Conjugate": a
 * submatrix is taken by truncating the row and column splits).  Every element
 * keeps its owner and its place in the owner's buffer, so the submatrix
 * layout addresses the parent's buffers; costa_layout_local_elems() of the
 * submatrix is the part of the parent's buffer it reaches (0 for a rank that
 * holds none of it).  The parent may be destroyed afterwards.  Errors:
 * INVALID_VALUE for a window outside the parent. */
costa_status costa_layout_submatrix(costa_layout parent, int64_t i0, int64_t j0, int64_t m, int64_t n,
                                    costa_layout* out);

/* Number of elements the buffer of `rank` must hold (0 if it owns nothing). */
costa_status costa_layout_local_elems(costa_layout layout, int32_t rank, int64_t* n);

/* Local view of one block (Figure 1): owner, element offset and leading
 * dimension.  Any output pointer may be NULL. */
costa_status costa_layout_block(costa_layout layout, int32_t bi, int32_t bj, int32_t* owner,
                                int64_t* offset, int64_t* ld);

/* Shape queries: any output pointer may be NULL. */
costa_status costa_layout_info(costa_layout layout, int64_t* nrows, int64_t* ncols, int32_t* nbr,
                               int32_t* nbc, int32_t* nranks, costa_order* block_order);

costa_status costa_layout_destroy(costa_layout layout);

/* ---------------------------------------------------------------------------
 * Communication volume and relabeling (Sections 2-4, Algorithms 1 and 2)
 * ------------------------------------------------------------------------- */

/* V_host[s*P + t] = number of elements that sender s (owner in L(B)) must
 * deliver to target label t (owner in L(A)) for A <- op(B): the package
 * volumes V(S_st) of Algorithm 2 in elements (multiply by the element size
 * for bytes, Section 2).  Computed on the device by the grid-overlay kernel
 * (Section 5 "Grid Overlay") on `stream`; the call synchronises `stream`
 * before returning.  V_host: P*P int64 host array, overwritten. */
costa_status costa_volume_matrix(costa_layout A, costa_layout B, costa_op op, int64_t* V_host,
                                 hipStream_t stream);

/* Communication-optimal process relabeling under the locally-free volume
 * cost (eq:locally_free_w): sigma maximises sum_t V[sigma[t]][t], which by the
 * gain remark (delta(p_x, p_y) = V(S_yx) - V(S_xx)), Lemma 2 and Theorems 1-2
 * minimises the total remote volume W(G_sigma).  Solved exactly on the host
 * (Hungarian algorithm, then among all optimal relabelings the
 * lexicographically smallest array sigma).  V_host: P*P int64, V[s*P+t] >= 0.
 * retained_identity / retained_sigma (may be NULL): local volume before and
 * after.  Host only; no device is needed. */
costa_status costa_relabel(int32_t P, const int64_t* V_host, int32_t* sigma, int64_t* retained_identity,
                           int64_t* retained_sigma);

/* Matching used for the relabeling (Section 4.3, Algorithm 1 "MWBPM"). */
typedef enum {
  COSTA_RELABEL_EXACT = 0,  /* Hungarian method: an optimal relabeling */
  COSTA_RELABEL_GREEDY = 1, /* the paper's greedy 2-approximation (Section 6): edges of G_delta
                               by decreasing gain (ties: smaller label, then smaller rank) are
                               taken while both ends are free; the identity when that perfect
                               matching's total gain is negative (gains can be) */
  COSTA_RELABEL_INT32 = 0x7fffffff
} costa_relabel_method;

/* Relabeling under a general communication cost (Section 3): a package s of
 * V(s) = V_host[i*P+j] * elem_bytes bytes sent from p_i to p_j costs
 *     w(p_i, p_j, s) = latency[i*P+j] + inv_bandwidth[i*P+j] * V(s)   (s non-empty),
 *     w = 0 for an empty package,
 * the latency-bandwidth model of the network-topology cost.  latency and
 * inv_bandwidth both NULL: the locally-free volume cost (eq:locally_free_w),
 * w = V(s) for i != j and 0 for i == j.  The gains delta(p_x, p_y) follow
 * eq:delta (sum over the left neighbours of p_x); sigma maximises
 * sum_t delta(p_t, p_sigma[t]) (Lemma 2), exactly or greedily.
 * cost_before / cost_after (may be NULL): W(G) and W(G_sigma) (def:WG).
 * Host only.  Errors: INVALID_VALUE for P < 0, null arrays, negative
 * volumes, non-finite or negative latency/bandwidth entries, unknown method. */
costa_status costa_relabel_cost(int32_t P, const int64_t* V_host, double elem_bytes, const double* latency,
                                const double* inv_bandwidth, costa_relabel_method method, int32_t* sigma,
                                double* cost_before, double* cost_after);

/* ---------------------------------------------------------------------------
 * The transform (Section 5 eq:costa and Algorithm 3; Section 6)
 * ------------------------------------------------------------------------- */

/* A <- alpha*op(B) + beta*A.  A is nrows x ncols of layout A; B is the same
 * shape for op N and the transposed shape otherwise; both layouts must have
 * the same number of ranks P.
 *   A_local : P device pointers, A_local[r] = buffer of PHYSICAL rank r, which
 *             holds the blocks of the label t with sigma[t] == r at the
 *             offsets layout A gives to label t.
 *   B_local : P device pointers, B_local[s] = buffer of rank s of layout B.
 * Buffers must hold costa_layout_local_elems() elements; a rank that owns
 * nothing may pass NULL.  A and B must not overlap.  Asynchronous on
 * `stream`; every argument error is returned before anything is enqueued.
 * The first call for a (layouts, op, sigma, type, whether beta is zero)
 * combination builds and caches a plan (host planning plus one upload).
 * Planning runs on up to 16 host threads, or on COSTA_PLAN_THREADS of them
 * when that environment variable is set (1: the calling thread only); the
 * plan does not depend on the count. */
costa_status costa_transform(costa_dtype dtype, costa_op op, const void* alpha, const void* beta,
                             costa_layout A, void* const* A_local, costa_layout B,
                             const void* const* B_local, const int32_t* sigma, hipStream_t stream);

/* One pair of a batched transform. */
typedef struct {
  costa_op op;
  const void* alpha;
  const void* beta;
  costa_layout A;
  void* const* A_local;
  costa_layout B;
  const void* const* B_local;
} costa_transform_desc;

/* n transforms of one element type as one job (Section 6 "Batched
 * Transformation"): one package per (sender, receiver) carries the blocks of
 * every pair, and each kernel launch covers all pairs.  One relabeling sigma
 * is shared by all pairs (a process is relabeled once).  All layouts must
 * have the same P. */
costa_status costa_transform_batched(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                     const int32_t* sigma, hipStream_t stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the batched
 * transform (same arguments, same results bit for bit as
 * costa_transform_batched) without any device or pinned-host allocation.
 * Its plan tables, the call's pointer table and the message buffers live in
 * one static device array of COSTA_NOALLOC_SCRATCH_BYTES per device, held
 * from the library's loading until the process ends: the first
 * COSTA_NOALLOC_TABLE_BYTES for the tables, the rest for the messages of one
 * wave (plans whose messages are larger run in more waves).  Nothing in the
 * array needs to start at zero.
 * Limits and errors: as costa_transform_batched(), plus NOT_SUPPORTED, returned
 * before any device work is enqueued, when the plan's rectangle and task
 * tables exceed COSTA_NOALLOC_TABLE_BYTES (very many rectangles or
 * workgroups; costa_transform_batched has no such limit).  No timing events
 * are recorded (costa_timing_enable does not cover this call).  Host memory
 * for planning and the plan cache comes from the C++ heap on the first call
 * of a (layouts, op, sigma, type) combination.
 * Every call on one device shares that device's array and keeps what the last
 * call left there: calls that overlap on one device (on different streams, or
 * from different threads without stream ordering) race and give undefined
 * results.  Calls on one stream are ordered by the stream. */
#define COSTA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
#define COSTA_NOALLOC_TABLE_BYTES ((size_t)16 << 20)
costa_status costa_transform_batched_noalloc(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                             const int32_t* sigma, hipStream_t stream);

/* Caps the message-buffer workspace.  A plan whose messages exceed the cap
 * is executed in waves (pack + unpack per wave).  0 = automatic (a share of
 * the free device memory at planning time).  Affects plans built afterwards. */
costa_status costa_set_workspace_limit(size_t bytes);

/* Statistics of the plan a transform with these arguments would use. */
typedef struct {
  int64_t total_elems;       /* sum over pairs of nrows*ncols */
  int64_t local_elems;       /* elements on the direct path (sender == receiver) */
  int64_t remote_elems;      /* elements through message buffers */
  int64_t model_bytes;       /* read B + read A (beta != 0) + write A + 2 * message bytes */
  int64_t message_bytes;     /* bytes written to (and read back from) message buffers */
  int64_t workspace_bytes;   /* size of the message workspace the plan needs */
  int64_t overlay_blocks;    /* blocks of the grid overlays, summed over pairs */
  int64_t pack_bytes;        /* algorithmic bytes of the pack kernels */
  int64_t unpack_bytes;      /* algorithmic bytes of the unpack-transform kernels */
  int64_t direct_bytes;      /* algorithmic bytes of the direct kernel */
  int32_t waves;             /* pack/unpack rounds */
  int32_t pieces_pack;       /* work rectangles of each kernel */
  int32_t pieces_unpack;
  int32_t pieces_direct;
  double plan_ms;            /* host time to build the plan */
} costa_stats;

/* Builds (or finds) the plan on the host only and reports it; no device work,
 * usable without a GPU.  alpha/beta of the descriptors may be NULL here
 * (beta is then taken as nonzero for the byte model). */
costa_status costa_plan_stats(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                              const int32_t* sigma, costa_stats* out);

/* One work rectangle of a plan, as the kernels see it (for inspection and
 * host-side checking of plans).  Coordinates follow the destination: x runs
 * along the destination's contiguous direction; dst(x, y) = dst_off +
 * y*dst_ld + x; the source is src_off + y*src_ld + x, or src_off + x*src_ld +
 * y when (flags & 1).  Buffer indices of a call with n pairs of P ranks:
 * A of pair k, physical rank r = k*P + r; B of pair k, rank s = n*P + k*P + s;
 * the message workspace = 2*n*P (offsets in elements). */
typedef struct {
  int32_t kind;   /* costa_kernel_kind: PACK, UNPACK or DIRECT */
  int32_t wave;   /* message round (0 for DIRECT) */
  int64_t group;  /* first workgroup of its launch that moves it */
  int64_t src_off, dst_off, src_ld, dst_ld;
  int32_t src_buf, dst_buf, nx, ny, item, flags;
  int64_t ntasks; /* workgroups that move it (LDS tiles or row-walk chunks); small
                     rectangles moved together by one workgroup report 1 each */
  int32_t tile_x, tile_y; /* LDS tile of a transposed rectangle (0 otherwise) */
  int32_t launch;         /* index of its kernel launch in the plan's launch order */
  int32_t reserved;
  int64_t wide_group;     /* launches of row walks only (else -1): its first task in the
                             launch's wide task table (tasks of 512 units, which the
                             launches that copy use) */
  int64_t wide_ntasks;    /* tasks of the wide table that move it (0 if none) */
} costa_piece_info;

/* Writes the rectangles of the plan a transform with these arguments would
 * use, in launch order (DIRECT, then PACK and UNPACK of each wave; a DIRECT
 * or UNPACK step that holds both transposed and other rectangles is two
 * launches, the transposed ones first), into
 * out[0..capacity); *count = their total number (call with capacity 0 to
 * size the array).  Host only; no device work. */
costa_status costa_plan_export(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                               const int32_t* sigma, costa_piece_info* out, int64_t capacity, int64_t* count);

/* ---------------------------------------------------------------------------
 * ScaLAPACK-compatible routines (Section 5: the operation eq:costa covers
 * pxgemr2d and pxtran(u/c); a submatrix by truncated splits)
 *
 * Arguments follow ScaLAPACK: 1-based global indices of each submatrix's
 * first element, 9-entry descriptors, m x n the shape of the destination
 * submatrix.  Each descriptor comes with its costa_grid in place of a BLACS
 * context, and each matrix is given as the P device pointers of its ranks
 * (P = the grid's nranks, the same for both grids, which may be grids of
 * different shapes over the same ranks, as for ScaLAPACK contexts within one
 * union context; NULL allowed for a rank that holds nothing of the
 * submatrix).  Elements land where the destination
 * descriptor puts them (no relabeling); elements outside the destination
 * submatrix are not touched.  m == 0 or n == 0: nothing is enqueued.
 * Asynchronous on `stream`.  The layouts of descriptor + submatrix pairs
 * (up to 1024 of them; past that the cache starts over) and the plans (up to
 * 32) are cached until costa_finalize(), so a repeated call only enqueues
 * kernels.  Errors: those of costa_layout_create_scalapack();
 * INVALID_VALUE for negative m/n, indices below 1 or submatrices past the
 * matrix, null pointers; SHAPE_MISMATCH when the grids have different nranks;
 * then those of costa_transform().
 * ------------------------------------------------------------------------- */

/* sub(B) = sub(A): B(ib+i, jb+j) = A(ia+i, ja+j) for 0 <= i < m, 0 <= j < n
 * (pxgemr2d for any element type; A is the source, B the destination). */
costa_status costa_pxgemr2d(costa_dtype dtype, int32_t m, int32_t n, const void* const* a, int32_t ia, int32_t ja,
                            const int32_t* desca, const costa_grid* grida, void* const* b, int32_t ib, int32_t jb,
                            const int32_t* descb, const costa_grid* gridb, hipStream_t stream);

/* sub(C) = beta*sub(C) + alpha*op(sub(A)), sub(C) m x n at (ic, jc), sub(A)
 * n x m at (ia, ja); op COSTA_OP_T (pxtran, pxtranu) or COSTA_OP_C (pxtranc).
 * alpha and beta point to one value of the element type (two for complex).
 * The element arithmetic is that of costa_transform(). */
costa_status costa_pxtran(costa_dtype dtype, costa_op op, int32_t m, int32_t n, const void* alpha,
                          const void* const* a, int32_t ia, int32_t ja, const int32_t* desca, const costa_grid* grida,
                          const void* beta, void* const* c, int32_t ic, int32_t jc, const int32_t* descc,
                          const costa_grid* gridc, hipStream_t stream);

/* The ScaLAPACK names: pdgemr2d and pdtran (double), pztranu and pztranc
 * (double complex; alpha and beta point to {re, im}). */
costa_status costa_pdgemr2d(int32_t m, int32_t n, const void* const* a, int32_t ia, int32_t ja, const int32_t* desca,
                            const costa_grid* grida, void* const* b, int32_t ib, int32_t jb, const int32_t* descb,
                            const costa_grid* gridb, hipStream_t stream);
costa_status costa_pdtran(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia, int32_t ja,
                          const int32_t* desca, const costa_grid* grida, const double* beta, void* const* c,
                          int32_t ic, int32_t jc, const int32_t* descc, const costa_grid* gridc, hipStream_t stream);
costa_status costa_pztranu(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia, int32_t ja,
                           const int32_t* desca, const costa_grid* grida, const double* beta, void* const* c,
                           int32_t ic, int32_t jc, const int32_t* descc, const costa_grid* gridc,
                           hipStream_t stream);
costa_status costa_pztranc(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia, int32_t ja,
                           const int32_t* desca, const costa_grid* grida, const double* beta, void* const* c,
                           int32_t ic, int32_t jc, const int32_t* descc, const costa_grid* gridc,
                           hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Kernel timing (HIP events around each launch, on the launch stream)
 * ------------------------------------------------------------------------- */
typedef enum { COSTA_KERNEL_PACK = 0, COSTA_KERNEL_UNPACK = 1, COSTA_KERNEL_DIRECT = 2,
               COSTA_KERNEL_VOLUME = 3, COSTA_KERNEL_KINDS = 4 } costa_kernel_kind;

typedef struct {
  double ms[COSTA_KERNEL_KINDS];        /* summed device time per kernel kind */
  int64_t launches[COSTA_KERNEL_KINDS]; /* number of launches */
  int64_t bytes[COSTA_KERNEL_KINDS];    /* summed algorithmic bytes */
} costa_timing;

/* on != 0: bracket every later launch with HIP events (2048 of them are
 * created here, on the current device, so that the timed calls do not create
 * them).  Resets the counters. */
costa_status costa_timing_enable(int on);
/* Waits for the recorded events, adds up their durations, returns the totals
 * since costa_timing_enable and keeps counting. */
costa_status costa_timing_read(costa_timing* out);

/* ---------------------------------------------------------------------------
 * Misc
 * ------------------------------------------------------------------------- */
/* Releases plans, workspaces and events (waits for the device first). */
costa_status costa_finalize(void);
const char* costa_status_string(costa_status status);
/* Detail of the last error on this thread ("" if none). */
const char* costa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* COSTA_H */
