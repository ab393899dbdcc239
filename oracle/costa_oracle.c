/*
 * CPU oracle for the COSTA layout transform.  TEST INFRASTRUCTURE ONLY: the
 * tests, the smoke check and the benchmark's CPU-baseline leg use it; the
 * product library never links or calls it, and it shares no code with it.
 *
 * Plain, slow and element-by-element on purpose.  Every global element (i, j)
 * of A is handled on its own: find its owner and address in each layout, read
 * op(B)(i, j), write alpha*op(B)(i,j) + beta*A(i,j).
 *
 * Paper passages followed:
 *   - the operation A = alpha*op(B) + beta*A, op in {N, T, C}: Section 5,
 *     equation (eq:costa);
 *   - the matrix layout L(A) = (Grid_A, P, Owners_A), block b_ij = rows
 *     [R(i), R(i+1)) x cols [C(j), C(j+1)): Section 5, "Matrix Layout";
 *   - the local view (each block with a pointer, a stride, dimensions and a
 *     row/col ordering): Section 6, Figure 1;
 *   - package volume V(s) = sum of block volumes: Section 2; packages S_ij
 *     built from the owners in both layouts: Section 5, Algorithm 2;
 *   - relabeled target: the receiver of package S_ij becomes p_sigma(j):
 *     Section 4.1, Definition of the relabeled graph, and Algorithm 3.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - sender of an element = its owner in L(B), receiver = its owner in L(A);
 *   - sigma[t] = physical rank that ends up holding target label t; the
 *     buffer of physical rank r therefore holds the blocks of label t with
 *     sigma[t] == r, at the addresses the layout of A gives to label t;
 *   - op(B) is B itself for N; for T and C, op(B)(i, j) = B(j, i), conjugated
 *     for C (C equals T for real types);
 *   - beta == 0: A is not read (BLAS convention); alpha == 1 and beta == 0:
 *     nothing to scale, A(i,j) = op(B)(i,j) exactly ("scale ... if needed",
 *     Algorithm 3); otherwise t1 = alpha*b, t2 = beta*a, result t1 + t2, each
 *     operation rounded on its own (built with -ffp-contract=off), complex
 *     products as (ar*br - ai*bi, ar*bi + ai*br);
 *   - block-cyclic local storage follows the ScaLAPACK convention (local
 *     rows from NUMROC, first block row/column on process row/column
 *     rsrc/csrc, leading dimension lld or the local extent);
 *   - a window (submatrix) keeps every element where the full layout stores
 *     it: taking a submatrix only truncates the splits (Section 5, "Scale and
 *     Transpose/Conjugate");
 *   - default storage of a general grid: a rank stores its blocks one after
 *     another in row-major order of (block row, block col), each block packed
 *     with its own leading extent.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "../synth/gen.h"

enum { O_BLOCK_CYCLIC = 0, O_GENERAL = 1 };
enum { O_OP_N = 0, O_OP_T = 1, O_OP_C = 2 };
enum { O_F64 = 0, O_C128 = 1, O_F32 = 2, O_C64 = 3 };

/* The oracle's own description of a layout.  Filled from Python. */
typedef struct {
  int32_t kind;
  int32_t row_major;      /* storage order of blocks (local matrix for block-cyclic) */
  int64_t nrows, ncols;
  int32_t nranks;
  /* block-cyclic */
  int64_t mb, nb;
  int32_t prow, pcol;
  int32_t rank_row_major; /* rank = pr*pcol + pc if set, else pr + pc*prow */
  /* general */
  int32_t nbr, nbc;
  const int64_t* rsplit;  /* nbr+1 */
  const int64_t* csplit;  /* nbc+1 */
  const int32_t* owners;  /* nbr*nbc, row-major over (bi, bj) */
  const int64_t* boff;    /* nbr*nbc element offsets inside the owner's buffer */
  const int64_t* bld;     /* nbr*nbc leading dimensions */
  /* block-cyclic, ScaLAPACK descriptor extras: process row/column holding the
   * first block row/column, and the local leading dimension (0: the local
   * extent from NUMROC, at least 1) */
  int32_t rsrc, csrc;
  int64_t lld;
  /* block-cyclic: process at grid position (pr, pc) is rank_map[pr + pc*prow]
   * (a BLACS-style map into nranks >= prow*pcol ranks; NULL: rank order) */
  const int32_t* rank_map;
} olayout;

/* ScaLAPACK NUMROC: how many of n rows (or cols), dealt in blocks of nb over
 * nprocs processes starting with process isrc, process iproc holds.  Its
 * distance from isrc along the cycle decides: the first n/nb full blocks go
 * round (nblocks/nprocs) full cycles, the next (nblocks mod nprocs) processes
 * get one more full block, and the one after them the partial last block. */
static int64_t numroc(int64_t n, int64_t nb, int64_t iproc, int64_t isrc, int64_t nprocs) {
  int64_t dist = (iproc - isrc + nprocs) % nprocs;
  int64_t nblocks = n / nb;
  int64_t num = (nblocks / nprocs) * nb;
  int64_t extra = nblocks % nprocs;
  if (dist < extra) num += nb;
  else if (dist == extra) num += n % nb;
  return num;
}

int64_t oracle_numroc(int64_t n, int64_t nb, int64_t iproc, int64_t isrc, int64_t nprocs) {
  return numroc(n, nb, iproc, isrc, nprocs);
}

/* Index k of the split interval [s[k], s[k+1]) containing x (binary search). */
static int32_t interval_of(const int64_t* s, int32_t nb, int64_t x) {
  int32_t lo = 0, hi = nb - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) / 2;
    if (s[mid] <= x) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

/* Owner rank and local element offset of global element (i, j). */
static void locate(const olayout* L, int64_t i, int64_t j, int32_t* rank, int64_t* off) {
  if (L->kind == O_BLOCK_CYCLIC) {
    /* block row i/mb lives on process row (rsrc + i/mb) mod prow, as the
     * (i/(mb*prow))-th block of that process row (ScaLAPACK INDXG2P and
     * INDXG2L); likewise for columns */
    int64_t pr = (i / L->mb + L->rsrc) % L->prow;
    int64_t pc = (j / L->nb + L->csrc) % L->pcol;
    if (L->rank_map) *rank = L->rank_map[pr + pc * L->prow];
    else *rank = (int32_t)(L->rank_row_major ? pr * L->pcol + pc : pr + pc * L->prow);
    int64_t li = (i / (L->mb * L->prow)) * L->mb + i % L->mb;
    int64_t lj = (j / (L->nb * L->pcol)) * L->nb + j % L->nb;
    if (L->row_major) {
      int64_t lc = numroc(L->ncols, L->nb, pc, L->csrc, L->pcol);
      int64_t ld = L->lld ? L->lld : (lc > 1 ? lc : 1);
      *off = li * ld + lj;
    } else {
      int64_t lr = numroc(L->nrows, L->mb, pr, L->rsrc, L->prow);
      int64_t ld = L->lld ? L->lld : (lr > 1 ? lr : 1);
      *off = li + lj * ld;
    }
  } else {
    int32_t bi = interval_of(L->rsplit, L->nbr, i);
    int32_t bj = interval_of(L->csplit, L->nbc, j);
    int64_t b = (int64_t)bi * L->nbc + bj;
    int64_t ri = i - L->rsplit[bi], cj = j - L->csplit[bj];
    *rank = L->owners[b];
    *off = L->boff[b] + (L->row_major ? ri * L->bld[b] + cj : ri + cj * L->bld[b]);
  }
}

/* Default storage of a general grid (see the header comment): fills boff/bld. */
int oracle_default_packing(int32_t nbr, int32_t nbc, const int64_t* rsplit, const int64_t* csplit,
                           const int32_t* owners, int32_t nranks, int32_t row_major, int64_t* boff,
                           int64_t* bld, int64_t* local_elems) {
  for (int32_t r = 0; r < nranks; ++r) local_elems[r] = 0;
  for (int32_t bi = 0; bi < nbr; ++bi)
    for (int32_t bj = 0; bj < nbc; ++bj) {
      int64_t b = (int64_t)bi * nbc + bj;
      int64_t h = rsplit[bi + 1] - rsplit[bi], w = csplit[bj + 1] - csplit[bj];
      int32_t r = owners[b];
      if (r < 0 || r >= nranks) return 1;
      boff[b] = local_elems[r];
      bld[b] = row_major ? w : h;
      local_elems[r] += h * w;
    }
  return 0;
}

/* Number of elements the buffer of `rank` must hold. */
int64_t oracle_local_elems(const olayout* L, int32_t rank) {
  if (L->kind == O_BLOCK_CYCLIC) {
    int64_t pr = -1, pc = -1;
    if (L->rank_map) {
      for (int64_t k = 0; k < (int64_t)L->prow * L->pcol; ++k)
        if (L->rank_map[k] == rank) { pr = k % L->prow; pc = k / L->prow; }
      if (pr < 0) return 0; /* not in the grid: holds nothing */
    } else {
      pr = L->rank_row_major ? rank / L->pcol : rank % L->prow;
      pc = L->rank_row_major ? rank % L->pcol : rank / L->prow;
    }
    int64_t lr = numroc(L->nrows, L->mb, pr, L->rsrc, L->prow);
    int64_t lc = numroc(L->ncols, L->nb, pc, L->csrc, L->pcol);
    if (lr == 0 || lc == 0) return 0;
    /* one past the last local element */
    if (L->row_major) return (lr - 1) * (L->lld ? L->lld : lc) + lc;
    return (lc - 1) * (L->lld ? L->lld : lr) + lr;
  }
  int64_t need = 0;
  for (int64_t b = 0; b < (int64_t)L->nbr * L->nbc; ++b) {
    if (L->owners[b] != rank) continue;
    int32_t bi = (int32_t)(b / L->nbc), bj = (int32_t)(b % L->nbc);
    int64_t h = L->rsplit[bi + 1] - L->rsplit[bi], w = L->csplit[bj + 1] - L->csplit[bj];
    int64_t end = L->row_major ? L->boff[b] + (h - 1) * L->bld[b] + w : L->boff[b] + (w - 1) * L->bld[b] + h;
    if (h > 0 && w > 0 && end > need) need = end;
  }
  return need;
}

/* Owner and offset of a list of points (for tests of the storage maps). */
void oracle_locate_many(const olayout* L, int64_t n, const int64_t* rows, const int64_t* cols, int32_t* rank,
                        int64_t* off) {
  for (int64_t k = 0; k < n; ++k) locate(L, rows[k], cols[k], &rank[k], &off[k]);
}

/* Element (i', j') of B that op(B)(i, j) reads. */
static void source_of(int op, int64_t i, int64_t j, int64_t* bi, int64_t* bj) {
  if (op == O_OP_N) { *bi = i; *bj = j; }
  else { *bi = j; *bj = i; }
}

/* Volume matrix by brute-force element counting (Section 2 volume, Algorithm 2
 * packages): V[s*P + t] += 1 for every element (i, j) of the m x n window of A
 * at (ia, ja) whose source, element op^-1(i, j) of the window of B at
 * (ib, jb), is owned by s in L(B), and which label t owns in L(A). */
int oracle_volume_window(const olayout* A, int64_t ia, int64_t ja, const olayout* B, int64_t ib, int64_t jb,
                         int64_t m, int64_t n, int op, int64_t* V) {
  int32_t P = A->nranks;
  if (B->nranks != P) return 1;
  memset(V, 0, sizeof(int64_t) * (size_t)P * (size_t)P);
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) {
      int32_t t, s;
      int64_t oa, ob, bi, bj;
      locate(A, ia + i, ja + j, &t, &oa);
      source_of(op, i, j, &bi, &bj);
      locate(B, ib + bi, jb + bj, &s, &ob);
      V[(int64_t)s * P + t] += 1;
    }
  return 0;
}

/* The volume matrix of the whole matrices. */
int oracle_volume(const olayout* A, const olayout* B, int op, int64_t* V) {
  return oracle_volume_window(A, 0, 0, B, 0, 0, A->nrows, A->ncols, op, V);
}

/* ---- element arithmetic, literally as equation (eq:costa) ---- */
typedef struct { double re, im; } cplx;

static cplx cmul(cplx a, cplx b) {
  cplx r;
  double p1 = a.re * b.re, p2 = a.im * b.im, p3 = a.re * b.im, p4 = a.im * b.re;
  r.re = p1 - p2;
  r.im = p3 + p4;
  return r;
}
static cplx cadd(cplx a, cplx b) {
  cplx r;
  r.re = a.re + b.re;
  r.im = a.im + b.im;
  return r;
}

/* One element: returns alpha*b + beta*a under the readings above. */
static cplx combine(int cpx, cplx alpha, cplx beta, cplx b, cplx a_old) {
  int alpha_one = alpha.re == 1.0 && alpha.im == 0.0;
  int beta_zero = beta.re == 0.0 && beta.im == 0.0;
  if (alpha_one && beta_zero) return b;
  cplx t1, t2;
  if (cpx) {
    t1 = cmul(alpha, b);
    if (beta_zero) return t1;
    t2 = cmul(beta, a_old);
    return cadd(t1, t2);
  }
  t1.re = alpha.re * b.re;
  t1.im = 0.0;
  if (beta_zero) return t1;
  t2.re = beta.re * a_old.re;
  t2.im = 0.0;
  return cadd(t1, t2);
}

/* 32-bit variant: every operation rounded to float. */
static void combine32(int cpx, const float* alpha, const float* beta, const float* b, const float* a_old,
                      float* out) {
  int alpha_one = alpha[0] == 1.0f && alpha[1] == 0.0f;
  int beta_zero = beta[0] == 0.0f && beta[1] == 0.0f;
  if (alpha_one && beta_zero) { out[0] = b[0]; if (cpx) out[1] = b[1]; return; }
  if (cpx) {
    float p1 = alpha[0] * b[0], p2 = alpha[1] * b[1], p3 = alpha[0] * b[1], p4 = alpha[1] * b[0];
    float t1r = p1 - p2, t1i = p3 + p4;
    if (beta_zero) { out[0] = t1r; out[1] = t1i; return; }
    float q1 = beta[0] * a_old[0], q2 = beta[1] * a_old[1], q3 = beta[0] * a_old[1], q4 = beta[1] * a_old[0];
    float t2r = q1 - q2, t2i = q3 + q4;
    out[0] = t1r + t2r;
    out[1] = t1i + t2i;
    return;
  }
  float t1 = alpha[0] * b[0];
  if (beta_zero) { out[0] = t1; return; }
  float t2 = beta[0] * a_old[0];
  out[0] = t1 + t2;
}

/* A window of A receives a window of op(B) (Section 5, "Scale and
 * Transpose/Conjugate": a submatrix is taken by truncating the splits, which
 * leaves every element where the full layout stores it):
 *     A(ia + i, ja + j) <- alpha * op(B~)(i, j) + beta * A(ia + i, ja + j),
 * for window rows i in [row_begin, row_end) and columns j in [0, n), where
 * B~ is the window of B starting at (ib, jb): op(B~)(i, j) = B(ib + i, jb + j)
 * for N, and B(ib + j, jb + i) for T and C.  Elements of A outside the window
 * are not touched.  alpha, beta: {re, im} (im ignored for real types).  sigma
 * may be NULL (identity).  A_local[r] / B_local[s]: host buffers of physical
 * ranks. */
int oracle_transform_window(int dtype, int op, const double* alpha, const double* beta, const olayout* A,
                            void* const* A_local, int64_t ia, int64_t ja, const olayout* B,
                            const void* const* B_local, int64_t ib, int64_t jb, int64_t n, const int32_t* sigma,
                            int64_t row_begin, int64_t row_end) {
  int cpx = dtype == O_C128 || dtype == O_C64;
  cplx al = {alpha[0], cpx ? alpha[1] : 0.0}, be = {beta[0], cpx ? beta[1] : 0.0};
  float al32[2] = {(float)alpha[0], cpx ? (float)alpha[1] : 0.0f};
  float be32[2] = {(float)beta[0], cpx ? (float)beta[1] : 0.0f};
  if (A->nranks != B->nranks) return 1;
  for (int64_t i = row_begin; i < row_end; ++i)
    for (int64_t j = 0; j < n; ++j) {
      int32_t t, s;
      int64_t oa, ob, bi, bj;
      locate(A, ia + i, ja + j, &t, &oa);
      int32_t r = sigma ? sigma[t] : t;
      source_of(op, i, j, &bi, &bj);
      locate(B, ib + bi, jb + bj, &s, &ob);
      if (dtype == O_F64 || dtype == O_C128) {
        const double* src = (const double*)B_local[s] + (cpx ? 2 * ob : ob);
        double* dst = (double*)A_local[r] + (cpx ? 2 * oa : oa);
        cplx b = {src[0], cpx ? src[1] : 0.0};
        if (op == O_OP_C && cpx) b.im = -b.im;
        cplx a_old = {0.0, 0.0};
        if (!(be.re == 0.0 && be.im == 0.0)) { a_old.re = dst[0]; a_old.im = cpx ? dst[1] : 0.0; }
        cplx res = combine(cpx, al, be, b, a_old);
        dst[0] = res.re;
        if (cpx) dst[1] = res.im;
      } else {
        const float* src = (const float*)B_local[s] + (cpx ? 2 * ob : ob);
        float* dst = (float*)A_local[r] + (cpx ? 2 * oa : oa);
        float b[2] = {src[0], cpx ? src[1] : 0.0f};
        if (op == O_OP_C && cpx) b[1] = -b[1];
        float a_old[2] = {0.0f, 0.0f};
        if (!(be32[0] == 0.0f && be32[1] == 0.0f)) { a_old[0] = dst[0]; a_old[1] = cpx ? dst[1] : 0.0f; }
        combine32(cpx, al32, be32, b, a_old, dst);
      }
    }
  return 0;
}

/* A <- alpha*op(B) + beta*A for the rows [row_begin, row_end) of A: the
 * window that is all of A and all of B. */
int oracle_transform(int dtype, int op, const double* alpha, const double* beta, const olayout* A,
                     void* const* A_local, const olayout* B, const void* const* B_local, const int32_t* sigma,
                     int64_t row_begin, int64_t row_end) {
  return oracle_transform_window(dtype, op, alpha, beta, A, A_local, 0, 0, B, B_local, 0, 0, A->ncols, sigma,
                                 row_begin, row_end);
}

/* Expected final A at sampled points, for inputs made by the seeded generator
 * (B of physical rank s: stream(B, item, s); initial A of physical rank r:
 * stream(A, item, r)).  out_val holds 2 doubles per point ({re, im}; for f32
 * and c64 the float values widened exactly).  Also returns where the point
 * lives: physical rank and element offset.  Points are given in the window
 * coordinates of oracle_transform_window. */
int oracle_expect_at_window(int dtype, int op, const double* alpha, const double* beta, const olayout* A,
                            int64_t ia, int64_t ja, const olayout* B, int64_t ib, int64_t jb, const int32_t* sigma,
                            uint64_t seed, uint32_t item, int64_t n, const int64_t* rows, const int64_t* cols,
                            int32_t* out_rank, int64_t* out_off, double* out_val) {
  int cpx = dtype == O_C128 || dtype == O_C64;
  int beta_zero = beta[0] == 0.0 && (!cpx || beta[1] == 0.0);
  for (int64_t k = 0; k < n; ++k) {
    int32_t t, s;
    int64_t oa, ob, bi, bj;
    locate(A, ia + rows[k], ja + cols[k], &t, &oa);
    int32_t r = sigma ? sigma[t] : t;
    source_of(op, rows[k], cols[k], &bi, &bj);
    locate(B, ib + bi, jb + bj, &s, &ob);
    uint64_t sb = synth_stream(SYNTH_ROLE_B, item, (uint32_t)s), sa = synth_stream(SYNTH_ROLE_A, item, (uint32_t)r);
    out_rank[k] = r;
    out_off[k] = oa;
    if (dtype == O_F64 || dtype == O_C128) {
      cplx b, a_old = {0.0, 0.0};
      cplx al = {alpha[0], cpx ? alpha[1] : 0.0}, be = {beta[0], cpx ? beta[1] : 0.0};
      if (cpx) { b.re = synth_c128_re(seed, sb, (uint64_t)ob); b.im = synth_c128_im(seed, sb, (uint64_t)ob); }
      else { b.re = synth_f64(seed, sb, (uint64_t)ob); b.im = 0.0; }
      if (op == O_OP_C && cpx) b.im = -b.im;
      if (!beta_zero) {
        if (cpx) { a_old.re = synth_c128_re(seed, sa, (uint64_t)oa); a_old.im = synth_c128_im(seed, sa, (uint64_t)oa); }
        else a_old.re = synth_f64(seed, sa, (uint64_t)oa);
      }
      cplx res = combine(cpx, al, be, b, a_old);
      out_val[2 * k] = res.re;
      out_val[2 * k + 1] = cpx ? res.im : 0.0;
    } else {
      float al32[2] = {(float)alpha[0], cpx ? (float)alpha[1] : 0.0f};
      float be32[2] = {(float)beta[0], cpx ? (float)beta[1] : 0.0f};
      float b[2], a_old[2] = {0.0f, 0.0f}, res[2] = {0.0f, 0.0f};
      if (cpx) { b[0] = synth_c64_re(seed, sb, (uint64_t)ob); b[1] = synth_c64_im(seed, sb, (uint64_t)ob); }
      else { b[0] = synth_f32(seed, sb, (uint64_t)ob); b[1] = 0.0f; }
      if (op == O_OP_C && cpx) b[1] = -b[1];
      if (!beta_zero) {
        if (cpx) { a_old[0] = synth_c64_re(seed, sa, (uint64_t)oa); a_old[1] = synth_c64_im(seed, sa, (uint64_t)oa); }
        else a_old[0] = synth_f32(seed, sa, (uint64_t)oa);
      }
      combine32(cpx, al32, be32, b, a_old, res);
      out_val[2 * k] = (double)res[0];
      out_val[2 * k + 1] = (double)res[1];
    }
  }
  return 0;
}

int oracle_expect_at(int dtype, int op, const double* alpha, const double* beta, const olayout* A, const olayout* B,
                     const int32_t* sigma, uint64_t seed, uint32_t item, int64_t n, const int64_t* rows,
                     const int64_t* cols, int32_t* out_rank, int64_t* out_off, double* out_val) {
  return oracle_expect_at_window(dtype, op, alpha, beta, A, 0, 0, B, 0, 0, sigma, seed, item, n, rows, cols,
                                 out_rank, out_off, out_val);
}

/* Host fill of a buffer with the generator (same values as the device fill). */
int oracle_fill(int dtype, void* dst, int64_t n, uint64_t seed, uint64_t stream) {
  for (int64_t i = 0; i < n; ++i) {
    switch (dtype) {
      case O_F64: ((double*)dst)[i] = synth_f64(seed, stream, (uint64_t)i); break;
      case O_C128:
        ((double*)dst)[2 * i] = synth_c128_re(seed, stream, (uint64_t)i);
        ((double*)dst)[2 * i + 1] = synth_c128_im(seed, stream, (uint64_t)i);
        break;
      case O_F32: ((float*)dst)[i] = synth_f32(seed, stream, (uint64_t)i); break;
      case O_C64:
        ((float*)dst)[2 * i] = synth_c64_re(seed, stream, (uint64_t)i);
        ((float*)dst)[2 * i + 1] = synth_c64_im(seed, stream, (uint64_t)i);
        break;
      default: return 1;
    }
  }
  return 0;
}
