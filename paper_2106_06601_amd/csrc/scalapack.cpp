// ScaLAPACK-compatible entry points.  A descriptor plus a 1-based submatrix
// becomes a submatrix layout (Section 5: a submatrix is taken by truncating
// the splits), and the call becomes one transform A <- alpha*op(B) + beta*A
// (Section 5, eq:costa, which covers pxgemr2d and pxtran).  The layouts are
// cached by descriptor, grid and window (a block-cyclic layout is a few
// hundred bytes, whatever the matrix size), so that repeated calls keep the
// same layouts and therefore find their cached plans; the cache holds at most
// kMaxCachedLayouts and starts over when a call would pass that, and
// costa_finalize empties it.
#include <map>
#include <mutex>

#include "internal.hpp"

namespace costa {
namespace {

// M_, N_, MB_, NB_, RSRC_, CSRC_, LLD_, nprow, npcol, rank order, nranks, i0,
// j0, m, n, then the rank map if there is one
using Key = std::vector<int64_t>;

// A call looks up two layouts; the cache starts over before a call whose two
// could pass the bound, never between its two lookups.
constexpr size_t kMaxCachedLayouts = 1024;

struct Cache {
  std::mutex mu;  // held for a whole call: its layouts stay alive until it returns
  std::map<Key, costa_layout> layouts;
};

void clear_locked(Cache& C) {
  for (auto& kv : C.layouts) costa_layout_destroy(kv.second);
  C.layouts.clear();
}

Cache& cache() {
  static Cache* c = new Cache();
  return *c;
}

costa_status check_desc(const char* name, const int32_t* desc, const costa_grid* grid) {
  if (!desc || !grid) return fail(COSTA_ERROR_INVALID_VALUE, std::string("null descriptor or grid of ") + name);
  return COSTA_SUCCESS;
}

// Layout of the rows x cols submatrix at 1-based (i1, j1) of the descriptor's
// matrix.  The caller holds the cache's lock.
costa_status window_layout(const char* name, const int32_t* desc, const costa_grid* grid, int32_t i1, int32_t j1,
                           int64_t rows, int64_t cols, costa_layout* out) {
  costa_status st = check_desc(name, desc, grid);
  if (st != COSTA_SUCCESS) return st;
  if (i1 < 1 || j1 < 1) return fail(COSTA_ERROR_INVALID_VALUE, std::string("indices of ") + name + " below 1");
  if ((int64_t)i1 - 1 + rows > desc[2] || (int64_t)j1 - 1 + cols > desc[3])
    return fail(COSTA_ERROR_INVALID_VALUE, std::string("submatrix of ") + name + " past the matrix");
  if (grid->nprow < 1 || grid->npcol < 1) return fail(COSTA_ERROR_INVALID_VALUE, "process grid must be at least 1x1");
  Key key{desc[2], desc[3], desc[4], desc[5], desc[6], desc[7], desc[8], grid->nprow, grid->npcol,
          (int64_t)grid->rank_order, grid->nranks, (int64_t)i1 - 1, (int64_t)j1 - 1, rows, cols};
  if (grid->rank_map) key.insert(key.end(), grid->rank_map, grid->rank_map + (size_t)grid->nprow * grid->npcol);
  Cache& C = cache();
  auto it = C.layouts.find(key);
  if (it != C.layouts.end()) {
    *out = it->second;
    return COSTA_SUCCESS;
  }
  if (desc[0] != 1) return fail(COSTA_ERROR_NOT_SUPPORTED, std::string("descriptor type of ") + name + " is not 1");
  costa_layout full = nullptr, sub = nullptr;
  st = costa_layout_create_scalapack(desc, grid, &full);
  if (st != COSTA_SUCCESS) return st;
  st = costa_layout_submatrix(full, (int64_t)i1 - 1, (int64_t)j1 - 1, rows, cols, &sub);
  costa_layout_destroy(full);
  if (st != COSTA_SUCCESS) return st;
  C.layouts.emplace(key, sub);
  *out = sub;
  return COSTA_SUCCESS;
}

// dst window (m x n) <- alpha * op(src window) + beta * dst window.
costa_status scalapack_transform(costa_dtype dtype, costa_op op, int32_t m, int32_t n, const void* alpha,
                                 const void* const* src, int32_t is, int32_t js, const int32_t* descs,
                                 const costa_grid* grids, const void* beta, void* const* dst, int32_t id,
                                 int32_t jd, const int32_t* descd, const costa_grid* gridd, hipStream_t stream) {
  if (m < 0 || n < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative m or n");
  costa_status st = check_desc("the source", descs, grids);
  if (st != COSTA_SUCCESS) return st;
  st = check_desc("the destination", descd, gridd);
  if (st != COSTA_SUCCESS) return st;
  auto world = [](const costa_grid* g) { return g->nranks ? (int64_t)g->nranks : (int64_t)g->nprow * g->npcol; };
  if (world(grids) != world(gridd))
    return fail(COSTA_ERROR_SHAPE_MISMATCH, "the two process grids live on different numbers of ranks");
  if (m == 0 || n == 0) return COSTA_SUCCESS;
  if (!src || !dst) return fail(COSTA_ERROR_INVALID_VALUE, "null buffer array");
  const bool tr = op != COSTA_OP_N;
  Cache& C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  if (C.layouts.size() + 2 > kMaxCachedLayouts) clear_locked(C);
  costa_layout ls = nullptr, ld = nullptr;
  st = window_layout("the source", descs, grids, is, js, tr ? n : m, tr ? m : n, &ls);
  if (st != COSTA_SUCCESS) return st;
  st = window_layout("the destination", descd, gridd, id, jd, m, n, &ld);
  if (st != COSTA_SUCCESS) return st;
  return costa_transform(dtype, op, alpha, beta, ld, dst, ls, src, nullptr, stream);
}

const void* one_of(costa_dtype dt) {
  static const double d1[2] = {1.0, 0.0};
  static const float f1[2] = {1.0f, 0.0f};
  return dt == COSTA_R32 || dt == COSTA_C64 ? (const void*)f1 : (const void*)d1;
}
const void* zero_of(costa_dtype dt) {
  static const double d0[2] = {0.0, 0.0};
  static const float f0[2] = {0.0f, 0.0f};
  return dt == COSTA_R32 || dt == COSTA_C64 ? (const void*)f0 : (const void*)d0;
}

}  // namespace

void release_scalapack_layouts() {
  Cache& C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  clear_locked(C);
}

}  // namespace costa

using namespace costa;

extern "C" costa_status costa_pxgemr2d(costa_dtype dtype, int32_t m, int32_t n, const void* const* a, int32_t ia,
                                       int32_t ja, const int32_t* desca, const costa_grid* grida, void* const* b,
                                       int32_t ib, int32_t jb, const int32_t* descb, const costa_grid* gridb,
                                       hipStream_t stream) {
  return guarded([&]() -> costa_status {
    if (dtype != COSTA_R64 && dtype != COSTA_C128 && dtype != COSTA_R32 && dtype != COSTA_C64)
      return fail(COSTA_ERROR_INVALID_VALUE, "unknown dtype");
    return scalapack_transform(dtype, COSTA_OP_N, m, n, one_of(dtype), a, ia, ja, desca, grida, zero_of(dtype), b, ib,
                               jb, descb, gridb, stream);
  });
}

extern "C" costa_status costa_pxtran(costa_dtype dtype, costa_op op, int32_t m, int32_t n, const void* alpha,
                                     const void* const* a, int32_t ia, int32_t ja, const int32_t* desca,
                                     const costa_grid* grida, const void* beta, void* const* c, int32_t ic,
                                     int32_t jc, const int32_t* descc, const costa_grid* gridc, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    if (op != COSTA_OP_T && op != COSTA_OP_C)
      return fail(COSTA_ERROR_INVALID_VALUE, "op must be T or C (pxgemr2d copies without transposing)");
    if (!alpha || !beta) return fail(COSTA_ERROR_INVALID_VALUE, "null alpha or beta");
    return scalapack_transform(dtype, op, m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc, stream);
  });
}

extern "C" costa_status costa_pdgemr2d(int32_t m, int32_t n, const void* const* a, int32_t ia, int32_t ja,
                                       const int32_t* desca, const costa_grid* grida, void* const* b, int32_t ib,
                                       int32_t jb, const int32_t* descb, const costa_grid* gridb, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    return costa_pxgemr2d(COSTA_R64, m, n, a, ia, ja, desca, grida, b, ib, jb, descb, gridb, stream);
  });
}

extern "C" costa_status costa_pdtran(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia,
                                     int32_t ja, const int32_t* desca, const costa_grid* grida, const double* beta,
                                     void* const* c, int32_t ic, int32_t jc, const int32_t* descc,
                                     const costa_grid* gridc, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    return costa_pxtran(COSTA_R64, COSTA_OP_T, m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                        stream);
  });
}

extern "C" costa_status costa_pztranu(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia,
                                      int32_t ja, const int32_t* desca, const costa_grid* grida, const double* beta,
                                      void* const* c, int32_t ic, int32_t jc, const int32_t* descc,
                                      const costa_grid* gridc, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    return costa_pxtran(COSTA_C128, COSTA_OP_T, m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                        stream);
  });
}

extern "C" costa_status costa_pztranc(int32_t m, int32_t n, const double* alpha, const void* const* a, int32_t ia,
                                      int32_t ja, const int32_t* desca, const costa_grid* grida, const double* beta,
                                      void* const* c, int32_t ic, int32_t jc, const int32_t* descc,
                                      const costa_grid* gridc, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    return costa_pxtran(COSTA_C128, COSTA_OP_C, m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                        stream);
  });
}
