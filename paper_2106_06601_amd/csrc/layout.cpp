// Layouts: the global grid (splits + owners) and the local view (per-block
// offset, leading dimension, ordering) of Section 5 "Matrix Layout" and
// Section 6 Figure 1.
#include <algorithm>
#include <atomic>
#include <climits>
#include <cstring>
#include <new>

#include "internal.hpp"

struct costa_layout_s {
  costa::Layout L;
};

namespace costa {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

costa_status fail(costa_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

static std::atomic<uint64_t> g_next_id{1};

static costa_status check_splits(const char* what, int64_t n, int32_t nb, const int64_t* s) {
  if (nb < 0) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": negative block count");
  if (n < 0) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": negative dimension");
  if (nb == 0) {
    if (n != 0) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": no blocks for a nonempty dimension");
    if (s && s[0] != 0) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": splits must start at 0");
    return COSTA_SUCCESS;
  }
  if (!s) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": null splits");
  if (s[0] != 0) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": splits must start at 0");
  if (s[nb] != n) return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": last split must equal the dimension");
  for (int32_t k = 0; k < nb; ++k)
    if (s[k + 1] <= s[k])
      return fail(COSTA_ERROR_INVALID_VALUE, std::string(what) + ": splits must be strictly increasing");
  return COSTA_SUCCESS;
}

// Fills local_elems from the per-block storage; checks offsets and strides.
static costa_status finish_layout(Layout& L) {
  L.local_elems.assign(L.nranks, 0);
  for (int32_t bi = 0; bi < L.nbr; ++bi)
    for (int32_t bj = 0; bj < L.nbc; ++bj) {
      int64_t b = L.block(bi, bj);
      int64_t h = L.rsplit[bi + 1] - L.rsplit[bi], w = L.csplit[bj + 1] - L.csplit[bj];
      int64_t fast = L.order == COSTA_COL_MAJOR ? h : w;
      int64_t slow = L.order == COSTA_COL_MAJOR ? w : h;
      if (L.boff[b] < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative block offset");
      if (L.bld[b] < fast || L.bld[b] < 1)
        return fail(COSTA_ERROR_INVALID_VALUE, "block leading dimension smaller than the block extent");
      int64_t end = L.boff[b] + (slow - 1) * L.bld[b] + fast;
      int32_t r = L.owner[b];
      if (end > L.local_elems[r]) L.local_elems[r] = end;
    }
  L.id = g_next_id.fetch_add(1);
  return COSTA_SUCCESS;
}

}  // namespace costa

using namespace costa;

extern "C" costa_status costa_layout_create(int64_t nrows, int64_t ncols, int32_t nbr, const int64_t* row_splits,
                                            int32_t nbc, const int64_t* col_splits, const int32_t* owners,
                                            int32_t nranks, costa_order block_order, const int64_t* block_offset,
                                            const int64_t* block_ld, costa_layout* out) {
  if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output handle");
  *out = nullptr;
  if (nranks < 1) return fail(COSTA_ERROR_INVALID_VALUE, "nranks must be >= 1");
  if (block_order != COSTA_COL_MAJOR && block_order != COSTA_ROW_MAJOR)
    return fail(COSTA_ERROR_INVALID_VALUE, "unknown block order");
  costa_status st = check_splits("rows", nrows, nbr, row_splits);
  if (st != COSTA_SUCCESS) return st;
  st = check_splits("cols", ncols, nbc, col_splits);
  if (st != COSTA_SUCCESS) return st;
  int64_t nblocks = (int64_t)nbr * nbc;
  if (nblocks > 0 && !owners) return fail(COSTA_ERROR_INVALID_VALUE, "null owners");
  if ((block_offset == nullptr) != (block_ld == nullptr))
    return fail(COSTA_ERROR_INVALID_VALUE, "block_offset and block_ld must both be given or both be NULL");
  for (int64_t b = 0; b < nblocks; ++b)
    if (owners[b] < 0 || owners[b] >= nranks) return fail(COSTA_ERROR_INVALID_VALUE, "owner out of range");

  costa_layout_s* h = new (std::nothrow) costa_layout_s();
  if (!h) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
  Layout& L = h->L;
  L.nrows = nrows;
  L.ncols = ncols;
  L.nbr = nbr;
  L.nbc = nbc;
  L.nranks = nranks;
  L.order = block_order;
  L.rsplit.assign(row_splits ? row_splits : nullptr, row_splits ? row_splits + nbr + 1 : nullptr);
  if (L.rsplit.empty()) L.rsplit.push_back(0);
  L.csplit.assign(col_splits ? col_splits : nullptr, col_splits ? col_splits + nbc + 1 : nullptr);
  if (L.csplit.empty()) L.csplit.push_back(0);
  L.owner.assign(owners, owners + nblocks);
  L.boff.assign(nblocks, 0);
  L.bld.assign(nblocks, 1);
  if (block_offset) {
    std::memcpy(L.boff.data(), block_offset, sizeof(int64_t) * nblocks);
    std::memcpy(L.bld.data(), block_ld, sizeof(int64_t) * nblocks);
  } else {
    // default packing: blocks of a rank one after another, row-major over (bi, bj)
    std::vector<int64_t> next(nranks, 0);
    for (int32_t bi = 0; bi < nbr; ++bi)
      for (int32_t bj = 0; bj < nbc; ++bj) {
        int64_t b = L.block(bi, bj);
        int64_t hgt = L.rsplit[bi + 1] - L.rsplit[bi], wid = L.csplit[bj + 1] - L.csplit[bj];
        L.boff[b] = next[L.owner[b]];
        L.bld[b] = block_order == COSTA_COL_MAJOR ? hgt : wid;
        next[L.owner[b]] += hgt * wid;
      }
  }
  st = finish_layout(L);
  if (st != COSTA_SUCCESS) {
    delete h;
    return st;
  }
  *out = h;
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_layout_create_block_cyclic(int64_t nrows, int64_t ncols, int64_t mb, int64_t nb,
                                                         int32_t prow, int32_t pcol, costa_order rank_order,
                                                         costa_order block_order, costa_layout* out) {
  if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output handle");
  *out = nullptr;
  if (nrows < 0 || ncols < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative dimension");
  if (mb < 1 || nb < 1) return fail(COSTA_ERROR_INVALID_VALUE, "block sizes must be >= 1");
  if (prow < 1 || pcol < 1) return fail(COSTA_ERROR_INVALID_VALUE, "process grid must be at least 1x1");
  if ((int64_t)prow * pcol > INT32_MAX) return fail(COSTA_ERROR_INVALID_VALUE, "too many processes");
  if (rank_order != COSTA_COL_MAJOR && rank_order != COSTA_ROW_MAJOR)
    return fail(COSTA_ERROR_INVALID_VALUE, "unknown rank order");
  if (block_order != COSTA_COL_MAJOR && block_order != COSTA_ROW_MAJOR)
    return fail(COSTA_ERROR_INVALID_VALUE, "unknown block order");
  int64_t nbr64 = (nrows + mb - 1) / mb, nbc64 = (ncols + nb - 1) / nb;
  if (nbr64 > INT32_MAX || nbc64 > INT32_MAX) return fail(COSTA_ERROR_INVALID_VALUE, "too many blocks");
  int32_t nbr = (int32_t)nbr64, nbc = (int32_t)nbc64;

  costa_layout_s* h = new (std::nothrow) costa_layout_s();
  if (!h) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
  Layout& L = h->L;
  L.nrows = nrows;
  L.ncols = ncols;
  L.nbr = nbr;
  L.nbc = nbc;
  L.nranks = prow * pcol;
  L.order = block_order;
  L.rsplit.resize(nbr + 1);
  for (int32_t k = 0; k <= nbr; ++k) L.rsplit[k] = std::min<int64_t>((int64_t)k * mb, nrows);
  L.csplit.resize(nbc + 1);
  for (int32_t k = 0; k <= nbc; ++k) L.csplit[k] = std::min<int64_t>((int64_t)k * nb, ncols);
  // local extents of each process row / column: the sum of the blocks it is dealt
  L.lrows.assign(prow, 0);
  L.lcols.assign(pcol, 0);
  for (int32_t bi = 0; bi < nbr; ++bi) L.lrows[bi % prow] += L.rsplit[bi + 1] - L.rsplit[bi];
  for (int32_t bj = 0; bj < nbc; ++bj) L.lcols[bj % pcol] += L.csplit[bj + 1] - L.csplit[bj];
  L.mb = mb;
  L.nb = nb;
  L.block_cyclic = true;
  L.prow = prow;
  L.pcol = pcol;
  L.rank_order = rank_order;
  // every rank holds its local matrix of lrows x lcols elements
  L.local_elems.assign(L.nranks, 0);
  for (int32_t pr = 0; pr < prow; ++pr)
    for (int32_t pc = 0; pc < pcol; ++pc)
      L.local_elems[rank_order == COSTA_ROW_MAJOR ? pr * pcol + pc : pr + pc * prow] = L.lrows[pr] * L.lcols[pc];
  L.id = g_next_id.fetch_add(1);
  *out = h;
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_layout_local_elems(costa_layout layout, int32_t rank, int64_t* n) {
  if (!layout || !n) return fail(COSTA_ERROR_INVALID_VALUE, "null argument");
  if (rank < 0 || rank >= layout->L.nranks) return fail(COSTA_ERROR_INVALID_VALUE, "rank out of range");
  *n = layout->L.local_elems[rank];
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_layout_block(costa_layout layout, int32_t bi, int32_t bj, int32_t* owner,
                                           int64_t* offset, int64_t* ld) {
  if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
  const Layout& L = layout->L;
  if (bi < 0 || bi >= L.nbr || bj < 0 || bj >= L.nbc) return fail(COSTA_ERROR_INVALID_VALUE, "block out of range");
  if (owner) *owner = L.owner_of(bi, bj);
  if (offset) *offset = L.offset_of(bi, bj);
  if (ld) *ld = L.ld_of(bi, bj);
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_layout_info(costa_layout layout, int64_t* nrows, int64_t* ncols, int32_t* nbr,
                                          int32_t* nbc, int32_t* nranks, costa_order* block_order) {
  if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
  const Layout& L = layout->L;
  if (nrows) *nrows = L.nrows;
  if (ncols) *ncols = L.ncols;
  if (nbr) *nbr = L.nbr;
  if (nbc) *nbc = L.nbc;
  if (nranks) *nranks = L.nranks;
  if (block_order) *block_order = L.order;
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_layout_destroy(costa_layout layout) {
  if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
  delete layout;
  return COSTA_SUCCESS;
}

extern "C" const char* costa_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* costa_status_string(costa_status s) {
  switch (s) {
    case COSTA_SUCCESS: return "success";
    case COSTA_ERROR_INVALID_VALUE: return "invalid value";
    case COSTA_ERROR_SHAPE_MISMATCH: return "shape mismatch";
    case COSTA_ERROR_OUT_OF_MEMORY: return "out of memory";
    case COSTA_ERROR_DEVICE: return "device error";
    case COSTA_ERROR_NOT_SUPPORTED: return "not supported";
  }
  return "unknown status";
}

namespace costa {
const Layout* layout_of(costa_layout h) { return h ? &h->L : nullptr; }
}  // namespace costa
