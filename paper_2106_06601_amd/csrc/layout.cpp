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
  return guarded([&]() -> costa_status {
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
  });
}

namespace costa {

// Splits of the window [r0, r0 + m) of a dimension dealt in blocks of mb: the
// full matrix's block boundaries inside the window, shifted to start at 0.
static bool window_splits(int64_t r0, int64_t m, int64_t mb, std::vector<int64_t>& s) {
  s.assign(1, 0);
  if (m == 0) return true;
  const int64_t first = r0 / mb, last = (r0 + m - 1) / mb;
  if (last - first + 1 > INT32_MAX) return false;
  for (int64_t k = first + 1; k <= last; ++k) s.push_back(k * mb - r0);
  s.push_back(m);
  return true;
}

// Sets the window of a block-cyclic layout (origin r0, c0 in the full
// matrix; m x n) and the buffer size each rank needs for it: one past the
// rank's last window element.
static costa_status set_window(Layout& L, int64_t r0, int64_t c0, int64_t m, int64_t n) {
  if (!window_splits(r0, m, L.mb, L.rsplit) || !window_splits(c0, n, L.nb, L.csplit))
    return fail(COSTA_ERROR_INVALID_VALUE, "too many blocks");
  L.nrows = m;
  L.ncols = n;
  L.nbr = (int32_t)(L.rsplit.size() - 1);
  L.nbc = (int32_t)(L.csplit.size() - 1);
  L.r0 = r0;
  L.c0 = c0;
  L.rb0 = r0 / L.mb;
  L.cb0 = c0 / L.nb;
  // one past the largest local row (column) index of the window on each
  // process row (column): the window's last block on it ends there
  std::vector<int64_t> rows_used(L.prow, 0), cols_used(L.pcol, 0);
  for (int32_t bi = 0; bi < L.nbr; ++bi) {
    const int64_t g = r0 + L.rsplit[bi + 1] - 1;
    rows_used[L.prow_of(bi)] = ((L.rb0 + bi) / L.prow) * L.mb + g % L.mb + 1;
  }
  for (int32_t bj = 0; bj < L.nbc; ++bj) {
    const int64_t g = c0 + L.csplit[bj + 1] - 1;
    cols_used[L.pcol_of(bj)] = ((L.cb0 + bj) / L.pcol) * L.nb + g % L.nb + 1;
  }
  L.local_elems.assign(L.nranks, 0);
  for (int32_t pr = 0; pr < L.prow; ++pr)
    for (int32_t pc = 0; pc < L.pcol; ++pc) {
      if (rows_used[pr] == 0 || cols_used[pc] == 0) continue;
      int64_t need;
      if (L.order == COSTA_COL_MAJOR) {
        const int64_t ld = L.lld ? L.lld : std::max<int64_t>(1, L.lrows[pr]);
        need = (cols_used[pc] - 1) * ld + rows_used[pr];
      } else {
        const int64_t ld = L.lld ? L.lld : std::max<int64_t>(1, L.lcols[pc]);
        need = (rows_used[pr] - 1) * ld + cols_used[pc];
      }
      L.local_elems[L.rank_at(pr, pc)] = need;
    }
  L.id = g_next_id.fetch_add(1);
  return COSTA_SUCCESS;
}

// Block-cyclic layout of a whole matrix dealt from process (rsrc, csrc).
static costa_status make_block_cyclic(int64_t nrows, int64_t ncols, int64_t mb, int64_t nb, int32_t prow,
                                      int32_t pcol, int32_t rsrc, int32_t csrc, int64_t lld, costa_order rank_order,
                                      costa_order block_order, int32_t nranks, const int32_t* rank_map,
                                      costa_layout* out) {
  if (nrows < 0 || ncols < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative dimension");
  if (mb < 1 || nb < 1) return fail(COSTA_ERROR_INVALID_VALUE, "block sizes must be >= 1");
  if (prow < 1 || pcol < 1) return fail(COSTA_ERROR_INVALID_VALUE, "process grid must be at least 1x1");
  if ((int64_t)prow * pcol > INT32_MAX) return fail(COSTA_ERROR_INVALID_VALUE, "too many processes");
  if (rank_order != COSTA_COL_MAJOR && rank_order != COSTA_ROW_MAJOR)
    return fail(COSTA_ERROR_INVALID_VALUE, "unknown rank order");
  if (block_order != COSTA_COL_MAJOR && block_order != COSTA_ROW_MAJOR)
    return fail(COSTA_ERROR_INVALID_VALUE, "unknown block order");
  if ((nrows + mb - 1) / mb > INT32_MAX || (ncols + nb - 1) / nb > INT32_MAX)
    return fail(COSTA_ERROR_INVALID_VALUE, "too many blocks");
  const int32_t grid_size = prow * pcol;
  if (nranks == 0) nranks = grid_size;
  if (nranks < grid_size) return fail(COSTA_ERROR_INVALID_VALUE, "fewer ranks than grid positions");
  if (!rank_map && nranks != grid_size)
    return fail(COSTA_ERROR_INVALID_VALUE, "a grid smaller than its set of ranks needs a rank map");
  if (rank_map) {
    std::vector<char> seen(nranks, 0);
    for (int32_t k = 0; k < grid_size; ++k) {
      if (rank_map[k] < 0 || rank_map[k] >= nranks || seen[rank_map[k]])
        return fail(COSTA_ERROR_INVALID_VALUE, "rank map entries must be distinct ranks in [0, nranks)");
      seen[rank_map[k]] = 1;
    }
  }
  costa_layout_s* h = new (std::nothrow) costa_layout_s();
  if (!h) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
  Layout& L = h->L;
  L.nranks = nranks;
  if (rank_map) L.rank_map.assign(rank_map, rank_map + grid_size);
  L.order = block_order;
  L.block_cyclic = true;
  L.prow = prow;
  L.pcol = pcol;
  L.rsrc = rsrc;
  L.csrc = csrc;
  L.rank_order = rank_order;
  L.mb = mb;
  L.nb = nb;
  // local extents of each process row / column: the blocks dealt to it, the
  // first block to process row rsrc (column csrc)
  L.lrows.assign(prow, 0);
  L.lcols.assign(pcol, 0);
  for (int64_t k = 0; k * mb < nrows; ++k) L.lrows[(k + rsrc) % prow] += std::min(mb, nrows - k * mb);
  for (int64_t k = 0; k * nb < ncols; ++k) L.lcols[(k + csrc) % pcol] += std::min(nb, ncols - k * nb);
  const int64_t need_ld = std::max<int64_t>(
      1, block_order == COSTA_COL_MAJOR ? *std::max_element(L.lrows.begin(), L.lrows.end())
                                        : *std::max_element(L.lcols.begin(), L.lcols.end()));
  if (lld != 0 && lld < need_ld) {
    delete h;
    return fail(COSTA_ERROR_INVALID_VALUE, "local leading dimension smaller than the local extent");
  }
  L.lld = lld;
  costa_status st = set_window(L, 0, 0, nrows, ncols);
  if (st != COSTA_SUCCESS) {
    delete h;
    return st;
  }
  *out = h;
  return COSTA_SUCCESS;
}

}  // namespace costa

extern "C" costa_status costa_layout_create_block_cyclic(int64_t nrows, int64_t ncols, int64_t mb, int64_t nb,
                                                         int32_t prow, int32_t pcol, costa_order rank_order,
                                                         costa_order block_order, costa_layout* out) {
  return guarded([&]() -> costa_status {
    if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output handle");
    *out = nullptr;
    return make_block_cyclic(nrows, ncols, mb, nb, prow, pcol, 0, 0, 0, rank_order, block_order, 0, nullptr, out);
  });
}

extern "C" costa_status costa_layout_create_scalapack(const int32_t* desc, const costa_grid* grid,
                                                      costa_layout* out) {
  return guarded([&]() -> costa_status {
    if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output handle");
    *out = nullptr;
    if (!desc || !grid) return fail(COSTA_ERROR_INVALID_VALUE, "null descriptor or grid");
    if (desc[0] != 1) return fail(COSTA_ERROR_NOT_SUPPORTED, "descriptor type (DTYPE_) other than 1 (dense)");
    if (grid->nprow < 1 || grid->npcol < 1) return fail(COSTA_ERROR_INVALID_VALUE, "process grid must be at least 1x1");
    if (desc[6] < 0 || desc[6] >= grid->nprow) return fail(COSTA_ERROR_INVALID_VALUE, "RSRC_ outside the process grid");
    if (desc[7] < 0 || desc[7] >= grid->npcol) return fail(COSTA_ERROR_INVALID_VALUE, "CSRC_ outside the process grid");
    if (desc[8] < 1) return fail(COSTA_ERROR_INVALID_VALUE, "LLD_ must be >= 1");
    if (grid->nranks < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative number of ranks");
    return make_block_cyclic(desc[2], desc[3], desc[4], desc[5], grid->nprow, grid->npcol, desc[6], desc[7], desc[8],
                             grid->rank_map ? COSTA_ROW_MAJOR : grid->rank_order, COSTA_COL_MAJOR, grid->nranks,
                             grid->rank_map, out);
  });
}

extern "C" costa_status costa_layout_submatrix(costa_layout parent, int64_t i0, int64_t j0, int64_t m, int64_t n,
                                               costa_layout* out) {
  return guarded([&]() -> costa_status {
    if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output handle");
    *out = nullptr;
    if (!parent) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
    const Layout& P = parent->L;
    if (i0 < 0 || j0 < 0 || m < 0 || n < 0 || i0 > P.nrows - m || j0 > P.ncols - n)
      return fail(COSTA_ERROR_INVALID_VALUE, "submatrix outside the matrix");
    costa_layout_s* h = new (std::nothrow) costa_layout_s();
    if (!h) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
    Layout& L = h->L;
    costa_status st;
    if (P.block_cyclic) {
      L = P;
      st = set_window(L, P.r0 + i0, P.c0 + j0, m, n);
    } else {
      // keep the blocks the window meets, cut to it; each keeps its storage,
      // the offset moving to the window's first element inside it
      auto range = [](const std::vector<int64_t>& s, int64_t lo, int64_t len, int32_t& first) -> int32_t {
        if (len == 0) {
          first = 0;
          return 0;
        }
        first = (int32_t)(std::upper_bound(s.begin(), s.end(), lo) - s.begin() - 1);
        const int32_t last = (int32_t)(std::upper_bound(s.begin(), s.end(), lo + len - 1) - s.begin() - 1);
        return last - first + 1;
      };
      int32_t fr, fc;
      const int32_t nbr = range(P.rsplit, i0, m, fr), nbc = range(P.csplit, j0, n, fc);
      L.nrows = m;
      L.ncols = n;
      L.nbr = nbr;
      L.nbc = nbc;
      L.nranks = P.nranks;
      L.order = P.order;
      L.rsplit.assign(nbr + 1, 0);
      for (int32_t k = 1; k < nbr; ++k) L.rsplit[k] = P.rsplit[fr + k] - i0;
      L.rsplit[nbr] = m;
      L.csplit.assign(nbc + 1, 0);
      for (int32_t k = 1; k < nbc; ++k) L.csplit[k] = P.csplit[fc + k] - j0;
      L.csplit[nbc] = n;
      const size_t nblocks = (size_t)nbr * nbc;
      L.owner.resize(nblocks);
      L.boff.resize(nblocks);
      L.bld.resize(nblocks);
      for (int32_t bi = 0; bi < nbr; ++bi)
        for (int32_t bj = 0; bj < nbc; ++bj) {
          const int64_t pb = P.block(fr + bi, fc + bj), b = L.block(bi, bj);
          const int64_t pi = i0 + L.rsplit[bi] - P.rsplit[fr + bi], pj = j0 + L.csplit[bj] - P.csplit[fc + bj];
          L.owner[b] = P.owner[pb];
          L.bld[b] = P.bld[pb];
          L.boff[b] = P.boff[pb] + (P.order == COSTA_COL_MAJOR ? pi + pj * P.bld[pb] : pi * P.bld[pb] + pj);
        }
      st = finish_layout(L);
    }
    if (st != COSTA_SUCCESS) {
      delete h;
      return st;
    }
    *out = h;
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_layout_local_elems(costa_layout layout, int32_t rank, int64_t* n) {
  return guarded([&]() -> costa_status {
    if (!layout || !n) return fail(COSTA_ERROR_INVALID_VALUE, "null argument");
    if (rank < 0 || rank >= layout->L.nranks) return fail(COSTA_ERROR_INVALID_VALUE, "rank out of range");
    *n = layout->L.local_elems[rank];
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_layout_block(costa_layout layout, int32_t bi, int32_t bj, int32_t* owner,
                                           int64_t* offset, int64_t* ld) {
  return guarded([&]() -> costa_status {
    if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
    const Layout& L = layout->L;
    if (bi < 0 || bi >= L.nbr || bj < 0 || bj >= L.nbc) return fail(COSTA_ERROR_INVALID_VALUE, "block out of range");
    if (owner) *owner = L.owner_of(bi, bj);
    if (offset) *offset = L.offset_of(bi, bj);
    if (ld) *ld = L.ld_of(bi, bj);
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_layout_info(costa_layout layout, int64_t* nrows, int64_t* ncols, int32_t* nbr,
                                          int32_t* nbc, int32_t* nranks, costa_order* block_order) {
  return guarded([&]() -> costa_status {
    if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
    const Layout& L = layout->L;
    if (nrows) *nrows = L.nrows;
    if (ncols) *ncols = L.ncols;
    if (nbr) *nbr = L.nbr;
    if (nbc) *nbc = L.nbc;
    if (nranks) *nranks = L.nranks;
    if (block_order) *block_order = L.order;
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_layout_destroy(costa_layout layout) {
  return guarded([&]() -> costa_status {
    if (!layout) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
    delete layout;
    return COSTA_SUCCESS;
  });
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
