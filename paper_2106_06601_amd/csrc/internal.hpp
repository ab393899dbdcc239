// Internal declarations shared by the host code and the kernels of the
// layout-transform library.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <new>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/costa.h"

namespace costa {

// ---- error reporting -------------------------------------------------------
void set_error(const std::string& msg);
costa_status fail(costa_status st, const std::string& msg);

// A valid request past what the kernels index: more than 2^31 rectangles or
// workgroups in one launch, or more than 2^32 rectangles to sort.
struct LimitExceeded : std::runtime_error {
  using std::runtime_error::runtime_error;
};

// Runs the body of a C entry point so that nothing it throws crosses the C
// ABI: a host allocation that fails (std::bad_alloc, or a container asked for
// more than it can hold) is COSTA_ERROR_OUT_OF_MEMORY, a LimitExceeded is
// COSTA_ERROR_NOT_SUPPORTED.
template <typename F>
costa_status guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const LimitExceeded& e) {
    return fail(COSTA_ERROR_NOT_SUPPORTED, e.what());
  } catch (const std::bad_alloc&) {
    return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
  } catch (const std::length_error&) {
    return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed (container size limit)");
  } catch (const std::exception& e) {
    return fail(COSTA_ERROR_NOT_SUPPORTED, std::string("unexpected host error: ") + e.what());
  } catch (...) {
    return fail(COSTA_ERROR_NOT_SUPPORTED, "unexpected host error");
  }
}

// ---- layouts (Section 5 "Matrix Layout", Figure 1) -------------------------
struct Layout {
  uint64_t id = 0;
  int64_t nrows = 0, ncols = 0;
  int32_t nbr = 0, nbc = 0;
  int32_t nranks = 0;
  costa_order order = COSTA_COL_MAJOR;
  std::vector<int64_t> rsplit, csplit;  // nbr+1, nbc+1
  std::vector<int64_t> local_elems;     // per rank
  // general grids: per block, row-major over (bi, bj)
  std::vector<int32_t> owner;
  std::vector<int64_t> boff, bld;
  // block-cyclic layouts keep no per-block arrays (a 10^5 x 10^5 matrix in
  // 1 x 1 blocks has 10^10 of them).  They follow a ScaLAPACK descriptor: the
  // full matrix is dealt in mb x nb blocks over a prow x pcol grid starting
  // at process (rsrc, csrc), and each rank keeps its local matrix with
  // leading dimension lld (0: its own local extent, at least 1).  A layout
  // may be a window of that matrix: its element (i, j) is element
  // (r0 + i, c0 + j) of the full one, and its block bi is the full
  // matrix's block row r0/mb + bi, truncated to the window (Section 5,
  // a submatrix by truncating the splits).
  bool block_cyclic = false;
  int32_t prow = 0, pcol = 0;
  int32_t rsrc = 0, csrc = 0;
  costa_order rank_order = COSTA_ROW_MAJOR;
  int64_t mb = 0, nb = 0;
  int64_t lld = 0;
  int64_t r0 = 0, c0 = 0;            // window origin in the full matrix
  int64_t rb0 = 0, cb0 = 0;          // r0 / mb, c0 / nb
  std::vector<int64_t> lrows, lcols;  // local extents of the full matrix per process row / column
  std::vector<int32_t> rank_map;      // empty, or the rank of grid position (pr, pc) at pr + pc*prow

  int64_t block(int32_t bi, int32_t bj) const { return (int64_t)bi * nbc + bj; }
  int32_t prow_of(int32_t bi) const { return (int32_t)((rb0 + bi + rsrc) % prow); }
  int32_t pcol_of(int32_t bj) const { return (int32_t)((cb0 + bj + csrc) % pcol); }
  int32_t rank_at(int32_t pr, int32_t pc) const {
    if (!rank_map.empty()) return rank_map[(size_t)pr + (size_t)pc * prow];
    return rank_order == COSTA_ROW_MAJOR ? pr * pcol + pc : pr + pc * prow;
  }
  int32_t owner_of(int32_t bi, int32_t bj) const {
    if (!block_cyclic) return owner[block(bi, bj)];
    return rank_at(prow_of(bi), pcol_of(bj));
  }
  int64_t ld_of(int32_t bi, int32_t bj) const {
    if (!block_cyclic) return bld[block(bi, bj)];
    if (lld) return lld;
    const int64_t ext = order == COSTA_COL_MAJOR ? lrows[prow_of(bi)] : lcols[pcol_of(bj)];
    return ext > 1 ? ext : 1;
  }
  int64_t offset_of(int32_t bi, int32_t bj) const {
    if (!block_cyclic) return boff[block(bi, bj)];
    // local position of the block's first element (ScaLAPACK INDXG2L)
    const int64_t gi = r0 + rsplit[bi], gj = c0 + csplit[bj];
    const int64_t li = ((rb0 + bi) / prow) * mb + gi % mb;
    const int64_t lj = ((cb0 + bj) / pcol) * nb + gj % nb;
    const int64_t ld = ld_of(bi, bj);
    return order == COSTA_COL_MAJOR ? li + lj * ld : li * ld + lj;
  }
};

// ---- grid overlay (Section 5 "Grid Overlay") -------------------------------
// One interval of the union of two split lists, with the index of the
// interval of each list that covers it.
struct Interval {
  int64_t start;
  int64_t len;
  int32_t a;  // covering block index in A's splits
  int32_t b;  // covering block index in op(B)'s splits
};
std::vector<Interval> overlay(const std::vector<int64_t>& sa, const std::vector<int64_t>& sb);

// ---- work rectangles -------------------------------------------------------
// A rectangle of elements moved with one addressing rule.  Coordinates are in
// the destination's orientation: x runs along the destination's contiguous
// direction.  dst(x, y) = dst_off + y*dst_ld + x.  The source is
//   src_off + y*src_ld + x   (flag TRANSPOSE clear: contiguous along x), or
//   src_off + x*src_ld + y   (flag TRANSPOSE set: contiguous along y).
// PIECE_WIDE: a non-transposed rectangle whose offsets, strides and width
//   allow 16-byte vectors.
// PIECE_GROUP_NEXT: the next rectangle of the launch is moved by the same
//   workgroup (a run of small rectangles shares one workgroup).
// PIECE_STACK: one of a stack of row walks -- consecutive rectangles of a
//   launch, of one pair, vector width and height ny, that follow one another
//   along x on one side (the source, or the destination with
//   PIECE_STACK_DST): the same buffer and stride there, each starting where
//   the previous one ends.  The stack is moved as one band of the summed
//   width (stack_tasks below); its first rectangle holds the number of
//   rectangles in flags bits 16-31, and every rectangle of the stack has the
//   stack's first task in task0 and aux.
// A transposed rectangle is moved in LDS tiles of tile_x x tile_y elements
// (tile_x along the destination's contiguous direction; choose_tile below),
// packed into `aux` with tile_pack.
enum : int32_t {
  PIECE_TRANSPOSE = 1,
  PIECE_WIDE = 2,
  PIECE_GROUP_NEXT = 16,
  PIECE_STACK = 32,
  PIECE_STACK_DST = 64
};
constexpr int32_t stack_size_of(int32_t flags) { return (int32_t)((uint32_t)flags >> 16); }

struct alignas(16) Piece {
  int64_t src_off;
  int64_t dst_off;
  int64_t src_ld;
  int64_t dst_ld;
  int32_t src_buf;  // index into the call's buffer table
  int32_t dst_buf;
  int32_t nx;
  int32_t ny;
  int32_t item;     // pair of a batched call (selects alpha, beta, mode)
  int32_t flags;
  int32_t task0;    // first workgroup of its launch that moves it
  int32_t aux;      // transposed rectangles: tile_pack(tile_x, tile_y); row walks in a
                    // launch without tiles: its first task in the launch's wide task table
};
static_assert(sizeof(Piece) == 64, "Piece must be 64 bytes");

// Work of one workgroup (kThreadsPerTask lanes): one LDS tile of a
// transposed rectangle, kThreadsPerTask units (16-byte vectors, or single
// elements when the rectangle is not PIECE_WIDE) of a rectangle walked along
// its rows, or a run of small rectangles moved at once.  A launch of row
// walks also has a wide task table whose tasks are kWideTaskUnits units (a
// run still one task); launches that copy use it, two units per lane.
constexpr int32_t kThreadsPerTask = 256;
#ifndef COSTA_COPY_UNITS
#define COSTA_COPY_UNITS 2  // units per lane in launches of row walks that copy
#endif
constexpr int32_t kWideTaskUnits = (COSTA_COPY_UNITS > 1 ? COSTA_COPY_UNITS : 2) * kThreadsPerTask;
constexpr int32_t kGroupUnitsMax = 128;  // rectangles of at most this many units may share a workgroup
constexpr int32_t kGroupPiecesMax = 8;

// Stacks (PIECE_STACK): rectangles whose rows are COSTA_STACK_MIN_RUN to
// COSTA_STACK_MAX_RUN bytes long stack, up to kStackPiecesMax of them.  A
// stack of height ny and summed width hu units (16-byte vectors when
// PIECE_WIDE, else elements) is cut into wave tasks of 64 units of x by
// kStackRows rows of y: wave task t covers units [64 * (t % wb), +64) and
// rows [kStackRows * (t / wb), +kStackRows), wb = ceil(hu / 64), and
// workgroup task c runs wave tasks 4c .. 4c + 3 (stack_tasks of them).
// COSTA_STACK_MAX_RUN 0 turns stacks off.
#ifndef COSTA_STACK_MIN_RUN
#define COSTA_STACK_MIN_RUN 128
#endif
#ifndef COSTA_STACK_MAX_RUN
#define COSTA_STACK_MAX_RUN 512
#endif
#ifndef COSTA_STACK_ROWS
#define COSTA_STACK_ROWS 4
#endif
#ifndef COSTA_STACK_MIN_UNITS
#define COSTA_STACK_MIN_UNITS 256  // narrower stacks, and stacks whose last wave would be mostly idle, do not form
#endif
constexpr int32_t kStackPiecesMax = 4096;
constexpr int32_t kStackRows = COSTA_STACK_ROWS;
constexpr int32_t kStackWave = 64;
constexpr int64_t kStackWaveTasksMax = (1 << 23) - 1;  // the kernel divides wave tasks in fp32
inline int64_t stack_wave_tasks(int64_t hu, int64_t ny) {
  return ((hu + kStackWave - 1) / kStackWave) * ((ny + kStackRows - 1) / kStackRows);
}
inline int64_t stack_tasks(int64_t hu, int64_t ny) {
  const int64_t per = kThreadsPerTask / kStackWave;
  return (stack_wave_tasks(hu, ny) + per - 1) / per;
}

// Elements per 16-byte unit of a PIECE_WIDE rectangle.
constexpr int32_t wide_elems(int32_t es) { return es >= 16 ? 1 : 16 / es; }

// LDS tiles of transposed rectangles.  A tile is at most tile_max_x(es)
// wide; its rows (one per x) take tile_y | 1 elements in LDS -- an odd
// stride, so that lanes reading one LDS row element each (consecutive x) hit
// distinct banks -- and all of them fit the tile's LDS array of
// tile_lds_elems(es) elements.  Small rectangles are one tile; larger ones
// are cut into tiles of equal width (at most tile_max_x) and equal height.
// When the rectangle's source columns start on 128-byte lines the height is
// what tile_budget(es) elements allow (for the usual shapes a whole number of
// lines per column, so no tile shares a line with the one below it, and the
// lanes storing a column to LDS do not straddle two columns).  Otherwise the
// height is odd and as large as the LDS array allows: the rows then need no
// padding, so the lanes storing a tile's columns one after another write
// consecutive LDS addresses (padded rows would make each group of lanes that
// crosses a column end hit one bank twice).
#ifndef COSTA_TILE_BUDGET16
#define COSTA_TILE_BUDGET16 3072  // three workgroups per CU (4096: two, -1 to -9%; 2048: four, shorter tiles)
#endif
#ifndef COSTA_TILE_MAXX16
#define COSTA_TILE_MAXX16 256
#endif
#ifndef COSTA_ODD_TILES
#define COSTA_ODD_TILES 0  // 1: cut tiles of misaligned columns with an odd height that fills the LDS array
#endif
constexpr int32_t tile_budget(int32_t es) { return es >= 16 ? COSTA_TILE_BUDGET16 : es == 8 ? 2048 : 4096; }
constexpr int32_t tile_max_x(int32_t es) { return es >= 16 ? COSTA_TILE_MAXX16 : 128; }
constexpr int32_t tile_lds_elems(int32_t es) { return tile_budget(es) + tile_max_x(es); }
// Elements of the largest tile (what a workgroup's lanes must cover).
constexpr int32_t tile_max_elems(int32_t es) { return COSTA_ODD_TILES ? tile_lds_elems(es) : tile_budget(es); }
constexpr int32_t tile_pack(int32_t tx, int32_t ty) { return tx | ty << 16; }
constexpr int32_t tile_x_of(int32_t t) { return t & 0xffff; }
constexpr int32_t tile_y_of(int32_t t) { return t >> 16; }
// aligned_cols: the source columns (runs along y) start on 128-byte lines.
inline void choose_tile(int32_t es, int32_t nx, int32_t ny, bool aligned_cols, int32_t& tx, int32_t& ty) {
  const int32_t maxx = tile_max_x(es);
  const bool odd = COSTA_ODD_TILES && !aligned_cols;
  const int32_t cap = tile_lds_elems(es), budget = tile_budget(es);
  if (nx <= maxx && (odd ? (int64_t)nx * (ny | 1) <= cap : (int64_t)nx * ny <= budget)) {
    tx = nx;
    ty = ny;
    return;
  }
  const int32_t ntx = (nx + maxx - 1) / maxx;
  tx = (nx + ntx - 1) / ntx;
  if (!odd) {
    ty = budget / tx;
    if (ty > ny) ty = ny;
    const int32_t nty = (ny + ty - 1) / ty;
    ty = (ny + nty - 1) / nty;
    return;
  }
  int32_t tymax = cap / tx;  // >= 1: tx <= maxx < cap
  if (tymax > 1 && tymax % 2 == 0) --tymax;  // odd: rows without padding
  if (ny <= tymax) {
    ty = ny;  // one tile row: (ny | 1) <= tymax since tymax is odd (or 1)
    return;
  }
  const int32_t nty = (ny + tymax - 1) / tymax;
  ty = (ny + nty - 1) / nty;
  if (ty % 2 == 0 && ty < tymax) ++ty;  // keeps at most nty tiles, the last one shorter
}

// Per-pair parameters of a call, read by the kernels.
enum : int32_t { MODE_COPY = 0, MODE_SCALE = 1, MODE_AXPBY = 2 };
struct alignas(16) ItemParam {
  double alpha[2];
  double beta[2];
  int32_t mode;
  int32_t conj;
  int32_t pad[2];
};
static_assert(sizeof(ItemParam) == 48, "ItemParam must be 48 bytes");

// One kernel launch of a plan: a range of rectangles and the workgroups
// (tasks) that move them.  tasks[task_begin + b] = index into Plan::pieces of
// the rectangle task b starts with; that rectangle's task0 is the first task
// that moves it, so task b takes its (b - task0)-th tile or chunk.  The wide
// table works the same way with the rectangle's aux in place of task0.
struct LaunchRange {
  int64_t piece_begin = 0, npieces = 0;
  int64_t task_begin = 0, ntasks = 0;
  int64_t wide_begin = 0, nwide = 0;  // wide task table (launches without tiles; 0 tasks otherwise)
  int64_t elems = 0;
  bool has_transpose = false;
  int32_t xcd_ranges = 0;  // 1: each XCD takes one contiguous range of the launch's tasks
  std::vector<int64_t> item_elems;  // elements of each pair in this launch
};

// A pack and its unpack-transform; the unpack is two launches when it holds
// both row walks and LDS tiles (each launch of one kind, see plan.cpp).
struct Wave {
  LaunchRange pack;
  std::vector<LaunchRange> unpack;
  int64_t msg_bytes = 0;
};

// ---- kernels (kernels.hip) -------------------------------------------------
enum MoverKind : int32_t { KIND_PACK = 0, KIND_UNPACK = 1, KIND_DIRECT = 2 };
// What one launch needs: the pairs' common arithmetic mode and conjugation
// (mode -1: the pairs differ, read per rectangle) and whether any rectangle
// of the launch is transposed.
struct LaunchSpec {
  int32_t mode;
  int32_t conj;
  bool has_transpose;
};
// pieces: the plan's rectangles (global indices); tasks: the launch's
// ntasks entries, wide: its wide task table (nwide entries, 0 in launches
// with tiles).
// xcd_ranges: 0 runs task b in workgroup b (workgroups are dispatched
// round-robin over the 8 XCDs); 1 hands each XCD one contiguous range of the
// tasks of each launch slice.
hipError_t launch_mover(MoverKind kind, costa_dtype dtype, const LaunchSpec& spec, const Piece* pieces,
                        const int32_t* tasks, int64_t ntasks, const int32_t* wide, int64_t nwide, void* const* bufs,
                        const ItemParam* items, int32_t allow_wide, int32_t xcd_ranges, hipStream_t stream);

struct VolumeArgs {
  const Interval* rows;
  int32_t K;
  const Interval* cols;
  int32_t L;
  const int32_t* ownerA;
  int32_t nbcA;
  const int32_t* ownerB;
  int32_t nbcB;
  int32_t transposed;
  int32_t P;
  unsigned long long* V;
};
hipError_t launch_volume(const VolumeArgs& a, hipStream_t stream);

// Separable volume of two block-cyclic layouts: per-dimension histograms of
// the overlay intervals over (class in B, class in A) -- Interval::a and ::b
// hold those classes here -- then V[s][t] as the product of a row and a
// column histogram entry.
struct SeparableArgs {
  const Interval* rows;
  int32_t K;
  const Interval* cols;
  int32_t L;
  int32_t nrb, nra;  // row classes of B (for rows of op(B)) and of A
  int32_t ncb, nca;  // column classes
  unsigned long long* hrow;  // nrb * nra, zeroed by the caller
  unsigned long long* hcol;  // ncb * nca, zeroed by the caller
  // per rank r: its row class at [2r] and column class at [2r + 1] in A's
  // grid (clsA) and in op(B)'s grid (clsB), or -1 for a rank outside the grid
  const int32_t* clsA;
  const int32_t* clsB;
  int32_t P;
  unsigned long long* V;
};
hipError_t launch_volume_separable(const SeparableArgs& a, hipStream_t stream);

// ---- ScaLAPACK-compatible routines (scalapack.cpp) ----------------------------
// Destroys the cached descriptor layouts (called by costa_finalize).
void release_scalapack_layouts();

// ---- relabeling (lap.cpp) --------------------------------------------------
// Lexicographically smallest sigma maximising sum_t V[sigma[t]][t].
void solve_relabel(int32_t P, const int64_t* V, int32_t* sigma);

}  // namespace costa
