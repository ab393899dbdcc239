// Planning of a transform (Section 5, Algorithm 2 and "Grid Overlay";
// Section 6 "Implementation" and "Batched Transformation").
//
// Every block of the grid overlay of L(A) and L(op(B)) lies inside exactly one
// block of each grid, so it has one sender s (owner in L(B)) and one receiver
// label t (owner in L(A)), i.e. it belongs to package S_st.  Under the
// relabeling sigma the label t lives on physical rank sigma[t]; the block is
// local when s == sigma[t] and goes straight from B to A, otherwise it is
// packed into the message of (s -> sigma[t]) and unpacked from there.
//
// Adjacent overlay blocks that are also adjacent in both the source and the
// destination storage (for instance the blocks of one process row of a 1 x P
// grid) are merged into one rectangle.  Each launch's rectangles are then cut
// into workgroup tasks of equal size (an LDS tile of a transposed rectangle,
// or a few KiB of a row walk); runs of small rectangles share one workgroup,
// and stacks of short rectangles that follow one another on one side move as
// one band.  The planning itself runs on host threads (plan_threads) and
// gives the same plan whatever their number.
#include <algorithm>
#include <chrono>
#include <cstdlib>
#include <exception>
#include <new>
#include <numeric>
#include <system_error>
#include <thread>
#include <tuple>

#include "plan.hpp"

// Put the direct rectangles into the last unpack launch instead of a launch
// of their own.
#ifndef COSTA_MERGE_DIRECT
#define COSTA_MERGE_DIRECT 1
#endif

namespace costa {

std::vector<Interval> overlay(const std::vector<int64_t>& sa, const std::vector<int64_t>& sb) {
  // Both lists start at 0 and end at the same n.  The union of their points
  // cuts [0, n) into intervals; each lies inside one interval of each list.
  std::vector<Interval> out;
  size_t na = sa.size() - 1, nb = sb.size() - 1;
  if (na == 0 || nb == 0) return out;
  out.reserve(na + nb);
  size_t ia = 0, ib = 0;
  int64_t pos = 0;
  while (ia < na && ib < nb) {
    int64_t end = std::min(sa[ia + 1], sb[ib + 1]);
    out.push_back(Interval{pos, end - pos, (int32_t)ia, (int32_t)ib});
    pos = end;
    if (sa[ia + 1] == end) ++ia;
    if (sb[ib + 1] == end) ++ib;
  }
  return out;
}

namespace {

// Host threads of the planner: COSTA_PLAN_THREADS if set (1 plans on the
// calling thread alone), else the hardware's threads, at most 16.  The plan
// is the same whatever the count: work is split into ranges whose results
// are joined in order, and sorts order unique keys.
int plan_threads() {
  if (const char* e = std::getenv("COSTA_PLAN_THREADS")) {
    const int v = std::atoi(e);
    if (v >= 1) return std::min(v, 64);
  }
  const unsigned h = std::thread::hardware_concurrency();
  return (int)std::max(1u, std::min(h, 16u));
}

// fn(t) for t in [0, n) on up to `threads` threads (the calling one
// included); an exception in any is rethrown here after all have joined.
template <typename Fn>
void parallel_for(int64_t n, int threads, Fn&& fn) {
  const int64_t nt = std::min<int64_t>(n, threads);
  if (nt <= 1) {
    for (int64_t t = 0; t < n; ++t) fn(t);
    return;
  }
  std::vector<std::exception_ptr> err((size_t)nt);
  auto worker = [&](int64_t w) {
    try {
      for (int64_t t = w; t < n; t += nt) fn(t);
    } catch (...) {
      err[(size_t)w] = std::current_exception();
    }
  };
  std::vector<std::thread> pool;
  pool.reserve((size_t)nt - 1);
  int64_t started = 1;
  try {
    for (; started < nt; ++started) pool.emplace_back(worker, started);
  } catch (const std::system_error&) {
    // no more threads: the calling thread takes the shares not started
  }
  for (int64_t w = started; w < nt; ++w) worker(w);
  worker(0);
  for (std::thread& th : pool) th.join();
  for (const std::exception_ptr& e : err)
    if (e) std::rethrow_exception(e);
}

struct Cand {
  Piece p;
  int32_t kx0, kx1;  // x-interval range [kx0, kx1)
  int32_t ly_start;  // y-interval index of its first strip
  int32_t ly_end;    // y-interval index following the last strip merged
  int32_t s, r;      // sender rank, receiving physical rank
};

inline bool same_kind(const Piece& a, const Piece& b) {
  return a.src_buf == b.src_buf && a.dst_buf == b.dst_buf && a.flags == b.flags && a.src_ld == b.src_ld &&
         a.dst_ld == b.dst_ld;
}

// Owner, leading dimension and local offset of a layout's blocks, with the
// per-block-row and per-block-column parts of a block-cyclic layout (process
// row or column and local start; ScaLAPACK INDXG2P / INDXG2L) taken once per
// row and column instead of once per block.
struct BlockMap {
  const Layout& L;
  std::vector<int32_t> prow, pcol;
  std::vector<int64_t> li, lj;
  explicit BlockMap(const Layout& l) : L(l) {
    if (!L.block_cyclic) return;
    prow.resize(L.nbr);
    li.resize(L.nbr);
    for (int32_t bi = 0; bi < L.nbr; ++bi) {
      prow[bi] = L.prow_of(bi);
      li[bi] = ((L.rb0 + bi) / L.prow) * L.mb + (L.r0 + L.rsplit[bi]) % L.mb;
    }
    pcol.resize(L.nbc);
    lj.resize(L.nbc);
    for (int32_t bj = 0; bj < L.nbc; ++bj) {
      pcol[bj] = L.pcol_of(bj);
      lj[bj] = ((L.cb0 + bj) / L.pcol) * L.nb + (L.c0 + L.csplit[bj]) % L.nb;
    }
  }
  int32_t owner(int32_t bi, int32_t bj) const {
    return L.block_cyclic ? L.rank_at(prow[bi], pcol[bj]) : L.owner[L.block(bi, bj)];
  }
  int64_t ld(int32_t bi, int32_t bj) const {
    if (!L.block_cyclic) return L.bld[L.block(bi, bj)];
    if (L.lld) return L.lld;
    const int64_t ext = L.order == COSTA_COL_MAJOR ? L.lrows[prow[bi]] : L.lcols[pcol[bj]];
    return ext > 1 ? ext : 1;
  }
  int64_t offset(int32_t bi, int32_t bj, int64_t ld_) const {
    if (!L.block_cyclic) return L.boff[L.block(bi, bj)];
    return L.order == COSTA_COL_MAJOR ? li[bi] + lj[bj] * ld_ : li[bi] * ld_ + lj[bj];
  }
};

// All overlay rectangles of one pair, merged; appended to `local` / `remote`.
// The strips along y are cut into ranges planned on up to `threads` threads
// (each range starts with no open rectangles); the ranges are then stitched
// in order, merging a range's rectangles that start on its first strip into
// the open rectangles of the ranges before it -- the merges a single pass
// over the strips makes, so the rectangles are the same.
void plan_pair(int32_t item, int32_t nitems, const ItemDesc& d, const std::vector<int32_t>& sigma,
               std::vector<Cand>& local, std::vector<Cand>& remote, int64_t& overlay_blocks, int64_t& n_local,
               int64_t& n_remote, int threads) {
  const Layout& A = *d.A;
  const Layout& B = *d.B;
  const BlockMap MA(A), MB(B);
  const bool tr = d.op != COSTA_OP_N;
  const int32_t P = A.nranks;
  // op(B) seen in A's coordinates: its row splits are B's column splits for T/C
  std::vector<Interval> rows = overlay(A.rsplit, tr ? B.csplit : B.rsplit);
  std::vector<Interval> cols = overlay(A.csplit, tr ? B.rsplit : B.csplit);
  const bool a_col = A.order == COSTA_COL_MAJOR;
  const bool b_col = B.order == COSTA_COL_MAJOR;
  // destination orientation: x along A's contiguous direction
  const std::vector<Interval>& X = a_col ? rows : cols;
  const std::vector<Interval>& Y = a_col ? cols : rows;
  const int32_t KX = (int32_t)X.size(), LY = (int32_t)Y.size();
  overlay_blocks += (int64_t)KX * LY;

  // whether c (starting on strip ly) continues q along y
  auto continues_y = [](const Cand& q, const Cand& c, int32_t ly) {
    const int64_t step = (q.p.flags & PIECE_TRANSPOSE) ? 1 : q.p.src_ld;
    return q.ly_end == ly && q.kx1 == c.kx1 && same_kind(q.p, c.p) &&
           c.p.dst_off == q.p.dst_off + (int64_t)q.p.ny * q.p.dst_ld &&
           c.p.src_off == q.p.src_off + (int64_t)q.p.ny * step && (int64_t)q.p.ny + c.p.ny <= INT32_MAX;
  };
  struct Range {
    std::vector<Cand> all;
    std::vector<int32_t> open;  // per kx0: candidate that may still grow along y
    int64_t n_local = 0, n_remote = 0;
  };
  const int64_t cells = (int64_t)KX * LY;
  const int nr = (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)threads, LY, cells / 65536 + 1}));
  std::vector<Range> R((size_t)nr);
  parallel_for(nr, nr, [&](int64_t ri_) {
    Range& rg = R[(size_t)ri_];
    const int32_t ly0 = (int32_t)((int64_t)LY * ri_ / nr), ly1 = (int32_t)((int64_t)LY * (ri_ + 1) / nr);
    rg.open.assign(KX, -1);
    std::vector<Cand> strip;
    for (int32_t ly = ly0; ly < ly1; ++ly) {
      strip.clear();
      const Interval& yi = Y[ly];
      for (int32_t kx = 0; kx < KX; ++kx) {
        const Interval& xi = X[kx];
        const Interval& ri = a_col ? xi : yi;  // row interval of this overlay block
        const Interval& ci = a_col ? yi : xi;  // column interval
        // destination block and label
        const int32_t t = MA.owner(ri.a, ci.a);
        const int32_t r = sigma.empty() ? t : sigma[t];
        const int64_t pi = ri.start - A.rsplit[ri.a], pj = ci.start - A.csplit[ci.a];
        const int64_t lda = MA.ld(ri.a, ci.a);
        const int64_t dst_off = MA.offset(ri.a, ci.a, lda) + (a_col ? pi + pj * lda : pi * lda + pj);
        // source block: op(B) block (ri.b, ci.b) is B block (ci.b, ri.b) for T/C
        const int32_t bi = tr ? ci.b : ri.b, bj = tr ? ri.b : ci.b;
        const int32_t s = MB.owner(bi, bj);
        const int64_t ldb = MB.ld(bi, bj);
        // B element of A's (i, j): B(i, j) for N, B(j, i) for T/C
        const int64_t qrow = tr ? ci.start - B.rsplit[bi] : ri.start - B.rsplit[bi];
        const int64_t qcol = tr ? ri.start - B.csplit[bj] : ci.start - B.csplit[bj];
        const int64_t s_brow = b_col ? 1 : ldb, s_bcol = b_col ? ldb : 1;  // strides of B's row / col index
        const int64_t src_off = MB.offset(bi, bj, ldb) + qrow * s_brow + qcol * s_bcol;
        const int64_t s_i = tr ? s_bcol : s_brow;  // stride along A's row index i
        const int64_t s_j = tr ? s_brow : s_bcol;  // stride along A's column index j
        const int64_t sx = a_col ? s_i : s_j, sy = a_col ? s_j : s_i;

        Cand c;
        Piece& p = c.p;
        p.dst_off = dst_off;
        p.dst_ld = lda;
        p.src_off = src_off;
        p.nx = (int32_t)xi.len;
        p.ny = (int32_t)yi.len;
        if (sx == 1 || p.nx == 1) {
          p.flags = 0;
          p.src_ld = sy;
        } else {
          p.flags = PIECE_TRANSPOSE;  // sy == 1 here: one of the strides is always 1
          p.src_ld = sx;
        }
        p.dst_buf = item * P + r;
        p.src_buf = nitems * P + item * P + s;
        p.item = item;
        p.task0 = 0;
        p.aux = 0;
        c.kx0 = kx;
        c.kx1 = kx + 1;
        c.ly_start = ly;
        c.ly_end = ly + 1;
        c.s = s;
        c.r = r;
        const int64_t ne = (int64_t)p.nx * p.ny;
        if (s == r) rg.n_local += ne;
        else rg.n_remote += ne;
        // merge along x with the previous rectangle of this strip
        if (!strip.empty()) {
          Piece& q = strip.back().p;
          const int64_t step = (q.flags & PIECE_TRANSPOSE) ? q.src_ld : 1;
          if (same_kind(q, p) && q.ny == p.ny && p.dst_off == q.dst_off + q.nx &&
              p.src_off == q.src_off + (int64_t)q.nx * step && (int64_t)q.nx + p.nx <= INT32_MAX) {
            q.nx += p.nx;
            strip.back().kx1 = kx + 1;
            continue;
          }
        }
        strip.push_back(c);
      }
      // merge along y with the rectangle of the previous strip with the same x range
      for (Cand& c : strip) {
        const int32_t o = rg.open[c.kx0];
        if (o >= 0 && continues_y(rg.all[o], c, ly)) {
          Cand& q = rg.all[o];
          q.p.ny += c.p.ny;
          q.ly_end = ly + 1;
          continue;
        }
        rg.open[c.kx0] = (int32_t)rg.all.size();
        rg.all.push_back(c);
      }
    }
  });
  // stitch the ranges in order: a rectangle on a range's first strip that
  // continues an open rectangle of the ranges before is merged into it
  std::vector<std::pair<int32_t, int32_t>> open((size_t)KX, {-1, -1});  // (range, index)
  std::vector<std::vector<char>> dead((size_t)nr);
  for (int r = 0; r < nr; ++r) {
    Range& rg = R[(size_t)r];
    n_local += rg.n_local;
    n_remote += rg.n_remote;
    dead[(size_t)r].assign(rg.all.size(), 0);
    const int32_t ly0 = (int32_t)((int64_t)LY * r / nr);
    std::vector<std::pair<int32_t, int32_t>> moved(rg.all.size());
    for (size_t j = 0; j < rg.all.size(); ++j) {
      Cand& c = rg.all[j];
      moved[j] = {r, (int32_t)j};
      if (r == 0 || c.ly_start != ly0) continue;
      const std::pair<int32_t, int32_t> o = open[(size_t)c.kx0];
      if (o.first < 0) continue;
      Cand& q = R[(size_t)o.first].all[(size_t)o.second];
      if (continues_y(q, c, ly0)) {
        q.p.ny += c.p.ny;
        q.ly_end = c.ly_end;
        moved[j] = o;
        dead[(size_t)r][j] = 1;
      }
    }
    for (int32_t kx = 0; kx < KX; ++kx)
      if (rg.open[kx] >= 0) open[(size_t)kx] = moved[(size_t)rg.open[kx]];
  }
  size_t nl = local.size(), nrem = remote.size();
  for (int r = 0; r < nr; ++r)
    for (size_t j = 0; j < R[(size_t)r].all.size(); ++j)
      if (!dead[(size_t)r][j]) (R[(size_t)r].all[j].s == R[(size_t)r].all[j].r ? nl : nrem) += 1;
  local.reserve(nl);
  remote.reserve(nrem);
  for (int r = 0; r < nr; ++r) {
    for (size_t j = 0; j < R[(size_t)r].all.size(); ++j) {
      const Cand& c = R[(size_t)r].all[j];
      if (!dead[(size_t)r][j]) (c.s == c.r ? local : remote).push_back(c);
    }
    std::vector<Cand>().swap(R[(size_t)r].all);
  }
}

// Cuts of a rectangle larger than max_elems elements: (x0, y0, nx, ny) of
// each sub-rectangle.  Row walks are cut into strips of whole rows where a row
// fits; transposed rectangles into strips whose width is a multiple of 128 and
// whose height is a multiple of 32 where possible, so that their LDS tiles
// stay full.
struct Cut {
  int64_t x0, y0, nx, ny;
};
void cuts_of(const Piece& p, int64_t max_elems, std::vector<Cut>& out) {
  out.clear();
  if ((int64_t)p.nx * p.ny <= max_elems) {
    out.push_back(Cut{0, 0, p.nx, p.ny});
    return;
  }
  const bool T = p.flags & PIECE_TRANSPOSE;
  int64_t cx, cy;
  if (T) {
    cx = std::min<int64_t>(p.nx, std::max<int64_t>(128, max_elems / 32));
    if (cx < p.nx && cx >= 128) cx -= cx % 128;
    cy = std::max<int64_t>(1, max_elems / cx);
    if (cy > 32) cy -= cy % 32;
  } else {
    cx = std::min<int64_t>(p.nx, max_elems);
    cy = std::max<int64_t>(1, max_elems / cx);
  }
  cy = std::min<int64_t>(cy, p.ny);
  for (int64_t y0 = 0; y0 < p.ny; y0 += cy)
    for (int64_t x0 = 0; x0 < p.nx; x0 += cx)
      out.push_back(Cut{x0, y0, std::min<int64_t>(cx, p.nx - x0), std::min<int64_t>(cy, p.ny - y0)});
}

// The sub-rectangle of p at cut c (source and destination offsets moved).
Piece sub_piece(const Piece& p, const Cut& c) {
  Piece d = p;
  const bool T = p.flags & PIECE_TRANSPOSE;
  d.nx = (int32_t)c.nx;
  d.ny = (int32_t)c.ny;
  d.dst_off = p.dst_off + c.y0 * p.dst_ld + c.x0;
  d.src_off = p.src_off + (T ? c.x0 * p.src_ld + c.y0 : c.y0 * p.src_ld + c.x0);
  return d;
}

// Splits rectangles larger than max_elems elements (see cuts_of).
void split_pieces(std::vector<Cand>& v, int64_t max_elems) {
  bool any = false;
  for (const Cand& c : v) any = any || (int64_t)c.p.nx * c.p.ny > max_elems;
  if (!any) return;
  std::vector<Cand> out;
  out.reserve(v.size());
  std::vector<Cut> cs;
  for (const Cand& c : v) {
    cuts_of(c.p, max_elems, cs);
    for (const Cut& k : cs) {
      Cand d = c;
      d.p = sub_piece(c.p, k);
      out.push_back(d);
    }
  }
  v.swap(out);
}

// Sets the flags the kernels read: 16-byte vectors for row walks, the LDS
// tile class of transposed rectangles.
void finish_piece(Piece& p, int elem_size) {
  p.flags &= ~(PIECE_WIDE | PIECE_GROUP_NEXT);
  p.task0 = 0;
  p.aux = 0;
  if (p.flags & PIECE_TRANSPOSE) {
    int32_t tx, ty;
    const bool aligned_cols = p.src_off * elem_size % 128 == 0 && (p.nx == 1 || p.src_ld * elem_size % 128 == 0);
    choose_tile(elem_size, p.nx, p.ny, aligned_cols, tx, ty);
    p.aux = tile_pack(tx, ty);
    return;
  }
  const int64_t want = wide_elems(elem_size);
  if (want > 1 && p.nx % want == 0 && p.src_off % want == 0 && p.dst_off % want == 0 &&
      (p.ny == 1 || (p.src_ld % want == 0 && p.dst_ld % want == 0)))
    p.flags |= PIECE_WIDE;
}

// Workgroup order per launch: one contiguous range of tasks per XCD when the
// launch's tasks are all of one kind (all row-walk chunks or all tiles, so
// that equal ranges are equal work) and nearly all of its elements lie in
// rectangles whose runs start and end on 128-byte lines; dispatch order
// otherwise.  Measured on MI355X: +5 to +8% on such launches; -5 to -8% on
// launches of short runs that share lines with their neighbours; -40% on a
// launch whose first half is row walks and second half LDS tiles (four XCDs
// idle while four finish the tiles).  COSTA_XCD_RANGES=0 turns it off.
#ifndef COSTA_XCD_RANGES
#define COSTA_XCD_RANGES 1
#endif
// Tenths of a launch's elements that must lie in line-aligned rectangles for
// the ranges (0: every launch of one kind; measured: the scaled transpose
// -8%, the complex case -4%, pdgemr2d's unpack +5% and its pack -1%).
#ifndef COSTA_XCD_ALIGNED_TENTHS
#define COSTA_XCD_ALIGNED_TENTHS 9
#endif
// 1: stacked rectangles count as aligned (measured: pdgemr2d -4%, pdtran -6%).
#ifndef COSTA_XCD_STACKS
#define COSTA_XCD_STACKS 0
#endif
// Row strides (bytes) from which rows count as far apart: such row walks
// cost more per task than walks of nearby rows, so a launch that holds both
// is not of one kind for the XCD ranges (measured on MI355X: the tall-skinny
// batch's pack, identity pairs with rows 32 KiB apart and transposed pairs
// with rows 4 MiB apart, +6 to +8% without the ranges, its step +2.5%; the
// transposed pairs alone -2 to -13% without them); it also decides the pack
// order below.
#ifndef COSTA_PACK_FAR_ROWS
#define COSTA_PACK_FAR_ROWS (1 << 20)
#endif
// 1: ranges also for launches whose rectangles are all contiguous on both
// sides (one sequential stream in task order; measured: the tall-skinny
// batch's identity pairs' unpack, 256 KiB blocks, step -0.9% with them).
#ifndef COSTA_XCD_DENSE
#define COSTA_XCD_DENSE 0
#endif

// Whether every run of the rectangle (its rows in the source and in the
// destination) starts and ends on a 128-byte line.
bool line_aligned(const Piece& p, int es) {
  auto al = [&](int64_t v) { return v * es % 128 == 0; };
  const bool T = p.flags & PIECE_TRANSPOSE;
  const int64_t srun = T ? p.ny : p.nx;  // source run length
  const int64_t sstep = T ? p.nx : p.ny;  // number of source runs
  return al(p.dst_off) && al(p.nx) && (p.ny == 1 || al(p.dst_ld)) && al(p.src_off) && al(srun) &&
         (sstep == 1 || al(p.src_ld));
}

// Whether rectangle `q` continues rectangle `p` along x on the source
// (side 0) or the destination (side 1): the same buffer and stride there, and
// q starting where p ends.
bool continues(const Piece& p, const Piece& q, int side) {
  if (side == 0)
    return q.src_buf == p.src_buf && (p.ny == 1 || q.src_ld == p.src_ld) && q.src_off == p.src_off + p.nx;
  return q.dst_buf == p.dst_buf && (p.ny == 1 || q.dst_ld == p.dst_ld) && q.dst_off == p.dst_off + p.nx;
}

// Marks the stacks of a launch of row walks (PIECE_STACK): maximal runs of
// consecutive rectangles of short rows that continue one another along x on
// one side.  Returns, per rectangle, the length of the stack it starts (0 when
// it starts none).  Rectangles cut from one block by the other layout's
// splits lie one after another in a local column on one side; moved as one
// band, each 64-lane access covers contiguous bytes there, and rows that end
// inside a 128-byte line are written whole by one wave.  Measured on MI355X:
// the ScaLAPACK-shaped copy with misaligned columns (32-row into 128-row
// blocks, 16 x 16 ranks) +7% per step; the scaled transpose's unpack with
// beta = 0 +4 to +7%, with beta != 0 -5% -- outside the pack (a copy), stacks
// form only from rectangles of pairs that do not read A (reads_a), and the
// kernel has no stack walk that reads A.
std::vector<int32_t> mark_stacks(std::vector<Piece>& ps, int es, bool is_pack, const std::vector<char>& reads_a) {
  std::vector<int32_t> len(ps.size(), 0);
  if (COSTA_STACK_MAX_RUN <= 0) return len;
  for (const Piece& p : ps)
    if (p.flags & PIECE_TRANSPOSE) return len;
  auto short_rows = [&](const Piece& p) {
    return (int64_t)p.nx * es >= COSTA_STACK_MIN_RUN && (int64_t)p.nx * es <= COSTA_STACK_MAX_RUN;
  };
  size_t k = 0;
  while (k < ps.size()) {
    const Piece& h = ps[k];
    size_t e = k + 1;
    int side = -1;
    int64_t width = h.nx;
    const int64_t epu = (h.flags & PIECE_WIDE) ? wide_elems(es) : 1;
    if (short_rows(h) && (is_pack || !reads_a[h.item])) {
      while (e < ps.size() && e - k < (size_t)kStackPiecesMax) {
        const Piece& q = ps[e];
        if (!short_rows(q) || q.item != h.item || q.ny != h.ny || (q.flags & PIECE_WIDE) != (h.flags & PIECE_WIDE) ||
            stack_wave_tasks((width + q.nx) / epu, h.ny) > kStackWaveTasksMax)
          break;
        if (side < 0) side = continues(ps[e - 1], q, 0) ? 0 : continues(ps[e - 1], q, 1) ? 1 : -1;
        if (side < 0 || !continues(ps[e - 1], q, side)) break;
        width += q.nx;
        ++e;
      }
    }
    // a stack narrower than a few waves leaves lanes of its last wave of
    // every row idle: keep the rectangles' own walks there (measured on
    // MI355X: stacks 50-300 units wide, the scaled transpose, 20% slower)
    const int64_t hu = width / epu;
    const int64_t lanes = (hu + kStackWave - 1) / kStackWave * kStackWave;
    if (e - k >= 2 && hu >= COSTA_STACK_MIN_UNITS && 10 * hu >= 9 * lanes) {
      len[k] = (int32_t)(e - k);
      for (size_t j = k; j < e; ++j) ps[j].flags |= PIECE_STACK | (side == 1 ? PIECE_STACK_DST : 0);
      ps[k].flags |= (int32_t)((uint32_t)(e - k) << 16);
    }
    k = e;
  }
  return len;
}

// Appends n tasks to a task table: task t of the launch moves the rectangle
// of the last segment (first task, rectangle) that starts at or before t.
void fill_tasks(std::vector<int32_t>& table, const std::vector<std::pair<int64_t, int32_t>>& seg, int64_t n) {
  const size_t at = table.size();
  table.resize(at + (size_t)n);
  int32_t* out = table.data() + at;
  const int threads = n >= (1 << 20) ? plan_threads() : 1;
  parallel_for(threads, threads, [&](int64_t t) {
    const size_t s0 = seg.size() * (size_t)t / (size_t)threads, s1 = seg.size() * (size_t)(t + 1) / (size_t)threads;
    for (size_t j = s0; j < s1; ++j) {
      const int64_t end = j + 1 < seg.size() ? seg[j + 1].first : n;
      std::fill(out + seg[j].first, out + end, seg[j].second);
    }
  });
}

// Appends one launch: its rectangles and the workgroups that move them, in
// rectangle order.  A transposed rectangle gets one workgroup per LDS tile
// (tiles along x first); a row walk one per kThreadsPerTask units; runs of
// small row walks of the same pair and vector width share one workgroup; a
// stack the workgroups of its bands (stack_tasks).
LaunchRange add_launch(HostPlan& hp, std::vector<Piece>& ps, int es, int32_t nitems, bool is_pack) {
  LaunchRange lr;
  lr.item_elems.assign(nitems, 0);
  lr.piece_begin = (int64_t)hp.pieces.size();
  lr.npieces = (int64_t)ps.size();
  lr.task_begin = (int64_t)hp.tasks.size();
  if (hp.pieces.size() + ps.size() > (size_t)INT32_MAX)
    throw LimitExceeded("more than 2^31-1 rectangles in one plan");
  const int32_t base = (int32_t)hp.pieces.size();
  const std::vector<int32_t> stack_len = mark_stacks(ps, es, is_pack, hp.item_reads_a);
  // tasks of the stack each rectangle starts (0 for the others)
  auto stack_ntasks = [&](size_t k) -> int64_t {
    const Piece& h = ps[k];
    const Piece& l = ps[k + stack_len[k] - 1];
    const int64_t width = (h.flags & PIECE_STACK_DST) ? l.dst_off + l.nx - h.dst_off : l.src_off + l.nx - h.src_off;
    return stack_tasks(width / ((h.flags & PIECE_WIDE) ? wide_elems(es) : 1), h.ny);
  };
  int64_t b = 0;
  // (first task, rectangle) of every rectangle that starts tasks; the tables
  // are filled from these once their sizes are known
  std::vector<std::pair<int64_t, int32_t>> seg;
  seg.reserve(ps.size());
  // the open run of small row walks
  int64_t g_task = -1;
  int64_t g_units = 0;
  int32_t g_count = 0;
  size_t g_last = 0;
  bool g_wide = false;
  int32_t g_item = 0;
  for (size_t k = 0; k < ps.size(); ++k) {
    Piece& p = ps[k];
    const int64_t ne = (int64_t)p.nx * p.ny;
    lr.elems += ne;
    lr.item_elems[p.item] += ne;
    const int32_t pi = base + (int32_t)k;
    if (p.flags & PIECE_STACK) {
      g_task = -1;
      if (stack_len[k] == 0) {  // a later rectangle of the stack
        p.task0 = ps[k - 1].task0;
        continue;
      }
      const int64_t n = stack_ntasks(k);
      p.task0 = (int32_t)b;
      seg.emplace_back(b, pi);
      b += n;
      continue;
    }
    if (p.flags & PIECE_TRANSPOSE) {
      lr.has_transpose = true;
      g_task = -1;
      const int32_t tx = tile_x_of(p.aux), ty = tile_y_of(p.aux);
      const int64_t n = (int64_t)((p.nx + tx - 1) / tx) * ((p.ny + ty - 1) / ty);
      p.task0 = (int32_t)b;
      seg.emplace_back(b, pi);
      b += n;
      continue;
    }
    const bool wide = p.flags & PIECE_WIDE;
    const int64_t units = wide ? ne / wide_elems(es) : ne;
    if (units <= kGroupUnitsMax && g_task >= 0 && wide == g_wide && p.item == g_item &&
        g_units + units <= kThreadsPerTask && g_count < kGroupPiecesMax) {
      ps[g_last].flags |= PIECE_GROUP_NEXT;
      p.task0 = (int32_t)g_task;
      g_units += units;
      ++g_count;
      g_last = k;
      continue;
    }
    const int64_t n = (units + kThreadsPerTask - 1) / kThreadsPerTask;
    p.task0 = (int32_t)b;
    seg.emplace_back(b, pi);
    b += n;
    if (units <= kGroupUnitsMax) {
      g_task = b - 1;
      g_units = units;
      g_count = 1;
      g_last = k;
      g_wide = wide;
      g_item = p.item;
    } else {
      g_task = -1;
    }
  }
  if (b > INT32_MAX) throw LimitExceeded("more than 2^31-1 workgroups in one launch");
  lr.ntasks = b;
  // Which tables the kernels read (the units per lane of each launch): the
  // pack always copies (the wide table, unless COSTA_COPY_UNITS is 1); an
  // unpack or direct launch copies only in calls that read no A, and a plan
  // built for pairs that read A serves only such calls (reads_a is part of
  // the plan key), so its launches never read the wide table.  The first
  // tasks and counts of both are kept whatever is filled.
  bool plan_reads_a = false;
  for (char r : hp.item_reads_a) plan_reads_a = plan_reads_a || r;
  const bool need_narrow = !is_pack || COSTA_COPY_UNITS <= 1;
  const bool need_wide = is_pack ? COSTA_COPY_UNITS > 1 : !plan_reads_a;
  if (need_narrow) fill_tasks(hp.tasks, seg, b);
  // the wide task table of a launch of row walks: kWideTaskUnits units per
  // task, a run of small rectangles still one task
  lr.wide_begin = (int64_t)hp.wide_tasks.size();
  if (!lr.has_transpose) {
    int64_t b2 = 0;
    seg.clear();
    for (size_t k = 0; k < ps.size(); ++k) {
      Piece& p = ps[k];
      if (k > 0 && ((ps[k - 1].flags & PIECE_GROUP_NEXT) || ((p.flags & PIECE_STACK) && stack_len[k] == 0))) {
        p.aux = ps[k - 1].aux;
        continue;
      }
      if (p.flags & PIECE_STACK) {  // the same tasks as in the task table
        const int64_t n = stack_ntasks(k);
        p.aux = (int32_t)b2;
        seg.emplace_back(b2, base + (int32_t)k);
        b2 += n;
        continue;
      }
      const int64_t ne = (int64_t)p.nx * p.ny;
      const int64_t units = (p.flags & PIECE_WIDE) ? ne / wide_elems(es) : ne;
      const int64_t n = (p.flags & PIECE_GROUP_NEXT) ? 1 : (units + kWideTaskUnits - 1) / kWideTaskUnits;
      p.aux = (int32_t)b2;
      seg.emplace_back(b2, base + (int32_t)k);
      b2 += n;
    }
    lr.nwide = b2;
    if (need_wide) fill_tasks(hp.wide_tasks, seg, b2);
  }
  int64_t aligned = 0, transposed = 0, far = 0, near = 0, dense = 0;
  for (const Piece& p : ps) {
    const int64_t ne = (int64_t)p.nx * p.ny;
    if (!(p.flags & PIECE_TRANSPOSE) && (p.ny == 1 || (p.src_ld == p.nx && p.dst_ld == p.nx))) dense += ne;
    if (line_aligned(p, es) || (COSTA_XCD_STACKS && (p.flags & PIECE_STACK))) aligned += ne;
    if (p.flags & PIECE_TRANSPOSE) transposed += ne;
    else if (p.ny > 1) (std::max(p.src_ld, p.dst_ld) * es >= COSTA_PACK_FAR_ROWS ? far : near) += ne;
  }
  const bool one_kind = (transposed == 0 || transposed == lr.elems) && (far == 0 || near == 0);
  lr.xcd_ranges = COSTA_XCD_RANGES && one_kind && (COSTA_XCD_DENSE || dense < lr.elems) && lr.elems > 0 && 10 * aligned >= COSTA_XCD_ALIGNED_TENTHS * lr.elems ? 1 : 0;
  hp.pieces.insert(hp.pieces.end(), ps.begin(), ps.end());
  return lr;
}

#ifndef COSTA_PACK_BY_SOURCE
#define COSTA_PACK_BY_SOURCE 1
#endif
// Split an unpack or direct launch that holds both row walks and LDS tiles
// into one launch of each kind (tiles first), so that each can take the
// per-XCD workgroup ranges (measured on MI355X: tall-skinny batch of 4
// identity + 4 transposed pairs: unpack +8%, whole step +4%).
#ifndef COSTA_SPLIT_KINDS
#define COSTA_SPLIT_KINDS 1
#endif

// The launches of one kernel kind over `ps` (sorted): one, or a tile launch
// and a row-walk launch.
std::vector<LaunchRange> add_launches(HostPlan& hp, std::vector<Piece>& ps, int es, int32_t nitems) {
  std::vector<LaunchRange> out;
  if (ps.empty()) return out;
  std::vector<Piece> tiles, walks;
  size_t ntiles = 0;
  for (const Piece& p : ps) ntiles += (p.flags & PIECE_TRANSPOSE) ? 1 : 0;
  if (COSTA_SPLIT_KINDS && ntiles > 0 && ntiles < ps.size()) {
    for (const Piece& p : ps) ((p.flags & PIECE_TRANSPOSE) ? tiles : walks).push_back(p);
  }
  if (tiles.empty() || walks.empty()) {
    out.push_back(add_launch(hp, ps, es, nitems, false));
  } else {
    out.push_back(add_launch(hp, tiles, es, nitems, false));
    out.push_back(add_launch(hp, walks, es, nitems, false));
  }
  return out;
}

// Sorts v by key(element) through an array of (key, index) pairs instead of
// moving the elements around.  Every key used below is unique (each element
// of A and of B lies in exactly one rectangle), so the order is the one a
// sort of the elements themselves gives.
template <typename T, typename KeyFn>
void sort_by_key(std::vector<T>& v, KeyFn key) {
  using K = decltype(key(v[0]));
  if (v.size() > (size_t)UINT32_MAX) throw LimitExceeded("more than 2^32-1 rectangles to order");
  const size_t n = v.size();
  std::vector<std::pair<K, uint32_t>> ix(n);
  // sorted runs on several threads, merged pairwise (the keys are unique, so
  // the order is the one a single sort gives)
  const int threads = n >= (1u << 16) ? plan_threads() : 1;
  int64_t runs = 1;
  while (runs < threads) runs *= 2;
  std::vector<size_t> bound((size_t)runs + 1);
  for (int64_t r = 0; r <= runs; ++r) bound[(size_t)r] = n * (size_t)r / (size_t)runs;
  parallel_for(runs, threads, [&](int64_t r) {
    for (size_t i = bound[(size_t)r]; i < bound[(size_t)r + 1]; ++i) ix[i] = {key(v[i]), (uint32_t)i};
    std::sort(ix.begin() + (ptrdiff_t)bound[(size_t)r], ix.begin() + (ptrdiff_t)bound[(size_t)r + 1]);
  });
  for (int64_t width = 1; width < runs; width *= 2) {
    parallel_for(runs / (2 * width), threads, [&](int64_t m) {
      const size_t lo = bound[(size_t)(2 * width * m)], mid = bound[(size_t)(2 * width * m + width)],
                   hi = bound[(size_t)(2 * width * m + 2 * width)];
      std::inplace_merge(ix.begin() + (ptrdiff_t)lo, ix.begin() + (ptrdiff_t)mid, ix.begin() + (ptrdiff_t)hi);
    });
  }
  std::vector<T> out(n);
  parallel_for(threads, threads, [&](int64_t r) {
    for (size_t i = n * (size_t)r / (size_t)threads; i < n * (size_t)(r + 1) / (size_t)threads; ++i)
      out[i] = std::move(v[ix[i].second]);
  });
  v.swap(out);
}

std::pair<int32_t, int64_t> dst_key(const Piece& p) { return {p.dst_buf, p.dst_off}; }
std::pair<int32_t, int64_t> src_key(const Piece& p) { return {p.src_buf, p.src_off}; }

}  // namespace

void build_plan(const std::vector<ItemDesc>& items, const std::vector<int32_t>& sigma, const PlanConfig& cfg,
                const std::function<int64_t(int64_t)>& choose_cap, HostPlan& hp) {
  auto t0 = std::chrono::steady_clock::now();
  const int32_t n = (int32_t)items.size();
  const int es = cfg.elem_size;
  hp = HostPlan();
  hp.item_total.assign(n, 0);
  hp.item_local.assign(n, 0);
  hp.item_remote.assign(n, 0);
  hp.item_reads_a.assign(n, 0);
  for (int32_t k = 0; k < n; ++k) hp.item_reads_a[k] = items[k].reads_a ? 1 : 0;
  std::vector<Cand> local, remote;
  {
    // the pairs on several threads, joined in pair order
    std::vector<std::vector<Cand>> loc((size_t)n), rem((size_t)n);
    std::vector<int64_t> blocks((size_t)n, 0);
    const int threads = plan_threads();
    const int inner = std::max(1, threads / std::max(1, n));  // threads per pair
    parallel_for(n, threads, [&](int64_t k) {
      hp.item_total[k] = items[k].A->nrows * items[k].A->ncols;
      plan_pair((int32_t)k, n, items[k], sigma, loc[k], rem[k], blocks[k], hp.item_local[k], hp.item_remote[k],
                inner);
    });
    size_t nl = 0, nr = 0;
    for (int32_t k = 0; k < n; ++k) {
      nl += loc[k].size();
      nr += rem[k].size();
      hp.overlay_blocks += blocks[k];
    }
    local.reserve(nl);
    remote.reserve(nr);
    for (int32_t k = 0; k < n; ++k) {
      local.insert(local.end(), loc[k].begin(), loc[k].end());
      remote.insert(remote.end(), rem[k].begin(), rem[k].end());
      std::vector<Cand>().swap(loc[k]);
      std::vector<Cand>().swap(rem[k]);
    }
  }
  split_pieces(local, cfg.max_piece_elems);
  split_pieces(remote, cfg.max_piece_elems);

  // direct path, in destination order
  std::vector<Piece> direct;
  direct.reserve(local.size());
  for (Cand& c : local) {
    finish_piece(c.p, es);
    direct.push_back(c.p);
  }
  sort_by_key(direct, dst_key);
  hp.pieces_direct = (int32_t)direct.size();

  // messages: packages ordered by sender, then receiver (each sender's send
  // buffer holds one contiguous package per receiver; plans of several waves
  // reorder them by receiver below); blocks in source order
  auto by_package = [](const Cand& c) { return std::make_tuple(c.s, c.r, c.p.src_buf, c.p.src_off); };
  sort_by_key(remote, by_package);
  auto chunk_bytes = [&](const Piece& p) {
    int64_t b = (int64_t)p.nx * p.ny * es;
    return (b + 255) / 256 * 256;  // every message block starts 256-byte aligned
  };
  int64_t total_msg = 0, biggest = 0;
  for (const Cand& c : remote) {
    total_msg += chunk_bytes(c.p);
    biggest = std::max(biggest, chunk_bytes(c.p));
  }
  int64_t cap = choose_cap ? choose_cap(total_msg) : cfg.workspace_cap;
  if (biggest > cap) {
    // a small workspace: cut the blocks so that each fits one wave
    split_pieces(remote, std::max<int64_t>(1, (cap - 255) / es));
    sort_by_key(remote, by_package);
    biggest = 0;
    for (const Cand& c : remote) biggest = std::max(biggest, chunk_bytes(c.p));
  }
  cap = std::max(cap, biggest);
  if (total_msg > cap) {
    // Several waves: packages ordered by receiver, then sender, so that each
    // wave holds every package of a range of receivers and the rectangles
    // that border one another in A (from different senders) are unpacked by
    // the same launch.  Cut by sender instead, neighbours land in different
    // waves and the lines they share are read and written once per wave
    // (measured on MI355X, the scaled transpose with a 1 GiB workspace, 3
    // waves: 3.63 ms by sender, 2.85 by receiver; the tall-skinny batch's 7
    // waves: equal).
    sort_by_key(remote, [](const Cand& c) { return std::make_tuple(c.r, c.s, c.p.src_buf, c.p.src_off); });
  }

  // room for the task tables and rectangles of every launch (an upper bound
  // of the tasks: one per 256 elements, plus the rounding of each
  // rectangle), so that appending launches does not move the tables
  {
    int64_t est = 0;
    for (const Cand& c : remote) est += 2 * ((int64_t)c.p.nx * c.p.ny / kThreadsPerTask + 2);
    for (const Piece& p : direct) est += (int64_t)p.nx * p.ny / kThreadsPerTask + 2;
    hp.tasks.reserve((size_t)est);
    hp.wide_tasks.reserve((size_t)est);
    hp.pieces.reserve(2 * remote.size() + direct.size());
  }
  const int32_t msg_buf = 2 * n * (items.empty() ? 0 : items[0].A->nranks);
  size_t k = 0;
  while (k < remote.size()) {
    std::vector<Piece> pack, unpack;
    int64_t off = 0;
    while (k < remote.size() && (off == 0 || off + chunk_bytes(remote[k].p) <= cap)) {
      const Piece& q = remote[k].p;
      const bool T = q.flags & PIECE_TRANSPOSE;
      // pack: B -> message, always in the source's orientation (a plain copy)
      Piece pk = q;
      pk.flags = 0;
      pk.nx = T ? q.ny : q.nx;
      pk.ny = T ? q.nx : q.ny;
      pk.src_ld = q.src_ld;
      pk.dst_buf = msg_buf;
      pk.dst_off = off / es;
      pk.dst_ld = pk.nx;
      finish_piece(pk, es);
      pack.push_back(pk);
      // unpack-transform: message -> A, the block read back in the source's
      // orientation
      Piece up = q;
      up.src_buf = msg_buf;
      up.src_off = off / es;
      up.src_ld = T ? q.ny : q.nx;
      finish_piece(up, es);
      unpack.push_back(up);
      off += chunk_bytes(q);
      ++k;
    }
    // When many source rows start or end inside a 128-byte line (blocks cut
    // by the other layout's splits), the pack walks the sources in storage
    // order, so that rectangles sharing an edge line are read by the same or
    // neighbouring workgroups while the line is still in L2; likewise when
    // many rectangles' source rows lie COSTA_PACK_FAR_ROWS bytes or more
    // apart (a tall source's local columns): in package order the workgroups
    // in flight then read rows of a few rectangles, all that far apart
    // (measured on MI355X: the tall-skinny batch's transposed pairs, rows
    // 4 MiB apart, pack +8.6% alone; the whole batch's pack +5%, four
    // processes each way).  Otherwise it keeps
    // package order (sequential message writes).  The message offsets stay
    // in package order either way.
    int64_t partial = 0;
    for (const Piece& pk : pack) {
      const int64_t a = pk.src_off * es % 128, e = (pk.src_off + pk.nx) * es % 128;
      if (a != 0 || e != 0 || (pk.ny > 1 && pk.src_ld * es % 128 != 0)) ++partial;
      else if (COSTA_PACK_FAR_ROWS > 0 && pk.ny > 1 && pk.src_ld * es >= COSTA_PACK_FAR_ROWS) ++partial;
    }
    if (COSTA_PACK_BY_SOURCE && 4 * partial > (int64_t)pack.size()) sort_by_key(pack, src_key);
    hp.pieces_pack += (int32_t)pack.size();
    hp.pieces_unpack += (int32_t)unpack.size();
    const bool last = k == remote.size();
    if (last && COSTA_MERGE_DIRECT) {
      // the direct rectangles join the last unpack launch: one pass writes A
      // in destination order (the kernel reads each rectangle's source from
      // the buffer its descriptor names, B or the message workspace)
      unpack.insert(unpack.end(), direct.begin(), direct.end());
      direct.clear();
    }
    sort_by_key(unpack, dst_key);
    Wave w;
    w.msg_bytes = off;
    w.pack = add_launch(hp, pack, es, n, true);
    w.unpack = add_launches(hp, unpack, es, n);
    hp.workspace_bytes = std::max(hp.workspace_bytes, off);
    hp.waves.push_back(w);
  }
  hp.direct = add_launches(hp, direct, es, n);  // empty when merged above
  hp.plan_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

}  // namespace costa
