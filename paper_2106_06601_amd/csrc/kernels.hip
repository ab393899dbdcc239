// HIP kernels for gfx950 (CDNA4): the rectangle mover used by the pack,
// unpack-transform and direct paths, and the grid-overlay volume kernel.
//
// All of them are bound by HBM bandwidth: per element they read at most two
// values and write one, with at most a few flops (Section 5 eq:costa).  The
// movers are therefore built from one-shot workgroups: each takes one task
// from the plan's task table -- 256 or 512 consecutive 16-byte units (or
// elements) of a rectangle walked along its rows, four wave tasks of a stack
// of short rectangles that follow one another along a local column, or one
// LDS tile of a rectangle whose source and destination run in different
// directions -- moves it with coalesced 64-lane accesses and exits, so the
// workgroups in flight sweep the buffers in task order.  A launch whose
// tasks are all alike may hand each XCD (one L2) a contiguous range of them.
#include <hip/hip_runtime.h>

#include "internal.hpp"

// Products and sums are rounded one by one, never fused into an FMA, so the
// results are reproducible bit for bit.
#pragma clang fp contract(off)

namespace costa {
namespace {

// Tuning switches (compile-time; the defaults are the measured best).
#ifndef COSTA_NT_LOADS
#define COSTA_NT_LOADS 1  // row walks: each source line is read once
#endif
#ifndef COSTA_NT_LOADS_MAX_ES
#define COSTA_NT_LOADS_MAX_ES 8  // ...for element sizes up to this (measured: helps fp64, hurts complex128)
#endif
#ifndef COSTA_NT_TILE_LOADS
#define COSTA_NT_TILE_LOADS 0  // tile loads: lines may serve two neighbouring tiles
#endif
#ifndef COSTA_NT_FULL_TILE_LOADS
#define COSTA_NT_FULL_TILE_LOADS 1  // ...except in a tile as tall as its rectangle (pdtran +2.7% per step;
#endif                              // all tile loads NT: the complex case -19%)
#ifndef COSTA_NT_STORES
#define COSTA_NT_STORES 1
#endif
#ifndef COSTA_NT_ALOADS
#define COSTA_NT_ALOADS 0  // loads of A in row walks (measured: 1 makes the scaled transpose's unpack 29% slower)
#endif
// Loads of A in LDS tiles.  Measured with 1: the tiles' unpack 1-2% slower,
// but the pack of the next call faster (pztranc's +7%, the tall-skinny
// batch's +1 to +3%): whole steps +1.2 to +1.4%.
#ifndef COSTA_NT_TILE_ALOADS
#define COSTA_NT_TILE_ALOADS 1
#endif

constexpr int kThreads = kThreadsPerTask;

// The task of workgroup b of n.  Workgroups are dispatched round-robin over
// the 8 XCDs (b % 8 is b's XCD).  ranges 0: task b.  ranges 1: XCD x takes
// the x-th of 8 contiguous ranges of tasks, workgroup b the (b/8)-th task of
// its XCD's range.
__device__ __forceinline__ int32_t xcd_order(int32_t b, int32_t n, int32_t ranges) {
  constexpr int32_t X = 8;
  if (!ranges) return b;
  const int32_t q = n / X, r = n % X;
  const int32_t xcd = b % X, idx = b / X;
  const int32_t start = xcd < r ? xcd * (q + 1) : r * (q + 1) + (xcd - r) * q;
  return start + idx;
}

template <typename S, int N>
struct alignas(sizeof(S) * N) Vec {
  S v[N];
};

// Raw integer vector of a given size, for loads and stores with an optional
// non-temporal hint (streaming data that is touched exactly once).
template <int BYTES>
struct Raw;
template <>
struct Raw<4> {
  using T = uint32_t;
};
template <>
struct Raw<8> {
  typedef uint32_t T __attribute__((ext_vector_type(2)));
};
template <>
struct Raw<16> {
  typedef uint32_t T __attribute__((ext_vector_type(4)));
};

// The buffers reach the kernels through a pointer table, so the compiler
// cannot see that they are global memory; the casts below make it emit global
// (not flat) loads and stores, which do not share a wait counter with LDS.
#define COSTA_GLOBAL __attribute__((address_space(1)))

template <bool NT = COSTA_NT_LOADS, typename U>
__device__ __forceinline__ U load(const U* p) {
  using R = typename Raw<sizeof(U)>::T;
  const COSTA_GLOBAL R* g = (const COSTA_GLOBAL R*)(p);
  R r;
  if constexpr (NT) r = __builtin_nontemporal_load(g);
  else r = *g;
  U u;
  __builtin_memcpy(&u, &r, sizeof(U));
  return u;
}

template <typename U>
__device__ __forceinline__ void store(U* p, const U& u) {
  using R = typename Raw<sizeof(U)>::T;
  COSTA_GLOBAL R* g = (COSTA_GLOBAL R*)(p);
  R r;
  __builtin_memcpy(&r, &u, sizeof(U));
  if constexpr (COSTA_NT_STORES) __builtin_nontemporal_store(r, g);
  else *g = r;
}

// Element arithmetic for a vector of NU scalars (pairs of them for complex).
template <typename S, int NU, bool CPLX, int MODE, bool CONJ>
__device__ __forceinline__ Vec<S, NU> combine(const Vec<S, NU>& b, const Vec<S, NU>& a, S ar, S ai, S br, S bi) {
  Vec<S, NU> o;
  if constexpr (CPLX) {
#pragma unroll
    for (int k = 0; k < NU; k += 2) {
      const S xr = b.v[k];
      const S xi = CONJ ? -b.v[k + 1] : b.v[k + 1];
      if constexpr (MODE == MODE_COPY) {
        o.v[k] = xr;
        o.v[k + 1] = xi;
      } else {
        const S p1 = ar * xr, p2 = ai * xi, p3 = ar * xi, p4 = ai * xr;
        S t1r = p1 - p2, t1i = p3 + p4;
        if constexpr (MODE == MODE_AXPBY) {
          const S q1 = br * a.v[k], q2 = bi * a.v[k + 1], q3 = br * a.v[k + 1], q4 = bi * a.v[k];
          const S t2r = q1 - q2, t2i = q3 + q4;
          t1r = t1r + t2r;
          t1i = t1i + t2i;
        }
        o.v[k] = t1r;
        o.v[k + 1] = t1i;
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      if constexpr (MODE == MODE_COPY) {
        o.v[k] = b.v[k];
      } else if constexpr (MODE == MODE_SCALE) {
        o.v[k] = ar * b.v[k];
      } else {
        const S t1 = ar * b.v[k];
        const S t2 = br * a.v[k];
        o.v[k] = t1 + t2;
      }
    }
  }
  return o;
}

template <typename S, bool CPLX>
struct TypeTraits {
  static constexpr int NS = CPLX ? 2 : 1;         // scalars per element
  static constexpr int ES = (int)sizeof(S) * NS;  // bytes per element
  static constexpr int WIDE_NEL = wide_elems(ES); // elements per 16-byte unit
  static constexpr bool NT_WALK = COSTA_NT_LOADS && ES <= COSTA_NT_LOADS_MAX_ES;
  static constexpr int LDS_ELEMS = tile_lds_elems(ES);
  static constexpr int TILE_PASSES = (tile_max_elems(ES) + kThreads - 1) / kThreads;  // elements per lane
};

// y = u / n and x = u - y*n from a float estimate of the quotient, corrected
// to the exact one (u, n < 2^24: at most one step each way).
__device__ __forceinline__ void divmod(int32_t u, int32_t n, int32_t& y, int32_t& x) {
  y = (int32_t)((float)u * (1.0f / (float)n));
  x = u - y * n;
  while (x < 0) {
    --y;
    x += n;
  }
  while (x >= n) {
    ++y;
    x -= n;
  }
}

// Row walk: dst[y*dst_ld + x] = f(src[y*src_ld + x]).  The task starts at
// unit u0 of rectangle pi (a unit is a 16-byte vector for PIECE_WIDE
// rectangles, else one element; the flattened (y, x) index of a rectangle
// numbers its units) and covers the next UL*kThreads units: lane l takes
// units u0 + l + k*kThreads, k < UL.  A run of small rectangles
// (PIECE_GROUP_NEXT) is flattened the same way, its units one rectangle after
// another.  A lane issues all its loads (and those of A when it is read)
// before its stores.
template <typename S, bool CPLX, int MODE, bool CONJ, int UL>
__device__ __forceinline__ void move_walk(const Piece* __restrict__ pieces, int32_t pi, int32_t u0,
                                          void* const* __restrict__ bufs, int32_t allow_wide, S ar, S ai, S br,
                                          S bi) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  constexpr int W = TT::WIDE_NEL;
  const Piece& p0 = pieces[pi];
  const bool wide = (p0.flags & PIECE_WIDE) != 0;  // the same over a run
  const int32_t epu = wide ? W : 1;                // elements per unit
  const S* __restrict__ srcs[UL];
  S* __restrict__ dsts[UL];
  int64_t soffs[UL], doffs[UL];
  const int32_t nxu0 = wide ? p0.nx / W : p0.nx;
  const int32_t units0 = nxu0 * p0.ny;
  if (u0 + UL * kThreads <= units0) {
    // the whole task lies in rectangle pi: its fields are the same for every lane
    const S* src = reinterpret_cast<const S*>(bufs[p0.src_buf]);
    S* dst = reinterpret_cast<S*>(bufs[p0.dst_buf]);
#pragma unroll
    for (int k = 0; k < UL; ++k) {
      int32_t y, x;
      divmod(u0 + k * kThreads + (int32_t)threadIdx.x, nxu0, y, x);
      soffs[k] = p0.src_off + (int64_t)y * p0.src_ld + (int64_t)x * epu;
      doffs[k] = p0.dst_off + (int64_t)y * p0.dst_ld + (int64_t)x * epu;
      srcs[k] = src;
      dsts[k] = dst;
    }
  } else {
    // the task runs past the end of rectangle pi (into the next ones of a
    // run of small rectangles, or past the rectangle's end): walk the
    // rectangles it spans one by one, the same for every lane, each lane
    // keeping the one that holds its unit
    int32_t uu[UL];
#pragma unroll
    for (int k = 0; k < UL; ++k) {
      uu[k] = u0 + k * kThreads + (int32_t)threadIdx.x;
      soffs[k] = -1;
      doffs[k] = 0;
      srcs[k] = nullptr;
      dsts[k] = nullptr;
    }
    int32_t q = pi;
    int32_t rem = u0 + UL * kThreads;  // units of the task at or past rectangle q
    while (true) {
      const Piece& p = pieces[q];
      const int32_t nxu = wide ? p.nx / W : p.nx;
      const int32_t units = nxu * p.ny;
#pragma unroll
      for (int k = 0; k < UL; ++k) {
        if (uu[k] >= 0 && uu[k] < units) {
          int32_t y, x;
          divmod(uu[k], nxu, y, x);
          soffs[k] = p.src_off + (int64_t)y * p.src_ld + (int64_t)x * epu;
          doffs[k] = p.dst_off + (int64_t)y * p.dst_ld + (int64_t)x * epu;
          srcs[k] = reinterpret_cast<const S*>(bufs[p.src_buf]);
          dsts[k] = reinterpret_cast<S*>(bufs[p.dst_buf]);
        }
        uu[k] -= units;
      }
      rem -= units;
      if (rem <= 0 || !(p.flags & PIECE_GROUP_NEXT)) break;
      ++q;
    }
  }
  if (W > 1 && wide && allow_wide) {
    using U = Vec<S, TT::NS * W>;
    U bv[UL], av[UL];
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        bv[k] = load<TT::NT_WALK>(reinterpret_cast<const U*>(srcs[k] + soffs[k] * TT::NS));
        if constexpr (MODE == MODE_AXPBY) av[k] = load<COSTA_NT_ALOADS>(reinterpret_cast<U*>(dsts[k] + doffs[k] * TT::NS));
      }
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0)
        store(reinterpret_cast<U*>(dsts[k] + doffs[k] * TT::NS),
              combine<S, TT::NS * W, CPLX, MODE, CONJ>(bv[k], av[k], ar, ai, br, bi));
  } else {
    // one element at a time (epu of them: a PIECE_WIDE rectangle in a call
    // whose buffers are not 16-byte aligned)
    E bv[UL][W], av[UL][W];
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        const E* se = reinterpret_cast<const E*>(srcs[k]) + soffs[k];
        E* de = reinterpret_cast<E*>(dsts[k]) + doffs[k];
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu) {
            bv[k][j] = load<TT::NT_WALK>(se + j);
            if constexpr (MODE == MODE_AXPBY) av[k][j] = load<COSTA_NT_ALOADS>(de + j);
          }
      }
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        E* de = reinterpret_cast<E*>(dsts[k]) + doffs[k];
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu) store(de + j, combine<S, TT::NS, CPLX, MODE, CONJ>(bv[k][j], av[k][j], ar, ai, br, bi));
      }
  }
}

// The same row walk, with each lane finding its rectangle of a run on its
// own (the rectangle's fields and buffer pointers then live in vector
// registers).  Used for 16-byte elements: measured on MI355X, the complex128
// pack of the COSMA-like case runs 9% faster this way than with the
// walk above, while the 8-byte and smaller walks of short rows run 3-5%
// slower.  Task c of the rectangle covers units [c*UL*kThreads,
// (c+1)*UL*kThreads) of its flattened (y, x) index.
template <typename S, bool CPLX, int MODE, bool CONJ, int UL>
__device__ __forceinline__ void move_walk_lanes(const Piece* __restrict__ pieces, int32_t pi, int32_t c,
                                          void* const* __restrict__ bufs, int32_t allow_wide, S ar, S ai, S br,
                                          S bi) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  constexpr int W = TT::WIDE_NEL;
  const bool wide = (pieces[pi].flags & PIECE_WIDE) != 0;  // the same over a run
  const int32_t epu = wide ? W : 1;                         // elements per unit
  const S* __restrict__ srcs[UL];
  S* __restrict__ dsts[UL];
  int64_t soffs[UL], doffs[UL];
#pragma unroll
  for (int k = 0; k < UL; ++k) {
    int32_t u = c * (UL * kThreads) + k * kThreads + (int32_t)threadIdx.x;
    int64_t soff = -1, doff = 0;
    int32_t sbuf = 0, dbuf = 0;
    int32_t q = pi;
    while (true) {
      const Piece& p = pieces[q];
      const int32_t nxu = wide ? p.nx / W : p.nx;
      const int32_t units = nxu * p.ny;
      if (u >= 0 && u < units) {
        int32_t y, x;
        divmod(u, nxu, y, x);
        soff = p.src_off + (int64_t)y * p.src_ld + (int64_t)x * epu;
        doff = p.dst_off + (int64_t)y * p.dst_ld + (int64_t)x * epu;
        sbuf = p.src_buf;
        dbuf = p.dst_buf;
      }
      u -= units;
      if (!(p.flags & PIECE_GROUP_NEXT)) break;
      ++q;
    }
    soffs[k] = soff;
    doffs[k] = doff;
    srcs[k] = reinterpret_cast<const S*>(bufs[sbuf]);
    dsts[k] = reinterpret_cast<S*>(bufs[dbuf]);
  }
  if (W > 1 && wide && allow_wide) {
    using U = Vec<S, TT::NS * W>;
    U bv[UL], av[UL];
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        bv[k] = load<TT::NT_WALK>(reinterpret_cast<const U*>(srcs[k] + soffs[k] * TT::NS));
        if constexpr (MODE == MODE_AXPBY) av[k] = load<COSTA_NT_ALOADS>(reinterpret_cast<U*>(dsts[k] + doffs[k] * TT::NS));
      }
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0)
        store(reinterpret_cast<U*>(dsts[k] + doffs[k] * TT::NS),
              combine<S, TT::NS * W, CPLX, MODE, CONJ>(bv[k], av[k], ar, ai, br, bi));
  } else {
    // one element at a time (epu of them: a PIECE_WIDE rectangle in a call
    // whose buffers are not 16-byte aligned)
    E bv[UL][W], av[UL][W];
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        const E* se = reinterpret_cast<const E*>(srcs[k]) + soffs[k];
        E* de = reinterpret_cast<E*>(dsts[k]) + doffs[k];
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu) {
            bv[k][j] = load<TT::NT_WALK>(se + j);
            if constexpr (MODE == MODE_AXPBY) av[k][j] = load<COSTA_NT_ALOADS>(de + j);
          }
      }
#pragma unroll
    for (int k = 0; k < UL; ++k)
      if (soffs[k] >= 0) {
        E* de = reinterpret_cast<E*>(dsts[k]) + doffs[k];
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu) store(de + j, combine<S, TT::NS, CPLX, MODE, CONJ>(bv[k][j], av[k][j], ar, ai, br, bi));
      }
  }
}

// Stack walk (PIECE_STACK): the rectangles of a stack follow one another
// along x on one side, so the stack is walked as one band of hu units per y,
// in wave tasks of 64 units by kStackRows rows: wave v of task c takes wave
// task t = 4c + v, units [64 * (t % wb), +64) of x -- one per lane, the same
// for every row -- and rows [kStackRows * (t / wb), +kStackRows) of y.  The
// wave finds once which rectangle holds each lane's unit (a binary search for
// the last rectangle that starts at or before its first unit, then a scan
// over those that start before its last), then moves its rows with up to
// kStackRowsInFlight loads in flight per lane.  Every 64-lane access is
// contiguous on the stacked side, wherever the rectangles' edges fall in a
// 128-byte line.
#ifndef COSTA_STACK_ROWS_IN_FLIGHT
#define COSTA_STACK_ROWS_IN_FLIGHT 4
#endif
constexpr int kStackRowsInFlight = COSTA_STACK_ROWS_IN_FLIGHT;

template <typename S, bool CPLX, int MODE, bool CONJ>
__device__ __forceinline__ void move_stack(const Piece* __restrict__ pieces, int32_t pi, int32_t c,
                                           void* const* __restrict__ bufs, int32_t allow_wide, S ar, S ai, S br,
                                           S bi) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  constexpr int W = TT::WIDE_NEL;
  constexpr int YU = kStackRowsInFlight;
  static_assert(MODE != MODE_AXPBY, "stacks hold no rectangles of pairs that read A");
  const Piece& h = pieces[pi];
  const int32_t np = stack_size_of(h.flags);
  const bool on_dst = (h.flags & PIECE_STACK_DST) != 0;
  const bool wide = (h.flags & PIECE_WIDE) != 0;
  const int32_t epu = wide ? W : 1;  // elements per unit
  const Piece& last = pieces[pi + np - 1];
  const int64_t base = on_dst ? h.dst_off : h.src_off;
  const int32_t hu = (int32_t)(((on_dst ? last.dst_off : last.src_off) + last.nx - base) / epu);
  const int32_t wb = (hu + kStackWave - 1) / kStackWave;
  const int32_t nt = wb * ((h.ny + kStackRows - 1) / kStackRows);
  // this wave's task (wave-uniform)
  const int32_t t = c * (kThreads / kStackWave) + __builtin_amdgcn_readfirstlane((int32_t)threadIdx.x / kStackWave);
  if (t >= nt) return;  // past the stack's last wave task (no barrier follows)
  int32_t chunk, band;
  divmod(t, wb, chunk, band);
  const int32_t w0 = band * kStackWave;
  const int32_t xu = w0 + (int32_t)(threadIdx.x % kStackWave);
  const int64_t x = (int64_t)xu * epu;  // this lane's element offset along the stack
  const int64_t xw0 = (int64_t)w0 * epu;
  const int64_t xw1 = (int64_t)min(w0 + kStackWave, hu) * epu;
  // the last rectangle that starts at or before the wave's first unit
  int32_t lo = 0, hi = np - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    const Piece& m = pieces[pi + mid];
    if ((on_dst ? m.dst_off : m.src_off) - base <= xw0) lo = mid;
    else hi = mid - 1;
  }
  int64_t soff = 0, doff = 0, sld = 0, dld = 0;
  int32_t sbuf = 0, dbuf = 0;
  for (int32_t k = lo; k < np; ++k) {
    const Piece& p = pieces[pi + k];
    const int64_t s0 = (on_dst ? p.dst_off : p.src_off) - base;
    if (s0 >= xw1) break;
    if (x >= s0 && x < s0 + p.nx) {
      soff = p.src_off + (x - s0);
      doff = p.dst_off + (x - s0);
      sld = p.src_ld;
      dld = p.dst_ld;
      sbuf = p.src_buf;
      dbuf = p.dst_buf;
    }
  }
  if (xu >= hu) return;
  const int32_t y0 = chunk * kStackRows;
  const int32_t y1 = min(y0 + kStackRows, h.ny);
  const S* sb = reinterpret_cast<const S*>(bufs[sbuf]) + (soff + (int64_t)y0 * sld) * TT::NS;
  S* db = reinterpret_cast<S*>(bufs[dbuf]) + (doff + (int64_t)y0 * dld) * TT::NS;
  const int64_t ss = sld * TT::NS, ds = dld * TT::NS;  // row strides in scalars
  int32_t y = y0;
  if (W > 1 && wide && allow_wide) {
    using U = Vec<S, TT::NS * W>;
    for (; y + YU <= y1; y += YU) {
      U bv[YU];
#pragma unroll
      for (int k = 0; k < YU; ++k) bv[k] = load<TT::NT_WALK>(reinterpret_cast<const U*>(sb + k * ss));
#pragma unroll
      for (int k = 0; k < YU; ++k)
        store(reinterpret_cast<U*>(db + k * ds), combine<S, TT::NS * W, CPLX, MODE, CONJ>(bv[k], bv[k], ar, ai, br, bi));
      sb += YU * ss;
      db += YU * ds;
    }
    for (; y < y1; ++y) {
      const U bv = load<TT::NT_WALK>(reinterpret_cast<const U*>(sb));
      store(reinterpret_cast<U*>(db), combine<S, TT::NS * W, CPLX, MODE, CONJ>(bv, bv, ar, ai, br, bi));
      sb += ss;
      db += ds;
    }
  } else {
    // one element at a time (epu of them: a PIECE_WIDE stack in a call whose
    // buffers are not 16-byte aligned)
    const E* se = reinterpret_cast<const E*>(sb);
    E* de = reinterpret_cast<E*>(db);
    for (; y + YU <= y1; y += YU) {
      E bv[YU][W];
#pragma unroll
      for (int k = 0; k < YU; ++k)
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu) bv[k][j] = load<TT::NT_WALK>(se + k * sld + j);
#pragma unroll
      for (int k = 0; k < YU; ++k)
#pragma unroll
        for (int j = 0; j < W; ++j)
          if (j < epu)
            store(de + k * dld + j, combine<S, TT::NS, CPLX, MODE, CONJ>(bv[k][j], bv[k][j], ar, ai, br, bi));
      se += YU * sld;
      de += YU * dld;
    }
    for (; y < y1; ++y) {
#pragma unroll
      for (int j = 0; j < W; ++j)
        if (j < epu) {
          const E bv = load<TT::NT_WALK>(se + j);
          store(de + j, combine<S, TT::NS, CPLX, MODE, CONJ>(bv, bv, ar, ai, br, bi));
        }
      se += sld;
      de += dld;
    }
  }
}

// One LDS tile of a rectangle whose source runs along y while the
// destination runs along x: tile c (tiles numbered along x first) of
// tile_x x tile_y elements, cut at the rectangle's edges to w x h.  Loads
// take the tile's elements in source order (y fastest: runs of h elements),
// stores in destination order (x fastest: runs of w elements); lanes walk
// the flattened tile, so every lane has work whatever its shape.  In LDS
// element (x, y) sits at x * (tile_y | 1) + y.  When A is read (beta != 0)
// its elements are loaded together with the source, before the barrier:
// loads issued between the stores could not be moved ahead of them (the
// compiler cannot tell that they touch other elements) and would each wait
// for a full memory round trip.
template <typename S, bool CPLX, int MODE, bool CONJ>
__device__ __forceinline__ void move_tile(const Piece* __restrict__ pieces, int32_t pi, int32_t c,
                                          void* const* __restrict__ bufs, Vec<S, CPLX ? 2 : 1>* lds, S ar, S ai,
                                          S br, S bi) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  constexpr int NP = TT::TILE_PASSES;
  const Piece& p = pieces[pi];
  const int32_t tid = threadIdx.x;
  const int32_t tx = tile_x_of(p.aux), ty = tile_y_of(p.aux);
  const int32_t stride = ty | 1;
  const int32_t ntx = (p.nx + tx - 1) / tx;
  const int32_t x0 = (c % ntx) * tx, y0 = (c / ntx) * ty;
  const int32_t w = min(tx, p.nx - x0), h = min(ty, p.ny - y0);
  const int32_t n = w * h;
  const E* __restrict__ se = reinterpret_cast<const E*>(bufs[p.src_buf]) + p.src_off + (int64_t)x0 * p.src_ld + y0;
  E* __restrict__ de = reinterpret_cast<E*>(bufs[p.dst_buf]) + p.dst_off + (int64_t)y0 * p.dst_ld + x0;
  E v[NP];
  // a tile as tall as its rectangle reads source lines no other tile reads
  if (COSTA_NT_FULL_TILE_LOADS && h == p.ny) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const int32_t i = k * kThreads + tid;
      if (i < n) {
        int32_t xl, yl;
        divmod(i, h, xl, yl);
        v[k] = load<true>(se + ((int64_t)xl * p.src_ld + yl));
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const int32_t i = k * kThreads + tid;
      if (i < n) {
        int32_t xl, yl;
        divmod(i, h, xl, yl);
        v[k] = load<COSTA_NT_TILE_LOADS>(se + ((int64_t)xl * p.src_ld + yl));
      }
    }
  }
  E a[MODE == MODE_AXPBY ? NP : 1];
  if constexpr (MODE == MODE_AXPBY) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const int32_t i = k * kThreads + tid;
      if (i < n) {
        int32_t yl, xl;
        divmod(i, w, yl, xl);
        a[k] = load<COSTA_NT_TILE_ALOADS>(de + ((int64_t)yl * p.dst_ld + xl));
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int32_t i = k * kThreads + tid;
    if (i < n) {
      int32_t xl, yl;
      divmod(i, h, xl, yl);
      lds[xl * stride + yl] = v[k];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int32_t i = k * kThreads + tid;
    if (i < n) {
      int32_t yl, xl;
      divmod(i, w, yl, xl);
      store(de + ((int64_t)yl * p.dst_ld + xl),
            combine<S, TT::NS, CPLX, MODE, CONJ>(lds[xl * stride + yl], a[MODE == MODE_AXPBY ? k : 0], ar, ai, br,
                                                 bi));
    }
  }
}

// The work of one workgroup for a fixed arithmetic mode.
template <typename S, bool CPLX, int MODE, bool CONJ, bool HAS_T, int UL>
__device__ __forceinline__ void move_task(const Piece* __restrict__ pieces, int32_t pi, int32_t flags, int32_t c,
                                          void* const* __restrict__ bufs, const ItemParam* __restrict__ ip,
                                          int32_t allow_wide, Vec<S, CPLX ? 2 : 1>* lds) {
  S ar = S(0), ai = S(0), br = S(0), bi = S(0);
  if constexpr (MODE != MODE_COPY) {
    ar = (S)ip->alpha[0];
    ai = (S)ip->alpha[1];
    br = (S)ip->beta[0];
    bi = (S)ip->beta[1];
  }
  if constexpr (HAS_T) {
    if (flags & PIECE_TRANSPOSE) {
      move_tile<S, CPLX, MODE, CONJ>(pieces, pi, c, bufs, lds, ar, ai, br, bi);
      return;
    }
  } else if constexpr (MODE != MODE_AXPBY) {
    // stacks outside the pack hold only rectangles of pairs that do not read A
    if (flags & PIECE_STACK) {
      move_stack<S, CPLX, MODE, CONJ>(pieces, pi, c, bufs, allow_wide, ar, ai, br, bi);
      return;
    }
  }
  if constexpr (TypeTraits<S, CPLX>::ES >= 16)
    move_walk_lanes<S, CPLX, MODE, CONJ, UL>(pieces, pi, c, bufs, allow_wide, ar, ai, br, bi);
  else
    move_walk<S, CPLX, MODE, CONJ, UL>(pieces, pi, c * (UL * kThreads), bufs, allow_wide, ar, ai, br, bi);
}

constexpr int MODE_ANY = 3;

// One launch slice: workgroup b moves task task_off + xcd_order(b) of the
// launch's task table.
//   KIND: pack (bitwise copy into message buffers, never transposed),
//         unpack-transform, or direct.
//   MODE: the arithmetic of every pair of the call, or MODE_ANY to read it
//         per workgroup (batches that mix modes; a workgroup's rectangles
//         belong to one pair); CONJ likewise.
//   HAS_T: whether the launch contains transposed rectangles (LDS tiles).
//   UL: units per lane of its row walks; with UL = 2 the table is the
//       launch's wide task table, whose first task of a rectangle is in aux.
template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T, int UL>
__device__ __forceinline__ void mover_body(const Piece* __restrict__ pieces, const int32_t* __restrict__ tasks,
                                           int32_t task_off, void* const* __restrict__ bufs,
                                           const ItemParam* __restrict__ items, int32_t allow_wide,
                                           int32_t ranges) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  __shared__ E lds[HAS_T ? TT::LDS_ELEMS : 1];
  const int32_t b = task_off + xcd_order((int32_t)blockIdx.x, (int32_t)gridDim.x, ranges);
  const int32_t pi = tasks[b];
  const int32_t c = b - (UL == 1 ? pieces[pi].task0 : pieces[pi].aux);
  if constexpr (KIND == KIND_PACK) {
    if (pieces[pi].flags & PIECE_STACK) {
      move_stack<S, CPLX, MODE_COPY, false>(pieces, pi, c, bufs, allow_wide, S(0), S(0), S(0), S(0));
      return;
    }
    if constexpr (TT::ES >= 16)
      move_walk_lanes<S, CPLX, MODE_COPY, false, UL>(pieces, pi, c, bufs, allow_wide, S(0), S(0), S(0), S(0));
    else
      move_walk<S, CPLX, MODE_COPY, false, UL>(pieces, pi, c * (UL * kThreads), bufs, allow_wide, S(0), S(0), S(0),
                                               S(0));
  } else {
    const int32_t flags = pieces[pi].flags;
    const ItemParam* ip = items + pieces[pi].item;
    if constexpr (MODE != MODE_ANY) {
      move_task<S, CPLX, MODE, CONJ, HAS_T, UL>(pieces, pi, flags, c, bufs, ip, allow_wide, lds);
    } else {
      const bool conj = CPLX && ip->conj;
      const int32_t mode = ip->mode;
#define COSTA_TASK(M, CJ) move_task<S, CPLX, M, CJ, HAS_T, UL>(pieces, pi, flags, c, bufs, ip, allow_wide, lds)
      if (mode == MODE_COPY) {
        if (conj) COSTA_TASK(MODE_COPY, CPLX);
        else COSTA_TASK(MODE_COPY, false);
      } else if (mode == MODE_SCALE) {
        if (conj) COSTA_TASK(MODE_SCALE, CPLX);
        else COSTA_TASK(MODE_SCALE, false);
      } else {
        if (conj) COSTA_TASK(MODE_AXPBY, CPLX);
        else COSTA_TASK(MODE_AXPBY, false);
      }
#undef COSTA_TASK
    }
  }
}

// Tile sizes that leave room for at least four workgroups per CU (160 KiB of
// LDS) are compiled for at least four waves per SIMD; larger tiles (the big
// complex128 tile) for two.
template <typename S, bool CPLX, bool HAS_T>
constexpr bool big_lds() {
  return HAS_T && TypeTraits<S, CPLX>::LDS_ELEMS * TypeTraits<S, CPLX>::ES > 40 * 1024;
}

// Units per lane of a launch: two (the wide task table) in launches of row
// walks that copy -- the pack, and unpack/direct launches with alpha = 1,
// beta = 0 -- one otherwise.  Measured on MI355X: two units per lane +2 to
// +11% on copies; on an axpby walk of short misaligned rows -19%.
template <int KIND, int MODE, bool HAS_T>
constexpr int units_per_lane() {
  return !HAS_T && (KIND == KIND_PACK || MODE == MODE_COPY) ? COSTA_COPY_UNITS : 1;
}

template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8)))
costa_mover(const Piece* __restrict__ pieces, const int32_t* __restrict__ tasks, int32_t task_off,
            void* const* __restrict__ bufs, const ItemParam* __restrict__ items, int32_t allow_wide,
            int32_t ranges) {
  mover_body<S, CPLX, KIND, MODE, CONJ, HAS_T, units_per_lane<KIND, MODE, HAS_T>()>(pieces, tasks, task_off, bufs,
                                                                                   items, allow_wide, ranges);
}

template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
costa_mover_lds(const Piece* __restrict__ pieces, const int32_t* __restrict__ tasks, int32_t task_off,
                void* const* __restrict__ bufs, const ItemParam* __restrict__ items, int32_t allow_wide,
                int32_t ranges) {
  mover_body<S, CPLX, KIND, MODE, CONJ, HAS_T, 1>(pieces, tasks, task_off, bufs, items, allow_wide, ranges);
}

// Volume of the grid overlay: every overlay block (k, l) adds its element
// count to V[s][t] (s: owner of its cover in L(B), t: owner of its cover in
// L(A)).  Histogram in LDS when P*P fits, flushed with 64-bit atomics.
__global__ void __launch_bounds__(kThreads) costa_volume(VolumeArgs a, int32_t use_lds) {
  extern __shared__ unsigned long long hist[];
  const int32_t PP = a.P * a.P;
  if (use_lds) {
    for (int32_t i = threadIdx.x; i < PP; i += kThreads) hist[i] = 0ull;
    __syncthreads();
  }
  const int64_t total = (int64_t)a.K * a.L;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total; idx += stride) {
    const int32_t k = (int32_t)(idx / a.L), l = (int32_t)(idx % a.L);
    const Interval ri = a.rows[k], ci = a.cols[l];
    const int32_t t = a.ownerA[(int64_t)ri.a * a.nbcA + ci.a];
    const int32_t bi = a.transposed ? ci.b : ri.b, bj = a.transposed ? ri.b : ci.b;
    const int32_t s = a.ownerB[(int64_t)bi * a.nbcB + bj];
    const unsigned long long vol = (unsigned long long)(ri.len * ci.len);
    if (use_lds) atomicAdd(&hist[s * a.P + t], vol);
    else atomicAdd(&a.V[(int64_t)s * a.P + t], vol);
  }
  if (use_lds) {
    __syncthreads();
    for (int32_t i = threadIdx.x; i < PP; i += kThreads)
      if (hist[i]) atomicAdd(&a.V[i], hist[i]);
  }
}

struct Launch {
  hipStream_t stream;
  const Piece* pieces;
  const int32_t* tasks;  // the launch's task table
  int64_t ntasks;
  const int32_t* wide;   // its wide task table (launches of row walks)
  int64_t nwide;
  void* const* bufs;
  const ItemParam* items;
  int32_t allow_wide;
  int32_t ranges;
};

// Separable volume, step 1: histogram of overlay interval lengths by (class
// of the covering block in op(B), class of the covering block in A), for the
// rows (blockIdx.y == 0) and the columns (blockIdx.y == 1).
__global__ void __launch_bounds__(kThreads) costa_volume_hist(SeparableArgs a) {
  const bool rows = blockIdx.y == 0;
  const Interval* iv = rows ? a.rows : a.cols;
  const int32_t n = rows ? a.K : a.L;
  unsigned long long* h = rows ? a.hrow : a.hcol;
  const int32_t na = rows ? a.nra : a.nca;
  for (int32_t i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads) {
    const Interval v = iv[i];
    atomicAdd(&h[(int64_t)v.b * na + v.a], (unsigned long long)v.len);
  }
}

// Separable volume, step 2: V[s][t] = hrow[row class of s][row class of t] *
// hcol[col class of s][col class of t], 0 when s or t has no place in its
// grid (for op T the row overlay of op(B) runs over B's process columns and
// the column overlay over its rows; the host folds that into clsB).
__global__ void __launch_bounds__(kThreads) costa_volume_outer(SeparableArgs a) {
  const int32_t PP = a.P * a.P;
  for (int32_t k = blockIdx.x * kThreads + threadIdx.x; k < PP; k += gridDim.x * kThreads) {
    const int32_t s = k / a.P, t = k % a.P;
    const int32_t ra = a.clsA[2 * t], ca = a.clsA[2 * t + 1];
    const int32_t rb = a.clsB[2 * s], cb = a.clsB[2 * s + 1];
    a.V[k] = (ra < 0 || rb < 0) ? 0ull : a.hrow[(int64_t)rb * a.nra + ra] * a.hcol[(int64_t)cb * a.nca + ca];
  }
}

// One workgroup per task of the table the launch runs on, in slices that
// keep the grid below 2^32 work-items.
template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T>
hipError_t go(const Launch& l) {
  constexpr bool WIDE = units_per_lane<KIND, MODE, HAS_T>() > 1;
  const int32_t* tasks = WIDE ? l.wide : l.tasks;
  const int64_t ntasks = WIDE ? l.nwide : l.ntasks;
  if (ntasks > INT32_MAX) return hipErrorInvalidValue;
  constexpr int64_t kSlice = (int64_t)1 << 23;
  for (int64_t off = 0; off < ntasks; off += kSlice) {
    const unsigned n = (unsigned)(ntasks - off < kSlice ? ntasks - off : kSlice);
    if constexpr (big_lds<S, CPLX, HAS_T>())
      hipLaunchKernelGGL((costa_mover_lds<S, CPLX, KIND, MODE, CONJ, HAS_T>), dim3(n), dim3(kThreads), 0, l.stream,
                         l.pieces, tasks, (int32_t)off, l.bufs, l.items, l.allow_wide, l.ranges);
    else
      hipLaunchKernelGGL((costa_mover<S, CPLX, KIND, MODE, CONJ, HAS_T>), dim3(n), dim3(kThreads), 0, l.stream,
                         l.pieces, tasks, (int32_t)off, l.bufs, l.items, l.allow_wide, l.ranges);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename S, bool CPLX, int KIND, bool HAS_T>
hipError_t go_mode(const Launch& l, int mode, int conj) {
  // fixed-mode kernels for the element types of the hot workloads; the rest
  // read the mode per rectangle
  constexpr bool SPECIALISE = sizeof(S) == 8;
  if constexpr (SPECIALISE) {
    if (mode == MODE_COPY) return conj ? go<S, CPLX, KIND, MODE_COPY, CPLX, HAS_T>(l)
                                       : go<S, CPLX, KIND, MODE_COPY, false, HAS_T>(l);
    if (mode == MODE_SCALE) return conj ? go<S, CPLX, KIND, MODE_SCALE, CPLX, HAS_T>(l)
                                        : go<S, CPLX, KIND, MODE_SCALE, false, HAS_T>(l);
    if (mode == MODE_AXPBY) return conj ? go<S, CPLX, KIND, MODE_AXPBY, CPLX, HAS_T>(l)
                                        : go<S, CPLX, KIND, MODE_AXPBY, false, HAS_T>(l);
  }
  return go<S, CPLX, KIND, MODE_ANY, false, HAS_T>(l);
}

template <typename S, bool CPLX>
hipError_t launch_typed(MoverKind kind, const LaunchSpec& spec, const Launch& l) {
  if (kind == KIND_PACK) return go<S, CPLX, KIND_PACK, MODE_COPY, false, false>(l);
  if (kind == KIND_UNPACK) {
    return spec.has_transpose ? go_mode<S, CPLX, KIND_UNPACK, true>(l, spec.mode, spec.conj)
                              : go_mode<S, CPLX, KIND_UNPACK, false>(l, spec.mode, spec.conj);
  }
  return spec.has_transpose ? go_mode<S, CPLX, KIND_DIRECT, true>(l, spec.mode, spec.conj)
                            : go_mode<S, CPLX, KIND_DIRECT, false>(l, spec.mode, spec.conj);
}

}  // namespace

hipError_t launch_mover(MoverKind kind, costa_dtype dtype, const LaunchSpec& spec, const Piece* pieces,
                        const int32_t* tasks, int64_t ntasks, const int32_t* wide, int64_t nwide, void* const* bufs,
                        const ItemParam* items, int32_t allow_wide, int32_t xcd_ranges, hipStream_t stream) {
  if (ntasks <= 0) return hipSuccess;
  if (!spec.has_transpose && nwide <= 0) return hipErrorInvalidValue;  // a launch of row walks has both tables
  Launch l{stream, pieces, tasks, ntasks, wide, nwide, bufs, items, allow_wide, xcd_ranges};
  switch (dtype) {
    case COSTA_R64: return launch_typed<double, false>(kind, spec, l);
    case COSTA_C128: return launch_typed<double, true>(kind, spec, l);
    case COSTA_R32: return launch_typed<float, false>(kind, spec, l);
    case COSTA_C64: return launch_typed<float, true>(kind, spec, l);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_volume_separable(const SeparableArgs& a, hipStream_t stream) {
  const int32_t nmax = a.K > a.L ? a.K : a.L;
  if (nmax > 0) {
    unsigned gx = (unsigned)((nmax + kThreads - 1) / kThreads);
    if (gx > 1024) gx = 1024;
    hipLaunchKernelGGL(costa_volume_hist, dim3(gx, 2), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int32_t PP = a.P * a.P;
  unsigned gx = (unsigned)((PP + kThreads - 1) / kThreads);
  if (gx > 1024) gx = 1024;
  if (gx == 0) return hipSuccess;
  hipLaunchKernelGGL(costa_volume_outer, dim3(gx), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_volume(const VolumeArgs& a, hipStream_t stream) {
  const int64_t total = (int64_t)a.K * a.L;
  if (total == 0) return hipSuccess;
  int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 2048) blocks = 2048;
  const size_t lds = (size_t)a.P * a.P * sizeof(unsigned long long);
  const int32_t use_lds = lds <= 64 * 1024 ? 1 : 0;
  hipLaunchKernelGGL(costa_volume, dim3((unsigned)blocks), dim3(kThreads), use_lds ? lds : 0, stream, a, use_lds);
  return hipGetLastError();
}

}  // namespace costa
