// HIP kernels for gfx950 (CDNA4): the rectangle mover used by the pack,
// unpack-transform and direct paths, and the grid-overlay volume kernel.
//
// All of them are bound by HBM bandwidth: per element they read at most two
// values and write one, with at most a few flops (Section 5 eq:costa).  The
// design goals are therefore coalesced 64-lane accesses, 16-byte vectors
// where the rectangle allows them, many independent loads in flight per lane,
// an LDS tile for the rectangles whose source and destination run in
// different directions, and a workgroup order that keeps neighbouring work on
// one XCD (one L2).
#include <hip/hip_runtime.h>

#include "internal.hpp"

// Products and sums are rounded one by one, never fused into an FMA, so the
// results are reproducible bit for bit.
#pragma clang fp contract(off)

namespace costa {
namespace {

// Tuning switches (compile-time; the defaults are the measured best).
#ifndef COSTA_UNROLL_WIDE
#define COSTA_UNROLL_WIDE 4  // 16-byte units in flight per lane on the row walk
#endif
#ifndef COSTA_UNROLL_WIDE_AXPBY
#define COSTA_UNROLL_WIDE_AXPBY 8  // ...when A is read too (beta != 0) in a launch without LDS tiles
#endif
#ifndef COSTA_UNROLL_NARROW16
#define COSTA_UNROLL_NARROW16 4  // 16-byte elements in flight per lane on the row walk
#endif
#ifndef COSTA_XCD_REMAP
#define COSTA_XCD_REMAP 1
#endif
#ifndef COSTA_TILE_X8
#define COSTA_TILE_X8 32
#endif
#ifndef COSTA_TILE_Y8
#define COSTA_TILE_Y8 32
#endif
#ifndef COSTA_TILE_X16
#define COSTA_TILE_X16 128  // 16-byte elements: 2 KiB store runs
#endif
#ifndef COSTA_TILE_Y16
#define COSTA_TILE_Y16 16
#endif
#ifndef COSTA_TILE_X16N
#define COSTA_TILE_X16N 64  // narrow rectangles of 16-byte elements
#endif
#ifndef COSTA_TILE_X8N
#define COSTA_TILE_X8N 16  // narrow rectangles of 8-byte elements
#endif
#ifndef COSTA_TILE_Y8N
#define COSTA_TILE_Y8N 32
#endif
#ifndef COSTA_TILE_Y16N
#define COSTA_TILE_Y16N 16
#endif
#ifndef COSTA_NT_LOADS
#define COSTA_NT_LOADS 1  // row walks: each source line is read once
#endif
#ifndef COSTA_NT_LOADS_MAX_ES
#define COSTA_NT_LOADS_MAX_ES 8  // ...for element sizes up to this (measured: helps fp64, hurts complex128)
#endif
#ifndef COSTA_NT_TILE_LOADS
#define COSTA_NT_TILE_LOADS 0  // tile loads: lines may serve two neighbouring tiles
#endif
#ifndef COSTA_NT_STORES
#define COSTA_NT_STORES 1
#endif
#ifndef COSTA_NT_ALOADS
#define COSTA_NT_ALOADS 0
#endif

constexpr int kThreads = 256;

// Workgroup b of n (dispatched round-robin over the 8 XCDs) gets the b-th
// slot of a contiguous range per XCD, so consecutive groups share an L2.
__device__ __forceinline__ int32_t xcd_remap(int32_t b, int32_t n) {
  if (!COSTA_XCD_REMAP) return b;
  constexpr int32_t X = 8;
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

// Rectangle whose source and destination both run along x:
// dst[y*dst_ld + x] = f(src[y*src_ld + x]).  Units of NU scalars (one element,
// or several when the rectangle is 16-byte aligned); lanes walk the flattened
// (y, x) index so short rows still fill a wavefront.
template <typename S, int NU, int NEL, bool CPLX, int MODE, bool CONJ, int UNROLL>
__device__ __forceinline__ void move_rows(const S* __restrict__ src, S* __restrict__ dst, const Piece& p, S ar,
                                          S ai, S br, S bi) {
  using U = Vec<S, NU>;
  const U* __restrict__ su = reinterpret_cast<const U*>(src) + p.src_off / NEL;
  U* __restrict__ du = reinterpret_cast<U*>(dst) + p.dst_off / NEL;
  const int64_t sld = p.src_ld / NEL, dld = p.dst_ld / NEL;
  const int32_t nxu = p.nx / NEL;
  const int32_t n = nxu * p.ny;
  const float inv = 1.0f / (float)nxu;
  const int32_t tid = threadIdx.x;
  for (int32_t base = 0; base < n; base += kThreads * UNROLL) {
    U bv[UNROLL], av[UNROLL];
    int64_t doff[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int32_t e = base + u * kThreads + tid;
      doff[u] = -1;
      if (e < n) {
        // y = e / nxu from a float estimate, corrected to the exact quotient
        int32_t y = (int32_t)((float)e * inv);
        int32_t x = e - y * nxu;
        while (x < 0) {
          --y;
          x += nxu;
        }
        while (x >= nxu) {
          ++y;
          x -= nxu;
        }
        bv[u] = load<COSTA_NT_LOADS && (int)sizeof(S) * (CPLX ? 2 : 1) <= COSTA_NT_LOADS_MAX_ES>(su + (y * sld + x));
        doff[u] = y * dld + x;
        if constexpr (MODE == MODE_AXPBY) av[u] = load<COSTA_NT_ALOADS>(du + doff[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      if (doff[u] >= 0) store(du + doff[u], combine<S, NU, CPLX, MODE, CONJ>(bv[u], av[u], ar, ai, br, bi));
  }
}

template <typename S, bool CPLX>
struct TypeTraits {
  static constexpr int NS = CPLX ? 2 : 1;                  // scalars per element
  static constexpr int ES = (int)sizeof(S) * NS;           // bytes per element
  static constexpr int WIDE_NEL = ES >= 16 ? 1 : 16 / ES;  // elements per 16-byte unit
  static constexpr int UNROLL_NARROW = ES >= 16 ? COSTA_UNROLL_NARROW16 : 8;
  // transpose tile: TX elements along the destination's contiguous direction
  // (store lanes), TY along the source's (load lanes).  Long store runs pay
  // off for 16-byte elements; 8-byte elements keep 32 x 32 (occupancy, and
  // the narrow transposed rectangles of block-cyclic layouts)
  static constexpr int TX = ES >= 16 ? COSTA_TILE_X16 : ES == 8 ? COSTA_TILE_X8 : 64;
  static constexpr int TY = ES >= 16 ? COSTA_TILE_Y16 : ES == 8 ? COSTA_TILE_Y8 : 64;
  // rectangles marked PIECE_NARROW_T: a narrower tile keeps the store lanes
  // busy
  static constexpr int TXN = ES >= 16 ? COSTA_TILE_X16N : ES == 8 ? COSTA_TILE_X8N : TX;
  static constexpr int TYN = ES >= 16 ? COSTA_TILE_Y16N : ES == 8 ? COSTA_TILE_Y8N : TY;
  static constexpr int LDS_ELEMS = TX * (TY + 1) > TXN * (TYN + 1) ? TX * (TY + 1) : TXN * (TYN + 1);
};

// Rectangles whose source runs along y while the destination runs along x:
// staged through an LDS tile of TX x TY elements (one padding column against
// bank conflicts).  Loads are coalesced along the source, stores along the
// destination.  The workgroup walks the tiles of the consecutive transposed
// rectangles [pi, p1) as one sequence, software pipelined across rectangle
// boundaries: the loads of the next tile (of this rectangle or of the next
// one) are in flight while the current tile is written out.  Returns the
// index of the first rectangle it did not process (the run stops at a
// rectangle that is not transposed or takes the other tile shape).  MODE_ANY
// callers pass p1 = pi + 1.
template <typename S, bool CPLX, int MODE, bool CONJ, int TX, int TY>
__device__ __forceinline__ int32_t move_transposed_run(const Piece* __restrict__ pieces, int32_t pi, int32_t p1,
                                                       void* const* __restrict__ bufs,
                                                       const ItemParam* __restrict__ items,
                                                       Vec<S, CPLX ? 2 : 1>* lds) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  E (*tile)[TY + 1] = reinterpret_cast<E (*)[TY + 1]>(lds);
  constexpr int LROWS = kThreads / TY;  // x rows per load pass
  constexpr int SROWS = kThreads / TX;  // y rows per store pass
  constexpr int NL = TX / LROWS;        // loads per thread per tile
  static_assert(kThreads % TX == 0 && kThreads % TY == 0 && TX % LROWS == 0 && TY % SROWS == 0,
                "the load and store passes must cover the tile exactly");
  const int32_t tid = threadIdx.x;
  const int32_t ly0 = tid % TY, lx0 = tid / TY;  // load mapping
  const int32_t sx0 = tid % TX, sy0 = tid / TX;  // store mapping
  auto tiles_x = [](const Piece& p) { return (p.nx + TX - 1) / TX; };
  auto tiles_of = [&](const Piece& p) { return tiles_x(p) * ((p.ny + TY - 1) / TY); };
  auto fetch = [&](const Piece& p, int32_t t, E (&b)[NL]) {
    const E* __restrict__ se = reinterpret_cast<const E*>(bufs[p.src_buf]) + p.src_off;
    const int32_t ntx = tiles_x(p);
    const int32_t tx = (t % ntx) * TX, ty = (t / ntx) * TY;
    const int32_t y = ty + ly0;
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int32_t x = tx + lx0 + k * LROWS;
      if (x < p.nx && y < p.ny) b[k] = load<COSTA_NT_TILE_LOADS>(se + ((int64_t)x * p.src_ld + y));
    }
  };
  Piece cur = pieces[pi];
  int32_t ntiles = tiles_of(cur);
  E b[NL];
  fetch(cur, 0, b);
  int32_t t = 0;
  while (true) {
    const int32_t ntx = tiles_x(cur);
    const int32_t tx = (t % ntx) * TX, ty = (t / ntx) * TY;
    // registers -> LDS
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int32_t lx = lx0 + k * LROWS;
      if (tx + lx < cur.nx && ty + ly0 < cur.ny) tile[lx][ly0] = b[k];
    }
    __syncthreads();
    // the next tile: of this rectangle, else the first of the next one if it
    // is transposed too; its loads go out before this tile is stored
    Piece nxt = cur;
    int32_t nt = t + 1;
    bool more = nt < ntiles;
    if (!more && pi + 1 < p1) {
      nxt = pieces[pi + 1];
      constexpr int32_t kClass = PIECE_TRANSPOSE | PIECE_NARROW_T;  // same tile shape
      more = (nxt.flags & kClass) == (cur.flags & kClass);
      nt = 0;
    }
    if (more) fetch(nxt, nt, b);
    // LDS -> destination
    E* __restrict__ de = reinterpret_cast<E*>(bufs[cur.dst_buf]) + cur.dst_off;
    S ar = S(0), ai = S(0), br = S(0), bi = S(0);
    if constexpr (MODE != MODE_COPY) {
      const ItemParam& ip = items[cur.item];
      ar = (S)ip.alpha[0];
      ai = (S)ip.alpha[1];
      br = (S)ip.beta[0];
      bi = (S)ip.beta[1];
    }
    const int32_t x = tx + sx0;
#pragma unroll
    for (int k = 0; k < TY / SROWS; ++k) {
      const int32_t ly = sy0 + k * SROWS;
      const int32_t yy = ty + ly;
      if (x < cur.nx && yy < cur.ny) {
        E* o = de + ((int64_t)yy * cur.dst_ld + x);
        E a;
        if constexpr (MODE == MODE_AXPBY) a = load<COSTA_NT_ALOADS>(o);
        store(o, combine<S, TT::NS, CPLX, MODE, CONJ>(tile[sx0][ly], a, ar, ai, br, bi));
      }
    }
    __syncthreads();
    if (!more) return pi + 1;
    if (nt == 0) {
      ++pi;
      cur = nxt;
      ntiles = tiles_of(cur);
    }
    t = nt;
  }
}

// A rectangle whose source and destination run the same way.  A launch that
// also holds transposed rectangles (HAS_T) keeps the shallower unroll: the
// register budget of its tile path sets the launch's occupancy.
template <typename S, bool CPLX, int MODE, bool CONJ, bool HAS_T>
__device__ __forceinline__ void move_piece(const S* src, S* dst, const Piece& p, bool wide, S ar, S ai, S br, S bi) {
  using TT = TypeTraits<S, CPLX>;
  if (wide && TT::WIDE_NEL > 1) {
    constexpr int U = MODE == MODE_AXPBY && !HAS_T ? COSTA_UNROLL_WIDE_AXPBY : COSTA_UNROLL_WIDE;
    move_rows<S, TT::NS * TT::WIDE_NEL, TT::WIDE_NEL, CPLX, MODE, CONJ, U>(src, dst, p, ar, ai, br, bi);
  } else {
    move_rows<S, TT::NS, 1, CPLX, MODE, CONJ, TT::UNROLL_NARROW>(src, dst, p, ar, ai, br, bi);
  }
}

constexpr int MODE_ANY = 3;

// One launch over groups of rectangles.
//   KIND: pack (bitwise copy into message buffers, never transposed),
//         unpack-transform, or direct.
//   MODE: the arithmetic of every pair of the call, or MODE_ANY to read it
//         per rectangle (batches that mix modes); CONJ likewise.
//   HAS_T: whether the launch contains transposed rectangles (LDS tile).
template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8)))
costa_mover(const Piece* __restrict__ pieces, const int32_t* __restrict__ groups, int32_t ngroups,
            void* const* __restrict__ bufs, const ItemParam* __restrict__ items, int32_t allow_wide) {
  using TT = TypeTraits<S, CPLX>;
  using E = Vec<S, TT::NS>;
  __shared__ E lds[HAS_T ? TT::LDS_ELEMS : 1];
  const int32_t g = xcd_remap((int32_t)blockIdx.x, ngroups);
  const int32_t p0 = groups[g], p1 = groups[g + 1];
  int32_t pi = p0;
  Piece ahead = pieces[p0];  // the next rectangle's descriptor, fetched while the current one moves
  int32_t ahead_i = p0;
  while (pi < p1) {
    const Piece p = ahead_i == pi ? ahead : pieces[pi];
    if (pi + 1 < p1) {
      ahead = pieces[pi + 1];
      ahead_i = pi + 1;
    }
    if constexpr (KIND == KIND_PACK) {
      const bool wide = allow_wide && (p.flags & PIECE_WIDE);
      move_piece<S, CPLX, MODE_COPY, false, false>(reinterpret_cast<const S*>(bufs[p.src_buf]),
                                            reinterpret_cast<S*>(bufs[p.dst_buf]), p, wide, S(0), S(0), S(0), S(0));
      ++pi;
      continue;
    } else {
      const ItemParam& ip = items[p.item];
      if constexpr (HAS_T) {
        if (p.flags & PIECE_TRANSPOSE) {
          if constexpr (MODE != MODE_ANY) {
            if (TT::TXN != TT::TX && (p.flags & PIECE_NARROW_T))
              pi = move_transposed_run<S, CPLX, MODE, CONJ, TT::TXN, TT::TYN>(pieces, pi, p1, bufs, items, lds);
            else
              pi = move_transposed_run<S, CPLX, MODE, CONJ, TT::TX, TT::TY>(pieces, pi, p1, bufs, items, lds);
          } else {
            // mixed batches: one rectangle at a time, the big tile
            const bool conj = CPLX && ip.conj;
            constexpr int X = TT::TX, Y = TT::TY;
            if (ip.mode == MODE_COPY)
              pi = conj ? move_transposed_run<S, CPLX, MODE_COPY, true, X, Y>(pieces, pi, pi + 1, bufs, items, lds)
                        : move_transposed_run<S, CPLX, MODE_COPY, false, X, Y>(pieces, pi, pi + 1, bufs, items, lds);
            else if (ip.mode == MODE_SCALE)
              pi = conj ? move_transposed_run<S, CPLX, MODE_SCALE, true, X, Y>(pieces, pi, pi + 1, bufs, items, lds)
                        : move_transposed_run<S, CPLX, MODE_SCALE, false, X, Y>(pieces, pi, pi + 1, bufs, items, lds);
            else
              pi = conj ? move_transposed_run<S, CPLX, MODE_AXPBY, true, X, Y>(pieces, pi, pi + 1, bufs, items, lds)
                        : move_transposed_run<S, CPLX, MODE_AXPBY, false, X, Y>(pieces, pi, pi + 1, bufs, items, lds);
          }
          continue;
        }
      }
      const S* src = reinterpret_cast<const S*>(bufs[p.src_buf]);
      S* dst = reinterpret_cast<S*>(bufs[p.dst_buf]);
      const bool wide = allow_wide && (p.flags & PIECE_WIDE);
      const S ar = (S)ip.alpha[0], ai = (S)ip.alpha[1], br = (S)ip.beta[0], bi = (S)ip.beta[1];
      if constexpr (MODE != MODE_ANY) {
        move_piece<S, CPLX, MODE, CONJ, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
      } else {
        const bool conj = CPLX && ip.conj;
        switch (ip.mode) {
          case MODE_COPY:
            if (conj) move_piece<S, CPLX, MODE_COPY, true, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            else move_piece<S, CPLX, MODE_COPY, false, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            break;
          case MODE_SCALE:
            if (conj) move_piece<S, CPLX, MODE_SCALE, true, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            else move_piece<S, CPLX, MODE_SCALE, false, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            break;
          default:
            if (conj) move_piece<S, CPLX, MODE_AXPBY, true, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            else move_piece<S, CPLX, MODE_AXPBY, false, HAS_T>(src, dst, p, wide, ar, ai, br, bi);
            break;
        }
      }
      ++pi;
    }
  }
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
  dim3 grid, block;
  hipStream_t stream;
  const Piece* pieces;
  const int32_t* groups;
  int32_t ngroups;
  void* const* bufs;
  const ItemParam* items;
  int32_t allow_wide;
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
// hcol[col class of s][col class of t] (for op T the row overlay of op(B)
// runs over B's process columns and the column overlay over its rows).
__global__ void __launch_bounds__(kThreads) costa_volume_outer(SeparableArgs a) {
  const int32_t PP = a.P * a.P;
  for (int32_t k = blockIdx.x * kThreads + threadIdx.x; k < PP; k += gridDim.x * kThreads) {
    const int32_t s = k / a.P, t = k % a.P;
    const int32_t prA = a.rowmajA ? t / a.pcolA : t % a.prowA;
    const int32_t pcA = a.rowmajA ? t % a.pcolA : t / a.prowA;
    const int32_t prB = a.rowmajB ? s / a.pcolB : s % a.prowB;
    const int32_t pcB = a.rowmajB ? s % a.pcolB : s / a.prowB;
    const int32_t rb = a.transposed ? pcB : prB;  // class of s in the row overlay
    const int32_t cb = a.transposed ? prB : pcB;  // class of s in the column overlay
    a.V[k] = a.hrow[(int64_t)rb * a.nra + prA] * a.hcol[(int64_t)cb * a.nca + pcA];
  }
}

template <typename S, bool CPLX, int KIND, int MODE, bool CONJ, bool HAS_T>
hipError_t go(const Launch& l) {
  hipLaunchKernelGGL((costa_mover<S, CPLX, KIND, MODE, CONJ, HAS_T>), l.grid, l.block, 0, l.stream, l.pieces,
                     l.groups, l.ngroups, l.bufs, l.items, l.allow_wide);
  return hipGetLastError();
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
                        const int32_t* groups, int64_t ngroups, void* const* bufs, const ItemParam* items,
                        int32_t allow_wide, hipStream_t stream) {
  if (ngroups <= 0) return hipSuccess;
  if (ngroups > INT32_MAX) return hipErrorInvalidValue;
  Launch l{dim3((unsigned)ngroups), dim3(kThreads), stream, pieces, groups, (int32_t)ngroups, bufs, items,
           allow_wide};
  switch (dtype) {
    case COSTA_R64: return launch_typed<double, false>(kind, spec, l);
    case COSTA_C128: return launch_typed<double, true>(kind, spec, l);
    case COSTA_R32: return launch_typed<float, false>(kind, spec, l);
    case COSTA_C64: return launch_typed<float, true>(kind, spec, l);
  }
  return hipErrorInvalidValue;
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
