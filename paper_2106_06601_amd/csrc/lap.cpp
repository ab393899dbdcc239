// Communication-optimal process relabeling (Section 4): with the locally-free
// volume cost the gain of moving label x to rank y is V(S_yx) - V(S_xx) (gain
// remark), so the optimal relabeling maximises sum_t V[sigma[t]][t] -- a
// linear assignment problem (Theorems 1 and 2), solved here exactly with the
// Hungarian (Kuhn-Munkres) method in O(P^3).
//
// Several relabelings may be optimal.  The library returns the
// lexicographically smallest array sigma among them: by complementary
// slackness every optimal assignment uses only edges that are tight for the
// optimal dual potentials the Hungarian method ends with, and every perfect
// matching of tight edges is optimal; so labels are fixed in increasing order
// to the smallest rank that still leaves a perfect matching of tight edges,
// checked with one augmenting-path search per candidate.
#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

#include "internal.hpp"

namespace costa {

using i128 = __int128;

namespace {

// Minimum-cost assignment on a dense n x n cost matrix, 1-based potentials u
// (rows) and v (cols) with u[i] + v[j] <= c[i][j], tight on the returned
// assignment.  colrow[j] = row assigned to column j.  T: __int128 for exact
// integer costs, long double for real ones.
template <typename T>
void hungarian(int n, const std::vector<T>& c, T INF, std::vector<T>& u, std::vector<T>& v,
               std::vector<int>& colrow) {
  u.assign(n + 1, 0);
  v.assign(n + 1, 0);
  std::vector<int> p(n + 1, 0), way(n + 1, 0);  // p[j]: row matched to column j (0 = none)
  for (int i = 1; i <= n; ++i) {
    p[0] = i;
    int j0 = 0;
    std::vector<T> minv(n + 1, INF);
    std::vector<char> used(n + 1, 0);
    do {
      used[j0] = 1;
      int i0 = p[j0], j1 = 0;
      T delta = INF;
      for (int j = 1; j <= n; ++j)
        if (!used[j]) {
          T cur = c[(size_t)(i0 - 1) * n + (j - 1)] - u[i0] - v[j];
          if (cur < minv[j]) {
            minv[j] = cur;
            way[j] = j0;
          }
          if (minv[j] < delta) {
            delta = minv[j];
            j1 = j;
          }
        }
      for (int j = 0; j <= n; ++j) {
        if (used[j]) {
          u[p[j]] += delta;
          v[j] -= delta;
        } else {
          minv[j] -= delta;
        }
      }
      j0 = j1;
    } while (p[j0] != 0);
    do {
      int j1 = way[j0];
      p[j0] = p[j1];
      j0 = j1;
    } while (j0);
  }
  colrow.assign(n, -1);
  for (int j = 1; j <= n; ++j) colrow[j - 1] = p[j] - 1;
}

struct Matcher {
  int n;
  const std::vector<char>& tight;     // tight[s*n + t]
  std::vector<int>& rank_of;          // label t -> rank s
  std::vector<int>& label_of;         // rank s -> label t
  const std::vector<char>& fixed_rank;
  const std::vector<char>& fixed_label;
  std::vector<char> seen;

  // Try to find a new partner rank for label t among unfixed ranks, moving
  // other unfixed labels along an alternating path; `banned` is excluded.
  bool augment(int t, int banned) {
    for (int s = 0; s < n; ++s) {
      if (s == banned || fixed_rank[s] || seen[s] || !tight[(size_t)s * n + t]) continue;
      seen[s] = 1;
      int t2 = label_of[s];
      if (t2 < 0 || (!fixed_label[t2] && augment(t2, banned))) {
        rank_of[t] = s;
        label_of[s] = t;
        return true;
      }
    }
    return false;
  }
};

}  // namespace

void solve_relabel(int32_t P, const int64_t* V, int32_t* sigma) {
  const int n = P;
  if (n == 0) return;
  int64_t vmax = 0;
  for (int64_t k = 0; k < (int64_t)n * n; ++k) vmax = std::max(vmax, V[k]);
  // cost[s][t] = vmax - V[s][t] >= 0: minimum cost = maximum retained volume
  std::vector<i128> cost((size_t)n * n);
  for (int s = 0; s < n; ++s)
    for (int t = 0; t < n; ++t) cost[(size_t)s * n + t] = (i128)vmax - V[(size_t)s * n + t];
  std::vector<i128> u, v;
  std::vector<int> colrow;
  hungarian<i128>(n, cost, ((i128)1) << 120, u, v, colrow);  // rows = ranks, cols = labels

  std::vector<char> tight((size_t)n * n);
  for (int s = 0; s < n; ++s)
    for (int t = 0; t < n; ++t) tight[(size_t)s * n + t] = (u[s + 1] + v[t + 1] == cost[(size_t)s * n + t]);

  std::vector<int> rank_of(colrow), label_of(n, -1);
  for (int t = 0; t < n; ++t) label_of[rank_of[t]] = t;
  std::vector<char> fixed_rank(n, 0), fixed_label(n, 0);
  Matcher m{n, tight, rank_of, label_of, fixed_rank, fixed_label, {}};

  for (int t = 0; t < n; ++t) {
    for (int s = 0; s < n; ++s) {
      if (fixed_rank[s] || !tight[(size_t)s * n + t]) continue;
      if (rank_of[t] == s) break;  // already matched to the smallest feasible candidate so far
      // try to match (s, t): free s's current label, re-match it elsewhere
      std::vector<int> save_r(rank_of), save_l(label_of);
      int t_old = label_of[s];  // unfixed label currently using s (t_old > t)
      int s_old = rank_of[t];
      label_of[s_old] = -1;
      rank_of[t] = s;
      label_of[s] = t;
      fixed_label[t] = 1;  // t is being fixed; keep it out of the search
      m.seen.assign(n, 0);
      bool ok = m.augment(t_old, s);
      fixed_label[t] = 0;
      if (ok) break;
      rank_of = save_r;
      label_of = save_l;
    }
    fixed_label[t] = 1;
    fixed_rank[rank_of[t]] = 1;
  }
  for (int t = 0; t < n; ++t) sigma[t] = rank_of[t];
}

namespace {

// The paper's greedy matching (Section 6): edges by decreasing weight, ties
// by smaller row then smaller column; an edge is taken while both ends are
// free.  weight[x*n + y]; returns rowcol[x] = y.  The weights (gains) can be
// negative: when the completed perfect matching has a total weight below
// zero, the identity (weight 0, always a perfect matching of the complete
// graph G_delta, Theorem 2) is returned instead, since a 2-approximation of a
// maximum that is >= 0 cannot be negative.
template <typename T>
void greedy_matching(int n, const std::vector<T>& weight, std::vector<int>& rowcol) {
  std::vector<int64_t> order((size_t)n * n);
  for (size_t k = 0; k < order.size(); ++k) order[k] = (int64_t)k;
  std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) { return weight[a] > weight[b]; });
  std::vector<char> row_used(n, 0), col_used(n, 0);
  rowcol.assign(n, -1);
  int taken = 0;
  for (int64_t k : order) {
    int x = (int)(k / n), y = (int)(k % n);
    if (row_used[x] || col_used[y]) continue;
    row_used[x] = col_used[y] = 1;
    rowcol[x] = y;
    if (++taken == n) break;
  }
  T total = 0;
  for (int x = 0; x < n; ++x) total += weight[(size_t)x * n + rowcol[x]];
  if (total < 0)
    for (int x = 0; x < n; ++x) rowcol[x] = x;
}

}  // namespace
}  // namespace costa

extern "C" costa_status costa_relabel_cost(int32_t P, const int64_t* V, double elem_bytes, const double* latency,
                                           const double* inv_bandwidth, costa_relabel_method method, int32_t* sigma,
                                           double* cost_before, double* cost_after) {
  return costa::guarded([&]() -> costa_status {
    using namespace costa;
    if (P < 0) return fail(COSTA_ERROR_INVALID_VALUE, "P must be >= 0");
    if (P > 0 && (!V || !sigma)) return fail(COSTA_ERROR_INVALID_VALUE, "null argument");
    if ((latency == nullptr) != (inv_bandwidth == nullptr))
      return fail(COSTA_ERROR_INVALID_VALUE, "latency and inv_bandwidth must both be given or both be NULL");
    if (method != COSTA_RELABEL_EXACT && method != COSTA_RELABEL_GREEDY)
      return fail(COSTA_ERROR_INVALID_VALUE, "unknown relabeling method");
    if (!(elem_bytes > 0) || !std::isfinite(elem_bytes)) return fail(COSTA_ERROR_INVALID_VALUE, "elem_bytes must be > 0");
    const bool general = latency != nullptr;
    if (P > (general ? 1024 : 4096)) return fail(COSTA_ERROR_NOT_SUPPORTED, "P too large for the relabeling");
    const size_t PP = (size_t)P * P;
    for (size_t k = 0; k < PP; ++k) {
      if (V[k] < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative volume");
      if (general && (!std::isfinite(latency[k]) || !std::isfinite(inv_bandwidth[k]) || latency[k] < 0 ||
                      inv_bandwidth[k] < 0))
        return fail(COSTA_ERROR_INVALID_VALUE, "latency and inv_bandwidth entries must be finite and >= 0");
    }
    // w(p_i, p_j, S_ij) of a non-empty package of `vol` elements
    auto w = [&](int i, int j, int64_t vol) -> long double {
      if (vol == 0) return 0.0L;
      const long double bytes = (long double)vol * elem_bytes;
      if (!general) return i == j ? 0.0L : bytes;
      return (long double)latency[(size_t)i * P + j] + (long double)inv_bandwidth[(size_t)i * P + j] * bytes;
    };
    auto total = [&](const int32_t* sg) {
      long double W = 0;
      for (int i = 0; i < P; ++i)
        for (int j = 0; j < P; ++j) {
          const int64_t vol = V[(size_t)i * P + j];
          if (vol) W += w(i, sg ? sg[j] : j, vol);
        }
      return W;
    };
    if (P > 0) {
      if (!general && method == COSTA_RELABEL_EXACT) {
        solve_relabel(P, V, sigma);  // integer path, canonical tie-break
      } else if (!general) {
        // gain remark: delta(p_x, p_y) = V(S_yx) - V(S_xx), exact in integers
        std::vector<int64_t> gain(PP);
        for (int x = 0; x < P; ++x)
          for (int y = 0; y < P; ++y) gain[(size_t)x * P + y] = V[(size_t)y * P + x] - V[(size_t)x * P + x];
        std::vector<int> rowcol;
        greedy_matching(P, gain, rowcol);
        for (int x = 0; x < P; ++x) sigma[x] = rowcol[x];
      } else {
        // eq:delta: sum over the left neighbours p_i of p_x (S_ix non-empty)
        std::vector<long double> gain(PP, 0.0L);
        for (int x = 0; x < P; ++x)
          for (int y = 0; y < P; ++y) {
            long double d = 0;
            for (int i = 0; i < P; ++i) {
              const int64_t vol = V[(size_t)i * P + x];
              if (vol) d += w(i, x, vol) - w(i, y, vol);
            }
            gain[(size_t)x * P + y] = d;
          }
        if (method == COSTA_RELABEL_GREEDY) {
          std::vector<int> rowcol;
          greedy_matching(P, gain, rowcol);
          for (int x = 0; x < P; ++x) sigma[x] = rowcol[x];
        } else {
          std::vector<long double> cost(PP);
          for (size_t k = 0; k < PP; ++k) cost[k] = -gain[k];
          std::vector<long double> u, v;
          std::vector<int> colrow;
          hungarian<long double>(P, cost, std::numeric_limits<long double>::infinity(), u, v, colrow);  // rows = labels
          for (int y = 0; y < P; ++y) sigma[colrow[y]] = y;
        }
      }
    }
    if (cost_before) *cost_before = (double)total(nullptr);
    if (cost_after) *cost_after = (double)total(sigma);
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_relabel(int32_t P, const int64_t* V_host, int32_t* sigma, int64_t* retained_identity,
                                      int64_t* retained_sigma) {
  return costa::guarded([&]() -> costa_status {
    using namespace costa;
    if (P < 0) return fail(COSTA_ERROR_INVALID_VALUE, "P must be >= 0");
    if (P > 0 && (!V_host || !sigma)) return fail(COSTA_ERROR_INVALID_VALUE, "null argument");
    if (P > 4096) return fail(COSTA_ERROR_NOT_SUPPORTED, "relabeling is limited to P <= 4096");
    for (int64_t k = 0; k < (int64_t)P * P; ++k)
      if (V_host[k] < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative volume");
    solve_relabel(P, V_host, sigma);
    if (retained_identity) {
      int64_t r = 0;
      for (int t = 0; t < P; ++t) r += V_host[(size_t)t * P + t];
      *retained_identity = r;
    }
    if (retained_sigma) {
      int64_t r = 0;
      for (int t = 0; t < P; ++t) r += V_host[(size_t)sigma[t] * P + t];
      *retained_sigma = r;
    }
    return COSTA_SUCCESS;
  });
}
