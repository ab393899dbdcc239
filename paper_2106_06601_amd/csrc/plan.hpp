// Host plan of a (batched) transform: the work rectangles of each kernel.
#pragma once

#include <functional>

#include "internal.hpp"

namespace costa {

const Layout* layout_of(costa_layout h);

struct ItemDesc {
  const Layout* A;
  const Layout* B;
  costa_op op;
  bool reads_a;  // beta != 0: the pair's unpack and direct rectangles read A
};

struct PlanConfig {
  int elem_size;           // bytes per element
  int64_t workspace_cap;   // max message bytes per wave (>= 1)
  int64_t max_piece_elems; // split rectangles larger than this (keeps per-rectangle indices in 32 bits)
};

struct HostPlan {
  std::vector<Piece> pieces;    // every launch's rectangles, concatenated
  std::vector<int32_t> tasks;   // every launch's workgroups: index of the rectangle each starts with
  std::vector<int32_t> wide_tasks;  // the wide task tables of the launches without tiles
  std::vector<LaunchRange> direct;  // empty when the direct rectangles join the last unpack
  std::vector<Wave> waves;
  int64_t workspace_bytes = 0;  // max message bytes of a wave
  // per pair: elements on each path
  std::vector<int64_t> item_total, item_local, item_remote;
  std::vector<char> item_reads_a;
  int64_t overlay_blocks = 0;
  int32_t pieces_pack = 0, pieces_unpack = 0, pieces_direct = 0;
  double plan_ms = 0.0;
};

// Builds the plan.  sigma: P entries or empty (identity).  Buffer table of a
// call with n pairs: [A of pair k, rank r] at k*P + r, [B of pair k, rank s]
// at n*P + k*P + s, the message workspace at 2*n*P.
// choose_cap(total message bytes) returns the workspace cap for the waves
// (cfg.workspace_cap is ignored when choose_cap is given).
void build_plan(const std::vector<ItemDesc>& items, const std::vector<int32_t>& sigma, const PlanConfig& cfg,
                const std::function<int64_t(int64_t)>& choose_cap, HostPlan& out);

}  // namespace costa
