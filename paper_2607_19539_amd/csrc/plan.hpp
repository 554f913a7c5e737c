// plan.hpp -- host construction of the static plan of one expert stage run.
//
// Builds, from the routing of one run (paper Section 3.2, Algorithm 1):
//   * the remote-owner-aligned row layout (Section 3.2.1),
//   * the remote-first tile schedule (Section 3.2.2),
//   * the combine plan: transfer segments with destination, offset and rows
//     (Sections 3.2.3 and 3.3.2).
// Pure C++; no HIP dependency, so it is testable without a GPU.
#pragma once
#include <stdint.h>

#include <array>
#include <string>
#include <vector>

#include "plan_types.hpp"

namespace moe {

struct PlanParams {
  int32_t H = 0, F = 0, E_l = 0, R = 0, self = 0;
  int32_t band_rows = 1;      // tb_M: remote owner groups start at multiples of it
  int32_t mid_pieces = 1;     // x (mgb): tile-row pieces per middle segment
  bool local_direct = true;   // local rows need no transfer
  bool overlapped = true;     // false: plan of the non-overlapped baseline
  int32_t gu_group = 4;       // tile rows an XCD sweeps its gate/up columns for together
  int32_t down_group = 4;     // tile rows an XCD sweeps its down (part, column) slice for together
  int32_t split_k = 0;        // K parts of every down tile (1..kMaxSplitK); 0 = split the tail
};

struct Plan {
  PlanParams p;
  int32_t gu_per_row = 0, down_per_row = 0;
  std::vector<TileRow> tile_rows;
  std::vector<uint32_t> items;
  std::vector<int32_t> row_x, row_rank, row_slot;
  std::vector<Segment> segs;
  std::vector<Group> groups;
  int64_t n_valid = 0, n_band_pad = 0, n_remote = 0;
  int32_t n_gu = 0, n_down = 0;
  int32_t tail_split = 1;     // K parts of the split tile rows (split_k when uniform)
  int32_t n_split_rows = 0;   // tile rows whose down tiles are split
  int32_t n_partials = 0;     // fp32 partial tiles the run uses
  // Per-XCD work queues of each launch: queue x holds items [q[x], q[x+1]) of that launch
  // (offsets from the launch's first item).
  std::array<int32_t, kXcds + 1> gu_queue{}, down_queue{};
  int64_t n_lrows() const { return (int64_t)row_x.size(); }
};

// Checks the routing of one run.  Returns 0, -1 (invalid argument) or -2 (bad routing)
// and describes the problem in *err.
int validate_routing(const PlanParams& p, int64_t rows, const int32_t* expert_offsets,
                     const int32_t* row_src_rank, const int32_t* row_slot,
                     const int64_t* return_rows, std::string* err);

// Builds the plan (validation included).  Same return codes as validate_routing.
int build_plan(const PlanParams& p, int64_t rows, const int32_t* expert_offsets,
               const int32_t* row_src_rank, const int32_t* row_slot, const int64_t* return_rows,
               Plan* out, std::string* err);

// Upper bound of logical rows of the padded layout for `max_rows` routed rows.
int64_t max_logical_rows(int64_t max_rows, int32_t E_l, int32_t R, int32_t band_rows);


// fp32 partial tiles a run may need: uniform splitting keeps one per part of every down tile;
// the default tail split keeps at most one round's worth (kRoundTiles).  nk = ffn / 64.
int64_t max_partial_tiles(int32_t split_k, int64_t max_tile_rows, int32_t down_per_row, int32_t nk);

}  // namespace moe
