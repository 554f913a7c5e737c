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

#include <string>
#include <vector>

#include "plan_types.hpp"

namespace moe {

struct PlanParams {
  int32_t H = 0, F = 0, E_l = 0, R = 0, self = 0;
  int32_t band_rows = 0;      // tb_M
  int32_t mid_bands = 1;      // x (mgb)
  bool local_direct = true;   // local rows need no transfer
  bool overlapped = true;     // false: plan of the non-overlapped baseline
  int32_t band_group = 8;     // tile rows that sweep the weight columns together
};

struct Plan {
  PlanParams p;
  int32_t gu_per_row = 0, down_per_row = 0;
  std::vector<TileRow> tile_rows;
  std::vector<uint32_t> items;
  std::vector<int32_t> row_x, row_rank, row_slot;
  std::vector<Segment> segs;
  std::vector<Band> bands;
  int64_t n_valid = 0, n_band_pad = 0, n_remote = 0;
  int32_t n_gu = 0, n_down = 0;
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

// Default band height: the largest power of two (16..256) whose expected owner-group
// padding stays within 2 % of max_rows.
int32_t default_band_rows(int32_t max_rows, int32_t E_l, int32_t R);

}  // namespace moe
