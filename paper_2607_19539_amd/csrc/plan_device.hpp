// plan_device.hpp -- launch interface of the device-side plan builder.
//
// Builds on the GPU, from routing that is already in device memory, the same plan the host
// builder makes (paper Section 3.2, Algorithm 1: the remote-owner-aligned layout, the
// remote-first tile schedule and the combine plan), in stream order and without a host round
// trip.  Its routing precondition is the order a dispatch all-to-all delivers rows in: within
// each expert, the rows of one source rank are contiguous and their slots ascend.  Routing
// that breaks it, or any rule the host validation enforces, leaves an empty plan and the error
// code in PlanHeader::status.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan_types.hpp"

namespace moe {

// Device scratch of the planner, carved from one allocation sized for the handle's capacity.
struct DevPlanWs {
  // Filled with all-ones bits by the init kernel, in one range: run bounds and the hash set.
  int32_t* run_lo;        // [E_l * R] first dispatched row of source rank r in expert e, or -1
  int32_t* run_hi;        // [E_l * R] one past its last row
  uint64_t* seen;         // [seen_cap] open-addressing set of (rank, slot) keys; ~0 = empty
  int64_t seen_cap;       // power of two, >= 2 * max_rows
  int64_t fill_words;     // 32-bit words from run_lo through the end of `seen`
  // Written by the planner before they are read.
  int32_t* ex_ntr;        // [E_l] tile rows of each expert; then their first tile row
  int32_t* ex_ng;         // [E_l] owner groups of each expert; then their first group
  int32_t* ex_hr;         // [E_l] tile rows holding remote rows
  int32_t* ex_bands;      // [E_l] remote bands (the schedule's expert key)
  int32_t* ex_roff;       // [E_l] schedule position of the expert's first remote tile row
  int32_t* ex_loff;       // [E_l] schedule position of its first local-only tile row
  int32_t* tmp;           // [E_l] scan scratch
  int32_t* g_lrow0;       // [E_l * R] internal group table (every plan kind)
  int32_t* g_rows;
  int32_t* g_dst;
  int32_t* g_src0;        // first dispatched row of the group
  int32_t* order;         // [max_tile_rows] schedule position -> tile row
  int32_t* ga_gu;         // [max_tile_rows] row group [ga, gb) of each schedule position,
  int32_t* gb_gu;         //   gate/up launch
  int32_t* ga_dn;         //   down launch
  int32_t* gb_dn;
  int32_t* pos_of_down;   // [max_tile_rows * down_per_row] latest queue position of a tile's parts
  int32_t* start_q;       // [max_tile_rows][256] per tile row: logical rows where segments start,
  int32_t* start_np;      //   the tile-row pieces each one's chunk covers,
  int32_t* end_q;         //   and one past the rows where segments end
  int32_t* cnt_s;         // [max_tile_rows] segment starts per tile row (then their prefix sums)
  int32_t* cnt_e;         // [max_tile_rows] segment ends per tile row (then their prefix sums)
  Segment* seg_tmp;       // [max_lrows] segments in layout order
  int32_t* seg_key;       // [max_lrows] ready position of each
  int32_t* hist;          // [max_items + 1] ready-position counts, then offsets
};

struct DevPlanArgs {
  const int32_t* off;     // [E_l + 1] expert offsets (device)
  const int32_t* src;     // [rows] source rank of each dispatched row (device)
  const int32_t* slot;    // [rows] receive slot of each dispatched row (device)
  const int64_t* return_rows;  // [R] receive-buffer rows (device copy)
  int32_t E_l, R, self, tb, mid_pieces, gu_group, down_group, split_k;
  int32_t gu_per_row, down_per_row, nk;
  int32_t overlapped, local_direct;
  int32_t no_lds;         // keep every table in device memory (testing the large-size path)
  int32_t max_rows, max_tile_rows;
  PlanHeader* hdr;
  TileRow* tile_rows;
  uint32_t* items;
  int32_t* queues;        // [2][kXcds + 1] absolute item indices of each launch's queues
  int32_t* row_x;
  int32_t* row_rank;
  int32_t* row_slot;
  Segment* segs;
  Group* groups;
  int32_t* tail_rows;     // [kMaxTailRows] split tile rows of the default tail split, schedule order
  DevPlanWs ws;
};

// Bytes of planner scratch for a handle of this capacity; carve() lays it out from `base`.
size_t devplan_ws_bytes(int32_t E_l, int32_t R, int32_t max_rows, int32_t max_tile_rows,
                        int32_t down_per_row, int64_t max_lrows, int64_t max_items);
DevPlanWs devplan_ws_carve(void* base, int32_t E_l, int32_t R, int32_t max_rows, int32_t max_tile_rows,
                           int32_t down_per_row, int64_t max_lrows, int64_t max_items);

// Enqueues the planner kernels on `s`.  The init kernel must already have filled the
// all-ones range of the scratch and reset the header (status 0, bad_row INT32_MAX).
hipError_t launch_devplan(const DevPlanArgs& a, int64_t max_items, int num_cus, hipStream_t s);

}  // namespace moe
