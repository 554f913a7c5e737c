// plan_types.hpp -- plain structs shared by the host plan builder and the gfx950 kernels.
//
// The plan is a set of flat tables the host builds per run and uploads once
// (paper Section 3.2.3: routing is resolved up front into per-tile device
// arrays so no kernel inspects individual rows' owners at transfer time).
#pragma once
#include <stdint.h>

namespace moe {

// GEMM tiling of the producer.  A tile row is kTileM consecutive rows of one
// expert's padded layout; a gate/up tile covers kGuTileF ffn features (and
// computes both the gate and the up projection for them); a down tile covers
// kDownTileN hidden columns.  K advances kTileK elements per step.
constexpr int kTileM = 256;
constexpr int kGuTileF = 128;
constexpr int kDownTileN = 256;
constexpr int kTileK = 64;

// Work-item encoding: bit 31 = down tile, bits 30..12 = tile row.  A gate/up item keeps its
// column tile in bits 11..0.  A down item keeps its column tile in bits 11..4 and, in bits
// 3..0, which of the tile's split_k parts it is: part p accumulates the K steps
// [p*nk/split_k, (p+1)*nk/split_k) of the nk = F/kTileK steps, and the part that finishes
// last adds all parts in part order and writes the tile.
constexpr uint32_t kItemDown = 0x80000000u;
constexpr int kItemRowShift = 12;
constexpr uint32_t kItemColMask = 0xFFFu;
constexpr int kDownColShift = 4;
constexpr uint32_t kDownColMask = 0xFFu;
constexpr uint32_t kDownPartMask = 0xFu;
constexpr int32_t kMaxTileRows = 1 << 19;
constexpr int32_t kMaxColTiles = 1 << 12;
constexpr int32_t kMaxDownColTiles = 1 << 8;
constexpr int32_t kMaxSplitK = 16;
// Down tiles the producer runs at once on MI355X (one workgroup per compute unit).  The
// default split (see build_plan) fills the last, partly occupied round of that many tiles.
constexpr int32_t kRoundTiles = 256;
// Split tile rows the default tail split can produce: each has at least two parts of its
// down_per_row tiles within one round.
constexpr int32_t kMaxTailRows = kRoundTiles / 2;

struct TileRow {
  int32_t expert;      // local expert index
  int32_t lrow0;       // first logical row (multiple of kTileM)
  int32_t nvalid;      // routed (non-padding) rows in this tile row
  int32_t has_remote;  // 1 if any row returns to another rank
  int32_t split;       // K parts of each of its down tiles (1 = whole tiles)
  int32_t part_base;   // first fp32 partial tile of its parts (split > 1), else -1
};

struct Segment {
  int32_t dst_rank;    // receive buffer the rows go to
  int32_t rows;        // rows in the segment (all valid, slot-contiguous)
  int32_t y_row0;      // first logical row in the staged output
  int32_t slot0;       // slot of the first row in the receive buffer
  int32_t flag_begin;  // first ready flag the segment waits for
  int32_t flag_count;  // consecutive flags it waits for
  int32_t ready_pos;   // schedule position of the last down item it needs
  int32_t npieces;     // tile-row pieces of its group it covers (1 for first/last segments)
};

// One owner group: the rows of one local expert that came from one source rank, contiguous
// in the padded layout.
struct Group {
  int32_t expert;
  int32_t lrow0;       // first logical row
  int32_t rows;
  int32_t dst_rank;    // the source rank the rows return to
};

// MI355X has 8 XCDs (accelerator dies), each with its own L2; the workgroups of a launch are
// dealt to them round-robin.  Each producer launch keeps one work queue per XCD.
constexpr int kXcds = 8;
// Items per chunk when a launch's item sequence is dealt round-robin to the XCD queues.
constexpr int kQueueChunk = 32;

// Counts of a plan in device memory, written by whichever side built it (the host uploads
// it with the tables; the device planner writes it itself).  The kernels take their item,
// segment and row counts from here, so a plan built on the device needs no host round trip.
struct PlanHeader {
  int32_t status;        // 0, or the MOE_E* code the device planner found (then the plan is empty)
  int32_t bad_row;       // first routing row that failed validation (INT32_MAX if none)
  int32_t n_tile_rows;
  int32_t n_groups;      // owner groups reported (overlapped plans only)
  int32_t n_gu;          // gate/up items
  int32_t n_down;        // down items
  int32_t n_segs;        // transfer segments
  int32_t tail_split;    // K parts of each split down tile
  int32_t n_split_rows;
  int32_t n_partials;
  int32_t down_qmax;     // longest down queue (items)
  int32_t n_groups_all;  // device planner: owner groups of the layout, any plan kind
  int32_t reserved[2];
  int64_t n_valid, n_lrows, n_band_pad, n_remote;
};

// Device-side counters of one run; the queue heads are zeroed by the init kernel.
struct RunCounters {
  uint32_t gu_next[kXcds];    // gate/up work queue heads, one per XCD
  uint32_t down_next[kXcds];  // down-projection work queue heads
  uint32_t seg_next;          // consumer copy-unit queue head
  // Watchdog reports, NOT reset per run (a query reads and clears them, so they are sticky):
  uint32_t timeouts;          // bounded waits that expired
  uint32_t timeout_where;     // bit 0 = consumer flag wait
  uint32_t timeout_seg;       // lowest segment (ready order) whose wait expired; UINT32_MAX if none
  uint32_t gu_active;         // gate/up workgroups that claimed at least one tile
  uint32_t down_active;       // down workgroups that claimed at least one tile
  uint32_t n_units;           // consumer copy units of the run (written by the consumer)
  uint32_t cons_exit;         // consumer waves done (runs that end with a drain launch)
  uint32_t go;                // epoch of the last run whose reset is complete (set after the
                              // init kernel by a kernel of its own; the init kernel leaves it)
  uint64_t units_pub;         // (copy units << 32) | early units, published by the consumer
  uint64_t poll_iters;        // consumer poll iterations
  uint64_t wait_ticks;        // consumer wait time, 100 MHz ticks
  // Timestamped runs only (100 MHz wall clock): first gate/up workgroup start and last
  // producer (down or tail) workgroup end.
  uint64_t prod_t0, prod_t1;
  uint32_t n_abandoned;       // copy units whose flag wait expired (the drain copies them)
  uint32_t pad_;
};

}  // namespace moe
