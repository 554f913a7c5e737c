// kernels.hpp -- launch interface of the gfx950 kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan_types.hpp"

namespace moe {

// Producer mode bits.
constexpr uint32_t kModeSignal = 1u;       // raise a ready flag per down tile of a transfer tile row
constexpr uint32_t kModeLocalDirect = 2u;  // local rows go straight to the local receive buffer
constexpr uint32_t kModeDirectAll = 4u;    // every row goes straight to its receive buffer
constexpr uint32_t kModeDeferTail = 8u;    // split tail tiles: parts only store their partials; the
                                           // tail kernel after the launch adds them and writes the tiles

// Timestamped runs: one record per producer workgroup of each launch (where it ran, how many
// items it took, when it started and ended; 100 MHz wall clock) and one per consumer copy unit.
struct WgRecord {
  uint32_t hw_id;   // HW_ID register of wave 0 (wave, SIMD, CU, shader array and engine ids)
  uint32_t xcc_id;  // XCD the workgroup ran on
  int32_t launch;   // 0 gate/up, 1 down
  int32_t items;    // work items it ran
  uint64_t t_start, t_end;
  uint64_t cycles;  // shader clock cycles of wave 0 between t_start and t_end
};
struct CopyRecord {
  int32_t segment;  // segment index (ready order)
  int32_t part;     // copy unit within the segment
  uint32_t hw_id;   // HW_ID register of the copying wave
  uint32_t xcc_id;
  uint64_t t_poll;  // the wave starts polling the segment's flags
  uint64_t t_ready; // every flag seen, acquire done: the copy starts
  uint64_t t_done;  // the wave's copy stores have completed
  int32_t source;   // 0 the consumer launch, 1 the drain launch
  int32_t reserved;
};
static_assert(sizeof(WgRecord) == 40 && sizeof(CopyRecord) == 48, "record layouts are part of the ABI");

struct ProducerArgs {
  const uint16_t* x;       // [rows, H] dispatched tokens
  const uint16_t* w1;      // [E_l, F, H]
  const uint16_t* w3;      // [E_l, F, H]
  const uint16_t* w2;      // [E_l, H, F]
  uint16_t* hws;           // [F / 64][hws_rows][64] gated activation (workspace, K-blocked)
  int64_t hws_rows;        // rows per K block of the workspace (the handle's row capacity)
  uint16_t* y;             // [n_lrows, H] staged output (workspace)
  const TileRow* tile_rows;
  const uint32_t* items;   // every work item of the run (gate/up tiles, then down items)
  const int32_t* queue;    // [kXcds + 1] of this launch: XCD x's queue is items
                           // [queue[x], queue[x+1]); queue[kXcds] ends the launch's items
  uint32_t* claim;         // [kXcds] queue heads of this launch
  uint32_t* active;        // count of workgroups that claimed work in this launch
  const int32_t* row_x;    // [n_lrows]
  const int32_t* row_rank; // [n_lrows], -1 = padding
  const int32_t* row_slot; // [n_lrows]
  uint16_t* const* ret;    // [R] receive buffers (device array of device pointers)
  uint32_t* flags;         // [n_tile_rows * down_per_row] ready flags (value = epoch)
  uint32_t epoch;
  int32_t H, F, self_rank, down_per_row;
  uint32_t mode;
  int32_t split_k;         // K parts of every down tile; 0 = per tile row (TileRow::split)
  float* partials;         // fp32 part tiles (256 threads x 256) from TileRow::part_base on
  uint32_t* arrivals;      // [tiles] parts finished this run (zeroed by the init kernel)
  WgRecord* wg_rec;        // timestamped runs: [grid] records of this launch, else null
  RunCounters* ctr;        // timestamped runs: the producer span (prod_t0 / prod_t1)
  uint64_t* tile_ready;    // timestamped runs: [tiles] when each down tile's flag was raised
  RunCounters* go_ctr;     // gate/up launch of an overlapped run: publishes go = epoch as it starts
  uint32_t* wcount;        // MOE_WRITE_COUNTS: [logical rows] 8-byte words stored into receive buffers
};

// The tail kernel: finishes the split down tiles after the down launch.  Reads the plan's tile
// rows and its partials; writes the tiles' rows exactly as the down epilogue would and raises
// their flags.
struct TailArgs {
  ProducerArgs p;              // the down launch's arguments (mode, outputs, flags, partials)
  const int32_t* tail_rows;    // device: the split tile rows, in schedule order
  const int32_t* n_split_rows; // device: how many
};

struct ConsumerArgs {
  const uint16_t* y;
  uint16_t* const* ret;
  const Segment* segs;
  const int32_t* n_segs;   // device: segments of the plan
  const int32_t* down_qmax; // device: longest down queue, in items
  const uint32_t* flags;
  uint32_t epoch;
  int32_t H;
  // Copy units per segment, as powers of two: segments ready before the down launch's last two
  // rounds take 2^early_shift units, later ones 2^late_shift.
  int32_t early_shift, late_shift;
  RunCounters* ctr;
  uint64_t watchdog_ticks;
  CopyRecord* rec;         // timestamped runs: one record per copy unit below rec_cap, else null
  uint32_t rec_cap;
  uint32_t* simd_waves;    // beside the producer: [kXcds * kSimdKeys] consumer waves per SIMD
  int64_t plain_n16;       // plain-copy measurement: 16-byte vectors to copy into ret[0]
  // Ticket dealing: tickets below 4 x map_grid go transposed to the waves of the consumer launch
  // of map_grid workgroups (0: this launch's grid), so the drain deals them like the consumer.
  uint32_t map_grid;
  int32_t role;            // kRoleConsumer, kRoleCounted or kRoleDrain
  uint32_t exit_waves;     // drain: consumer waves whose exit it waits for
  uint32_t wait_go;        // 1: wait until ctr->go holds this run's epoch before anything else
  uint32_t map_wpg;        // waves per workgroup of the launch map_grid describes (0: this launch's)
  uint32_t max_waves_cu;   // beside the producer: consumer waves a compute unit keeps (0: no limit)
  uint32_t* abandoned;     // [abandoned_cap] copy units whose flag wait expired, for the drain
  uint32_t abandoned_cap;
  uint32_t* wcount;        // MOE_WRITE_COUNTS: [logical rows] 8-byte words stored into receive buffers
};
// Consumer launch roles.  A counted consumer's waves each add one to ctr->cons_exit once their
// stores are written back; a drain launch (after the producer, in its stream) claims the copy
// units still unclaimed, then waits until every consumer wave has counted its exit, so the end
// of the drain is the end of every copy of the run.
constexpr int32_t kRoleConsumer = 0;
constexpr int32_t kRoleCounted = 1;
constexpr int32_t kRoleDrain = 2;

struct ScatterArgs {
  const uint16_t* y;
  uint16_t* const* ret;
  const int32_t* row_rank;
  const int32_t* row_slot;
  const int64_t* n_lrows;  // device: logical rows of the plan
  int32_t H;
  uint32_t* wcount;        // MOE_WRITE_COUNTS: [logical rows] 8-byte words stored into receive buffers
};

struct InitArgs {
  RunCounters* ctr;
  uint16_t* poison;        // optional: filled with bf16 NaN
  int64_t poison_elems;    // multiple of 8
  uint32_t* arrivals;      // split-K arrival counters to zero
  int32_t n_arrivals;
  uint32_t* wcount;        // optional: write counts to zero
  int64_t n_wcount;
  uint64_t* tile_ready;    // optional: per-tile flag times to zero (as many as arrivals)
  uint32_t* simd_waves;    // optional: consumer per-SIMD wave counts to zero
  uint32_t* publish;       // optional: ready flags to set to `epoch` (consumer-only measurement)
  int32_t n_publish;
  uint32_t epoch;
  uint32_t* fill_ones;     // optional: words to set to all-ones bits (device planner scratch)
  int64_t n_fill_ones;
  PlanHeader* plan_hdr;    // optional: header the device planner fills; reset to no error
};


struct CombineArgs {
  const uint16_t* recv;    // [recv_rows, H] receive buffer of this source rank
  const int32_t* slot;     // [tokens, k] receive slot of each choice
  const float* gate;       // [tokens, k] gate weights
  uint16_t* out;           // [tokens, H]
  uint32_t* bad_slots;     // optional: incremented once per out-of-range slot
  int64_t recv_rows, tokens;
  int32_t k, H;
};

hipError_t launch_init(const InitArgs& a, hipStream_t s);
// Gate-weighted sum of each token's k returned rows (16-byte vectors, fp32 sum, bf16 out).
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
// Gate/up tiles (down = false) or down-projection tiles with ready flags (down = true).
hipError_t launch_producer(const ProducerArgs& a, bool down, int grid, hipStream_t s);
// own_cus: the consumer has its compute units to itself (a reserved partition, or no producer).
hipError_t launch_consumer(const ConsumerArgs& a, bool own_cus, int grid, int threads, hipStream_t s);
// After the producer, in its stream: the copy units the consumer has not claimed yet, on the
// producer's compute units, and the wait for the consumer's last wave.
hipError_t launch_drain(const ConsumerArgs& a, int grid, hipStream_t s);
// One thread stores `epoch` into ctr->go (agent scope): the run's reset is complete (for runs
// without a gate/up launch, which otherwise publishes it).
hipError_t launch_go(RunCounters* ctr, uint32_t epoch, hipStream_t s);
// Measurement aid: a flat grid-stride copy of plain_n16 vectors from the staged output into the
// first receive buffer (no flags, no copy units).
hipError_t launch_plain_copy(const ConsumerArgs& a, int grid, hipStream_t s);
// Split tail tiles of a kModeDeferTail down launch: one accumulator block of one tile per pass.
hipError_t launch_tail(const TailArgs& a, int grid, hipStream_t s);
hipError_t launch_scatter(const ScatterArgs& a, int grid, hipStream_t s);
// One 100 MHz real-time counter reading into *dst (host-visible memory) in stream order.
hipError_t launch_stamp(uint64_t* dst, hipStream_t s);
// Resident producer workgroups per compute unit.
int producer_blocks_per_cu();
constexpr int kProducerThreads = 256;
constexpr int kConsumerThreads = 256;
// 16-byte vectors per consumer lane and copy chunk (two chunks in flight): beside the producer,
// within 56 VGPRs (two such waves and a producer wave of 136 VGPRs + 256 AGPRs fill a SIMD's
// 512 registers); on compute units of its own, within 128.
constexpr int kCopyUnroll = 3;
constexpr int kCopyUnrollOwn = 10;
// Consumer copy units (one wave each) per segment, as a power of two.  Beside the producer
// (shared compute units) a copying wave slows the producer workgroup on its compute unit, so
// segments take few units (kCopyPartsShift) until the last two rounds of the down queues
// (kLatePositions positions: two rounds of an XCD's 32 compute units), after which little
// producer work is left and the last segments take up to kCopyPartsLateShift units each.  On
// compute units of its own the consumer cuts every segment into units of about 64 KiB (at
// most kCopyPartsOwnShift), so its waves copy in parallel whatever the segment count.
constexpr int kCopyPartsShift = 2;
constexpr int kCopyPartsLateShift = 4;
constexpr int kCopyPartsOwnShift = 6;
constexpr int kLatePositions = 64;
// Copy records a timestamped handle keeps per run (units past it are not recorded).
constexpr uint32_t kMaxCopyRecords = 1u << 18;
// Consumer flag polls sleep kPollSleep x 64 cycles, doubling the count of sleeps per poll up to
// kPollBackoffMax (about 2.5 us between polls at the loaded clock).
constexpr int kPollSleep = 4;
constexpr uint32_t kPollBackoffMax = 16;
constexpr int kTailGrid = 1024; // tail kernel workgroups (one pass each on the usual tail)
// Consumer waves per SIMD the register budget must allow: at most 512 / 8 = 64 VGPRs each (the
// copy chunk keeps the kernel at 56, so two waves fit beside a producer wave of 392 registers).
constexpr int kConsumerMinWaves = 8;
// Consumer waves beside the producer in all (their copy rate is latency-bound per wave; about 256
// waves saturate it), spread over however many compute units the split gives the consumer.
constexpr int kConsumerWavesShared = 256;
// Consumer waves a SIMD keeps beside the producer (the register budget above), counted per SIMD
// key (shader engine, shader array, compute unit, SIMD) of each XCD.
constexpr int kMaxConsumerWavesPerSimd = 2;
constexpr int kSimdKeys = 1024;
constexpr int kCuKeys = kSimdKeys / 4;
// Consumer wave counters beside the producer: per SIMD key, then per compute-unit key, per XCD.
constexpr int kWaveCounters = kXcds * (kSimdKeys + kCuKeys);
// On compute units of its own: up to 128 VGPRs, four waves per SIMD (four workgroups per CU).
constexpr int kConsumerOwnMinWaves = 4;
constexpr int kConsumerOwnPerCu = 4;
// Entries of the abandoned-unit list: a consumer wave abandons at most one unit (then exits), and a
// launch has at most 16 waves on each of 256 compute units.
constexpr uint32_t kMaxAbandoned = 4096;

}  // namespace moe
