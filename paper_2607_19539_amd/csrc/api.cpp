// api.cpp -- the C ABI of include/moe_stage.h: handle, validation, plan upload,
// CU-masked stream pair and the fork/join of producer and consumer.
//
// Co-scheduling (paper Section 3.3.3): the consumer and the producer are two
// persistent kernels on two streams whose compute-unit masks are disjoint, so
// each keeps a stable CU budget; they coordinate only through device memory.
// The consumer is enqueued first so its workgroups are resident before the
// producer fills the remaining compute units.  Stream priorities are left at
// the default: with disjoint CU masks there is nothing left for a priority to
// arbitrate.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>
#include <stddef.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/moe_stage.h"
#include "kernels.hpp"
#include "plan.hpp"
#include "plan_device.hpp"

using namespace moe;

static_assert(sizeof(WgRecord) == sizeof(moe_wg_record_t) && offsetof(WgRecord, t_start) == offsetof(moe_wg_record_t, t_start) &&
                  offsetof(WgRecord, cycles) == offsetof(moe_wg_record_t, cycles),
              "producer record layout");
static_assert(sizeof(CopyRecord) == sizeof(moe_copy_record_t) && offsetof(CopyRecord, t_poll) == offsetof(moe_copy_record_t, t_poll),
              "copy record layout");

namespace {

thread_local std::string g_create_error;

constexpr int kTimingRing = 512;

// Adaptive CU split (cu_split = 0): the consumer sizes tried, the completed runs measured for
// each, and the event pairs kept in flight for the measurements.
// With shared CUs the consumer's waves are best spread thinly over many compute units (each
// slows the producer workgroup beside it); a reserved partition takes its CUs from the producer,
// so it stays small.
constexpr int kAutoSplitsShared[] = {32, 64, 128, 248};
constexpr int kAutoSplitsPartitioned[] = {8, 16, 32, 64};
constexpr int kNumAutoSplits = sizeof(kAutoSplitsShared) / sizeof(kAutoSplitsShared[0]);
static_assert(sizeof(kAutoSplitsPartitioned) == sizeof(kAutoSplitsShared), "one candidate count");
constexpr int kAutoSamples = 3;
constexpr int kAutoRing = 8;

struct AutoSplit {
  int cand = 0;     // candidate being measured
  int chosen = -1;  // index of the split in use once every candidate is measured
  std::vector<float> ms[kNumAutoSplits];
  // Per measured run: GPU wall-clock stamps at its start and after its join (pinned host
  // memory, written by a one-thread kernel) and an event without timing that marks them done.
  uint64_t* stamps = nullptr;  // [kAutoRing][2]
  hipEvent_t done[kAutoRing] = {};
  int ev_cand[kAutoRing] = {};
  bool busy[kAutoRing] = {};
  int next = 0;
};

struct TimingRec {
  hipEvent_t ev[8];  // 0 stage start, 1 producer start, 2 producer end, 3 consumer start,
                     // 4 consumer end / scatter start, 5 stage end / scatter end, 6 gate/up end,
                     // 7 plan ready (upload or device planner, and the counter reset, done)
  int kind = -1;     // 0 overlapped, 1 serial
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Byte layout of the device plan blob.  The host builder packs it to the plan's own sizes;
// the device builder writes into the layout of the handle's capacity.
struct BlobLayout {
  size_t hdr, tile_rows, items, queues, row_x, row_rank, row_slot, segs, groups, tail, ret, total;
};

BlobLayout blob_layout(int64_t n_tr, int64_t n_items, int64_t n_lrows, int64_t n_segs, int64_t n_groups,
                       int32_t R) {
  BlobLayout b{};
  size_t o = 0;
  b.hdr = o;       o = align256(o + sizeof(PlanHeader));
  b.tile_rows = o; o = align256(o + sizeof(TileRow) * (size_t)n_tr);
  b.items = o;     o = align256(o + sizeof(uint32_t) * (size_t)n_items);
  b.queues = o;    o = align256(o + sizeof(int32_t) * 2 * (kXcds + 1));
  b.row_x = o;     o = align256(o + sizeof(int32_t) * (size_t)n_lrows);
  b.row_rank = o;  o = align256(o + sizeof(int32_t) * (size_t)n_lrows);
  b.row_slot = o;  o = align256(o + sizeof(int32_t) * (size_t)n_lrows);
  b.segs = o;      o = align256(o + sizeof(Segment) * (size_t)n_segs);
  b.groups = o;    o = align256(o + sizeof(Group) * (size_t)n_groups);
  b.tail = o;      o = align256(o + sizeof(int32_t) * (size_t)kMaxTailRows);  // split tile rows (default split)
  b.ret = o;       o = align256(o + (sizeof(void*) + sizeof(int64_t)) * (size_t)R);  // pointers, then rows
  b.total = o;
  return b;
}

}  // namespace

struct moe_stage_s {
  moe_stage_config_t cfg{};
  int device = 0;
  int num_cus = 0;
  int n_xcd = 1;
  int producer_bpc = 1;
  int64_t max_lrows = 0;
  int32_t max_tile_rows = 0;
  int32_t down_per_row = 0;

  uint16_t* hws = nullptr;
  uint16_t* y = nullptr;
  uint32_t* flags = nullptr;
  float* partials = nullptr;
  uint32_t* arrivals = nullptr;
  uint32_t* abandoned = nullptr;   // [kMaxAbandoned] copy units a consumer wave gave up on
  uint32_t* wcount = nullptr;      // MOE_WRITE_COUNTS: [max logical rows] words stored per row
  RunCounters* ctr = nullptr;
  WgRecord* wg_rec = nullptr;      // MOE_TIMESTAMPS: [2][num_cus * producer_bpc] per launch
  CopyRecord* copy_rec = nullptr;  // MOE_TIMESTAMPS: [kMaxCopyRecords]
  uint64_t* tile_ready = nullptr;  // MOE_TIMESTAMPS: [max_tile_rows * down_per_row] flag times
  uint32_t* simd_waves = nullptr;  // consumer waves per SIMD and per CU beside the producer [kWaveCounters]
  int32_t last_tiles = 0;          // down tiles of the last run (tile rows x down_per_row)
  uint8_t* d_plan = nullptr;
  size_t plan_cap = 0;
  BlobLayout cap_lay{};   // the blob at the handle's capacity (device-built plans)
  BlobLayout last_lay{};  // the blob of the last run
  void* dev_ws = nullptr; // device planner scratch
  int64_t max_items = 0;
  DevPlanWs ws{};
  bool last_dev = false;         // the last run's plan was built on the device
  bool last_overlapped = false;
  bool dev_hdr_pending = false;  // its header has not been read back yet
  int32_t dev_status = 0, dev_bad_row = 0;
  uint8_t* h_stage[2] = {nullptr, nullptr};
  hipEvent_t stage_free[2] = {nullptr, nullptr};
  int stage_idx = 0;
  uint32_t epoch = 0;

  // CU-masked queues of the consumer split in use (and, while the adaptive selector measures,
  // of each candidate, so a switch costs no queue teardown); s_cons / s_prod are the current
  // split's pair.  Partitioned runs give each split a producer queue on the complementary
  // mask; with shared CUs one every-CU producer queue serves every split, made only when a
  // run needs it (a caller on the legacy null stream).  Every hardware queue a process keeps
  // costs: past a few dozen the scheduler time-slices them and every kernel slows down, and even
  // a few idle ones slow the stage, so a handle keeps only the current split's pair.
  struct SplitQueues {
    int c;
    hipStream_t cons, prod;  // prod: partitioned runs only
  };
  std::vector<SplitQueues> queues;
  hipStream_t shared_prod = nullptr;
  int cached_split = -1;
  hipStream_t s_cons = nullptr, s_prod = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join_c = nullptr, ev_join_p = nullptr, ev_done = nullptr;
  bool ran = false;
  bool counters_pending = false;  // the last run's device counters have not been read yet
  uint64_t last_span[2] = {0, 0};  // producer span of the last timestamped run
  uint32_t last_timeouts = 0, last_timeout_where = 0;

  std::vector<TimingRec> ring;
  int ring_next = 0, ring_count = 0;
  AutoSplit autos;

  Plan plan;
  std::string err;
  moe_stage_stats_t last{};
};

namespace {

int set_err(moe_stage_s* h, int code, const std::string& msg) {
  if (h)
    h->err = msg;
  else
    g_create_error = msg;
  return code;
}

#define HIP_TRY(h, call)                                                                   \
  do {                                                                                     \
    hipError_t e__ = (call);                                                               \
    if (e__ != hipSuccess)                                                                 \
      return set_err((h), MOE_EHIP, std::string(#call) + ": " + hipGetErrorString(e__));   \
  } while (0)

PlanParams params_of(const moe_stage_config_t& c, bool overlapped) {
  PlanParams p;
  p.H = c.hidden;
  p.F = c.ffn;
  p.E_l = c.num_local_experts;
  p.R = c.num_ranks;
  p.self = c.self_rank;
  p.band_rows = c.band_rows;
  p.mid_pieces = std::max(c.mid_segment_pieces, 1);
  p.local_direct = (c.flags & MOE_LOCAL_DIRECT) != 0;
  p.overlapped = overlapped;
  p.split_k = c.down_split_k;
  return p;
}

int check_config(const moe_stage_config_t* c) {
  if (!c) return MOE_EINVAL;
  if (c->hidden <= 0 || c->ffn <= 0 || c->num_local_experts <= 0 || c->num_ranks <= 0 ||
      c->self_rank < 0 || c->self_rank >= c->num_ranks || c->max_rows < 0 ||
      c->mid_segment_pieces < 0 || c->watchdog_ms < 0)
    return MOE_EINVAL;
  constexpr uint32_t kKnownFlags = MOE_LOCAL_DIRECT | MOE_KERNEL_TIMING | MOE_POISON |
                                   MOE_TEST_NO_SIGNAL | MOE_SHARED_CUS | MOE_DIRECT_ALL |
                                   MOE_TEST_CONSUMER_ONLY | MOE_TEST_PLAN_NO_LDS | MOE_TIMESTAMPS |
                                   MOE_TEST_PLAIN_COPY | MOE_WRITE_COUNTS;
  if (c->flags & ~kKnownFlags) return MOE_EINVAL;
  if (c->band_rows < 0 || c->band_rows > 256 || (c->band_rows & (c->band_rows - 1)) != 0)
    return MOE_EINVAL;
  if (c->down_split_k < 0 || c->down_split_k > kMaxSplitK ||
      (c->ffn > 0 && c->down_split_k > c->ffn / kTileK))
    return MOE_EINVAL;
  if (c->hidden % 64 != 0 || c->ffn % 64 != 0 || c->hidden > kMaxDownColTiles * kDownTileN ||
      c->max_rows >= (1 << 24))
    return MOE_EUNSUPPORTED;
  // The kernels address within one operand with 32-bit lane offsets: the gathered token rows of
  // dispatched_x (row x 2*hidden bytes) and the K blocks of the activation workspace (its
  // logical rows x 128 bytes).
  if ((int64_t)c->max_rows * c->hidden * 2 > (int64_t)UINT32_MAX) return MOE_EUNSUPPORTED;
  const int64_t tile_rows =
      (max_logical_rows(c->max_rows, c->num_local_experts, c->num_ranks, std::max(c->band_rows, 1)) + kTileM - 1) /
          kTileM + c->num_local_experts;
  if (tile_rows > kMaxTileRows || tile_rows * kTileM * kTileK * 2 > (int64_t)UINT32_MAX) return MOE_EUNSUPPORTED;
  return MOE_OK;
}

uint64_t watchdog_ticks(const moe_stage_s* h) {
  const int ms = h->cfg.watchdog_ms > 0 ? h->cfg.watchdog_ms : 2000;
  return (uint64_t)ms * 100000ull;  // wall clock runs at 100 MHz
}

// Resets the run counters on `stream` (and, before a device-built plan, the planner's scratch
// and header), and advances the flag epoch.
int enqueue_init(moe_stage_s* h, bool overlapped, bool dev, int32_t n_tile_rows, int64_t n_lrows,
                 hipStream_t stream) {
  const moe_stage_config_t& c = h->cfg;
  InitArgs ia{};
  ia.ctr = h->ctr;
  ia.arrivals = h->arrivals;
  ia.n_arrivals = n_tile_rows * h->down_per_row;
  ia.tile_ready = h->tile_ready;
  h->last_tiles = ia.n_arrivals;
  ia.wcount = h->wcount;
  ia.n_wcount = h->wcount ? h->max_lrows : 0;
  if (overlapped && (c.flags & MOE_SHARED_CUS)) ia.simd_waves = h->simd_waves;
  if (c.flags & MOE_POISON) {
    ia.poison = h->y;
    ia.poison_elems = n_lrows * c.hidden;
  }
  const uint32_t epoch = h->epoch + 1 == 0 ? 1 : h->epoch + 1;  // flags hold the epoch of the run that set them
  if (overlapped && (c.flags & MOE_TEST_CONSUMER_ONLY)) {
    ia.publish = h->flags;
    ia.n_publish = ia.n_arrivals;
    ia.epoch = epoch;
  }
  if (dev) {
    ia.fill_ones = (uint32_t*)h->ws.run_lo;
    ia.n_fill_ones = h->ws.fill_words;
    ia.plan_hdr = (PlanHeader*)(h->d_plan + h->cap_lay.hdr);
  }
  HIP_TRY(h, launch_init(ia, stream));
  h->epoch = epoch;
  return MOE_OK;
}

// Host arguments both planners check before anything is enqueued.
int check_run_args(moe_stage_s* h, const void* const* ret, const int64_t* return_rows) {
  if (!return_rows || !ret) return set_err(h, MOE_EINVAL, "null receive-buffer array");
  for (int r = 0; r < h->cfg.num_ranks; ++r) {
    if (return_rows[r] < 0) return set_err(h, MOE_EINVAL, "return_rows[" + std::to_string(r) + "] < 0");
    if (!ret[r] && return_rows[r] > 0) return set_err(h, MOE_EINVAL, "null return buffer");
  }
  return MOE_OK;
}

// Validates and builds the plan on the host, uploads it and resets the run counters, all on
// `stream`.
int prepare(moe_stage_s* h, bool overlapped, const void* x,
            const int32_t* off, const int32_t* src, const int32_t* slot, const void* w1,
            const void* w3, const void* w2, void* const* ret, const int64_t* return_rows,
            hipStream_t stream, BlobLayout* lay) {
  const auto t0 = std::chrono::steady_clock::now();
  const moe_stage_config_t& c = h->cfg;
  if (!off) return set_err(h, MOE_EINVAL, "null routing array");
  int rc = check_run_args(h, ret, return_rows);
  if (rc) return rc;
  const int64_t rows = off[c.num_local_experts];
  if (rows < 0) return set_err(h, MOE_EROUTING, "expert_offsets[E_l] < 0");
  if (rows > c.max_rows)
    return set_err(h, MOE_ECAPACITY, "rows " + std::to_string(rows) + " > max_rows " +
                                         std::to_string(c.max_rows));
  if (rows > 0 && (!x || !w1 || !w3 || !w2)) return set_err(h, MOE_EINVAL, "null tensor pointer");

  std::string msg;
  rc = build_plan(params_of(c, overlapped), rows, off, src, slot, return_rows, &h->plan, &msg);
  if (rc) return set_err(h, rc, msg);
  const Plan& P = h->plan;
  if (P.n_lrows() > h->max_lrows || (int64_t)P.tile_rows.size() > h->max_tile_rows)
    return set_err(h, MOE_ECAPACITY, "plan exceeds the handle's workspaces");
  *lay = blob_layout((int64_t)P.tile_rows.size(), (int64_t)P.items.size(), P.n_lrows(),
                     (int64_t)P.segs.size(), (int64_t)P.groups.size(), c.num_ranks);
  if (lay->total > h->plan_cap) return set_err(h, MOE_ECAPACITY, "plan exceeds the plan buffer");

  h->last.plan_us =
      std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
  PlanHeader hd{};
  hd.bad_row = INT32_MAX;
  hd.n_tile_rows = (int32_t)P.tile_rows.size();
  hd.n_groups = hd.n_groups_all = (int32_t)P.groups.size();
  hd.n_gu = P.n_gu;
  hd.n_down = P.n_down;
  hd.n_segs = (int32_t)P.segs.size();
  hd.tail_split = P.tail_split;
  hd.n_split_rows = P.n_split_rows;
  hd.n_partials = P.n_partials;
  for (int x = 0; x < kXcds; ++x)
    hd.down_qmax = std::max(hd.down_qmax, P.down_queue[x + 1] - P.down_queue[x]);
  hd.n_valid = P.n_valid;
  hd.n_lrows = P.n_lrows();
  hd.n_band_pad = P.n_band_pad;
  hd.n_remote = P.n_remote;
  // The kernels index the whole item table: the down queues follow the gate/up items.
  int32_t queues[2 * (kXcds + 1)];
  for (int x = 0; x <= kXcds; ++x) {
    queues[x] = P.gu_queue[x];
    queues[kXcds + 1 + x] = P.n_gu + P.down_queue[x];
  }
  // Stage into pinned memory (wait until the copy that last used this half finished).
  const int si = h->stage_idx;
  h->stage_idx ^= 1;
  HIP_TRY(h, hipEventSynchronize(h->stage_free[si]));
  uint8_t* hs = h->h_stage[si];
  memcpy(hs + lay->hdr, &hd, sizeof hd);
  memcpy(hs + lay->tile_rows, P.tile_rows.data(), sizeof(TileRow) * P.tile_rows.size());
  memcpy(hs + lay->items, P.items.data(), sizeof(uint32_t) * P.items.size());
  memcpy(hs + lay->queues, queues, sizeof queues);
  memcpy(hs + lay->row_x, P.row_x.data(), sizeof(int32_t) * P.row_x.size());
  memcpy(hs + lay->row_rank, P.row_rank.data(), sizeof(int32_t) * P.row_rank.size());
  memcpy(hs + lay->row_slot, P.row_slot.data(), sizeof(int32_t) * P.row_slot.size());
  memcpy(hs + lay->segs, P.segs.data(), sizeof(Segment) * P.segs.size());
  memcpy(hs + lay->groups, P.groups.data(), sizeof(Group) * P.groups.size());
  if (c.down_split_k == 0) {  // the tail kernel's list of split tile rows, in schedule order
    int32_t* tail = (int32_t*)(hs + lay->tail);
    for (size_t t = 0; t < P.tile_rows.size(); ++t)
      if (P.tile_rows[t].split > 1) tail[P.tile_rows[t].part_base / (P.down_per_row * P.tail_split)] = (int32_t)t;
  }
  memcpy(hs + lay->ret, ret, sizeof(void*) * (size_t)c.num_ranks);
  memcpy(hs + lay->ret + sizeof(void*) * (size_t)c.num_ranks, return_rows, sizeof(int64_t) * (size_t)c.num_ranks);

  HIP_TRY(h, hipMemcpyAsync(h->d_plan, hs, lay->total, hipMemcpyHostToDevice, stream));
  HIP_TRY(h, hipEventRecord(h->stage_free[si], stream));
  rc = enqueue_init(h, overlapped, false, (int32_t)P.tile_rows.size(), P.n_lrows(), stream);
  if (rc) return rc;
  h->last_lay = *lay;
  h->last_dev = false;
  h->dev_hdr_pending = false;
  h->last_overlapped = overlapped;
  moe_stage_stats_t& st = h->last;
  st.n_valid = P.n_valid;
  st.n_logical_rows = P.n_lrows();
  st.n_band_padding = P.n_band_pad;
  st.n_remote_rows = P.n_remote;
  st.n_tile_rows = (int32_t)P.tile_rows.size();
  st.n_groups = (int32_t)P.groups.size();
  st.n_gu_items = P.n_gu;
  st.n_down_items = P.n_down;
  st.n_segments = (int32_t)P.segs.size();
  st.split_k = P.tail_split;
  st.split_rows = P.n_split_rows;
  return MOE_OK;
}

// Enqueues the device planner on `stream` for routing already in device memory: only the
// receive-buffer pointers and sizes go up from the host.  Routing errors are found on the
// device; the plan is then empty and moe_stage_query reports them.
int prepare_device(moe_stage_s* h, bool overlapped, const void* x, const int32_t* off,
                   const int32_t* src, const int32_t* slot, const void* w1, const void* w3,
                   const void* w2, void* const* ret, const int64_t* return_rows, hipStream_t stream,
                   BlobLayout* lay) {
  const auto t0 = std::chrono::steady_clock::now();
  const moe_stage_config_t& c = h->cfg;
  if (!off || !src || !slot) return set_err(h, MOE_EINVAL, "null routing array");
  if (!x || !w1 || !w3 || !w2) return set_err(h, MOE_EINVAL, "null tensor pointer");
  int rc = check_run_args(h, ret, return_rows);
  if (rc) return rc;
  const int32_t gu_per_row = (c.ffn + kGuTileF - 1) / kGuTileF;
  if (gu_per_row >= kMaxColTiles || h->down_per_row > kMaxDownColTiles)
    return set_err(h, MOE_EUNSUPPORTED, "hidden or ffn too large for the work-item encoding");
  *lay = h->cap_lay;
  const size_t R = (size_t)c.num_ranks;
  if (h->h_stage[0]) {
    const int si = h->stage_idx;
    h->stage_idx ^= 1;
    HIP_TRY(h, hipEventSynchronize(h->stage_free[si]));
    uint8_t* hs = h->h_stage[si];
    memcpy(hs, ret, sizeof(void*) * R);
    memcpy(hs + sizeof(void*) * R, return_rows, sizeof(int64_t) * R);
    HIP_TRY(h, hipMemcpyAsync(h->d_plan + lay->ret, hs, (sizeof(void*) + sizeof(int64_t)) * R,
                              hipMemcpyHostToDevice, stream));
    HIP_TRY(h, hipEventRecord(h->stage_free[si], stream));
  } else {  // a handle without pinned staging (the no-allocation entry point): pageable copies
    HIP_TRY(h, hipMemcpyAsync(h->d_plan + lay->ret, ret, sizeof(void*) * R, hipMemcpyHostToDevice, stream));
    HIP_TRY(h, hipMemcpyAsync(h->d_plan + lay->ret + sizeof(void*) * R, return_rows, sizeof(int64_t) * R,
                              hipMemcpyHostToDevice, stream));
  }
  rc = enqueue_init(h, overlapped, true, h->max_tile_rows, h->max_lrows, stream);
  if (rc) return rc;

  DevPlanArgs a{};
  a.off = off;
  a.src = src;
  a.slot = slot;
  a.return_rows = (const int64_t*)(h->d_plan + lay->ret + sizeof(void*) * R);
  a.E_l = c.num_local_experts;
  a.R = c.num_ranks;
  a.self = c.self_rank;
  a.tb = std::max(c.band_rows, 1);
  a.mid_pieces = std::max(c.mid_segment_pieces, 1);
  const PlanParams pp;
  a.gu_group = pp.gu_group;
  a.down_group = pp.down_group;
  a.split_k = c.down_split_k;
  a.gu_per_row = gu_per_row;
  a.down_per_row = h->down_per_row;
  a.nk = c.ffn / kTileK;
  a.overlapped = overlapped ? 1 : 0;
  a.local_direct = (c.flags & MOE_LOCAL_DIRECT) ? 1 : 0;
  a.no_lds = (c.flags & MOE_TEST_PLAN_NO_LDS) ? 1 : 0;
  a.max_rows = c.max_rows;
  a.max_tile_rows = h->max_tile_rows;
  a.hdr = (PlanHeader*)(h->d_plan + lay->hdr);
  a.tile_rows = (TileRow*)(h->d_plan + lay->tile_rows);
  a.items = (uint32_t*)(h->d_plan + lay->items);
  a.queues = (int32_t*)(h->d_plan + lay->queues);
  a.row_x = (int32_t*)(h->d_plan + lay->row_x);
  a.row_rank = (int32_t*)(h->d_plan + lay->row_rank);
  a.row_slot = (int32_t*)(h->d_plan + lay->row_slot);
  a.segs = (Segment*)(h->d_plan + lay->segs);
  a.groups = (Group*)(h->d_plan + lay->groups);
  a.tail_rows = (int32_t*)(h->d_plan + lay->tail);
  a.ws = h->ws;
  HIP_TRY(h, launch_devplan(a, h->max_items, h->num_cus, stream));
  h->last.plan_us =
      std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
  h->last_lay = *lay;
  h->last_dev = true;
  h->dev_hdr_pending = true;
  h->last_overlapped = overlapped;
  return MOE_OK;
}

ProducerArgs producer_args(moe_stage_s* h, const BlobLayout& lay, const void* x, const void* w1,
                           const void* w3, const void* w2, uint32_t mode, bool down) {
  ProducerArgs a{};
  a.x = (const uint16_t*)x;
  a.w1 = (const uint16_t*)w1;
  a.w3 = (const uint16_t*)w3;
  a.w2 = (const uint16_t*)w2;
  a.hws = h->hws;
  a.hws_rows = h->max_lrows;
  a.y = h->y;
  a.tile_rows = (const TileRow*)(h->d_plan + lay.tile_rows);
  a.items = (const uint32_t*)(h->d_plan + lay.items);
  a.queue = (const int32_t*)(h->d_plan + lay.queues) + (down ? kXcds + 1 : 0);
  a.claim = down ? h->ctr->down_next : h->ctr->gu_next;
  a.active = down ? &h->ctr->down_active : &h->ctr->gu_active;
  a.row_x = (const int32_t*)(h->d_plan + lay.row_x);
  a.row_rank = (const int32_t*)(h->d_plan + lay.row_rank);
  a.row_slot = (const int32_t*)(h->d_plan + lay.row_slot);
  a.ret = (uint16_t* const*)(h->d_plan + lay.ret);
  a.flags = h->flags;
  a.epoch = h->epoch;
  a.H = h->cfg.hidden;
  a.F = h->cfg.ffn;
  a.self_rank = h->cfg.self_rank;
  a.down_per_row = h->down_per_row;
  a.mode = mode;
  a.split_k = h->cfg.down_split_k;
  a.partials = h->partials;
  a.arrivals = h->arrivals;
  a.wcount = h->wcount;
  if (h->wg_rec) {
    a.wg_rec = h->wg_rec + (down ? (size_t)h->num_cus * h->producer_bpc : 0);
    a.ctr = h->ctr;
    a.tile_ready = h->tile_ready;
  }
  return a;
}

TailArgs tail_args(moe_stage_s* h, const BlobLayout& lay, const ProducerArgs& down) {
  TailArgs t{};
  t.p = down;
  t.tail_rows = (const int32_t*)(h->d_plan + lay.tail);
  t.n_split_rows = &((const PlanHeader*)(h->d_plan + lay.hdr))->n_split_rows;
  return t;
}

TimingRec* timing_slot(moe_stage_s* h) {
  if (!(h->cfg.flags & MOE_KERNEL_TIMING)) return nullptr;
  TimingRec* r = &h->ring[h->ring_next];
  h->ring_next = (h->ring_next + 1) % kTimingRing;
  h->ring_count = std::min(h->ring_count + 1, kTimingRing);
  return r;
}

// CU masks for the consumer/producer partition.  Workgroups of a launch are dealt
// round-robin to the XCDs, so a queue must own CUs on every XCD, and an even split keeps
// the per-XCD share symmetric: the consumer gets m = c / n_xcd CUs on each XCD.  Mask bit b
// selects compute unit b / n_xcd of XCD b mod n_xcd, and consecutive compute units of an XCD
// sit in different shader engines (both read from the placement records on MI355X), so the first
// c bits give the consumer m compute units on every XCD spread over its shader engines.  (Bits
// (cus_per_xcd + 1) * i + j, j < m, which also land on every XCD, put all m of an XCD's compute
// units in one shader engine for m <= 8, whose shared path to L2 held a 16- to 64-CU copy at
// the same 1.5 TB/s.)  The producer gets the complement, or every CU when `shared`.
void make_masks(int num_cus, int n_xcd, int c, bool shared, std::vector<uint32_t>* mc,
                std::vector<uint32_t>* mp) {
  (void)n_xcd;
  const int words = (num_cus + 31) / 32;
  mc->assign(words, 0);
  mp->assign(words, 0);
  for (int cu = 0; cu < num_cus; ++cu) {
    const bool is_c = cu < c;
    if (is_c) (*mc)[cu / 32] |= 1u << (cu % 32);
    if (shared || !is_c) (*mp)[cu / 32] |= 1u << (cu % 32);
  }
}

// Adaptive split: collects the stage times of finished measured runs (never waits).
void harvest_auto(moe_stage_s* h) {
  AutoSplit& a = h->autos;
  for (int i = 0; i < kAutoRing; ++i) {
    if (!a.busy[i] || hipEventQuery(a.done[i]) != hipSuccess) continue;
    const volatile uint64_t* st = a.stamps + 2 * i;
    const uint64_t t0 = st[0], t1 = st[1];
    if (t1 > t0) a.ms[a.ev_cand[i]].push_back((float)((double)(t1 - t0) * 1e-5));  // 100 MHz ticks
    a.busy[i] = false;
  }
}

int auto_split(const moe_stage_s* h, int i) {
  return (h->cfg.flags & MOE_SHARED_CUS) ? kAutoSplitsShared[i] : kAutoSplitsPartitioned[i];
}

// The split of the next auto run: the candidates are measured one after another, each alone
// (its CU-masked queue is the only one the handle keeps, as in the steady state it is chosen
// for: live queues of other splits slow the stage by amounts that differ from split to split),
// 1 + kAutoSamples finished runs each; the one with the lowest median stage time over all but
// its first (which pays for the new queue) is kept.  Returns the candidate index.
int pick_auto(moe_stage_s* h) {
  AutoSplit& a = h->autos;
  if (a.chosen >= 0) return a.chosen;
  auto valid = [&](int c) { return auto_split(h, c) <= h->num_cus - h->n_xcd; };
  bool any = false;
  for (int c = 0; c < kNumAutoSplits; ++c) any |= valid(c);
  if (!any) return 0;  // no candidate fits this GPU: the run reports the split as unsupported
  while (a.cand < kNumAutoSplits && (!valid(a.cand) || (int)a.ms[a.cand].size() >= 1 + kAutoSamples))
    ++a.cand;
  if (a.cand < kNumAutoSplits) return a.cand;
  float best = 0.f;
  for (int c = 0; c < kNumAutoSplits; ++c) {
    if (!valid(c)) continue;
    std::vector<float> v(a.ms[c].begin() + 1, a.ms[c].end());
    std::nth_element(v.begin(), v.begin() + v.size() / 2, v.end());
    if (a.chosen < 0 || v[v.size() / 2] < best) {
      a.chosen = c;
      best = v[v.size() / 2];
    }
  }
  return a.chosen >= 0 ? a.chosen : 0;
}

// Copy units per segment (powers of two).  Beside the producer, few: a copying wave slows the
// producer workgroup on its compute unit; segments ready in the down launch's last two rounds
// take H / 256 units (about 128 KiB of each 256-row piece, 4..16).  On compute units of its own
// the consumer cuts each 256-row piece into units of about 64 KiB (H / 128, 4..64), so its
// waves copy in parallel whatever the segment count.
void copy_units(int32_t H, bool shared, int32_t* early_shift, int32_t* late_shift) {
  auto log2_floor = [](int32_t v) { return v > 1 ? 31 - __builtin_clz((uint32_t)v) : 0; };
  if (shared) {
    *early_shift = kCopyPartsShift;
    *late_shift = std::min(std::max(log2_floor(H / 256), kCopyPartsShift), kCopyPartsLateShift);
  } else {
    *early_shift = *late_shift = std::min(std::max(log2_floor(H / 128), kCopyPartsShift), kCopyPartsOwnShift);
  }
}

// The copy units of a host-built plan, as the consumer counts them from the uploaded plan: the
// segments ready before the last kLatePositions positions of the longest down queue take
// 2^early_shift units each, the others 2^late_shift.
int64_t host_copy_units(const Plan& P, int32_t early_shift, int32_t late_shift) {
  int32_t qmax = 0;
  for (int x = 0; x < kXcds; ++x) qmax = std::max(qmax, P.down_queue[x + 1] - P.down_queue[x]);
  int64_t early = 0;
  while (early < (int64_t)P.segs.size() && P.segs[early].ready_pos < qmax - kLatePositions) ++early;
  return (early << early_shift) + (((int64_t)P.segs.size() - early) << late_shift);
}

// Consumer waves per compute unit beside the producer for a split of c compute units: a power of
// two, 1 to 8, so that about kConsumerWavesShared waves copy in all.
int consumer_waves_per_cu(int c) {
  int w = 1;
  while (w < 8 && (w * 2) * c <= kConsumerWavesShared) w *= 2;
  return w;
}

// Consumer CUs actually reserved for a requested split: a multiple of the XCD count.
int effective_split(const moe_stage_s* h, int c) {
  const int n = h->n_xcd;
  return std::min((c + n - 1) / n * n, h->num_cus - n);
}

void destroy_split(moe_stage_s::SplitQueues& q) {
  (void)hipStreamSynchronize(q.cons);
  (void)hipStreamDestroy(q.cons);
  if (q.prod) {
    (void)hipStreamSynchronize(q.prod);
    (void)hipStreamDestroy(q.prod);
  }
}

// Releases the queues of every split but `keep` (waiting for work still on them).
void release_other_queues(moe_stage_s* h, int keep) {
  std::vector<moe_stage_s::SplitQueues> kept;
  for (auto& q : h->queues) {
    if (q.c == keep)
      kept.push_back(q);
    else
      destroy_split(q);
  }
  h->queues.swap(kept);
  if (h->cached_split != keep) h->cached_split = -1;
}

// Makes the consumer queue of split c (and its producer queue where the run needs one)
// current, releasing every other split's queues: live CU-masked queues slow the stage.
int ensure_streams(moe_stage_s* h, int c, bool need_prod) {
  const bool shared = (h->cfg.flags & MOE_SHARED_CUS) != 0;
  if (h->queues.size() > 1 || (h->queues.size() == 1 && h->queues[0].c != c)) release_other_queues(h, c);
  moe_stage_s::SplitQueues* cur = nullptr;
  for (auto& q : h->queues)
    if (q.c == c) cur = &q;
  if (!cur) {
    std::vector<uint32_t> mc, mp;
    make_masks(h->num_cus, h->n_xcd, c, shared, &mc, &mp);
    moe_stage_s::SplitQueues q{c, nullptr, nullptr};
    HIP_TRY(h, hipExtStreamCreateWithCUMask(&q.cons, (uint32_t)mc.size(), mc.data()));
    if (!shared && hipExtStreamCreateWithCUMask(&q.prod, (uint32_t)mp.size(), mp.data()) != hipSuccess) {
      (void)hipStreamDestroy(q.cons);
      return set_err(h, MOE_EHIP, "hipExtStreamCreateWithCUMask(producer)");
    }
    h->queues.push_back(q);
    cur = &h->queues.back();
  }
  if (shared && need_prod && !h->shared_prod) {
    std::vector<uint32_t> mc, mp;
    make_masks(h->num_cus, h->n_xcd, c, true, &mc, &mp);
    HIP_TRY(h, hipExtStreamCreateWithCUMask(&h->shared_prod, (uint32_t)mp.size(), mp.data()));
  }
  h->s_cons = cur->cons;
  h->s_prod = shared ? h->shared_prod : cur->prod;
  h->cached_split = c;
  return MOE_OK;
}

// Workspace sizes of a handle (its configuration set): the capacities every run fits in.
struct WsBytes {
  size_t hws, y, flags, partials, planner;
};

WsBytes size_workspaces(moe_stage_s* h) {
  const moe_stage_config_t& c = h->cfg;
  h->max_lrows = max_logical_rows(c.max_rows, c.num_local_experts, c.num_ranks, c.band_rows);
  h->max_tile_rows = (int32_t)((h->max_lrows + kTileM - 1) / kTileM) + c.num_local_experts;
  h->max_lrows = (int64_t)h->max_tile_rows * kTileM;
  h->down_per_row = (c.hidden + kDownTileN - 1) / kDownTileN;
  const int gu_per_row = (c.ffn + kGuTileF - 1) / kGuTileF;
  const int32_t S = c.down_split_k;
  // Down items: one per part of every tile (uniform split), or one per tile plus at most one
  // round of parts for the split tail rows (default).
  h->max_items = (int64_t)h->max_tile_rows * (gu_per_row + (int64_t)h->down_per_row * std::max(S, 1)) +
                 (S == 0 ? kRoundTiles : 0);
  // Segments: at most one per routed row.  Groups: one per (local expert, source rank).
  h->cap_lay = blob_layout(h->max_tile_rows, h->max_items, h->max_lrows, h->max_lrows,
                           (int64_t)c.num_local_experts * c.num_ranks, c.num_ranks);
  h->plan_cap = h->cap_lay.total;
  WsBytes b;
  b.planner = devplan_ws_bytes(c.num_local_experts, c.num_ranks, c.max_rows, h->max_tile_rows, h->down_per_row,
                               h->max_lrows, h->max_items);
  b.hws = (size_t)h->max_lrows * c.ffn * 2;
  b.y = (size_t)h->max_lrows * c.hidden * 2;
  b.flags = (size_t)h->max_tile_rows * h->down_per_row * 4;
  // One fp32 partial tile (256 threads x 256 accumulators) per K part of a split down tile.
  b.partials = (size_t)max_partial_tiles(S, h->max_tile_rows, h->down_per_row, c.ffn / kTileK) * kProducerThreads *
               256 * 4;
  return b;
}

}  // namespace

extern "C" {

int moe_stage_create(const moe_stage_config_t* cfg, moe_stage_t* out) {
  if (!out) return set_err(nullptr, MOE_EINVAL, "out is null");
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc) return set_err(nullptr, rc, "invalid configuration");
  auto* h = new moe_stage_s();
  h->cfg = *cfg;
  if (h->cfg.mid_segment_pieces == 0) h->cfg.mid_segment_pieces = 1;
  if (h->cfg.band_rows == 0) h->cfg.band_rows = 1;
  auto bail = [&](int code) {
    moe_stage_destroy(h);
    return code;
  };
  hipError_t e = hipGetDevice(&h->device);
  hipDeviceProp_t prop{};
  if (e == hipSuccess) e = hipGetDeviceProperties(&prop, h->device);
  if (e != hipSuccess) {
    set_err(nullptr, MOE_EHIP, std::string("no HIP device: ") + hipGetErrorString(e));
    delete h;
    return MOE_EHIP;
  }
  h->num_cus = prop.multiProcessorCount;
  if (hipDeviceGetAttribute(&h->n_xcd, hipDeviceAttributeNumberOfXccs, h->device) != hipSuccess ||
      h->n_xcd < 1 || h->num_cus % h->n_xcd != 0)
    h->n_xcd = 1;
  h->producer_bpc = producer_blocks_per_cu();
  const WsBytes wb = size_workspaces(h);
  const size_t ws_bytes = wb.planner, hws_bytes = wb.hws, y_bytes = wb.y, flag_bytes = wb.flags,
               part_bytes = wb.partials;

  auto try_hip = [&](hipError_t err, const char* what) {
    if (err != hipSuccess) {
      set_err(nullptr, MOE_EHIP, std::string(what) + ": " + hipGetErrorString(err));
      return false;
    }
    return true;
  };
  if ((part_bytes && !try_hip(hipMalloc(&h->partials, part_bytes), "hipMalloc(partials)")) ||
      !try_hip(hipMalloc(&h->arrivals, flag_bytes), "hipMalloc(arrivals)") ||
      !try_hip(hipMalloc(&h->abandoned, sizeof(uint32_t) * kMaxAbandoned), "hipMalloc(counters)") ||
      !try_hip(hipMemset(h->arrivals, 0, flag_bytes), "hipMemset(arrivals)") ||
      !try_hip(hipMalloc(&h->hws, hws_bytes), "hipMalloc(hws)") ||
      !try_hip(hipMalloc(&h->y, y_bytes), "hipMalloc(y)") ||
      !try_hip(hipMalloc(&h->flags, flag_bytes), "hipMalloc(flags)") ||
      !try_hip(hipMalloc(&h->ctr, sizeof(RunCounters)), "hipMalloc(counters)") ||
      !try_hip(hipMalloc(&h->simd_waves, sizeof(uint32_t) * kWaveCounters), "hipMalloc(counters)") ||
      !try_hip(hipMemset(h->simd_waves, 0, sizeof(uint32_t) * kWaveCounters), "hipMemset(counters)") ||
      !try_hip(hipMalloc(&h->d_plan, h->plan_cap), "hipMalloc(plan)") ||
      !try_hip(hipMalloc(&h->dev_ws, ws_bytes), "hipMalloc(planner scratch)") ||
      !try_hip(hipHostMalloc(&h->h_stage[0], h->plan_cap, hipHostMallocDefault), "hipHostMalloc") ||
      !try_hip(hipHostMalloc(&h->h_stage[1], h->plan_cap, hipHostMallocDefault), "hipHostMalloc") ||
      !try_hip(hipMemset(h->hws, 0, hws_bytes), "hipMemset(hws)") ||
      !try_hip(hipMemset(h->y, 0, y_bytes), "hipMemset(y)") ||
      !try_hip(hipMemset(h->flags, 0, flag_bytes), "hipMemset(flags)") ||
      !try_hip(hipMemset(h->ctr, 0, sizeof(RunCounters)), "hipMemset(counters)") ||
      !try_hip(hipMemset(&h->ctr->timeout_seg, 0xFF, sizeof(uint32_t)), "hipMemset(counters)"))
    return bail(MOE_EHIP);
  if ((cfg->flags & MOE_WRITE_COUNTS) &&
      (!try_hip(hipMalloc(&h->wcount, (size_t)h->max_lrows * 4), "hipMalloc(write counts)") ||
       !try_hip(hipMemset(h->wcount, 0, (size_t)h->max_lrows * 4), "hipMemset(write counts)")))
    return bail(MOE_EHIP);
  if (cfg->flags & MOE_TIMESTAMPS) {
    const size_t wg_bytes = 2 * (size_t)h->num_cus * h->producer_bpc * sizeof(WgRecord);
    const size_t cp_bytes = (size_t)kMaxCopyRecords * sizeof(CopyRecord);
    if (!try_hip(hipMalloc(&h->wg_rec, wg_bytes), "hipMalloc(records)") ||
        !try_hip(hipMalloc(&h->copy_rec, cp_bytes), "hipMalloc(records)") ||
        !try_hip(hipMalloc(&h->tile_ready, flag_bytes * 2), "hipMalloc(records)") ||
        !try_hip(hipMemset(h->wg_rec, 0, wg_bytes), "hipMemset(records)") ||
        !try_hip(hipMemset(h->copy_rec, 0, cp_bytes), "hipMemset(records)"))
      return bail(MOE_EHIP);
  }
  h->ws = devplan_ws_carve(h->dev_ws, cfg->num_local_experts, cfg->num_ranks, cfg->max_rows,
                           h->max_tile_rows, h->down_per_row, h->max_lrows, h->max_items);
  // Every event here orders work on this device or marks completion for the host; none
  // publishes device writes to the host (results are read through the caller's own copies),
  // so a device-scope release suffices and no system-scope cache writeback sits between
  // launches.
  constexpr unsigned kSyncEv = hipEventDisableTiming | hipEventReleaseToDevice;
  for (int i = 0; i < 2; ++i)
    if (!try_hip(hipEventCreateWithFlags(&h->stage_free[i], kSyncEv), "hipEventCreate") ||
        !try_hip(hipEventRecord(h->stage_free[i], nullptr), "hipEventRecord"))
      return bail(MOE_EHIP);
  if (!try_hip(hipEventCreateWithFlags(&h->ev_fork, kSyncEv), "hipEventCreate") ||
      !try_hip(hipEventCreateWithFlags(&h->ev_join_c, kSyncEv), "hipEventCreate") ||
      !try_hip(hipEventCreateWithFlags(&h->ev_join_p, kSyncEv), "hipEventCreate") ||
      !try_hip(hipEventCreateWithFlags(&h->ev_done, kSyncEv), "hipEventCreate"))
    return bail(MOE_EHIP);
  for (auto& ev : h->autos.done)
    if (!try_hip(hipEventCreateWithFlags(&ev, kSyncEv), "hipEventCreate")) return bail(MOE_EHIP);
  if (!try_hip(hipHostMalloc((void**)&h->autos.stamps, 2 * kAutoRing * sizeof(uint64_t),
                             hipHostMallocCoherent | hipHostMallocMapped),
               "hipHostMalloc"))
    return bail(MOE_EHIP);
  if (h->cfg.flags & MOE_KERNEL_TIMING) {
    h->ring.resize(kTimingRing);
    for (auto& r : h->ring)
      for (auto& ev : r.ev)
        if (!try_hip(hipEventCreateWithFlags(&ev, hipEventReleaseToDevice), "hipEventCreate"))
          return bail(MOE_EHIP);
  }
  if (!try_hip(hipDeviceSynchronize(), "hipDeviceSynchronize")) return bail(MOE_EHIP);
  *out = h;
  return MOE_OK;
}

static int run_overlapped(moe_stage_t h, bool dev, const void* x, const int32_t* off,
                          const int32_t* src, const int32_t* slot, const void* w1, const void* w3,
                          const void* w2, void* const* ret, const int64_t* return_rows,
                          int32_t cu_split, void* stream_) {
  if (!h) return MOE_EINVAL;
  hipStream_t stream = (hipStream_t)stream_;
  const bool autosplit = cu_split == 0;
  int auto_cand = -1, auto_slot = -1;
  if (autosplit) {
    harvest_auto(h);
    auto_cand = pick_auto(h);
    cu_split = auto_split(h, auto_cand);
    if (!h->autos.busy[h->autos.next]) auto_slot = h->autos.next;  // else: this run is not measured
  }
  if (cu_split < 1 || cu_split > h->num_cus - h->n_xcd)
    return set_err(h, MOE_EUNSUPPORTED, "cu_split must be in [0, compute units - XCDs]");
  const int c_eff = effective_split(h, cu_split);
  const bool shared = (h->cfg.flags & MOE_SHARED_CUS) != 0;
  const int pgrid = (shared ? h->num_cus : h->num_cus - c_eff) * h->producer_bpc;
  // Consumer workgroups per CU: two beside a producer workgroup (their registers fill what a
  // producer wave leaves free), four of the wider variant when the consumer owns its CUs.
  const bool own_cus = !shared;
  // Consumer waves beside the producer: about kConsumerWavesShared in all, spread over the c_eff
  // compute units (8 per CU on 32 CUs, 1 per CU on 248): each copying wave slows the producer
  // workgroup on its compute unit, so a wide split copies thinly everywhere, and the down launch's
  // last workgroups are not held back on a few busy compute units.  On compute units of its own the
  // consumer runs kConsumerOwnPerCu workgroups of four waves per compute unit.
  const int wpc = own_cus ? 4 * kConsumerOwnPerCu : consumer_waves_per_cu(c_eff);
  const int cthreads = own_cus ? kConsumerThreads : 64 * std::min(wpc, 4);
  int cgrid = own_cus ? c_eff * kConsumerOwnPerCu : c_eff * std::max(1, wpc / 4);
  const bool legacy = stream == nullptr || stream == hipStreamLegacy;
  const bool on_caller = shared && !legacy;
  // The adaptive selector keeps its candidates' queues until it has settled.
  int rc = ensure_streams(h, c_eff, !on_caller);
  if (rc) return rc;
  BlobLayout lay{};
  TimingRec* tr = timing_slot(h);
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[0], stream));
  if (auto_slot >= 0) HIP_TRY(h, launch_stamp(&h->autos.stamps[2 * auto_slot], stream));
  rc = dev ? prepare_device(h, true, x, off, src, slot, w1, w3, w2, ret, return_rows, stream, &lay)
           : prepare(h, true, x, off, src, slot, w1, w3, w2, ret, return_rows, stream, &lay);
  if (rc) {
    if (tr) h->ring_next = (h->ring_next + kTimingRing - 1) % kTimingRing, --h->ring_count;
    return rc;
  }
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[7], stream));
  int32_t early_shift = 0, late_shift = 0;
  copy_units(h->cfg.hidden, !own_cus, &early_shift, &late_shift);
  // A host-built plan's copy units are known: launch no more consumer waves than there are units
  // (a small stage's few units would otherwise send hundreds of waves claiming nothing), and a
  // drain of about one workgroup per four units.
  int dgrid = shared ? h->num_cus : h->num_cus - c_eff;
  if (!dev) {
    const int64_t units = host_copy_units(h->plan, early_shift, late_shift);
    cgrid = (int)std::min<int64_t>(cgrid, std::max<int64_t>(1, (units + cthreads / 64 - 1) / (cthreads / 64)));
    dgrid = (int)std::min<int64_t>(dgrid, std::max<int64_t>(h->n_xcd, (units + 3) / 4));
  }
  h->last.producer_grid = pgrid;
  h->last.consumer_grid = cgrid;
  h->last.consumer_cus = c_eff;
  uint32_t mode = (h->cfg.flags & MOE_TEST_NO_SIGNAL) ? 0u : kModeSignal;
  if (h->cfg.flags & MOE_LOCAL_DIRECT) mode |= kModeLocalDirect;
  if (h->cfg.down_split_k == 0) mode |= kModeDeferTail;
  ProducerArgs pgu = producer_args(h, lay, x, w1, w3, w2, mode, false);
  const ProducerArgs pdn = producer_args(h, lay, x, w1, w3, w2, mode, true);
  ConsumerArgs ca{};
  ca.y = h->y;
  ca.ret = pgu.ret;
  ca.segs = (const Segment*)(h->d_plan + lay.segs);
  ca.n_segs = &((const PlanHeader*)(h->d_plan + lay.hdr))->n_segs;
  ca.down_qmax = &((const PlanHeader*)(h->d_plan + lay.hdr))->down_qmax;
  ca.flags = h->flags;
  ca.epoch = h->epoch;
  ca.H = h->cfg.hidden;
  ca.ctr = h->ctr;
  ca.watchdog_ticks = watchdog_ticks(h);
  ca.early_shift = early_shift;
  ca.late_shift = late_shift;
  ca.abandoned = h->abandoned;
  ca.abandoned_cap = kMaxAbandoned;
  ca.wcount = h->wcount;
  if (!own_cus) {
    ca.simd_waves = h->simd_waves;
    ca.max_waves_cu = (uint32_t)wpc;
  }
  if (h->copy_rec) {
    ca.rec = h->copy_rec;
    ca.rec_cap = kMaxCopyRecords;
  }

  // No event orders the consumer after this run's reset: the consumer launch waits for the run's
  // epoch in the counters, which the gate/up launch publishes as it starts (it follows the init
  // kernel), so the caller's stream carries no cross-queue packet (an event there stalled it
  // ~6 us per run, a kernel of its own ~5 us).
  // Its queue holds it behind the previous run's consumer, whose waves the previous drain saw
  // leave before this run's reset.  Should the caller's stream hold back the reset past the
  // watchdog, the consumer leaves without copying and the drain launch copies every unit.
  // With shared CUs the producer stays on the caller's stream and is enqueued first, so the
  // host's consumer launch overlaps the gate/up launch -- unless that stream is the legacy null
  // stream, whose launches wait for all earlier work on blocking streams, the still-polling
  // consumer included: that would be a cycle, so the producer then forks to the handle's own
  // stream like the partitioned launch, after an event that orders it behind the reset.
  hipStream_t ps = on_caller ? stream : h->s_prod;
  const bool producer = !(h->cfg.flags & MOE_TEST_CONSUMER_ONLY);
  // A host-built plan's counts are known here, so empty launches are skipped; a device-built
  // plan's kernels read them and return at once when there is nothing to do.
  const bool known = !dev;
  const bool gu_launch = producer && (!known || h->plan.n_gu > 0);
  if (gu_launch)
    pgu.go_ctr = h->ctr;
  else
    HIP_TRY(h, launch_go(h->ctr, h->epoch, stream));
  if (!on_caller || !producer) {
    // The handle's producer stream follows the reset through an event; so does the consumer of
    // the consumer-only measurement, whose timing then starts at the reset.
    HIP_TRY(h, hipEventRecord(h->ev_fork, stream));
    if (!on_caller) HIP_TRY(h, hipStreamWaitEvent(h->s_prod, h->ev_fork, 0));
    if (!producer) HIP_TRY(h, hipStreamWaitEvent(h->s_cons, h->ev_fork, 0));
  }
  const bool plain = (h->cfg.flags & MOE_TEST_CONSUMER_ONLY) && (h->cfg.flags & MOE_TEST_PLAIN_COPY);
  // With a producer, the run ends with a drain launch in the producer's stream: it copies the
  // units the consumer has not claimed by then on the producer's compute units and waits for the
  // consumer's last wave, so the caller's stream needs no event from the consumer's queue.
  const bool drain = producer && (!known || !h->plan.segs.empty());
  if (drain) {
    ca.role = kRoleCounted;
    ca.map_grid = (uint32_t)cgrid;
    ca.map_wpg = (uint32_t)(cthreads / 64);
  }
  ca.wait_go = 1;
  auto gate_up = [&]() -> int {
    if (tr) HIP_TRY(h, hipEventRecord(tr->ev[1], ps));
    if (gu_launch) HIP_TRY(h, launch_producer(pgu, false, pgrid, ps));
    return MOE_OK;
  };
  if (on_caller && (rc = gate_up()) != MOE_OK) return rc;
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[3], h->s_cons));
  if (plain && known) {
    // As many rows as the segments hold, bounded by the staged output and the first receive buffer.
    int64_t rows = 0;
    for (const Segment& sg : h->plan.segs) rows += sg.rows;
    rows = std::min<int64_t>(std::min<int64_t>(rows, return_rows[0]), h->max_lrows);
    ca.plain_n16 = rows * h->cfg.hidden / 8;
    if (ca.plain_n16 > 0) HIP_TRY(h, launch_plain_copy(ca, c_eff * kConsumerOwnPerCu, h->s_cons));
  } else if (!known || !h->plan.segs.empty()) {
    HIP_TRY(h, launch_consumer(ca, own_cus, cgrid, cthreads, h->s_cons));
  }
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[4], h->s_cons));
  HIP_TRY(h, hipEventRecord(h->ev_join_c, h->s_cons));
  if (!on_caller && (rc = gate_up()) != MOE_OK) return rc;
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[6], ps));
  if (producer && (!known || h->plan.n_down > 0)) HIP_TRY(h, launch_producer(pdn, true, pgrid, ps));
  if (producer && (pdn.mode & kModeDeferTail) && (!known || h->plan.n_split_rows > 0))
    HIP_TRY(h, launch_tail(tail_args(h, lay, pdn), kTailGrid, ps));
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[2], ps));
  if (drain) {
    ConsumerArgs da = ca;
    da.role = kRoleDrain;
    da.wait_go = 0;  // behind the producer in its stream, so behind the reset
    da.simd_waves = nullptr;
    da.exit_waves = (uint32_t)cgrid * (uint32_t)(cthreads / 64);
    HIP_TRY(h, launch_drain(da, dgrid, ps));
  }
  if (!on_caller) {
    HIP_TRY(h, hipEventRecord(h->ev_join_p, h->s_prod));
    HIP_TRY(h, hipStreamWaitEvent(stream, h->ev_join_p, 0));
  }
  if (!drain) HIP_TRY(h, hipStreamWaitEvent(stream, h->ev_join_c, 0));
  if (tr) {
    HIP_TRY(h, hipEventRecord(tr->ev[5], stream));
    tr->kind = 0;
  }
  HIP_TRY(h, hipEventRecord(h->ev_done, stream));
  if (auto_slot >= 0) {
    HIP_TRY(h, launch_stamp(&h->autos.stamps[2 * auto_slot + 1], stream));
    HIP_TRY(h, hipEventRecord(h->autos.done[auto_slot], stream));
    h->autos.busy[auto_slot] = true;
    h->autos.ev_cand[auto_slot] = auto_cand;
    h->autos.next = (auto_slot + 1) % kAutoRing;
  }
  h->last.auto_cu_split = autosplit ? (h->autos.chosen >= 0 ? auto_split(h, h->autos.chosen) : 0) : -1;
  h->ran = true;
  h->counters_pending = true;
  return MOE_OK;
}

static int run_serial(moe_stage_t h, bool dev, const void* x, const int32_t* off,
                      const int32_t* src, const int32_t* slot, const void* w1, const void* w3,
                      const void* w2, void* const* ret, const int64_t* return_rows, void* stream_) {
  if (!h) return MOE_EINVAL;
  hipStream_t stream = (hipStream_t)stream_;
  const int pgrid = h->num_cus * h->producer_bpc;
  BlobLayout lay{};
  TimingRec* tr = timing_slot(h);
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[0], stream));
  int rc = dev ? prepare_device(h, false, x, off, src, slot, w1, w3, w2, ret, return_rows, stream, &lay)
               : prepare(h, false, x, off, src, slot, w1, w3, w2, ret, return_rows, stream, &lay);
  if (rc) {
    if (tr) h->ring_next = (h->ring_next + kTimingRing - 1) % kTimingRing, --h->ring_count;
    return rc;
  }
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[7], stream));
  h->last.producer_grid = pgrid;
  h->last.consumer_grid = 0;
  h->last.auto_cu_split = -1;
  h->last.consumer_cus = 0;
  const bool direct_all = (h->cfg.flags & MOE_DIRECT_ALL) != 0;
  const uint32_t mode = (direct_all ? kModeDirectAll : 0u) | (h->cfg.down_split_k == 0 ? kModeDeferTail : 0u);
  const ProducerArgs pgu = producer_args(h, lay, x, w1, w3, w2, mode, false);
  const ProducerArgs pa = producer_args(h, lay, x, w1, w3, w2, mode, true);
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[1], stream));
  const bool known = !dev;
  if (!known || h->plan.n_gu > 0) HIP_TRY(h, launch_producer(pgu, false, pgrid, stream));
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[6], stream));
  if (!known || h->plan.n_down > 0) HIP_TRY(h, launch_producer(pa, true, pgrid, stream));
  if ((pa.mode & kModeDeferTail) && (!known || h->plan.n_split_rows > 0))
    HIP_TRY(h, launch_tail(tail_args(h, lay, pa), kTailGrid, stream));
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[2], stream));
  ScatterArgs sa{};
  sa.y = h->y;
  sa.ret = pa.ret;
  sa.row_rank = pa.row_rank;
  sa.row_slot = pa.row_slot;
  sa.n_lrows = &((const PlanHeader*)(h->d_plan + lay.hdr))->n_lrows;
  sa.H = h->cfg.hidden;
  sa.wcount = h->wcount;
  if (tr) HIP_TRY(h, hipEventRecord(tr->ev[4], stream));
  const int64_t scatter_rows = known ? h->plan.n_lrows() : h->max_lrows;
  if (scatter_rows > 0 && !direct_all)
    HIP_TRY(h, launch_scatter(sa, (int)std::min<int64_t>(scatter_rows, (int64_t)h->num_cus * 8), stream));
  if (tr) {
    HIP_TRY(h, hipEventRecord(tr->ev[5], stream));
    tr->kind = 1;
  }
  if (h->ev_done) HIP_TRY(h, hipEventRecord(h->ev_done, stream));
  h->ran = true;
  h->counters_pending = true;
  return MOE_OK;
}

int moe_stage_run(moe_stage_t h, const void* x, const int32_t* off, const int32_t* src,
                  const int32_t* slot, const void* w1, const void* w3, const void* w2,
                  void* const* ret, const int64_t* return_rows, int32_t cu_split, void* stream) {
  return run_overlapped(h, false, x, off, src, slot, w1, w3, w2, ret, return_rows, cu_split, stream);
}

int moe_stage_run_serial(moe_stage_t h, const void* x, const int32_t* off, const int32_t* src,
                         const int32_t* slot, const void* w1, const void* w3, const void* w2,
                         void* const* ret, const int64_t* return_rows, void* stream) {
  return run_serial(h, false, x, off, src, slot, w1, w3, w2, ret, return_rows, stream);
}

int moe_stage_run_devplan(moe_stage_t h, const void* x, const int32_t* off, const int32_t* src,
                          const int32_t* slot, const void* w1, const void* w3, const void* w2,
                          void* const* ret, const int64_t* return_rows, int32_t cu_split,
                          void* stream) {
  return run_overlapped(h, true, x, off, src, slot, w1, w3, w2, ret, return_rows, cu_split, stream);
}

int moe_stage_run_serial_devplan(moe_stage_t h, const void* x, const int32_t* off,
                                 const int32_t* src, const int32_t* slot, const void* w1,
                                 const void* w3, const void* w2, void* const* ret,
                                 const int64_t* return_rows, void* stream) {
  return run_serial(h, true, x, off, src, slot, w1, w3, w2, ret, return_rows, stream);
}

// Waits for the last run and reads its device counters once (the watchdog reports stay in
// h->last until a query returns them).
static int sync_counters(moe_stage_t h) {
  if (h->ran) HIP_TRY(h, hipEventSynchronize(h->ev_done));
  if (h->counters_pending) {
    h->counters_pending = false;
    RunCounters c{};
    HIP_TRY(h, hipMemcpy(&c, h->ctr, sizeof c, hipMemcpyDeviceToHost));
    h->last.poll_iters = c.poll_iters;
    h->last.wait_ticks = c.wait_ticks;
    h->last.gu_workgroups = (int32_t)c.gu_active;
    h->last.down_workgroups = (int32_t)c.down_active;
    h->last.timeout = c.timeouts ? 1 : 0;
    h->last.timeout_segment = c.timeouts ? (int32_t)c.timeout_seg : -1;
    h->last.copy_units = (int32_t)c.n_units;
    h->last_timeouts = c.timeouts;
    h->last_timeout_where = c.timeout_where;
    h->last_span[0] = c.prod_t0;
    h->last_span[1] = c.prod_t1;
    if (c.timeouts) {  // sticky across runs until reported here
      const uint32_t reset[3] = {0, 0, UINT32_MAX};  // timeouts, timeout_where, timeout_seg
      HIP_TRY(h, hipMemcpy(&h->ctr->timeouts, reset, sizeof reset, hipMemcpyHostToDevice));
    }
  }
  return MOE_OK;
}

int moe_stage_query(moe_stage_t h, moe_stage_stats_t* out) {
  if (!h || !out) return MOE_EINVAL;
  const int rc = sync_counters(h);
  if (rc) return rc;
  if (h->dev_hdr_pending) {  // a device-built plan: its counts and verdict are on the device
    h->dev_hdr_pending = false;
    PlanHeader hd{};
    HIP_TRY(h, hipMemcpy(&hd, h->d_plan + h->last_lay.hdr, sizeof hd, hipMemcpyDeviceToHost));
    moe_stage_stats_t& st = h->last;
    st.n_valid = hd.n_valid;
    st.n_logical_rows = hd.n_lrows;
    st.n_band_padding = hd.n_band_pad;
    st.n_remote_rows = hd.n_remote;
    st.n_tile_rows = hd.n_tile_rows;
    st.n_groups = hd.n_groups;
    st.n_gu_items = hd.n_gu;
    st.n_down_items = hd.n_down;
    st.n_segments = hd.n_segs;
    st.split_k = hd.tail_split;
    st.split_rows = hd.n_split_rows;
    h->dev_status = hd.status;
    h->dev_bad_row = hd.bad_row;
  }
  *out = h->last;
  if (h->dev_status) {
    const int code = h->dev_status;
    h->dev_status = 0;
    std::string what = code == MOE_ECAPACITY ? "rows > max_rows, or the plan exceeds the handle's workspaces"
                                             : "invalid routing";
    if (h->dev_bad_row != INT32_MAX && code == MOE_EROUTING) what += " at row " + std::to_string(h->dev_bad_row);
    return set_err(h, code, "device plan: " + what + "; the run did no work");
  }
  if (h->last.timeout) {
    h->last.timeout = 0;
    return set_err(h, MOE_ETIMEOUT,
                   std::to_string(h->last_timeouts) + " device wait(s) hit the watchdog since the last query (" +
                       ((h->last_timeout_where & 1) ? "consumer flag wait" : "") +
                       ((h->last_timeout_where & 3) == 3 ? ", " : "") +
                       ((h->last_timeout_where & 2) ? "end-of-stage wait for the consumer" : "") + ", first at segment " +
                       std::to_string(h->last.timeout_segment) + ")");
  }
  return MOE_OK;
}

int moe_stage_times(moe_stage_t h, int32_t reset, moe_stage_times_t* out) {
  if (!h || !out) return MOE_EINVAL;
  *out = moe_stage_times_t{};
  if (!(h->cfg.flags & MOE_KERNEL_TIMING)) return set_err(h, MOE_EINVAL, "MOE_KERNEL_TIMING not set");
  if (h->ran) HIP_TRY(h, hipEventSynchronize(h->ev_done));
  for (int k = 0; k < h->ring_count; ++k) {
    TimingRec& r = h->ring[(h->ring_next - 1 - k + 2 * kTimingRing) % kTimingRing];
    float ms = 0;
    HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[0], r.ev[5]));
    out->stage_ms += ms;
    HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[1], r.ev[2]));
    out->producer_ms += ms;
    HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[1], r.ev[6]));
    out->gate_up_ms += ms;
    HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[0], r.ev[7]));
    out->plan_ms += ms;
    if (r.kind == 0) {
      HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[3], r.ev[4]));
      out->consumer_ms += ms;
    } else {
      HIP_TRY(h, hipEventElapsedTime(&ms, r.ev[4], r.ev[5]));
      out->scatter_ms += ms;
    }
    ++out->runs;
  }
  if (reset) h->ring_count = 0;
  return MOE_OK;
}

// The last run's plan as the kernels saw it, read back from the device blob.
static int read_header(moe_stage_t h, PlanHeader* hd) {
  if (!h->ran) return set_err(h, MOE_EINVAL, "no run yet");
  HIP_TRY(h, hipEventSynchronize(h->ev_done));
  HIP_TRY(h, hipMemcpy(hd, h->d_plan + h->last_lay.hdr, sizeof *hd, hipMemcpyDeviceToHost));
  return MOE_OK;
}

int moe_stage_plan_info(moe_stage_t h, moe_plan_info_t* o) {
  if (!h || !o) return MOE_EINVAL;
  PlanHeader hd{};
  int rc = read_header(h, &hd);
  if (rc) return rc;
  *o = moe_plan_info_t{};
  o->n_tile_rows = hd.n_tile_rows;
  o->n_items = hd.n_gu + hd.n_down;
  o->n_gu_items = hd.n_gu;
  o->n_down_items = hd.n_down;
  o->n_segments = hd.n_segs;
  o->n_groups = hd.n_groups;
  o->gu_tiles_per_row = (h->cfg.ffn + kGuTileF - 1) / kGuTileF;
  o->down_tiles_per_row = h->down_per_row;
  o->tile_m = kTileM;
  o->band_rows = h->last_overlapped ? h->cfg.band_rows : 1;
  o->split_k = hd.tail_split;
  o->split_rows = hd.n_split_rows;
  o->n_logical_rows = hd.n_lrows;
  o->n_valid = hd.n_valid;
  o->n_band_padding = hd.n_band_pad;
  o->n_remote_rows = hd.n_remote;
  return MOE_OK;
}

int64_t moe_stage_plan_copy(moe_stage_t h, int32_t which, void* dst, int64_t bytes) {
  if (!h) return MOE_EINVAL;
  PlanHeader hd{};
  int rc = read_header(h, &hd);
  if (rc) return rc;
  const BlobLayout& L = h->last_lay;
  size_t off = 0;
  int64_t need = 0;
  switch (which) {
    case MOE_PLAN_TILE_ROWS: off = L.tile_rows; need = (int64_t)sizeof(TileRow) * hd.n_tile_rows; break;
    case MOE_PLAN_ITEMS: off = L.items; need = 4 * ((int64_t)hd.n_gu + hd.n_down); break;
    case MOE_PLAN_ROW_X: off = L.row_x; need = 4 * hd.n_lrows; break;
    case MOE_PLAN_ROW_RANK: off = L.row_rank; need = 4 * hd.n_lrows; break;
    case MOE_PLAN_ROW_SLOT: off = L.row_slot; need = 4 * hd.n_lrows; break;
    case MOE_PLAN_SEGMENTS: off = L.segs; need = (int64_t)sizeof(Segment) * hd.n_segs; break;
    case MOE_PLAN_GROUPS: off = L.groups; need = (int64_t)sizeof(Group) * hd.n_groups; break;
    case MOE_PLAN_QUEUES: off = L.queues; need = 4 * 2 * (kXcds + 1); break;
    default: return set_err(h, MOE_EINVAL, "unknown plan table");
  }
  if (!dst) return need;
  if (bytes < need) return set_err(h, MOE_EINVAL, "destination too small");
  if (need) HIP_TRY(h, hipMemcpy(dst, h->d_plan + off, (size_t)need, hipMemcpyDeviceToHost));
  if (which == MOE_PLAN_QUEUES) {  // the blob's down queues index the whole item table
    int32_t* q = (int32_t*)dst;
    for (int x = 0; x <= kXcds; ++x) q[kXcds + 1 + x] -= hd.n_gu;
  }
  return MOE_OK;
}

int64_t moe_stage_records(moe_stage_t h, int32_t which, void* dst, int64_t bytes) {
  if (!h) return MOE_EINVAL;
  if (which == MOE_RECORDS_WRITES) {
    if (!h->wcount) return set_err(h, MOE_EINVAL, "MOE_WRITE_COUNTS not set");
    if (!h->ran) return set_err(h, MOE_EINVAL, "no run yet");
    const int64_t need = h->max_lrows * 4;
    if (!dst) return need;
    if (bytes < need) return set_err(h, MOE_EINVAL, "destination too small");
    const int rc = sync_counters(h);
    if (rc) return rc;
    HIP_TRY(h, hipMemcpy(dst, h->wcount, (size_t)need, hipMemcpyDeviceToHost));
    return MOE_OK;
  }
  if (!(h->cfg.flags & MOE_TIMESTAMPS)) return set_err(h, MOE_EINVAL, "MOE_TIMESTAMPS not set");
  if (!h->ran) return set_err(h, MOE_EINVAL, "no run yet");
  const int rc = sync_counters(h);
  if (rc) return rc;
  const int32_t recorded = std::min<int32_t>(h->last.copy_units, (int32_t)kMaxCopyRecords);
  int64_t need = 0;
  switch (which) {
    case MOE_RECORDS_PRODUCER: need = 2 * (int64_t)h->last.producer_grid * (int64_t)sizeof(WgRecord); break;
    case MOE_RECORDS_COPY: need = (int64_t)recorded * (int64_t)sizeof(CopyRecord); break;
    case MOE_RECORDS_SPAN: need = (int64_t)sizeof(moe_span_t); break;
    case MOE_RECORDS_TILES: need = (int64_t)h->last_tiles * (int64_t)sizeof(uint64_t); break;
    default: return set_err(h, MOE_EINVAL, "unknown record kind");
  }
  if (!dst) return need;
  if (bytes < need) return set_err(h, MOE_EINVAL, "destination too small");
  if (which == MOE_RECORDS_PRODUCER) {
    const size_t per = (size_t)h->last.producer_grid * sizeof(WgRecord);
    const size_t stride = (size_t)h->num_cus * h->producer_bpc;
    HIP_TRY(h, hipMemcpy(dst, h->wg_rec, per, hipMemcpyDeviceToHost));
    HIP_TRY(h, hipMemcpy((uint8_t*)dst + per, h->wg_rec + stride, per, hipMemcpyDeviceToHost));
  } else if (which == MOE_RECORDS_COPY) {
    if (need) HIP_TRY(h, hipMemcpy(dst, h->copy_rec, (size_t)need, hipMemcpyDeviceToHost));
  } else if (which == MOE_RECORDS_TILES) {
    if (need) HIP_TRY(h, hipMemcpy(dst, h->tile_ready, (size_t)need, hipMemcpyDeviceToHost));
  } else {
    moe_span_t sp{};
    sp.producer_start = h->last_span[0];
    sp.producer_end = h->last_span[1];
    sp.copy_units = h->last.copy_units;
    sp.copy_recorded = recorded;
    sp.producer_grid = h->last.producer_grid;
    memcpy(dst, &sp, sizeof sp);
  }
  return MOE_OK;
}

const char* moe_stage_last_error(moe_stage_t h) { return h ? h->err.c_str() : g_create_error.c_str(); }

int moe_stage_destroy(moe_stage_t h) {
  if (!h) return MOE_EINVAL;
  (void)hipDeviceSynchronize();
  for (auto& r : h->ring)
    for (auto& ev : r.ev)
      if (ev) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : {h->stage_free[0], h->stage_free[1], h->ev_fork, h->ev_join_c, h->ev_join_p,
                        h->ev_done})
    if (ev) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : h->autos.done)
    if (ev) (void)hipEventDestroy(ev);
  if (h->autos.stamps) (void)hipHostFree(h->autos.stamps);
  for (const auto& q : h->queues) {
    (void)hipStreamDestroy(q.cons);
    if (q.prod) (void)hipStreamDestroy(q.prod);
  }
  if (h->shared_prod) (void)hipStreamDestroy(h->shared_prod);
  for (void* p : {(void*)h->hws, (void*)h->y, (void*)h->flags, (void*)h->ctr, (void*)h->d_plan,
                  (void*)h->partials, (void*)h->arrivals, h->dev_ws, (void*)h->wg_rec, (void*)h->copy_rec,
                  (void*)h->tile_ready, (void*)h->simd_waves, (void*)h->abandoned, (void*)h->wcount})
    if (p) (void)hipFree(p);
  for (uint8_t* p : h->h_stage)
    if (p) (void)hipHostFree(p);
  delete h;
  return MOE_OK;
}

// ----------------------------------------------------------------- weighted combine
int moe_combine(const void* recv, int64_t recv_rows, int32_t hidden, const int32_t* slot,
                const float* gate, int64_t tokens, int32_t k, void* out, uint32_t* bad_slots,
                void* stream) {
  if (hidden <= 0 || k <= 0 || tokens < 0 || recv_rows < 0)
    return set_err(nullptr, MOE_EINVAL, "moe_combine: hidden and k must be positive, sizes >= 0");
  if (tokens == 0) return MOE_OK;
  if (!slot || !gate || !out || (recv_rows > 0 && !recv))
    return set_err(nullptr, MOE_EINVAL, "moe_combine: null pointer");
  if (hidden % 8 || hidden > 65536)
    return set_err(nullptr, MOE_EUNSUPPORTED, "moe_combine: hidden must be a multiple of 8, <= 65536");
  if (((uintptr_t)recv | (uintptr_t)out) & 15)
    return set_err(nullptr, MOE_EUNSUPPORTED, "moe_combine: recv and out must be 16-byte aligned");
  if (recv_rows > INT32_MAX)
    return set_err(nullptr, MOE_EUNSUPPORTED, "moe_combine: recv_rows must fit a 32-bit slot");
  CombineArgs a{};
  a.recv = (const uint16_t*)recv;
  a.slot = slot;
  a.gate = gate;
  a.out = (uint16_t*)out;
  a.bad_slots = bad_slots;
  a.recv_rows = recv_rows;
  a.tokens = tokens;
  a.k = k;
  a.H = hidden;
  const hipError_t e = launch_combine(a, (hipStream_t)stream);
  if (e != hipSuccess)
    return set_err(nullptr, MOE_EHIP, std::string("moe_combine launch: ") + hipGetErrorString(e));
  return MOE_OK;
}

// ----------------------------------------------------------------- no-allocation entry point
// Every workspace of moe_stage_run_serial_static lives in one fixed array per GPU.  In host code
// `scratch` only names the symbol: its device address comes from hipGetSymbolAddress, looked up
// once per device with that device current, and only that address is passed to kernels.
static __device__ __align__(256) uint8_t scratch[MOE_STATIC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch[kMaxDevices] = {};

int scratch_of_device(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return set_err(nullptr, MOE_EUNSUPPORTED, "device index beyond 64");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_err(nullptr, MOE_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch[dev] = (uint8_t*)p;
  }
  *out = g_scratch[dev];
  return MOE_OK;
}
}  // namespace

int moe_stage_run_serial_static(const moe_stage_config_t* cfg, const void* x, const int32_t* off,
                                const int32_t* src, const int32_t* slot, const void* w1, const void* w3,
                                const void* w2, void* const* ret, const int64_t* return_rows, void* stream) {
  int rc = check_config(cfg);
  if (rc) return set_err(nullptr, rc, "moe_stage_run_serial_static: invalid configuration");
  moe_stage_s h;  // a handle view over the scratch array: no streams, events or pinned staging
  h.cfg = *cfg;
  if (h.cfg.mid_segment_pieces == 0) h.cfg.mid_segment_pieces = 1;
  if (h.cfg.band_rows == 0) h.cfg.band_rows = 1;
  h.cfg.flags &= ~(uint32_t)MOE_KERNEL_TIMING;
  if (hipGetDevice(&h.device) != hipSuccess ||
      hipDeviceGetAttribute(&h.num_cus, hipDeviceAttributeMultiprocessorCount, h.device) != hipSuccess)
    return set_err(nullptr, MOE_EHIP, "moe_stage_run_serial_static: no HIP device");
  h.producer_bpc = producer_blocks_per_cu();
  const WsBytes wb = size_workspaces(&h);
  size_t off_b = 0;
  auto carve = [&](size_t bytes) {
    const size_t at = off_b;
    off_b = align256(off_b + bytes);
    return at;
  };
  const size_t o_hws = carve(wb.hws), o_y = carve(wb.y), o_arr = carve(wb.flags), o_part = carve(wb.partials),
               o_ctr = carve(sizeof(RunCounters)), o_plan = carve(h.plan_cap), o_ws = carve(wb.planner);
  if (off_b > (size_t)MOE_STATIC_SCRATCH_BYTES)
    return set_err(nullptr, MOE_ECAPACITY,
                   "moe_stage_run_serial_static: the configuration needs " + std::to_string(off_b) +
                       " bytes of workspace, more than the " + std::to_string((size_t)MOE_STATIC_SCRATCH_BYTES) +
                       " of the static array");
  uint8_t* base = nullptr;
  rc = scratch_of_device(h.device, &base);
  if (rc) return rc;
  h.hws = (uint16_t*)(base + o_hws);
  h.y = (uint16_t*)(base + o_y);
  h.arrivals = (uint32_t*)(base + o_arr);
  h.partials = wb.partials ? (float*)(base + o_part) : nullptr;
  h.ctr = (RunCounters*)(base + o_ctr);
  h.d_plan = base + o_plan;
  h.dev_ws = base + o_ws;
  h.ws = devplan_ws_carve(h.dev_ws, h.cfg.num_local_experts, h.cfg.num_ranks, h.cfg.max_rows, h.max_tile_rows,
                          h.down_per_row, h.max_lrows, h.max_items);
  rc = run_serial(&h, true, x, off, src, slot, w1, w3, w2, ret, return_rows, stream);
  if (rc) g_create_error = "moe_stage_run_serial_static: " + h.err;
  return rc;
}

// ----------------------------------------------------------------- plan inspection
struct moe_plan_s {
  Plan plan;
  int32_t band_rows = 0;
  int32_t queues[2 * (kXcds + 1)] = {};  // gate/up then down queue offsets
};

int moe_plan_build(const moe_stage_config_t* cfg, int64_t rows, const int32_t* off,
                   const int32_t* src, const int32_t* slot, const int64_t* return_rows,
                   int32_t overlapped, moe_plan_t* out) {
  if (!out) return MOE_EINVAL;
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc) return set_err(nullptr, rc, "invalid configuration");
  if (rows > cfg->max_rows) return set_err(nullptr, MOE_ECAPACITY, "rows > max_rows");
  moe_stage_config_t c = *cfg;
  if (c.band_rows == 0) c.band_rows = 1;
  if (off && off[c.num_local_experts] != rows)
    return set_err(nullptr, MOE_EROUTING, "expert_offsets[E_l] must equal rows");
  auto* p = new moe_plan_s();
  std::string msg;
  rc = build_plan(params_of(c, overlapped != 0), rows, off, src, slot, return_rows, &p->plan, &msg);
  if (rc) {
    delete p;
    return set_err(nullptr, rc, msg);
  }
  p->band_rows = overlapped ? c.band_rows : 1;
  std::copy(p->plan.gu_queue.begin(), p->plan.gu_queue.end(), p->queues);
  std::copy(p->plan.down_queue.begin(), p->plan.down_queue.end(), p->queues + kXcds + 1);
  *out = p;
  return MOE_OK;
}

int moe_plan_info(moe_plan_t p, moe_plan_info_t* o) {
  if (!p || !o) return MOE_EINVAL;
  const Plan& P = p->plan;
  o->n_tile_rows = (int32_t)P.tile_rows.size();
  o->n_items = (int32_t)P.items.size();
  o->n_gu_items = P.n_gu;
  o->n_down_items = P.n_down;
  o->n_segments = (int32_t)P.segs.size();
  o->n_groups = (int32_t)P.groups.size();
  o->gu_tiles_per_row = P.gu_per_row;
  o->down_tiles_per_row = P.down_per_row;
  o->tile_m = kTileM;
  o->band_rows = p->band_rows;
  o->split_k = P.tail_split;
  o->split_rows = P.n_split_rows;
  o->n_logical_rows = P.n_lrows();
  o->n_valid = P.n_valid;
  o->n_band_padding = P.n_band_pad;
  o->n_remote_rows = P.n_remote;
  return MOE_OK;
}

int64_t moe_plan_copy(moe_plan_t p, int32_t which, void* dst, int64_t bytes) {
  if (!p) return MOE_EINVAL;
  const Plan& P = p->plan;
  const void* src = nullptr;
  int64_t need = 0;
  switch (which) {
    case MOE_PLAN_TILE_ROWS: src = P.tile_rows.data(); need = sizeof(TileRow) * P.tile_rows.size(); break;
    case MOE_PLAN_ITEMS: src = P.items.data(); need = sizeof(uint32_t) * P.items.size(); break;
    case MOE_PLAN_ROW_X: src = P.row_x.data(); need = sizeof(int32_t) * P.row_x.size(); break;
    case MOE_PLAN_ROW_RANK: src = P.row_rank.data(); need = sizeof(int32_t) * P.row_rank.size(); break;
    case MOE_PLAN_ROW_SLOT: src = P.row_slot.data(); need = sizeof(int32_t) * P.row_slot.size(); break;
    case MOE_PLAN_SEGMENTS: src = P.segs.data(); need = sizeof(Segment) * P.segs.size(); break;
    case MOE_PLAN_GROUPS: src = P.groups.data(); need = sizeof(Group) * P.groups.size(); break;
    case MOE_PLAN_QUEUES: src = p->queues; need = sizeof p->queues; break;
    default: return MOE_EINVAL;
  }
  if (!dst) return need;
  if (bytes < need) return MOE_EINVAL;
  if (need) memcpy(dst, src, (size_t)need);
  return MOE_OK;
}

void moe_plan_free(moe_plan_t p) { delete p; }

}  // extern "C"
