/*
 * moe_stage.h -- C ABI of the MI355X (gfx950) MoE expert stage.
 *
 * One expert-parallel rank's expert stage with the return all-to-all
 * overlapped by tile-level signaling (paper Section 3: "Fine-grained
 * Computation-Communication Overlap via Tile-level Signaling and Scheduling
 * for Mixture-of-Experts").
 *
 * Problem (paper Section 2.1, steps 3-4, and Section 3.1): the rank owns
 * num_local_experts experts.  After the dispatch all-to-all it holds `rows`
 * routed token copies, expert-contiguous in `dispatched_x`.  For every row i
 * of local expert e it computes the SiLU-gated FFN
 *     y_i = W2_e * bf16( silu(W1_e x_i) (.) (W3_e x_i) ),  silu(g) = g/(1+e^-g)
 * and returns y_i to the rank the token came from, at the slot that rank
 * reserved for it:
 *     return_bufs[row_src_rank[i]][row_slot[i], :] = bf16_rne(y_i)
 * No other byte of the return buffers is written.  The outputs are not
 * gate-weighted (the weighted reduction happens on the owner, Section 2.1
 * step 5).  On one GPU, `return_bufs[r]` stands in for source rank r's receive
 * buffer; the transfer is a device copy inside local HBM.
 *
 * Layouts (all bf16 tensors row-major, 2-byte elements):
 *   dispatched_x  device  [rows, hidden]
 *   w1, w3        device  [num_local_experts, ffn, hidden]   (row f = output feature f)
 *   w2            device  [num_local_experts, hidden, ffn]
 *   return_bufs   host array of num_ranks device pointers; buffer r is
 *                 [return_rows[r], hidden]
 *   expert_offsets, row_src_rank, row_slot, return_rows: host arrays.
 *
 * Ownership: the caller owns every tensor and keeps it alive until the work
 * enqueued on `stream` has completed.  Host arrays may be freed as soon as a
 * call returns.  The handle owns its workspaces (intermediate activation,
 * staged output, flags, counters, plan buffers), the CU-masked streams and
 * events it creates; no device memory is allocated per run.  A handle is not
 * thread-safe and runs one stage at a time (a run waits for the previous
 * run's plan upload before reusing its staging memory).
 *
 * Errors: every call returns MOE_OK (0) or a negative code.  Validation runs
 * before anything is enqueued, so a failed call leaves the stream untouched.
 * moe_stage_last_error() describes the most recent failure of a handle.
 */
#ifndef MOE_STAGE_H
#define MOE_STAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_OK 0
#define MOE_EINVAL (-1)       /* null pointer, non-positive dimension, bad config value        */
#define MOE_EROUTING (-2)     /* offsets not 0..rows monotone, rank out of range, slot outside  */
                              /* its receive buffer, or two rows with the same (rank, slot)     */
#define MOE_ECAPACITY (-3)    /* rows > max_rows, or the plan exceeds the handle's workspaces   */
#define MOE_EHIP (-4)         /* a HIP runtime call failed (message names it)                  */
#define MOE_ETIMEOUT (-5)     /* a bounded device wait expired; sticky until the next query.
                                 A consumer wave whose flag wait expires hands its copy unit to
                                 the drain launch, which copies it after the producer, so an
                                 overlapped run's output is still complete; the run took at least
                                 watchdog_ms.  Only an expired wait of the drain itself (for the
                                 consumer's last wave) can leave rows uncopied               */
#define MOE_EUNSUPPORTED (-6) /* hidden/ffn not multiples of 64, hidden > 65536, max_rows >=
                                 2^24, max_rows * hidden * 2 > 2^32 - 1 (gathered rows are
                                 addressed with 32-bit offsets), a padded layout of more than
                                 2^24 rows, cu_split out of range                              */

/* Config flags */
#define MOE_LOCAL_DIRECT (1u << 0) /* overlapped run: rows whose source is self_rank are written
                                      by the producer epilogue straight into return_bufs[self];
                                      local tiles need no transfer (paper Section 3.2.3)       */
#define MOE_KERNEL_TIMING (1u << 1) /* record HIP events around each kernel of every run       */
#define MOE_POISON (1u << 2)        /* fill the staged output with NaN before each run, so a
                                       copy that races ahead of its data is detectable          */
#define MOE_TEST_NO_SIGNAL (1u << 3) /* testing aid: the producer raises no ready flags, so every
                                       consumer wait runs into watchdog_ms and the run reports
                                       MOE_ETIMEOUT; the kernels still exit normally and the drain
                                       launch copies every unit                                 */
#define MOE_TEST_CONSUMER_ONLY (1u << 6) /* measurement aid: moe_stage_run launches no producer
                                       work; the run's reset publishes every ready flag, so the
                                       consumer copies the staged output (whatever it holds) at
                                       the rate its cu_split compute units allow.  The receive
                                       buffers then hold no results                            */
#define MOE_TEST_PLAIN_COPY (1u << 9) /* measurement aid, with MOE_TEST_CONSUMER_ONLY and a
                                       host-built plan: instead of the consumer, a flat grid-stride
                                       copy of as many bytes as the segments hold (8 vectors in
                                       flight per lane, no flags, no copy units) from the staged
                                       output into return_bufs[0] runs on the same cu_split compute
                                       units: the copy ceiling of those compute units.  It overwrites
                                       return_bufs[0]                                            */
#define MOE_TEST_PLAN_NO_LDS (1u << 7) /* testing aid: the device planner keeps every table in
                                       device memory even where it fits in LDS, so the path taken
                                       by very large configurations is exercised on small ones */
#define MOE_SHARED_CUS (1u << 4)   /* overlapped run: the producer keeps every compute unit and
                                      the consumer, still confined to its cu_split units, runs
                                      beside producer workgroups there (a consumer workgroup's
                                      registers and LDS fit next to a producer workgroup's), so
                                      the partition costs the producer issue slots, not CUs    */
#define MOE_TIMESTAMPS (1u << 8)   /* measurement: every run records, in 100 MHz wall-clock ticks,
                                      when each producer workgroup started and ended and where it
                                      ran, and when each consumer copy unit began polling, saw its
                                      flags and finished its copy (moe_stage_records); the handle
                                      allocates the record buffers at create                   */
#define MOE_WRITE_COUNTS (1u << 10) /* testing aid: every run counts, per logical row of its plan,
                                      the 8-byte words stored into the receive buffers (by the down
                                      epilogue, the tail kernel, the consumer, the drain or the
                                      scatter), so a test can check that every routed row was
                                      written exactly once and nothing else
                                      (moe_stage_records, MOE_RECORDS_WRITES); the handle
                                      allocates the counters at create                          */
#define MOE_DIRECT_ALL (1u << 5)   /* ablation, serial runs only: the down epilogue writes every
                                      row straight to its slot in return_bufs and no scatter
                                      runs -- the bound of a stage with no consumer at all     */

typedef struct moe_stage_s* moe_stage_t;

typedef struct {
  int32_t hidden;            /* H, multiple of 64                                             */
  int32_t ffn;               /* F, multiple of 64                                             */
  int32_t num_local_experts; /* E_l >= 1                                                      */
  int32_t num_ranks;         /* R >= 1 source ranks                                           */
  int32_t self_rank;         /* 0 <= self_rank < R; rows from it are local (Section 3.2.1)    */
  int32_t max_rows;          /* capacity of one run (< 2^24, and max_rows * hidden * 2 bytes
                                < 4 GiB); sizes the workspaces                                */
  int32_t band_rows;         /* tb_M of the remote-owner-aligned layout (Section 3.2.1): each
                                remote owner group is padded to a multiple of it, so every
                                band of band_rows rows has one destination.  Power of two in
                                [1, 256]; 0 means 1, the default: readiness is tracked per
                                256-row tile row, so alignment would only add padding rows. */
  int32_t mid_segment_pieces; /* x of Section 3.3.2 (mgb in the evaluation): an owner group is
                                cut at 256-row tile-row boundaries into pieces; its first and
                                last pieces are one transfer segment each and middle segments
                                coalesce x pieces.  >= 1; 0 means 1.                         */
  uint32_t flags;            /* MOE_* flags above                                            */
  int32_t watchdog_ms;       /* bound on every device spin-wait; 0 = 2000 ms                  */
  int32_t down_split_k;      /* K parts per down-projection tile, 0..16 and <= ffn / 64.  A
                                split tile's parts each accumulate one contiguous K range in
                                fp32; the part that finishes last adds them in part order and
                                writes the tile.  Nonzero: every tile is split so.  0 (default):
                                only the tile rows holding the last, partly filled round of 256
                                down tiles are split, into as many parts as fill that round (at
                                most 16), so the launch's tail keeps every compute unit busy
                                for at most 256 fp32 partial tiles of traffic.  Which rows are
                                split depends on the routing only, never on the launch: with
                                band_rows = 1 the serial and overlapped runs of a routing give
                                identical bits.                                               */
} moe_stage_config_t;

/* Statistics of the most recent run (moe_stage_query). */
typedef struct {
  int64_t n_valid;          /* routed rows                                                   */
  int64_t n_logical_rows;   /* rows of the padded layout, incl. band and tile padding        */
  int64_t n_band_padding;   /* zero rows inserted at owner-group boundaries (Section 4.5)    */
  int64_t n_remote_rows;    /* rows whose source rank is not self_rank                      */
  int32_t n_tile_rows;      /* 256-row GEMM tile rows                                        */
  int32_t n_groups;         /* owner groups: (local expert, source rank) row groups          */
  int32_t n_gu_items;       /* gate/up tiles                                                */
  int32_t n_down_items;     /* down-projection work items: one per part of each tile (each
                               tile raises one ready flag when its last part is done)        */
  int32_t n_segments;       /* transfer segments issued by the consumer                      */
  int32_t producer_grid;    /* persistent producer workgroups launched                      */
  int32_t consumer_grid;    /* persistent consumer workgroups launched                      */
  int32_t consumer_cus;     /* compute units the consumer is confined to (cu_split rounded up
                               to a multiple of the XCD count; 0 for serial runs); with
                               MOE_SHARED_CUS the producer runs on them too                  */
  int32_t timeout;          /* 1 if a device wait hit the watchdog in any run since the last
                               query (sticky across runs)                                    */
  double plan_us;           /* host time to validate and build the plan (device-built plans:
                               to enqueue the planner)                                       */
  uint64_t poll_iters;      /* consumer flag-poll iterations summed over segments            */
  uint64_t wait_ticks;      /* consumer time spent waiting for flags (100 MHz ticks)         */
  int32_t gu_workgroups;    /* producer workgroups that claimed at least one tile in the last
                               run's gate/up launch (fewer than producer_grid means some
                               were not resident while the queue still held work)            */
  int32_t down_workgroups;  /* the same for the down-projection launch                       */
  int32_t split_k;          /* K parts of each split down-projection tile (1: none split)    */
  int32_t split_rows;       /* tile rows whose down-projection tiles are split               */
  int32_t auto_cu_split;    /* cu_split = 0 runs: the split the selector settled on, 0 while
                               it is still measuring candidates; -1 for other runs          */
  int32_t timeout_segment;  /* with timeout = 1: the lowest segment (ready order, as in
                               moe_stage_plan_copy(MOE_PLAN_SEGMENTS)) whose flag wait expired;
                               -1 otherwise                                                  */
  int32_t copy_units;       /* overlapped runs: consumer copy units (one wave each) the run's
                               segments were cut into; 0 for serial runs                     */
  int32_t reserved;
} moe_stage_stats_t;

/* Accumulated kernel times (MOE_KERNEL_TIMING), milliseconds, over runs since the last reset. */
typedef struct {
  int32_t runs;
  double stage_ms;     /* fork to join of each run (overlapped) or first to last kernel (serial) */
  double producer_ms;  /* producer: gate/up launch start to down launch end              */
  double gate_up_ms;   /* gate/up launch                                                 */
  double consumer_ms;  /* consumer kernel (overlapped runs)                              */
  double scatter_ms;   /* scatter kernel (serial runs)                                   */
  double plan_ms;      /* stage start until the plan is on the device and the counters are
                          reset: the upload of a host-built plan, or the device planner    */
} moe_stage_times_t;

/* Creates a handle and its device workspaces on the current HIP device. */
int moe_stage_create(const moe_stage_config_t* cfg, moe_stage_t* out);

/*
 * Overlapped stage (paper Section 3.3): builds the remote-owner-aligned row
 * layout, remote-first tile schedule and combine plan (Section 3.2, Algorithm
 * 1) on the host, then runs the persistent rank-wide producer (a gate/up launch,
 * then the down-projection launch) on all but `cu_split` compute units and a
 * persistent consumer on the others.  The down launch raises a ready flag per
 * finished tile; the consumer, released once the run's queues are reset,
 * copies each ready segment into return_bufs[destination].  The
 * work is ordered after prior work on `stream` (a hipStream_t; NULL = null
 * stream) and later work on `stream` sees the results.  The consumer runs on a
 * CU-masked stream of the handle; the producer runs on another one, or directly
 * on `stream` under MOE_SHARED_CUS when `stream` is not the legacy null stream
 * (whose launches would wait for the polling consumer).  A drain launch follows
 * the producer in its stream: it copies the units the consumer has not claimed
 * when the producer ends, on the producer's compute units, and waits (bounded by
 * the watchdog) until every consumer wave has finished, so the stage ends with it.
 *
 * cu_split: compute units for the consumer, 1 <= cu_split <= CUs - XCDs, or 0 to let the
 * handle choose (a runtime-adaptive selector, the future work of paper Sections 4.3.4
 * and 6): it measures
 * the stage time of its own runs at consumer splits of 32, 64, 128 and 248 CUs under
 * MOE_SHARED_CUS (8, 16, 32 and 64 without it), one after another and each with only its own
 * CU-masked queue alive, four finished runs each (the first a warm-up), skipping any above
 * CUs - XCDs, then keeps the one with the lowest median (stats: auto_cu_split).
 * Results do not depend on the split.  Workgroups
 * are dealt round-robin over the XCDs (8 on MI355X) and a CU-masked queue must own
 * CUs on each of them, so the split is rounded up to a multiple of the XCD count
 * (the stats report the effective value); the producer gets every other CU, or every
 * CU under MOE_SHARED_CUS.  Beside the producer (MOE_SHARED_CUS) the consumer runs about
 * 256 waves spread over its cu_split CUs (8 per CU on 32 CUs, 1 per CU on 248); on CUs of
 * its own it runs 16 waves per CU.
 */
int moe_stage_run(moe_stage_t h, const void* dispatched_x, const int32_t* expert_offsets,
                  const int32_t* row_src_rank, const int32_t* row_slot, const void* w1,
                  const void* w3, const void* w2, void* const* return_bufs,
                  const int64_t* return_rows, int32_t cu_split, void* stream);

/*
 * Non-overlapped baseline (paper Section 4.1.3: expert compute, then the
 * whole return transfer): the same producer on all compute units with no
 * signaling, then one scatter kernel that copies every routed row to its slot.
 */
int moe_stage_run_serial(moe_stage_t h, const void* dispatched_x, const int32_t* expert_offsets,
                         const int32_t* row_src_rank, const int32_t* row_slot, const void* w1,
                         const void* w3, const void* w2, void* const* return_bufs,
                         const int64_t* return_rows, void* stream);

/*
 * The same two runs with the plan built on the GPU (paper Section 3.2, Algorithm 1: layout,
 * schedule and combine plan; Section 3.3.2: segments) from routing already in device memory:
 *   expert_offsets  device int32 [num_local_experts + 1]
 *   row_src_rank    device int32 [rows]  (rows = expert_offsets[num_local_experts])
 *   row_slot        device int32 [rows]
 * return_bufs and return_rows stay host arrays (the receive buffers' places and sizes).  A few
 * small kernels on `stream` validate the routing and write the plan tables; the producer and
 * consumer read their counts from device memory, so nothing waits for the host between the
 * routing and the stage.  The tables are identical to those the host builder makes for the same
 * routing (moe_stage_plan_copy reads them back).
 *
 * Precondition: the order a dispatch all-to-all delivers rows in -- within each expert, the
 * rows of one source rank are contiguous and their slots ascend (source ranks may come in any
 * order).  The host-planned entry points accept any order.
 *
 * Errors: argument errors (null pointers, negative return_rows) return at once and enqueue
 * nothing.  Routing errors (the host path's MOE_EROUTING and MOE_ECAPACITY cases, and routing
 * that breaks the precondition) are found on the device: the run then does no work, writes
 * nothing to return_bufs, and the next moe_stage_query returns the code (the message names the
 * first offending row).  Workspaces are sized at create; no run allocates memory.
 */
int moe_stage_run_devplan(moe_stage_t h, const void* dispatched_x, const int32_t* expert_offsets,
                          const int32_t* row_src_rank, const int32_t* row_slot, const void* w1,
                          const void* w3, const void* w2, void* const* return_bufs,
                          const int64_t* return_rows, int32_t cu_split, void* stream);
int moe_stage_run_serial_devplan(moe_stage_t h, const void* dispatched_x,
                                 const int32_t* expert_offsets, const int32_t* row_src_rank,
                                 const int32_t* row_slot, const void* w1, const void* w3,
                                 const void* w2, void* const* return_bufs,
                                 const int64_t* return_rows, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the non-overlapped run of
 * moe_stage_run_serial_devplan without a handle.  Arguments are those of
 * moe_stage_run_serial_devplan with the configuration in place of the handle (routing in device
 * memory, in the order a dispatch all-to-all delivers it).  Every workspace (activations, staged
 * output, K-part partials, counters, plan tables, planner scratch) lives in one fixed device
 * array of MOE_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on until the
 * process ends; the call allocates nothing: no hipMalloc, hipFree, stream, event or pinned host
 * memory.  It enqueues on `stream` (a hipStream_t; NULL = null stream) and returns; the two
 * receive-buffer tables go up with hipMemcpyAsync from the caller's host arrays.  Every call on
 * a GPU shares that GPU's array and leaves its contents behind (each run's kernels reset what
 * must start at zero): calls that overlap on one GPU -- on different streams, or from different
 * threads -- race and must not be made.  Errors: MOE_ECAPACITY when the configuration's
 * workspaces (sized by max_rows as for moe_stage_create) exceed the array, the other codes as
 * for moe_stage_run_serial_devplan; routing errors found on the device leave return_bufs
 * untouched.  The message is moe_stage_last_error(NULL).  Results are bit-identical to
 * moe_stage_run_serial_devplan on a handle of the same configuration.
 */
#define MOE_STATIC_SCRATCH_BYTES (64u * 1024u * 1024u)
int moe_stage_run_serial_static(const moe_stage_config_t* cfg, const void* dispatched_x,
                                const int32_t* expert_offsets, const int32_t* row_src_rank,
                                const int32_t* row_slot, const void* w1, const void* w3, const void* w2,
                                void* const* return_bufs, const int64_t* return_rows, void* stream);

/* Statistics of the last run; synchronizes with it.  Returns MOE_ETIMEOUT (once) if any run
 * since the previous query had a device wait expire; its outputs are then incomplete.  After a
 * device-planned run it returns the planner's routing error (once), if any; its plan counts
 * come from the device.  plan_us is the host time spent building (or enqueueing) the plan. */
int moe_stage_query(moe_stage_t h, moe_stage_stats_t* out);

/* Kernel times accumulated since the last reset (needs MOE_KERNEL_TIMING); synchronizes. */
int moe_stage_times(moe_stage_t h, int32_t reset, moe_stage_times_t* out);

/*
 * Timing and placement records of the last run of a handle created with MOE_TIMESTAMPS
 * (measurement of the overlap of paper Section 4.2.2 and of the compute-unit partition of
 * Section 3.3.3).  Times are the GPU's 100 MHz wall clock.  `which` selects:
 *   MOE_RECORDS_PRODUCER  moe_wg_record_t[2 * producer_grid]: the gate/up launch's workgroups
 *                         (index = workgroup), then the down launch's;
 *   MOE_RECORDS_COPY      moe_copy_record_t[min(copy_units, 2^18)]: one per consumer copy unit
 *                         (overlapped runs; index = unit);
 *   MOE_RECORDS_SPAN      moe_span_t: the producer's span (first gate/up workgroup start, last
 *                         down or tail workgroup end) and the unit counts;
 *   MOE_RECORDS_TILES     uint64_t[tile rows * down tiles per row]: when each down tile's ready
 *                         flag was raised (index = tile row * down tiles per row + column tile;
 *                         0 = no flag this run: local-only tile rows, serial runs).
 *   MOE_RECORDS_WRITES    uint32_t[the handle's logical-row capacity]: with MOE_WRITE_COUNTS
 *                         instead of MOE_TIMESTAMPS, the 8-byte words the last run stored into the
 *                         receive buffers for each logical row of its plan (hidden / 4 for every
 *                         routed row, 0 for padding rows and past the plan's rows).
 * With dst == NULL returns the bytes needed; else copies them (bytes must be at least that) and
 * returns MOE_OK.  Synchronizes with the last run.  MOE_EINVAL without MOE_TIMESTAMPS (or, for
 * MOE_RECORDS_WRITES, MOE_WRITE_COUNTS) or without a run.
 */
#define MOE_RECORDS_PRODUCER 0
#define MOE_RECORDS_COPY 1
#define MOE_RECORDS_SPAN 2
#define MOE_RECORDS_TILES 3
#define MOE_RECORDS_WRITES 4
typedef struct {
  uint32_t hw_id;   /* HW_ID register of the workgroup's first wave: wave slot [3:0], SIMD
                       [5:4], compute unit [11:8], shader array [12], shader engine [15:13]   */
  uint32_t xcc_id;  /* XCD (accelerator die)                                               */
  int32_t launch;   /* 0 gate/up, 1 down                                                   */
  int32_t items;    /* work items the workgroup ran                                        */
  uint64_t t_start, t_end;
  uint64_t cycles;  /* shader clock cycles that passed between t_start and t_end: the
                       workgroup's mean clock is cycles / (t_end - t_start) x 100 MHz          */
} moe_wg_record_t;
typedef struct {
  int32_t segment;  /* segment index (ready order)                                         */
  int32_t part;     /* copy unit within the segment                                        */
  uint32_t hw_id;   /* HW_ID register of the copying wave (fields as above)                */
  uint32_t xcc_id;
  uint64_t t_poll;  /* the wave starts polling the segment's ready flags                   */
  uint64_t t_ready; /* every flag seen and acquired: the copy starts                       */
  uint64_t t_done;  /* the unit's stores have completed                                    */
  int32_t source;   /* 0: copied by the consumer launch; 1: by the drain launch that follows
                       the producer (units still unclaimed when the producer ended)          */
  int32_t reserved;
} moe_copy_record_t;
typedef struct {
  uint64_t producer_start, producer_end;
  int32_t copy_units;     /* units of the last run (0 for serial runs)                      */
  int32_t copy_recorded;  /* of them recorded                                               */
  int32_t producer_grid;  /* workgroups per producer launch                                 */
  int32_t reserved;
} moe_span_t;
int64_t moe_stage_records(moe_stage_t h, int32_t which, void* dst, int64_t bytes);

/* Human-readable description of the handle's last error ("" if none).  Valid until the next call. */
const char* moe_stage_last_error(moe_stage_t h);

/* Waits for outstanding work, then frees the handle and everything it owns. */
int moe_stage_destroy(moe_stage_t h);

/*
 * Weighted combine on a source rank (paper Section 2.1, step 5: after the
 * return transfer, the rank that sent a token reduces the token's k expert
 * outputs, weighted by the router's gate values).  Stateless, needs no handle:
 *
 *   out[t, :] = bf16_rne( sum_{j = 0..k-1} gate[t*k + j] * recv[slot[t*k + j], :] )
 *
 * summed in fp32 in ascending j, each term a rounded fp32 product followed by a
 * rounded fp32 add (no fused multiply-add), starting from +0.
 *   recv       device, [recv_rows, hidden] bf16 row-major: this rank's receive
 *              buffer, as filled by every owner's moe_stage_run / _run_serial;
 *   slot       device, [tokens, k] int32: receive slot of choice j of token t;
 *   gate       device, [tokens, k] fp32 gate weights;
 *   out        device, [tokens, hidden] bf16 row-major, written in full;
 *   bad_slots  optional device uint32: incremented once per slot outside
 *              [0, recv_rows) (the term is skipped and the output still written);
 *              the caller zeroes it.
 * hidden must be a multiple of 8 and <= 65536, recv and out 16-byte aligned.  The
 * buffers stay owned by the caller; the call only enqueues a kernel on `stream`
 * (a hipStream_t; NULL = null stream) and returns without waiting.  Errors
 * (MOE_EINVAL, MOE_EUNSUPPORTED, MOE_EHIP) enqueue nothing; the message is
 * moe_stage_last_error(NULL).
 */
int moe_combine(const void* recv, int64_t recv_rows, int32_t hidden, const int32_t* slot,
                const float* gate, int64_t tokens, int32_t k, void* out, uint32_t* bad_slots,
                void* stream);

/* ---------------------------------------------------------------------------
 * Host-only plan inspection (no GPU needed).  Builds exactly the plan that
 * moe_stage_run would use for these arguments and lets the caller read its
 * tables, so the layout, schedule and combine plan can be checked on a CPU.
 * ------------------------------------------------------------------------- */
typedef struct moe_plan_s* moe_plan_t;

typedef struct {
  int32_t n_tile_rows, n_items, n_gu_items, n_down_items, n_segments, n_groups;
  int32_t gu_tiles_per_row;   /* gate/up tiles per tile row (ffn / 128, rounded up)          */
  int32_t down_tiles_per_row; /* down tiles per tile row (hidden / 256, rounded up)          */
  int32_t tile_m, band_rows;
  int32_t split_k;            /* K parts of each split down tile (1: none split)             */
  int32_t split_rows;         /* tile rows whose down tiles are split                         */
  int64_t n_logical_rows, n_valid, n_band_padding, n_remote_rows;
} moe_plan_info_t;

/* Tables readable with moe_plan_copy:
 *   MOE_PLAN_TILE_ROWS  int32 [n_tile_rows][6]: expert, first logical row, valid rows,
 *                       has_remote, K parts of its down tiles, first fp32 partial tile (-1)
 *   MOE_PLAN_ITEMS      uint32 [n_items]: bit 31 = down tile, bits 30..12 tile row; gate/up
 *                       items: bits 11..0 column tile; down items: bits 11..4 column tile,
 *                       bits 3..0 K part; all gate/up tiles (first launch) precede all down
 *                       items, and each launch's items are its 8 per-XCD queues in turn
 *   MOE_PLAN_ROW_X      int32 [n_logical_rows]: dispatched_x row feeding each logical row
 *                       (padding rows repeat a valid row of the same expert)
 *   MOE_PLAN_ROW_RANK   int32 [n_logical_rows]: source rank, -1 for padding
 *   MOE_PLAN_ROW_SLOT   int32 [n_logical_rows]: receive slot, -1 for padding
 *   MOE_PLAN_SEGMENTS   int32 [n_segments][8]: dst rank, rows, first logical row, first slot,
 *                       first flag, flag count, latest queue position (within its XCD queue)
 *                       of the down items it waits for, tile-row pieces of its group it covers
 *   MOE_PLAN_GROUPS     int32 [n_groups][4]: expert, first logical row, rows, source rank
 *   MOE_PLAN_QUEUES     int32 [2][9]: per launch (gate/up, then down), queue x of the XCD x
 *                       workgroups is that launch's items [q[x], q[x+1]); a workgroup whose
 *                       queue is empty continues with the following queues.  The queues are
 *                       the launch's item sequence in schedule order dealt round-robin in
 *                       chunks of 32 items (queue x holds chunks x, x + 8, ...)
 */
#define MOE_PLAN_TILE_ROWS 0
#define MOE_PLAN_ITEMS 1
#define MOE_PLAN_ROW_X 2
#define MOE_PLAN_ROW_RANK 3
#define MOE_PLAN_ROW_SLOT 4
#define MOE_PLAN_SEGMENTS 5
#define MOE_PLAN_GROUPS 6
#define MOE_PLAN_QUEUES 7

/* `overlapped` selects the plan of moe_stage_run (1) or moe_stage_run_serial (0). */
int moe_plan_build(const moe_stage_config_t* cfg, int64_t rows, const int32_t* expert_offsets,
                   const int32_t* row_src_rank, const int32_t* row_slot,
                   const int64_t* return_rows, int32_t overlapped, moe_plan_t* out);
int moe_plan_info(moe_plan_t p, moe_plan_info_t* out);
/* Copies table `which` into `dst` (host memory of at least `bytes`); returns bytes needed if
 * dst is NULL, else MOE_OK or MOE_EINVAL when bytes is too small. */
int64_t moe_plan_copy(moe_plan_t p, int32_t which, void* dst, int64_t bytes);
void moe_plan_free(moe_plan_t p);

/* The plan of a handle's last run (host- or device-built), read back from device memory in
 * the layouts above; both synchronize with that run.  MOE_EINVAL before the first run. */
int moe_stage_plan_info(moe_stage_t h, moe_plan_info_t* out);
int64_t moe_stage_plan_copy(moe_stage_t h, int32_t which, void* dst, int64_t bytes);

#ifdef __cplusplus
}
#endif
#endif /* MOE_STAGE_H */
