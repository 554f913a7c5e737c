// plan_device.hip -- the plan of one expert-stage run, built on the GPU (gfx950).
//
// The host builder (plan.cpp) walks the routing serially.  Here the same plan -- layout,
// schedule, work queues and combine plan (paper Section 3.2, Algorithm 1; segment
// composition of Section 3.3.2) -- comes from four kernels in stream order:
//
//   rows    grid over dispatched rows: validates the routing and records, per (expert, source
//           rank), the run of rows it occupies (a histogram by run bounds: the dispatch order
//           keeps each source rank's rows of an expert contiguous); a hash set of (rank, slot)
//           catches duplicates.
//   layout  one workgroup: per expert, the owner groups in rank order (remote ranks ascending,
//           then the local rank) with band padding, prefix sums into tile rows and groups, the
//           remote-first schedule (experts by remote band count, descending), the tail split,
//           each schedule position's row group and the per-XCD queue bounds -- all closed forms
//           of the host's greedy walks.
//   fill    grid: every work item straight to its queue slot; the row tables; per tile row, the
//           logical rows where transfer segments start and end, compacted into short lists.
//   segs    one workgroup: prefix sums of the per-tile-row counts pair the k-th start with the
//           k-th end; each segment's fields and ready position; then a stable counting sort by
//           ready position (the order the consumer claims them in).
//
// Every step reproduces the host's tables exactly for routing in dispatch order.  The
// single-workgroup kernels keep their tables in LDS when they fit, and need only workgroup
// barriers between phases: every wave of a workgroup shares one compute unit, whose vector
// cache is coherent for it, so no device-scope fence (an L2 write-back on this chip) is paid.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/moe_stage.h"
#include "plan_device.hpp"

namespace moe {
namespace {

constexpr int kWg = 1024;   // threads of the single-workgroup kernels
constexpr int kBlk = 256;   // threads of the grid kernels; one logical row each in a tile row
static_assert(kBlk == kTileM, "the fill and segment kernels give each tile row one workgroup");

__device__ __forceinline__ int32_t round_up_i(int32_t v, int32_t m) { return (v + m - 1) / m * m; }

// Inclusive prefix sum of x over a workgroup of kThreads threads: a shuffle scan within each
// 64-lane wave, then one over the wave totals.  `sh` holds kThreads / 64 ints of LDS; *total
// gets the workgroup's sum.  Every thread must call it.
template <int kThreads>
__device__ __forceinline__ int32_t wg_incl_scan(int32_t x, int32_t* sh, int32_t* total) {
  constexpr int kWaves = kThreads / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) sh[wv] = x;
  __syncthreads();
  if (wv == 0) {
    int32_t t = lane < kWaves ? sh[lane] : 0;
    for (int d = 1; d < kWaves; d <<= 1) {
      const int32_t y = __shfl_up(t, d, 64);
      if (lane >= d) t += y;
    }
    if (lane < kWaves) sh[lane] = t;
  }
  __syncthreads();
  const int32_t r = x + (wv ? sh[wv - 1] : 0);
  *total = sh[kWaves - 1];
  __syncthreads();  // sh may be reused at once
  return r;
}

// Exclusive prefix sum of v[0, n) in place by one workgroup of kThreads threads (v in LDS or
// global memory); returns the total, the same in every thread.
// kAtomicIn: v was last written by atomics; read it with device-coherent loads.
template <int kThreads, bool kAtomicIn = false>
__device__ int32_t wg_scan(int32_t* v, int32_t n, int32_t* sh) {
  const int tid = threadIdx.x;
  int32_t carry = 0;
  for (int32_t c0 = 0; c0 < n; c0 += kThreads) {
    const int32_t i = c0 + tid;
    int32_t x = 0;
    if (i < n) x = kAtomicIn ? __hip_atomic_load(&v[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : v[i];
    int32_t tot;
    const int32_t incl = wg_incl_scan<kThreads>(x, sh, &tot);
    if (i < n) v[i] = carry + incl - x;
    carry += tot;
  }
  __syncthreads();
  return carry;
}

// Largest e in [0, n) with begin[e] <= i, for non-decreasing begin[] with begin[0] <= i: the
// expert (or owner) whose range holds i when empty ranges share their successor's start.
__device__ __forceinline__ int32_t range_of(const int32_t* begin, int32_t n, int32_t i) {
  int32_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (begin[mid] <= i)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Inserts key into the open-addressing set; true if it was there already.  The set holds at
// most half its capacity, so a free entry is always found.
__device__ bool seen_insert(uint64_t* set, int64_t cap, uint64_t key) {
  uint64_t h = key * 0x9E3779B97F4A7C15ull;
  h ^= h >> 29;
  const uint64_t mask = (uint64_t)cap - 1;
  h &= mask;
  for (int64_t probe = 0; probe < cap; ++probe) {
    const unsigned long long prev = atomicCAS((unsigned long long*)&set[h], ~0ull, (unsigned long long)key);
    if (prev == ~0ull) return false;
    if (prev == key) return true;
    h = (h + 1) & mask;
  }
  return true;
}

// Rank order of the layout (Section 3.2.1): remote ranks ascending, the local rank last.
__device__ __forceinline__ int32_t rank_at(int32_t j, int32_t R, int32_t self) {
  return j == R - 1 ? self : (j < self ? j : j + 1);
}

__device__ void write_empty(const DevPlanArgs& a) {
  if (threadIdx.x < 2 * (kXcds + 1)) a.queues[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    PlanHeader* H = a.hdr;
    H->n_tile_rows = H->n_groups = H->n_gu = H->n_down = H->n_segs = 0;
    H->tail_split = 1;
    H->n_split_rows = H->n_partials = H->down_qmax = H->n_groups_all = 0;
    H->n_valid = H->n_lrows = H->n_band_pad = H->n_remote = 0;
  }
}

// ---------------------------------------------------------------------------------------------
// rows: validation and the per-(expert, rank) runs.
// ---------------------------------------------------------------------------------------------
constexpr int kLdsOffsets = 4096;  // expert offsets staged in LDS up to this many experts
constexpr int kLdsRanks = 1024;    // receive-buffer sizes staged in LDS up to this many ranks

__global__ __launch_bounds__(kBlk) void plan_rows_kernel(DevPlanArgs a) {
  __shared__ int32_t off_lds[kLdsOffsets + 1];
  __shared__ int64_t rr_lds[kLdsRanks];
  const bool in_lds = !a.no_lds && a.E_l <= kLdsOffsets;
  const bool rr_in_lds = !a.no_lds && a.R <= kLdsRanks;
  const int32_t* off = in_lds ? off_lds : a.off;
  const int64_t* rrows = rr_in_lds ? rr_lds : a.return_rows;
  int bad_off = 0;
  for (int e = threadIdx.x; e <= a.E_l; e += kBlk) {
    const int32_t v = a.off[e];
    if (in_lds) off_lds[e] = v;
    if (e < a.E_l) bad_off |= v > a.off[e + 1];
  }
  if (rr_in_lds)
    for (int r = threadIdx.x; r < a.R; r += kBlk) rr_lds[r] = a.return_rows[r];
  bad_off = __syncthreads_or(bad_off);
  const int32_t rows = off[a.E_l];
  int32_t code = 0;
  if (rows < 0)
    code = MOE_EROUTING;
  else if (rows > a.max_rows)
    code = MOE_ECAPACITY;
  else if (off[0] != 0 || bad_off)
    code = MOE_EROUTING;
  if (code) {
    if (blockIdx.x == 0 && threadIdx.x == 0) a.hdr->status = code;
    return;
  }
  const int32_t R = a.R;
  for (int32_t i = blockIdx.x * kBlk + threadIdx.x; i < rows; i += gridDim.x * kBlk) {
    // Neighbours are loaded with the row itself (clamped indices), so one round trip serves all.
    const int32_t ip = i > 0 ? i - 1 : i, in = i + 1 < rows ? i + 1 : i;
    const int32_t r = a.src[i], s = a.slot[i], r_prev = a.src[ip], r_next = a.src[in], s_prev = a.slot[ip];
    const int32_t e = range_of(off, a.E_l, i);
    const int32_t lo = off[e], hi = off[e + 1];
    bool bad = r < 0 || r >= R || s < 0 || (int64_t)s >= rrows[r];
    if (!bad) {
      const bool first = i == lo || r_prev != r;
      const bool last = i == hi - 1 || r_next != r;
      if (!first && s_prev >= s) bad = true;  // slots ascend within a rank's run
      if (first && atomicCAS(&a.ws.run_lo[e * R + r], -1, i) != -1) bad = true;  // a second run
      if (last) a.ws.run_hi[e * R + r] = i + 1;
      if (seen_insert(a.ws.seen, a.ws.seen_cap, ((uint64_t)r << 32) | (uint32_t)s)) bad = true;
    }
    if (bad) {
      atomicMin(&a.hdr->bad_row, i);
      a.hdr->status = MOE_EROUTING;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// layout: one workgroup.
// ---------------------------------------------------------------------------------------------
constexpr int kLdsExperts = 1024;  // per-expert tables in LDS up to this many experts
constexpr int kLdsGroups = 2048;   // group table in LDS up to this many (expert, rank) pairs

__global__ __launch_bounds__(kWg) void plan_layout_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kWg];
  __shared__ int32_t ex_lds[7 * kLdsExperts];
  __shared__ int32_t g_lds[3 * kLdsGroups];
  __shared__ unsigned long long s_pad, s_remote;
  PlanHeader* H = a.hdr;
  const int tid = threadIdx.x;
  if (H->status != 0) {
    write_empty(a);
    return;
  }
  if (tid == 0) s_pad = s_remote = 0;
  const int32_t E_l = a.E_l, R = a.R, self = a.self;
  const int32_t tb = a.overlapped ? a.tb : 1;
  const DevPlanWs& w = a.ws;
  // Per-expert and group tables: LDS when they fit, else the global scratch (generic pointers,
  // so the code is the same either way).
  const bool ex_in_lds = !a.no_lds && E_l <= kLdsExperts;
  int32_t* ex_ntr = ex_in_lds ? ex_lds : w.ex_ntr;
  int32_t* ex_ng = ex_in_lds ? ex_lds + kLdsExperts : w.ex_ng;
  int32_t* ex_hr = ex_in_lds ? ex_lds + 2 * kLdsExperts : w.ex_hr;
  int32_t* ex_bands = ex_in_lds ? ex_lds + 3 * kLdsExperts : w.ex_bands;
  int32_t* ex_roff = ex_in_lds ? ex_lds + 4 * kLdsExperts : w.ex_roff;
  int32_t* ex_loff = ex_in_lds ? ex_lds + 5 * kLdsExperts : w.ex_loff;
  int32_t* tmp = ex_in_lds ? ex_lds + 6 * kLdsExperts : w.tmp;
  const bool g_in_lds = !a.no_lds && (int64_t)E_l * R <= kLdsGroups;
  int32_t* gl_lrow0 = g_in_lds ? g_lds : w.g_lrow0;
  int32_t* gl_rows = g_in_lds ? g_lds + kLdsGroups : w.g_rows;
  int32_t* gl_dst = g_in_lds ? g_lds + 2 * kLdsGroups : w.g_dst;
  __syncthreads();

  // Per expert: its owner groups in rank order, band padding after each remote group (only
  // in the overlapped layout), its extent in tile rows, and its schedule key.
  for (int32_t e = tid; e < E_l; e += kWg) {
    int32_t pos = 0, bands = 0, ng = 0, remote_end = 0;
    int64_t pad_e = 0, remote_e = 0;
    for (int32_t j = 0; j < R; ++j) {
      const int32_t r = rank_at(j, R, self);
      const int32_t lo = w.run_lo[e * R + r];
      if (lo < 0) continue;
      const int32_t n = w.run_hi[e * R + r] - lo;
      ++ng;
      pos += n;
      if (r != self) {
        remote_e += n;
        bands += (n + tb - 1) / tb;
        remote_end = pos;
        if (a.overlapped) {
          const int32_t p = round_up_i(pos, tb) - pos;
          pad_e += p;
          pos += p;
        }
      }
    }
    ex_ntr[e] = round_up_i(pos, kTileM) / kTileM;
    // Remote rows precede local ones, and padding never fills a whole tile row, so the tile
    // rows holding remote rows are the expert's first ones, through the last remote row's.
    ex_hr[e] = remote_end > 0 ? (remote_end - 1) / kTileM + 1 : 0;
    ex_bands[e] = bands;
    ex_ng[e] = ng;
    if (pad_e) atomicAdd(&s_pad, (unsigned long long)pad_e);
    if (remote_e) atomicAdd(&s_remote, (unsigned long long)remote_e);
  }
  __syncthreads();
  const int32_t n_tr = wg_scan<kWg>(ex_ntr, E_l, sh);   // ex_ntr: first tile row of each expert
  const int32_t n_grp = wg_scan<kWg>(ex_ng, E_l, sh);   // ex_ng: first group of each expert
  if (n_tr > a.max_tile_rows || n_tr >= kMaxTileRows) {
    if (tid == 0) H->status = MOE_ECAPACITY;
    write_empty(a);
    return;
  }

  // Remote-first schedule (Section 3.2.2): experts by remote band count, descending, ties by
  // id, each contributing its remote tile rows; then every expert's local-only tile rows in
  // expert order.  tmp[rank] takes each expert's remote tile-row count for the prefix sum.
  for (int32_t e = tid; e < E_l; e += kWg) {
    const int32_t b = ex_bands[e];
    int32_t rank = 0;
    for (int32_t f = 0; f < E_l; ++f) {
      const int32_t c = ex_bands[f];
      rank += (c > b) || (c == b && f < e);
    }
    tmp[rank] = ex_hr[e];
    ex_roff[e] = rank;
    const int32_t ntr_e = (e + 1 < E_l ? ex_ntr[e + 1] : n_tr) - ex_ntr[e];
    ex_loff[e] = ntr_e - ex_hr[e];
  }
  __syncthreads();
  const int32_t n_hr = wg_scan<kWg>(tmp, E_l, sh);
  wg_scan<kWg>(ex_loff, E_l, sh);  // + n_hr: first local-only position of each expert
  for (int32_t e = tid; e < E_l; e += kWg) ex_roff[e] = tmp[ex_roff[e]];

  // Owner groups with their places in the padded layout (the fill kernel reads the global
  // copies of the group table and of each expert's first group).
  for (int32_t e = tid; e < E_l; e += kWg) {
    const int32_t base = ex_ntr[e] * kTileM;
    int32_t g = ex_ng[e], pos = base;
    if (ex_in_lds) w.ex_ng[e] = g;
    for (int32_t j = 0; j < R; ++j) {
      const int32_t r = rank_at(j, R, self);
      const int32_t lo = w.run_lo[e * R + r];
      if (lo < 0) continue;
      const int32_t n = w.run_hi[e * R + r] - lo;
      w.g_lrow0[g] = pos;
      w.g_rows[g] = n;
      w.g_dst[g] = r;
      w.g_src0[g] = lo;
      if (g_in_lds) {
        gl_lrow0[g] = pos;
        gl_rows[g] = n;
        gl_dst[g] = r;
      }
      if (a.overlapped) a.groups[g] = Group{e, pos, n, r};
      ++g;
      pos += n;
      if (a.overlapped && r != self) pos = base + round_up_i(pos - base, tb);
    }
  }

  // K parts of the down tiles: an explicit split_k splits every tile row; by default the tile
  // rows holding the last, partly filled round of kRoundTiles down tiles are split into as
  // many parts as fill that round.
  const int32_t dpr = a.down_per_row, gpr = a.gu_per_row;
  int32_t S = 1, n_split = 0;
  if (a.split_k > 0) {
    S = a.split_k;
    n_split = a.split_k > 1 ? n_tr : 0;
  } else if (n_tr > 0) {
    const int64_t rem = ((int64_t)n_tr * dpr) % kRoundTiles;
    if (rem > 0) {
      const int32_t rows = (int32_t)((rem + dpr - 1) / dpr);
      const int64_t s = kRoundTiles / ((int64_t)rows * dpr);
      const int32_t s2 = (int32_t)min(min(s, (int64_t)kMaxSplitK), (int64_t)a.nk);
      if (s2 > 1) {
        S = s2;
        n_split = rows;
      }
    }
  }
  const int32_t n_whole = n_tr - n_split;
  __syncthreads();

  // Tile rows, their schedule positions and row groups.  A position's class run [cs, ce) is
  // its expert's remote (or local-only) tile rows, consecutive in the schedule; the host's
  // greedy grouping in closed form: within the run, clipped to the range [a0, a1) being
  // grouped, groups of g positions start at max(cs, a0).
  const int32_t ggu = max(a.gu_group, 1), gdn = max(a.down_group, 1);
  for (int32_t t = tid; t < n_tr; t += kWg) {
    const int32_t e = range_of(ex_ntr, E_l, t);
    const int32_t j = t - ex_ntr[e], hr = ex_hr[e];
    const int32_t ntr_e = (e + 1 < E_l ? ex_ntr[e + 1] : n_tr) - ex_ntr[e];
    const int32_t t0 = t * kTileM;
    int32_t nvalid = 0, has_remote = 0;
    const int32_t g1 = e + 1 < E_l ? ex_ng[e + 1] : n_grp;
    for (int32_t g = ex_ng[e]; g < g1; ++g) {
      const int32_t L0 = gl_lrow0[g];
      const int32_t lo = max(t0, L0), hi = min(t0 + kTileM, L0 + gl_rows[g]);
      if (hi > lo) {
        nvalid += hi - lo;
        if (gl_dst[g] != self) has_remote = 1;
      }
    }
    int32_t cs, ce, q;
    if (j < hr) {
      cs = ex_roff[e];
      ce = cs + hr;
      q = cs + j;
    } else {
      cs = n_hr + ex_loff[e];
      ce = cs + (ntr_e - hr);
      q = cs + (j - hr);
    }
    w.order[q] = t;
    {
      const int32_t A = cs + (q - cs) / ggu * ggu;
      w.ga_gu[q] = A;
      w.gb_gu[q] = min(A + ggu, ce);
    }
    {
      const int32_t a0 = q < n_whole ? 0 : n_whole, a1 = q < n_whole ? n_whole : n_tr;
      const int32_t base = max(cs, a0);
      const int32_t A = base + (q - base) / gdn * gdn;
      w.ga_dn[q] = A;
      w.gb_dn[q] = min(A + gdn, min(ce, a1));
    }
    const bool split = q >= n_whole;
    a.tile_rows[t] = TileRow{e, t0, nvalid, has_remote, split ? S : 1, split ? (q - n_whole) * dpr * S : -1};
    if (split && a.split_k == 0) a.tail_rows[q - n_whole] = t;
    for (int32_t n = 0; n < dpr; ++n) w.pos_of_down[t * dpr + n] = -1;
  }

  // Queue bounds: each launch's item sequence dealt round-robin to the XCD queues in chunks of
  // kQueueChunk items (queue x holds chunks x, x + kXcds, ...).  Absolute item indices.
  const int32_t n_gu = n_tr * gpr;
  const int32_t n_down = n_whole * dpr + n_split * dpr * S;
  if (tid < 2) {
    const int32_t N = tid == 0 ? n_gu : n_down, base = tid == 0 ? 0 : n_gu;
    const int32_t nf = N / kQueueChunk, part = N % kQueueChunk;
    int32_t acc = 0, qmax = 0;
    for (int x = 0; x < kXcds; ++x) {
      a.queues[tid * (kXcds + 1) + x] = base + acc;
      int32_t L = (nf > x ? (nf - x + kXcds - 1) / kXcds : 0) * kQueueChunk;
      if (part && nf % kXcds == x) L += part;
      acc += L;
      qmax = max(qmax, L);
    }
    a.queues[tid * (kXcds + 1) + kXcds] = base + acc;
    if (tid == 1) H->down_qmax = qmax;
  }
  if (tid == 0) {
    H->n_tile_rows = n_tr;
    H->n_groups = a.overlapped ? n_grp : 0;
    H->n_groups_all = n_grp;
    H->n_gu = n_gu;
    H->n_down = n_down;
    H->n_segs = 0;
    H->tail_split = S;
    H->n_split_rows = n_split;
    H->n_partials = n_split * dpr * S;
    H->n_valid = a.off[E_l];
    H->n_lrows = (int64_t)n_tr * kTileM;
    H->n_band_pad = (int64_t)s_pad;
    H->n_remote = (int64_t)s_remote;
  }
}

// ---------------------------------------------------------------------------------------------
// fill: work items, row tables, segment boundaries.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlk) void plan_fill_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kBlk];
  const PlanHeader* H = a.hdr;
  if (H->status != 0) return;
  const DevPlanWs& w = a.ws;
  const int32_t n_tr = H->n_tile_rows, n_gu = H->n_gu, n_down = H->n_down;
  const int32_t S = H->tail_split, n_whole = n_tr - H->n_split_rows, n_grp = H->n_groups_all;
  const int32_t gpr = a.gu_per_row, dpr = a.down_per_row;
  const int32_t gid = blockIdx.x * kBlk + threadIdx.x, gsz = gridDim.x * kBlk;

  // A sequence index s of a launch lies in the row group [A, B) of the schedule position
  // s / cols (every group of a range has the same columns), column-major within the group.
  for (int32_t s = gid; s < n_gu; s += gsz) {
    const int32_t p = s / gpr, A = w.ga_gu[p], m = w.gb_gu[p] - A, loc = s - A * gpr;
    const int32_t c = loc / m, q = A + loc % m;
    const int32_t ch = s / kQueueChunk, x = ch % kXcds;
    const int32_t pos = ch / kXcds * kQueueChunk + s % kQueueChunk;
    a.items[a.queues[x] + pos] = ((uint32_t)w.order[q] << kItemRowShift) | (uint32_t)c;
  }
  const int32_t n_wd = n_whole * dpr;
  for (int32_t s = gid; s < n_down; s += gsz) {
    int32_t p, A, loc;
    if (s < n_wd) {
      p = s / dpr;
      A = w.ga_dn[p];
      loc = s - A * dpr;
    } else {
      const int32_t cols = dpr * S, s2 = s - n_wd;
      p = n_whole + s2 / cols;
      A = w.ga_dn[p];
      loc = s2 - (A - n_whole) * cols;
    }
    const int32_t m = w.gb_dn[p] - A;
    const int32_t pc = loc / m, q = A + loc % m, t = w.order[q];
    const int32_t part = pc / dpr, n = pc % dpr;  // (part, column) pairs, part-major
    const int32_t ch = s / kQueueChunk, x = ch % kXcds;
    const int32_t pos = ch / kXcds * kQueueChunk + s % kQueueChunk;
    a.items[a.queues[kXcds + 1 + x] + pos] =
        kItemDown | ((uint32_t)t << kItemRowShift) | ((uint32_t)n << kDownColShift) | (uint32_t)part;
    atomicMax(&w.pos_of_down[t * dpr + n], pos);
  }

  // Logical rows, one tile row per workgroup pass.  A transfer group (Section 3.3.2) is cut at
  // tile-row boundaries into k pieces; its first and last pieces are one chunk each and the
  // middle ones coalesce mid_pieces at a time; a slot gap also starts a segment.
  const int32_t xm = max(a.mid_pieces, 1);
  const int tid = threadIdx.x;
  for (int32_t t = blockIdx.x; t < n_tr; t += gridDim.x) {
    const int32_t q = t * kTileM + tid;
    const int32_t e = a.tile_rows[t].expert;
    const int32_t g1 = e + 1 < a.E_l ? w.ex_ng[e + 1] : n_grp;
    int32_t g = -1;
    for (int32_t k = w.ex_ng[e]; k < g1; ++k)
      if (q >= w.g_lrow0[k] && q < w.g_lrow0[k] + w.g_rows[k]) {
        g = k;
        break;
      }
    int32_t start = 0, end = 0, np = 1;
    if (g >= 0) {
      const int32_t L0 = w.g_lrow0[g], L1 = L0 + w.g_rows[g];
      const int32_t i = w.g_src0[g] + (q - L0);
      const int32_t r = w.g_dst[g], sl = a.slot[i];
      a.row_x[q] = i;
      a.row_rank[q] = r;
      a.row_slot[q] = sl;
      if (a.overlapped && (r != a.self || !a.local_direct)) {
        const int32_t first_t = L0 / kTileM, k = (L1 - 1) / kTileM - first_t + 1, b = t - first_t;
        auto chunk_start = [&](int32_t pb) { return pb == 0 || k <= 2 || pb == k - 1 || (pb - 1) % xm == 0; };
        start = q == L0 || (q % kTileM == 0 && chunk_start(b)) || (int64_t)a.slot[i - 1] + 1 != sl;
        end = q == L1 - 1 || ((q + 1) % kTileM == 0 && chunk_start(b + 1)) ||
              (int64_t)a.slot[i + 1] != (int64_t)sl + 1;
        if (k > 2 && b > 0 && b < k - 1) {
          const int32_t cb = 1 + (b - 1) / xm * xm;
          np = min(cb + xm, k - 1) - cb;
        }
      }
    } else {
      a.row_x[q] = a.off[e];
      a.row_rank[q] = -1;
      a.row_slot[q] = -1;
    }
    // Compact this tile row's segment starts and ends (counts packed in one scan).
    const int32_t v = start | (end << 16);
    int32_t tot;
    const int32_t ex = wg_incl_scan<kBlk>(v, sh, &tot) - v;
    if (start) {
      w.start_q[t * kTileM + (ex & 0xFFFF)] = q;
      w.start_np[t * kTileM + (ex & 0xFFFF)] = np;
    }
    if (end) w.end_q[t * kTileM + (ex >> 16)] = q + 1;
    if (tid == 0) {
      w.cnt_s[t] = tot & 0xFFFF;
      w.cnt_e[t] = tot >> 16;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// segs: one workgroup pairs starts with ends, finishes each segment, and orders them by ready
// position, stably.
// ---------------------------------------------------------------------------------------------
constexpr int kLdsTileRows = 4096;  // per-tile-row counts in LDS up to this many tile rows
constexpr int kLdsHist = 8192;      // ready-position histogram in LDS up to this many positions

__global__ __launch_bounds__(kWg) void plan_segs_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kWg];
  __shared__ int32_t cnt_lds[2 * kLdsTileRows];
  __shared__ int32_t hist_lds[kLdsHist];
  PlanHeader* H = a.hdr;
  if (H->status != 0) return;
  const DevPlanWs& w = a.ws;
  const int32_t n_tr = H->n_tile_rows, K = H->down_qmax, dpr = a.down_per_row;
  const int tid = threadIdx.x;
  const bool c_in_lds = !a.no_lds && n_tr <= kLdsTileRows;
  int32_t* cs = c_in_lds ? cnt_lds : w.cnt_s;
  int32_t* ce = c_in_lds ? cnt_lds + kLdsTileRows : w.cnt_e;
  if (c_in_lds)
    for (int32_t t = tid; t < n_tr; t += kWg) {
      cs[t] = w.cnt_s[t];
      ce[t] = w.cnt_e[t];
    }
  __syncthreads();
  const int32_t n = wg_scan<kWg>(cs, n_tr, sh);
  wg_scan<kWg>(ce, n_tr, sh);  // the k-th end closes the k-th start's segment
  if (tid == 0) H->n_segs = n;
  if (n == 0) return;
  int32_t* hist = !a.no_lds && K <= kLdsHist ? hist_lds : w.hist;
  for (int32_t i = tid; i < K; i += kWg) hist[i] = 0;
  __syncthreads();
  for (int32_t k = tid; k < n; k += kWg) {
    const int32_t ts = range_of(cs, n_tr, k), te = range_of(ce, n_tr, k);
    const int32_t js = ts * kTileM + (k - cs[ts]);
    const int32_t q0 = w.start_q[js], q1 = w.end_q[te * kTileM + (k - ce[te])];
    Segment sg;
    sg.dst_rank = a.row_rank[q0];
    sg.rows = q1 - q0;
    sg.y_row0 = q0;
    sg.slot0 = a.row_slot[q0];
    const int32_t t0 = q0 / kTileM, t1 = (q1 - 1) / kTileM;
    sg.flag_begin = t0 * dpr;
    sg.flag_count = (t1 - t0 + 1) * dpr;
    int32_t rp = 0;
    for (int32_t f = sg.flag_begin; f < sg.flag_begin + sg.flag_count; ++f) rp = max(rp, w.pos_of_down[f]);
    sg.ready_pos = rp;
    sg.npieces = w.start_np[js];
    w.seg_tmp[k] = sg;
    w.seg_key[k] = rp;
    atomicAdd(&hist[rp], 1);
  }
  __syncthreads();
  wg_scan<kWg, true>(hist, K, sh);
  // Stable placement, kWg segments at a time: a segment goes after every earlier one with
  // the same ready position.
  for (int32_t c0 = 0; c0 < n; c0 += kWg) {
    const int32_t i = c0 + tid;
    const int32_t k = i < n ? w.seg_key[i] : -1;
    sh[tid] = k;
    __syncthreads();
    int32_t dest = 0;
    if (i < n) {
      int32_t rank = 0;
      for (int j = 0; j < tid; ++j) rank += sh[j] == k;
      dest = __hip_atomic_load(&hist[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + rank;
    }
    __syncthreads();
    if (i < n) {
      a.segs[dest] = w.seg_tmp[i];
      atomicAdd(&hist[k], 1);
    }
    __syncthreads();
  }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct WsLayout {
  size_t run_lo, run_hi, seen, ex, g, order, ga, pod, lists, cnt, seg_tmp, seg_key, hist, total;
  int64_t seen_cap;
};

WsLayout ws_layout(int32_t E_l, int32_t R, int32_t max_rows, int32_t max_tile_rows, int32_t dpr,
                   int64_t max_lrows, int64_t max_items) {
  WsLayout L{};
  int64_t cap = 64;
  while (cap < 2 * (int64_t)max_rows) cap <<= 1;
  L.seen_cap = cap;
  const size_t er = (size_t)E_l * R;
  size_t o = 0;
  // run_lo, run_hi and seen are contiguous (one all-ones fill); seen is 8-byte aligned.
  L.run_lo = o;   o += 4 * er;
  L.run_hi = o;   o += 4 * er;
  o = (o + 7) & ~(size_t)7;
  L.seen = o;     o += 8 * (size_t)cap;
  o = align256(o);
  L.ex = o;       o = align256(o + 4 * 7 * (size_t)E_l);
  L.g = o;        o = align256(o + 4 * 4 * er);
  L.order = o;    o = align256(o + 4 * (size_t)max_tile_rows);
  L.ga = o;       o = align256(o + 4 * 4 * (size_t)max_tile_rows);
  L.pod = o;      o = align256(o + 4 * (size_t)max_tile_rows * dpr);
  L.lists = o;    o = align256(o + 4 * 3 * (size_t)max_lrows);
  L.cnt = o;      o = align256(o + 4 * 2 * (size_t)max_tile_rows);
  L.seg_tmp = o;  o = align256(o + sizeof(Segment) * (size_t)max_lrows);
  L.seg_key = o;  o = align256(o + 4 * (size_t)max_lrows);
  L.hist = o;     o = align256(o + 4 * (size_t)(max_items + 1));
  L.total = o;
  return L;
}

}  // namespace

size_t devplan_ws_bytes(int32_t E_l, int32_t R, int32_t max_rows, int32_t max_tile_rows,
                        int32_t down_per_row, int64_t max_lrows, int64_t max_items) {
  return ws_layout(E_l, R, max_rows, max_tile_rows, down_per_row, max_lrows, max_items).total;
}

DevPlanWs devplan_ws_carve(void* base_, int32_t E_l, int32_t R, int32_t max_rows, int32_t max_tile_rows,
                           int32_t down_per_row, int64_t max_lrows, int64_t max_items) {
  const WsLayout L = ws_layout(E_l, R, max_rows, max_tile_rows, down_per_row, max_lrows, max_items);
  uint8_t* b = (uint8_t*)base_;
  DevPlanWs w{};
  w.run_lo = (int32_t*)(b + L.run_lo);
  w.run_hi = (int32_t*)(b + L.run_hi);
  w.seen = (uint64_t*)(b + L.seen);
  w.seen_cap = L.seen_cap;
  w.fill_words = (int64_t)((L.seen + 8 * (size_t)L.seen_cap - L.run_lo) / 4);
  int32_t* ex = (int32_t*)(b + L.ex);
  w.ex_ntr = ex;
  w.ex_ng = ex + E_l;
  w.ex_hr = ex + 2 * E_l;
  w.ex_bands = ex + 3 * E_l;
  w.ex_roff = ex + 4 * E_l;
  w.ex_loff = ex + 5 * E_l;
  w.tmp = ex + 6 * E_l;
  const size_t er = (size_t)E_l * R;
  int32_t* g = (int32_t*)(b + L.g);
  w.g_lrow0 = g;
  w.g_rows = g + er;
  w.g_dst = g + 2 * er;
  w.g_src0 = g + 3 * er;
  w.order = (int32_t*)(b + L.order);
  int32_t* ga = (int32_t*)(b + L.ga);
  w.ga_gu = ga;
  w.gb_gu = ga + max_tile_rows;
  w.ga_dn = ga + 2 * (size_t)max_tile_rows;
  w.gb_dn = ga + 3 * (size_t)max_tile_rows;
  w.pos_of_down = (int32_t*)(b + L.pod);
  int32_t* lists = (int32_t*)(b + L.lists);
  w.start_q = lists;
  w.start_np = lists + max_lrows;
  w.end_q = lists + 2 * max_lrows;
  w.cnt_s = (int32_t*)(b + L.cnt);
  w.cnt_e = w.cnt_s + max_tile_rows;
  w.seg_tmp = (Segment*)(b + L.seg_tmp);
  w.seg_key = (int32_t*)(b + L.seg_key);
  w.hist = (int32_t*)(b + L.hist);
  return w;
}

hipError_t launch_devplan(const DevPlanArgs& a, int64_t max_items, int num_cus, hipStream_t s) {
  const int64_t wide = (int64_t)std::max(num_cus, 1) * 4;
  const int rows_grid = (int)std::max<int64_t>(1, std::min<int64_t>(wide, ((int64_t)a.max_rows + kBlk - 1) / kBlk));
  // The fill kernel: a workgroup per tile row, and enough threads for the work items.
  const int fill_grid = (int)std::max<int64_t>(
      1, std::min<int64_t>(wide, std::max<int64_t>(a.max_tile_rows, (max_items + kBlk - 1) / kBlk)));
  hipLaunchKernelGGL(plan_rows_kernel, dim3(rows_grid), dim3(kBlk), 0, s, a);
  hipLaunchKernelGGL(plan_layout_kernel, dim3(1), dim3(kWg), 0, s, a);
  hipLaunchKernelGGL(plan_fill_kernel, dim3(fill_grid), dim3(kBlk), 0, s, a);
  if (a.overlapped) hipLaunchKernelGGL(plan_segs_kernel, dim3(1), dim3(kWg), 0, s, a);
  return hipGetLastError();
}

}  // namespace moe
