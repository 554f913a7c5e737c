// plan_device.hip -- the plan of one expert-stage run, built on the GPU (gfx950).
//
// The host builder (plan.cpp) walks the routing serially.  Here the same plan -- layout,
// schedule, work queues and combine plan (paper Section 3.2, Algorithm 1; segment
// composition of Section 3.3.2) -- comes from five kernels in stream order:
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
//   fill    grid: every work item straight to its queue slot; the row tables; per logical row,
//           whether a transfer segment starts or ends there; segment starts counted per tile
//           row, and the last workgroup to finish scans the counts.
//   segs    grid: each segment's fields from its first and last rows.
//   sort    one workgroup: rows, flags and ready position of every segment, then a stable
//           counting sort by ready position (the order the consumer claims them in).
//
// Every step reproduces the host's tables exactly for routing in dispatch order.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

#include "../../include/moe_stage.h"
#include "plan_device.hpp"

namespace moe {
namespace {

constexpr int kWg = 1024;   // threads of the single-workgroup kernels
constexpr int kBlk = 256;   // threads of the grid kernels; one logical row each in a tile row
static_assert(kBlk == kTileM, "the fill and segment kernels give each tile row one workgroup");

__device__ __forceinline__ int32_t round_up_i(int32_t v, int32_t m) { return (v + m - 1) / m * m; }

// Global writes of this workgroup are complete and visible to every wave of it after this
// (device-scope fence, so L1 lines read earlier are dropped), then a barrier.
__device__ __forceinline__ void wg_sync() {
  __threadfence();
  __syncthreads();
}

// Exclusive prefix sum of v[0, n) in place by one workgroup of kThreads threads (global memory,
// LDS scratch `sh` of kThreads ints); returns the total, the same in every thread.
template <int kThreads>
__device__ int32_t wg_scan(int32_t* v, int32_t n, int32_t* sh) {
  const int tid = threadIdx.x;
  int32_t carry = 0;
  for (int32_t c0 = 0; c0 < n; c0 += kThreads) {
    const int32_t i = c0 + tid;
    const int32_t x = i < n ? v[i] : 0;
    sh[tid] = x;
    __syncthreads();
    for (int d = 1; d < kThreads; d <<= 1) {
      const int32_t y = tid >= d ? sh[tid - d] : 0;
      __syncthreads();
      sh[tid] += y;
      __syncthreads();
    }
    if (i < n) v[i] = carry + sh[tid] - x;
    carry += sh[kThreads - 1];
    __syncthreads();
  }
  wg_sync();
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
__global__ __launch_bounds__(kBlk) void plan_rows_kernel(DevPlanArgs a) {
  const int32_t rows = a.off[a.E_l];
  int bad_off = 0;
  for (int e = threadIdx.x; e < a.E_l; e += kBlk) bad_off |= a.off[e] > a.off[e + 1];
  bad_off = __syncthreads_or(bad_off);
  int32_t code = 0;
  if (rows < 0)
    code = MOE_EROUTING;
  else if (rows > a.max_rows)
    code = MOE_ECAPACITY;
  else if (a.off[0] != 0 || bad_off)
    code = MOE_EROUTING;
  if (code) {
    if (blockIdx.x == 0 && threadIdx.x == 0) a.hdr->status = code;
    return;
  }
  const int32_t R = a.R;
  for (int32_t i = blockIdx.x * kBlk + threadIdx.x; i < rows; i += gridDim.x * kBlk) {
    const int32_t e = range_of(a.off, a.E_l, i);
    const int32_t lo = a.off[e], hi = a.off[e + 1];
    const int32_t r = a.src[i], s = a.slot[i];
    bool bad = r < 0 || r >= R || s < 0 || (int64_t)s >= a.return_rows[r];
    if (!bad) {
      const bool first = i == lo || a.src[i - 1] != r;
      const bool last = i == hi - 1 || a.src[i + 1] != r;
      if (!first && a.slot[i - 1] >= s) bad = true;  // slots ascend within a rank's run
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
__global__ __launch_bounds__(kWg) void plan_layout_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kWg];
  __shared__ unsigned long long s_pad, s_remote;
  PlanHeader* H = a.hdr;
  const int tid = threadIdx.x;
  if (H->status != 0) {
    write_empty(a);
    return;
  }
  if (tid == 0) s_pad = s_remote = 0;
  __syncthreads();
  const int32_t E_l = a.E_l, R = a.R, self = a.self;
  const int32_t tb = a.overlapped ? a.tb : 1;
  const DevPlanWs& w = a.ws;

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
    w.ex_ntr[e] = round_up_i(pos, kTileM) / kTileM;
    // Remote rows precede local ones, and padding never fills a whole tile row, so the tile
    // rows holding remote rows are the expert's first ones, through the last remote row's.
    w.ex_hr[e] = remote_end > 0 ? (remote_end - 1) / kTileM + 1 : 0;
    w.ex_bands[e] = bands;
    w.ex_ng[e] = ng;
    if (pad_e) atomicAdd(&s_pad, (unsigned long long)pad_e);
    if (remote_e) atomicAdd(&s_remote, (unsigned long long)remote_e);
  }
  wg_sync();
  const int32_t n_tr = wg_scan<kWg>(w.ex_ntr, E_l, sh);   // ex_ntr: first tile row of each expert
  const int32_t n_grp = wg_scan<kWg>(w.ex_ng, E_l, sh);   // ex_ng: first group of each expert
  if (n_tr > a.max_tile_rows || n_tr >= kMaxTileRows) {
    if (tid == 0) H->status = MOE_ECAPACITY;
    write_empty(a);
    return;
  }

  // Remote-first schedule (Section 3.2.2): experts by remote band count, descending, ties by
  // id, each contributing its remote tile rows; then every expert's local-only tile rows in
  // expert order.  tmp[rank] takes each expert's remote tile-row count for the prefix sum.
  for (int32_t e = tid; e < E_l; e += kWg) {
    const int32_t b = w.ex_bands[e];
    int32_t rank = 0;
    for (int32_t f = 0; f < E_l; ++f) {
      const int32_t c = w.ex_bands[f];
      rank += (c > b) || (c == b && f < e);
    }
    w.tmp[rank] = w.ex_hr[e];
    w.ex_roff[e] = rank;
  }
  wg_sync();
  const int32_t n_hr = wg_scan<kWg>(w.tmp, E_l, sh);
  for (int32_t e = tid; e < E_l; e += kWg) {
    w.ex_roff[e] = w.tmp[w.ex_roff[e]];
    const int32_t ntr_e = (e + 1 < E_l ? w.ex_ntr[e + 1] : n_tr) - w.ex_ntr[e];
    w.ex_loff[e] = ntr_e - w.ex_hr[e];
  }
  wg_sync();
  wg_scan<kWg>(w.ex_loff, E_l, sh);  // + n_hr: first local-only position of each expert

  // Owner groups with their places in the padded layout.
  for (int32_t e = tid; e < E_l; e += kWg) {
    const int32_t base = w.ex_ntr[e] * kTileM;
    int32_t g = w.ex_ng[e], pos = base;
    for (int32_t j = 0; j < R; ++j) {
      const int32_t r = rank_at(j, R, self);
      const int32_t lo = w.run_lo[e * R + r];
      if (lo < 0) continue;
      const int32_t n = w.run_hi[e * R + r] - lo;
      w.g_lrow0[g] = pos;
      w.g_rows[g] = n;
      w.g_dst[g] = r;
      w.g_src0[g] = lo;
      if (a.overlapped) a.groups[g] = Group{e, pos, n, r};
      ++g;
      pos += n;
      if (a.overlapped && r != self) pos = base + round_up_i(pos - base, tb);
    }
  }
  wg_sync();

  // Tile rows and the schedule.  ga_gu/gb_gu first hold each position's class run: the
  // expert's remote or local-only tile rows, consecutive in the schedule.
  for (int32_t t = tid; t < n_tr; t += kWg) {
    const int32_t e = range_of(w.ex_ntr, E_l, t);
    const int32_t j = t - w.ex_ntr[e], hr = w.ex_hr[e];
    const int32_t ntr_e = (e + 1 < E_l ? w.ex_ntr[e + 1] : n_tr) - w.ex_ntr[e];
    const int32_t t0 = t * kTileM;
    int32_t nvalid = 0, has_remote = 0;
    const int32_t g1 = e + 1 < E_l ? w.ex_ng[e + 1] : n_grp;
    for (int32_t g = w.ex_ng[e]; g < g1; ++g) {
      const int32_t lo = max(t0, w.g_lrow0[g]), hi = min(t0 + kTileM, w.g_lrow0[g] + w.g_rows[g]);
      if (hi > lo) {
        nvalid += hi - lo;
        if (w.g_dst[g] != self) has_remote = 1;
      }
    }
    int32_t cs, ce, q;
    if (j < hr) {
      cs = w.ex_roff[e];
      ce = cs + hr;
      q = cs + j;
    } else {
      cs = n_hr + w.ex_loff[e];
      ce = cs + (ntr_e - hr);
      q = cs + (j - hr);
    }
    w.order[q] = t;
    w.ga_gu[q] = cs;
    w.gb_gu[q] = ce;
    a.tile_rows[t] = TileRow{e, t0, nvalid, has_remote, 1, -1};
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
  wg_sync();

  // Row groups (the host's greedy walk in closed form): within a class run [cs, ce), clipped
  // to the range [a0, a1) being grouped, groups of g positions start at max(cs, a0).
  const int32_t ggu = max(a.gu_group, 1), gdn = max(a.down_group, 1);
  for (int32_t q = tid; q < n_tr; q += kWg) {
    const int32_t cs = w.ga_gu[q], ce = w.gb_gu[q];
    {
      const int32_t A = cs + (q - cs) / ggu * ggu;
      w.ga_gu[q] = A;
      w.gb_gu[q] = min(A + ggu, min(ce, n_tr));
    }
    {
      const int32_t a0 = q < n_whole ? 0 : n_whole, a1 = q < n_whole ? n_whole : n_tr;
      const int32_t base = max(cs, a0);
      const int32_t A = base + (q - base) / gdn * gdn;
      w.ga_dn[q] = A;
      w.gb_dn[q] = min(A + gdn, min(ce, a1));
    }
    if (q >= n_whole) {
      TileRow* tr = &a.tile_rows[w.order[q]];
      tr->split = S;
      tr->part_base = (q - n_whole) * dpr * S;
    }
  }
  for (int32_t i = tid; i < n_tr * dpr; i += kWg) w.pos_of_down[i] = -1;

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
  __shared__ int s_last;
  PlanHeader* H = a.hdr;
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
  for (int32_t t = blockIdx.x; t < n_tr; t += gridDim.x) {
    const int32_t q = t * kTileM + threadIdx.x;
    const int32_t e = a.tile_rows[t].expert;
    const int32_t g1 = e + 1 < a.E_l ? w.ex_ng[e + 1] : n_grp;
    int32_t g = -1;
    for (int32_t k = w.ex_ng[e]; k < g1; ++k)
      if (q >= w.g_lrow0[k] && q < w.g_lrow0[k] + w.g_rows[k]) {
        g = k;
        break;
      }
    uint32_t flag = 0;
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
        const bool start = q == L0 || (q % kTileM == 0 && chunk_start(b)) || (int64_t)a.slot[i - 1] + 1 != sl;
        const bool end = q == L1 - 1 || ((q + 1) % kTileM == 0 && chunk_start(b + 1)) ||
                         (int64_t)a.slot[i + 1] != (int64_t)sl + 1;
        int32_t np = 1;
        if (k > 2 && b > 0 && b < k - 1) {
          const int32_t cb = 1 + (b - 1) / xm * xm;
          np = min(cb + xm, k - 1) - cb;
        }
        flag = (start ? 1u : 0u) | (end ? 2u : 0u) | ((uint32_t)np << 8);
      }
    } else {
      a.row_x[q] = a.off[e];
      a.row_rank[q] = -1;
      a.row_slot[q] = -1;
    }
    w.row_flag[q] = flag;
    const int cnt = __syncthreads_count(flag & 1u);
    if (threadIdx.x == 0) w.blk_cnt[t] = cnt;
  }

  // The last workgroup to finish turns the per-tile-row counts into segment offsets.
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&H->ticket, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  const int32_t total = wg_scan<kBlk>(w.blk_cnt, n_tr, sh);
  if (threadIdx.x == 0) {
    H->n_segs = total;
    H->ticket = 0;
  }
}

// ---------------------------------------------------------------------------------------------
// segs: each segment's first-row fields and its end, in layout order.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlk) void plan_segs_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kBlk];
  const PlanHeader* H = a.hdr;
  if (H->status != 0 || H->n_segs == 0) return;
  const DevPlanWs& w = a.ws;
  const int32_t n_tr = H->n_tile_rows;
  const int tid = threadIdx.x;
  for (int32_t t = blockIdx.x; t < n_tr; t += gridDim.x) {
    const int32_t q = t * kTileM + tid;
    const uint32_t f = w.row_flag[q];
    const int32_t st = (int32_t)(f & 1u);
    sh[tid] = st;
    __syncthreads();
    for (int d = 1; d < kBlk; d <<= 1) {
      const int32_t y = tid >= d ? sh[tid - d] : 0;
      __syncthreads();
      sh[tid] += y;
      __syncthreads();
    }
    const int32_t incl = w.blk_cnt[t] + sh[tid];  // segment starts up to and including q
    if (st) {
      Segment sg{};
      sg.dst_rank = a.row_rank[q];
      sg.y_row0 = q;
      sg.slot0 = a.row_slot[q];
      sg.npieces = (int32_t)(f >> 8);
      w.seg_tmp[incl - 1] = sg;
    }
    if (f & 2u) w.seg_end[incl - 1] = q + 1;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------------------------
// sort: finish each segment, then order them by ready position, stably.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kWg) void plan_sort_kernel(DevPlanArgs a) {
  __shared__ int32_t sh[kWg];
  const PlanHeader* H = a.hdr;
  if (H->status != 0 || H->n_segs == 0) return;
  const DevPlanWs& w = a.ws;
  const int32_t n = H->n_segs, K = H->down_qmax, dpr = a.down_per_row;
  const int tid = threadIdx.x;
  for (int32_t i = tid; i < K; i += kWg) w.hist[i] = 0;
  wg_sync();
  for (int32_t i = tid; i < n; i += kWg) {
    Segment sg = w.seg_tmp[i];
    const int32_t end = w.seg_end[i];
    sg.rows = end - sg.y_row0;
    const int32_t t0 = sg.y_row0 / kTileM, t1 = (end - 1) / kTileM;
    sg.flag_begin = t0 * dpr;
    sg.flag_count = (t1 - t0 + 1) * dpr;
    int32_t rp = 0;
    for (int32_t f = sg.flag_begin; f < sg.flag_begin + sg.flag_count; ++f) rp = max(rp, w.pos_of_down[f]);
    sg.ready_pos = rp;
    w.seg_tmp[i] = sg;
    w.seg_key[i] = rp;
    atomicAdd(&w.hist[rp], 1);
  }
  wg_sync();
  wg_scan<kWg>(w.hist, K, sh);
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
      dest = w.hist[k] + rank;
    }
    wg_sync();
    if (i < n) {
      a.segs[dest] = w.seg_tmp[i];
      atomicAdd(&w.hist[k], 1);
    }
    wg_sync();
  }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct WsLayout {
  size_t run_lo, run_hi, seen, ex, g, order, ga, pod, row_flag, blk, seg_end, seg_tmp, seg_key, hist, total;
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
  L.row_flag = o; o = align256(o + 4 * (size_t)max_lrows);
  L.blk = o;      o = align256(o + 4 * (size_t)max_tile_rows);
  L.seg_end = o;  o = align256(o + 4 * (size_t)max_lrows);
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
  w.row_flag = (uint32_t*)(b + L.row_flag);
  w.blk_cnt = (int32_t*)(b + L.blk);
  w.seg_end = (int32_t*)(b + L.seg_end);
  w.seg_tmp = (Segment*)(b + L.seg_tmp);
  w.seg_key = (int32_t*)(b + L.seg_key);
  w.hist = (int32_t*)(b + L.hist);
  return w;
}

hipError_t launch_devplan(const DevPlanArgs& a, int num_cus, hipStream_t s) {
  const int wide = std::max(num_cus, 1) * 4;
  const int rows_grid = (int)std::max<int64_t>(1, std::min<int64_t>(wide, ((int64_t)a.max_rows + kBlk - 1) / kBlk));
  const int tr_grid = std::max(1, std::min(wide, a.max_tile_rows));
  hipLaunchKernelGGL(plan_rows_kernel, dim3(rows_grid), dim3(kBlk), 0, s, a);
  hipLaunchKernelGGL(plan_layout_kernel, dim3(1), dim3(kWg), 0, s, a);
  hipLaunchKernelGGL(plan_fill_kernel, dim3(wide), dim3(kBlk), 0, s, a);
  hipLaunchKernelGGL(plan_segs_kernel, dim3(tr_grid), dim3(kBlk), 0, s, a);
  hipLaunchKernelGGL(plan_sort_kernel, dim3(1), dim3(kWg), 0, s, a);
  return hipGetLastError();
}

}  // namespace moe
