// plan.cpp -- host construction of the remote-owner-aligned layout, the
// remote-first tile schedule and the combine plan (paper Section 3.2,
// Algorithm 1, and the segment composition of Section 3.3.2).
#include "plan.hpp"

#include <algorithm>
#include <numeric>
#include <string>

namespace moe {

namespace {

int fail(std::string* err, int code, const std::string& msg) {
  if (err) *err = msg;
  return code;
}

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

uint32_t gu_item(int32_t t, int32_t j) { return ((uint32_t)t << kItemRowShift) | (uint32_t)j; }
uint32_t down_item(int32_t t, int32_t n, int32_t part) {
  return kItemDown | ((uint32_t)t << kItemRowShift) | ((uint32_t)n << kDownColShift) | (uint32_t)part;
}

}  // namespace

int64_t max_logical_rows(int64_t max_rows, int32_t E_l, int32_t R, int32_t band_rows) {
  const int64_t tb = std::max<int32_t>(band_rows, 1);
  return max_rows + (int64_t)E_l * ((int64_t)(R - 1) * (tb - 1) + kTileM - 1);
}

int64_t max_partial_tiles(int32_t split_k, int64_t max_tile_rows, int32_t down_per_row, int32_t nk) {
  // The default tail split keeps at most one round of tiles' parts, and no more parts than the
  // tile rows have tiles times the parts a tile can take.
  if (split_k == 0)
    return std::min<int64_t>(kRoundTiles, max_tile_rows * down_per_row * std::min<int32_t>(kMaxSplitK, nk));
  return split_k > 1 ? max_tile_rows * down_per_row * split_k : 0;
}

int validate_routing(const PlanParams& p, int64_t rows, const int32_t* off, const int32_t* src,
                     const int32_t* slot, const int64_t* return_rows, std::string* err) {
  if (!off || !return_rows) return fail(err, -1, "expert_offsets and return_rows must not be null");
  if (rows < 0) return fail(err, -1, "rows must be >= 0");
  if (rows > 0 && (!src || !slot)) return fail(err, -1, "row_src_rank and row_slot must not be null");
  for (int r = 0; r < p.R; ++r)
    if (return_rows[r] < 0) return fail(err, -1, "return_rows[" + std::to_string(r) + "] < 0");
  if (off[0] != 0) return fail(err, -2, "expert_offsets[0] must be 0");
  for (int e = 0; e < p.E_l; ++e)
    if (off[e] > off[e + 1])
      return fail(err, -2, "expert_offsets not monotone at expert " + std::to_string(e));
  if (off[p.E_l] != rows) return fail(err, -2, "expert_offsets[E_l] must equal rows");

  std::vector<int64_t> per_rank(p.R, 0);
  for (int64_t i = 0; i < rows; ++i) {
    const int32_t r = src[i];
    if (r < 0 || r >= p.R)
      return fail(err, -2, "row " + std::to_string(i) + ": source rank out of range");
    if (slot[i] < 0 || (int64_t)slot[i] >= return_rows[r])
      return fail(err, -2, "row " + std::to_string(i) + ": slot outside its receive buffer");
    ++per_rank[r];
  }
  // Duplicate (rank, slot): a bitmap per rank when the buffers are modest, else a sort.
  bool small = true;
  for (int r = 0; r < p.R; ++r) small &= return_rows[r] <= 64 * (rows + 64);
  if (small) {
    std::vector<std::vector<uint64_t>> seen(p.R);
    for (int r = 0; r < p.R; ++r) seen[r].assign((size_t)(return_rows[r] + 63) / 64, 0);
    for (int64_t i = 0; i < rows; ++i) {
      uint64_t& w = seen[src[i]][(size_t)slot[i] >> 6];
      const uint64_t bit = 1ull << (slot[i] & 63);
      if (w & bit) return fail(err, -2, "row " + std::to_string(i) + ": duplicate (rank, slot)");
      w |= bit;
    }
  } else {
    std::vector<uint64_t> keys((size_t)rows);
    for (int64_t i = 0; i < rows; ++i) keys[i] = ((uint64_t)src[i] << 32) | (uint32_t)slot[i];
    std::sort(keys.begin(), keys.end());
    for (size_t i = 1; i < keys.size(); ++i)
      if (keys[i] == keys[i - 1]) return fail(err, -2, "duplicate (rank, slot)");
  }
  return 0;
}

int build_plan(const PlanParams& p, int64_t rows, const int32_t* off, const int32_t* src,
               const int32_t* slot, const int64_t* return_rows, Plan* out, std::string* err) {
  int rc = validate_routing(p, rows, off, src, slot, return_rows, err);
  if (rc) return rc;
  Plan& P = *out;
  P.p = p;
  P.tile_rows.clear();
  P.items.clear();
  P.row_x.clear();
  P.row_rank.clear();
  P.row_slot.clear();
  P.segs.clear();
  P.groups.clear();
  P.n_valid = rows;
  P.n_band_pad = 0;
  P.n_remote = 0;
  P.gu_per_row = (p.F + kGuTileF - 1) / kGuTileF;
  P.down_per_row = (p.H + kDownTileN - 1) / kDownTileN;

  // The baseline uses no alignment padding.  Both paths order an expert's rows by owner
  // group (Section 3.2.1, Algorithm 1): remote ranks in ascending order first, the local
  // rank last; with the default tb_M = 1 the two layouts, and so every tile, coincide.
  const int32_t tb = p.overlapped ? std::max<int32_t>(p.band_rows, 1) : 1;
  std::vector<int32_t> rank_order;
  for (int r = 0; r < p.R; ++r)
    if (r != p.self) rank_order.push_back(r);
  rank_order.push_back(p.self);

  std::vector<int32_t> tr_begin(p.E_l, 0), tr_end(p.E_l, 0), remote_bands(p.E_l, 0);
  std::vector<int64_t> bucket_start(p.R + 1);
  std::vector<int32_t> order_buf;
  for (int e = 0; e < p.E_l; ++e) {
    const int64_t lo = off[e], hi = off[e + 1];
    const int64_t base = (int64_t)P.row_x.size();  // multiple of kTileM
    tr_begin[e] = tr_end[e] = (int32_t)(base / kTileM);
    if (hi == lo) continue;

    // Bucket the expert's rows by source rank (stable), then order each bucket by slot so
    // that consecutive rows of a group fill consecutive receive slots when possible.
    std::fill(bucket_start.begin(), bucket_start.end(), 0);
    for (int64_t i = lo; i < hi; ++i) ++bucket_start[src[i] + 1];
    for (int r = 0; r < p.R; ++r) bucket_start[r + 1] += bucket_start[r];
    order_buf.resize((size_t)(hi - lo));
    {
      std::vector<int64_t> fillp(bucket_start.begin(), bucket_start.end() - 1);
      for (int64_t i = lo; i < hi; ++i) order_buf[(size_t)fillp[src[i]]++] = (int32_t)i;
    }
    for (int r = 0; r < p.R; ++r) {
      auto b = order_buf.begin() + bucket_start[r], en = order_buf.begin() + bucket_start[r + 1];
      if (!std::is_sorted(b, en, [&](int32_t a, int32_t c) { return slot[a] < slot[c]; }))
        std::stable_sort(b, en, [&](int32_t a, int32_t c) { return slot[a] < slot[c]; });
    }

    int64_t pos = base;
    for (int32_t r : rank_order) {
      const int64_t n = bucket_start[r + 1] - bucket_start[r];
      if (n == 0) continue;
      for (int64_t q = bucket_start[r]; q < bucket_start[r + 1]; ++q) {
        const int32_t i = order_buf[(size_t)q];
        P.row_x.push_back(i);
        P.row_rank.push_back(r);
        P.row_slot.push_back(slot[i]);
      }
      if (r != p.self) P.n_remote += n;
      if (p.overlapped) P.groups.push_back(Group{e, (int32_t)pos, (int32_t)n, r});
      if (r != p.self) remote_bands[e] += (int32_t)((n + tb - 1) / tb);
      pos += n;
      if (p.overlapped && r != p.self) {
        // Zero-row padding up to the next band boundary (Algorithm 1): the next group then
        // starts band-aligned and every band of tb_M rows has a single destination (none
        // with the default tb_M = 1).  Padding rows repeat the expert's first row as input;
        // their outputs are never stored or transferred.
        const int64_t pad = round_up(pos - base, tb) - (pos - base);
        for (int64_t q = 0; q < pad; ++q) {
          P.row_x.push_back((int32_t)lo);
          P.row_rank.push_back(-1);
          P.row_slot.push_back(-1);
        }
        P.n_band_pad += pad;
        pos += pad;
      }
    }
    const int64_t end = base + round_up(pos - base, kTileM);
    while ((int64_t)P.row_x.size() < end) {
      P.row_x.push_back((int32_t)lo);
      P.row_rank.push_back(-1);
      P.row_slot.push_back(-1);
    }
    for (int64_t t0 = base; t0 < end; t0 += kTileM) {
      TileRow tr{e, (int32_t)t0, 0, 0, 1, -1};
      for (int64_t q = t0; q < t0 + kTileM; ++q) {
        if (P.row_rank[q] >= 0) ++tr.nvalid;
        if (P.row_rank[q] >= 0 && P.row_rank[q] != p.self) tr.has_remote = 1;
      }
      P.tile_rows.push_back(tr);
    }
    tr_end[e] = (int32_t)(end / kTileM);
  }
  const int32_t n_tr = (int32_t)P.tile_rows.size();
  if (n_tr >= kMaxTileRows) return fail(err, -3, "too many tile rows");
  if (P.gu_per_row >= kMaxColTiles || P.down_per_row > kMaxDownColTiles)
    return fail(err, -6, "hidden or ffn too large for the work-item encoding");
  if (p.split_k < 0 || p.split_k > kMaxSplitK || p.split_k > p.F / kTileK)
    return fail(err, -1, "split_k out of range");

  // Remote-first tile schedule (Section 3.2.2), for both paths: rule (ii) experts by remote
  // band count (bands of tb_M rows, so remote rows when tb_M = 1), descending, ties by expert
  // id; rule (i) every tile row holding remote rows before any tile row of only local rows.
  std::vector<int32_t> order;
  order.reserve(n_tr);
  {
    std::vector<int32_t> experts(p.E_l);
    std::iota(experts.begin(), experts.end(), 0);
    std::stable_sort(experts.begin(), experts.end(),
                     [&](int32_t a, int32_t b) { return remote_bands[a] > remote_bands[b]; });
    for (int32_t e : experts)
      for (int32_t t = tr_begin[e]; t < tr_end[e]; ++t)
        if (P.tile_rows[t].has_remote) order.push_back(t);
    for (int32_t e = 0; e < p.E_l; ++e)
      for (int32_t t = tr_begin[e]; t < tr_end[e]; ++t)
        if (!P.tile_rows[t].has_remote) order.push_back(t);
  }

  // K parts per down tile.  An explicit split_k splits every tile.  By default only the
  // tile rows at the end of the schedule are split: the down tiles fill whole rounds of
  // kRoundTiles, and the tile rows holding the remainder -- the last, partly filled round --
  // are split into as many parts as that round has room for, so it runs full instead of
  // leaving most compute units idle, while the added fp32 partial traffic stays within one
  // round's worth of tiles.  The choice depends on the tile count only, never on the path or
  // the launch, so a given routing always gets the same parts.
  const int32_t nk = p.F / kTileK;
  P.tail_split = 1;
  P.n_split_rows = 0;
  if (p.split_k > 0) {
    P.tail_split = p.split_k;
    P.n_split_rows = p.split_k > 1 ? n_tr : 0;
  } else if (n_tr > 0) {
    const int64_t n_tiles = (int64_t)n_tr * P.down_per_row;
    const int64_t rem = n_tiles % kRoundTiles;
    if (rem > 0) {
      const int32_t rows = (int32_t)((rem + P.down_per_row - 1) / P.down_per_row);
      const int64_t s = kRoundTiles / ((int64_t)rows * P.down_per_row);
      const int32_t S = (int32_t)std::min<int64_t>(std::min<int64_t>(s, kMaxSplitK), nk);
      if (S > 1) {
        P.tail_split = S;
        P.n_split_rows = rows;
      }
    }
  }
  P.n_partials = 0;
  for (int32_t q = n_tr - P.n_split_rows; q < n_tr; ++q) {
    TileRow& tr = P.tile_rows[order[q]];
    tr.split = P.tail_split;
    tr.part_base = P.n_partials;
    P.n_partials += P.down_per_row * P.tail_split;
  }

  // Per-XCD work queues.  Each XCD has its own L2, and an item streams two operand panels
  // (a token or activation panel of its tile row and a weight panel of its column) through
  // it.  Each launch's items are laid out in schedule order as blocks: a row group (up to 4
  // consecutive tile rows of one expert and one class) times a slice of its columns -- gate/up
  // feature tiles, down (K part, column tile) pairs -- wide enough for about 32 items, columns
  // outer and rows inner.  That sequence is cut into chunks of 32 items dealt round-robin to
  // the XCD queues, so every queue holds the same work to within one chunk (whatever the
  // row-group sizes) and advances through the schedule at the same pace (tile rows still
  // finish in schedule order), and an XCD's 32 CUs run about 4 rows x 8 columns at once,
  // sharing every panel through L2.  A workgroup whose queue is empty takes items from the
  // next XCD's queue.
  auto row_groups = [&](int32_t g, int32_t a0, int32_t a1) {
    std::vector<std::pair<int32_t, int32_t>> out;
    g = std::max<int32_t>(g, 1);
    for (int32_t a = a0; a < a1;) {
      int32_t b = a + 1;
      while (b < a1 && b - a < g && P.tile_rows[order[b]].expert == P.tile_rows[order[a]].expert &&
             P.tile_rows[order[b]].has_remote == P.tile_rows[order[a]].has_remote)
        ++b;
      out.emplace_back(a, b);
      a = b;
    }
    return out;
  };
  // Appends the blocks of `groups` (tile rows of `cols` columns each) to `seq` as (q, column).
  auto blocks = [&](const std::vector<std::pair<int32_t, int32_t>>& groups, int32_t cols,
                    std::vector<std::pair<int32_t, int32_t>>* seq) {
    for (const auto& g : groups) {
      const int32_t w = std::max<int32_t>(1, kQueueChunk / (g.second - g.first));
      for (int32_t c0 = 0; c0 < cols; c0 += w)
        for (int32_t c = c0; c < std::min(cols, c0 + w); ++c)
          for (int32_t q = g.first; q < g.second; ++q) seq->emplace_back(q, c);
    }
  };
  // Deals `seq` to the XCD queues in chunks of kQueueChunk items, round-robin: queue x gets
  // chunks x, x + 8, ...; calls begin_queue(x) and push(q, column) queue by queue.
  auto deal = [&](const std::vector<std::pair<int32_t, int32_t>>& seq, auto&& begin_queue, auto&& push) {
    for (int32_t x = 0; x < kXcds; ++x) {
      begin_queue(x);
      for (size_t c0 = (size_t)x * kQueueChunk; c0 < seq.size(); c0 += (size_t)kXcds * kQueueChunk)
        for (size_t i = c0; i < std::min(seq.size(), c0 + kQueueChunk); ++i) push(seq[i].first, seq[i].second);
    }
  };
  std::vector<std::pair<int32_t, int32_t>> seq;

  blocks(row_groups(p.gu_group, 0, n_tr), P.gu_per_row, &seq);
  deal(seq, [&](int32_t x) { P.gu_queue[x] = (int32_t)P.items.size(); },
       [&](int32_t q, int32_t j) { P.items.push_back(gu_item(order[q], j)); });
  P.n_gu = (int32_t)P.items.size();
  P.gu_queue[kXcds] = P.n_gu;

  // Down tiles, the signaling GEMM of Section 3.3.1, run after every gate/up tile (a separate
  // launch on the producer stream).  A tile is ready once all its K parts are done; its
  // position in the run is taken as the latest queue position of its parts.
  std::vector<int32_t> pos_of_down((size_t)n_tr * P.down_per_row, -1);
  const int32_t n_whole = n_tr - P.n_split_rows;  // whole-tile rows first, split rows last
  seq.clear();
  blocks(row_groups(p.down_group, 0, n_whole), P.down_per_row, &seq);
  blocks(row_groups(p.down_group, n_whole, n_tr), P.down_per_row * P.tail_split, &seq);
  int32_t q0 = 0;
  deal(seq,
       [&](int32_t x) {
         q0 = (int32_t)P.items.size();
         P.down_queue[x] = q0 - P.n_gu;
       },
       [&](int32_t q, int32_t pc) {  // pc: (part, column) pair, part-major
         const int32_t t = order[q], part = pc / P.down_per_row, n = pc % P.down_per_row;
         P.items.push_back(down_item(t, n, part));
         int32_t& pos = pos_of_down[(size_t)t * P.down_per_row + n];
         pos = std::max(pos, (int32_t)P.items.size() - 1 - q0);
       });
  P.n_down = (int32_t)P.items.size() - P.n_gu;
  P.down_queue[kXcds] = P.n_down;

  // Combine plan (Section 3.2.3) and segment composition (Section 3.3.2).  A row is ready
  // when the down tiles of its 256-row tile row are, so each owner group is cut at tile-row
  // boundaries into pieces; per group the first and the last piece are one segment each and
  // middle segments coalesce x pieces.  Rows of a segment are contiguous in the staged output
  // and in the receive buffer; a slot gap splits a segment.  Local groups need no transfer
  // when the producer writes them directly.
  if (p.overlapped) {
    const int32_t x = std::max<int32_t>(p.mid_pieces, 1);
    std::vector<std::pair<int32_t, int32_t>> pieces, chunks;
    for (const Group& g : P.groups) {
      if (g.dst_rank == p.self && p.local_direct) continue;
      pieces.clear();
      for (int32_t s0 = g.lrow0; s0 < g.lrow0 + g.rows;) {
        const int32_t s1 = std::min(g.lrow0 + g.rows, (s0 / kTileM + 1) * kTileM);
        pieces.emplace_back(s0, s1);
        s0 = s1;
      }
      const int32_t k = (int32_t)pieces.size();
      chunks.clear();
      if (k <= 2) {
        for (int32_t b = 0; b < k; ++b) chunks.emplace_back(b, b + 1);
      } else {
        chunks.emplace_back(0, 1);
        for (int32_t b = 1; b < k - 1; b += x) chunks.emplace_back(b, std::min(b + x, k - 1));
        chunks.emplace_back(k - 1, k);
      }
      for (auto& c : chunks) {
        const int32_t r0 = pieces[c.first].first, r1 = pieces[c.second - 1].second;
        int32_t s = r0;
        while (s < r1) {
          int32_t e_ = s + 1;
          while (e_ < r1 && P.row_slot[e_] == P.row_slot[e_ - 1] + 1) ++e_;
          Segment sg{};
          sg.dst_rank = g.dst_rank;
          sg.rows = e_ - s;
          sg.y_row0 = s;
          sg.slot0 = P.row_slot[s];
          const int32_t t0 = s / kTileM, t1 = (e_ - 1) / kTileM;
          sg.flag_begin = t0 * P.down_per_row;
          sg.flag_count = (t1 - t0 + 1) * P.down_per_row;
          int32_t rp = 0;
          for (int32_t f = sg.flag_begin; f < sg.flag_begin + sg.flag_count; ++f)
            rp = std::max(rp, pos_of_down[f]);
          sg.ready_pos = rp;
          sg.npieces = c.second - c.first;
          P.segs.push_back(sg);
          s = e_;
        }
      }
    }
    // The consumer claims segments in the order their data becomes ready.
    std::stable_sort(P.segs.begin(), P.segs.end(),
                     [](const Segment& a, const Segment& b) { return a.ready_pos < b.ready_pos; });
  }
  return 0;
}

}  // namespace moe
