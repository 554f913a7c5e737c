"""Host plan builder through the C ABI (no GPU): row layout, tile schedule, combine plan.

Checks the properties the paper states for the remote-owner-aligned layout
(Section 3.2.1, Algorithm 1), the remote-first schedule (Section 3.2.2), the
combine plan (Section 3.2.3), the segment composition (Section 3.3.2) and the
padding bound (Section 4.5, per-expert reading), plus the worked example of
Section 3.2.2 stored in tests/golden/schedule_example.json.
"""
import json
import os

import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TILE_M = 256


def cfg_for(H, F, E_l, R, self_rank, max_rows, band_rows=32, mgb=1, flags=B.MOE_LOCAL_DIRECT, split_k=0):
    return B.make_config(H, F, E_l, R, self_rank, max_rows, band_rows, mgb, flags, down_split_k=split_k)


def routing_from_groups(groups, E_l, R):
    """groups[e][r] = rows of local expert e from rank r; slots follow (expert, row) per rank."""
    src, slot, off = [], [], [0]
    next_slot = [0] * R
    for e in range(E_l):
        for r in range(R):
            for _ in range(groups[e].get(r, 0)):
                src.append(r)
                slot.append(next_slot[r])
                next_slot[r] += 1
        off.append(len(src))
    return (np.array(off, np.int32), np.array(src, np.int32), np.array(slot, np.int32),
            np.array([max(n, 1) for n in next_slot], np.int64))


def decode(items):
    """(down, tile row, column tile, K part) of each work item."""
    down = (items >> 31) & 1
    t = (items >> 12) & ((1 << 19) - 1)
    col = np.where(down == 1, (items >> 4) & 0xFF, items & 0xFFF)
    part = np.where(down == 1, items & 0xF, 0)
    return down.astype(int), t.astype(int), col.astype(int), part.astype(int)


def schedule_order(p, launch):
    """Tile rows in order of first appearance in a launch's item sequence, restored from its
    per-XCD queues by interleaving their 32-item chunks round-robin (queue x holds chunks x,
    x + 8, ... of the sequence)."""
    down, t, _, _ = decode(p["items"])
    lo = 0 if launch == 0 else p["info"]["n_gu_items"]
    q = p["queues"][launch]
    chunks = [[t[lo + c:lo + min(c + 32, q[x + 1])] for c in range(q[x], q[x + 1], 32)] for x in range(8)]
    seq = []
    for c in range(max((len(ch) for ch in chunks), default=0)):
        for x in range(8):
            if c < len(chunks[x]):
                seq.extend(chunks[x][c].tolist())
    return list(dict.fromkeys(seq))


def check_plan(p, off, src, slot, self_rank, R, band_rows, mgb, overlapped=True, local_direct=True):
    info = p["info"]
    rows = int(off[-1])
    rank, lslot, rx = p["row_rank"], p["row_slot"], p["row_x"]
    valid = rank >= 0
    # every routed row appears exactly once, with its own rank and slot
    assert valid.sum() == rows
    assert np.array_equal(np.sort(rx[valid]), np.arange(rows))
    assert np.array_equal(rank[valid], src[rx[valid]])
    assert np.array_equal(lslot[valid], slot[rx[valid]])
    # padding rows feed from a row of the same expert (finite input) and are never stored
    e_of_row = np.searchsorted(off, np.arange(rows), side="right") - 1
    tr = p["tile_rows"]
    assert np.all(tr[:, 1] % TILE_M == 0)
    for t, (e, l0, nvalid, has_remote, *_split) in enumerate(tr):
        seg = slice(l0, l0 + TILE_M)
        assert np.all(e_of_row[rx[seg]] == e)
        assert nvalid == valid[seg].sum()
        assert has_remote == int(np.any(valid[seg] & (rank[seg] != self_rank)))
    # items: each gate/up tile and each K part of each down tile exactly once
    down, t, col, part = decode(p["items"])
    n_tr = len(tr)
    dpr = info["down_tiles_per_row"]
    # K parts per tile row: one split count for the split rows, 1 elsewhere; the split rows'
    # partial tiles are numbered consecutively
    splits = tr[:, 4]
    assert set(np.unique(splits).tolist()) <= {1, info["split_k"]}
    assert int(np.sum(splits > 1)) == info["split_rows"]
    split_rows = np.flatnonzero(splits > 1)
    bases = sorted(int(b) for b in tr[split_rows, 5])
    assert bases == [i * dpr * info["split_k"] for i in range(len(split_rows))]
    assert np.all(tr[splits == 1, 5] == -1)
    gu_pos = {}
    for pos, (d, ti, c, k) in enumerate(zip(down, t, col, part)):
        key = (d, ti, c, k)
        assert key not in gu_pos
        gu_pos[key] = pos
    assert info["n_down_items"] == int(np.sum(splits)) * dpr
    assert len(gu_pos) == n_tr * info["gu_tiles_per_row"] + info["n_down_items"]
    for (d, ti, c, k) in gu_pos:
        assert k < (splits[ti] if d else 1)
    # two launches: every gate/up tile precedes every down item
    n_gu = info["n_gu_items"]
    assert np.all(down[:n_gu] == 0) and np.all(down[n_gu:] == 1)
    # each launch's items are 8 per-XCD queues of near-equal size, which take tile rows in one
    # common order
    qs = p["queues"]
    assert qs.shape == (2, 9)
    qpos = np.empty(len(down), np.int64)   # position of each item within its queue
    sched_of = []
    for li, (lo, n) in enumerate(((0, n_gu), (n_gu, info["n_down_items"]))):
        q = qs[li]
        assert q[0] == 0 and q[8] == n and np.all(np.diff(q) >= 0)
        for x in range(8):
            qpos[lo + q[x]:lo + q[x + 1]] = np.arange(q[x + 1] - q[x])
        sizes = np.diff(q)   # chunks of 32 items are dealt round-robin: sizes within one chunk
        assert sizes.max() - sizes.min() <= 32
        # the launch's sequence, restored from its queues, takes tile rows in schedule order:
        # remote-first, and the same order in both launches
        sched = schedule_order(p, li)
        assert sorted(sched) == list(range(n_tr)) or n == 0
        hr = [int(tr[tt, 3]) for tt in sched]
        assert hr == sorted(hr, reverse=True)
        sched_of.append(sched)
    if n_gu and info["n_down_items"]:
        assert sched_of[0] == sched_of[1]

    if not overlapped:
        assert info["n_band_padding"] == 0 and info["n_segments"] == 0
        return
    # owner groups: one source rank each, every routed row in exactly one group
    groups = p["groups"]
    in_group = np.zeros(len(rank), int)
    for e, l0, nrows, dst in groups:
        seg = slice(l0, l0 + nrows)
        assert nrows > 0 and np.all(rank[seg] == dst) and np.all(e_of_row[rx[seg]] == e)
        in_group[seg] += 1
    assert np.array_equal(in_group, valid.astype(int))
    E_l = len(off) - 1
    for e in range(E_l):
        te = tr[tr[:, 0] == e]
        if len(te) == 0:
            continue
        base, end = te[0, 1], te[-1, 1] + TILE_M
        r_seq = rank[base:end]
        starts, order_seen = {}, []
        for i, r in enumerate(r_seq):
            if r >= 0 and r not in starts:
                starts[r] = i
                order_seen.append(r)
        remote = [r for r in order_seen if r != self_rank]
        assert remote == sorted(remote)
        if self_rank in order_seen:
            assert order_seen[-1] == self_rank
        for r in remote:
            assert starts[r] % band_rows == 0
        # padding bound: (R - 1)(tb_M - 1) band padding per expert (Section 4.5, per expert)
        n_pad_band = sum((-int(np.sum(r_seq == r))) % band_rows for r in remote)
        assert n_pad_band <= (R - 1) * (band_rows - 1)
    # segments cover every row that needs a transfer exactly once
    segs = p["segments"]
    covered = np.zeros(len(rank), int)
    for dst, nrows, y0, s0, fb, fc, rp, nb in segs:
        assert nrows > 0
        assert np.all(rank[y0:y0 + nrows] == dst)
        # a segment spans at most its pieces' tile rows: nb pieces cover at most nb tile rows
        assert (y0 + nrows - 1) // TILE_M - y0 // TILE_M + 1 <= nb
        assert np.array_equal(lslot[y0:y0 + nrows], s0 + np.arange(nrows))
        covered[y0:y0 + nrows] += 1
        t0, t1 = y0 // TILE_M, (y0 + nrows - 1) // TILE_M
        assert fb == t0 * dpr and fc == (t1 - t0 + 1) * dpr
        assert rp == max(qpos[gu_pos[(1, ti, n, k)]] for ti in range(t0, t1 + 1) for n in range(dpr)
                         for k in range(splits[ti]))
        assert 1 <= nb <= max(mgb, 1)
    need = valid & ((rank != self_rank) | (not local_direct))
    assert np.array_equal(covered, need.astype(int))
    assert np.all(np.diff(segs[:, 6]) >= 0) if len(segs) else True
    # first and last segments of every (expert, destination) group are a single tile-row piece
    group_of = {}
    for s_idx, (dst, nrows, y0, *_rest) in enumerate(segs):
        e = int(tr[y0 // TILE_M, 0])
        group_of.setdefault((e, int(dst)), []).append((y0, s_idx))
    for (e, dst), lst in group_of.items():
        lst.sort()
        assert segs[lst[0][1], 7] == 1 and segs[lst[-1][1], 7] == 1


def test_golden_schedule_example():
    g = json.load(open(os.path.join(GOLDEN, "schedule_example.json")))
    R, E_l, me, tb = g["num_ranks"], g["experts_per_rank"], g["self_rank"], g["band_rows"]
    glob = [me * E_l + i for i in range(E_l)]
    groups = [{int(r): n for r, n in g["rows_per_group"][str(e)].items()} for e in glob]
    off, src, slot, rr = routing_from_groups(groups, E_l, R)
    cfg = cfg_for(g["hidden"], g["ffn"], E_l, R, me, int(off[-1]), tb)
    p = B.moe_plan_build(cfg, off, src, slot, rr)
    check_plan(p, off, src, slot, me, R, tb, 1)
    assert p["tile_rows"][:, 0].tolist() == g["expected_tile_row_experts"]
    # both launches take the tile rows in the schedule order of the prose example
    assert schedule_order(p, 0) == g["expected_tile_row_order"]
    assert schedule_order(p, 1) == g["expected_tile_row_order"]
    pg = p["groups"]
    for e_glob, want in g["expected_remote_bands"].items():
        e = glob.index(int(e_glob))
        remote = pg[(pg[:, 0] == e) & (pg[:, 3] != me)]
        assert int(np.sum((remote[:, 2] + tb - 1) // tb)) == want
    # the group from rank 3 is padded up to the band height
    for e_glob, want in g["expected_padding_from_rank3"].items():
        e = glob.index(int(e_glob))
        n3 = groups[e][3]
        assert (-n3) % tb == want


@pytest.mark.parametrize("name,band_rows,mgb,split_k", [("tiny", 16, 1, 0), ("tiny", 32, 2, 3), ("fine", 32, 2, 0),
                                                        ("large_fine", 16, 1, 2), ("mixtral_zipf", 64, 2, 0)])
def test_plan_properties_generated(name, band_rows, mgb, split_k):
    ov = {"T_r": 512} if name != "tiny" else None
    wl = make_workload(name, weights=None, overrides=ov)
    cfg = cfg_for(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows, band_rows, mgb, split_k=split_k)
    p = B.moe_plan_build(cfg, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.return_rows)
    check_plan(p, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.self_rank, wl.R, band_rows, mgb)
    ps = B.moe_plan_build(cfg, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.return_rows, overlapped=False)
    check_plan(ps, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.self_rank, wl.R, 1, 1, overlapped=False)


@pytest.mark.parametrize("groups", [
    [{0: 0, 1: 0, 2: 0}, {0: 5, 1: 0, 2: 0}],          # empty expert, remote-only expert
    [{0: 300, 1: 0, 2: 0}, {0: 0, 1: 0, 2: 0}],         # all local, one empty expert
    [{0: 0, 1: 64, 2: 64}, {0: 1, 1: 1, 2: 1}],         # exact band multiples; single rows
    [{0: 31, 1: 33, 2: 257}, {0: 700, 1: 2, 2: 0}],     # groups smaller/larger than bands and tiles
])
def test_plan_edge_cases(groups):
    R, E_l, me, tb = 3, 2, 0, 32
    off, src, slot, rr = routing_from_groups(groups, E_l, R)
    cfg = cfg_for(128, 192, E_l, R, me, max(int(off[-1]), 1), tb, 2)
    for ld in (True, False):
        flags = B.MOE_LOCAL_DIRECT if ld else 0
        cfg.flags = flags
        p = B.moe_plan_build(cfg, off, src, slot, rr)
        check_plan(p, off, src, slot, me, R, tb, 2, local_direct=ld)


def test_empty_routing():
    cfg = cfg_for(128, 128, 2, 2, 0, 16)
    p = B.moe_plan_build(cfg, np.zeros(3, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                         np.array([4, 4], np.int64))
    assert p["info"]["n_items"] == 0 and p["info"]["n_segments"] == 0 and p["info"]["n_logical_rows"] == 0


def test_slot_gaps_split_segments():
    """Rows of one group whose slots are not consecutive go out as separate contiguous segments."""
    R, E_l, me = 2, 1, 0
    off = np.array([0, 40], np.int32)
    src = np.ones(40, np.int32)
    slot = np.concatenate([np.arange(20), 30 + np.arange(20)]).astype(np.int32)[::-1].copy()
    rr = np.array([1, 64], np.int64)
    cfg = cfg_for(64, 64, E_l, R, me, 40, 16, 4)
    p = B.moe_plan_build(cfg, off, src, slot, rr)
    check_plan(p, off, src, slot, me, R, 16, 4)
    segs = p["segments"]
    starts = sorted(int(s) for s in segs[:, 3])
    assert 0 in starts and 30 in starts


def test_validation_codes_via_plan():
    wl = make_workload("tiny", weights=None)
    cfg = cfg_for(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows)

    def code(off=wl.expert_offsets, src=wl.row_src_rank, slot=wl.row_slot, rr=wl.return_rows, c=cfg):
        try:
            B.moe_plan_build(c, off, src, slot, rr)
            return 0
        except B.MoeError as e:
            return e.code

    assert code() == 0
    off = wl.expert_offsets.copy(); off[1] = off[2] + 1
    assert code(off=off) == B.MOE_EROUTING
    src = wl.row_src_rank.copy(); src[0] = -1
    assert code(src=src) == B.MOE_EROUTING
    slot = wl.row_slot.copy(); slot[2] = wl.return_rows[wl.row_src_rank[2]]
    assert code(slot=slot) == B.MOE_EROUTING
    slot = wl.row_slot.copy(); src = wl.row_src_rank.copy(); src[4], slot[4] = src[9], slot[9]
    assert code(src=src, slot=slot) == B.MOE_EROUTING
    small = cfg_for(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows - 1)
    assert code(c=small) == B.MOE_ECAPACITY
    assert code(c=cfg_for(wl.H + 32, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows)) == B.MOE_EUNSUPPORTED
    assert code(c=cfg_for(wl.H, wl.F, wl.E_l, wl.R, wl.R, wl.rows)) == B.MOE_EINVAL
    assert code(c=cfg_for(wl.H, wl.F, wl.E_l, wl.R, 0, wl.rows, band_rows=48)) == B.MOE_EINVAL
    assert code(c=cfg_for(wl.H, wl.F, wl.E_l, wl.R, 0, wl.rows, split_k=17)) == B.MOE_EINVAL
    assert code(c=cfg_for(wl.H, wl.F, wl.E_l, wl.R, 0, wl.rows, split_k=wl.F // 64 + 1)) == B.MOE_EINVAL
    assert code(c=cfg_for(65536 + 64, wl.F, wl.E_l, wl.R, 0, wl.rows)) == B.MOE_EUNSUPPORTED
    assert code(c=cfg_for(wl.H, wl.F, wl.E_l, wl.R, 0, 1 << 24)) == B.MOE_EUNSUPPORTED


def _tail_case(H, F, tile_rows_per_expert, E_l=1, split_k=0, overlapped=True):
    """A routing whose experts each fill exactly `tile_rows_per_expert` 256-row tile rows."""
    n = 256 * tile_rows_per_expert
    off = np.arange(E_l + 1, dtype=np.int32) * n
    rows = int(off[-1])
    return B.moe_plan_build(cfg_for(H, F, E_l, 1, 0, rows, 1, split_k=split_k), off,
                            np.zeros(rows, np.int32), np.arange(rows, dtype=np.int32),
                            np.array([rows], np.int64), overlapped=overlapped)


@pytest.mark.parametrize("H,F,rows_per_expert,E_l,want_rows,want_split", [
    (4096, 14336, 16, 2, 0, 1),      # 32 tile rows x 16 tiles = 512: two full rounds
    (4096, 14336, 33, 1, 1, 16),     # 33 x 16 = 528 tiles: the last row's 16 tiles split 16 ways
    (4096, 2048, 33, 1, 1, 16),
    (4096, 512, 33, 1, 1, 8),        # capped at the 8 K steps of ffn 512
    (7168, 2048, 127, 1, 0, 1),      # 127 x 28 = 3556: the last round is 89 % full, no split
    (2048, 1408, 3, 1, 3, 10),       # 24 tiles in all: 256 // 24 = 10 parts
    (256, 512, 1, 1, 1, 8),          # one tile: as many parts as K steps (8)
])
def test_default_split_fills_the_last_round(H, F, rows_per_expert, E_l, want_rows, want_split):
    """Default split: only the tile rows of the last, partly filled round of 256 down tiles
    are split, into as many parts as that round has room for (at most 16 and ffn/64)."""
    p = _tail_case(H, F, rows_per_expert, E_l)
    info = p["info"]
    assert info["split_rows"] == want_rows and info["split_k"] == want_split
    tr = p["tile_rows"]
    dpr = info["down_tiles_per_row"]
    assert int(np.sum(tr[:, 4] > 1)) == want_rows
    assert int(np.sum(tr[:, 4] > 1)) * dpr * info["split_k"] <= 256
    # the split rows are the last rows of the schedule: their items end every down queue
    down, t, _, part = decode(p["items"])
    q = p["queues"][1]
    dn_t, dn_part = t[down == 1], part[down == 1]
    split_set = set(np.flatnonzero(tr[:, 4] > 1).tolist())
    for x in range(8):
        ts = dn_t[q[x]:q[x + 1]].tolist()
        flags = [tt in split_set for tt in ts]
        assert flags == sorted(flags)   # whole-tile items first, then split items
    # serial and overlapped plans split the same rows (same layout and order at tb_M = 1)
    ps = _tail_case(H, F, rows_per_expert, E_l, overlapped=False)
    assert np.array_equal(ps["tile_rows"], tr)


def test_explicit_split_splits_every_tile():
    p = _tail_case(4096, 14336, 3, 1, split_k=3)
    assert p["info"]["split_k"] == 3 and p["info"]["split_rows"] == 3
    assert np.all(p["tile_rows"][:, 4] == 3)
    assert p["info"]["n_down_items"] == 3 * 16 * 3


def test_split_k_part_ranges_cover_k():
    """The K steps [p*nk/S, (p+1)*nk/S) of the S parts tile [0, nk) with no gap or overlap."""
    for nk in (2, 3, 16, 18, 44, 448):
        for S in range(1, min(16, nk) + 1):
            bounds = [p * nk // S for p in range(S + 1)]
            assert bounds[0] == 0 and bounds[-1] == nk
            assert all(b1 > b0 for b0, b1 in zip(bounds, bounds[1:]))


def test_band_group_rasterisation_reuses_weights():
    """Gate/up tiles sweep the ffn columns for a group of tile rows before moving on."""
    wl = make_workload("mixtral", weights=None, overrides={"T_r": 2048})
    cfg = cfg_for(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows, 32)
    p = B.moe_plan_build(cfg, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.return_rows)
    down, t, col, _ = decode(p["items"])
    gu_t, gu_c = t[down == 0], col[down == 0]
    # consecutive gate/up tiles share the weight column tile far more often than they change it
    same_col = np.mean(gu_c[1:] == gu_c[:-1])
    assert same_col > 0.5


@pytest.mark.parametrize("name", ["mixtral", "mixtral_zipf", "fine", "large_fine"])
def test_default_layout_costs_no_extra_tiles(name):
    """With the default tb_M = 1 the owner-grouped layout has exactly the tile rows of the
    expert-contiguous baseline: the overlapped path does no extra MFMA work."""
    wl = make_workload(name, weights=None)
    cfg = B.make_config(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows)
    po = B.moe_plan_build(cfg, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.return_rows)
    ps = B.moe_plan_build(cfg, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.return_rows, overlapped=False)
    assert po["info"]["band_rows"] == 1 and po["info"]["n_band_padding"] == 0
    assert po["info"]["n_tile_rows"] == ps["info"]["n_tile_rows"]
    check_plan(po, wl.expert_offsets, wl.row_src_rank, wl.row_slot, wl.self_rank, wl.R, 1, 1)
