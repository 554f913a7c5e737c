"""Full-size GPU parity at the workload sizes the benchmark uses, in its launch configuration.

Placement (every routed slot written, nothing else touched) and bitwise equality across
consumer splits, CU modes and the serial path hold at any size and are checked on every row.
Values are checked against the oracle, row by row, on a stratified sample drawn from the
plan the GPU ran: at least one routed row of every 256-row tile row, of every (expert,
source rank) owner group (so every local expert's weights and the local-direct rows), every
row of the first split tile row (the K-split tail, whose parts a tail kernel adds), and
random rows on top.  Each sampled row is checked on all hidden columns, so every 256-column
down tile is covered.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, SENTINEL

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

BENCH_CU_SPLIT = 64
BENCH_FLAGS = B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS   # bench.py's default mode, on its own stream
RANDOM_ROWS = 24


def written_mask(buf_dev):
    s = SENTINEL - 65536
    return (~(buf_dev == s).all(dim=1)).cpu().numpy()


def stratified_rows(wl, plan, seed=3):
    """Dispatched-row indices of the value sample, and how many each stratum contributed."""
    g = np.random.default_rng(seed)
    tr = plan["tile_rows"]            # expert, lrow0, nvalid, has_remote, split, part_base
    row_x, row_rank = plan["row_x"], plan["row_rank"]
    picked = set()
    counts = {"tile_rows": 0, "groups": 0, "split_tail_rows": 0, "local_rows": 0, "random": 0}
    for t in range(len(tr)):
        l0 = int(tr[t, 1])
        valid = np.nonzero(row_rank[l0:l0 + 256] >= 0)[0]
        if len(valid):
            picked.add(int(row_x[l0 + int(g.choice(valid))]))
            counts["tile_rows"] += 1
    split = [t for t in range(len(tr)) if int(tr[t, 4]) > 1]
    if split:
        l0 = int(tr[split[0], 1])
        for lr in range(l0, l0 + 256):
            if row_rank[lr] >= 0:
                picked.add(int(row_x[lr]))
                counts["split_tail_rows"] += 1
    e_of = np.searchsorted(wl.expert_offsets, np.arange(wl.rows), side="right") - 1
    for e in range(wl.E_l):
        for r in range(wl.R):
            rows = np.nonzero((e_of == e) & (wl.row_src_rank == r))[0]
            if len(rows):
                picked.add(int(g.choice(rows)))
                counts["groups"] += 1
                counts["local_rows"] += int(r == wl.self_rank)
    for i in g.choice(wl.rows, size=min(RANDOM_ROWS, wl.rows), replace=False):
        picked.add(int(i))
        counts["random"] += 1
    return np.array(sorted(picked), np.int64), counts, len(split)


def compact_oracle(wl, idx):
    """Oracle outputs of the rows `idx` with each source rank's slots renumbered densely (the
    oracle computes every row on its own, so the values are those of the full stage)."""
    from oracle import oracle as orc
    sub = wl.subset(idx)
    slot = np.empty(sub.rows, np.int32)
    rows = np.zeros(wl.R, np.int64)
    for r in range(wl.R):
        m = np.nonzero(sub.row_src_rank == r)[0]
        order = m[np.argsort(sub.row_slot[m], kind="stable")]
        slot[order] = np.arange(len(order), dtype=np.int32)
        rows[r] = len(order)
    bufs = [np.full((int(n), wl.H), SENTINEL, np.uint16) for n in rows]
    rc = orc.get().run(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, sub.dispatched_x, sub.expert_offsets,
                       sub.row_src_rank, slot, wl.w1, wl.w3, wl.w2, bufs, rows, 0)
    assert rc == 0, rc
    return sub, slot, bufs


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["mixtral", "mixtral_zipf", "fine", "large_fine", "layer_e4", "layer_e64"])
def test_fullsize_stratified(name):
    log(f"full-size {name}: generating")
    wl = make_workload(name)
    log(f"full-size {name}: rows={wl.rows}")
    dw = DeviceWorkload(torch, wl)
    side = torch.cuda.Stream()
    with make_stage(wl, flags=BENCH_FLAGS) as st:
        dw.fill()
        torch.cuda.synchronize()
        st.run(*dw.args(), cu_split=BENCH_CU_SPLIT, stream=side)
        torch.cuda.synchronize()
        stats = st.query()
        plan = st.plan()
        log(f"full-size {name}: overlapped done, segments={stats['n_segments']} units={stats['copy_units']} "
            f"tiles={stats['n_tile_rows']} split_k={stats['split_k']} workgroups={stats['gu_workgroups']}/"
            f"{stats['down_workgroups']}")
        assert stats["timeout"] == 0
        # placement on every row: exactly the routed slots are written
        for r in range(wl.R):
            want = np.zeros(int(dw.return_rows[r]), bool)
            want[wl.row_slot[wl.row_src_rank == r]] = True
            assert np.array_equal(written_mask(dw.bufs[r]), want), f"rank {r} placement"
        over = [b.clone() for b in dw.bufs]
        # Narrower and wider consumers beside the producer: with 8 CUs (eight waves each) most
        # units are claimed after each wave's first one; with 248 (one wave each) many waves find
        # no unit left.
        for c in (8, 32, 248):
            dw.fill()
            torch.cuda.synchronize()
            st.run(*dw.args(), cu_split=c, stream=side)
            torch.cuda.synchronize()
            other = st.query()
            log(f"full-size {name}: c={c} shared units={other['copy_units']} consumer workgroups={other['consumer_grid']}")
            assert other["timeout"] == 0
            for a, b in zip(over, dw.bufs):
                assert torch.equal(a, b), f"consumer splits differ (c={c})"
        dw.fill()
        torch.cuda.synchronize()
        st.run_serial(*dw.args(), stream=side)
        torch.cuda.synchronize()
        st.query()
        for a, b in zip(over, dw.bufs):
            assert torch.equal(a, b), "serial and overlapped differ"
    # The consumer on compute units of its own cuts segments into ~64 KiB units.
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT) as st:
        dw.fill()
        torch.cuda.synchronize()
        st.run(*dw.args(), cu_split=32, stream=side)
        torch.cuda.synchronize()
        part = st.query()
        log(f"full-size {name}: c=32 partitioned units={part['copy_units']} segments={part['n_segments']}")
        assert part["timeout"] == 0
        for a, b in zip(over, dw.bufs):
            assert torch.equal(a, b), "partitioned consumer differs"
    del over
    idx, counts, n_split = stratified_rows(wl, plan)
    log(f"full-size {name}: value sample {len(idx)} rows: {counts} ({n_split} split tile rows in the plan)")
    assert counts["tile_rows"] == int((plan["tile_rows"][:, 2] > 0).sum())
    assert n_split == 0 or counts["split_tail_rows"] > 0
    sub, slot, ref = compact_oracle(wl, idx)
    got = []
    for r in range(wl.R):
        m = np.nonzero(sub.row_src_rank == r)[0]
        g = np.full((len(m), wl.H), SENTINEL, np.uint16)
        if len(m):
            rows = torch.from_numpy(sub.row_slot[m].astype(np.int64)).to("cuda")
            g[slot[m]] = dw.bufs[r].index_select(0, rows).cpu().numpy().view(np.uint16)
        got.append(g)
    worst, worst_rel = compare(got, ref)
    log(f"full-size {name}: sampled max scaled err {worst:.2e}, max row rel-L2 {worst_rel:.2e}")


@pytest.mark.timeout(300)
def test_watchdog_expiry_is_reported():
    """With ready flags suppressed from the host, the consumer's bounded wait expires, the
    kernels exit, the run reports MOE_ETIMEOUT with the first segment that expired, and the next
    run on a fresh handle is correct.  The expired run's output is complete too: each consumer
    wave that gives up hands its unit to the drain launch, which copies it after the producer."""
    from tests.gpu_helpers import oracle_bufs
    wl = make_workload("tiny", owner=1)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    for c, mode in ((8, B.MOE_SHARED_CUS), (64, B.MOE_SHARED_CUS), (16, 0)):
        dw.fill()
        with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_TEST_NO_SIGNAL | mode, watchdog_ms=20) as st:
            st.run(*dw.args(), cu_split=c)
            q = st.query(check=False)
            assert q["rc"] == B.MOE_ETIMEOUT and q["timeout"] == 1
            assert 0 <= q["timeout_segment"] < q["n_segments"]
            assert "segment" in B.moe_stage_last_error(st.h)
            q2 = st.query()
            assert q2["timeout"] == 0   # reported once
        compare(dw.host_bufs(), ref)
        log(f"watchdog: c={c} {'shared' if mode else 'partitioned'} expired run complete")
    with make_stage(wl) as st:
        dw.fill()
        st.run(*dw.args(), cu_split=8)
        assert st.query()["timeout_segment"] == -1
    compare(dw.host_bufs(), ref)
