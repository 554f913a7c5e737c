"""GPU tests of the device-side plan builder (moe_stage_run_devplan / _run_serial_devplan).

The device planner must produce exactly the host builder's plan (paper Section 3.2,
Algorithm 1: layout, schedule and combine plan; Section 3.3.2: segments): every table read
back from the device -- tile rows, work items and XCD queues, row tables, segments, groups --
is compared bit for bit with moe_plan_build's tables for the same routing, over the generated
workloads, the configuration knobs (band rows, segment coalescing, local-direct, split K) and
seeded random routings in dispatch order (empty experts, single ranks, slot gaps, ranks in any
order).  A run on a device-built plan must then give the same bits as the host-planned run
(same tables, same kernels), and one case is checked against the oracle directly.  Routing
errors are reported by the next query, with nothing written.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, SENTINEL, compare, log, oracle_bufs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TABLES = ("tile_rows", "items", "row_x", "row_rank", "row_slot", "segments", "groups", "queues")
NO_LDS = B.MOE_TEST_PLAN_NO_LDS


def _bf16_rand(shape, seed, scale=0.05):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda") * scale).to(torch.bfloat16).view(torch.int16)


class Case:
    """One owner's stage inputs on the device: routing (host and device copies), random weights."""

    def __init__(self, H, F, E_l, R, self_rank, off, src, slot, rr, seed=0, x=None, w=None):
        self.H, self.F, self.E_l, self.R, self.self_rank = H, F, E_l, R, self_rank
        self.off = np.ascontiguousarray(off, np.int32)
        self.src = np.ascontiguousarray(src, np.int32)
        self.slot = np.ascontiguousarray(slot, np.int32)
        self.rr = np.ascontiguousarray(rr, np.int64)
        self.rows = int(self.off[-1])
        self.d_off = torch.from_numpy(self.off).cuda()
        self.d_src = torch.from_numpy(self.src if self.rows else np.zeros(1, np.int32)).cuda()
        self.d_slot = torch.from_numpy(self.slot if self.rows else np.zeros(1, np.int32)).cuda()
        self.x = x if x is not None else _bf16_rand((max(self.rows, 1), H), seed, 1.0)
        if w is None:
            w = (_bf16_rand((E_l, F, H), seed + 1), _bf16_rand((E_l, F, H), seed + 2), _bf16_rand((E_l, H, F), seed + 3))
        self.w1, self.w3, self.w2 = w
        self.bufs = [torch.empty((int(n), H), dtype=torch.int16, device="cuda") for n in self.rr]

    @classmethod
    def from_workload(cls, wl, seed=0, device_weights=True):
        if device_weights:
            return cls(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.expert_offsets, wl.row_src_rank, wl.row_slot,
                       wl.return_rows, seed)
        dw = DeviceWorkload(torch, wl)
        return cls(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.expert_offsets, wl.row_src_rank, wl.row_slot,
                   wl.return_rows, seed, x=dw.x, w=(dw.w1, dw.w3, dw.w2))

    def fill(self):
        for b in self.bufs:
            b.fill_(SENTINEL - 65536 if SENTINEL >= 32768 else SENTINEL)

    def host_args(self):
        return (self.x, self.off, self.src, self.slot, self.w1, self.w3, self.w2, self.bufs, self.rr)

    def dev_args(self):
        return (self.x, self.d_off, self.d_src, self.d_slot, self.w1, self.w3, self.w2, self.bufs, self.rr)

    def out(self):
        torch.cuda.synchronize()
        return [b.cpu().numpy().view(np.uint16).copy() for b in self.bufs]


def stage_for(c, max_rows=None, band_rows=0, mgb=1, flags=B.MOE_LOCAL_DIRECT, split_k=0):
    return B.MoeStage(c.H, c.F, c.E_l, c.R, c.self_rank, max_rows or max(c.rows, 1), band_rows, mgb, flags, 0,
                      split_k)


def host_tables(st, c, overlapped):
    return B.moe_plan_build(st.cfg, c.off, c.src, c.slot, c.rr, overlapped=overlapped)


def assert_same_plan(dev, host, what=""):
    for k in ("n_tile_rows", "n_items", "n_gu_items", "n_down_items", "n_segments", "n_groups",
              "split_k", "split_rows", "n_logical_rows", "n_valid", "n_band_padding", "n_remote_rows",
              "band_rows", "gu_tiles_per_row", "down_tiles_per_row"):
        assert dev["info"][k] == host["info"][k], f"{what}: info {k}: device {dev['info'][k]} host {host['info'][k]}"
    for k in TABLES:
        a, b = dev[k], host[k]
        assert a.shape == b.shape, f"{what}: {k} shape {a.shape} vs {b.shape}"
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[:4]
            raise AssertionError(f"{what}: table {k} differs at {bad.tolist()}")


def check_both_paths(c, overlapped=True, cu_split=8, compare_outputs=True, **kw):
    """Host-planned and device-planned runs of one case: identical plans and identical bits."""
    with stage_for(c, **kw) as st:
        run_h = st.run if overlapped else st.run_serial
        run_d = st.run_devplan if overlapped else st.run_serial_devplan
        extra = dict(cu_split=cu_split) if overlapped else {}
        c.fill()
        run_h(*c.host_args(), **extra)
        host_out = c.out() if compare_outputs else None
        sh = st.query()
        c.fill()
        run_d(*c.dev_args(), **extra)
        dev_out = c.out() if compare_outputs else None
        sd = st.query()
        dev = st.plan()
        host = host_tables(st, c, overlapped)
        assert_same_plan(dev, host, f"overlapped={overlapped} {kw}")
        for k in ("n_valid", "n_logical_rows", "n_band_padding", "n_remote_rows", "n_tile_rows", "n_groups",
                  "n_gu_items", "n_down_items", "n_segments", "split_k", "split_rows"):
            assert sd[k] == sh[k], f"stats {k}: {sd[k]} vs {sh[k]}"
        assert sd["timeout"] == 0
        if compare_outputs:
            for r, (a, b) in enumerate(zip(dev_out, host_out)):
                assert np.array_equal(a, b), f"rank {r}: device-planned output differs from host-planned"
        return dev_out


# ------------------------------------------------------------------------------------ workloads

@pytest.mark.parametrize("name", ["tiny", "mixtral", "mixtral_zipf", "fine", "large_fine", "layer_e64"])
def test_workload_plans_match_host(name):
    log(f"devplan workload {name}")
    c = Case.from_workload(make_workload(name, weights=None), seed=3)
    check_both_paths(c, overlapped=True, cu_split=32)
    check_both_paths(c, overlapped=False)
    # the planner's device-memory path (taken by configurations too large for its LDS tables)
    check_both_paths(c, overlapped=True, cu_split=32, flags=B.MOE_LOCAL_DIRECT | NO_LDS)


RAGGED = dict(H=320, F=576, E_t=8, k=2, R=4, T_r=512, E_l=2)


@pytest.mark.parametrize("band_rows,mgb,flags,split_k", [
    (0, 1, B.MOE_LOCAL_DIRECT, 0), (16, 3, B.MOE_LOCAL_DIRECT, 0), (256, 2, 0, 0), (1, 1, 0, 3),
    (64, 4, B.MOE_LOCAL_DIRECT, 1), (32, 1, B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS, 2),
    (0, 1, B.MOE_LOCAL_DIRECT | NO_LDS, 0), (16, 3, NO_LDS, 2),
])
@pytest.mark.parametrize("owner", [0, 3])
def test_config_matrix(band_rows, mgb, flags, split_k, owner):
    log(f"devplan config tb={band_rows} mgb={mgb} flags={flags} split_k={split_k} owner={owner}")
    wl = make_workload("tiny", owner=owner, weights=None, overrides=RAGGED)
    c = Case.from_workload(wl, seed=owner)
    check_both_paths(c, overlapped=True, cu_split=8, band_rows=band_rows, mgb=mgb, flags=flags, split_k=split_k)
    check_both_paths(c, overlapped=False, band_rows=band_rows, mgb=mgb, flags=flags, split_k=split_k)


def test_oracle_through_device_plan():
    """Every owner of the tiny workload, device-planned, against the oracle."""
    for owner in range(4):
        wl = make_workload("tiny", owner=owner)
        log(f"devplan oracle owner={owner}")
        c = Case.from_workload(wl, device_weights=False)
        ref = oracle_bufs(wl)
        with stage_for(c, band_rows=16, mgb=2) as st:
            c.fill()
            st.run_devplan(*c.dev_args(), cu_split=8)
            compare(c.out(), ref)
            st.query()
            c.fill()
            st.run_serial_devplan(*c.dev_args())
            compare(c.out(), ref)
            st.query()


# ------------------------------------------------------------------------------- random routing

def dispatch_routing(rng, counts, R, contiguous, extra_slots=0):
    """Routing in dispatch order: counts[e][r] rows of expert e from rank r; within an expert each
    rank's rows are contiguous (ranks in random order) with ascending slots.  Slots of a rank are
    distinct across experts: consecutive per (expert, rank) when `contiguous`, else scattered."""
    E_l = len(counts)
    per_rank = [sum(counts[e][r] for e in range(E_l)) for r in range(R)]
    rr = np.array([n + extra_slots for n in per_rank], np.int64)
    pools = []
    for r in range(R):
        if contiguous:
            pools.append(list(range(per_rank[r])))
        else:
            pools.append(list(rng.choice(int(rr[r]), size=per_rank[r], replace=False)) if per_rank[r] else [])
    used = [0] * R
    off, src, slot = [0], [], []
    for e in range(E_l):
        ranks = list(range(R))
        rng.shuffle(ranks)
        for r in ranks:
            n = counts[e][r]
            s = sorted(pools[r][used[r]:used[r] + n])
            used[r] += n
            src += [r] * n
            slot += s
        off.append(len(src))
    return np.array(off, np.int32), np.array(src, np.int32), np.array(slot, np.int32), rr


def random_case(seed):
    rng = np.random.default_rng(seed)
    E_l = int(rng.choice([1, 2, 3, 8]))
    R = int(rng.choice([1, 2, 3, 5]))
    me = int(rng.integers(R))
    kind = seed % 4
    counts = []
    for _ in range(E_l):
        row = []
        for _ in range(R):
            if rng.random() < 0.25:
                row.append(0)
            elif kind == 0:
                row.append(int(rng.integers(1, 40)))
            else:
                row.append(int(rng.integers(1, 700)))
        counts.append(row)
    off, src, slot, rr = dispatch_routing(rng, counts, R, contiguous=seed % 3 != 0, extra_slots=int(rng.integers(0, 50)))
    return Case(128, 192, E_l, R, me, off, src, slot, rr, seed=seed), rng


@pytest.mark.parametrize("seed", range(16))
def test_random_routings(seed):
    c, rng = random_case(seed)
    band = int(rng.choice([0, 1, 8, 64, 256]))
    mgb = int(rng.integers(1, 4))
    flags = int(rng.choice([0, B.MOE_LOCAL_DIRECT])) | (NO_LDS if seed % 2 else 0)
    split_k = int(rng.choice([0, 0, 1, 2]))
    max_rows = c.rows + int(rng.choice([0, 1, 1000]))
    log(f"devplan random seed={seed} E_l={c.E_l} R={c.R} rows={c.rows} tb={band} mgb={mgb} flags={flags} "
        f"split_k={split_k} max_rows={max_rows}")
    kw = dict(max_rows=max(max_rows, 1), band_rows=band, mgb=mgb, flags=flags, split_k=split_k)
    check_both_paths(c, overlapped=True, cu_split=8, **kw)
    check_both_paths(c, overlapped=False, **kw)


def test_empty_routing():
    off = np.zeros(3, np.int32)
    c = Case(128, 128, 2, 2, 0, off, np.zeros(0, np.int32), np.zeros(0, np.int32), np.array([4, 4], np.int64))
    check_both_paths(c, overlapped=True)
    check_both_paths(c, overlapped=False)


def test_alternating_runs_on_one_handle():
    """Host- and device-planned runs of different routings, larger then smaller, share a handle."""
    c0 = Case(128, 192, 8, 5, 1, *dispatch_routing(np.random.default_rng(7), [[300, 0, 20, 600, 5]] * 8, 5, True))
    c1 = Case(128, 192, 8, 5, 1, *dispatch_routing(np.random.default_rng(8), [[3, 9, 0, 1, 60]] * 8, 5, False, 40))
    with B.MoeStage(128, 192, 8, 5, 1, c0.rows, 0, 2, B.MOE_LOCAL_DIRECT, 0, 0) as st:
        for c, dev in ((c0, True), (c1, False), (c1, True), (c0, False), (c0, True)):
            log(f"alternating rows={c.rows} dev={dev}")
            c.fill()
            if dev:
                st.run_devplan(*c.dev_args(), cu_split=8)
            else:
                st.run(*c.host_args(), cu_split=8)
            c.out()
            st.query()
            assert_same_plan(st.plan(), host_tables(st, c, True), f"rows={c.rows} dev={dev}")


# ---------------------------------------------------------------------------------------- errors

def _expect_device_error(st, c, code, serial=False):
    c.fill()
    if serial:
        st.run_serial_devplan(*c.dev_args())
    else:
        st.run_devplan(*c.dev_args(), cu_split=8)
    out = c.out()
    with pytest.raises(B.MoeError) as e:
        st.query()
    assert e.value.code == code, e.value
    for b in out:
        assert np.all(b == SENTINEL), "a run with a routing error wrote to a receive buffer"
    assert st.query()["n_segments"] == 0  # reported once; the empty plan's stats remain


def test_routing_errors_found_on_device():
    wl = make_workload("tiny", weights=None)
    good = Case.from_workload(wl, seed=1)

    def variant(off=None, src=None, slot=None, rr=None):
        return Case(good.H, good.F, good.E_l, good.R, good.self_rank,
                    good.off if off is None else off, good.src if src is None else src,
                    good.slot if slot is None else slot, good.rr if rr is None else rr,
                    x=good.x, w=(good.w1, good.w3, good.w2))

    with stage_for(good, max_rows=good.rows) as st:
        off = good.off.copy(); off[1] = off[2] + 1
        _expect_device_error(st, variant(off=off), B.MOE_EROUTING)
        off = good.off.copy(); off[0] = 1
        _expect_device_error(st, variant(off=off), B.MOE_EROUTING)
        src = good.src.copy(); src[0] = -1
        _expect_device_error(st, variant(src=src), B.MOE_EROUTING)
        src = good.src.copy(); src[5] = good.R
        _expect_device_error(st, variant(src=src), B.MOE_EROUTING, serial=True)
        slot = good.slot.copy(); slot[2] = good.rr[good.src[2]]
        _expect_device_error(st, variant(slot=slot), B.MOE_EROUTING)
        # the same (rank, slot) in two experts
        e1 = int(good.off[1])
        i = next(j for j in range(e1, good.rows) if good.src[j] == good.src[0])
        slot = good.slot.copy(); slot[i] = good.slot[0]
        _expect_device_error(st, variant(slot=slot), B.MOE_EROUTING)
        # dispatch-order precondition: a rank's rows in two runs (the first row of expert 0 moved
        # to its end, behind other ranks' rows), and descending slots within a run
        lo, hi = int(good.off[0]), int(good.off[1])
        assert len(set(good.src[lo:hi].tolist())) > 1
        src = good.src.copy(); src[lo:hi] = np.roll(src[lo:hi], -1)
        slot = good.slot.copy(); slot[lo:hi] = np.roll(slot[lo:hi], -1)
        _expect_device_error(st, variant(src=src, slot=slot), B.MOE_EROUTING)
        slot = good.slot.copy(); slot[0], slot[1] = slot[1], slot[0]
        assert good.src[0] == good.src[1]
        _expect_device_error(st, variant(slot=slot), B.MOE_EROUTING)
        # a valid run on the same handle afterwards
        good.fill()
        st.run_devplan(*good.dev_args(), cu_split=8)
        good.out()
        st.query()
        assert_same_plan(st.plan(), host_tables(st, good, True), "after errors")
    with stage_for(good, max_rows=good.rows - 1) as st:
        _expect_device_error(st, good, B.MOE_ECAPACITY)


def test_argument_errors_enqueue_nothing():
    wl = make_workload("tiny", weights=None)
    c = Case.from_workload(wl, seed=1)
    with stage_for(c) as st:
        with pytest.raises(ValueError):
            st.run_devplan(c.x, c.off, c.src, c.slot, c.w1, c.w3, c.w2, c.bufs, c.rr)  # host routing
        rr = c.rr.copy(); rr[0] = -1
        with pytest.raises(B.MoeError) as e:
            st.run_devplan(c.x, c.d_off, c.d_src, c.d_slot, c.w1, c.w3, c.w2, c.bufs, rr)
        assert e.value.code == B.MOE_EINVAL
