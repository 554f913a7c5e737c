"""Exactly-once writes: with MOE_WRITE_COUNTS every store into a receive buffer (down epilogue, tail
kernel, consumer, drain, scatter) counts its 8-byte words against the logical row it belongs to.
Every routed row must receive exactly hidden / 4 words and every padding row none, whichever path,
split, segment size or plan builder ran -- including a run whose consumer gave up on its units (the
drain copies them) -- so no row is copied twice, e.g. by both the consumer and the drain.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, oracle_bufs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

RAGGED = dict(H=320, F=576, E_t=8, k=2, R=4, T_r=2048, E_l=2)


def check_counts(st, wl, what):
    counts = st.records(B.MOE_RECORDS_WRITES)
    rank = st.plan()["row_rank"]
    n = len(rank)
    want = np.where(rank >= 0, wl.H // 4, 0).astype(np.int64)
    got = counts[:n].astype(np.int64)
    bad = np.nonzero(got != want)[0]
    assert len(bad) == 0, (f"{what}: {len(bad)} logical rows written a wrong number of words, first {bad[:5]}: "
                           f"got {got[bad[:5]]}, want {want[bad[:5]]}")
    assert not counts[n:].any(), f"{what}: words counted past the plan's rows"
    log(f"{what}: {int((rank >= 0).sum())} routed rows written exactly once, {int((rank < 0).sum())} padding rows untouched")


def run(dw, st, path, cu_split=8, device_plan=False):
    dw.fill()
    wl = dw.wl
    if device_plan:
        d = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
             for a in (wl.expert_offsets, wl.row_src_rank, wl.row_slot)]
        args = (dw.x, *d, dw.w1, dw.w3, dw.w2, dw.bufs, dw.return_rows)
        if path == "serial":
            st.run_serial_devplan(*args)
        else:
            st.run_devplan(*args, cu_split=cu_split)
    elif path == "serial":
        st.run_serial(*dw.args())
    else:
        st.run(*dw.args(), cu_split=cu_split)
    return dw.host_bufs()


CASES = [
    # (name, flags, path, cu_split, band_rows, mgb, split_k, device_plan)
    ("overlapped shared c=8", B.MOE_SHARED_CUS, "overlapped", 8, 0, 1, 0, False),
    ("overlapped shared c=64", B.MOE_SHARED_CUS, "overlapped", 64, 0, 1, 0, False),
    ("overlapped shared c=248", B.MOE_SHARED_CUS, "overlapped", 248, 0, 1, 0, False),
    ("overlapped partitioned c=16", 0, "overlapped", 16, 0, 1, 0, False),
    ("overlapped band_rows=32 mgb=2", B.MOE_SHARED_CUS, "overlapped", 32, 32, 2, 0, False),
    ("overlapped split_k=3", B.MOE_SHARED_CUS, "overlapped", 32, 0, 1, 3, False),
    ("overlapped device-built plan", B.MOE_SHARED_CUS, "overlapped", 64, 0, 1, 0, True),
    ("serial", 0, "serial", 0, 0, 1, 0, False),
    ("serial device-built plan", 0, "serial", 0, 0, 1, 0, True),
    ("epilogue-direct ablation", B.MOE_DIRECT_ALL, "serial", 0, 0, 1, 0, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_every_routed_row_written_once(case):
    name, flags, path, cu, band, mgb, split, dev = case
    wl = make_workload("tiny", owner=1, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=band, mgb=mgb, split_k=split,
                    flags=B.MOE_LOCAL_DIRECT | B.MOE_WRITE_COUNTS | flags) as st:
        for i in range(2):   # the counts are per run
            out = run(dw, st, path, cu, dev)
            assert st.query()["timeout"] == 0
            check_counts(st, wl, f"{name} (run {i})")
    compare(out, ref)


def test_abandoned_units_written_once():
    """Flags suppressed: every consumer wave gives up on its unit after the watchdog, and the drain
    copies each abandoned unit exactly once."""
    wl = make_workload("tiny", owner=1, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, watchdog_ms=20,
                    flags=B.MOE_LOCAL_DIRECT | B.MOE_WRITE_COUNTS | B.MOE_TEST_NO_SIGNAL | B.MOE_SHARED_CUS) as st:
        out = run(dw, st, "overlapped", 32)
        q = st.query(check=False)
        assert q["rc"] == B.MOE_ETIMEOUT
        check_counts(st, wl, "expired consumer")
    compare(out, ref)


@pytest.mark.parametrize("name", ["mixtral", "large_fine"])
def test_fullsize_written_once(name):
    log(f"write counts {name}: generating")
    wl = make_workload(name)
    dw = DeviceWorkload(torch, wl)
    side = torch.cuda.Stream()
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_WRITE_COUNTS | B.MOE_SHARED_CUS) as st:
        for c in (64, 248):
            dw.fill()
            st.run(*dw.args(), cu_split=c, stream=side)
            torch.cuda.synchronize()
            assert st.query()["timeout"] == 0
            check_counts(st, wl, f"{name} overlapped c={c}")
        dw.fill()
        st.run_serial(*dw.args(), stream=side)
        torch.cuda.synchronize()
        st.query()
        check_counts(st, wl, f"{name} serial")
