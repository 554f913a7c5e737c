"""Full-size GPU parity at the workload sizes the benchmark uses, in its launch configuration.

The oracle computes a seeded sample of routed rows one by one; placement (every
routed slot written, nothing else touched) and serial == overlapped bitwise are
checked on every row, since they hold at any size.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, oracle_bufs, SENTINEL

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

BENCH_CU_SPLIT = 248
BENCH_FLAGS = B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS   # bench.py's default mode, on its own stream
SAMPLE_ROWS = 24


def written_mask(buf_dev):
    s = SENTINEL - 65536
    return (~(buf_dev == s).all(dim=1)).cpu().numpy()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["mixtral", "mixtral_zipf", "fine", "large_fine"])
def test_fullsize_sampled(name):
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
        log(f"full-size {name}: overlapped done, segments={stats['n_segments']} tiles={stats['n_tile_rows']} "
            f"split_k={stats['split_k']} workgroups={stats['gu_workgroups']}/{stats['down_workgroups']}")
        assert stats["timeout"] == 0
        # placement on every row: exactly the routed slots are written
        for r in range(wl.R):
            want = np.zeros(int(dw.return_rows[r]), bool)
            want[wl.row_slot[wl.row_src_rank == r]] = True
            assert np.array_equal(written_mask(dw.bufs[r]), want), f"rank {r} placement"
        over = [b.clone() for b in dw.bufs]
        # A narrow consumer: four copy units per segment, far more than its waves, so most
        # units are claimed from the counter after each wave's fixed first one.
        dw.fill()
        torch.cuda.synchronize()
        st.run(*dw.args(), cu_split=8, stream=side)
        torch.cuda.synchronize()
        narrow = st.query()
        log(f"full-size {name}: c=8 units={4 * narrow['n_segments']} consumer waves={4 * narrow['consumer_grid']}")
        assert narrow["timeout"] == 0
        for a, b in zip(over, dw.bufs):
            assert torch.equal(a, b), "consumer splits differ"
        dw.fill()
        torch.cuda.synchronize()
        st.run_serial(*dw.args(), stream=side)
        torch.cuda.synchronize()
        st.query()
        for a, b in zip(over, dw.bufs):
            assert torch.equal(a, b), "serial and overlapped differ"
        del over
    # values on a seeded sample of rows, against the oracle row by row
    sub = wl.sample(SAMPLE_ROWS, seed=3)
    ref = oracle_bufs(sub)
    got = []
    for r in range(wl.R):
        g = np.full((int(wl.return_rows[r]), wl.H), SENTINEL, np.uint16)
        slots = sub.row_slot[sub.row_src_rank == r]
        if len(slots):
            idx = torch.from_numpy(slots.astype(np.int64)).to("cuda")
            g[slots] = dw.bufs[r].index_select(0, idx).cpu().numpy().view(np.uint16)
        got.append(g)
    worst, worst_rel = compare(got, ref)
    log(f"full-size {name}: sampled max scaled err {worst:.2e}, max row rel-L2 {worst_rel:.2e}")


@pytest.mark.timeout(300)
def test_watchdog_expiry_is_reported():
    """With ready flags suppressed from the host, the consumer's bounded wait expires, the
    kernels exit, the run reports MOE_ETIMEOUT, and the next run on a fresh handle is correct."""
    wl = make_workload("tiny", owner=1)
    dw = DeviceWorkload(torch, wl)
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_TEST_NO_SIGNAL, watchdog_ms=20) as st:
        st.run(*dw.args(), cu_split=8)
        q = st.query(check=False)
        assert q["rc"] == B.MOE_ETIMEOUT and q["timeout"] == 1
        assert st.query()["timeout"] == 0   # reported once
    ref = oracle_bufs(wl)
    with make_stage(wl) as st:
        dw.fill()
        st.run(*dw.args(), cu_split=8)
        st.query()
    compare(dw.host_bufs(), ref)
