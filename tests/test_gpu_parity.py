"""GPU parity of the HIP expert stage against the CPU oracle, through the C ABI.

Placement (which receive-buffer rows are written) is compared bit for bit;
values within |gpu - oracle| <= 1e-2 * max(1, |oracle|) elementwise, plus a
per-row relative L2 gate of 8e-3 (the paper's correctness tolerance,
Section 4.4).  Every output element comes from one tile with a fixed K order,
so results are also compared bitwise across launch configurations and
between the overlapped and the serial path.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, oracle_bufs, SENTINEL

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# A shape with ragged tiles: 320 = 256 + 64 hidden columns, 576 = 4 * 128 + 64 ffn features,
# several 256-row tile rows per expert and a partial last tile row.
RAGGED = dict(H=320, F=576, E_t=8, k=2, R=4, T_r=512, E_l=2)


def run_overlapped(dw, stage, cu_split=4):
    dw.fill()
    stage.run(*dw.args(), cu_split=cu_split)
    out = dw.host_bufs()
    st = stage.query()
    return out, st


def run_serial(dw, stage):
    dw.fill()
    stage.run_serial(*dw.args())
    out = dw.host_bufs()
    stage.query()
    return out


@pytest.mark.parametrize("owner", [0, 1, 2, 3])
def test_tiny_each_owner(owner):
    log(f"tiny owner={owner}")
    wl = make_workload("tiny", owner=owner)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=16) as st:
        out, stats = run_overlapped(dw, st, cu_split=4)
        compare(out, ref)
        assert stats["timeout"] == 0
        ser = run_serial(dw, st)
        for a, b in zip(out, ser):
            assert np.array_equal(a, b)


def test_tiny_all_owners_every_token_k_times():
    wl0 = make_workload("tiny", weights=None)
    bufs = None
    for owner in range(wl0.R):
        wl = make_workload("tiny", owner=owner)
        dw = DeviceWorkload(torch, wl)
        if bufs is not None:
            for b, h in zip(dw.bufs, bufs):
                b.copy_(torch.from_numpy(h.view(np.int16)))
        with make_stage(wl) as st:
            st.run(*dw.args(), cu_split=8)
            bufs = dw.host_bufs()
            st.query()
    for b in bufs:
        assert not np.any(np.all(b == SENTINEL, axis=1))
    ref = None
    for owner in range(wl0.R):
        wl = make_workload("tiny", owner=owner)
        r = oracle_bufs(wl)
        if ref is None:
            ref = r
        else:
            for a, o in zip(ref, r):
                m = ~np.all(o == SENTINEL, axis=1)
                a[m] = o[m]
    compare(bufs, ref)


@pytest.mark.parametrize("owner", [0, 3])
def test_ragged_multi_tile(owner):
    log(f"ragged owner={owner}")
    wl = make_workload("tiny", owner=owner, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    baseline = None
    for band_rows, mgb, split in ((16, 1, 2), (64, 2, 16), (32, 3, 64)):
        with make_stage(wl, band_rows=band_rows, mgb=mgb) as st:
            out, stats = run_overlapped(dw, st, cu_split=split)
            assert stats["n_tile_rows"] >= 3 and stats["timeout"] == 0
            compare(out, ref)
            if baseline is None:
                baseline = out
                with make_stage(wl, band_rows=band_rows) as st2:
                    ser = run_serial(dw, st2)
                for a, b in zip(out, ser):
                    assert np.array_equal(a, b)
            for a, b in zip(out, baseline):
                assert np.array_equal(a, b), "output depends on the launch configuration"


def test_local_rows_through_consumer():
    """Without LOCAL_DIRECT the local group is staged and copied by the consumer as well."""
    wl = make_workload("tiny", owner=2, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=32, flags=0) as st:
        out, stats = run_overlapped(dw, st, cu_split=8)
    compare(out, ref)


def test_poison_mode_catches_no_early_copy():
    """Staged output poisoned with NaN before the run: a copy racing its data would deliver NaN."""
    wl = make_workload("tiny", owner=1, overrides=dict(RAGGED, T_r=2048))
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=16, flags=B.MOE_LOCAL_DIRECT | B.MOE_POISON) as st:
        for split in (1, 8):
            out, _ = run_overlapped(dw, st, cu_split=split)
            compare(out, ref)


def test_direct_all_matches_serial():
    """MOE_DIRECT_ALL (no-consumer ablation): the down epilogue writes every row to its slot and
    no scatter runs; the output is bitwise the serial path's and within tolerance of the oracle."""
    wl = make_workload("tiny", owner=3, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=16) as st:
        ser = run_serial(dw, st)
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_DIRECT_ALL | B.MOE_KERNEL_TIMING) as st:
        out = run_serial(dw, st)
        t = st.times()
        assert t["runs"] == 1 and t["scatter_ms"] < 0.01  # nothing between the down launch and the end
    compare(out, ref)
    for a, b in zip(out, ser):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("split_k", [2, 3, 5, 9])
def test_split_k_down_tiles(split_k):
    """Down tiles split into K parts (9 K steps of 64 here, so parts of 1..5 steps, uneven for 2
    and 5, a single step each for 9):
    within tolerance of the oracle, bitwise equal between the overlapped and the serial path of
    one handle (the parts are added in part order whichever part finishes last), and poisoned
    staging shows no tile was published before its last part."""
    log(f"split_k={split_k}")
    wl = make_workload("tiny", owner=2, overrides=dict(RAGGED, T_r=1024))
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=16, flags=B.MOE_LOCAL_DIRECT | B.MOE_POISON, split_k=split_k) as st:
        out, stats = run_overlapped(dw, st, cu_split=8)
        assert stats["split_k"] == split_k and stats["timeout"] == 0
        assert stats["n_down_items"] == stats["n_tile_rows"] * 2 * split_k
        compare(out, ref)
        again, _ = run_overlapped(dw, st, cu_split=8)
        ser = run_serial(dw, st)
        for a, b, c in zip(out, again, ser):
            assert np.array_equal(a, b) and np.array_equal(a, c)
    with make_stage(wl, band_rows=16, split_k=1) as st:
        whole, _ = run_overlapped(dw, st, cu_split=8)
    compare(whole, ref)


@pytest.mark.parametrize("local_direct", [True, False])
def test_shared_cus_matches_partitioned(local_direct):
    """MOE_SHARED_CUS: the producer also runs on the consumer's CUs; results are bitwise those
    of the partitioned launch, and poisoned staging shows no copy ran ahead of its flag."""
    log(f"shared cus local_direct={local_direct}")
    wl = make_workload("tiny", owner=1, overrides=dict(RAGGED, T_r=2048))
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    base = B.MOE_LOCAL_DIRECT if local_direct else 0
    with make_stage(wl, band_rows=16, flags=base) as st:
        part, _ = run_overlapped(dw, st, cu_split=8)
    compare(part, ref)
    side = torch.cuda.Stream()
    with make_stage(wl, band_rows=16, flags=base | B.MOE_SHARED_CUS | B.MOE_POISON) as st:
        # Null stream: the producer forks to the handle's stream.  Created stream: the
        # producer runs on it directly, beside the consumer's CU-masked stream.
        for stream, split in ((None, 1), (None, 8), (side, 8), (side, 32), (None, 248), (side, 248)):
            dw.fill()
            torch.cuda.synchronize()
            st.run(*dw.args(), cu_split=split, stream=stream)
            torch.cuda.synchronize()
            out = dw.host_bufs()
            stats = st.query()
            assert stats["timeout"] == 0
            assert stats["producer_grid"] >= 256 and stats["consumer_cus"] >= 8
            compare(out, ref)
            for a, b in zip(out, part):
                assert np.array_equal(a, b)


@pytest.mark.parametrize("kind", ["identity", "zero_w1", "zero_w3", "zero_w2"])
def test_special_weights(kind):
    wl = make_workload("tiny", owner=0, weights=kind)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl) as st:
        out, _ = run_overlapped(dw, st, cu_split=4)
    compare(out, ref)
    if kind.startswith("zero"):
        for r in range(wl.R):
            m = wl.row_src_rank == r
            v = out[r][wl.row_slot[m]]
            assert np.all((v == 0) | (v == 0x8000))   # +0 or -0


def test_capacity_slack_untouched():
    wl = make_workload("tiny", owner=3)
    dw = DeviceWorkload(torch, wl, extra_rows=9)
    ref = oracle_bufs(wl, extra_rows=9)
    with make_stage(wl) as st:
        out, _ = run_overlapped(dw, st, cu_split=4)
    compare(out, ref)


def test_empty_run_writes_nothing():
    wl = make_workload("tiny", owner=0)
    dw = DeviceWorkload(torch, wl)
    off = np.zeros(wl.E_l + 1, np.int32)
    z = np.zeros(0, np.int32)
    with make_stage(wl) as st:
        st.run(dw.x, off, z, z, dw.w1, dw.w3, dw.w2, dw.bufs, dw.return_rows, cu_split=4)
        st.run_serial(dw.x, off, z, z, dw.w1, dw.w3, dw.w2, dw.bufs, dw.return_rows)
        st.query()
    for b in dw.host_bufs():
        assert np.all(b == SENTINEL)


def test_invalid_routing_enqueues_nothing():
    wl = make_workload("tiny", owner=0)
    dw = DeviceWorkload(torch, wl)
    bad = wl.row_slot.copy()
    bad[0] = bad[1]
    bad_src = wl.row_src_rank.copy()
    bad_src[0] = bad_src[1]
    with make_stage(wl) as st:
        with pytest.raises(B.MoeError) as ei:
            st.run(dw.x, wl.expert_offsets, bad_src, bad, dw.w1, dw.w3, dw.w2, dw.bufs, dw.return_rows,
                   cu_split=4)
        assert ei.value.code == B.MOE_EROUTING
        for bad_split in (-1, 10 ** 6):   # 0 asks for the adaptive selector, negative is invalid
            with pytest.raises(B.MoeError) as ei:
                st.run(*dw.args(), cu_split=bad_split)
            assert ei.value.code == B.MOE_EUNSUPPORTED
    for b in dw.host_bufs():
        assert np.all(b == SENTINEL)


def test_repeated_runs_reuse_flags_across_epochs():
    wl = make_workload("tiny", owner=1, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, band_rows=32) as st:
        for i in range(5):
            dw.fill()
            st.run(*dw.args(), cu_split=4 + 4 * (i % 2))
        out = dw.host_bufs()
        st.query()
    compare(out, ref)


@pytest.mark.parametrize("mode", ["shared", "partitioned"])
def test_alternating_inputs_read_fresh_staged_rows(mode):
    """Runs on one handle alternate two activation sets under the same routing, so every run
    stages its rows at the same addresses and raises the same flags.  A copy that read a staged
    row still cached from the previous run would deliver the other input's value: each run must
    match its own oracle output and be bitwise equal to the serial path on the same input."""
    import copy
    log(f"alternating inputs, {mode} compute units")
    wl_a = make_workload("tiny", owner=1, overrides=dict(RAGGED, T_r=2048))
    wl_b = copy.copy(wl_a)
    wl_b.dispatched_x = (wl_a.dispatched_x ^ np.uint16(0x8000)).astype(np.uint16)  # -x exactly
    dws = [DeviceWorkload(torch, wl) for wl in (wl_a, wl_b)]
    refs = [oracle_bufs(wl) for wl in (wl_a, wl_b)]
    sers = []
    # Unaligned layout (band_rows 1): serial and overlapped plans then split the same tile rows,
    # so their outputs are bitwise equal.
    with make_stage(wl_a) as st:
        for dw in dws:
            sers.append(run_serial(dw, st))
    flags = B.MOE_LOCAL_DIRECT | (B.MOE_SHARED_CUS if mode == "shared" else 0)
    with make_stage(wl_a, flags=flags) as st:
        for i in range(6):
            out, stats = run_overlapped(dws[i % 2], st, cu_split=(8, 32)[(i // 2) % 2])
            assert stats["timeout"] == 0
            compare(out, refs[i % 2])
            for a, b in zip(out, sers[i % 2]):
                assert np.array_equal(a, b), f"run {i}: overlapped differs from serial on its own input"


def test_consumer_only_copies_staged_rows():
    """MOE_TEST_CONSUMER_ONLY (copy-ceiling measurement): no producer work, every flag published
    by the run's reset, so the consumer copies the staged output -- zeros on a fresh handle --
    into every remote slot and leaves local slots (written by the producer otherwise) alone."""
    wl = make_workload("tiny", owner=2, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS | B.MOE_TEST_CONSUMER_ONLY) as st:
        out, stats = run_overlapped(dw, st, cu_split=8)
        assert stats["timeout"] == 0 and stats["n_segments"] > 0
    for r, b in enumerate(out):
        mine = wl.row_slot[wl.row_src_rank == r]
        if r == wl.self_rank:
            assert np.all(b[mine] == SENTINEL)
        else:
            assert np.all(b[mine] == 0)
        other = np.setdiff1d(np.arange(b.shape[0]), mine)
        assert np.all(b[other] == SENTINEL)


def test_auto_cu_split_settles_and_keeps_results():
    """cu_split = 0: the handle measures its own runs at several consumer splits, settles on
    one, and the output stays bitwise that of a fixed split (results never depend on it)."""
    wl = make_workload("tiny", owner=0, overrides=RAGGED)
    dw = DeviceWorkload(torch, wl)
    ref = oracle_bufs(wl)
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS) as st:
        fixed, _ = run_overlapped(dw, st, cu_split=8)
    compare(fixed, ref)
    seen = set()
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS) as st:
        for i in range(20):
            out, stats = run_overlapped(dw, st, cu_split=0)   # synchronises: every run measured
            seen.add(stats["consumer_cus"])
            for a, b in zip(out, fixed):
                assert np.array_equal(a, b)
        assert stats["auto_cu_split"] in (32, 64, 128, 248)
        assert stats["consumer_cus"] == stats["auto_cu_split"]
    assert seen >= {32, 64, 128, 248}
    # A reserved partition takes its CUs from the producer: the candidates stay small.
    seen = set()
    with make_stage(wl, flags=B.MOE_LOCAL_DIRECT) as st:
        for i in range(20):
            out, stats = run_overlapped(dw, st, cu_split=0)
            seen.add(stats["consumer_cus"])
            for a, b in zip(out, fixed):
                assert np.array_equal(a, b)
        assert stats["auto_cu_split"] in (8, 16, 32, 64)
    assert seen >= {8, 16, 32, 64}
    with make_stage(wl) as st:
        st.run_serial(*dw.args())
        assert st.query()["auto_cu_split"] == -1
