"""In-kernel timestamps and placement records (MOE_TIMESTAMPS) through the C ABI.

The records must be complete and consistent with the protocol of paper Section 3.3: every
copy unit is recorded once; a unit starts copying only after every ready flag of its segment
was raised (the tile's raise time precedes the consumer's observation of it) and finishes
after it starts; the producer's span covers its launches.  They also show where the kernels
ran (Section 3.3.3): with a reserved partition the consumer's waves stay on at most
consumer_cus compute units, none of which runs a producer workgroup; with shared compute units
the producer covers the whole GPU.  Results are unchanged by recording.
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, oracle_bufs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# The GPU wall clock is one 100 MHz counter; a reading taken after observing a flag can trail the
# writer's reading by up to a tick of skew between compute units.
SKEW_TICKS = 2


def cu_keys(hw, xcc):
    return {(int(x) & 0xF, (int(h) >> 8) & 0xFF) for h, x in zip(hw, xcc)}


def run_recorded(wl, flags, cu_split, mgb=1):
    dw = DeviceWorkload(torch, wl)
    side = torch.cuda.Stream()
    with make_stage(wl, flags=flags | B.MOE_TIMESTAMPS, mgb=mgb) as st:
        st.run(*dw.args(), cu_split=cu_split, stream=side)
        torch.cuda.synchronize()
        stats = st.query()
        rec = {"span": st.records(B.MOE_RECORDS_SPAN)[0], "copy": st.records(B.MOE_RECORDS_COPY),
               "wg": st.records(B.MOE_RECORDS_PRODUCER), "tiles": st.records(B.MOE_RECORDS_TILES),
               "plan": st.plan(), "stats": stats}
    return dw, rec


def check_protocol(rec):
    span, cp, wg, tiles, segs = rec["span"], rec["copy"], rec["wg"], rec["tiles"], rec["plan"]["segments"]
    stats = rec["stats"]
    n_units = int(span["copy_units"])
    assert n_units == stats["copy_units"] > 0
    assert len(cp) == min(n_units, 1 << 18)
    # every unit of every segment recorded exactly once
    per_seg = np.bincount(cp["segment"], minlength=len(segs))
    assert per_seg.min() >= 1 and per_seg.sum() == len(cp)
    pairs = set(zip(cp["segment"].tolist(), cp["part"].tolist()))
    assert len(pairs) == len(cp)
    assert np.all(cp["t_poll"] <= cp["t_ready"]) and np.all(cp["t_ready"] <= cp["t_done"])
    assert set(np.unique(cp["source"]).tolist()) <= {0, 1}
    # the drain launch starts after the producer's last launch: its units start copying after it ended
    dr = cp["source"] == 1
    if dr.any():
        assert int(cp["t_ready"][dr].min()) + SKEW_TICKS >= int(span["producer_end"])
    # a unit starts after every flag of its segment was raised
    for s in range(len(segs)):
        fb, fc = int(segs[s, 4]), int(segs[s, 5])
        raised = tiles[fb:fb + fc]
        assert np.all(raised > 0), f"segment {s}: a flag it waited for was never raised"
        m = cp["segment"] == s
        assert int(cp["t_ready"][m].min()) + SKEW_TICKS >= int(raised.max()), f"segment {s} copied before its flag"
    grid = int(span["producer_grid"])
    assert len(wg) == 2 * grid
    assert np.all(wg["launch"][:grid] == 0) and np.all(wg["launch"][grid:] == 1)
    assert int(wg["items"][:grid].sum()) == stats["n_gu_items"]
    assert int(wg["items"][grid:].sum()) == stats["n_down_items"]
    p0, p1 = int(span["producer_start"]), int(span["producer_end"])
    assert p0 == int(wg["t_start"][:grid].min()) and p1 >= int(wg["t_end"][grid:].max())
    assert p1 >= int(tiles.max())


@pytest.mark.timeout(300)
@pytest.mark.parametrize("shape", ["tiny", "ragged"])
def test_records_follow_the_protocol_and_keep_results(shape):
    if shape == "tiny":
        wl = make_workload("tiny", owner=1)
    else:
        wl = make_workload("tiny", overrides={"H": 320, "F": 576, "T_r": 400}, owner=2)
    dw, rec = run_recorded(wl, B.MOE_LOCAL_DIRECT | B.MOE_SHARED_CUS, 16)
    log(f"{shape}: units={rec['stats']['copy_units']} segments={rec['stats']['n_segments']} "
        f"span={(int(rec['span']['producer_end']) - int(rec['span']['producer_start'])) / 100:.1f} us")
    check_protocol(rec)
    compare(dw.host_bufs(), oracle_bufs(wl))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("mode", ["partitioned", "shared"])
def test_consumer_stays_on_its_compute_units(mode):
    """Where the waves ran, from the HW_ID and XCC_ID registers (mixtral-sized ranks so every
    producer workgroup has work in both launches)."""
    wl = make_workload("layer_e8")
    c = 32
    flags = B.MOE_LOCAL_DIRECT | (B.MOE_SHARED_CUS if mode == "shared" else 0)
    dw, rec = run_recorded(wl, flags, c)
    check_protocol(rec)
    stats, cp, wg = rec["stats"], rec["copy"], rec["wg"]
    grid = int(rec["span"]["producer_grid"])
    drained = int((cp["source"] == 1).sum())
    cp = cp[cp["source"] == 0]        # units the drain copied after the producer ran anywhere
    cons = cu_keys(cp["hw_id"], cp["xcc_id"])
    prod = cu_keys(wg["hw_id"][grid:], wg["xcc_id"][grid:]) | cu_keys(wg["hw_id"][:grid], wg["xcc_id"][:grid])
    per_xcd = np.bincount([k[0] for k in cons], minlength=8)
    se = {}
    for x, key in cons:
        se.setdefault(x, set()).add(key >> 5)       # shader engine (HW_ID bits 15:13)
    log(f"{mode}: units={len(rec['copy'])} drained={drained}; consumer_cus={stats['consumer_cus']} used={len(cons)} "
        f"per XCD {per_xcd.tolist()}; shader engines "
        f"per XCD {[len(se.get(x, ())) for x in range(8)]}; producer grid={grid} CUs={len(prod)} shared={len(cons & prod)}")
    assert len(cons) <= stats["consumer_cus"]
    if mode == "partitioned":
        assert grid == 256 - stats["consumer_cus"]
        assert len(prod) == grid          # one producer workgroup per compute unit
        assert not (cons & prod), "a consumer wave ran on a producer compute unit"
    else:
        assert grid == 256 and len(prod) == 256
        assert cons <= prod
        # at most two copying consumer waves per SIMD (wave slots of one SIMD key)
        slots = {}
        for h, x in zip(cp["hw_id"], cp["xcc_id"]):
            key = (int(x) & 0xF, (int(h) >> 4) & 0xFFF)
            slots.setdefault(key, set()).add(int(h) & 0xF)
        assert max(len(v) for v in slots.values()) <= 2, max(len(v) for v in slots.values())
