"""The no-allocation entry point (moe_stage_run_serial_static) through the C ABI.

Its output must equal, bit for bit, that of moe_stage_run_serial_devplan on a handle of the same
configuration (the same kernels over workspaces in the library's fixed per-GPU array), on two
calls in a row, the second with a smaller routing, and stay within the oracle's tolerance."""
import ctypes

import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload
from tests.gpu_helpers import DeviceWorkload, compare, log, make_stage, oracle_bufs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def dev_routing(wl):
    return [torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
            for a in (wl.expert_offsets, wl.row_src_rank, wl.row_slot)]


@pytest.mark.timeout(300)
def test_static_entry_point_matches_the_handle():
    full = make_workload("tiny", overrides={"H": 320, "F": 576, "T_r": 200}, owner=1)
    small = full.subset(np.arange(0, full.rows, 3))          # the second call: a third of the rows
    cfg = B.make_config(full.H, full.F, full.E_l, full.R, full.self_rank, full.rows)
    for i, wl in enumerate((full, small)):
        dw = DeviceWorkload(torch, wl)
        x, w1, w3, w2 = dw.x, dw.w1, dw.w3, dw.w2
        routing = dev_routing(wl)
        B.moe_stage_run_serial_static(cfg, x, *routing, w1, w3, w2, dw.bufs, dw.return_rows)
        torch.cuda.synchronize()
        got = [b.clone() for b in dw.bufs]
        dw.fill()
        with make_stage(wl, max_rows=full.rows) as st:
            st.run_serial_devplan(x, *routing, w1, w3, w2, dw.bufs, dw.return_rows)
            st.query()
        torch.cuda.synchronize()
        for a, b in zip(got, dw.bufs):
            assert torch.equal(a, b), f"call {i}: static entry point differs from the handle"
        worst, _ = compare(dw.host_bufs(), oracle_bufs(wl))
        log(f"call {i}: rows={wl.rows} equal to the handle's output, max scaled err vs oracle {worst:.2e}")


def test_static_entry_point_rejects_configurations_past_its_array():
    # hidden 7168 x ffn 2048 with 65536 rows needs far more than the fixed array
    cfg = B.make_config(7168, 2048, 32, 8, 0, 65536)
    z = torch.zeros(1, dtype=torch.int32, device="cuda")
    rc = B.load().moe_stage_run_serial_static(ctypes.byref(cfg), 16, z.data_ptr(), z.data_ptr(), z.data_ptr(),
                                              16, 16, 16, None, None, None)
    assert rc == B.MOE_ECAPACITY
    assert "static array" in B.moe_stage_last_error(None)
