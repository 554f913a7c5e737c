"""Helpers for the GPU parity tests: upload a workload, run the library, compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import bf16_bits_to_f32

SENTINEL = 0x7FC1  # bf16 quiet-NaN pattern the stage never produces


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_u16(torch, a: np.ndarray):
    """Device tensor holding the bf16 bit patterns of a uint16 array."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda")


class DeviceWorkload:
    def __init__(self, torch, wl, extra_rows: int = 0):
        self.torch = torch
        self.wl = wl
        self.x = dev_u16(torch, wl.dispatched_x)
        self.w1 = dev_u16(torch, wl.w1)
        self.w3 = dev_u16(torch, wl.w3)
        self.w2 = dev_u16(torch, wl.w2)
        self.return_rows = (wl.return_rows + extra_rows).astype(np.int64)
        self.bufs = [torch.empty((int(n), wl.H), dtype=torch.int16, device="cuda") for n in self.return_rows]
        self.fill()

    def fill(self, value: int = SENTINEL):
        v = value - 65536 if value >= 32768 else value
        for b in self.bufs:
            b.fill_(v)

    def args(self):
        wl = self.wl
        return (self.x, wl.expert_offsets, wl.row_src_rank, wl.row_slot, self.w1, self.w3, self.w2, self.bufs,
                self.return_rows)

    def host_bufs(self):
        self.torch.cuda.synchronize()
        return [b.cpu().numpy().view(np.uint16) for b in self.bufs]


def make_stage(wl, band_rows=0, mgb=1, flags=B.MOE_LOCAL_DIRECT, watchdog_ms=0, max_rows=None, split_k=0):
    return B.MoeStage(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, max_rows or max(wl.rows, 1), band_rows, mgb,
                      flags, watchdog_ms, split_k)


def oracle_bufs(wl, extra_rows: int = 0, threads: int = 0):
    from oracle import oracle as orc
    bufs = [np.full((int(n) + extra_rows, wl.H), SENTINEL, np.uint16) for n in wl.return_rows]
    rc = orc.get().run(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.dispatched_x, wl.expert_offsets,
                       wl.row_src_rank, wl.row_slot, wl.w1, wl.w3, wl.w2, bufs, wl.return_rows + extra_rows,
                       threads)
    assert rc == 0, rc
    return bufs


def compare(gpu, ref, rel_l2=8e-3):
    """Bit-exact placement; values within |g - o| <= 1e-2 max(1, |o|); per-row relative L2 gate."""
    worst = 0.0
    worst_rel = 0.0
    for r, (g, o) in enumerate(zip(gpu, ref)):
        assert g.shape == o.shape
        g_sent = np.all(g == SENTINEL, axis=1)
        o_sent = np.all(o == SENTINEL, axis=1)
        assert np.array_equal(g_sent, o_sent), f"rank {r}: written slots differ"
        if not np.any(~o_sent):
            continue
        gv = bf16_bits_to_f32(g[~o_sent]).astype(np.float64)
        ov = bf16_bits_to_f32(o[~o_sent]).astype(np.float64)
        assert np.all(np.isfinite(gv)), f"rank {r}: non-finite output"
        err = np.abs(gv - ov) / np.maximum(1.0, np.abs(ov))
        worst = max(worst, float(err.max()))
        assert err.max() <= 1e-2, f"rank {r}: max scaled error {err.max():.3e}"
        rel = np.linalg.norm(gv - ov, axis=1) / np.maximum(np.linalg.norm(ov, axis=1), 1e-30)
        worst_rel = max(worst_rel, float(rel.max()))
        assert rel.max() <= rel_l2, f"rank {r}: per-row relative L2 {rel.max():.3e}"
    return worst, worst_rel


def sub_workload(wl, rows_idx):
    """The same stage restricted to a subset of routed rows (for sampled full-size checks)."""
    return wl.subset(rows_idx)
