#!/usr/bin/env python3
"""Benchmark of the MI355X MoE expert stage (one expert-parallel rank, one GPU).

A step is one overlapped expert-stage run (moe_stage_run): host plan build and
upload, the persistent gated-FFN producer (gate/up launch, then the signaling
down launch) and the CU-confined consumer copying finished segments into the
per-source-rank receive buffers.  Inputs (activations, weights, receive
buffers) are resident in HBM before the timed region; the routing arrays are
host inputs by design of the C ABI, so each step re-validates and re-uploads
the plan.

The LAST stdout line is one compact JSON object (the headline: ``value`` is the
stage's algorithmic bf16 throughput, 6*H*F flops per routed row, padding
excluded, in TFLOP/s on the headline workload; ``ms_per_step`` its expert-stage
time; ``overlap_speedup`` serial / overlapped; ``roofline`` the gate/up launch
against the bf16 dense peak; ``cpu_baseline`` the CPU oracle).  Everything else
-- per-workload serial / overlapped / device-planned / ablation timings, the
consumer CU-split sweep in both CU modes and both segment sizes, the consumer
copy ceiling, the overlap ratio and flag latencies from in-kernel timestamps,
the compute units each kernel ran on, the band_rows = 256 layout and the
expert-count sweep -- goes to the ``--detail-out`` JSON file, which earlier
stdout lines name.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE expert-stage µs + bf16 MFMA TFLOP/s vs peak; overlap speedup vs serial"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA peak
PEAK_HBM_GBS = 8000.0
TICK_US = 0.01              # the GPU wall clock runs at 100 MHz
KERNEL_SRC = os.path.join(ROOT, "paper_2607_19539_amd", "csrc", "kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "producer_mixtral_traffic.md")

DESCRIPTIONS = {
    "tiny": "tiny: H256 F512, SiLU-gated FFN, 8 experts top-2, 4 source ranks x 64 tokens, 2 local experts",
    "mixtral": "mixtral: H4096 F14336, SiLU-gated FFN, 8 experts top-2, 4 source ranks x 4096 tokens, "
               "2 local experts, uniform router",
    "mixtral_zipf": "mixtral_zipf: mixtral shapes, Zipf(1.2) expert popularity (this rank owns the two hottest)",
    "fine": "fine: H2048 F1408, 64 experts top-6, 4 source ranks x 8192 tokens, 16 local experts",
    "large_fine": "large_fine: H7168 F2048, 256 experts top-8, 8 source ranks x 4096 tokens, 32 local experts",
}
for _e in (4, 8, 16, 32, 64):
    DESCRIPTIONS[f"layer_e{_e}"] = (f"layer_e{_e}: H1024 F4096, {4 * _e} experts top-2, 4 source ranks x 8192 tokens, "
                                    f"{_e} local experts (expert-count sweep)")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--warm-s", type=float, default=1.5,
                    help="warm-up time floor of the headline timings (after --warmup steps, runs continue until "
                         "this many seconds have passed, so the clocks have settled whatever --warmup is)")
    ap.add_argument("--warm-s-other", type=float, default=0.4, help="the same floor for every other timing")
    ap.add_argument("--workload", default="mixtral", choices=sorted(DESCRIPTIONS), help="headline workload")
    ap.add_argument("--extra-workloads", default="tiny,mixtral_zipf,fine,large_fine",
                    help="further workloads measured into the detail file ('' = none)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cu-split", type=int, default=64,
                    help="consumer compute units of the headline path (a quarter of the GPU, one wave per SIMD)")
    ap.add_argument("--mode", choices=["shared", "partitioned"], default="shared",
                    help="shared: the producer keeps every CU and the consumer runs beside it on its "
                         "cu_split CUs; partitioned: the consumer's CUs are reserved for it")
    ap.add_argument("--band-rows", type=int, default=0, help="tb_M of the row layout (0 = 1, no alignment)")
    ap.add_argument("--split-k", type=int, default=0, help="K parts per down tile (0 = library default)")
    ap.add_argument("--mgb", type=int, default=1, help="tile-row pieces per middle transfer segment")
    ap.add_argument("--small", default="4,8,16,24,32",
                    help="small consumer partitions (paper's range): measured in both CU modes and mgb 1 and 2 "
                         "(a partition owns CUs on every XCD, so requests round up to multiples of 8)")
    ap.add_argument("--grid", default="2,4,6,8,10,12,14,16,18,20,22,24,26,28,30,32",
                    help="consumer CU requests of the large_fine shared-CU grid (the paper's consumer-CTA grid)")
    ap.add_argument("--sweep", default="64,128,248", help="further shared-CU splits of the sweep")
    ap.add_argument("--copy-curve", default="8,16,32,64,128",
                    help="consumer CU counts for the consumer-only copy ceiling ('' to skip)")
    ap.add_argument("--esweep", default="4,8,16,32,64",
                    help="experts per rank for the single-layer expert-count sweep ('' to skip)")
    ap.add_argument("--only", choices=["all", "serial", "overlapped", "copy"], default="all",
                    help="time only one path of the headline workload, or only its consumer-only copy "
                         "curve (profiler runs)")
    ap.add_argument("--detail-out", default=os.path.join("gpurun_out", "bench_detail.json"))
    ap.add_argument("--esweep-child", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    return ap.parse_args()


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, target_s, threads=None):
    """Time the CPU oracle on a bounded sample of the workload's routed rows."""
    from oracle import oracle as orc
    if threads is None:
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    o = orc.get()

    def run(n):
        sub = wl.sample(n)
        bufs = [np.zeros((int(r), wl.H), np.uint16) for r in wl.return_rows]
        t0 = time.perf_counter()
        rc = o.run_workload(sub, bufs, threads)
        dt = time.perf_counter() - t0
        assert rc == 0, rc
        return sub.rows, dt

    n0, t_probe = run(max(threads, 4))
    rate = n0 / max(t_probe, 1e-6)                         # rows per second
    n = int(min(wl.rows, max(n0, rate * target_s)))
    n, dt = run(n)
    flops = 6.0 * wl.H * wl.F * n
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{n} of {wl.rows} routed rows ({n / wl.rows:.1%}) of {wl.name}, {dt:.1f} s wall; the full "
                      f"stage would take ~{dt * wl.rows / n:.0f} s on these cores"}


def stored_traffic():
    """HBM bytes per gate/up launch from the committed counter summary, if it was taken on the
    current kernel source (its sha256 is recorded next to the figure); else None."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    m_b = re.search(r"^traffic_bytes_per_launch:\s*([0-9.eE+]+)", text, re.M)
    m_h = re.search(r"^kernel_sha256:\s*([0-9a-f]{64})", text, re.M)
    if not m_b or not m_h:
        return None
    cur = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    return float(m_b.group(1)) if cur == m_h.group(1) else None


def union_length(iv):
    """Total length of the union of intervals [(a, b)], and the sorted disjoint pieces."""
    pieces = []
    for a, b in sorted(iv):
        if pieces and a <= pieces[-1][1]:
            pieces[-1][1] = max(pieces[-1][1], b)
        else:
            pieces.append([a, b])
    return sum(b - a for a, b in pieces), pieces


def cu_key(hw_id, xcc):
    """A compute unit's identity from the HW_ID register (CU, shader array, shader engine) and XCD."""
    return (int(xcc) & 0xF, (int(hw_id) >> 8) & 0xFF)


def producer_clocks(wg, grid, cons_cu=None):
    """Mean shader clock (GHz) of each producer launch from its workgroups' records: cycles over
    wall-clock ticks, summed over the workgroups that took work.  With a consumer CU set, the
    down launch's figure is also split into workgroups on those compute units and the rest."""
    out = {}
    for name, sl in (("gate_up", slice(0, grid)), ("down", slice(grid, 2 * grid))):
        w = wg[sl]
        w = w[w["items"] > 0]
        dt = (w["t_end"].astype(np.int64) - w["t_start"].astype(np.int64)).sum()
        out[name] = round(float(w["cycles"].astype(np.float64).sum() / dt / TICK_US * 1e-3), 3) if dt > 0 else None
    if cons_cu:
        w = wg[grid:2 * grid]
        w = w[w["items"] > 0]
        on = np.array([cu_key(h, x) in cons_cu for h, x in zip(w["hw_id"], w["xcc_id"])], bool)
        for key, m in (("down_on_consumer_cus", on), ("down_elsewhere", ~on)):
            dt = (w["t_end"][m].astype(np.int64) - w["t_start"][m].astype(np.int64)).sum()
            out[key] = round(float(w["cycles"][m].astype(np.float64).sum() / dt / TICK_US * 1e-3), 3) if dt > 0 else None
    return out


def overlap_analysis(B, stg, wl):
    """Overlap of the return copy with the expert compute (paper Section 4.2.2, Fig. 5b) from the
    last run's in-kernel timestamps: the share of the consumer's busy time (the union of its copy
    intervals) that lies inside the producer's span, the copy time left after the producer ended,
    how long each segment waited after its last flag was raised before a wave saw it, and where
    each kernel's workgroups ran."""
    span = stg.records(B.MOE_RECORDS_SPAN)[0]
    cp = stg.records(B.MOE_RECORDS_COPY)
    wg = stg.records(B.MOE_RECORDS_PRODUCER)
    tiles = stg.records(B.MOE_RECORDS_TILES)
    segs = stg.plan()["segments"]          # dst, rows, y_row0, slot0, flag_begin, flag_count, ready_pos, npieces
    p0, p1 = int(span["producer_start"]), int(span["producer_end"])
    out = {"copy_units": int(span["copy_units"]), "recorded": int(len(cp))}
    if len(cp) == 0 or p1 <= p0:
        return out
    busy, pieces = union_length(list(zip(cp["t_ready"].astype(np.int64), cp["t_done"].astype(np.int64))))
    hidden = sum(max(0, min(b, p1) - max(a, p0)) for a, b in pieces)
    t_end = int(cp["t_done"].max())
    nbytes = 4.0 * wl.H * float(segs[:, 1].sum())
    lag, deliver = [], []
    for s in range(len(segs)):
        m = cp["segment"] == s
        if not m.any():
            continue
        fb, fc = int(segs[s, 4]), int(segs[s, 5])
        t_flag = int(tiles[fb:fb + fc].max()) if fc else 0
        if t_flag:
            lag.append((int(cp["t_ready"][m].min()) - t_flag) * TICK_US)
            deliver.append((int(cp["t_done"][m].max()) - t_flag) * TICK_US)
    own = cp["source"] == 0
    cons_cu = {cu_key(h, x) for h, x in zip(cp["hw_id"][own], cp["xcc_id"][own])}
    grid = int(span["producer_grid"])
    prod_cu = {cu_key(h, x) for h, x in zip(wg["hw_id"][grid:], wg["xcc_id"][grid:])}
    per_cu = {}
    for h, x in zip(wg["hw_id"][grid:], wg["xcc_id"][grid:]):
        per_cu[cu_key(h, x)] = per_cu.get(cu_key(h, x), 0) + 1
    out.update({
        "producer_span_us": (p1 - p0) * TICK_US,
        "consumer_busy_us": busy * TICK_US,
        "overlap_ratio": hidden / busy if busy else None,
        "exposed_copy_us": max(0, t_end - p1) * TICK_US,
        "consumer_GBps_while_busy": nbytes / (busy * TICK_US * 1e-6) / 1e9 if busy else None,
        "copy_bytes": nbytes,
        "flag_to_copy_start_us_p50_p90_max": [round(float(np.percentile(lag, q)), 2) for q in (50, 90, 100)] if lag else None,
        "flag_to_delivered_us_p50_p90_max": [round(float(np.percentile(deliver, q)), 2) for q in (50, 90, 100)]
        if deliver else None,
        "segments_timed": len(lag),
        "units_drained": int((~own).sum()),
        "consumer_cus_used": len(cons_cu),
        "producer_down_cus_used": len(prod_cu),
        "producer_down_workgroups_per_cu_max": max(per_cu.values()) if per_cu else 0,
        "consumer_cus_shared_with_producer": len(cons_cu & prod_cu),
        "producer_clock_GHz": producer_clocks(wg, grid, cons_cu),
        "down_end_spread": down_end_spread(wg, grid, cons_cu),
    })
    return out


def down_end_spread(wg, grid, cons_cu):
    """When the down launch's workgroups finished, relative to the launch's first start: the
    median and the last, and the last among workgroups on the consumer's compute units and on
    the others (the launch ends with its slowest workgroup)."""
    w = wg[grid:2 * grid]
    w = w[w["items"] > 0]
    if len(w) == 0:
        return None
    t0 = int(w["t_start"].min())
    end = (w["t_end"].astype(np.int64) - t0) * TICK_US
    on = np.array([cu_key(h, x) in cons_cu for h, x in zip(w["hw_id"], w["xcc_id"])], bool)
    r = {"median_end_us": round(float(np.median(end)), 1), "last_end_us": round(float(end.max()), 1)}
    if on.any():
        r["last_end_on_consumer_cus_us"] = round(float(end[on].max()), 1)
    if (~on).any():
        r["last_end_elsewhere_us"] = round(float(end[~on].max()), 1)
    return r


class Bench:
    """One workload resident on the GPU.  Handles are created per measurement and closed right
    after it: every live handle keeps CU-masked hardware queues, and idle queues slow the stage."""

    def __init__(self, torch, B, wl, args):
        self.torch, self.B, self.wl, self.args = torch, B, wl, args

        def dev(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda")

        self.x, self.w1, self.w3, self.w2 = dev(wl.dispatched_x), dev(wl.w1), dev(wl.w3), dev(wl.w2)
        self.bufs = [torch.zeros((int(n), wl.H), dtype=torch.int16, device="cuda") for n in wl.return_rows]
        self.run_args = (self.x, wl.expert_offsets, wl.row_src_rank, wl.row_slot, self.w1, self.w3, self.w2,
                         self.bufs, wl.return_rows)
        d_routing = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
                     for a in (wl.expert_offsets, wl.row_src_rank, wl.row_slot)]
        self.dev_run_args = (self.x, *d_routing, self.w1, self.w3, self.w2, self.bufs, wl.return_rows)
        torch.cuda.synchronize()
        # The stage runs on a stream of its own, as in a serving loop (on the legacy null stream
        # the shared-CU producer would have to fork to a second queue; see moe_stage_run).
        self.stream = torch.cuda.Stream()
        self.timeouts = []

    def handle(self, mode, mgb=None, timing=False, extra=0, band_rows=None):
        B, wl, args = self.B, self.wl, self.args
        flags = B.MOE_LOCAL_DIRECT | extra | {"shared": B.MOE_SHARED_CUS, "partitioned": 0, "direct": B.MOE_DIRECT_ALL}[mode]
        if timing:
            flags |= B.MOE_KERNEL_TIMING
        return B.MoeStage(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows,
                          args.band_rows if band_rows is None else band_rows, mgb or args.mgb, flags, 0, args.split_k)

    def fn(self, stg, path, cu_split, device_plan=False):
        if path == "serial":
            if device_plan:
                return lambda: stg.run_serial_devplan(*self.dev_run_args, stream=self.stream)
            return lambda: stg.run_serial(*self.run_args, stream=self.stream)
        if device_plan:
            return lambda: stg.run_devplan(*self.dev_run_args, cu_split=cu_split, stream=self.stream)
        return lambda: stg.run(*self.run_args, cu_split=cu_split, stream=self.stream)

    def timed(self, stg, fn, steps, warmup, warm_s):
        """`warmup` untimed steps (continued until `warm_s` seconds have passed), then exactly
        `steps` timed steps bracketed by device synchronisation, one event between consecutive
        steps: the whole loop's time gives the mean, the per-step differences the median and
        spread."""
        torch = self.torch
        t0 = time.perf_counter()
        i = 0
        while i < warmup or time.perf_counter() - t0 < warm_s:
            fn()
            i += 1
            if i % 16 == 0:
                torch.cuda.synchronize()
        stg.query(check=False)
        if stg.cfg.flags & self.B.MOE_KERNEL_TIMING:
            stg.times(reset=True)
        # A garbage-collection pass inside the timed loop stalls the host while the GPU idles.
        gc.collect()
        gc.disable()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record(self.stream)
        for k in range(steps):
            fn()
            ev[k + 1].record(self.stream)
        torch.cuda.synchronize()
        gc.enable()
        per_step = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(steps)])
        st = stg.query(check=False)
        if st["rc"] != 0:
            msg = self.B.moe_stage_last_error(stg.h)
            log(f"ERROR: {msg} -- timing invalid")
            self.timeouts.append(msg)
        r = {"ms": ev[0].elapsed_time(ev[steps]) / steps, "p10_ms": float(np.percentile(per_step, 10)),
             "p50_ms": float(np.median(per_step)), "p90_ms": float(np.percentile(per_step, 90)),
             "warmup_runs": i, "stats": st}
        if stg.cfg.flags & self.B.MOE_KERNEL_TIMING:
            tm = stg.times(reset=True)
            runs = max(tm["runs"], 1)
            for k in ("producer_ms", "gate_up_ms", "consumer_ms", "scatter_ms", "plan_ms"):
                r[k] = tm[k] / runs
        return r

    def measure(self, mode, path, cu_split, steps, warmup, warm_s, mgb=None, device_plan=False, band_rows=None):
        """Stage time from a handle without per-kernel events (they cost the overlapped stage about
        1 %), then kernel durations from an event-timed handle on the same configuration."""
        stg = self.handle(mode, mgb, band_rows=band_rows)
        try:
            plain = self.timed(stg, self.fn(stg, path, cu_split, device_plan), steps, warmup, warm_s)
        finally:
            stg.close()
        stg = self.handle(mode, mgb, timing=True, band_rows=band_rows)
        try:
            ev = self.timed(stg, self.fn(stg, path, cu_split, device_plan), steps, warmup, warm_s)
        finally:
            stg.close()
        r = dict(ev)
        r["ms_with_kernel_events"] = ev["ms"]
        for k in ("ms", "p10_ms", "p50_ms", "p90_ms", "warmup_runs"):
            r[k] = plain[k]
        return r

    def plain(self, mode, path, cu_split, steps, warmup, warm_s, mgb=None):
        stg = self.handle(mode, mgb)
        try:
            return self.timed(stg, self.fn(stg, path, cu_split), steps, warmup, warm_s)
        finally:
            stg.close()

    def timestamps(self, mode, cu_split, warmup, warm_s, mgb=None, path="overlapped"):
        """One timestamped run after warm-up: for the overlapped path the overlap ratio, flag
        latencies and placement, for the serial path the producer's clocks."""
        stg = self.handle(mode, mgb, extra=self.B.MOE_TIMESTAMPS)
        try:
            fn = self.fn(stg, path, cu_split)
            self.timed(stg, fn, 5, warmup, warm_s)
            fn()
            stg.query(check=False)
            if path == "serial":
                span = stg.records(self.B.MOE_RECORDS_SPAN)[0]
                wg = stg.records(self.B.MOE_RECORDS_PRODUCER)
                return {"producer_clock_GHz": producer_clocks(wg, int(span["producer_grid"])),
                        "down_end_spread": down_end_spread(wg, int(span["producer_grid"]), set())}
            return overlap_analysis(self.B, stg, self.wl)
        finally:
            stg.close()

    def copy_curve(self, mode, splits, steps, warmup):
        """Consumer copy rate with no producer work (every flag published up front), per consumer
        CU count: the ceiling a c-CU consumer reaches on this workload's segments.  mode "plain":
        a plain grid-stride copy of the same segments on the same compute units, the rate those
        compute units reach with no protocol (the c-CU copy ceiling)."""
        torch, B = self.torch, self.B
        out = []
        for c in splits:
            extra = B.MOE_TEST_CONSUMER_ONLY | (B.MOE_TEST_PLAIN_COPY if mode == "plain" else 0)
            stg = self.handle("partitioned" if mode == "plain" else mode, timing=True, extra=extra)
            try:
                fn = self.fn(stg, "overlapped", c)
                for _ in range(warmup):
                    fn()
                torch.cuda.synchronize()
                stg.times(reset=True)
                for _ in range(steps):
                    fn()
                torch.cuda.synchronize()
                st = stg.query(check=False)
                tm = stg.times(reset=True)
            finally:
                stg.close()
            us = tm["consumer_ms"] / max(tm["runs"], 1) * 1e3
            nbytes = 4.0 * self.wl.H * st["n_remote_rows"]
            out.append({"cu_split": c, "mode": mode, "consumer_cus": st["consumer_cus"], "units": st["copy_units"],
                        "us": us, "bytes": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9,
                        "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, "rc": st["rc"]})
        return out

    def timed_combine(self, steps, warmup):
        """The weighted combine of this rank's own tokens (k returned rows each) from its receive
        buffer: HBM-bound, timed with events on the stream it runs on."""
        torch, B, wl = self.torch, self.B, self.wl
        r = wl.self_rank
        slot = torch.from_numpy(np.ascontiguousarray(wl.slots[r]).astype(np.int32)).cuda()
        gate = torch.from_numpy(np.ascontiguousarray(wl.gates[r]).astype(np.float32)).cuda()
        out = torch.empty((wl.T_r, wl.H), dtype=torch.int16, device="cuda")
        recv = self.bufs[r]
        fn = lambda: B.moe_combine(recv, slot, gate, out, stream=self.stream)
        for _ in range(warmup):
            fn()
        gc.collect()
        gc.disable()
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(self.stream)
        for _ in range(steps):
            fn()
        end.record(self.stream)
        torch.cuda.synchronize()
        gc.enable()
        us = start.elapsed_time(end) / steps * 1e3
        nbytes = 2.0 * wl.H * wl.T_r * (wl.k + 1) + 8.0 * wl.T_r * wl.k
        return {"us": us, "tokens": wl.T_r, "k": wl.k, "bytes": nbytes,
                "GBps": nbytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}


def down_kernel_name(split_k, st):
    """Instantiation the down launch runs: whole tiles with split tail rows by default."""
    if split_k == 0:
        return (f"moe::producer_kernel<true, -1> (down launch: whole tiles, last {st['split_rows']} "
                f"tile rows split {st['split_k']} ways)")
    return f"moe::producer_kernel<true, {split_k if split_k <= 4 else 0}> (down launch, {split_k} K parts)"


def path_summary(wl, r, serial):
    flops = wl.flops()
    gu = r["gate_up_ms"]
    dn = r["producer_ms"] - gu
    out = {"stage_us": r["ms"] * 1e3, "tflops": flops / (r["ms"] * 1e-3) / 1e12,
           "stage_us_median": r["p50_ms"] * 1e3,
           "stage_us_with_kernel_events": r["ms_with_kernel_events"] * 1e3,
           "step_us_p10_p50_p90": [round(r["p10_ms"] * 1e3, 1), round(r["p50_ms"] * 1e3, 1), round(r["p90_ms"] * 1e3, 1)],
           "warmup_runs": r["warmup_runs"],
           "producer_us": r["producer_ms"] * 1e3, "gate_up_us": gu * 1e3, "down_us": dn * 1e3,
           "gate_up_frac_of_peak": 4.0 * wl.H * wl.F * wl.rows / (gu * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "down_frac_of_peak": 2.0 * wl.H * wl.F * wl.rows / (dn * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "producer_frac_of_peak": flops / (r["producer_ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "workgroups_gate_up_down": [int(r["stats"]["gu_workgroups"]), int(r["stats"]["down_workgroups"])]}
    if serial:
        out["scatter_us"] = r["scatter_ms"] * 1e3
    else:
        out["consumer_us"] = r["consumer_ms"] * 1e3
        out["copy_units"] = int(r["stats"]["copy_units"])
    return out


def measure_workload(torch, B, wl, args, headline):
    """Every figure of one workload; returns (detail dict, raw results of the headline paths)."""
    bench = Bench(torch, B, wl, args)
    name = wl.name
    steps = args.steps if headline else max(args.steps, 20)
    warmup = args.warmup
    warm_s = args.warm_s if headline else args.warm_s_other
    wo = args.warm_s_other
    d = {"description": DESCRIPTIONS[name], "routed_rows": wl.rows, "gflop": wl.flops() / 1e9}
    only = args.only if headline else "all"
    raw = {}
    try:
        if only == "copy":
            cs = [int(v) for v in args.copy_curve.split(",")]
            d["consumer_copy_ceiling"] = (bench.copy_curve("partitioned", cs, 10, 3) + bench.copy_curve("shared", cs, 10, 3)
                                          + bench.copy_curve("plain", cs, 10, 3))
            for r in d["consumer_copy_ceiling"]:
                log(f"{name} consumer-only copy c={r['cu_split']} {r['mode']}: {r['us']:.1f} us, {r['GBps']:.0f} GB/s")
            return d, raw
        ser = ovl = None
        if only in ("all", "serial"):
            ser = bench.measure(args.mode, "serial", 0, steps, warmup, warm_s)
            d["serial"] = path_summary(wl, ser, True)
            log(f"{name} serial: {ser['ms'] * 1e3:.1f} us (median {ser['p50_ms'] * 1e3:.1f}; producer "
                f"{ser['producer_ms'] * 1e3:.1f}, gate/up {ser['gate_up_ms'] * 1e3:.1f}, scatter "
                f"{ser['scatter_ms'] * 1e3:.1f})")
        if only in ("all", "overlapped"):
            ovl = bench.measure(args.mode, "overlapped", args.cu_split, steps, warmup, warm_s)
            d["overlapped"] = path_summary(wl, ovl, False)
            d["overlapped"]["config"] = {"cu_split": args.cu_split, "cu_mode": args.mode, "mgb": args.mgb,
                                         "consumer_cus": int(ovl["stats"]["consumer_cus"])}
            st = ovl["stats"]
            log(f"{name} overlapped ({args.mode}, c={args.cu_split}): {ovl['ms'] * 1e3:.1f} us (median "
                f"{ovl['p50_ms'] * 1e3:.1f}; producer {ovl['producer_ms'] * 1e3:.1f}, gate/up "
                f"{ovl['gate_up_ms'] * 1e3:.1f}, consumer {ovl['consumer_ms'] * 1e3:.1f}); segments "
                f"{st['n_segments']}, units {st['copy_units']}, workgroups {st['gu_workgroups']}/{st['down_workgroups']}")
        raw = {"serial": ser, "overlapped": ovl}
        if ser is not None and ovl is not None:
            d["overlap_speedup"] = ser["ms"] / ovl["ms"]
            d["overlap_speedup_median"] = ser["p50_ms"] / ovl["p50_ms"]
        if only != "all":
            return d, raw
        ts = bench.timestamps(args.mode, args.cu_split, warmup, wo)
        d["overlapped"]["timestamps"] = ts
        raw["timestamps"] = ts
        ts_ser = bench.timestamps(args.mode, 0, warmup, wo, path="serial")
        d["serial"]["producer_clock_GHz"] = ts_ser["producer_clock_GHz"]
        d["serial"]["down_end_spread"] = ts_ser["down_end_spread"]
        log(f"{name} down launch ends (median / last / last on consumer CUs / last elsewhere): serial "
            f"{ts_ser['down_end_spread']}, overlapped {ts.get('down_end_spread')}")
        raw["serial_clock"] = ts_ser["producer_clock_GHz"]
        raw["serial_end_spread"] = ts_ser["down_end_spread"]
        log(f"{name} producer clock GHz: serial {ts_ser['producer_clock_GHz']}, overlapped {ts.get('producer_clock_GHz')}")
        log(f"{name} timestamps: overlap ratio {ts.get('overlap_ratio')}, exposed copy {ts.get('exposed_copy_us')} us, "
            f"flag->copy start p50/p90/max {ts.get('flag_to_copy_start_us_p50_p90_max')} us, consumer CUs "
            f"{ts.get('consumer_cus_used')}, producer CUs {ts.get('producer_down_cus_used')}")
        dp = bench.measure(args.mode, "overlapped", args.cu_split, steps, warmup, wo, device_plan=True)
        d["device_plan"] = {"stage_us": dp["ms"] * 1e3, "planner_gpu_us": dp["plan_ms"] * 1e3,
                            "host_plan_host_us": ovl["stats"]["plan_us"],
                            "host_plan_upload_gpu_us": ovl["plan_ms"] * 1e3}
        log(f"{name} overlapped, device-built plan: {dp['ms'] * 1e3:.1f} us (planner {dp['plan_ms'] * 1e3:.1f} us)")
        direct = bench.measure("direct", "serial", 0, steps, warmup, wo)
        d["epilogue_direct_ablation_us"] = direct["ms"] * 1e3
        log(f"{name} epilogue-direct ablation: {direct['ms'] * 1e3:.1f} us")
        # The paper's single-destination layout: every 256-row band belongs to one source rank.
        b256 = bench.handle(args.mode, band_rows=256)
        try:
            r = bench.timed(b256, bench.fn(b256, "overlapped", args.cu_split), steps, warmup, wo)
        finally:
            b256.close()
        d["band_rows_256"] = {"stage_us": r["ms"] * 1e3, "stage_us_median": r["p50_ms"] * 1e3,
                              "padding_rows": int(r["stats"]["n_band_padding"]),
                              "tile_rows": int(r["stats"]["n_tile_rows"]),
                              "vs_default_band_rows": ovl["ms"] / r["ms"]}
        log(f"{name} band_rows=256: {r['ms'] * 1e3:.1f} us, {r['stats']['n_band_padding']} padding rows, "
            f"{r['stats']['n_tile_rows']} tile rows")
        # Consumer CU-split sweep: the paper's small partitions in both CU modes and both segment
        # sizes, and wider shared splits; the main configuration is re-measured first, so the sweep
        # can be checked against it.
        sweep = []
        small = [int(v) for v in args.small.split(",") if v]
        wide = [int(v) for v in args.sweep.split(",") if v]
        points = [(args.cu_split, args.mode, args.mgb)]
        points += [(c, m, g) for g in (1, 2) for c in small for m in ("shared", "partitioned")]
        points += [(c, "shared", 1) for c in wide if (c, "shared", 1) not in points]
        if name == "large_fine":
            grid = [int(v) for v in args.grid.split(",") if v]
            points += [(c, "shared", 1) for c in grid if (c, "shared", 1) not in points]
        # The serial stage is re-measured right before the sweep, and the sweep's ratios use it: the
        # sweep runs minutes after the main measurements, and the box's clock drifts meanwhile.
        ser_sw = bench.plain(args.mode, "serial", 0, max(steps // 2, 20), warmup, wo)
        d["sweep_serial_us_median"] = ser_sw["p50_ms"] * 1e3
        d["sweep_serial_drift"] = ser_sw["p50_ms"] / ser["p50_ms"]
        for c, m, g in points:
            r = bench.plain(m, "overlapped", c, max(steps // 2, 20), warmup, wo, mgb=g)
            sweep.append({"cu_split": c, "cu_mode": m, "mgb": g, "consumer_cus": int(r["stats"]["consumer_cus"]),
                          "segments": int(r["stats"]["n_segments"]), "units": int(r["stats"]["copy_units"]),
                          "stage_us": r["ms"] * 1e3, "stage_us_median": r["p50_ms"] * 1e3,
                          "speedup_vs_serial": ser_sw["ms"] / r["ms"],
                          "speedup_vs_serial_median": ser_sw["p50_ms"] / r["p50_ms"],
                          "beats_serial": bool(r["p50_ms"] < ser_sw["p50_ms"])})
            log(f"{name} sweep c={c} {m} mgb={g}: {r['ms'] * 1e3:.1f} us (median {r['p50_ms'] * 1e3:.1f}), "
                f"speedup {ser_sw['ms'] / r['ms']:.3f}")
        d["cu_split_sweep"] = sweep
        # The sweep's first point repeats the main configuration: its stage time against the main
        # measurement (includes the drift), and its overlapped / serial ratio against the main one.
        d["sweep_main_agreement"] = sweep[0]["stage_us_median"] / (ovl["p50_ms"] * 1e3)
        d["sweep_main_speedup_agreement"] = sweep[0]["speedup_vs_serial_median"] / (ser["p50_ms"] / ovl["p50_ms"])
        best = max(sweep, key=lambda x: x["speedup_vs_serial_median"])
        d["best_sweep_point"] = {k: best[k] for k in ("cu_split", "cu_mode", "mgb", "stage_us_median",
                                                      "speedup_vs_serial_median")}
        smalls = [x for x in sweep if x["cu_split"] <= 32]
        bs = max(smalls, key=lambda x: x["speedup_vs_serial_median"]) if smalls else None
        if bs:
            d["best_small_partition"] = {k: bs[k] for k in ("cu_split", "cu_mode", "mgb", "stage_us_median",
                                                            "speedup_vs_serial_median")}
            ts_small = bench.timestamps(bs["cu_mode"], bs["cu_split"], warmup, wo, mgb=bs["mgb"])
            d["best_small_partition"]["timestamps"] = ts_small
        if args.copy_curve:
            cs = [int(v) for v in args.copy_curve.split(",")]
            d["consumer_copy_ceiling"] = (bench.copy_curve("partitioned", cs, 10, 3) + bench.copy_curve("shared", cs, 10, 3)
                                          + bench.copy_curve("plain", cs, 10, 3))
            for r in d["consumer_copy_ceiling"]:
                log(f"{name} consumer-only copy c={r['cu_split']} {r['mode']}: {r['us']:.1f} us, {r['GBps']:.0f} GB/s "
                    f"({r['units']} units)")
        d["combine"] = bench.timed_combine(max(steps, 20), max(warmup, 5))
        log(f"{name} combine ({wl.T_r} tokens, k={wl.k}): {d['combine']['us']:.1f} us, {d['combine']['GBps']:.0f} GB/s")
        return d, raw
    finally:
        if bench.timeouts:
            d["watchdog"] = bench.timeouts
        del bench
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def expert_count_sweep(torch, B, make_workload, args, counts):
    """Single-layer sweep over experts per rank (paper Section 4.2.2): serial and overlapped stage
    times, the split the adaptive selector (cu_split = 0) settles on, and the overlap ratio from the
    in-kernel timestamps of a run at that split (share of the consumer's copy time inside the
    producer's span)."""
    rows = []
    for E in counts:
        name = f"layer_e{E}"
        log(f"generating workload {name} seed {args.seed}")
        wl = make_workload(name, seed=args.seed)
        bench = Bench(torch, B, wl, args)
        steps, warmup, wo = max(args.steps, 20), args.warmup, args.warm_s_other
        ser = bench.plain("shared", "serial", 0, steps, warmup, wo)
        stg = bench.handle("shared")
        try:
            # Let the adaptive selector finish measuring its candidates, then time it.
            for i in range(200):
                stg.run(*bench.run_args, cu_split=0, stream=bench.stream)
                if i % 4 == 3:
                    torch.cuda.synchronize()
                    if stg.query(check=False)["auto_cu_split"] > 0:
                        break
            ovl = bench.timed(stg, bench.fn(stg, "overlapped", 0), steps, warmup, wo)
        finally:
            stg.close()
        c = int(ovl["stats"]["auto_cu_split"])
        ts = bench.timestamps("shared", c, warmup, wo)
        rows.append({"experts_per_rank": E, "routed_rows": wl.rows, "serial_us": ser["ms"] * 1e3,
                     "overlapped_us": ovl["ms"] * 1e3, "speedup": ser["ms"] / ovl["ms"],
                     "speedup_median": ser["p50_ms"] / ovl["p50_ms"], "auto_cu_split": c,
                     "overlap_ratio": ts.get("overlap_ratio"), "exposed_copy_us": ts.get("exposed_copy_us"),
                     "consumer_busy_us": ts.get("consumer_busy_us"),
                     "tflops_overlapped": wl.flops() / (ovl["ms"] * 1e-3) / 1e12})
        log(f"{name}: serial {ser['ms'] * 1e3:.1f} us, overlapped {ovl['ms'] * 1e3:.1f} us (auto c={c}), speedup "
            f"{ser['ms'] / ovl['ms']:.3f}, overlap ratio {ts.get('overlap_ratio')}")
        del bench, wl
        torch.cuda.empty_cache()
    return rows


def compact_line(args, detail, name, raw, wl):
    """The headline object: what the metric asks for, well under 4 KB."""
    d = detail["workloads"][name]
    ser, ovl = raw.get("serial"), raw.get("overlapped")
    main_r = ovl if ovl is not None else ser
    if main_r is None:
        return {"metric": METRIC, "value": None, "unit": "TFLOP/s", "n_gpus": 1, "note": f"--only {args.only}",
                "detail": args.detail_out}
    st = main_r["stats"]
    out = {"metric": METRIC, "value": wl.flops() / (main_r["ms"] * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": main_r["ms"], "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded generator, random-init weights N(0,0.02^2), activations N(0,1))"}
    out["config"] = {"workload": DESCRIPTIONS[name], "routed_rows": wl.rows,
                     "path": "overlapped" if ovl is not None else "serial",
                     "cu_split": args.cu_split, "consumer_cus": int(st.get("consumer_cus", 0)), "cu_mode": args.mode,
                     "band_rows": args.band_rows or 1, "mid_segment_pieces": args.mgb,
                     "down_split_k": int(st["split_k"]), "down_split_rows": int(st["split_rows"]),
                     "plan_us": round(st["plan_us"], 1), "seed": args.seed}
    out["expert_stage_us"] = main_r["ms"] * 1e3
    out["expert_stage_us_median"] = main_r["p50_ms"] * 1e3
    if ser is not None:
        out["serial_stage_us"] = ser["ms"] * 1e3
        out["serial_stage_us_median"] = ser["p50_ms"] * 1e3
    if ser is not None and ovl is not None:
        out["overlap_speedup"] = ser["ms"] / ovl["ms"]
        out["overlap_speedup_median"] = ser["p50_ms"] / ovl["p50_ms"]
    # Dominant kernel: the producer's gate/up launch (4*H*F flops per routed row, two thirds of the
    # stage), timed by HIP events the library records on the producer's own stream around every
    # launch in the timed region.
    gu_flops = 4.0 * wl.H * wl.F * wl.rows
    gu_ms = main_r["gate_up_ms"]
    ach = gu_flops / (gu_ms * 1e-3) / 1e12
    out["roofline"] = {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                       "frac": ach / PEAK_BF16_TFLOPS, "traffic": stored_traffic(),
                       "kernel": "moe::producer_kernel<false, 1> (gate/up launch)",
                       "flops_per_launch": gu_flops, "launch_us": gu_ms * 1e3}
    dn_ms = main_r["producer_ms"] - gu_ms
    dn = 2.0 * wl.H * wl.F * wl.rows / (dn_ms * 1e-3) / 1e12
    out["roofline_down"] = {"bound": "mfma", "achieved": dn, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                            "frac": dn / PEAK_BF16_TFLOPS, "kernel": down_kernel_name(args.split_k, st),
                            "launch_us": dn_ms * 1e3}
    prod = wl.flops() / (main_r["producer_ms"] * 1e-3) / 1e12
    out["producer"] = {"us": main_r["producer_ms"] * 1e3, "tflops": prod, "frac": prod / PEAK_BF16_TFLOPS}
    ts = raw.get("timestamps") or {}
    if raw.get("serial_clock") or ts.get("producer_clock_GHz"):
        # Mean shader clock of the gate/up and down launches, from the workgroups' cycle counts.
        out["producer"]["clock_GHz"] = {"serial": raw.get("serial_clock"), "overlapped": ts.get("producer_clock_GHz")}
        # When the down launch's workgroups finished (us after its start): median and last.
        out["producer"]["down_end_us"] = {"serial": raw.get("serial_end_spread"), "overlapped": ts.get("down_end_spread")}
    if ovl is not None:
        out["consumer"] = {"us": ovl["consumer_ms"] * 1e3, "copy_bytes": ts.get("copy_bytes"),
                           "units": int(st["copy_units"]),
                           "busy_us": ts.get("consumer_busy_us"), "GBps_while_busy": ts.get("consumer_GBps_while_busy"),
                           "overlap_ratio": ts.get("overlap_ratio"), "exposed_copy_us": ts.get("exposed_copy_us"),
                           "flag_to_copy_start_us_p50_p90_max": ts.get("flag_to_copy_start_us_p50_p90_max"),
                           "cus_used": ts.get("consumer_cus_used")}
        for mode, key in (("partitioned", "copy_alone_GBps_by_cus"), ("plain", "plain_copy_GBps_by_cus")):
            cc = [r for r in d.get("consumer_copy_ceiling", []) if r["mode"] == mode]
            if cc:
                out["consumer"][key] = {str(r["consumer_cus"]): round(r["GBps"]) for r in cc}
    if "best_small_partition" in d:
        b = d["best_small_partition"]
        out["best_small_partition"] = {k: b[k] for k in ("cu_split", "cu_mode", "mgb", "speedup_vs_serial_median")}
    if "sweep_main_agreement" in d:
        out["sweep_main_agreement"] = round(d["sweep_main_agreement"], 4)
        out["sweep_main_speedup_agreement"] = round(d["sweep_main_speedup_agreement"], 4)
        out["sweep_serial_drift"] = round(d["sweep_serial_drift"], 4)
    out["workloads"] = {}
    for n, w in detail["workloads"].items():
        s = {}
        if "serial" in w:
            s["serial_us"] = round(w["serial"]["stage_us"], 1)
            s["gate_up_frac"] = round(w["serial"]["gate_up_frac_of_peak"], 3)
        if "overlapped" in w:
            s["overlapped_us"] = round(w["overlapped"]["stage_us"], 1)
        if "overlap_speedup_median" in w:
            s["speedup_median"] = round(w["overlap_speedup_median"], 3)
        if "best_small_partition" in w:
            s["best_small_c_speedup"] = round(w["best_small_partition"]["speedup_vs_serial_median"], 3)
        if "sweep_main_speedup_agreement" in w:
            s["sweep_speedup_agreement"] = round(w["sweep_main_speedup_agreement"], 4)
        out["workloads"][n] = s
    if "cpu_baseline" in detail:
        out["cpu_baseline"] = detail["cpu_baseline"]
    out["watchdog_timeouts"] = len(detail.get("watchdog_timeouts", []))
    out["detail"] = args.detail_out
    return out


def short_floats(o):
    """The headline line with every float kept to 6 significant digits (the line stays a few KB)."""
    if isinstance(o, float):
        return float(f"{o:.6g}")
    if isinstance(o, dict):
        return {k: short_floats(v) for k, v in o.items()}
    if isinstance(o, list):
        return [short_floats(v) for v in o]
    return o


def main():
    t_start = time.time()
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the expert stage runs on one GPU: the return all-to-all is modelled by "
                                   "copies into per-source-rank buffers in local HBM; --gpus must be 1"}))
        sys.exit(2)
    import torch
    from paper_2607_19539_amd import binding as B
    from paper_2607_19539_amd.workload import make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.esweep_child:
        # The expert-count sweep alone, in a process of its own: handles, queues and allocations
        # of the earlier workloads do not carry over into its timings.
        rows = expert_count_sweep(torch, B, make_workload, args, [int(v) for v in args.esweep.split(",")])
        print(json.dumps({"expert_count_sweep": rows}), flush=True)
        return
    names = [args.workload] + [w for w in args.extra_workloads.split(",") if w and w != args.workload]
    detail = {"metric": METRIC, "args": vars(args), "workloads": {}}
    timeouts = []
    head_raw, head_wl = None, None
    for wi, name in enumerate(names):
        headline = wi == 0
        log(f"generating workload {name} seed {args.seed}")
        wl = make_workload(name, seed=args.seed)
        log(f"{name}: rows={wl.rows} H={wl.H} F={wl.F} E_l={wl.E_l} R={wl.R}")
        d, raw = measure_workload(torch, B, wl, args, headline)
        detail["workloads"][name] = d
        timeouts += d.get("watchdog", [])
        if headline:
            head_raw, head_wl = raw, wl
            if not args.no_cpu_baseline:
                log("timing the CPU oracle on a bounded sample")
                detail["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
                log(f"cpu baseline: {detail['cpu_baseline']['value']:.4f} TFLOP/s on {detail['cpu_baseline']['cores']} "
                    f"threads ({detail['cpu_baseline']['cpu_model']})")
        else:
            del wl
        if name == "tiny" and not args.no_cpu_baseline:
            # The tiny workload's whole stage on one host thread (it finishes in seconds).
            tb = cpu_baseline(make_workload("tiny", seed=args.seed), 1e9, threads=1)
            detail["cpu_baseline_tiny_1thread"] = tb
    if args.esweep and args.only == "all":
        import subprocess
        cmd = [sys.executable, "-u", os.path.abspath(__file__), "--esweep-child", "--esweep", args.esweep,
               "--steps", str(args.steps), "--warmup", str(args.warmup), "--seed", str(args.seed),
               "--band-rows", str(args.band_rows), "--split-k", str(args.split_k), "--mgb", str(args.mgb),
               "--warm-s-other", str(args.warm_s_other)]
        child = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)  # progress lines pass through stderr
        lines = [l for l in child.stdout.splitlines() if l.startswith("{")]
        if child.returncode != 0 or not lines:
            log(f"ERROR: expert-count sweep exited with {child.returncode}")
            timeouts.append(f"expert-count sweep exited with {child.returncode}")
        else:
            detail["expert_count_sweep"] = json.loads(lines[-1])["expert_count_sweep"]
    detail["watchdog_timeouts"] = timeouts
    detail["elapsed_s"] = time.time() - t_start
    line = compact_line(args, detail, names[0], head_raw, head_wl)
    if "expert_count_sweep" in detail:
        line["expert_count_sweep"] = [{"E": r["experts_per_rank"], "speedup": round(r["speedup_median"], 3),
                                       "overlap_ratio": None if r["overlap_ratio"] is None else round(r["overlap_ratio"], 3),
                                       "c": r["auto_cu_split"]} for r in detail["expert_count_sweep"]]
    detail["headline"] = line
    if args.detail_out:
        os.makedirs(os.path.dirname(os.path.abspath(args.detail_out)), exist_ok=True)
        with open(args.detail_out, "w") as f:
            json.dump(detail, f, indent=1)
        log(f"detail written to {args.detail_out}")
    log(f"done in {time.time() - t_start:.0f} s")
    print(json.dumps(short_floats(line)), flush=True)


if __name__ == "__main__":
    main()
