#!/usr/bin/env python3
"""Benchmark of the MI355X MoE expert stage (one expert-parallel rank, one GPU).

A step is one overlapped expert-stage run (moe_stage_run): host plan build and
upload, the persistent gated-FFN producer (gate/up launch, then the signaling
down launch) and the CU-confined consumer copying finished segments into the
per-source-rank receive buffers.  Inputs (activations, weights, receive
buffers) are resident in HBM before the timed region; the routing arrays are
host inputs by design of the C ABI, so each step re-validates and re-uploads
the plan.

Prints one JSON line.  ``value`` is the stage's algorithmic bf16 throughput
(6*H*F flops per routed row, padding excluded) in TFLOP/s on the headline
workload; ``ms_per_step`` is its expert-stage time; ``overlap_speedup`` is
serial time / overlapped time.  ``workloads`` holds the same figures and the
consumer CU-split sweep (both CU modes) for every workload measured.
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
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="mixtral", choices=sorted(DESCRIPTIONS), help="headline workload")
    ap.add_argument("--extra-workloads", default="mixtral_zipf,fine,large_fine",
                    help="further workloads measured into 'workloads' ('' = none)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cu-split", type=int, default=248, help="consumer compute units")
    ap.add_argument("--mode", choices=["shared", "partitioned"], default="shared",
                    help="shared: the producer keeps every CU and the consumer runs beside it on its "
                         "cu_split CUs; partitioned: the consumer's CUs are reserved for it")
    ap.add_argument("--band-rows", type=int, default=0, help="tb_M of the row layout (0 = 1, no alignment)")
    ap.add_argument("--split-k", type=int, default=0, help="K parts per down tile (0 = library default)")
    ap.add_argument("--mgb", type=int, default=1, help="tile-row pieces per middle transfer segment")
    ap.add_argument("--copy-curve", default="8,16,32,64,128",
                    help="consumer CU counts for the consumer-only copy ceiling ('' to skip)")
    ap.add_argument("--sweep", default="8,16,32,64,128,248",
                    help="CU splits for the overlap-speedup sweep: shared CUs at each, a reserved "
                         "partition at those up to 64 ('' = none)")
    ap.add_argument("--esweep", default="4,8,16,32,64",
                    help="experts per rank for the single-layer expert-count sweep ('' to skip)")
    ap.add_argument("--only", choices=["all", "serial", "overlapped"], default="all",
                    help="run only one path of the headline workload (counter collection)")
    ap.add_argument("--esweep-child", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    return ap.parse_args()


def cpu_baseline(wl, target_s):
    """Time the CPU oracle on a bounded sample of the workload's routed rows."""
    from oracle import oracle as orc
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
            "sample": f"{n} of {wl.rows} routed rows ({n / wl.rows:.1%}), {dt:.1f} s wall; full stage "
                      f"would take ~{dt * wl.rows / n:.0f} s on these cores"}


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


class Bench:
    """One workload resident on the GPU, with a handle per CU mode on a dedicated stream."""

    def __init__(self, torch, B, wl, args):
        self.torch, self.B, self.wl, self.args = torch, B, wl, args

        def dev(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda")

        self.x, self.w1, self.w3, self.w2 = dev(wl.dispatched_x), dev(wl.w1), dev(wl.w3), dev(wl.w2)
        self.bufs = [torch.zeros((int(n), wl.H), dtype=torch.int16, device="cuda") for n in wl.return_rows]
        self.run_args = (self.x, wl.expert_offsets, wl.row_src_rank, wl.row_slot, self.w1, self.w3, self.w2,
                         self.bufs, wl.return_rows)
        # The same routing resident on the device, for the device-planned runs.
        d_routing = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
                     for a in (wl.expert_offsets, wl.row_src_rank, wl.row_slot)]
        self.dev_run_args = (self.x, *d_routing, self.w1, self.w3, self.w2, self.bufs, wl.return_rows)
        self.base_flags = B.MOE_LOCAL_DIRECT | B.MOE_KERNEL_TIMING
        extra = {"shared": B.MOE_SHARED_CUS, "partitioned": 0, "direct": B.MOE_DIRECT_ALL}
        self.stages = {m: self.make_stage(f, args.mgb) for m, f in extra.items()}
        # The same CU modes without per-kernel events: the events a timed handle records inside
        # every run (eight on two queues) cost the overlapped stage ~1%, so the stage time is
        # taken from these, and kernel durations from the timed handles.
        for m in ("shared", "partitioned"):
            self.stages[m + ":plain"] = self.make_stage(extra[m], args.mgb, timing=False)
        torch.cuda.synchronize()
        # The stage runs on a stream of its own, as in a serving loop (on the legacy null stream
        # the shared-CU producer would have to fork to a second queue; see moe_stage_run).
        self.stream = torch.cuda.Stream()
        self.timeouts = []

    def make_stage(self, flags, mgb, timing=True):
        wl, args = self.wl, self.args
        base = self.base_flags if timing else self.base_flags & ~self.B.MOE_KERNEL_TIMING
        return self.B.MoeStage(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows, args.band_rows, mgb,
                               base | flags, 0, args.split_k)

    def stage(self, mode, mgb):
        """Event-free handle of a CU mode and mid-segment piece count (created on first use)."""
        key = f"{mode}:plain" if mgb == self.args.mgb else f"{mode}:mgb{mgb}:plain"
        if key not in self.stages:
            f = {"shared": self.B.MOE_SHARED_CUS, "partitioned": 0}[mode]
            self.stages[key] = self.make_stage(f, mgb, timing=False)
        return key

    def close(self):
        for s in self.stages.values():
            s.close()
        self.torch.cuda.synchronize()

    def timed(self, mode, path, cu_split, steps, warmup, device_plan=False):
        """W untimed steps, then exactly `steps` timed steps bracketed by device synchronisation.
        device_plan: the routing is on the device and the plan is built there."""
        torch, stg = self.torch, self.stages[mode]
        if path == "serial":
            fn = ((lambda: stg.run_serial_devplan(*self.dev_run_args, stream=self.stream)) if device_plan else
                  (lambda: stg.run_serial(*self.run_args, stream=self.stream)))
        else:
            fn = ((lambda: stg.run_devplan(*self.dev_run_args, cu_split=cu_split, stream=self.stream))
                  if device_plan else (lambda: stg.run(*self.run_args, cu_split=cu_split, stream=self.stream)))
        for _ in range(warmup):
            fn()
        stg.query(check=False)
        if stg.cfg.flags & self.B.MOE_KERNEL_TIMING:
            stg.times(reset=True)
        # A garbage-collection pass inside the timed loop stalls the host for tens of ms while
        # the GPU idles; collect before and keep the collector off while timing.
        gc.collect()
        gc.disable()
        torch.cuda.synchronize()
        # One event between consecutive steps: the whole loop's time gives the mean, the
        # per-step differences its spread (an event between steps costs no GPU time).
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record(self.stream)
        for i in range(steps):
            fn()
            ev[i + 1].record(self.stream)
        torch.cuda.synchronize()
        gc.enable()
        ms = ev[0].elapsed_time(ev[steps]) / steps
        per_step = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
        st = stg.query(check=False)
        if st["rc"] != 0:
            msg = self.B.moe_stage_last_error(stg.h)
            log(f"ERROR: {msg} -- timing invalid")
            self.timeouts.append(msg)
        tm = stg.times(reset=True) if stg.cfg.flags & self.B.MOE_KERNEL_TIMING else {
            "runs": 0, "producer_ms": 0.0, "gate_up_ms": 0.0, "consumer_ms": 0.0, "scatter_ms": 0.0, "plan_ms": 0.0}
        runs = max(tm["runs"], 1)
        return {"ms": ms, "stats": st, "producer_ms": tm["producer_ms"] / runs,
                "gate_up_ms": tm["gate_up_ms"] / runs, "consumer_ms": tm["consumer_ms"] / runs,
                "scatter_ms": tm["scatter_ms"] / runs, "plan_ms": tm["plan_ms"] / runs,
                "p10_ms": float(np.percentile(per_step, 10)), "p50_ms": float(np.median(per_step)),
                "p90_ms": float(np.percentile(per_step, 90))}

    def copy_curve(self, splits, steps, warmup):
        """Consumer copy rate with no producer work (every flag published up front), per
        consumer CU count: the ceiling a c-CU consumer can reach on this workload's segments."""
        torch, B = self.torch, self.B
        stg = self.make_stage(B.MOE_SHARED_CUS | B.MOE_TEST_CONSUMER_ONLY, self.args.mgb)
        out = []
        try:
            for c in splits:
                fn = lambda: stg.run(*self.run_args, cu_split=c, stream=self.stream)
                for _ in range(warmup):
                    fn()
                torch.cuda.synchronize()
                stg.times(reset=True)
                for _ in range(steps):
                    fn()
                torch.cuda.synchronize()
                st = stg.query(check=False)
                tm = stg.times(reset=True)
                us = tm["consumer_ms"] / max(tm["runs"], 1) * 1e3
                nbytes = 4.0 * self.wl.H * st["n_remote_rows"]
                out.append({"cu_split": c, "consumer_cus": st["consumer_cus"], "us": us,
                            "bytes": nbytes, "GBps": nbytes / (us * 1e-6) / 1e9, "rc": st["rc"]})
        finally:
            stg.close()
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


def with_plain_times(timed_r, plain_r):
    """Kernel durations and stats from the event-timed handle, stage times from the plain one."""
    r = dict(timed_r)
    r["ms_with_kernel_events"] = timed_r["ms"]
    for k in ("ms", "p10_ms", "p50_ms", "p90_ms"):
        r[k] = plain_r[k]
    return r


def summarize(wl, ser, ovl, sweep):
    """Per-workload figures: stage times, producer launches, throughput against the bf16 peak."""
    flops = wl.flops()
    out = {"routed_rows": wl.rows, "gflop": flops / 1e9}
    for key, r in (("serial", ser), ("overlapped", ovl)):
        if r is None:
            continue
        gu = r["gate_up_ms"]
        dn = r["producer_ms"] - gu
        out[key] = {"stage_us": r["ms"] * 1e3, "tflops": flops / (r["ms"] * 1e-3) / 1e12,
                    "stage_us_with_kernel_events": r.get("ms_with_kernel_events", r["ms"]) * 1e3,
                    "step_us_p10_p50_p90": [round(r["p10_ms"] * 1e3, 1), round(r["p50_ms"] * 1e3, 1),
                                            round(r["p90_ms"] * 1e3, 1)],
                    "producer_us": r["producer_ms"] * 1e3, "gate_up_us": gu * 1e3, "down_us": dn * 1e3,
                    "producer_frac_of_peak": flops / (r["producer_ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}
        if key == "serial":
            out[key]["scatter_us"] = r["scatter_ms"] * 1e3
        else:
            out[key]["consumer_us"] = r["consumer_ms"] * 1e3
    if ser is not None and ovl is not None:
        out["overlap_speedup"] = ser["ms"] / ovl["ms"]
    if sweep:
        out["cu_split_sweep"] = sweep
    return out


def expert_count_sweep(torch, B, make_workload, args, counts, timeouts):
    """Single-layer sweep over experts per rank (paper Section 4.2.2): serial and overlapped
    stage times, the split the adaptive selector (cu_split = 0) settles on, and the overlap
    ratio -- the share of the consumer's stand-alone copy time hidden behind the producer:
    1 - (overlapped stage - serial producer) / consumer-only copy time, clamped to [0, 1]."""
    rows = []
    for E in counts:
        name = f"layer_e{E}"
        log(f"generating workload {name} seed {args.seed}")
        wl = make_workload(name, seed=args.seed)
        bench = Bench(torch, B, wl, args)
        steps, warmup = max(args.steps // 2, 10), max(args.warmup // 2, 5)
        # Stage times and the selector run on a handle without per-kernel events (those events
        # slow some consumer splits down, which would steer the selector); the event-timed
        # handle gives only the serial producer time of the overlap ratio.
        ser_t = bench.timed("shared", "serial", 0, steps, warmup)
        ser = bench.timed("shared:plain", "serial", 0, steps, warmup)
        # Let the adaptive selector finish measuring its candidates before timing.
        stg = bench.stages["shared:plain"]
        for i in range(160):
            stg.run(*bench.run_args, cu_split=0, stream=bench.stream)
            if i % 4 == 3:
                torch.cuda.synchronize()
                if stg.query(check=False)["auto_cu_split"] > 0:
                    break
        ovl = bench.timed("shared:plain", "overlapped", 0, steps, warmup)
        st = ovl["stats"]
        c = st["consumer_cus"]
        curve = bench.copy_curve([c], 10, 3)[0]
        t_o, t_p, t_c = ovl["ms"] * 1e3, ser_t["producer_ms"] * 1e3, curve["us"]
        ratio = min(max(1.0 - (t_o - t_p) / t_c, 0.0), 1.0) if t_c > 0 else None
        rows.append({"experts_per_rank": E, "routed_rows": wl.rows, "serial_us": ser["ms"] * 1e3,
                     "overlapped_us": t_o, "speedup": ser["ms"] / ovl["ms"], "serial_producer_us": t_p,
                     "consumer_only_copy_us": t_c, "overlap_ratio": ratio,
                     "auto_cu_split": st["auto_cu_split"], "consumer_cus": c,
                     "tflops_overlapped": wl.flops() / (ovl["ms"] * 1e-3) / 1e12})
        log(f"{name}: serial {ser['ms'] * 1e3:.1f} us, overlapped {t_o:.1f} us (auto c={st['auto_cu_split']}), "
            f"speedup {ser['ms'] / ovl['ms']:.3f}, overlap ratio {ratio if ratio is None else round(ratio, 3)}")
        timeouts += bench.timeouts
        bench.close()
        del bench, wl
        torch.cuda.empty_cache()
    return rows


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
    if args.esweep_child:
        # The expert-count sweep alone, in a process of its own: handles, queues and allocations
        # of the earlier workloads do not carry over into its timings.
        torch.cuda.set_device(0)
        timeouts = []
        rows = expert_count_sweep(torch, B, make_workload, args, [int(v) for v in args.esweep.split(",")], timeouts)
        print(json.dumps({"expert_count_sweep": rows, "watchdog_timeouts": timeouts}), flush=True)
        return
    torch.cuda.set_device(0)
    sweep_cs = [int(v) for v in args.sweep.split(",") if v]
    names = [args.workload] + [w for w in args.extra_workloads.split(",") if w and w != args.workload]
    out = {"metric": METRIC, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded generator, random-init weights N(0,0.02^2), activations N(0,1))"}
    per_wl = {}
    timeouts = []
    for wi, name in enumerate(names):
        headline = wi == 0
        log(f"generating workload {name} seed {args.seed}")
        wl = make_workload(name, seed=args.seed)
        log(f"{name}: rows={wl.rows} H={wl.H} F={wl.F} E_l={wl.E_l} R={wl.R}")
        bench = Bench(torch, B, wl, args)
        steps, warmup = (args.steps, args.warmup) if headline else (max(args.steps // 2, 10),
                                                                    max(args.warmup // 2, 5))
        only = args.only if headline else "all"
        ser = ovl = None
        ser_plain = ovl_plain = None
        if only in ("all", "serial"):
            ser_plain = bench.timed(args.mode + ":plain", "serial", 0, steps, warmup)
            ser = with_plain_times(bench.timed(args.mode, "serial", 0, steps, warmup), ser_plain)
            log(f"{name} serial: {ser['ms'] * 1e3:.1f} us (producer {ser['producer_ms'] * 1e3:.1f}, gate/up "
                f"{ser['gate_up_ms'] * 1e3:.1f}, scatter {ser['scatter_ms'] * 1e3:.1f})")
        if only in ("all", "overlapped"):
            ovl_plain = bench.timed(args.mode + ":plain", "overlapped", args.cu_split, steps, warmup)
            ovl = with_plain_times(bench.timed(args.mode, "overlapped", args.cu_split, steps, warmup), ovl_plain)
            st = ovl["stats"]
            log(f"{name} overlapped ({args.mode}, c={args.cu_split}): {ovl['ms'] * 1e3:.1f} us (producer "
                f"{ovl['producer_ms'] * 1e3:.1f}, gate/up {ovl['gate_up_ms'] * 1e3:.1f}, consumer "
                f"{ovl['consumer_ms'] * 1e3:.1f}); segments {st['n_segments']}, workgroups "
                f"{st['gu_workgroups']}/{st['down_workgroups']}")
        dplan = None
        if only == "all" and ovl is not None:
            # The same overlapped stage with the plan built on the GPU from device-resident routing.
            dplan_plain = bench.timed(args.mode + ":plain", "overlapped", args.cu_split, steps, warmup,
                                      device_plan=True)
            dplan = with_plain_times(bench.timed(args.mode, "overlapped", args.cu_split, steps, warmup,
                                                 device_plan=True), dplan_plain)
            log(f"{name} overlapped, device-built plan: {dplan['ms'] * 1e3:.1f} us (planner on the GPU "
                f"{dplan['plan_ms'] * 1e3:.1f} us; host-built plan: {ovl['stats']['plan_us']:.1f} us on the host, "
                f"upload {ovl['plan_ms'] * 1e3:.1f} us on the GPU)")
        direct = None
        if only == "all":
            # Ablation: no consumer at all, the down epilogue writes every row to its slot.
            direct = bench.timed("direct", "serial", 0, steps, warmup)
            log(f"{name} epilogue-direct ablation: {direct['ms'] * 1e3:.1f} us (producer "
                f"{direct['producer_ms'] * 1e3:.1f}, gate/up {direct['gate_up_ms'] * 1e3:.1f})")
        sweep = []
        if sweep_cs and ser is not None and only == "all":
            for mgb in (1, 2):
                for c in sweep_cs:
                    for mode in ("shared", "partitioned") if c <= 64 else ("shared",):
                        key = bench.stage(mode, mgb)
                        r = bench.timed(key, "overlapped", c, max(steps // 2, 5), max(warmup // 2, 3))
                        sweep.append({"cu_split": c, "cu_mode": mode, "mgb": mgb,
                                      "consumer_cus": r["stats"]["consumer_cus"],
                                      "segments": r["stats"]["n_segments"], "stage_us": r["ms"] * 1e3,
                                      "speedup_vs_serial": ser["ms"] / r["ms"]})
                        log(f"{name} sweep c={c} {mode} mgb={mgb}: {r['ms'] * 1e3:.1f} us, "
                            f"speedup {ser['ms'] / r['ms']:.3f}")
        per_wl[name] = summarize(wl, ser, ovl, sweep)
        if only == "all" and args.copy_curve:
            curve = bench.copy_curve([int(v) for v in args.copy_curve.split(",")], 10, 3)
            per_wl_curve = curve
            for r in curve:
                log(f"{name} consumer copy ceiling c={r['cu_split']} ({r['consumer_cus']} CUs): "
                    f"{r['us']:.1f} us, {r['GBps']:.0f} GB/s")
        else:
            per_wl_curve = None
        comb = bench.timed_combine(max(steps, 20), max(warmup, 5))
        per_wl[name]["combine"] = comb
        if per_wl_curve is not None:
            per_wl[name]["consumer_copy_ceiling"] = per_wl_curve
        log(f"{name} combine ({wl.T_r} tokens, k={wl.k}): {comb['us']:.1f} us, {comb['GBps']:.0f} GB/s")
        if direct is not None:
            per_wl[name]["epilogue_direct_ablation_us"] = direct["ms"] * 1e3
        if dplan is not None:
            per_wl[name]["device_plan"] = {
                "stage_us": dplan["ms"] * 1e3, "planner_gpu_us": dplan["plan_ms"] * 1e3,
                "host_plan_host_us": ovl["stats"]["plan_us"], "host_plan_upload_gpu_us": ovl["plan_ms"] * 1e3,
                "host_planned_stage_us": ovl["ms"] * 1e3}
        timeouts += bench.timeouts
        if headline:
            main_r = ovl if ovl is not None else ser
            st = main_r["stats"]
            out["value"] = wl.flops() / (main_r["ms"] * 1e-3) / 1e12
            out["ms_per_step"] = main_r["ms"]
            out["expert_stage_us"] = main_r["ms"] * 1e3
            if ser is not None:
                out["serial_stage_us"] = ser["ms"] * 1e3
            if ser is not None and ovl is not None:
                out["overlap_speedup"] = ser["ms"] / ovl["ms"]
            out["config"] = {"workload": DESCRIPTIONS[name], "routed_rows": wl.rows,
                             "path": "overlapped" if ovl is not None else "serial",
                             "cu_split": args.cu_split, "consumer_cus": st.get("consumer_cus", 0),
                             "cu_mode": args.mode, "band_rows": args.band_rows or 1,
                             "mid_segment_pieces": args.mgb, "down_split_k": st["split_k"],
                             "down_split_rows": st["split_rows"],
                             "padding_rows": int(st["n_logical_rows"] - st["n_valid"]),
                             "plan_us": round(st["plan_us"], 1), "seed": args.seed}
            # Dominant kernel: the gate/up launch of the producer (4*H*F flops per routed row, two
            # thirds of the stage).  Its duration comes from HIP events the library records on the
            # producer's own stream around every launch in the timed region.
            gu_flops = 4.0 * wl.H * wl.F * wl.rows
            gu_ms = main_r["gate_up_ms"]
            achieved = gu_flops / (gu_ms * 1e-3) / 1e12
            out["roofline"] = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                               "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                               "traffic": stored_traffic(),
                               "kernel": "moe::producer_kernel<false, 1> (gate/up launch)",
                               "flops_per_launch": gu_flops, "launch_us": gu_ms * 1e3}
            dn_ms = main_r["producer_ms"] - gu_ms
            dn_flops = 2.0 * wl.H * wl.F * wl.rows
            out["roofline_down"] = {"bound": "mfma", "achieved": dn_flops / (dn_ms * 1e-3) / 1e12,
                                    "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                                    "frac": dn_flops / (dn_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                                    "kernel": down_kernel_name(args.split_k, st),
                                    "flops_per_launch": dn_flops, "launch_us": dn_ms * 1e3}
            prod = wl.flops() / (main_r["producer_ms"] * 1e-3) / 1e12
            out["producer"] = {"us": main_r["producer_ms"] * 1e3, "tflops": prod, "frac": prod / PEAK_BF16_TFLOPS}
            if ovl is not None:
                cons_bytes = 4.0 * wl.H * st["n_remote_rows"]
                out["consumer"] = {"us": ovl["consumer_ms"] * 1e3, "bytes": cons_bytes,
                                   "busy_GBps_lower_bound": cons_bytes / (ovl["consumer_ms"] * 1e-3) / 1e9,
                                   "flag_wait_us_summed": st["wait_ticks"] / 100.0,
                                   "poll_iters": int(st["poll_iters"]), "segments": int(st["n_segments"])}
            if not args.no_cpu_baseline:
                log("timing the CPU oracle on a bounded sample")
                out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
        bench.close()
        del bench, wl
        torch.cuda.empty_cache()
    out["workloads"] = per_wl
    if args.esweep and args.only == "all":
        import subprocess
        cmd = [sys.executable, "-u", os.path.abspath(__file__), "--esweep-child", "--esweep", args.esweep,
               "--steps", str(args.steps), "--warmup", str(args.warmup), "--seed", str(args.seed),
               "--band-rows", str(args.band_rows), "--split-k", str(args.split_k), "--mgb", str(args.mgb)]
        child = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)  # progress lines pass through stderr
        lines = [l for l in child.stdout.splitlines() if l.startswith("{")]
        if child.returncode != 0 or not lines:
            log(f"ERROR: expert-count sweep exited with {child.returncode}")
            timeouts.append(f"expert-count sweep exited with {child.returncode}")
        else:
            res = json.loads(lines[-1])
            out["expert_count_sweep"] = res["expert_count_sweep"]
            timeouts += res["watchdog_timeouts"]
    out["watchdog_timeouts"] = timeouts
    log(f"done in {time.time() - t_start:.0f} s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
