"""Thin ctypes binding of ``include/moe_stage.h``.

Argument marshalling only: every step of the expert stage runs in the HIP
library ``_lib/libmoe_stage.so``.  Functions keep the C names; ``MoeStage`` is a
small convenience wrapper that accepts torch tensors (device memory) and numpy
or CPU arrays (routing).  There is no fallback: if the library is missing or no
GPU is present, calls fail loudly.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import sys
from typing import Dict, Optional, Sequence

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "_lib", "libmoe_stage.so")

MOE_OK, MOE_EINVAL, MOE_EROUTING, MOE_ECAPACITY, MOE_EHIP, MOE_ETIMEOUT, MOE_EUNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
(MOE_LOCAL_DIRECT, MOE_KERNEL_TIMING, MOE_POISON, MOE_TEST_NO_SIGNAL, MOE_SHARED_CUS, MOE_DIRECT_ALL,
 MOE_TEST_CONSUMER_ONLY, MOE_TEST_PLAN_NO_LDS, MOE_TIMESTAMPS) = 1, 2, 4, 8, 16, 32, 64, 128, 256
MOE_TEST_PLAIN_COPY, MOE_WRITE_COUNTS = 512, 1024
MOE_RECORDS_PRODUCER, MOE_RECORDS_COPY, MOE_RECORDS_SPAN, MOE_RECORDS_TILES, MOE_RECORDS_WRITES = 0, 1, 2, 3, 4
(MOE_PLAN_TILE_ROWS, MOE_PLAN_ITEMS, MOE_PLAN_ROW_X, MOE_PLAN_ROW_RANK, MOE_PLAN_ROW_SLOT, MOE_PLAN_SEGMENTS,
 MOE_PLAN_GROUPS, MOE_PLAN_QUEUES) = range(8)
ERROR_NAMES = {0: "MOE_OK", -1: "MOE_EINVAL", -2: "MOE_EROUTING", -3: "MOE_ECAPACITY", -4: "MOE_EHIP",
               -5: "MOE_ETIMEOUT", -6: "MOE_EUNSUPPORTED"}

EXPORTED = ["moe_stage_create", "moe_stage_run", "moe_stage_run_serial", "moe_stage_query", "moe_stage_times",
            "moe_stage_last_error", "moe_stage_destroy", "moe_plan_build", "moe_plan_info", "moe_plan_copy",
            "moe_plan_free", "moe_combine", "moe_stage_run_devplan", "moe_stage_run_serial_devplan",
            "moe_stage_plan_info", "moe_stage_plan_copy", "moe_stage_records", "moe_stage_run_serial_static"]
MOE_STATIC_SCRATCH_BYTES = 64 * 1024 * 1024


class moe_stage_config_t(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32), ("num_local_experts", ctypes.c_int32),
                ("num_ranks", ctypes.c_int32), ("self_rank", ctypes.c_int32), ("max_rows", ctypes.c_int32),
                ("band_rows", ctypes.c_int32), ("mid_segment_pieces", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("watchdog_ms", ctypes.c_int32), ("down_split_k", ctypes.c_int32)]


class moe_stage_stats_t(ctypes.Structure):
    _fields_ = [("n_valid", ctypes.c_int64), ("n_logical_rows", ctypes.c_int64), ("n_band_padding", ctypes.c_int64),
                ("n_remote_rows", ctypes.c_int64), ("n_tile_rows", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("n_gu_items", ctypes.c_int32), ("n_down_items", ctypes.c_int32), ("n_segments", ctypes.c_int32),
                ("producer_grid", ctypes.c_int32), ("consumer_grid", ctypes.c_int32), ("consumer_cus", ctypes.c_int32),
                ("timeout", ctypes.c_int32),
                ("plan_us", ctypes.c_double), ("poll_iters", ctypes.c_uint64), ("wait_ticks", ctypes.c_uint64),
                ("gu_workgroups", ctypes.c_int32), ("down_workgroups", ctypes.c_int32),
                ("split_k", ctypes.c_int32), ("split_rows", ctypes.c_int32),
                ("auto_cu_split", ctypes.c_int32), ("timeout_segment", ctypes.c_int32),
                ("copy_units", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class moe_wg_record_t(ctypes.Structure):
    _fields_ = [("hw_id", ctypes.c_uint32), ("xcc_id", ctypes.c_uint32), ("launch", ctypes.c_int32),
                ("items", ctypes.c_int32), ("t_start", ctypes.c_uint64), ("t_end", ctypes.c_uint64),
                ("cycles", ctypes.c_uint64)]


class moe_copy_record_t(ctypes.Structure):
    _fields_ = [("segment", ctypes.c_int32), ("part", ctypes.c_int32), ("hw_id", ctypes.c_uint32),
                ("xcc_id", ctypes.c_uint32), ("t_poll", ctypes.c_uint64), ("t_ready", ctypes.c_uint64),
                ("t_done", ctypes.c_uint64), ("source", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class moe_span_t(ctypes.Structure):
    _fields_ = [("producer_start", ctypes.c_uint64), ("producer_end", ctypes.c_uint64),
                ("copy_units", ctypes.c_int32), ("copy_recorded", ctypes.c_int32),
                ("producer_grid", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class moe_stage_times_t(ctypes.Structure):
    _fields_ = [("runs", ctypes.c_int32), ("stage_ms", ctypes.c_double), ("producer_ms", ctypes.c_double),
                ("gate_up_ms", ctypes.c_double), ("consumer_ms", ctypes.c_double), ("scatter_ms", ctypes.c_double),
                ("plan_ms", ctypes.c_double)]


class moe_plan_info_t(ctypes.Structure):
    _fields_ = [("n_tile_rows", ctypes.c_int32), ("n_items", ctypes.c_int32), ("n_gu_items", ctypes.c_int32),
                ("n_down_items", ctypes.c_int32), ("n_segments", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("gu_tiles_per_row", ctypes.c_int32), ("down_tiles_per_row", ctypes.c_int32),
                ("tile_m", ctypes.c_int32), ("band_rows", ctypes.c_int32), ("split_k", ctypes.c_int32),
                ("split_rows", ctypes.c_int32), ("n_logical_rows", ctypes.c_int64),
                ("n_valid", ctypes.c_int64), ("n_band_padding", ctypes.c_int64), ("n_remote_rows", ctypes.c_int64)]


def _struct_dict(s) -> dict:
    return {name: getattr(s, name) for name, _ in s._fields_}


_lib: Optional[ctypes.CDLL] = None
# Live handles and their configurations: the run wrappers check buffer shapes against them, and
# the exit hook destroys whatever is still alive while the HIP runtime is intact.
_handles: Dict[int, moe_stage_config_t] = {}


def _destroy_live_handles():
    """Exit hook: destroy every live handle before the HIP runtime's own teardown.  Registered
    after torch is imported, so it runs before torch's exit hooks (atexit runs last-in first-out);
    a handle destroyed from a garbage-collector pass during interpreter finalization would tear
    down its streams and pinned memory after the runtime has started unloading."""
    lib = _lib
    for h in list(_handles):
        _handles.pop(h, None)
        if lib is not None:
            lib.moe_stage_destroy(h)


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library not built: {path} (run `python -m paper_2607_19539_amd.build`)")
    try:
        import torch  # noqa: F401  (its exit hooks must be registered before ours)
    except ImportError:
        pass
    atexit.register(_destroy_live_handles)
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.moe_stage_create.argtypes = [ctypes.POINTER(moe_stage_config_t), ctypes.POINTER(vp)]
    lib.moe_stage_run.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    lib.moe_stage_run_serial.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.moe_stage_query.argtypes = [vp, ctypes.POINTER(moe_stage_stats_t)]
    lib.moe_stage_times.argtypes = [vp, i32, ctypes.POINTER(moe_stage_times_t)]
    lib.moe_stage_last_error.argtypes = [vp]
    lib.moe_stage_last_error.restype = ctypes.c_char_p
    lib.moe_stage_destroy.argtypes = [vp]
    lib.moe_plan_build.argtypes = [ctypes.POINTER(moe_stage_config_t), i64, vp, vp, vp, vp, i32,
                                   ctypes.POINTER(vp)]
    lib.moe_plan_info.argtypes = [vp, ctypes.POINTER(moe_plan_info_t)]
    lib.moe_plan_copy.argtypes = [vp, i32, vp, i64]
    lib.moe_plan_copy.restype = ctypes.c_int64
    lib.moe_plan_free.argtypes = [vp]
    lib.moe_plan_free.restype = None
    lib.moe_combine.argtypes = [vp, i64, i32, vp, vp, i64, i32, vp, vp, vp]
    lib.moe_stage_run_devplan.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    lib.moe_stage_run_serial_devplan.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.moe_stage_plan_info.argtypes = [vp, ctypes.POINTER(moe_plan_info_t)]
    lib.moe_stage_plan_copy.argtypes = [vp, i32, vp, i64]
    lib.moe_stage_plan_copy.restype = ctypes.c_int64
    lib.moe_stage_run_serial_static.argtypes = [ctypes.POINTER(moe_stage_config_t), vp, vp, vp, vp, vp, vp, vp, vp,
                                                vp, vp]
    lib.moe_stage_run_serial_static.restype = ctypes.c_int
    lib.moe_stage_records.argtypes = [vp, i32, vp, i64]
    lib.moe_stage_records.restype = ctypes.c_int64
    for name in ("moe_combine", "moe_stage_create", "moe_stage_run", "moe_stage_run_serial", "moe_stage_query",
                 "moe_stage_times", "moe_stage_destroy", "moe_plan_build", "moe_plan_info"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


class MoeError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


def _host_i32(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=np.int32)


def _host_i64(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=np.int64)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dev_ptr(t) -> int:
    """Device pointer of a contiguous torch tensor (or a raw integer address)."""
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return t.data_ptr()


# ----------------------------------------------------------------------------- C-named functions

def make_config(hidden, ffn, num_local_experts, num_ranks, self_rank, max_rows, band_rows=0,
                mid_segment_pieces=1, flags=MOE_LOCAL_DIRECT, watchdog_ms=0, down_split_k=0) -> moe_stage_config_t:
    return moe_stage_config_t(hidden, ffn, num_local_experts, num_ranks, self_rank, max_rows, band_rows,
                              mid_segment_pieces, flags, watchdog_ms, down_split_k)


def moe_stage_last_error(h=None) -> str:
    s = load().moe_stage_last_error(h)
    return s.decode() if s else ""


def _check(rc: int, h=None) -> int:
    if rc != MOE_OK:
        raise MoeError(rc, moe_stage_last_error(h))
    return rc


def moe_stage_create(cfg: moe_stage_config_t) -> int:
    h = ctypes.c_void_p()
    _check(load().moe_stage_create(ctypes.byref(cfg), ctypes.byref(h)))
    _handles[h.value] = moe_stage_config_t.from_buffer_copy(cfg)
    return h.value


def _shape(t):
    """(shape, element size) of a tensor or array; None for a raw integer address or None."""
    if t is None or isinstance(t, int):
        return None
    esize = t.element_size() if hasattr(t, "element_size") else t.itemsize
    return tuple(int(d) for d in t.shape), int(esize)


def validate_run_args(cfg, x, rows, n_routing, w1, w3, w2, return_bufs, return_rows):
    """Checks that every buffer is as large as the call says, before anything reaches the library
    (whose kernels would otherwise read or write past a short buffer).  ``rows`` is the routed-row
    count (expert_offsets[E_l]; None when the routing lives on the device), ``n_routing`` the
    lengths of (expert_offsets, row_src_rank, row_slot).  Raw integer addresses are not checked.
    Raises ValueError."""
    H, F, E, R = cfg.hidden, cfg.ffn, cfg.num_local_experts, cfg.num_ranks
    n_off, n_src, n_slot = n_routing
    if n_off != E + 1:
        raise ValueError(f"expert_offsets must have num_local_experts + 1 = {E + 1} entries, not {n_off}")
    if n_src != n_slot:
        raise ValueError(f"row_src_rank ({n_src}) and row_slot ({n_slot}) differ in length")
    if rows is not None and rows >= 0 and n_src != rows:
        raise ValueError(f"row_src_rank and row_slot must have expert_offsets[-1] = {rows} entries, not {n_src}")
    n_rows = n_src if rows is None else max(rows, 0)
    for name, t, want in (("w1", w1, (E, F, H)), ("w3", w3, (E, F, H)), ("w2", w2, (E, H, F))):
        sh = _shape(t)
        if sh is not None and (sh[0] != want or sh[1] != 2):
            raise ValueError(f"{name} must be [{', '.join(map(str, want))}] with 2-byte elements, got {sh[0]} "
                             f"of {sh[1]}-byte elements")
    sh = _shape(x)
    if sh is not None and (len(sh[0]) != 2 or sh[0][1] != H or sh[0][0] < n_rows or sh[1] != 2):
        raise ValueError(f"dispatched_x must be [>= {n_rows}, {H}] with 2-byte elements, got {sh[0]} of "
                         f"{sh[1]}-byte elements")
    if len(return_bufs) != R:
        raise ValueError(f"return_bufs must hold num_ranks = {R} buffers, not {len(return_bufs)}")
    if len(return_rows) != R:
        raise ValueError(f"return_rows must hold num_ranks = {R} entries, not {len(return_rows)}")
    for r, (b, n) in enumerate(zip(return_bufs, return_rows)):
        sh = _shape(b)
        if sh is not None and (len(sh[0]) != 2 or sh[0][1] != H or sh[0][0] < int(n) or sh[1] != 2):
            raise ValueError(f"return_bufs[{r}] must be [>= return_rows[{r}] = {int(n)}, {H}] with 2-byte "
                             f"elements, got {sh[0]} of {sh[1]}-byte elements")


def _cfg_of(h) -> moe_stage_config_t:
    cfg = _handles.get(h)
    if cfg is None:
        raise ValueError("not a live handle of this binding")
    return cfg


def _run_args(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows, cfg=None):
    off, src, slot = _host_i32(expert_offsets), _host_i32(row_src_rank), _host_i32(row_slot)
    rr = _host_i64(return_rows if return_rows is not None else [b.shape[0] for b in return_bufs])
    if cfg is not None:
        validate_run_args(cfg, x, int(off[-1]) if off.size else None, (off.size, src.size, slot.size),
                          w1, w3, w2, return_bufs, rr)
    ptrs = (ctypes.c_void_p * len(return_bufs))(*[_dev_ptr(b) for b in return_bufs])
    keep = (off, src, slot, rr, ptrs)
    args = [_dev_ptr(x) if x is not None else None, _np_ptr(off), _np_ptr(src), _np_ptr(slot),
            _dev_ptr(w1) if w1 is not None else None, _dev_ptr(w3) if w3 is not None else None,
            _dev_ptr(w2) if w2 is not None else None, ctypes.cast(ptrs, ctypes.c_void_p), _np_ptr(rr)]
    return args, keep


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def moe_stage_run(h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs: Sequence,
                  return_rows=None, cu_split: int = 8, stream=None) -> int:
    args, keep = _run_args(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows,
                           _cfg_of(h))
    rc = load().moe_stage_run(h, *args, int(cu_split), _stream_ptr(stream))
    del keep
    return _check(rc, h)


def moe_stage_run_serial(h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs: Sequence,
                         return_rows=None, stream=None) -> int:
    args, keep = _run_args(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows,
                           _cfg_of(h))
    rc = load().moe_stage_run_serial(h, *args, _stream_ptr(stream))
    del keep
    return _check(rc, h)


def _run_args_dev(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows, cfg=None):
    import torch
    for name, t in (("expert_offsets", expert_offsets), ("row_src_rank", row_src_rank), ("row_slot", row_slot)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.int32 or t.dim() != 1:
            raise ValueError(f"{name} must be a one-dimensional int32 device tensor")
    rr = _host_i64(return_rows if return_rows is not None else [b.shape[0] for b in return_bufs])
    if cfg is not None:
        # The routed-row count lives on the device; the routing arrays' own lengths bound it.
        validate_run_args(cfg, x, None, (expert_offsets.numel(), row_src_rank.numel(), row_slot.numel()),
                          w1, w3, w2, return_bufs, rr)
    ptrs = (ctypes.c_void_p * len(return_bufs))(*[_dev_ptr(b) for b in return_bufs])
    keep = (rr, ptrs)
    args = [_dev_ptr(x), _dev_ptr(expert_offsets), _dev_ptr(row_src_rank), _dev_ptr(row_slot),
            _dev_ptr(w1), _dev_ptr(w3), _dev_ptr(w2), ctypes.cast(ptrs, ctypes.c_void_p), _np_ptr(rr)]
    return args, keep


def moe_stage_run_devplan(h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs: Sequence,
                          return_rows=None, cu_split: int = 8, stream=None) -> int:
    """moe_stage_run with the routing (int32 device tensors) planned on the device."""
    args, keep = _run_args_dev(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows,
                               _cfg_of(h))
    rc = load().moe_stage_run_devplan(h, *args, int(cu_split), _stream_ptr(stream))
    del keep
    return _check(rc, h)


def moe_stage_run_serial_devplan(h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2,
                                 return_bufs: Sequence, return_rows=None, stream=None) -> int:
    args, keep = _run_args_dev(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows,
                               _cfg_of(h))
    rc = load().moe_stage_run_serial_devplan(h, *args, _stream_ptr(stream))
    del keep
    return _check(rc, h)


def moe_stage_run_serial_static(cfg: moe_stage_config_t, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2,
                                return_bufs: Sequence, return_rows=None, stream=None) -> int:
    """moe_stage_run_serial_devplan without a handle: every workspace in the library's fixed
    per-GPU array (no allocation); routing as int32 device tensors."""
    args, keep = _run_args_dev(x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows,
                               cfg)
    rc = load().moe_stage_run_serial_static(ctypes.byref(cfg), *args, _stream_ptr(stream))
    del keep
    return _check(rc)


def moe_combine(recv, slot, gate, out, bad_slots=None, stream=None) -> int:
    """Weighted combine of one source rank on the device.

    ``recv`` [recv_rows, H] and ``out`` [T, H] are 2-byte device tensors (bf16 bits),
    ``slot`` [T, k] int32 and ``gate`` [T, k] float32 device tensors, ``bad_slots`` an
    optional one-element int32/uint32 device tensor that counts out-of-range slots."""
    if recv.dim() != 2 or out.dim() != 2 or slot.dim() != 2 or gate.shape != slot.shape:
        raise ValueError("recv [rows, H], out [T, H], slot and gate [T, k] expected")
    if recv.element_size() != 2 or out.element_size() != 2:
        raise ValueError("recv and out must hold 2-byte elements (bf16 bits)")
    import torch
    if slot.dtype != torch.int32 or gate.dtype != torch.float32:
        raise ValueError("slot must be int32 and gate float32")
    T, k = slot.shape
    if out.shape[0] != T or out.shape[1] != recv.shape[1]:
        raise ValueError("out must be [T, H] with the receive buffer's H")
    bad = None if bad_slots is None else _dev_ptr(bad_slots)
    rc = load().moe_combine(_dev_ptr(recv), int(recv.shape[0]), int(recv.shape[1]), _dev_ptr(slot),
                            _dev_ptr(gate), int(T), int(k), _dev_ptr(out), bad, _stream_ptr(stream))
    return _check(rc)


def moe_stage_query(h, check: bool = True) -> dict:
    st = moe_stage_stats_t()
    rc = load().moe_stage_query(h, ctypes.byref(st))
    d = _struct_dict(st)
    d["rc"] = rc
    if check:
        _check(rc, h)
    return d


def moe_stage_times(h, reset: bool = False) -> dict:
    t = moe_stage_times_t()
    _check(load().moe_stage_times(h, int(reset), ctypes.byref(t)), h)
    return _struct_dict(t)


def moe_stage_destroy(h) -> int:
    _handles.pop(h, None)
    return _check(load().moe_stage_destroy(h))


def moe_stage_records(h, which: int) -> np.ndarray:
    """Records of the handle's last run (MOE_TIMESTAMPS) as a numpy structured array (the span: a
    one-element array)."""
    lib = load()
    ctype = {MOE_RECORDS_PRODUCER: moe_wg_record_t, MOE_RECORDS_COPY: moe_copy_record_t,
             MOE_RECORDS_SPAN: moe_span_t, MOE_RECORDS_TILES: np.uint64, MOE_RECORDS_WRITES: np.uint32}[which]
    need = lib.moe_stage_records(h, int(which), None, 0)
    if need < 0:
        _check(int(need), h)
    if ctype in (np.uint64, np.uint32):
        dt = np.dtype(ctype)
    else:
        dt = np.dtype([(n, np.dtype(t)) for n, t in ctype._fields_], align=True)
        assert dt.itemsize == ctypes.sizeof(ctype)
    out = np.zeros(need // dt.itemsize, dt)
    if need:
        _check(int(lib.moe_stage_records(h, int(which), _np_ptr(out), int(need))), h)
    return out


def moe_plan_build(cfg: moe_stage_config_t, expert_offsets, row_src_rank, row_slot, return_rows,
                   overlapped: bool = True) -> dict:
    """Build the plan on the host and return its tables as numpy arrays (no GPU needed)."""
    lib = load()
    off, src, slot, rr = _host_i32(expert_offsets), _host_i32(row_src_rank), _host_i32(row_slot), _host_i64(return_rows)
    p = ctypes.c_void_p()
    rows = int(off[-1]) if off.size else 0
    _check(lib.moe_plan_build(ctypes.byref(cfg), rows, _np_ptr(off), _np_ptr(src), _np_ptr(slot), _np_ptr(rr),
                              int(bool(overlapped)), ctypes.byref(p)))
    try:
        return _read_plan(lambda o: lib.moe_plan_info(p, o), lambda w, d, n: lib.moe_plan_copy(p, w, d, n))
    finally:
        lib.moe_plan_free(p)


_PLAN_TABLES = (("tile_rows", MOE_PLAN_TILE_ROWS, np.int32, 6), ("items", MOE_PLAN_ITEMS, np.uint32, 1),
                ("row_x", MOE_PLAN_ROW_X, np.int32, 1), ("row_rank", MOE_PLAN_ROW_RANK, np.int32, 1),
                ("row_slot", MOE_PLAN_ROW_SLOT, np.int32, 1), ("segments", MOE_PLAN_SEGMENTS, np.int32, 8),
                ("groups", MOE_PLAN_GROUPS, np.int32, 4), ("queues", MOE_PLAN_QUEUES, np.int32, 9))


def _read_plan(info_fn, copy_fn, h=None) -> dict:
    info = moe_plan_info_t()
    _check(info_fn(ctypes.byref(info)), h)
    out = {"info": _struct_dict(info)}
    for key, which, dt, width in _PLAN_TABLES:
        need = copy_fn(which, None, 0)
        if need < 0:
            _check(int(need), h)
        arr = np.empty(need // np.dtype(dt).itemsize, dt)
        if need:
            _check(int(copy_fn(which, _np_ptr(arr), need)), h)
        out[key] = arr.reshape(-1, width) if width > 1 else arr
    return out


def moe_stage_plan(h) -> dict:
    """The plan of the handle's last run, read back from the device (same tables as moe_plan_build)."""
    lib = load()
    return _read_plan(lambda o: lib.moe_stage_plan_info(h, o), lambda w, d, n: lib.moe_stage_plan_copy(h, w, d, n), h)


# ----------------------------------------------------------------------------- convenience wrapper

class MoeStage:
    """Owns one library handle.  Tensors are torch device tensors holding bf16 (or int16 bit patterns)."""

    def __init__(self, hidden, ffn, num_local_experts, num_ranks, self_rank, max_rows, band_rows=0,
                 mid_segment_pieces=1, flags=MOE_LOCAL_DIRECT, watchdog_ms=0, down_split_k=0):
        self.cfg = make_config(hidden, ffn, num_local_experts, num_ranks, self_rank, max_rows, band_rows,
                               mid_segment_pieces, flags, watchdog_ms, down_split_k)
        self.h = moe_stage_create(self.cfg)

    def run(self, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows=None,
            cu_split=8, stream=None):
        return moe_stage_run(self.h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs,
                             return_rows, cu_split, stream)

    def run_serial(self, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows=None,
                   stream=None):
        return moe_stage_run_serial(self.h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs,
                                    return_rows, stream)

    def run_devplan(self, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs, return_rows=None,
                    cu_split=8, stream=None):
        return moe_stage_run_devplan(self.h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs,
                                     return_rows, cu_split, stream)

    def run_serial_devplan(self, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2, return_bufs,
                           return_rows=None, stream=None):
        return moe_stage_run_serial_devplan(self.h, x, expert_offsets, row_src_rank, row_slot, w1, w3, w2,
                                            return_bufs, return_rows, stream)

    def plan(self) -> dict:
        return moe_stage_plan(self.h)

    def query(self, check=True) -> dict:
        return moe_stage_query(self.h, check)

    def times(self, reset=False) -> dict:
        return moe_stage_times(self.h, reset)

    def records(self, which) -> np.ndarray:
        return moe_stage_records(self.h, which)

    def close(self):
        if self.h:
            moe_stage_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self, _finalizing=sys.is_finalizing):
        # During interpreter finalization the exit hook has already destroyed live handles (and
        # module globals may already be gone, hence the bound default).
        if _finalizing():
            return
        try:
            self.close()
        except Exception:
            pass
