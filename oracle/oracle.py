"""ctypes wrapper and build step for the plain-C CPU oracle (``moe_oracle.c``).

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the CPU
baseline leg of the benchmark.  The product library never imports this module.

``run`` takes numpy arrays holding bf16 bit patterns (``uint16``) and writes the
expert outputs into the given per-source-rank receive buffers, exactly as the
library's ``moe_stage_run`` does on the GPU.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "moe_oracle.c")
LIB = os.path.join(HERE, "libmoe_oracle.so")

EINVAL, EROUTING = -1, -2


def build(out: str = LIB, mutation: int = 0) -> str:
    """Compile the oracle into a shared library (portable x86-64 code, OpenMP)."""
    cmd = ["gcc", "-O3", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           f"-DORACLE_MUTATION={int(mutation)}",
           SRC, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _stale(lib: str) -> bool:
    return not os.path.exists(lib) or os.path.getmtime(lib) < os.path.getmtime(SRC)


class Oracle:
    def __init__(self, lib_path: Optional[str] = None):
        path = lib_path or LIB
        if lib_path is None and _stale(path):
            build(path)
        self.lib = ctypes.CDLL(path)
        i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        self.lib.moe_oracle_run.argtypes = [i32, i32, i32, i32, i32, i64, vp, vp, vp, vp, vp, vp, vp,
                                            ctypes.POINTER(vp), vp, i32]
        self.lib.moe_oracle_run.restype = ctypes.c_int
        self.lib.moe_oracle_validate.argtypes = [i32, i32, i32, i32, i32, i64, vp, vp, vp, vp]
        self.lib.moe_oracle_validate.restype = ctypes.c_int
        self.lib.moe_oracle_combine.argtypes = [i32, i32, i64, i64, vp, vp, vp, vp, i32]
        self.lib.moe_oracle_combine.restype = ctypes.c_int

    @staticmethod
    def _p(a: Optional[np.ndarray]):
        return None if a is None else a.ctypes.data_as(ctypes.c_void_p)

    def run(self, H: int, F: int, E_l: int, R: int, self_rank: int, x: np.ndarray,
            expert_offsets: np.ndarray, row_src_rank: np.ndarray, row_slot: np.ndarray,
            w1: np.ndarray, w3: np.ndarray, w2: np.ndarray, return_bufs: Sequence[np.ndarray],
            return_rows: Optional[np.ndarray] = None, num_threads: int = 0) -> int:
        """Run the oracle; ``return_bufs[r]`` is a C-contiguous ``uint16`` array of shape [rows_r, H]."""
        x = np.ascontiguousarray(x, np.uint16)
        off = np.ascontiguousarray(expert_offsets, np.int32)
        src = np.ascontiguousarray(row_src_rank, np.int32)
        slot = np.ascontiguousarray(row_slot, np.int32)
        w1 = np.ascontiguousarray(w1, np.uint16)
        w3 = np.ascontiguousarray(w3, np.uint16)
        w2 = np.ascontiguousarray(w2, np.uint16)
        for b in return_bufs:
            if b.dtype != np.uint16 or not b.flags.c_contiguous:
                raise ValueError("return buffers must be C-contiguous uint16 arrays")
        if return_rows is None:
            return_rows = np.array([b.shape[0] for b in return_bufs], np.int64)
        rr = np.ascontiguousarray(return_rows, np.int64)
        ptrs = (ctypes.c_void_p * len(return_bufs))(*[b.ctypes.data for b in return_bufs])
        return self.lib.moe_oracle_run(H, F, E_l, R, self_rank, int(x.shape[0]), self._p(x), self._p(off),
                                       self._p(src), self._p(slot), self._p(w1), self._p(w3), self._p(w2),
                                       ptrs, self._p(rr), int(num_threads))

    def validate(self, H: int, F: int, E_l: int, R: int, self_rank: int, rows: int,
                 expert_offsets, row_src_rank, row_slot, return_rows) -> int:
        off = np.ascontiguousarray(expert_offsets, np.int32)
        src = np.ascontiguousarray(row_src_rank, np.int32)
        slot = np.ascontiguousarray(row_slot, np.int32)
        rr = np.ascontiguousarray(return_rows, np.int64)
        return self.lib.moe_oracle_validate(H, F, E_l, R, self_rank, rows, self._p(off), self._p(src),
                                            self._p(slot), self._p(rr))

    def combine(self, recv: np.ndarray, slot: np.ndarray, gate: np.ndarray, out: np.ndarray,
                num_threads: int = 0) -> int:
        """Weighted combine of one source rank: ``recv`` [recv_rows, H] u16, ``slot`` [T, k] i32,
        ``gate`` [T, k] f32; writes ``out`` [T, H] u16 (bf16 bits)."""
        recv = np.ascontiguousarray(recv, np.uint16)
        slot = np.ascontiguousarray(slot, np.int32)
        gate = np.ascontiguousarray(gate, np.float32)
        if out.dtype != np.uint16 or not out.flags.c_contiguous:
            raise ValueError("out must be a C-contiguous uint16 array")
        T, k = slot.shape
        return self.lib.moe_oracle_combine(int(recv.shape[1]), int(k), int(T), int(recv.shape[0]),
                                           self._p(recv), self._p(slot), self._p(gate), self._p(out),
                                           int(num_threads))

    def run_workload(self, wl, return_bufs: Sequence[np.ndarray], num_threads: int = 0) -> int:
        """Convenience: run on a ``Workload`` from the synthetic generator."""
        return self.run(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.dispatched_x, wl.expert_offsets,
                        wl.row_src_rank, wl.row_slot, wl.w1, wl.w3, wl.w2, return_bufs,
                        wl.return_rows, num_threads)


_default: Optional[Oracle] = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
