"""Independent numpy float64 brute force of the expert stage, used to pin the oracle.

Structure deliberately differs from the oracle: token-major and dense (every
local expert is applied to every token of every source rank with matrix
products), then the rows that the router actually sent are picked out.  The
receive slot of copy (t, j) of source rank r is recomputed from its definition
(rank of (expert, t, j) in r's send list), not taken from the generator.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def round_to_bf16(v: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), returned as float64.

    Goes through float32 first only when that is exact for the bf16 decision: values are
    rounded directly from float64 by scaling the mantissa.
    """
    v = np.asarray(v, np.float64)
    out = np.zeros_like(v)
    nz = (v != 0) & np.isfinite(v)
    m, e = np.frexp(v[nz])                 # v = m * 2^e, 0.5 <= |m| < 1
    scaled = np.ldexp(m, 8)                # 8 significant bits of bf16
    out[nz] = np.ldexp(np.round(scaled), e - 8)   # np.round is round-half-to-even
    out[~np.isfinite(v)] = v[~np.isfinite(v)]
    return out


def send_slots(topk: np.ndarray) -> np.ndarray:
    """slot[r, t, j] = position of copy (t, j) in source r's list sorted by (expert, t, j)."""
    R, T, k = topk.shape
    slots = np.empty((R, T, k), np.int64)
    for r in range(R):
        e = topk[r].astype(np.int64)
        for t in range(T):
            for j in range(k):
                before = np.count_nonzero(e < e[t, j])
                same = (e == e[t, j])
                # copies of the same expert that come earlier in (t, j) order
                earlier = np.count_nonzero(same[:t]) + np.count_nonzero(same[t, :j])
                slots[r, t, j] = before + earlier
    return slots


def expert_outputs(x_src, w1, w3, w2, round_activation: bool):
    """Dense outputs of every local expert for every token: list over r of [E_l, T, H] float64."""
    outs = []
    for xr in x_src:
        X = bf16_to_f64(xr)                              # [T, H]
        per_e = []
        for e in range(w1.shape[0]):
            G = X @ bf16_to_f64(w1[e]).T                 # [T, F]
            U = X @ bf16_to_f64(w3[e]).T
            A = G / (1.0 + np.exp(-G)) * U
            if round_activation:
                A = round_to_bf16(A)
            per_e.append(A @ bf16_to_f64(w2[e]).T)       # [T, H]
        outs.append(np.stack(per_e))
    return outs


def expected_return(wl_list, round_activation: bool):
    """Expected float64 receive buffers after every owner in ``wl_list`` has run.

    Returns (bufs, written) where bufs[r] is [T*k, H] and written[r] marks the slots
    the owners in ``wl_list`` fill.
    """
    wl0 = wl_list[0]
    R, T, k, H = wl0.R, wl0.T_r, wl0.k, wl0.H
    slots = send_slots(wl0.topk_experts)
    bufs = [np.zeros((T * k, H)) for _ in range(R)]
    written = [np.zeros(T * k, bool) for _ in range(R)]
    for wl in wl_list:
        outs = expert_outputs(wl.x_src, wl.w1, wl.w3, wl.w2, round_activation)
        lo = wl.self_rank * wl.E_l
        for r in range(R):
            for t in range(T):
                for j in range(k):
                    e = int(wl.topk_experts[r, t, j])
                    if lo <= e < lo + wl.E_l:
                        s = slots[r, t, j]
                        bufs[r][s] = outs[r][e - lo, t]
                        written[r][s] = True
    return bufs, written
