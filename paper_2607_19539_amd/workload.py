"""Seeded synthetic inputs for one expert-parallel rank's MoE expert stage.

This module only *creates inputs*: token activations, expert weights, a
synthetic router and the dispatch (first all-to-all) that delivers routed token
copies to the rank that owns their expert.  It contains none of the expert
stage's arithmetic (no FFN, no row layout, no tile schedule, no combine plan),
so both the CPU oracle and the HIP path can consume the same bytes.

Workload shapes follow the paper's setting of expert parallelism (Section 2.1:
routing, dispatch, expert compute, combine, scale) with the sizes of the
workloads this library is measured on:

==============  ====  =====  ====  ==  ==  =====  ====  ============================
name            H     F      E_t   k   R   T_r    E_l   router logits
==============  ====  =====  ====  ==  ==  =====  ====  ============================
tiny            256   512    8     2   4   64     2     N(0,1)
mixtral         4096  14336  8     2   4   4096   2     U(0,1) iid
mixtral_zipf    4096  14336  8     2   4   4096   2     Gumbel-top-k, p_e~(e+1)^-1.2
fine            2048  1408   64    6   4   8192   16    N(0,1) + b_e, b_e~N(0,1)
large_fine      7168  2048   256   8   8   4096   32    U(0,1) iid
layer_e<E>      1024  4096   4E    2   4   8192   E     U(0,1) iid, E in 4..64
==============  ====  =====  ====  ==  ==  =====  ====  ============================

The ``layer_e<E>`` family is the single-layer expert-count sweep of Section 4.2.2
(one MoE block, 16 x 512 tokens per rank, top-2, model width 1024, E experts per
rank); the paper states no FFN width, and the usual 4x width is taken.

Conventions (see the dispatch description in Section 3.2.3, "non-overlapping
offsets per peer across experts"):

* activations x ~ N(0,1) and weights ~ N(0, 0.02^2), rounded to bf16 (RNE);
* top-k = stable argsort of the negated logits (ties go to the lower expert id);
  gate weights = softmax over the selected logits (kept for the scale step);
* source rank r sends its routed copies sorted by (global expert, token, j); the
  index of copy (t, j) in that list is its *slot*; every source rank owns a
  receive buffer of ``T_r * k`` rows;
* the owner rank's ``dispatched_x`` is expert-contiguous (local experts in id
  order), and inside an expert sorted by (source rank, token, j).

Random streams are independent per purpose, so any subset is reproducible:
``SeedSequence([seed, 1])`` router, ``[seed, 100 + r]`` activations of source
rank r, ``[seed, 1000 + 3e + {0,1,2}]`` W1/W3/W2 of global expert e.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

__all__ = ["CONFIGS", "Workload", "make_workload", "f32_to_bf16_bits", "bf16_bits_to_f32"]

CONFIGS: Dict[str, dict] = {
    "tiny": dict(H=256, F=512, E_t=8, k=2, R=4, T_r=64, E_l=2, router="normal"),
    "mixtral": dict(H=4096, F=14336, E_t=8, k=2, R=4, T_r=4096, E_l=2, router="uniform"),
    "mixtral_zipf": dict(H=4096, F=14336, E_t=8, k=2, R=4, T_r=4096, E_l=2, router="zipf"),
    "fine": dict(H=2048, F=1408, E_t=64, k=6, R=4, T_r=8192, E_l=16, router="normal_bias"),
    "large_fine": dict(H=7168, F=2048, E_t=256, k=8, R=8, T_r=4096, E_l=32, router="uniform"),
}
for _e in (4, 8, 16, 32, 64):
    CONFIGS[f"layer_e{_e}"] = dict(H=1024, F=4096, E_t=4 * _e, k=2, R=4, T_r=8192, E_l=_e, router="uniform")

ZIPF_S = 1.2
WEIGHT_STD = 0.02


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even) and return the bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    out = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, stream]))


@dataclass
class Workload:
    """All inputs of one owner rank's expert stage (bf16 tensors as uint16 bit patterns)."""

    name: str
    H: int
    F: int
    E_t: int
    k: int
    R: int
    T_r: int
    E_l: int
    self_rank: int
    seed: int
    dispatched_x: np.ndarray          # [rows, H] u16, expert-contiguous
    expert_offsets: np.ndarray        # [E_l + 1] i32
    row_src_rank: np.ndarray          # [rows] i32
    row_slot: np.ndarray              # [rows] i32
    row_token: np.ndarray             # [rows] i32 (token index on its source rank)
    row_j: np.ndarray                 # [rows] i32 (which of the token's k choices)
    w1: Optional[np.ndarray]          # [E_l, F, H] u16 (gate projection, K = H contiguous)
    w3: Optional[np.ndarray]          # [E_l, F, H] u16 (up projection)
    w2: Optional[np.ndarray]          # [E_l, H, F] u16 (down projection, K = F contiguous)
    return_rows: np.ndarray           # [R] i64, receive-buffer rows per source rank (= T_r * k)
    topk_experts: np.ndarray          # [R, T_r, k] i32 global expert ids
    gates: np.ndarray                 # [R, T_r, k] f32 gate weights
    slots: Optional[np.ndarray] = None  # [R, T_r, k] i32 receive slot of each (source, token, choice)
    x_src: List[np.ndarray] = field(default_factory=list)  # per source rank [T_r, H] u16 (optional)

    @property
    def rows(self) -> int:
        return int(self.dispatched_x.shape[0])

    @property
    def local_experts(self) -> range:
        return range(self.self_rank * self.E_l, (self.self_rank + 1) * self.E_l)

    def flops(self) -> float:
        """Algorithmic flops of the stage: 6*H*F per routed row (gate + up + down)."""
        return 6.0 * self.H * self.F * self.rows

    def subset(self, rows_idx) -> "Workload":
        """The same stage restricted to some routed rows (weights and receive buffers unchanged)."""
        import copy
        idx = np.sort(np.asarray(rows_idx, dtype=np.int64))
        e_of = np.searchsorted(self.expert_offsets, idx, side="right") - 1
        s = copy.copy(self)
        s.dispatched_x = self.dispatched_x[idx]
        s.row_src_rank = self.row_src_rank[idx]
        s.row_slot = self.row_slot[idx]
        s.row_token = self.row_token[idx]
        s.row_j = self.row_j[idx]
        off = np.zeros(self.E_l + 1, np.int32)
        off[1:] = np.cumsum(np.bincount(e_of, minlength=self.E_l))
        s.expert_offsets = off
        return s

    def sample(self, n: int, seed: int = 12345) -> "Workload":
        """A seeded uniform sample of n routed rows (all rows if n >= rows)."""
        if n >= self.rows:
            return self
        g = np.random.default_rng(np.random.SeedSequence([seed, 7]))
        return self.subset(g.choice(self.rows, size=n, replace=False))


def _router_logits(name: str, cfg: dict, seed: int) -> np.ndarray:
    R, T, E = cfg["R"], cfg["T_r"], cfg["E_t"]
    g = _rng(seed, 1)
    kind = cfg["router"]
    if kind == "normal":
        return g.standard_normal((R, T, E), dtype=np.float32)
    if kind == "uniform":
        return g.random((R, T, E), dtype=np.float32)
    if kind == "normal_bias":
        bias = g.standard_normal(E, dtype=np.float32)  # per-expert bias, drawn first
        return g.standard_normal((R, T, E), dtype=np.float32) + bias[None, None, :]
    if kind == "zipf":
        # Gumbel-top-k over log-popularity samples k distinct experts without replacement
        # with probabilities proportional to p_e = (e+1)^-s (expert 0 most popular).
        logp = (-ZIPF_S * np.log(np.arange(1, E + 1, dtype=np.float64))).astype(np.float32)
        gumbel = -np.log(-np.log(g.random((R, T, E), dtype=np.float64).clip(1e-300, None)))
        return (logp[None, None, :] + gumbel.astype(np.float32)).astype(np.float32)
    raise ValueError(f"unknown router kind {kind!r}")


def _normal_bf16_into(dst: np.ndarray, seed: int, stream: int, scale: float, chunk_rows: int = 2048) -> None:
    """dst[:] = bf16(N(0,1) * scale) from one stream, drawn in row chunks (the same values as a
    single draw of the whole matrix)."""
    g = _rng(seed, stream)
    for r0 in range(0, dst.shape[0], chunk_rows):
        r1 = min(dst.shape[0], r0 + chunk_rows)
        v = g.standard_normal((r1 - r0, dst.shape[1]), dtype=np.float32)
        v *= np.float32(scale)
        dst[r0:r1] = f32_to_bf16_bits(v)


def _normal_weights_into(w1, w3, w2, seed: int, first_expert: int) -> None:
    """Fill all local experts' weights, one thread per matrix (each has its own stream)."""
    jobs = []
    for i in range(w1.shape[0]):
        e = first_expert + i
        jobs += [(w1[i], 1000 + 3 * e + 0), (w3[i], 1000 + 3 * e + 1), (w2[i], 1000 + 3 * e + 2)]
    workers = max(1, min(16, len(jobs), len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(lambda j: _normal_bf16_into(j[0], seed, j[1], WEIGHT_STD), jobs))


def _expert_weights(seed: int, e: int, H: int, F: int, kind: str, E_l_index: int):
    if kind == "normal":
        w1, w3, w2 = np.empty((F, H), np.uint16), np.empty((F, H), np.uint16), np.empty((H, F), np.uint16)
        _normal_bf16_into(w1, seed, 1000 + 3 * e + 0, WEIGHT_STD)
        _normal_bf16_into(w3, seed, 1000 + 3 * e + 1, WEIGHT_STD)
        _normal_bf16_into(w2, seed, 1000 + 3 * e + 2, WEIGHT_STD)
        return w1, w3, w2
    if kind == "identity":
        # W1 = W3 = [I_H; 0] (F x H), W2 = s_e [I_H 0] (H x F), s_e = 2^-(e mod 4).
        if F < H:
            raise ValueError("identity-like weights need F >= H")
        one = np.uint16(0x3F80)
        w1 = np.zeros((F, H), np.uint16)
        w1[np.arange(H), np.arange(H)] = one
        w3 = w1.copy()
        s_bits = np.uint16(0x3F80 - (e % 4) * 0x80)  # 2^-(e mod 4) in bf16
        w2 = np.zeros((H, F), np.uint16)
        w2[np.arange(H), np.arange(H)] = s_bits
        return w1, w3, w2
    w1, w3, w2 = _expert_weights(seed, e, H, F, "normal", E_l_index)
    if kind == "zero_w1":
        w1 = np.zeros_like(w1)
    elif kind == "zero_w3":
        w3 = np.zeros_like(w3)
    elif kind == "zero_w2":
        w2 = np.zeros_like(w2)
    else:
        raise ValueError(f"unknown weight kind {kind!r}")
    return w1, w3, w2


def make_workload(
    name: str,
    seed: int = 0,
    owner: int = 0,
    weights: Optional[str] = "normal",
    keep_sources: bool = False,
    overrides: Optional[dict] = None,
) -> Workload:
    """Build the inputs of owner rank ``owner``'s expert stage for workload ``name``.

    ``weights``: "normal" (N(0, 0.02^2)), "identity" (closed-form check weights),
    "zero_w1" / "zero_w3" / "zero_w2", or None to skip weight generation.
    ``overrides`` replaces shape entries (e.g. ``{"T_r": 16}``) for small test cases.
    """
    cfg = dict(CONFIGS[name])
    if overrides:
        cfg.update(overrides)
    H, F, E_t, k, R, T, E_l = (cfg[n] for n in ("H", "F", "E_t", "k", "R", "T_r", "E_l"))
    if E_t != E_l * R:
        raise ValueError("experts must divide evenly across ranks")
    if not 0 <= owner < R:
        raise ValueError("owner out of range")

    logits = _router_logits(name, cfg, seed)                            # [R, T, E_t]
    order = np.argsort(-logits, axis=-1, kind="stable")[..., :k].astype(np.int32)
    sel = np.take_along_axis(logits, order, axis=-1).astype(np.float64)
    sel = np.exp(sel - sel.max(axis=-1, keepdims=True))
    gates = (sel / sel.sum(axis=-1, keepdims=True)).astype(np.float32)

    # Slots: source r's send list sorted by (global expert, token, j).
    slots = np.empty((R, T, k), np.int32)
    for r in range(R):
        e_flat = order[r].reshape(-1).astype(np.int64)
        t_flat = np.repeat(np.arange(T, dtype=np.int64), k)
        j_flat = np.tile(np.arange(k, dtype=np.int64), T)
        key = (e_flat * T + t_flat) * k + j_flat
        perm = np.argsort(key, kind="stable")
        s = np.empty(T * k, np.int32)
        s[perm] = np.arange(T * k, dtype=np.int32)
        slots[r] = s.reshape(T, k)

    # Rows delivered to the owner: local experts in id order, then source rank, token, j.
    lo = owner * E_l
    x_src: List[np.ndarray] = []
    rows_e, rows_r, rows_t, rows_j = [], [], [], []
    for r in range(R):
        t_idx, j_idx = np.nonzero((order[r] >= lo) & (order[r] < lo + E_l))
        rows_e.append(order[r][t_idx, j_idx] - lo)
        rows_r.append(np.full(t_idx.shape, r, np.int32))
        rows_t.append(t_idx.astype(np.int32))
        rows_j.append(j_idx.astype(np.int32))
    e_all = np.concatenate(rows_e).astype(np.int64)
    r_all = np.concatenate(rows_r).astype(np.int64)
    t_all = np.concatenate(rows_t).astype(np.int64)
    j_all = np.concatenate(rows_j).astype(np.int64)
    perm = np.lexsort((j_all, t_all, r_all, e_all))
    e_all, r_all, t_all, j_all = e_all[perm], r_all[perm], t_all[perm], j_all[perm]
    n = e_all.shape[0]

    dispatched = np.empty((n, H), np.uint16)
    for r in range(R):
        xr = f32_to_bf16_bits(_rng(seed, 100 + r).standard_normal((T, H), dtype=np.float32))
        m = r_all == r
        dispatched[m] = xr[t_all[m]]
        if keep_sources:
            x_src.append(xr)

    offsets = np.zeros(E_l + 1, np.int32)
    offsets[1:] = np.cumsum(np.bincount(e_all, minlength=E_l))
    row_slot = slots[r_all, t_all, j_all].astype(np.int32)

    w1 = w3 = w2 = None
    if weights is not None:
        w1 = np.empty((E_l, F, H), np.uint16)
        w3 = np.empty((E_l, F, H), np.uint16)
        w2 = np.empty((E_l, H, F), np.uint16)
        if weights == "identity":
            for i in range(E_l):
                w1[i], w3[i], w2[i] = _expert_weights(seed, lo + i, H, F, weights, i)
        else:
            _normal_weights_into(w1, w3, w2, seed, lo)
            if weights == "zero_w1":
                w1[:] = 0
            elif weights == "zero_w3":
                w3[:] = 0
            elif weights == "zero_w2":
                w2[:] = 0
            elif weights != "normal":
                raise ValueError(f"unknown weight kind {weights!r}")

    return Workload(
        name=name, H=H, F=F, E_t=E_t, k=k, R=R, T_r=T, E_l=E_l, self_rank=owner, seed=seed,
        dispatched_x=dispatched, expert_offsets=offsets,
        row_src_rank=r_all.astype(np.int32), row_slot=row_slot,
        row_token=t_all.astype(np.int32), row_j=j_all.astype(np.int32),
        w1=w1, w3=w3, w2=w2,
        return_rows=np.full(R, T * k, np.int64),
        topk_experts=order, gates=gates, slots=slots, x_src=x_src,
    )
