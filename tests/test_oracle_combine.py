"""Pins for the oracle's weighted combine (paper Section 2.1, step 5), no GPU.

The combine is pinned against:
  * a numpy float64 brute force whose receive slots are recomputed from their definition
    (rank of (expert, t, j) in the source's send list), not taken from the generator,
  * closed forms: k = 1 with gate 1 is an exact row copy; zero gates give zeros; doubling
    every gate doubles every output exactly (a power-of-two scale commutes with rounding),
  * the whole layer: every owner's stage followed by the combine against a dense float64
    mixture-of-experts layer (sum over the chosen experts of gate * expert(x)),
  * validation codes,
and a meta-test rebuilds the oracle with planted combine mistakes and checks that the pins
reject each of them.
"""
import os
import tempfile

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2607_19539_amd.workload import make_workload, bf16_bits_to_f32
from tests import bruteforce as bf

SENTINEL = np.uint16(0x7FC1)


@pytest.fixture(scope="module")
def o():
    return orc.get()


def _ulp(v):
    a = np.abs(np.asarray(v, np.float64))
    a = np.where(a < 1e-30, 1e-30, a)
    return np.ldexp(1.0, np.floor(np.log2(a)).astype(np.int64) - 7)


def _random_recv(rng, rows, H):
    """bf16 bit patterns of N(0, 1) values (finite, normal range)."""
    v = rng.standard_normal((rows, H)).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def _combine(o, recv, slot, gate):
    T, _ = slot.shape
    out = np.full((T, recv.shape[1]), SENTINEL, np.uint16)
    rc = o.combine(recv, slot, gate, out)
    return rc, out


def _check_combine(o, recv, topk, gate):
    """Failures of the oracle's combine of one source rank against the float64 brute force.

    ``topk`` [T, k] are the expert choices; the slots are recomputed from them."""
    fails = []
    slot = bf.send_slots(topk[None])[0].astype(np.int32)
    rc, out = _combine(o, recv, slot, gate)
    if rc != 0:
        return [f"rc {rc}"]
    X = bf.bf16_to_f64(recv)
    terms = gate[:, :, None].astype(np.float64) * X[slot]          # [T, k, H]
    ref = terms.sum(axis=1)
    got = bf16_bits_to_f32(out).astype(np.float64)
    # fp32 products and sums against float64: at most a few fp32 ulps of sum |terms|, then
    # the bf16 rounding of the fp32 value (the double rounding can flip one bf16 tie)
    bound = _ulp(ref) + 4.0 * 2.0 ** -24 * np.abs(terms).sum(axis=1) + 1e-30
    if np.any(np.abs(got - ref) > bound):
        fails.append(f"max |oracle - brute| / bound = {np.max(np.abs(got - ref) / bound):.2f}")
    if np.mean(got == bf.round_to_bf16(ref)) < 0.99:
        fails.append("fewer than 99% of outputs equal the correctly rounded float64 sum")
    return fails


def _topk_and_gate(rng, T, k, E):
    topk = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    g = rng.random((T, k)).astype(np.float32) + np.float32(0.05)
    return topk, (g / g.sum(axis=1, keepdims=True)).astype(np.float32)


@pytest.mark.parametrize("T,k,E,H", [(64, 2, 8, 256), (37, 4, 16, 72), (5, 8, 8, 8), (1, 1, 3, 16)])
def test_combine_vs_bruteforce(o, T, k, E, H):
    """Pin C1: random receive rows and gates, slots recomputed from the expert choices."""
    rng = np.random.default_rng(T * 1000 + k)
    topk, gate = _topk_and_gate(rng, T, k, E)
    recv = _random_recv(rng, T * k, H)
    assert _check_combine(o, recv, topk, gate) == []


def test_combine_k1_gate1_is_a_copy(o):
    """Pin C2: with one choice and gate 1 the combine gathers receive rows unchanged."""
    rng = np.random.default_rng(3)
    recv = _random_recv(rng, 50, 64)
    slot = rng.permutation(50)[:40].astype(np.int32)[:, None]
    rc, out = _combine(o, recv, slot, np.ones((40, 1), np.float32))
    assert rc == 0
    assert np.array_equal(out, recv[slot[:, 0]])


def test_combine_zero_and_doubled_gates(o):
    """Pin C3: zero gates give +0 everywhere; doubling all gates doubles every output exactly."""
    rng = np.random.default_rng(4)
    topk, gate = _topk_and_gate(rng, 30, 3, 9)
    slot = bf.send_slots(topk[None])[0].astype(np.int32)
    recv = _random_recv(rng, 90, 40)
    rc, z = _combine(o, recv, slot, np.zeros_like(gate))
    assert rc == 0 and np.all(z == 0)
    rc1, a = _combine(o, recv, slot, gate)
    rc2, b = _combine(o, recv, slot, gate * np.float32(2))
    assert rc1 == 0 and rc2 == 0
    assert np.array_equal(bf16_bits_to_f32(b), 2 * bf16_bits_to_f32(a))


def test_layer_end_to_end(o):
    """Pin C4: all owners' stages, then every source rank's combine, against a dense float64
    MoE layer: out[r, t] = sum_j gate[r, t, j] * expert_{e(r, t, j)}(x[r, t])."""
    name = "tiny"
    R = make_workload(name, weights=None).R
    wls = [make_workload(name, owner=r, keep_sources=True) for r in range(R)]
    bufs = [np.full((int(n), wls[0].H), SENTINEL, np.uint16) for n in wls[0].return_rows]
    for wl in wls:
        assert o.run_workload(wl, bufs) == 0
    wl0 = wls[0]
    assert np.array_equal(wl0.slots, bf.send_slots(wl0.topk_experts))
    # dense expert outputs of every global expert for every token (activation unrounded)
    dense = {}
    for wl in wls:
        outs = bf.expert_outputs(wl.x_src, wl.w1, wl.w3, wl.w2, round_activation=False)
        for el in range(wl.E_l):
            dense[wl.self_rank * wl.E_l + el] = [outs[r][el] for r in range(R)]
    for r in range(R):
        out = np.full((wl0.T_r, wl0.H), SENTINEL, np.uint16)
        slot = bf.send_slots(wl0.topk_experts)[r].astype(np.int32)
        assert o.combine(bufs[r], slot, wl0.gates[r], out) == 0
        ref = np.zeros((wl0.T_r, wl0.H))
        for t in range(wl0.T_r):
            for j in range(wl0.k):
                ref[t] += float(wl0.gates[r, t, j]) * dense[int(wl0.topk_experts[r, t, j])][r][t]
        got = bf16_bits_to_f32(out).astype(np.float64)
        assert np.all(np.abs(got - ref) <= 1e-2 * np.maximum(1.0, np.abs(ref)))
        rel = np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
        assert rel.max() < 8e-3


def test_combine_validation(o):
    rng = np.random.default_rng(5)
    recv = _random_recv(rng, 10, 16)
    gate = np.ones((4, 2), np.float32)
    slot = np.arange(8, dtype=np.int32).reshape(4, 2)
    for bad in (-1, 10):
        s = slot.copy(); s[2, 1] = bad
        rc, out = _combine(o, recv, s, gate)
        assert rc == orc.EROUTING and np.all(out == SENTINEL)
    out = np.zeros((0, 16), np.uint16)
    assert o.combine(recv, np.zeros((0, 2), np.int32), np.zeros((0, 2), np.float32), out) == 0
    assert o.lib.moe_oracle_combine(0, 2, 4, 10, None, None, None, None, 0) == orc.EINVAL
    assert o.lib.moe_oracle_combine(16, 0, 4, 10, None, None, None, None, 0) == orc.EINVAL


@pytest.mark.parametrize("mutation", [6, 7])
def test_combine_pins_catch_planted_mistakes(mutation):
    with tempfile.TemporaryDirectory() as d:
        bad = orc.Oracle(orc.build(os.path.join(d, f"libmut{mutation}.so"), mutation=mutation))
        rng = np.random.default_rng(0)
        topk, gate = _topk_and_gate(rng, 64, 2, 8)
        assert _check_combine(bad, _random_recv(rng, 128, 64), topk, gate), \
            f"planted combine mistake {mutation} went undetected"
