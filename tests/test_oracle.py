"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself:
  * an independent numpy float64 brute force (dense, token-major, all experts),
  * a library special case (one rank, one expert: a plain gated MLP in torch),
  * a closed form (identity-like weights give y = s_e * x * silu(x) elementwise),
  * zero invariants (a zero W1, W3 or W2 gives exactly zero output),
  * placement invariants (sentinel-filled receive buffers; every token lands k times),
  * validation codes,
and a meta-test rebuilds the oracle with planted mistakes and checks that the
pins reject every one of them.
"""
import os
import tempfile

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2607_19539_amd.workload import make_workload, bf16_bits_to_f32
from tests import bruteforce as bf

SENTINEL = np.uint16(0x7FC1)   # a quiet-NaN bf16 pattern no computation produces here


def _bufs(wl, extra=0):
    return [np.full((int(n) + extra, wl.H), SENTINEL, np.uint16) for n in wl.return_rows]


def _run_all_owners(o, name="tiny", weights="normal", overrides=None):
    wls = [make_workload(name, owner=r, weights=weights, keep_sources=True, overrides=overrides)
           for r in range(make_workload(name, weights=None, overrides=overrides).R)]
    bufs = _bufs(wls[0])
    for wl in wls:
        assert o.run_workload(wl, bufs) == 0
    return wls, bufs


def _bf16_ulp(v):
    a = np.abs(v).astype(np.float64)
    a = np.where(a < 1e-30, 1e-30, a)
    return np.ldexp(1.0, np.floor(np.log2(a)).astype(np.int64) - 7)


def _check_vs_bruteforce(o, wls, bufs):
    """Returns a list of failure strings (empty when the oracle matches the brute force)."""
    fails = []
    exp_r, written = bf.expected_return(wls, round_activation=True)
    exp_u, _ = bf.expected_return(wls, round_activation=False)
    for r in range(len(bufs)):
        got_bits = bufs[r]
        if np.any(got_bits[~written[r]] != SENTINEL):
            fails.append(f"rank {r}: unrouted slot overwritten")
        if np.any(np.all(got_bits[written[r]] == SENTINEL, axis=1)):
            fails.append(f"rank {r}: routed slot left unwritten")
        got = bf16_bits_to_f32(got_bits[written[r]]).astype(np.float64)
        ref = exp_r[r][written[r]]
        # Same bf16 rounding of the activation: what remains is fp32-vs-fp64 summation, the
        # final bf16 rounding (<= 1 ulp) and rare one-ulp flips of a rounded activation when
        # fp32 and fp64 land on opposite sides of a bf16 tie point.  A flip moves y by at most
        # |w2| * ulp(a), a few percent of the row's RMS, and flips are rare.
        d = np.abs(got - ref)
        rms = np.sqrt(np.mean(ref * ref, axis=1, keepdims=True))
        over = d > _bf16_ulp(ref) + 1e-30
        if np.any(d > _bf16_ulp(ref) + 0.02 * rms):
            fails.append(f"rank {r}: max |oracle - brute(a rounded)| / rms = {np.max(d / rms):.3f}")
        if over.mean() > 1e-3:
            fails.append(f"rank {r}: {over.mean():.2e} of elements differ by more than 1 ulp")
        refu = exp_u[r][written[r]]
        if np.any(np.abs(got - refu) > 1e-2 * np.maximum(1.0, np.abs(refu))):
            fails.append(f"rank {r}: elementwise tolerance vs unrounded brute force")
        rel = np.linalg.norm(got - refu, axis=1) / np.maximum(np.linalg.norm(refu, axis=1), 1e-30)
        if np.any(rel > 8e-3):
            fails.append(f"rank {r}: per-row relative L2 {rel.max():.3e} > 8e-3")
    return fails


@pytest.fixture(scope="module")
def o():
    return orc.get()


def test_bruteforce_all_owners(o):
    """Pin P1: all four owner ranks of the tiny workload vs the float64 brute force."""
    wls, bufs = _run_all_owners(o)
    assert _check_vs_bruteforce(o, wls, bufs) == []
    # every token of every source rank appears exactly k times across the receive buffers
    for r, b in enumerate(bufs):
        assert not np.any(np.all(b == SENTINEL, axis=1)), "a receive slot stayed empty"
    wl = wls[0]
    seen = np.zeros((wl.R, wl.T_r), int)
    for w in wls:
        np.add.at(seen, (w.row_src_rank, w.row_token), 1)
    assert np.all(seen == wl.k)


def test_library_special_case(o):
    """Pin P2: one rank, one expert -> the stage is a gated MLP plus a slot permutation."""
    torch = pytest.importorskip("torch")
    F_ = torch.nn.functional
    wl = make_workload("tiny", overrides=dict(R=1, E_t=1, k=1, E_l=1, T_r=48))
    bufs = _bufs(wl)
    assert o.run_workload(wl, bufs) == 0
    X = torch.from_numpy(bf16_bits_to_f32(wl.dispatched_x)).double()
    W1 = torch.from_numpy(bf16_bits_to_f32(wl.w1[0])).double()
    W3 = torch.from_numpy(bf16_bits_to_f32(wl.w3[0])).double()
    W2 = torch.from_numpy(bf16_bits_to_f32(wl.w2[0])).double()
    A = (F_.silu(X @ W1.T) * (X @ W3.T)).to(torch.bfloat16).double()
    Y = (A @ W2.T).numpy()
    got = bf16_bits_to_f32(bufs[0][wl.row_slot]).astype(np.float64)
    assert np.all(np.abs(got - Y) <= _bf16_ulp(Y) + 1e-6)


def test_identity_closed_form(o):
    """Pin P3: W1 = W3 = [I; 0], W2 = s_e [I 0] gives y = s_e * bf16(x * silu(x)) elementwise."""
    wls, bufs = _run_all_owners(o, weights="identity")
    wl0 = wls[0]
    for wl in wls:
        for i in range(wl.rows):
            e = wl.self_rank * wl.E_l + int(np.searchsorted(wl.expert_offsets, i, side="right") - 1)
            s_e = 2.0 ** -(e % 4)
            x = bf16_bits_to_f32(wl.x_src[wl.row_src_rank[i]][wl.row_token[i]]).astype(np.float64)
            want = s_e * bf.round_to_bf16(x * x / (1.0 + np.exp(-x)))
            got = bf16_bits_to_f32(bufs[wl.row_src_rank[i]][wl.row_slot[i]]).astype(np.float64)
            # fp32 silu may flip the single bf16 rounding of the activation: <= 1 ulp
            assert np.all(np.abs(got - want) <= _bf16_ulp(want) + 1e-30), (wl.self_rank, i)
            assert np.mean(got == want) > 0.99
    assert all(not np.any(np.all(b == SENTINEL, axis=1)) for b in bufs)
    assert wl0.k * wl0.R * wl0.T_r == sum(w.rows for w in wls)


@pytest.mark.parametrize("kind", ["zero_w1", "zero_w3", "zero_w2"])
def test_zero_weights_give_zero(o, kind):
    """Pin P4: silu(0) = 0 and x * 0 = 0, so any zero projection zeroes the output."""
    wl = make_workload("tiny", owner=2, weights=kind)
    bufs = _bufs(wl)
    assert o.run_workload(wl, bufs) == 0
    for i in range(wl.rows):
        v = bf16_bits_to_f32(bufs[wl.row_src_rank[i]][wl.row_slot[i]])
        assert np.all(v == 0.0)


def test_single_owner_touches_only_its_slots(o):
    """Pin P5: one owner writes exactly its routed slots; other slots and capacity slack stay intact."""
    wl = make_workload("tiny", owner=1)
    bufs = _bufs(wl, extra=7)
    rr = wl.return_rows + 7
    assert o.run(wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.dispatched_x, wl.expert_offsets,
                 wl.row_src_rank, wl.row_slot, wl.w1, wl.w3, wl.w2, bufs, rr) == 0
    mask = [np.zeros(b.shape[0], bool) for b in bufs]
    for r, s in zip(wl.row_src_rank, wl.row_slot):
        mask[r][s] = True
    for r, b in enumerate(bufs):
        assert np.all(b[~mask[r]] == SENTINEL)
        assert not np.any(np.all(b[mask[r]] == SENTINEL, axis=1))


def test_validation_codes(o):
    wl = make_workload("tiny", weights=None)
    args = (wl.H, wl.F, wl.E_l, wl.R, wl.self_rank, wl.rows)

    def v(off=wl.expert_offsets, src=wl.row_src_rank, slot=wl.row_slot, rr=wl.return_rows, a=args):
        return o.validate(*a, off, src, slot, rr)

    assert v() == 0
    off = wl.expert_offsets.copy(); off[1] = off[2] + 1
    assert v(off=off) == orc.EROUTING                      # non-monotone offsets
    off = wl.expert_offsets.copy(); off[-1] -= 1
    assert v(off=off) == orc.EROUTING                      # offsets do not end at rows
    src = wl.row_src_rank.copy(); src[3] = wl.R
    assert v(src=src) == orc.EROUTING                      # source rank out of range
    slot = wl.row_slot.copy(); slot[5] = wl.return_rows[wl.row_src_rank[5]]
    assert v(slot=slot) == orc.EROUTING                    # slot beyond the receive buffer
    slot = wl.row_slot.copy(); src = wl.row_src_rank.copy()
    src[7], slot[7] = src[8], slot[8]
    assert v(src=src, slot=slot) == orc.EROUTING           # duplicate (rank, slot)
    assert v(a=(0,) + args[1:]) == orc.EINVAL
    assert v(a=args[:4] + (wl.R,) + args[5:]) == orc.EINVAL  # self rank out of range


def test_empty_stage(o):
    """No routed rows: nothing is written and the call succeeds."""
    bufs = [np.full((4, 64), SENTINEL, np.uint16)]
    z = np.zeros(0, np.int32)
    w = np.zeros((1, 64, 64), np.uint16)
    assert o.run(64, 64, 1, 1, 0, np.zeros((0, 64), np.uint16), np.zeros(2, np.int32), z, z,
                 w, w, w, bufs) == 0
    assert np.all(bufs[0] == SENTINEL)


@pytest.mark.parametrize("mutation", [1, 2, 3, 4, 5])
def test_pins_catch_planted_mistakes(mutation):
    """A plausible mistake anywhere in the oracle must fail at least one pin."""
    with tempfile.TemporaryDirectory() as d:
        lib = orc.build(os.path.join(d, f"libmut{mutation}.so"), mutation=mutation)
        bad = orc.Oracle(lib)
        wls, bufs = _run_all_owners(bad)
        fails = _check_vs_bruteforce(bad, wls, bufs)
        if not fails:   # the identity closed form must catch what the brute force missed
            wls, bufs = _run_all_owners(bad, weights="identity")
            fails = _check_vs_bruteforce(bad, wls, bufs)
        assert fails, f"planted mistake {mutation} went undetected"
