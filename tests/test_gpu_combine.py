"""GPU parity of the weighted combine (paper Section 2.1, step 5) against the CPU oracle.

The kernel and the oracle take the same fp32 steps in the same order (a rounded product,
then a rounded add, choices in ascending order, from +0) and the same bf16 rounding, so
outputs are compared bit for bit.  The whole-layer test runs every owner's stage on the
GPU into shared receive buffers, then each source rank's combine, and checks the result
against the oracle's combine of the same receive buffers (bitwise) and against the
oracle's own stage + combine (the stage tolerance).
"""
import numpy as np
import pytest

from paper_2607_19539_amd import binding as B
from paper_2607_19539_amd.workload import make_workload, bf16_bits_to_f32
from tests.gpu_helpers import DeviceWorkload, dev_u16, log, make_stage, oracle_bufs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _oracle():
    from oracle import oracle as orc
    return orc.get()


def _inputs(seed, T, k, H, recv_rows=None):
    rng = np.random.default_rng(seed)
    recv_rows = T * k if recv_rows is None else recv_rows
    recv = (rng.standard_normal((recv_rows, H)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    slot = np.stack([rng.permutation(recv_rows)[:k] for _ in range(T)]).astype(np.int32) if T else \
        np.zeros((0, k), np.int32)
    g = rng.random((T, k)).astype(np.float32) + np.float32(0.05)
    gate = (g / g.sum(axis=1, keepdims=True)).astype(np.float32) if T else np.zeros((0, k), np.float32)
    return recv, slot, gate


def _gpu_combine(recv, slot, gate, bad=None):
    T, _ = slot.shape
    out = torch.full((T, recv.shape[1]), 0x7FC1, dtype=torch.int16, device="cuda")
    B.moe_combine(dev_u16(torch, recv), torch.from_numpy(slot).cuda(), torch.from_numpy(gate).cuda(), out,
                  bad_slots=bad)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint16)


def _oracle_combine(recv, slot, gate):
    out = np.empty((slot.shape[0], recv.shape[1]), np.uint16)
    assert _oracle().combine(recv, slot, gate, out) == 0
    return out


# (T, k, H): one vector per thread, two, four; several spans per token; ragged spans;
# k above and below the kernel's batch of four choices; one token; no tokens.
SHAPES = [(64, 2, 256), (37, 4, 72), (5, 8, 8), (300, 2, 4096), (17, 3, 7168), (3, 5, 65536),
          (1, 1, 2056), (129, 6, 2048), (0, 2, 512)]


@pytest.mark.parametrize("T,k,H", SHAPES)
def test_combine_bitexact(T, k, H):
    log(f"combine T={T} k={k} H={H}")
    recv, slot, gate = _inputs(T * 7 + k, T, k, H)
    got = _gpu_combine(recv, slot, gate)
    assert np.array_equal(got, _oracle_combine(recv, slot, gate))


def test_combine_full_size():
    """Source rank of the Mixtral-8x7B workload: 4096 tokens, k = 2, H = 4096."""
    wl = make_workload("mixtral", weights=None)
    log("combine mixtral full size")
    recv, _, _ = _inputs(11, wl.T_r, wl.k, wl.H)
    slot = np.ascontiguousarray(wl.slots[0]).astype(np.int32)
    gate = np.ascontiguousarray(wl.gates[0]).astype(np.float32)
    got = _gpu_combine(recv, slot, gate)
    assert np.array_equal(got, _oracle_combine(recv, slot, gate))


def test_combine_counts_and_skips_bad_slots():
    recv, slot, gate = _inputs(5, 40, 3, 256)
    slot[3, 1] = -1
    slot[17, 2] = recv.shape[0]
    slot[17, 0] = 2 ** 31 - 1
    bad = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = _gpu_combine(recv, slot, gate, bad)
    assert int(bad.item()) == 3
    # a skipped term equals a zero-weight term on a valid row (finite inputs, sum from +0)
    s2, g2 = slot.copy(), gate.copy()
    for t, j in ((3, 1), (17, 2), (17, 0)):
        s2[t, j], g2[t, j] = 0, 0.0
    assert np.array_equal(got, _oracle_combine(recv, s2, g2))


def test_combine_rejects_bad_arguments():
    recv = torch.zeros((8, 12), dtype=torch.int16, device="cuda")
    slot = torch.zeros((2, 2), dtype=torch.int32, device="cuda")
    gate = torch.zeros((2, 2), dtype=torch.float32, device="cuda")
    out = torch.zeros((2, 12), dtype=torch.int16, device="cuda")
    with pytest.raises(B.MoeError) as e:
        B.moe_combine(recv, slot, gate, out)
    assert e.value.code == B.MOE_EUNSUPPORTED


def test_layer_end_to_end():
    """Every owner's stage on the GPU, then every source rank's combine."""
    name = "tiny"
    R = make_workload(name, weights=None).R
    wls = [make_workload(name, owner=r, keep_sources=True) for r in range(R)]
    dws = [DeviceWorkload(torch, wl) for wl in wls]
    shared = dws[0].bufs
    ref_bufs = [np.full((int(n), wls[0].H), 0x7FC1, np.uint16) for n in wls[0].return_rows]
    for wl, dw in zip(wls, dws):
        dw.bufs = shared
        log(f"layer: owner {wl.self_rank}")
        with make_stage(wl) as st:
            st.run(*dw.args(), cu_split=8)
            torch.cuda.synchronize()
            st.query()
        ob = oracle_bufs(wl)
        for r in range(R):
            w = ~np.all(ob[r] == 0x7FC1, axis=1)
            ref_bufs[r][w] = ob[r][w]
    gpu_recv = [b.cpu().numpy().view(np.uint16) for b in shared]
    wl0 = wls[0]
    for r in range(R):
        slot = np.ascontiguousarray(wl0.slots[r]).astype(np.int32)
        gate = np.ascontiguousarray(wl0.gates[r]).astype(np.float32)
        got = _gpu_combine(gpu_recv[r], slot, gate)
        assert np.array_equal(got, _oracle_combine(gpu_recv[r], slot, gate))
        want = bf16_bits_to_f32(_oracle_combine(ref_bufs[r], slot, gate)).astype(np.float64)
        g = bf16_bits_to_f32(got).astype(np.float64)
        assert np.all(np.abs(g - want) <= 1e-2 * np.maximum(1.0, np.abs(want)))
