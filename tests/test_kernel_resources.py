"""Register and scratch budget of the gfx950 kernels, read from the compiler's code-object
metadata (no GPU needed).

A producer wave holds 256 accumulation registers plus its vector registers; in a shared-CU
run two consumer waves must fit beside it on each SIMD (512 registers), and no kernel may
spill to scratch (a spill in the MFMA loop costs an order of magnitude).
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_19539_amd", "csrc")
SOURCES = ["kernels.hip", "combine.hip", "plan_device.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SIMD_REGISTERS = 512
CONSUMER_WAVES_BESIDE_PRODUCER = 2


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    found = {}
    for src in SOURCES:
        out = tmp_path_factory.mktemp("dev") / (src + ".s")
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-x", "hip", "--cuda-device-only",
                        "-S", os.path.join(CSRC, src), f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", "-o", str(out),
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"],
                       check=True, capture_output=True)
        meta = out.read_text().split("amdhsa.kernels:", 1)[1]
        for block in re.split(r"\n  - ", meta)[1:]:
            fields = dict(re.findall(r"^\s*\.(\w+):\s+(\S+)", block, re.M))
            if "name" in fields:
                found[fields["name"]] = fields
    return found


def by_name(kernels, fragment):
    hits = {n: f for n, f in kernels.items() if fragment in n}
    assert hits, fragment
    return hits


def test_no_kernel_spills(kernels):
    for name, f in kernels.items():
        assert int(f["private_segment_fixed_size"]) == 0, name
        assert int(f["vgpr_spill_count"]) == 0, name


def test_consumer_fits_beside_a_producer_wave(kernels):
    """The shared-CU consumer variant (kOwn = false) leaves a producer wave its registers; the
    variant for compute units of its own keeps four waves per SIMD."""
    (cons,) = by_name(kernels, "consumer_kernelILb0ELb0E").values()   # the MOE_WRITE_COUNTS
    (own,) = by_name(kernels, "consumer_kernelILb1ELb0E").values()    # variants are outside it
    assert int(own["vgpr_count"]) <= 128
    granule = 8  # registers are allocated to a wave in blocks of 8
    cons_alloc = -(-int(cons["vgpr_count"]) // granule) * granule
    budget = SIMD_REGISTERS - CONSUMER_WAVES_BESIDE_PRODUCER * cons_alloc
    # The launches taken by default (split 1 to 4 parts) must leave that room.
    for name, f in by_name(kernels, "producer_kernel").items():
        tag = re.search(r"ILb[01]ELi(n?\d+)E", name).group(1)
        split = -int(tag[1:]) if tag.startswith("n") else int(tag)
        if split in (-1, 1, 2, 3, 4):
            assert int(f["vgpr_count"]) <= budget, (name, f["vgpr_count"], budget)
        assert int(f["agpr_count"]) == 256, name


def test_every_split_variant_is_instantiated(kernels):
    names = set(by_name(kernels, "producer_kernel"))
    for down, split in ((0, 1), (1, 1), (1, 2), (1, 3), (1, 4), (1, 0), (1, "n1")):
        assert any(f"ILb{down}ELi{split}E" in n for n in names), (down, split)


def test_combine_variants_present(kernels):
    names = set(by_name(kernels, "combine_kernel"))
    assert len(names) == 3, names


def test_consumer_leaves_lds_to_the_producer(kernels):
    """A producer workgroup takes all of a CU's LDS; a consumer workgroup holding any LDS would
    keep producer workgroups off the compute units the two are meant to share."""
    for cons in by_name(kernels, "consumer_kernel").values():
        assert int(cons["group_segment_fixed_size"]) == 0
    for name, f in by_name(kernels, "producer_kernel").items():
        assert int(f["group_segment_fixed_size"]) == 160 * 1024, name


def test_tail_kernel_fits_beside_the_polling_consumer(kernels):
    """The tail kernel runs while the consumer polls on shared CUs: it holds no LDS (so no
    workgroup waits for LDS it holds) and at most 128 vector registers per wave."""
    (tail,) = by_name(kernels, "tail_kernel").values()
    assert int(tail["group_segment_fixed_size"]) == 0
    assert int(tail["vgpr_count"]) <= 128


def test_device_planner_kernels_present_and_small(kernels):
    """The four planner kernels: single-workgroup ones stay within the 160 KiB of LDS a workgroup
    may hold on gfx950, grid ones use little."""
    names = {n.split("_kernel")[0].rsplit("plan_", 1)[1]: f for n, f in by_name(kernels, "plan_").items()
             if "_kernel" in n}
    assert set(names) == {"rows", "layout", "fill", "segs"}, names
    for part, f in names.items():
        lds = int(f["group_segment_fixed_size"])
        assert lds <= 160 * 1024, (part, lds)
        if part in ("rows", "fill"):
            assert lds <= 32 * 1024, (part, lds)
