"""The C-ABI library loads and exports exactly what include/moe_stage.h declares (no GPU)."""
import ctypes
import os
import re

import pytest

from paper_2607_19539_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "moe_stage.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_\w+)\s*\(", text)))


def test_header_declares_the_binding_surface():
    assert declared_functions() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = B.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_sizes_match_header_layout():
    # int32 x 9 + uint32 = 40 bytes; stats and plan-info contain int64 fields (8-byte aligned)
    assert ctypes.sizeof(B.moe_stage_config_t) == 40
    assert ctypes.sizeof(B.moe_stage_stats_t) == 4 * 8 + 9 * 4 + 4 + 8 + 2 * 8  # 9 int32 + pad
    assert ctypes.sizeof(B.moe_plan_info_t) == 10 * 4 + 4 * 8


def test_create_without_gpu_fails_loudly():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    cfg = B.make_config(256, 512, 2, 4, 0, 128)
    with pytest.raises(B.MoeError) as ei:
        B.moe_stage_create(cfg)
    assert ei.value.code == B.MOE_EHIP


def test_create_rejects_bad_config_before_touching_the_device():
    for cfg, code in ((B.make_config(200, 512, 2, 4, 0, 128), B.MOE_EUNSUPPORTED),
                      (B.make_config(256, 512, 0, 4, 0, 128), B.MOE_EINVAL),
                      (B.make_config(256, 512, 2, 4, 4, 128), B.MOE_EINVAL),
                      (B.make_config(256, 512, 2, 4, 0, 128, band_rows=24), B.MOE_EINVAL)):
        with pytest.raises(B.MoeError) as ei:
            B.moe_stage_create(cfg)
        assert ei.value.code == code
