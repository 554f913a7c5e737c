"""The C-ABI library loads and exports exactly what include/moe_stage.h declares (no GPU)."""
import ctypes
import os
import re
import subprocess

import numpy as np
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


def _c_layout(tmp_path, struct, fields):
    """sizeof and offsetof of `fields` in `struct` as the C compiler lays it out from the header."""
    src = tmp_path / "layout.c"
    body = "".join(f'  printf("%zu\\n", offsetof({struct}, {f}));\n' for f in fields)
    src.write_text(f'#include <stddef.h>\n#include <stdio.h>\n#include "moe_stage.h"\n'
                   f'int main(void) {{\n  printf("%zu\\n", sizeof({struct}));\n{body}  return 0;\n}}\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True,
                                           text=True).stdout.split()]
    return vals[0], vals[1:]


@pytest.mark.parametrize("cname, cls", [("moe_stage_config_t", B.moe_stage_config_t),
                                        ("moe_stage_stats_t", B.moe_stage_stats_t),
                                        ("moe_stage_times_t", B.moe_stage_times_t),
                                        ("moe_plan_info_t", B.moe_plan_info_t),
                                        ("moe_wg_record_t", B.moe_wg_record_t),
                                        ("moe_copy_record_t", B.moe_copy_record_t),
                                        ("moe_span_t", B.moe_span_t)])
def test_struct_layout_matches_header(tmp_path, cname, cls):
    fields = [f for f, _ in cls._fields_]
    size, offsets = _c_layout(tmp_path, cname, fields)
    assert ctypes.sizeof(cls) == size
    assert [getattr(cls, f).offset for f in fields] == offsets


def test_unknown_config_flags_rejected():
    with pytest.raises(B.MoeError) as ei:
        B.moe_stage_create(B.make_config(256, 512, 2, 4, 0, 128, flags=1 << 20))
    assert ei.value.code == B.MOE_EINVAL


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


def test_combine_checks_arguments_before_touching_the_device():
    lib = B.load()
    p = 4096  # an aligned stand-in address; no call below reaches the device
    assert lib.moe_combine(None, 0, 64, None, None, 0, 2, None, None, None) == B.MOE_OK   # no tokens
    assert lib.moe_combine(p, 8, 0, p, p, 4, 2, p, None, None) == B.MOE_EINVAL           # hidden 0
    assert lib.moe_combine(p, 8, 64, p, p, 4, 0, p, None, None) == B.MOE_EINVAL          # k 0
    assert lib.moe_combine(p, 8, 64, None, p, 4, 2, p, None, None) == B.MOE_EINVAL       # null slot
    assert lib.moe_combine(None, 8, 64, p, p, 4, 2, p, None, None) == B.MOE_EINVAL       # null recv
    assert lib.moe_combine(p, 8, 12, p, p, 4, 2, p, None, None) == B.MOE_EUNSUPPORTED    # H % 8
    assert lib.moe_combine(p + 8, 8, 64, p, p, 4, 2, p, None, None) == B.MOE_EUNSUPPORTED  # alignment
    assert lib.moe_combine(p, 2 ** 31, 64, p, p, 4, 2, p, None, None) == B.MOE_EUNSUPPORTED
    assert "moe_combine" in B.moe_stage_last_error(None)


def test_handle_entry_points_reject_a_null_handle():
    """Every handle entry point checks its handle before anything else (no device needed)."""
    lib = B.load()
    st = B.moe_stage_stats_t()
    tm = B.moe_stage_times_t()
    info = B.moe_plan_info_t()
    null10 = [None] * 9
    assert lib.moe_stage_run(None, *null10, 8, None) == B.MOE_EINVAL
    assert lib.moe_stage_run_serial(None, *null10, None) == B.MOE_EINVAL
    assert lib.moe_stage_run_devplan(None, *null10, 8, None) == B.MOE_EINVAL
    assert lib.moe_stage_run_serial_devplan(None, *null10, None) == B.MOE_EINVAL
    assert lib.moe_stage_query(None, ctypes.byref(st)) == B.MOE_EINVAL
    assert lib.moe_stage_times(None, 0, ctypes.byref(tm)) == B.MOE_EINVAL
    assert lib.moe_stage_plan_info(None, ctypes.byref(info)) == B.MOE_EINVAL
    assert lib.moe_stage_plan_copy(None, B.MOE_PLAN_ITEMS, None, 0) == B.MOE_EINVAL
    assert lib.moe_stage_records(None, B.MOE_RECORDS_SPAN, None, 0) == B.MOE_EINVAL
    assert lib.moe_stage_destroy(None) == B.MOE_EINVAL


def test_device_plan_flag_is_a_known_config_flag():
    """MOE_TEST_PLAN_NO_LDS passes configuration checks (the host planner ignores it)."""
    wl_cfg = B.make_config(256, 512, 2, 4, 0, 128, flags=B.MOE_LOCAL_DIRECT | B.MOE_TEST_PLAN_NO_LDS)
    off = [0, 1, 2]
    p = B.moe_plan_build(wl_cfg, off, [1, 2], [0, 0], [4, 4, 4, 4])
    assert p["info"]["n_valid"] == 2


def test_configs_whose_offsets_would_wrap_32_bits_are_rejected():
    """Gathered token rows and the activation workspace's K blocks are addressed with 32-bit
    offsets: a configuration past 4 GiB for either is refused before the device is touched."""
    ok = B.make_config(65536, 512, 1, 1, 0, 32767)           # 32767 x 64 Ki x 2 B < 4 GiB
    p = B.moe_plan_build(ok, [0, 1], [0], [0], [1])
    assert p["info"]["n_valid"] == 1
    for cfg in (B.make_config(65536, 512, 1, 1, 0, 32768),    # exactly 4 GiB of dispatched_x
                B.make_config(7168, 2048, 32, 8, 0, 1 << 23 | 1 << 22)):  # 12 Mi rows x 14 KiB
        with pytest.raises(B.MoeError) as ei:
            B.moe_plan_build(cfg, [0] * (cfg.num_local_experts + 1), [], [], [1] * cfg.num_ranks)
        assert ei.value.code == B.MOE_EUNSUPPORTED
        with pytest.raises(B.MoeError) as ei:
            B.moe_stage_create(cfg)
        assert ei.value.code == B.MOE_EUNSUPPORTED
    # a padded layout whose workspace K blocks pass 4 GiB (2^25 rows of 128 bytes)
    big = B.make_config(64, 64, 4096, 64, 0, (1 << 24) - 1, band_rows=256)
    with pytest.raises(B.MoeError) as ei:
        B.moe_stage_create(big)
    assert ei.value.code == B.MOE_EUNSUPPORTED


def _meta(torch, *shape, dtype=None):
    return torch.empty(*shape, dtype=dtype or torch.int16, device="meta")


@pytest.mark.parametrize("case", ["return_count", "return_rows", "return_width", "x_rows", "x_width", "w1", "w3",
                                  "w2", "dtype", "offsets", "routing_len", "ok"])
def test_binding_checks_buffer_shapes_before_the_library(case):
    """The run wrappers refuse buffers smaller than the call describes (ValueError) before any
    pointer reaches the library; meta tensors carry shapes without memory, so no GPU is needed."""
    torch = pytest.importorskip("torch")
    H, F, E, R = 256, 512, 2, 4
    cfg = B.make_config(H, F, E, R, 0, 64)
    off, src, slot = np.array([0, 3, 5]), np.zeros(5, np.int32), np.arange(5, dtype=np.int32)
    x, w1, w3, w2 = _meta(torch, 5, H), _meta(torch, E, F, H), _meta(torch, E, F, H), _meta(torch, E, H, F)
    bufs, rr = [_meta(torch, 8, H) for _ in range(R)], np.full(R, 8)
    if case == "return_count":
        bufs = bufs[:3]
    elif case == "return_rows":
        rr = np.array([8, 8, 9, 8])
    elif case == "return_width":
        bufs[1] = _meta(torch, 8, H + 64)
    elif case == "x_rows":
        x = _meta(torch, 4, H)
    elif case == "x_width":
        x = _meta(torch, 5, H * 2)
    elif case == "w1":
        w1 = _meta(torch, E, F, H - 64)
    elif case == "w3":
        w3 = _meta(torch, E + 1, F, H)
    elif case == "w2":
        w2 = _meta(torch, E, F, H)          # transposed
    elif case == "dtype":
        w2 = _meta(torch, E, H, F, dtype=torch.float32)
    elif case == "offsets":
        off = np.array([0, 5])
    elif case == "routing_len":
        src = np.zeros(4, np.int32)
    args = (cfg, x, int(off[-1]), (off.size, src.size, slot.size), w1, w3, w2, bufs, rr)
    if case == "ok":
        B.validate_run_args(*args)
    else:
        with pytest.raises(ValueError):
            B.validate_run_args(*args)


def test_run_wrappers_refuse_a_handle_they_did_not_create():
    with pytest.raises(ValueError):
        B.moe_stage_run(12345, None, [0, 0, 0], [], [], None, None, None, [], None)
