"""The C-ABI library loads and exports exactly what include/moe_stage.h declares (no GPU)."""
import ctypes
import os
import re
import subprocess

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
                                        ("moe_plan_info_t", B.moe_plan_info_t)])
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
    assert lib.moe_stage_destroy(None) == B.MOE_EINVAL


def test_device_plan_flag_is_a_known_config_flag():
    """MOE_TEST_PLAN_NO_LDS passes configuration checks (the host planner ignores it)."""
    wl_cfg = B.make_config(256, 512, 2, 4, 0, 128, flags=B.MOE_LOCAL_DIRECT | B.MOE_TEST_PLAN_NO_LDS)
    off = [0, 1, 2]
    p = B.moe_plan_build(wl_cfg, off, [1, 2], [0, 0], [4, 4, 4, 4])
    assert p["info"]["n_valid"] == 2
