"""Host logic of bench.py (no GPU): the headline line's number formatting, the interval union
behind the overlap ratio, and the rule that the stored traffic figure is reported only for the
kernel source it was measured on."""
import hashlib
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def test_short_floats_keeps_structure_and_six_digits(bench):
    line = {"value": 1233.2812345678, "n": 7, "flag": True, "none": None, "s": "x",
            "roofline": {"frac": 0.514555123, "traffic": 3292755693.83},
            "sweep": [{"speedup": 0.99209912345}, 1.0]}
    out = bench.short_floats(line)
    assert out == {"value": 1233.28, "n": 7, "flag": True, "none": None, "s": "x",
                   "roofline": {"frac": 0.514555, "traffic": 3292760000.0},
                   "sweep": [{"speedup": 0.992099}, 1.0]}
    assert isinstance(out["n"], int) and isinstance(out["flag"], bool)
    json.dumps(out)  # still one JSON object


def test_union_length(bench):
    total, pieces = bench.union_length([(5, 7), (0, 2), (1, 3), (6, 9)])
    assert total == 3 + 4
    assert pieces == [[0, 3], [5, 9]]
    assert bench.union_length([])[0] == 0


def test_stored_traffic_only_for_the_measured_source(bench, tmp_path, monkeypatch):
    src = tmp_path / "kernels.hip"
    src.write_text("// kernel source\n")
    sha = hashlib.sha256(src.read_bytes()).hexdigest()
    rec = tmp_path / "traffic.md"
    rec.write_text(f"traffic_bytes_per_launch: 3.2916e+09\nkernel_sha256: {sha}\n")
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(rec))
    assert bench.stored_traffic() == pytest.approx(3.2916e9)
    src.write_text("// kernel source, changed\n")  # counters taken on another source: no figure
    assert bench.stored_traffic() is None
    rec.write_text("no figure here\n")
    assert bench.stored_traffic() is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.md"))
    assert bench.stored_traffic() is None

