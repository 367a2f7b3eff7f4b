"""Host-side logic of bench.py (no GPU): the one-GPU guard, the roofline
object, the source hash that ties committed counter summaries to the kernels,
and reading those summaries."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr and r.stdout == ""


def test_roofline_fields(bench):
    rf = bench.roofline(1_000_000_000, 0.25, None)        # 1 GB in 0.25 ms = 4000 GB/s
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["achieved"] == pytest.approx(4000.0) and rf["frac"] == pytest.approx(0.5)
    assert rf["traffic"] is None and rf["algorithmic_bytes"] == 1_000_000_000


def test_source_hash_ignores_comments_only(bench):
    a = "int f(int x) { return x + 1; }  // add one\n/* block */\n"
    b = "int f(int x) { return x + 1; }\n"
    c = "int f(int x) { return x + 2; }\n"
    assert bench._code_only(a) == bench._code_only(b) != bench._code_only(c)
    assert len(bench.kernel_source_hash()) == 16


def test_traffic_summary_read_only_for_the_current_sources(bench, tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    f = tmp_path / "profiles" / "traffic_verify_demo.txt"
    f.write_text("# comment: ignored\nsource_hash: abc\nhbm_bytes_per_launch: 1234\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.load_traffic("verify", "demo", "abc") == 1234.0
    assert bench.load_traffic("verify", "demo", "other") is None
    assert bench.load_traffic("commit", "demo", "abc") is None
