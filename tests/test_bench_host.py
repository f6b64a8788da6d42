"""Host-side logic of bench.py (no GPU): the one-GPU refusal, the roofline
table over per-call timings, and the lookup of hardware-counter traffic,
which must give nothing once the kernel sources differ from those the
counters were taken with."""
import hashlib
import importlib.util
import json
import os
import subprocess
import sys
from types import SimpleNamespace

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_roofline_takes_the_kind_with_the_largest_total_time(bench):
    # two matmuls of 1e12 FLOP (1 ms, 2 ms), one quantise of 4e9 bytes (1 ms) per step
    step = SimpleNamespace(calls=[("a", "gemm_fwd", 1e12, None), ("b", "quantise", 4e9, None),
                                  ("c", "gemm_dw", 1e12, None)])
    per_call = [[1e-3, 1e-3, 2e-3], [1e-3, 1e-3, 2e-3]]
    roof, table = bench.roofline(step, per_call)
    assert roof["kernel"] == "gemm_dw" and roof["bound"] == "mfma"
    assert roof["achieved"] == pytest.approx(500.0)          # 1e12 FLOP / 2 ms, in TFLOP/s
    assert roof["frac"] == pytest.approx(500.0 / bench.FP8_PEAK_TFLOPS)
    assert table["quantise"]["achieved"] == pytest.approx(4000.0)  # 4e9 B / 1 ms, in GB/s
    assert table["quantise"]["bound"] == "hbm" and table["gemm_fwd"]["achieved"] == pytest.approx(1000.0)


def test_decode_matmuls_are_priced_against_hbm(bench):
    step = SimpleNamespace(calls=[("d", "gemm_decode", 8e9, None)])
    roof, table = bench.roofline(step, [[2e-3]])
    assert roof["bound"] == "hbm" and roof["achieved"] == pytest.approx(4000.0)
    assert "gemm_decode" in bench.COLD_KINDS


def _fake_tree(tmp_path, sources, record):
    csrc = tmp_path / "paper_2309_17224_amd" / "csrc"
    csrc.mkdir(parents=True)
    for name, text in sources.items():
        (csrc / name).write_bytes(text)
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "hbm_traffic_w.json").write_text(json.dumps(record))


def test_traffic_is_given_only_for_the_sources_it_was_measured_with(bench, tmp_path, monkeypatch):
    sources = {"fp8lin_gemm.hip": b"g", "fp8lin_amax_cast.hip": b"a", "fp8lin_fp8.h": b"f"}
    h = hashlib.sha256()
    for name in ("fp8lin_gemm.hip", "fp8lin_amax_cast.hip", "fp8lin_fp8.h"):
        h.update(sources[name])
    _fake_tree(tmp_path, sources, {"kernel_sources_sha256": h.hexdigest(),
                                   "bytes_per_launch": {"gemm_dw": 123}})
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w", "gemm_dw") == 123
    assert bench.measured_traffic("w", "gemm_fwd") is None
    assert bench.measured_traffic("other", "gemm_dw") is None
    (tmp_path / "paper_2309_17224_amd" / "csrc" / "fp8lin_gemm.hip").write_bytes(b"changed")
    assert bench.measured_traffic("w", "gemm_dw") is None


def test_committed_traffic_matches_the_committed_sources(bench):
    """The counters under profiles/ were taken with the kernels as they are
    now; when a kernel has changed since, bench.py reports no traffic, and
    this says so rather than failing the suite."""
    rec = json.load(open(os.path.join(ROOT, "profiles", "hbm_traffic_llama2-7b-up.json")))
    got = bench.measured_traffic("llama2-7b-up", "gemm_dw")
    if got is None:
        pytest.skip("kernel sources changed since the HBM counters were taken: re-take them")
    assert got == rec["bytes_per_launch"]["gemm_dw"]
