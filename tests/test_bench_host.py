"""bench.py pieces that run without a GPU: the one-GPU refusal, the lookup of the committed
traffic record and the oracle baseline leg."""
import importlib.util
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_record_needs_the_same_source_and_flags(bench, tmp_path, monkeypatch):
    from paper_2608_11688_amd import build, configs
    cfg = configs.CONFIGS["granite-1b-a400m"]
    rec = json.load(open(os.path.join(ROOT, "profiles", "moe_ffn_traffic.json")))["records"][0]
    assert bench.measured_traffic(cfg, 1) == rec["traffic_bytes_per_call"]
    assert bench.measured_traffic(cfg, 8) is None                  # no record for batch 8
    assert bench.measured_traffic(cfg, 1, weights="fp8") is None
    monkeypatch.setattr(build, "HIPCC_FLAGS", build.HIPCC_FLAGS + ["-DOTHER"])
    assert bench.measured_traffic(cfg, 1) is None                  # other compiler flags


def test_cpu_baseline_fields(bench):
    from paper_2608_11688_amd import configs
    cfg = configs.CONFIGS["tiny"]
    base, ties = bench.cpu_baseline(cfg, 1, 0, cfg.tau, budget_s=1.0)
    assert set(base) == {"value", "unit", "cores", "kind", "sample"}
    assert base["kind"] == "oracle" and base["unit"] == "us/token/layer" and base["value"] > 0
    assert ties["token_layers"] >= 1 and 0 <= ties["gate_cut"] <= ties["token_layers"]
    one, _ = bench.cpu_baseline(cfg, 1, 0, cfg.tau, budget_s=0.5, threads_limit=1)
    assert one["cores"] == 1
