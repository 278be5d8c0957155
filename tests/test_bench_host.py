"""bench.py pieces that run without a GPU: the one-GPU refusal, the lookup of the committed
traffic record and the oracle baseline leg."""
import importlib.util
import json
import os
import subprocess
import sys

import numpy as np
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
    cfg = configs.CONFIGS["mixtral-8x7b"]          # the bench's default workload
    recs = json.load(open(os.path.join(ROOT, "profiles", "moe_ffn_traffic.json")))["records"]
    pick = lambda w: [r for r in recs if r["workload"] == cfg.name and r["batch"] == 1 and
                      r["weights"] == w][0]
    assert bench.measured_traffic(cfg, 1) == pick("bf16")["traffic_bytes_per_call"]
    assert bench.measured_traffic(cfg, 1, weights="fp8") == pick("fp8")["traffic_bytes_per_call"]
    assert bench.measured_traffic(cfg, 8) is None                  # no record for batch 8
    assert bench.measured_traffic(cfg, 1, weights="fp32") is None  # nor for fp32 experts
    monkeypatch.setattr(build, "HIPCC_FLAGS", build.HIPCC_FLAGS + ["-DOTHER"])
    assert bench.measured_traffic(cfg, 1) is None                  # other compiler flags


def test_cpu_baseline_fields(bench):
    from paper_2608_11688_amd import configs
    cfg = configs.CONFIGS["tiny"]
    sample = bench.oracle_sample(cfg, 1, "bf16", 0, None)
    assert sample["layers"] == [0] and sample["steps"] == 64
    # every expert of the sampled layers is drawn before the timed run
    assert len(sample["states"][0]._bits) == cfg.E
    base, ties = bench.cpu_baseline(cfg, 1, 0, cfg.tau, 1.0, sample)
    assert set(base) == {"value", "unit", "cores", "kind", "sample"}
    assert base["kind"] == "oracle" and base["unit"] == "us/token/layer" and base["value"] > 0
    assert "drawn before timing" in base["sample"]
    assert ties["token_layers"] >= 1 and 0 <= ties["gate_cut"] <= ties["token_layers"]
    one, _ = bench.cpu_baseline(cfg, 1, 0, cfg.tau, 0.5, sample, threads_limit=1)
    assert one["cores"] == 1


def test_oracle_sample_of_large_experts(bench):
    # experts of 352 MB: two layers (under 8 GB of drawn weights), 16 steps
    from paper_2608_11688_amd import configs
    cfg = configs.CONFIGS["mixtral-8x7b"]
    S = 6 * cfg.d * cfg.I
    assert int(8e9 // (cfg.E * S)) == 2 and S >= (64 << 20)


def test_selection_stats_match_the_oracle_metrics(bench):
    """The per-layer leg's host accounting against the oracle's enumerations of Eq. 2, Eq. 3
    and the overlap of Sec. V-C, on random rankings, routed sets and prefix sizes
    (m = 0, the no-prefetch case, included)."""
    from oracle import metrics
    rng = np.random.default_rng(7)
    N, k, k_max, n = 12, 3, 8, 400
    ranked = np.stack([rng.permutation(N) for _ in range(n)])
    routed = np.stack([rng.choice(N, k, replace=False) for _ in range(n)])
    m = rng.integers(0, k_max + 1, n)
    m[:10] = 0
    sel = np.where(np.arange(k_max)[None, :] < m[:, None], ranked[:, :k_max], -1)
    st = bench.selection_stats(ranked, routed, sel, m, k)
    for i in range(n):
        K_p = [int(e) for e in sel[i] if e >= 0]
        assert st["delta_star"][i] == metrics.delta_star(list(ranked[i]), list(routed[i]), k)
        assert st["delta_hat"][i] == max(int(m[i]) - k, 0)
        assert st["overlap"][i] == pytest.approx(metrics.overlap(routed[i], K_p, k))
        assert bool(st["coverage"][i]) == metrics.full_coverage(routed[i], K_p)
    # entries past m are ignored even when they hold expert ids
    st2 = bench.selection_stats(ranked, routed, ranked[:, :k_max], m, k)
    assert np.array_equal(st2["overlap"], st["overlap"])


def test_every_weight_format_names_its_kernels(bench):
    for w in ("bf16", "fp8", "mxfp4", "fp32"):
        assert (w, True) in bench.FFN_KERNELS
        if w != "fp32":                    # fp32 experts run at batch 1 only
            assert (w, False) in bench.FFN_KERNELS
    assert abs(bench.PCIE_PEAK_GBPS - 63.015) < 1e-2
