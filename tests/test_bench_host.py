"""The host side of bench.py, without a GPU: the one-GPU contract, the HBM
traffic figure that follows the kernel source, and the CPU oracle legs."""
from __future__ import annotations

import os
import re
import shutil
import sys

import pytest

import bench
import seeded_inputs as si


def test_more_than_one_gpu_exits_with_a_message(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err


def _profiles_fresh():
    """Whether the committed counter summaries were taken on the current kernel
    source (after a kernel change they are stale until measured again, and
    bench.py reports no traffic figure meanwhile)."""
    text = open(bench.TRAFFIC_SUMMARY).read()
    return re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text).group(1) == \
        bench.kernel_source_sha256()


def test_traffic_is_reported_only_for_the_profiled_kernel_source(monkeypatch, tmp_path):
    text = open(bench.TRAFFIC_SUMMARY).read()
    value = float(re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text).group(1))
    recorded = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text).group(1)
    if not _profiles_fresh():
        assert bench.committed_traffic() is None
    # the source the counters were taken on gets their figure ...
    monkeypatch.setattr(bench, "kernel_source_sha256", lambda: recorded)
    assert bench.committed_traffic() == value
    monkeypatch.undo()
    # the counter summary is for the current kernel source; any other source
    # (here: one more comment line) gets no traffic figure
    src = tmp_path / "kernel.hip"
    shutil.copy(bench.KERNEL_SOURCE, src)
    with open(src, "a") as f:
        f.write("// edited\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    assert bench.committed_traffic() is None


def test_every_traffic_summary_gives_its_workloads_bytes():
    """Each workload with a counter summary gets its traffic figure, at least
    the algorithmic bytes (Q, K, V read once, O and lse written once)."""
    if not _profiles_fresh():
        pytest.skip("the counter summaries predate the current kernel source")
    for wl in bench.TRAFFIC_SUMMARIES:
        w = si.WORKLOADS[wl]
        es = 1 if w.dtype == "e4m3" else 2
        alg = (w.B * w.N * (w.H * w.d + w.kv_heads * (w.d + w.d_v)) * es
               + w.B * w.H * w.N * (2 * w.d_v + 4))
        t = bench.committed_traffic(wl)
        assert t is not None and 0.99 * alg <= t <= 4 * alg, (wl, t, alg)
    assert bench.committed_traffic("mha_b1_h2_n128_d64_f16") is None


def test_every_profile_summary_names_the_current_kernel_source():
    """Each committed rocprofv3 summary that records a kernel source hash
    records the current one (a kernel change needs fresh profiles)."""
    if not _profiles_fresh():
        pytest.skip("the profile summaries predate the current kernel source")
    sha = bench.kernel_source_sha256()
    prof = os.path.join(os.path.dirname(bench.TRAFFIC_SUMMARY))
    found = 0
    for name in sorted(os.listdir(prof)):
        m = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", open(os.path.join(prof, name)).read())
        if m:
            found += 1
            assert m.group(1) == sha, f"{name} was measured on another kernel source"
    assert found >= 2


def test_cpu_baseline_reports_the_oracle_on_host_cores():
    w = si.WORKLOADS["mha_b1_h2_n128_d64_f16"]
    q, k, v = w.inputs()
    r = bench.cpu_baseline(w, q, k, v)
    affinity, usable = bench.usable_cpus()
    assert r["kind"] == "oracle" and r["unit"] == "TFLOPS"
    assert r["cores"] == usable and r["cores_in_affinity"] == affinity and r["value"] > 0
    assert 1 <= usable <= affinity == len(os.sched_getaffinity(0))
    assert "2 of 2 (batch, head) slices" in r["sample"]


def test_cpu_single_core_times_whole_small_workloads():
    r = bench.cpu_single_core(names=("mha_b1_h2_n128_d64_f16",))
    assert set(r) == {"mha_b1_h2_n128_d64_f16"}
    assert r["mha_b1_h2_n128_d64_f16"]["seconds"] >= 0
    assert r["mha_b1_h2_n128_d64_f16"]["gflops"] > 0


def test_rocm_smi_json_gives_clock_and_power():
    """The sampler reads SCLK and a package-power key (rocm-smi JSON)."""
    import json
    text = json.dumps({"card0": {"sclk clock speed:": "(1804Mhz)",
                                 "Current Socket Graphics Package Power (W)": "1397.0"},
                       "system": {"Driver version": "6.x"}})
    assert bench.SclkSampler.parse(text) == (1804, 1397.0)
    assert bench.SclkSampler.parse(json.dumps({"card0": {}})) == (None, None)
