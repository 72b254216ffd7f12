"""``bench.py --sustain``: each launch of a workload run back to back while the
shader clock is sampled, one JSON line per launch; ``--library`` loads a given
build of the library.  Runs bench.py as a child process on the smallest
workload."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*extra):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "mha_b1_h2_n128_d64_f16",
           "--no-cpu-baseline", "--sustain", "0.3", *extra]
    print("running", " ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert res.returncode == 0, res.stderr[-2000:]
    return [json.loads(l) for l in res.stdout.splitlines() if l.startswith("{")]


def test_sustain_reports_each_launch():
    lines = _run()
    assert [l["launch"] for l in lines] == ["unmasked"]
    (l,) = lines
    assert l["sustained"] and l["library"] == "in-tree"
    assert l["launches"] >= 16 and l["tflops"] > 0
    if l["sclk_mhz"] is not None:   # rocm-smi present
        assert 100 < l["sclk_mhz"] < 5000
        # tflops_per_ghz is rounded to one decimal
        assert l["tflops_per_ghz"] == pytest.approx(l["tflops"] / (l["sclk_mhz"] / 1000), rel=1e-3, abs=0.051)


def test_sustain_with_a_given_library():
    from paper_2506_12355_amd import LIB_PATH
    lines = _run("--library", LIB_PATH)
    assert len(lines) == 1 and lines[0]["library"] == os.path.abspath(LIB_PATH)
    assert lines[0]["tflops"] > 0
