"""The measurement contract of bench.py: one JSON line with the fields the harness reads.

bench.main() runs in the test process (argv patched, output captured): no program is started
from a process that may already hold the GPU."""
import json

import pytest

import bench


def run_bench(monkeypatch, capsys, *argv):
    monkeypatch.setattr("sys.argv", ["bench.py", *argv])
    code = 0
    try:
        bench.main()
    except SystemExit as e:
        code = e.code
    out = capsys.readouterr()
    return code, out.out, out.err


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    """Only one GPU is measured: --gpus 2 exits non-zero with a message saying so, before any
    device is touched."""
    code, out, err = run_bench(monkeypatch, capsys, "--gpus", "2")
    assert code not in (0, None)
    assert "one GPU" in err and out == ""


@pytest.mark.gpu
def test_bench_line_contract(monkeypatch, capsys, gpu_ok):
    """A short run (one timed step of the default 100,000 x 32 workload, no side legs) prints one JSON
    line carrying the contract's fields, a roofline whose fraction is achieved / peak, and the
    configuration named by its workload."""
    code, out, err = run_bench(monkeypatch, capsys, "--steps", "1", "--warmup", "0", "--cpu-seconds", "0", "--no-ovo",
                               "--no-paper-shapes", "--no-workloads", "--ws-q=", "--row-path-steps", "0",
                               "--row-large-n", "0")
    assert code in (0, None), err[-2000:]
    lines = [l for l in out.splitlines() if l.strip()]
    assert len(lines) == 1
    b = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline"):
        assert k in b, k
    assert b["n_gpus"] == 1 and b["steps"] == 1 and b["warmup"] == 0
    assert b["value"] > 0 and b["ms_per_step"] > 0 and b["higher_is_better"] is True
    assert "workload" in b["config"] and "model" not in b["config"]
    rf = b["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in rf, k
    assert rf["bound"] in ("hbm", "mfma", "alu")
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) <= 1e-9 * rf["frac"]
    assert "cpu_baseline" not in b  # --cpu-seconds 0 skips the oracle leg
