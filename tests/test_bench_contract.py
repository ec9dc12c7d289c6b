"""bench.py's JSON line meets the measurement contract (tests/bench_contract.py):
the line recorded in profiles/ (CPU), and a short run of bench.py itself on
the GPU."""
import json
import os
import re
import subprocess

import pytest

import bench_contract

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_recorded_bench_line_meets_the_contract():
    text = open(os.path.join(ROOT, "profiles", "bench_other_workloads.md")).read()
    m = re.search(r"^    (\{\"metric\".*\})$", text, re.M)
    assert m, "no JSON line in the workloads profile"
    line = json.loads(m.group(1))
    assert bench_contract.problems(line) == []
    assert set(line["workloads"]) == {"llava_k128", "llava_k192", "llava_fp32", "llava_fp32_k192", "llava_next",
                                      "qwen_ragged", "video"}


def test_validator_catches_broken_lines():
    good = {"metric": "m", "value": 100.0, "unit": "images/s", "n_gpus": 1, "steps": 2, "warmup": 1,
            "ms_per_step": 10.0, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic", "config": {"workload": "w", "images": 1},
            "roofline": {"bound": "hbm", "achieved": 4000.0, "peak": 8000.0, "unit": "GB/s", "frac": 0.5,
                         "traffic": None},
            "cpu_baseline": {"value": 1.0, "unit": "images/s", "cores": 1, "kind": "oracle", "sample": "s"}}
    assert bench_contract.problems(good) == []
    for mutate in (lambda d: d.pop("roofline"), lambda d: d.update(n_gpus=2), lambda d: d.update(vs_baseline=1.0),
                   lambda d: d["roofline"].update(frac=0.7), lambda d: d["roofline"].update(peak=5000.0),
                   lambda d: d.update(value=200.0), lambda d: d["cpu_baseline"].update(kind="tuned"),
                   lambda d: d.pop("cpu_baseline"), lambda d: d["config"].pop("workload")):
        bad = json.loads(json.dumps(good))
        mutate(bad)
        assert bench_contract.problems(bad), bad


@pytest.mark.gpu
def test_bench_line_from_a_short_run():
    print("[case] bench.py --steps 3 --warmup 1 --no-workloads --cpu-seconds 0.5", flush=True)
    res = subprocess.run(["python3", os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1", "--no-workloads",
                          "--cpu-seconds", "0.5"], capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, res.stdout
    line = json.loads(lines[0])
    assert bench_contract.problems(line) == []
    assert line["roofline"]["traffic_source"]["status"] == "current", line["roofline"]["traffic_source"]
    assert line["roofline"]["traffic"] is not None
