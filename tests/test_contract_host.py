"""Host-side checks of the product boundary (CPU).

* bench.py measures one GPU only and says so for --gpus N > 1.
* The binding refuses to run without a GPU: there is no CPU fallback.
* The product (the HIP library and its binding) and the oracle share no code:
  neither imports nor includes the other, and the oracle's C source uses no
  HIP header.
"""
import os
import re
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_13500_amd")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the behaviour without a GPU")
def test_reducer_fails_loudly_without_a_gpu():
    import paper_2607_13500_amd as tr
    with pytest.raises(RuntimeError, match="GPU"):
        tr.Reducer(64, 64, torch.bfloat16, max_images=1, max_tokens=64, max_N=64)


def _sources(top, exts):
    for dirpath, _, files in os.walk(top):
        for f in files:
            if f.endswith(exts):
                yield os.path.join(dirpath, f)


def test_product_never_uses_the_oracle():
    for path in _sources(PKG, (".py", ".hip", ".h", ".cpp", ".c")):
        text = open(path).read()
        assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), path
        assert not re.search(r'#\s*include\s*[<"][^>"]*(oracle|altr_oracle)', text), path
        assert "libaltr_oracle" not in text, path


def test_oracle_uses_no_product_code():
    for path in _sources(os.path.join(ROOT, "oracle"), (".py", ".c", ".h")):
        text = open(path).read()
        assert not re.search(r"^\s*(import|from)\s+paper_2607_13500_amd\b", text, re.M), path
        assert not re.search(r'#\s*include\s*[<"](hip/|tr\.h|tr_internal|tr_wave)', text), path
        assert "libaltr.so" not in text, path
