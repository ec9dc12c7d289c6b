"""The C ABI from plain C: tests/c_client/reduce_client.c uses only
include/tr.h and the HIP runtime's C API (no C++, no torch).  The CPU test
compiles it with warnings as errors; the GPU test runs it and checks the
outputs it writes against the fp64 oracle with the parity protocol."""
import os
import subprocess

import numpy as np
import pytest
import torch

import parity
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2607_13500_amd")
N = [576, 300, 1000]
K = [64, 40, 111]
D, DC = 1024, 768


def _build(tmp_path):
    exe = tmp_path / "reduce_client"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-O2", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "c_client", "reduce_client.c"),
           "-L", LIBDIR, "-laltr", "-L", "/opt/rocm/lib", "-lamdhip64", "-lm",
           "-Wl,-rpath," + LIBDIR, "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return exe


def test_c_client_compiles_against_the_header(tmp_path):
    from paper_2607_13500_amd import _lib
    _lib.load()   # the library it links is built
    assert _build(tmp_path).exists()


MODES = {"fp32": dict(), "bf16": dict(), "bf16-shannon": dict(entropy=1), "fp32-stride-real": dict(stride_mode=1)}


@pytest.mark.gpu
@pytest.mark.parametrize("mode", list(MODES))
def test_c_client_matches_the_oracle(mode, tmp_path):
    print("[case] plain C client, %s: 3 images (576, 300, 1000 tokens) x 1024, states 768" % mode, flush=True)
    exe = _build(tmp_path)
    run = subprocess.run([str(exe), str(tmp_path), mode], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "c client ok (%s)" % mode in run.stdout
    rows, kept = sum(N), sum(K)

    def load(name, dtype, shape):
        return torch.from_numpy(np.fromfile(str(tmp_path / name), dtype=dtype).reshape(shape))

    # (bf16 modes: the arrays hold the bf16 values the library read, widened
    # exactly to fp32, and the kept rows widened the same way)
    X = load("X.f32", np.float32, (rows, D))
    P = load("P.f32", np.float32, (rows, DC))
    Q = load("Q.f32", np.float32, (rows, DC))
    from paper_2607_13500_amd import ReduceResult
    res = ReduceResult(out=load("out.f32", np.float32, (kept, D)),
                       idx=load("idx.i32", np.int32, (kept,)),
                       src=load("src.u8", np.uint8, (kept,)),
                       h2=load("h2.f32", np.float32, (rows,)),
                       s=load("s.f32", np.float32, (rows,)))
    w = synth.Workload("c-client", X, P, Q, list(N), list(K), synth.LAMBDA)
    kw = MODES[mode]
    rep = parity.check(w, res, parity.oracle_reference(w, **kw), **kw)
    print("   ", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
