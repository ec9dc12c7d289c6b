"""CPU checks of the C ABI library: symbols, host budget plan, validation.

Nothing here launches a kernel.  The plan is checked against the budget split
the paper prints and the keep ratios it runs (tests/golden/).
"""
import ctypes
import os
import re
import subprocess
from fractions import Fraction

import pytest

import paper_2607_13500_amd as tr
from paper_2607_13500_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "tr.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tr_[a-z_A-Z0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert {"tr_create", "tr_reduce", "tr_destroy", "tr_strerror", "tr_score", "tr_select",
            "tr_plan"} <= set(names)
    lib = _lib.load()
    for n in names:
        assert hasattr(lib, n), n
    dyn = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (tr_\w+)", dyn))
    assert set(names) <= exported
    # the product library links the HIP runtime and nothing from the oracle
    assert "altr_oracle" not in dyn


def test_library_built_for_gfx950_only(tmp_path):
    blob = tmp_path / "fatbin.bin"
    res = subprocess.run(["objcopy", "-O", "binary", "--only-section=.hip_fatbin", _lib.LIB_PATH,
                          str(blob)], capture_output=True, text=True)
    if res.returncode != 0:
        pytest.skip("objcopy unavailable")
    targets = set(re.findall(rb"amdgcn-amd-amdhsa--(gfx[0-9a-z]+)", blob.read_bytes()))
    assert targets == {b"gfx950"}


def test_strerror():
    lib = _lib.load()
    assert lib.tr_strerror(0) == b"success"
    assert lib.tr_strerror(1) == b"invalid argument"
    assert lib.tr_strerror(4) == b"HIP device error"
    assert lib.tr_strerror(99) == b"unknown status"


def _rows(name):
    out = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if line:
            out.append(line.split())
    return out


def test_plan_matches_golden_budget_split():
    rows = _rows("budget_split.txt")
    assert any(r[-1] == "paper" for r in rows)
    for N, K, ln, ld, K1, K2, t, _ in rows:
        lam = int(ln) / int(ld)
        Kb, K1b, K2b, tb = tr.plan([int(N)], [int(K)], lam=lam)
        assert (Kb[0], K1b[0], K2b[0], tb[0]) == (int(K), int(K1), int(K2), int(t)), (N, K, lam)


def test_plan_keep_ratio_matches_paper_budgets():
    for N, rn, rd, K in _rows("keep_ratio.txt"):
        ratio = int(rn) / int(rd)
        Kb, _, _, _ = tr.plan([int(N)], None, keep_ratio=ratio)
        assert Kb[0] == int(K), (N, ratio)


def test_plan_keep_ratio_clamps_and_floors():
    Kb, K1, K2, t = tr.plan([1, 5, 9, 16384, 256], None, keep_ratio=0.11)
    assert Kb == [1, 1, 1, 1802, 28]
    # floor(lambda K) with lambda = 1/3
    assert K1 == [0, 0, 0, 600, 9]
    assert all(k1 + k2 == k for k, k1, k2 in zip(Kb, K1, K2))
    Kb, _, _, _ = tr.plan([7], None, keep_ratio=1.0)
    assert Kb == [7]


def test_plan_budget_exhaustive_small():
    # Algorithm 1's split and stride over every (N, K, lambda) on a small grid,
    # checked with exact rational arithmetic (floor of lambda*K for a rational
    # lambda is exact here because lambda*K is never within 1e-12 of an integer
    # unless it is one).
    for N in range(1, 40):
        for K in range(1, N + 1):
            for lam in (Fraction(0), Fraction(1, 4), Fraction(1, 3), Fraction(1, 2), Fraction(2, 3),
                        Fraction(1)):
                Kb, K1b, K2b, tb = tr.plan([N], [K], lam=float(lam))
                k1 = (lam * K).numerator // (lam * K).denominator
                k2 = K - k1
                t = max(1, (N - k1) // k2) if k2 else 0
                assert (Kb[0], K1b[0], K2b[0], tb[0]) == (K, k1, k2, t)
                if k2:
                    assert (k2 - 1) * t < N - k1     # every pick lands inside X^rem


@pytest.mark.parametrize("N,K,kw", [
    ([0], [1], {}),
    ([5], [0], {}),
    ([5], [6], {}),
    ([5, 7], [2, -1], {}),
    ([70000], [5], {}),
    ([5], None, {}),                      # no K and no keep ratio
    ([5], [2], {"lam": 1.5}),
    ([5], [2], {"lam": -0.01}),
    ([5], [2], {"lam": float("nan")}),
    ([5], None, {"keep_ratio": 1.5}),
])
def test_plan_rejects_invalid(N, K, kw):
    with pytest.raises(tr.TRError) as e:
        tr.plan(N, K, **kw)
    assert e.value.status == _lib.TR_EINVAL


def test_plan_empty_batch():
    assert tr.plan([], []) == ([], [], [], [])


def test_create_rejects_bad_params_before_touching_a_device():
    lib = _lib.load()
    ctx = ctypes.c_void_p()
    good = dict(D=64, Dc=0, dtype=1, max_images=4, max_tokens=1024, max_N=512, flags=0,
                lam=1 / 3, keep_ratio=0.0)
    bad = [dict(D=0), dict(Dc=-1), dict(dtype=7), dict(max_images=0), dict(max_tokens=0),
           dict(max_tokens=1 << 31), dict(max_N=0), dict(flags=8), dict(flags=-1), dict(lam=2.0),
           dict(keep_ratio=-0.5)]
    for b in bad:
        p = _lib.Params(**{**good, **b})
        assert lib.tr_create(ctypes.byref(p), ctypes.byref(ctx)) == _lib.TR_EINVAL, b
        assert ctx.value is None
    assert lib.tr_create(None, ctypes.byref(ctx)) == _lib.TR_EINVAL
    assert lib.tr_last_error() != b""


def test_null_context_calls_are_rejected():
    lib = _lib.load()
    N = (ctypes.c_int32 * 1)(4)
    assert lib.tr_reduce(None, None, None, None, 1, N, None, None, None, None, None, None, None) == _lib.TR_EINVAL
    assert lib.tr_select(None, None, None, 1, N, None, None, None, None) == _lib.TR_EINVAL
    assert lib.tr_score(None, None, None, None, 1, None, None, None, None) == _lib.TR_EINVAL
    assert lib.tr_nonfinite_rows(None, None, 0, None) == _lib.TR_EINVAL
    lib.tr_destroy(None)


def test_every_variant_flag_is_accepted_and_others_are_not():
    """TR_FLAG_STRIDE_REAL, TR_FLAG_SHANNON and TR_FLAG_CHECK_FINITE (and
    their combinations) pass the host checks; any other bit is TR_EINVAL."""
    lib = _lib.load()
    N = (ctypes.c_int32 * 1)(100)
    K = (ctypes.c_int32 * 1)(10)
    g = 1 << 20
    known = _lib.TR_FLAG_STRIDE_REAL | _lib.TR_FLAG_SHANNON | _lib.TR_FLAG_CHECK_FINITE
    for flags in range(16):
        p = _lib.Params(D=64, Dc=0, dtype=_lib.TR_BF16, max_images=0, max_tokens=0, max_N=0, flags=flags,
                        lam=1.0 / 3.0, keep_ratio=0.0)
        want = _lib.TR_OK if flags & ~known == 0 else _lib.TR_EINVAL
        assert lib.tr_check_reduce(ctypes.byref(p), g, g, g, 1, N, K, g, g, None, None, None) == want, flags
        assert lib.tr_plan(ctypes.byref(p), 1, N, K, None, None, None, None) == want, flags


def test_gemm_and_fused_entry_points_validate_before_touching_a_device():
    """Argument errors of the GEMM entry points come back synchronously (no context needed)."""
    lib = _lib.load()
    assert lib.tr_gemm_bf16(None, None, 64, None, 0, None, 64, None, 128, 1, 128, 64, None) == _lib.TR_EINVAL
    assert lib.tr_mlp_out_cos(None, None, 64, None, 64, None, None, 1, 64, None, None) == _lib.TR_EINVAL
    N = (ctypes.c_int32 * 1)(4)
    assert lib.tr_reduce_given_s(None, None, None, 1, N, None, None, None, None, None, None) == _lib.TR_EINVAL
    assert lib.tr_reduce_project(None, None, None, None, 1, N, None, None, 64, 128, None, None, None, None) == _lib.TR_EINVAL
    assert lib.tr_last_error() != b""


def _read_args(ptrs, sizes):
    n = len(ptrs)
    p = (ctypes.c_void_p * max(n, 1))(*ptrs)
    b = (ctypes.c_int64 * max(n, 1))(*sizes)
    return ctypes.cast(p, ctypes.c_void_p), ctypes.cast(b, ctypes.c_void_p), n


def test_read_bandwidth_validates_before_touching_a_device():
    """The read hook rejects sets, sizes and pointers it cannot stream, and
    reads nothing for 0 bytes, all without a device call."""
    lib = _lib.load()
    sink = ctypes.c_void_p(64)   # never dereferenced: every call below returns first
    ok = lambda ptrs, sizes, sk=sink, words=1: lib.tr_read_bandwidth(*_read_args(ptrs, sizes), sk, words, None)
    assert ok([None], [0], None, 0) == _lib.TR_OK                       # nothing to read
    assert ok([None, None], [0, 0], None, 0) == _lib.TR_OK
    assert lib.tr_read_bandwidth(None, None, 1, sink, 1, None) == _lib.TR_EINVAL   # no arrays
    assert ok([], []) == _lib.TR_EINVAL                                  # n = 0
    assert ok([256] * 9, [16] * 9) == _lib.TR_EINVAL                     # more than 8 buffers
    assert ok([256], [-16]) == _lib.TR_EINVAL
    assert ok([256], [24]) == _lib.TR_EINVAL                             # not a multiple of 16
    assert ok([None], [16]) == _lib.TR_EINVAL
    assert ok([256, 264], [16, 16]) == _lib.TR_EINVAL                    # misaligned second buffer
    assert ok([256], [16], sink, 0) == _lib.TR_EINVAL                    # no sink words
    assert ok([256], [16], ctypes.c_void_p(66), 1) == _lib.TR_EINVAL     # misaligned sink
    assert b"sink" in lib.tr_last_error()


def test_last_error_is_per_thread():
    """tr_last_error reports the calling thread's latest failure only."""
    import threading
    lib = _lib.load()
    seen = {}

    def failing():
        assert lib.tr_read_bandwidth(None, None, 0, None, 0, None) == _lib.TR_EINVAL
        seen["failing"] = lib.tr_last_error()

    def quiet():
        seen["quiet_before"] = lib.tr_last_error()
        t = threading.Thread(target=failing)
        t.start()
        t.join()
        seen["quiet_after"] = lib.tr_last_error()

    t = threading.Thread(target=quiet)
    t.start()
    t.join()
    assert seen["failing"] != b""
    assert seen["quiet_before"] == b"" and seen["quiet_after"] == b""


# ----------------------------------------------------------- host sanitizers

def _sanitizer_flags():
    return ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
            "-fno-omit-frame-pointer"]


def test_host_planner_under_sanitizers(tmp_path):
    """The host-only planner (tr_plan.cpp: parameter checks, Algorithm 1's
    budget plan, the argument rules of a reduce call, the error buffer) built
    on its own with the address and undefined-behaviour sanitizers and driven
    over valid and invalid calls, batches above and below its inline storage."""
    exe = tmp_path / "plan_driver"
    src = [os.path.join(ROOT, "tests", "sanitize", "plan_driver.cpp"),
           os.path.join(ROOT, "paper_2607_13500_amd", "csrc", "tr_plan.cpp")]
    res = subprocess.run(["g++", "-std=c++17", "-Wall", "-Wextra", "-I", os.path.join(ROOT, "include")]
                         + _sanitizer_flags() + ["-o", str(exe)] + src, capture_output=True, text=True)
    if res.returncode != 0 and "asan" in (res.stderr or "").lower():
        pytest.skip("no sanitizer runtime: " + res.stderr[-200:])
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert run.returncode == 0, run.stdout + run.stderr
    assert "planner ok" in run.stdout


def test_check_reduce_states_the_alignment_rule():
    """tr_check_reduce (host-only, no device) applies tr_reduce's argument
    rules: a base not aligned to its element size is TR_EUNSUPPORTED, an
    element-aligned one is accepted (scalar path), and inputs of a score the
    call does not compute are neither required nor checked."""
    lib = _lib.load()
    N = (ctypes.c_int32 * 2)(100, 50)
    K = (ctypes.c_int32 * 2)(10, 5)
    g = 1 << 20   # addresses are inspected, never dereferenced
    for dtype, e in ((_lib.TR_BF16, 2), (_lib.TR_FP32, 4)):
        p = _lib.Params(D=64, Dc=0, dtype=dtype, max_images=0, max_tokens=0, max_N=0, flags=0,
                        lam=1.0 / 3.0, keep_ratio=0.0)

        def chk(X=g, P=g, Q=g, out=g, idx=g, h2=None, s=None):
            return lib.tr_check_reduce(ctypes.byref(p), X, P, Q, 2, N, K, out, idx, None, h2, s)

        assert chk() == _lib.TR_OK
        assert chk(X=g + e, P=g + 3 * e, out=g + e) == _lib.TR_OK
        for bad in (dict(X=g + 1), dict(P=g + 1), dict(Q=g + 1), dict(out=g + 1), dict(idx=g + 2),
                    dict(h2=g + 2), dict(s=g + 2)):
            assert chk(**bad) == _lib.TR_EUNSUPPORTED, bad
            assert b"aligned" in lib.tr_last_error()
        if dtype == _lib.TR_FP32:
            assert chk(X=g + 2) == _lib.TR_EUNSUPPORTED
        for missing in (dict(X=None), dict(P=None), dict(Q=None), dict(out=None), dict(idx=None)):
            assert chk(**missing) == _lib.TR_EINVAL, missing
        p.lam = 1.0
        assert chk(P=None, Q=None) == _lib.TR_OK
        assert chk(P=g + 1, Q=g + 1) == _lib.TR_OK
        assert chk(P=None, Q=None, s=g) == _lib.TR_EINVAL       # asking for s needs the states


def _run_with_env(env_extra, code):
    env = dict(os.environ)
    env.update(env_extra)
    return subprocess.run(["python3", "-c", code], capture_output=True, text=True, env=env, cwd=ROOT, timeout=300)


_BAD_PLAN = """
import ctypes
from paper_2607_13500_amd import _lib
lib = _lib.load()
p = _lib.Params(D=0, Dc=0, dtype=1, max_images=0, max_tokens=0, max_N=0, flags=0, lam=0.5, keep_ratio=0.0)
N = (ctypes.c_int32 * 1)(4)
print(lib.tr_plan(ctypes.byref(p), 1, N, None, None, None, None, None))
print(lib.tr_read_bandwidth(None, None, 0, None, 0, None))
"""


def test_log_is_opt_in():
    """The library prints nothing unless TR_LOG=1; then each failure is one
    stderr line naming the status and the reason."""
    quiet = _run_with_env({"TR_LOG": "0"}, _BAD_PLAN)
    assert quiet.returncode == 0, quiet.stderr
    assert quiet.stdout.split() == [str(_lib.TR_EINVAL)] * 2
    assert "tr:" not in quiet.stderr
    loud = _run_with_env({"TR_LOG": "1"}, _BAD_PLAN)
    assert loud.returncode == 0, loud.stderr
    lines = [l for l in loud.stderr.splitlines() if l.startswith("tr: ")]
    assert len(lines) == 2, loud.stderr
    assert lines[0].startswith("tr: invalid argument: ") and "D" in lines[0]
    assert "n must be in [1, 8]" in lines[1]


def test_roctx_ranges_are_opt_in_and_harmless():
    """TR_ROCTX=1 opens the roctx library at the first entry point that
    enqueues work and brackets each such call in a range (here calls that
    fail their argument checks, so no device is needed); the process runs
    and ends normally with the ranges balanced.  Without it no range is
    made."""
    on = _run_with_env({"TR_ROCTX": "1", "TR_LOG": "1"}, _BAD_PLAN)
    assert on.returncode == 0, on.stderr
    assert on.stdout.split() == [str(_lib.TR_EINVAL)] * 2
    assert "tr: roctx ranges on" in on.stderr, on.stderr
    off = _run_with_env({"TR_ROCTX": "0", "TR_LOG": "1"}, _BAD_PLAN)
    assert off.returncode == 0, off.stderr
    assert "roctx" not in off.stderr, off.stderr
