"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value is a closed
form, an invariant, a value the paper prints (tests/golden/), a library routine
(numpy lexsort) or the exact brute force of tests/brute.py.
"""
import math
import os

import numpy as np
import pytest
import torch

import brute
import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
RNG = np.random.default_rng(20260712)


def bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (round to nearest even, via torch)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_to_f32(u: np.ndarray) -> np.ndarray:
    return (u.astype(np.uint32) << 16).view(np.float32)


def both_dtypes(row: np.ndarray):
    """The same row as float32 and, if exactly representable, as bfloat16."""
    f = np.ascontiguousarray(row, dtype=np.float32)
    out = [f]
    b = bf16(f)
    if np.array_equal(bf16_to_f32(b), f):
        out.append(b)
    return out


# ---------------------------------------------------------------- Eq. (3)-(4)

@pytest.mark.parametrize("D", [1, 2, 3, 7, 64, 1000, 1024, 3584, 4096])
def test_h2_uniform_magnitude_is_log_D(D):
    signs = RNG.choice([-1.0, 1.0], size=D)
    for c in (1.0, 0.5, 3.0, 1e-20, 1e20):
        for row in both_dtypes(c * signs):
            assert oracle.renyi2(row) == pytest.approx(math.log(D), rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("D", [1, 5, 1024, 4096])
def test_h2_one_hot_is_zero(D):
    for pos in {0, D // 2, D - 1}:
        row = np.zeros(D, np.float32)
        row[pos] = -2.5
        for r in both_dtypes(row):
            assert abs(oracle.renyi2(r)) < 1e-15


@pytest.mark.parametrize("D,k", [(8, 3), (64, 17), (4096, 1000), (4096, 4096)])
def test_h2_k_equal_nonzeros_is_log_k(D, k):
    row = np.zeros(D, np.float32)
    pos = RNG.choice(D, size=k, replace=False)
    row[pos] = 0.75 * RNG.choice([-1.0, 1.0], size=k)
    for r in both_dtypes(row):
        assert oracle.renyi2(r) == pytest.approx(math.log(k), rel=1e-12)


@pytest.mark.parametrize("na,a,nb,b", [(3, 1.0, 5, 2.0), (100, 0.25, 1, 64.0), (2000, 1.0, 2096, 1.5)])
def test_h2_two_level_closed_form(na, a, nb, b):
    row = np.concatenate([np.full(na, a), -np.full(nb, b)]).astype(np.float32)
    RNG.shuffle(row)
    want = math.log((na * a + nb * b) ** 2 / (na * a * a + nb * b * b))
    for r in both_dtypes(row):
        assert oracle.renyi2(r) == pytest.approx(want, rel=1e-12)


def test_h2_small_rational_examples():
    # [3, 4]: p = (3/7, 4/7), sum p^2 = 25/49.   [1, -2, 2]: p = (1,2,2)/5, sum = 9/25.
    assert oracle.renyi2(np.array([3, 4], np.float32)) == pytest.approx(math.log(49 / 25), rel=1e-14)
    assert oracle.renyi2(np.array([1, -2, 2], np.float32)) == pytest.approx(math.log(25 / 9), rel=1e-14)


def test_h2_all_zero_row_reading():
    # Eq. (3) is 0/0 here; the reading used throughout is H2 = 0.
    for D in (1, 16, 4096):
        assert oracle.renyi2(np.zeros(D, np.float32)) == 0.0


def test_h2_invariances_and_bounds():
    for D in (5, 300, 4096):
        x = RNG.standard_normal(D).astype(np.float32) * RNG.lognormal(0, 1, D).astype(np.float32)
        h = oracle.renyi2(x)
        assert 0.0 <= h <= math.log(D) + 1e-12
        assert oracle.renyi2(np.float32(-4.0) * x) == pytest.approx(h, rel=1e-12)   # scale (exact in fp32)
        assert oracle.renyi2(np.float32(0.125) * x) == pytest.approx(h, rel=1e-12)
        flip = x * RNG.choice([-1, 1], size=D).astype(np.float32)                  # signs
        assert oracle.renyi2(flip) == pytest.approx(h, rel=1e-12)
        assert oracle.renyi2(RNG.permutation(x)) == pytest.approx(h, rel=1e-12)   # channels


def test_h2_two_forms_agree():
    for D in (3, 1024, 4096):
        for kind in range(4):
            if kind == 0:
                x = RNG.standard_normal(D)
            elif kind == 1:   # near-constant magnitude, H2 close to log D
                x = 1.7 * (1 + 1e-3 * RNG.standard_normal(D))
            elif kind == 2:   # heavy tail
                x = RNG.standard_t(3, D)
            else:             # sparse spikes
                x = np.where(RNG.random(D) < 0.01, 50.0, 1e-3) * RNG.standard_normal(D)
            for r in both_dtypes(x.astype(np.float32)):
                a, b = oracle.renyi2(r), oracle.renyi2_cv(r)
                assert abs(a - b) <= 1e-12 * max(1.0, abs(a))


def test_h2_gaussian_row_statistics():
    # i.i.d. N(0,1) channels: E[H2] ~ log D + log(2/pi) and, by the delta method,
    # sd(H2) ~ sqrt(2*pi - 6) / sqrt(D) = 0.532 / sqrt(D).
    D, n = 4096, 600
    rng = np.random.default_rng(7)
    h = np.array([oracle.renyi2(rng.standard_normal(D).astype(np.float32)) for _ in range(n)])
    sd_pred = math.sqrt(2 * math.pi - 6) / math.sqrt(D)
    assert abs(h.mean() - (math.log(D) + math.log(2 / math.pi))) < 4 * sd_pred / math.sqrt(n) + 2e-4
    assert 0.85 < h.std() / sd_pred < 1.15


# ------------------------------------------- Shannon variant of the score

@pytest.mark.parametrize("D", [1, 2, 7, 1024, 4096])
def test_h1_closed_forms(D):
    signs = RNG.choice([-1.0, 1.0], size=D)
    for c in (1.0, 3.0, 1e-20):
        for row in both_dtypes(c * signs):                     # uniform magnitude: log D
            assert oracle.shannon(row) == pytest.approx(math.log(D), rel=1e-12, abs=1e-15)
    row = np.zeros(D, np.float32)
    row[D // 2] = -2.5
    assert oracle.shannon(row) == 0.0                          # one-hot: 0
    k = max(1, D // 3)
    row = np.zeros(D, np.float32)
    row[RNG.choice(D, size=k, replace=False)] = 0.75           # k equal non-zeros: log k
    assert oracle.shannon(row) == pytest.approx(math.log(k), rel=1e-12, abs=1e-15)
    assert oracle.shannon(np.zeros(D, np.float32)) == 0.0      # all-zero row: the H2 reading


def test_h1_against_scipy_entropy():
    import scipy.stats
    for D in (2, 3, 64, 1000, 4096):
        for kind in range(4):
            if kind == 0:
                x = RNG.standard_normal(D)
            elif kind == 1:
                x = 1.7 * (1 + 1e-3 * RNG.standard_normal(D))
            elif kind == 2:
                x = RNG.standard_t(3, D)
            else:
                x = np.where(RNG.random(D) < 0.05, 50.0, 0.0) * RNG.standard_normal(D)
                x[0] = 1.0
            for r in both_dtypes(x.astype(np.float32)):
                a = np.abs(oracle.as_raw(r)[0].astype(np.float64)) if r.dtype == np.float32 \
                    else np.abs(bf16_to_f32(r).astype(np.float64))
                want = scipy.stats.entropy(a)               # normalises, natural log, 0 log 0 = 0
                assert oracle.shannon(r) == pytest.approx(want, rel=1e-12, abs=1e-13)


def test_h1_renyi_order_and_invariances():
    # Renyi entropies do not increase with the order: H2 <= H1 <= log D, with
    # equality only for a uniform magnitude distribution over the support.
    for D in (5, 300, 4096):
        x = (RNG.standard_normal(D) * RNG.lognormal(0, 1, D)).astype(np.float32)
        h1, h2 = oracle.shannon(x), oracle.renyi2(x)
        assert h2 < h1 < math.log(D)
        assert oracle.shannon(np.float32(-4.0) * x) == pytest.approx(h1, rel=1e-12)
        assert oracle.shannon(RNG.permutation(x)) == pytest.approx(h1, rel=1e-12)
        assert oracle.shannon(x * RNG.choice([-1, 1], size=D).astype(np.float32)) == pytest.approx(h1, rel=1e-12)


def test_h1_drives_stage1_in_the_variant():
    # With entropy=1 the oracle's scores are H1 per row and lambda = 1 keeps
    # the K highest-H1 tokens (numpy lexsort on (index, -H1)).
    N, D, K = 300, 64, 40
    X = (RNG.standard_normal((N, D)) * RNG.lognormal(0, 1, (N, 1))).astype(np.float32)
    X[::7] = np.abs(X[::7]).mean()                            # planted exact ties (uniform rows)
    P = RNG.standard_normal((N, D)).astype(np.float32)
    h1, s = oracle.scores(X, P, P, entropy=1)
    assert np.array_equal(h1, np.array([oracle.shannon(r) for r in X]))
    ref = oracle.reduce(X, P, P, [N], [K], 1.0, entropy=1)
    want = np.sort(np.lexsort((np.arange(N), -h1))[:K])
    assert np.array_equal(ref["idx"], want)
    assert np.array_equal(ref["h2"], h1)


# ---------------------------------------------------------------- Eq. (6)

def test_cosine_closed_forms():
    for Dc in (1, 2, 17, 4096):
        x = RNG.standard_normal(Dc).astype(np.float32)
        assert oracle.cosine(x, x) == pytest.approx(1.0, abs=1e-14)
        assert oracle.cosine(x, -x) == pytest.approx(-1.0, abs=1e-14)
        assert oracle.cosine(x, np.float32(2.5) * x) == pytest.approx(1.0, abs=1e-14)
        assert oracle.cosine(x, np.float32(-0.25) * x) == pytest.approx(-1.0, abs=1e-14)
        y = RNG.standard_normal(Dc).astype(np.float32)
        c = oracle.cosine(x, y)
        assert -1.0 <= c <= 1.0
        assert oracle.cosine(y, x) == c                                        # symmetry
        assert oracle.cosine(np.float32(4) * x, np.float32(0.5) * y) == pytest.approx(c, rel=1e-12)
    # known angles
    assert oracle.cosine(np.array([1, 0], np.float32), np.array([1, 1], np.float32)) == pytest.approx(1 / math.sqrt(2), rel=1e-15)
    assert oracle.cosine(np.array([3, 4], np.float32), np.array([4, 3], np.float32)) == pytest.approx(24 / 25, rel=1e-15)
    assert oracle.cosine(np.array([1, 1, 0, 0], np.float32), np.array([1, -1, 5, 0], np.float32)) == 0.0
    assert oracle.cosine(np.array([2, 0, 0], np.float32), np.array([0, 0, -7], np.float32)) == 0.0
    # zero norm reading
    z = np.zeros(8, np.float32)
    assert oracle.cosine(z, RNG.standard_normal(8).astype(np.float32)) == 0.0
    assert oracle.cosine(RNG.standard_normal(8).astype(np.float32), z) == 0.0


def test_cosine_f64_rows():
    # the same closed forms on float64 rows (the exact product of two bf16
    # matrices is compared against in float64)
    for Dc in (1, 3, 1024):
        x = RNG.standard_normal(Dc)
        assert oracle.cosine(x, x) == pytest.approx(1.0, abs=1e-14)
        assert oracle.cosine(x, -3.0 * x) == pytest.approx(-1.0, abs=1e-14)
        y = RNG.standard_normal(Dc)
        assert oracle.cosine(x, y) == pytest.approx(float(x @ y / math.sqrt((x @ x) * (y @ y))), rel=1e-12, abs=1e-15)
    assert oracle.cosine(np.array([3.0, 4.0]), np.array([4.0, 3.0])) == pytest.approx(24 / 25, rel=1e-15)
    assert oracle.cosine(np.zeros(4), np.ones(4)) == 0.0
    # float32 rows widened to float64 give the same value
    x32 = RNG.standard_normal(64).astype(np.float32)
    y32 = RNG.standard_normal(64).astype(np.float32)
    assert oracle.cosine(x32.astype(np.float64), y32.astype(np.float64)) == oracle.cosine(x32, y32)


def test_matmul_bt_small_integer_brute_force():
    rng = np.random.default_rng(5)
    for M, N, K in ((1, 1, 1), (3, 5, 7), (17, 4, 33)):
        A = rng.integers(-4, 5, (M, K)).astype(np.float32)
        B = rng.integers(-4, 5, (N, K)).astype(np.float32)
        want = [[sum(float(A[m, k]) * float(B[n, k]) for k in range(K)) for n in range(N)] for m in range(M)]
        assert np.array_equal(oracle.matmul_bt(A, B), np.array(want))
        assert np.array_equal(oracle.matmul_bt(bf16(A), bf16(B)), np.array(want))   # exact in bf16 too


def test_scores_batch_matches_single_rows():
    X = RNG.standard_normal((9, 33)).astype(np.float32)
    P = RNG.standard_normal((9, 20)).astype(np.float32)
    Q = RNG.standard_normal((9, 20)).astype(np.float32)
    h2, s = oracle.scores(bf16(X), bf16(P), bf16(Q))
    for i in range(9):
        assert h2[i] == oracle.renyi2(bf16(X[i]))
        assert s[i] == oracle.cosine(bf16(P[i]), bf16(Q[i]))


# ---------------------------------------------------------------- Algorithm 1

def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_budget_golden_table():
    rows = _golden("budget_split.txt")
    assert any(r[-1] == "paper" for r in rows)
    for N, K, ln, ld, K1, K2, t, _ in rows:
        lam = int(ln) / int(ld)
        assert oracle.budget(int(N), int(K), lam) == (int(K1), int(K2), int(t))


def test_budget_rejects_invalid():
    for args in [(0, 1, 0.5), (5, 0, 0.5), (5, 6, 0.5), (5, 3, -0.1), (5, 3, 1.5), (5, 3, float("nan"))]:
        with pytest.raises(ValueError):
            oracle.budget(*args)


def test_lambda_one_is_textbook_topk():
    # lambda = 1: Algorithm 1 reduces to the K highest-entropy tokens, ties to
    # the lower index, i.e. numpy lexsort on (index, -H2).
    for trial in range(200):
        N = int(RNG.integers(1, 400))
        K = int(RNG.integers(1, N + 1))
        h2 = RNG.choice(RNG.random(max(1, N // 3)), size=N)   # planted exact ties
        s = RNG.random(N)
        idx, src = oracle.select(h2, s, K, 1.0)
        want = np.sort(np.lexsort((np.arange(N), -h2))[:K])
        assert np.array_equal(idx, want)
        assert not src.any()


def test_lambda_zero_is_sorted_stride():
    # lambda = 0: no Stage I; the picks are positions 0, t, 2t, ... of the
    # stable ascending order of s (numpy lexsort on (index, s)).
    for trial in range(200):
        N = int(RNG.integers(1, 400))
        K = int(RNG.integers(1, N + 1))
        s = RNG.choice(RNG.standard_normal(max(1, N // 2)), size=N)
        h2 = RNG.random(N)
        t = max(1, N // K)
        idx, src = oracle.select(h2, s, K, 0.0)
        want = np.sort(np.lexsort((np.arange(N), s))[::t][:K])
        assert np.array_equal(idx, want)
        assert src.all()


def test_select_invariants():
    for trial in range(300):
        N = int(RNG.integers(1, 300))
        K = int(RNG.integers(1, N + 1))
        lam = float(RNG.choice([0.0, 0.25, 1 / 3, 0.5, 0.9, 1.0]))
        h2 = RNG.choice(RNG.random(max(1, N // 2)), size=N)
        s = RNG.choice(RNG.standard_normal(max(1, N // 2)), size=N)
        K1, K2, t = oracle.budget(N, K, lam)
        idx, src = oracle.select(h2, s, K, lam)
        assert idx.size == K and np.all(np.diff(idx) > 0)
        assert 0 <= idx.min() and idx.max() < N
        imp = idx[src == 0]
        div = idx[src == 1]
        assert imp.size == K1 and div.size == K2
        rest = np.setdiff1d(np.arange(N), imp)
        if imp.size and rest.size:
            # every X^imp token precedes every remaining token in (H2 desc, index asc)
            worst = max(imp, key=lambda i: (-h2[i], i))
            best = min(rest, key=lambda i: (-h2[i], i))
            assert (-h2[worst], worst) < (-h2[best], best)
        if K2:
            order = rest[np.lexsort((rest, s[rest]))]
            pos = np.sort(np.nonzero(np.isin(order, div))[0])
            assert np.array_equal(pos, np.arange(K2) * t)


def _small_int_case(N, D, Dc):
    vals = np.array([-2, -1, 0, 1, 2], np.float32)
    X = RNG.choice(vals, size=(N, D))
    P = RNG.choice(vals, size=(N, Dc))
    Q = RNG.choice(vals, size=(N, Dc))
    return X, P, Q


def test_bruteforce_small_integer_inputs_with_exact_ties():
    # Entries in {-2..2} force many exact ties in both stages; two-channel rows
    # keep every tie exact in double too (a two-term sum is order-free).
    cases = 0
    for trial in range(1500):
        N = int(RNG.integers(1, 7))
        K = int(RNG.integers(1, N + 1))
        lam = float(RNG.choice([0.0, 1 / 3, 0.5, 2 / 3, 1.0]))
        D = int(RNG.integers(1, 3))
        X, P, Q = _small_int_case(N, D, D)
        want = brute.reduce_rows(X, P, Q, K, lam)
        got = oracle.reduce(X, P, Q, [N], [K], lam)
        assert list(got["idx"]) == want[0], (X, P, Q, K, lam)
        assert list(got["src"]) == want[1]
        for dt in (bf16,):
            got2 = oracle.reduce(dt(X), dt(P), dt(Q), [N], [K], lam)
            assert list(got2["idx"]) == want[0]
        cases += 1
    assert cases == 1500


def test_bruteforce_continuous_inputs():
    for trial in range(400):
        N = int(RNG.integers(1, 11))
        K = int(RNG.integers(1, N + 1))
        lam = float(RNG.choice([0.0, 1 / 3, 0.5, 1.0]))
        D = int(RNG.integers(1, 9))
        Dc = int(RNG.integers(1, 9))
        X = (RNG.standard_normal((N, D)) * RNG.lognormal(0, 1, (N, 1))).astype(np.float32)
        P = RNG.standard_normal((N, Dc)).astype(np.float32)
        Q = (P + 0.7 * RNG.standard_normal((N, Dc))).astype(np.float32)
        want = brute.reduce_rows(X, P, Q, K, lam)
        got = oracle.reduce(X, P, Q, [N], [K], lam)
        assert list(got["idx"]) == want[0]
        assert list(got["src"]) == want[1]


def test_bruteforce_real_interval_stride_variant():
    for trial in range(300):
        N = int(RNG.integers(1, 11))
        K = int(RNG.integers(1, N + 1))
        lam = float(RNG.choice([0.0, 1 / 3, 0.5]))
        X, P, Q = _small_int_case(N, 2, 2)
        want = brute.reduce_rows(X, P, Q, K, lam, stride_mode=1)
        got = oracle.reduce(X, P, Q, [N], [K], lam, stride_mode=1)
        assert list(got["idx"]) == want[0]


def test_conditional_mode():
    for trial in range(300):
        N = int(RNG.integers(1, 9))
        K = int(RNG.integers(1, N + 1))
        lam = float(RNG.choice([0.0, 1 / 3, 0.5, 1.0]))
        X, P, Q = _small_int_case(N, 2, 2)
        K1 = math.floor(lam * K)
        # its own X^imp reproduces the unconditional result
        base = oracle.reduce(X, P, Q, [N], [K], lam)
        own = np.zeros(N, bool)
        own[base["idx"][base["src"] == 0]] = True
        again = oracle.reduce(X, P, Q, [N], [K], lam, given_imp=own)
        assert np.array_equal(again["idx"], base["idx"])
        # an arbitrary X^imp of the right size matches the brute force given it
        gi = np.zeros(N, bool)
        gi[RNG.choice(N, size=K1, replace=False)] = True
        want = brute.reduce_rows(X, P, Q, K, lam, given_imp=gi)
        got = oracle.reduce(X, P, Q, [N], [K], lam, given_imp=gi)
        assert list(got["idx"]) == want[0] and list(got["src"]) == want[1]


def test_batch_gather_bytes_and_offsets():
    N = [5, 1, 12, 7]
    K = [2, 1, 12, 3]
    D, Dc = 6, 4
    X = bf16(RNG.standard_normal((sum(N), D)))
    P = bf16(RNG.standard_normal((sum(N), Dc)))
    Q = bf16(RNG.standard_normal((sum(N), Dc)))
    res = oracle.reduce(X, P, Q, N, K, 1 / 3)
    r0 = o0 = 0
    for n, k in zip(N, K):
        idx, src = oracle.select(res["h2"][r0:r0 + n], res["s"][r0:r0 + n], k, 1 / 3)
        assert np.array_equal(res["idx"][o0:o0 + k], idx)
        assert np.array_equal(res["src"][o0:o0 + k], src)
        assert np.array_equal(res["out"][o0:o0 + k], X[r0 + idx])      # byte copy
        r0 += n
        o0 += k


def test_select_rejects_invalid():
    with pytest.raises(ValueError):
        oracle.select(np.zeros(4), np.zeros(4), 5, 0.5)
    with pytest.raises(ValueError):   # conditional X^imp of the wrong size
        oracle.select(np.zeros(4), np.zeros(4), 2, 0.5, given_imp=np.array([1, 1, 0, 0]))


# ----------------------------------------------------------- host sanitizers

def _asan_runtime():
    import subprocess
    path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _sanitized_oracle(tmp_path, source=None):
    import subprocess
    src = source or os.path.join(os.path.dirname(oracle.__file__), "altr_oracle.c")
    lib = str(tmp_path / "liboracle_sanitized.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c99", "-fPIC", "-shared", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", lib, src, "-lm"])
    return lib


def _pins_under_sanitizers(lib, select):
    import subprocess
    import sys
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(), ALTR_ORACLE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # -s: a sanitizer report goes to the real stderr, not pytest's capture
    return subprocess.run([sys.executable, "-u", "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider", "-k",
                           select, os.path.abspath(__file__)], capture_output=True, text=True, timeout=600, env=env,
                          cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def test_pins_hold_under_sanitizers(tmp_path):
    """Every pin above, run against the oracle built with the address and
    undefined-behaviour sanitizers (inputs come from numpy, whose buffers the
    preloaded runtime guards): no out-of-bounds access, no undefined
    arithmetic, same results."""
    if _asan_runtime() is None:
        pytest.skip("no address-sanitizer runtime")
    res = _pins_under_sanitizers(_sanitized_oracle(tmp_path), "not sanitizer")
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-2000:]
    assert " passed" in res.stdout


def test_sanitizer_build_catches_an_out_of_bounds_read(tmp_path):
    """The sanitized run is not vacuous: a copy of the oracle whose entropy
    loop reads one element past the row is stopped by it."""
    if _asan_runtime() is None:
        pytest.skip("no address-sanitizer runtime")
    text = open(os.path.join(os.path.dirname(oracle.__file__), "altr_oracle.c")).read()
    start = text.index("double altr_oracle_renyi2(")
    body = text[start:]
    loop = body.index("j < D")
    mutated = text[:start] + body[:loop] + "j <= D" + body[loop + len("j < D"):]
    src = tmp_path / "altr_oracle_oob.c"
    src.write_text(mutated)
    res = _pins_under_sanitizers(_sanitized_oracle(tmp_path, str(src)), "h2_uniform")
    assert res.returncode != 0
    assert "AddressSanitizer" in res.stdout + res.stderr

