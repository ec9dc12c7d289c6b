"""GPU parity of the HIP path against the fp64 oracle (through the C ABI).

Every case prints its name, seed and shape before touching the GPU.  Small
cases span several 64-token tiles and ragged tails; the `full` cases run the
benchmark workloads at their real sizes in the launch configuration bench.py
times, and check every image with the protocol of tests/parity.py.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def reducer_for(w, **kw):
    import paper_2607_13500_amd as tr
    return tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, keep_ratio=w.keep_ratio,
                      max_images=max(1, w.B), max_tokens=max(1, sum(w.N)),
                      max_N=max(w.N) if w.N else 1, **kw)


def run_and_check(w, *, use_keep_ratio=False, tol=parity.TOL):
    r = reducer_for(w)
    K = None if use_keep_ratio else w.K
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, K, want_scores=True)
    cv2, s2, h2b = r.score(w.X, w.Xpre, w.Xpost, want_h2=True)
    torch.cuda.synchronize()
    # the stand-alone scoring entry point is the same kernel, bit for bit
    assert torch.equal(s2, res.s) and torch.equal(h2b, res.h2)
    ref = parity.oracle_reference(w)
    rep = parity.check(w, res, ref, cv2_gpu=cv2, tol=tol)
    print("   ", w.name, rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    r.close()
    return rep, res


SMALL = [
    ("llava_fp32", dict()),                                          # B=1, 576 x 1024 fp32
    ("llava", dict(B=6, N=576, D=4096)),
    ("llava", dict(B=3, N=577, D=520, K=100)),                        # ragged tail tile, D % 64 != 0
    ("llava_next", dict(B=2, D=4096, K=320)),
    ("qwen_ragged", dict(B=5, n_lo=256, n_hi=3000, D=3584)),
    ("video", dict(B=1, frames=6, positions=576, D=4096, K=216)),
    ("llava", dict(B=2, N=300, D=4096, K=40, dtype=torch.float32)),   # 16 KiB rows: one per wavefront
    ("llava", dict(B=2, N=200, D=8192, K=30, dtype=torch.float32)),   # 32 KiB rows
    ("llava", dict(B=2, N=200, D=12288, K=30)),                       # 24 KiB bf16 rows, six loop passes
]


@pytest.mark.parametrize("name,kw", SMALL, ids=[f"{n}-{i}" for i, (n, _) in enumerate(SMALL)])
def test_reduce_parity_small(name, kw):
    say("small", name, kw)
    w = synth.make(name, device=DEV, **kw)
    rep, _ = run_and_check(w, use_keep_ratio=(name == "qwen_ragged"))
    assert rep.stage1_swaps <= max(1, rep.images // 10)


def test_reduce_deterministic_and_duplicates_tie_exactly():
    say("determinism llava B=4")
    w = synth.llava(device=DEV, B=4, N=576, D=4096)
    r = reducer_for(w)
    a = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    outs = [r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True) for _ in range(2)]
    torch.cuda.synchronize()
    for o in outs:
        for u, v in zip(a, o):
            assert torch.equal(u, v)
    # exact duplicate rows (5 % of tokens) have bit-identical scores
    Xi = w.X.view(torch.int16)
    uniq, inv = torch.unique(Xi, dim=0, return_inverse=True)
    assert uniq.shape[0] < Xi.shape[0]
    for g in range(uniq.shape[0]):
        members = torch.nonzero(inv == g).flatten()
        if members.numel() > 1:
            assert torch.unique(a.h2[members]).numel() == 1
            assert torch.unique(a.s[members]).numel() == 1
    r.close()


def _edge_workload(D, Dc, dtype, rows_kind, n, seed=5):
    g = torch.Generator(device="cpu").manual_seed(seed)
    X = torch.randn(n, D, generator=g)
    P = torch.randn(n, Dc, generator=g)
    Q = P + 0.5 * torch.randn(n, Dc, generator=g)
    k = 0
    for kind in rows_kind:
        if kind == "zero":
            X[k] = 0
        elif kind == "onehot":
            X[k] = 0
            X[k, (7 * k) % D] = -3.0
        elif kind == "uniform":
            X[k] = 0.75 * torch.where(torch.rand(D, generator=g) < 0.5, -1.0, 1.0)
        elif kind == "near_uniform":
            X[k] = 1.3 * (1 + 1e-3 * torch.randn(D, generator=g))
        elif kind == "zero_pre":
            P[k] = 0
        elif kind == "zero_post":
            Q[k] = 0
        elif kind == "antiparallel":
            Q[k] = -2 * P[k]
        elif kind == "dup":
            X[k], P[k], Q[k] = X[0], P[0], Q[0]
        k += 1
    cast = lambda t: t.to(dtype).to(DEV).contiguous()
    return synth.Workload("edge", cast(X), cast(P), cast(Q), [n], [min(n, 40)], synth.LAMBDA)


EDGE_KINDS = ["zero", "onehot", "uniform", "near_uniform", "zero_pre", "zero_post", "antiparallel",
              "dup", "zero", "onehot", "uniform", "near_uniform", "dup"]


@pytest.mark.parametrize("D,Dc,dtype", [(4096, 4096, torch.bfloat16), (1024, 1024, torch.float32),
                                        (37, 45, torch.bfloat16), (5, 3, torch.float32),
                                        (1, 1, torch.bfloat16), (3584, 1024, torch.bfloat16)])
def test_degenerate_rows(D, Dc, dtype):
    say("degenerate rows", D, Dc, dtype)
    w = _edge_workload(D, Dc, dtype, EDGE_KINDS, 150)
    rep, res = run_and_check(w)
    h2 = res.h2.cpu().numpy()
    s = res.s.cpu().numpy()
    if D > 1:
        assert h2[0] == 0.0 and h2[8] == 0.0                       # all-zero rows
        assert abs(h2[1]) < 1e-6                                    # one-hot
        assert abs(h2[2] - math.log(D)) < 1e-5 * math.log(D)        # uniform magnitude
    assert s[4] == 0.0 and s[5] == 0.0                              # zero-norm states
    assert abs(s[6] + 1.0) < 1e-6                                   # cos(x, -2x) = -1


# Magnitudes where fp32 squares of the raw values underflow or overflow.
SCALES = [1e-30, 1e-20, 1e-19, 1e18, 1e30]


def _magnitude_workload(D, Dc, dtype, n=240, seed=9):
    """Rows far from O(1): X near-uniform and Gaussian at every scale of SCALES
    and at 1e37 (the probe's sum overflows fp32) and 1e-40 (denormal values);
    rows mixing magnitudes (a block of 1e25 after O(1) values, a zero probe
    before 1e-30 values, values spread log-uniformly over 1e-30..1e30); and
    x', x'' Gaussian or nearly parallel with every pair of scales, scaled
    independently, plus norms so small that their squares underflow."""
    g = torch.Generator().manual_seed(seed)
    f64 = dict(dtype=torch.float64)
    X = torch.randn(n, D, generator=g, **f64)
    P = torch.randn(n, Dc, generator=g, **f64)
    # per-row noise levels spread s over (0.3, 1): distinct s values, so that
    # the selection's near ties stay rare
    sigma = 0.2 + 2.8 * torch.rand(n, 1, generator=g, **f64)
    Q = P + sigma * torch.randn(n, Dc, generator=g, **f64)
    eps = 10.0 ** (-2.5 + 2 * torch.rand(n, generator=g, **f64))
    xs = []
    for sc in SCALES + [1e37, 1e-40]:
        xs.append(("gauss", sc))
        xs.append(("near_uniform", sc))
    xs += [("spike", 1.0), ("zero_probe", 1e-30), ("log_uniform", 1.0)]
    cs = []
    for sp in SCALES:
        for sq in SCALES:
            cs.append(("indep", sp, sq))
            cs.append(("parallel", sp, sq))
    cs += [("indep", 1e-35, 1e-35), ("indep", 1e-40, 1.0), ("parallel", 1e-38, 1e30), ("indep", 1e36, 1e36)]
    for r in range(n):
        kind, sc = xs[r % len(xs)]
        if kind == "gauss":
            X[r] *= sc
        elif kind == "near_uniform":   # (1e-2: still distinct rows in bf16 at D = 37)
            X[r] = sc * 1.3 * (1 + 1e-2 * torch.randn(D, generator=g, **f64))
        elif kind == "spike":
            X[r, D // 2:] *= 1e25
        elif kind == "zero_probe":
            X[r] *= sc
            X[r, :min(D, 512)] = 0
        elif kind == "log_uniform":
            X[r] = torch.sign(X[r]) * 10.0 ** (60 * torch.rand(D, generator=g, **f64) - 30)
        ck, sp, sq = cs[r % len(cs)]
        if ck == "parallel":   # s from 1 - 5e-6 to about 0.95
            Q[r] = P[r] * (1 + eps[r] * torch.randn(Dc, generator=g, **f64))
        P[r] *= sp
        Q[r] *= sq
    cast = lambda t: t.to(dtype).to(DEV).contiguous()
    return synth.Workload("magnitudes", cast(X), cast(P), cast(Q), [n], [40], synth.LAMBDA)


@pytest.mark.parametrize("entropy", [2, 1])
@pytest.mark.parametrize("D,Dc,dtype", [(4096, 4096, torch.bfloat16), (1024, 1024, torch.float32),
                                        (4096, 3584, torch.float32), (37, 45, torch.bfloat16),
                                        (600, 520, torch.bfloat16)])
def test_extreme_magnitudes_match_the_oracle(D, Dc, dtype, entropy):
    """Finite rows at magnitudes 1e-40..1e37 score like the fp64 oracle, token
    by token (P1), and select like it (P2-P4): both scores are scale-invariant
    and the kernel keeps its fp32 sums in range for any finite row."""
    say("extreme magnitudes", D, Dc, dtype, "entropy", entropy)
    w = _magnitude_workload(D, Dc, dtype)
    r = reducer_for(w, shannon=(entropy == 1))
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    key, s2, h2 = r.score(w.X, w.Xpre, w.Xpost, want_h2=True)
    torch.cuda.synchronize()
    assert torch.equal(s2, res.s) and torch.equal(h2, res.h2)
    assert torch.isfinite(key).all() and torch.isfinite(res.s).all() and torch.isfinite(res.h2).all()
    rep = parity.check(w, res, parity.oracle_reference(w, entropy=entropy), cv2_gpu=key, entropy=entropy)
    print("   ", w.name, "entropy", entropy, rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    r.close()


@pytest.mark.parametrize("shannon", [False, True])
@pytest.mark.parametrize("D,dtype", [(4096, torch.bfloat16), (37, torch.bfloat16), (1000, torch.float32)])
def test_uniform_rows_tie_exactly_at_any_magnitude(D, dtype, shannon):
    """Rows of one repeated magnitude (any signs) have the maximum entropy
    log D exactly (Eq. 3 gives p = 1/D): their Stage I key is exactly 0 at
    every magnitude, normal or not, so they tie and resolve by index."""
    say("uniform rows", D, dtype, "shannon", shannon)
    g = torch.Generator().manual_seed(D)
    mags = [1.3e-40, 1e-30, 3.7e-20, 0.75, 1.1, 5e18, 2e30, 1e37]
    X = torch.stack([m * torch.where(torch.rand(D, generator=g) < 0.5, -1.0, 1.0).double() for m in mags])
    X = X.to(dtype).to(DEV).contiguous()
    assert all(torch.unique(X[i].abs()).numel() == 1 for i in range(len(mags)))
    r = tr_reducer(D, dtype, len(mags), shannon)
    key, _, h = r.score(X, None, None, want_h2=True)
    torch.cuda.synchronize()
    assert torch.all(key == 0), key
    assert torch.all(h == h[0]), h
    r.close()


def tr_reducer(D, dtype, rows, shannon=False):
    import paper_2607_13500_amd as tr
    return tr.Reducer(D, D, dtype, max_images=1, max_tokens=rows, max_N=rows, shannon=shannon)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_scores_are_invariant_to_power_of_two_scaling(dtype):
    """Scaling a row of X, x' or x'' by 2^k (values staying normal) leaves
    every score bit for bit unchanged: X is accumulated relative to the power
    of two of its probe mean, and the cosine's sums scale exactly."""
    D = Dc = 1024
    say("power-of-two invariance", dtype)
    w = _edge_workload(D, Dc, dtype, EDGE_KINDS, 150)
    r = reducer_for(w)
    key0, s0, h0 = r.score(w.X, w.Xpre, w.Xpost, want_h2=True)
    # (the squared norms of x' and x'' stay inside the window where the
    # cosine takes its one-pass form: 2^-60 .. 2^127)
    for kx, kp, kq in ((-60, 10, -20), (40, -25, 25), (-20, -20, -20), (60, 0, 0)):
        key, s, h = r.score((w.X * 2.0 ** kx).contiguous(), (w.Xpre * 2.0 ** kp).contiguous(),
                            (w.Xpost * 2.0 ** kq).contiguous(), want_h2=True)
        torch.cuda.synchronize()
        assert torch.equal(key, key0) and torch.equal(h, h0), (kx, kp, kq)
        assert torch.equal(s, s0), (kx, kp, kq)
    r.close()


def test_misaligned_pointers_give_identical_results():
    say("misaligned bf16 views, D=4096")
    w = synth.llava(device=DEV, B=2, N=300, D=4096, K=64)
    import paper_2607_13500_amd as tr
    r = reducer_for(w)
    a = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    # copies whose base addresses are 2 bytes past a 16-byte boundary
    def shifted(t):
        buf = torch.empty(t.numel() + 8, dtype=t.dtype, device=t.device)
        v = buf[1:1 + t.numel()].view_as(t)
        v.copy_(t)
        return v
    Xs, Ps, Qs = shifted(w.X), shifted(w.Xpre), shifted(w.Xpost)
    outb = torch.empty(sum(w.K) * w.D + 8, dtype=w.dtype, device=DEV)[1:1 + sum(w.K) * w.D].view(sum(w.K), w.D)
    b = r.reduce(Xs, Ps, Qs, w.N, w.K, out=outb, want_scores=True)
    torch.cuda.synchronize()
    assert torch.equal(a.h2, b.h2) and torch.equal(a.s, b.s)
    assert torch.equal(a.idx, b.idx) and torch.equal(a.src, b.src)
    assert torch.equal(a.out.view(torch.int16), b.out.view(torch.int16))
    r.close()


def _select_cases(rng, trials=200):
    cases = []
    for trial in range(trials):
        B = int(rng.integers(1, 7))
        N = [int(rng.choice([1, 2, 63, 64, 65, 200, 576, 1000, 2880, 4097, 9000]))
             for _ in range(B)]
        K = [int(rng.integers(1, n + 1)) for n in N]
        lam = float(rng.choice([0.0, 1 / 3, 0.5, 0.9, 1.0]))
        cases.append((N, K, lam))
    cases.append(([18432], [1152], 1 / 3))
    cases.append(([65] * 40, [13] * 40, 1 / 3))                       # > 32 images, uniform
    cases.append(([65, 70] * 20, [13, 14] * 20, 1 / 3))               # > 32 images, ragged
    # the smallest remainders ranked bucket-by-bucket across split groups
    # (R = N - K1 >= 4096): the per-wavefront staging rows fill the LDS
    # above the remainder list exactly at N = 4096
    cases.append(([4096], [512], 0.0))
    cases.append(([4097, 4099, 4096], [3, 700, 4096], 0.0))
    cases.append(([4098], [6], 1 / 3))
    # a launch whose largest image (4096 tokens) has no packed-remainder
    # region while a smaller one (4095) has it: the launch must reserve the
    # larger layout of the smaller image
    cases.append(([4096, 4095, 2048, 1100], [400, 409, 256, 120], 1 / 3))
    # key shapes that steer the selection's internal paths: all keys equal,
    # one outlier that puts every other key in one bucket, narrow clusters
    shaped = []
    for n in (100, 576, 3000, 4096, 5000):
        for shape in ("const", "outlier", "narrow", "denormal"):
            shaped.append(([n], [max(1, n // 9)], 1 / 3, shape))
    return [c + ("mixed",) for c in cases] + shaped


def _select_keys(rng, shape, total):
    if shape == "mixed":
        # keys drawn from small value sets plant exact ties, and include -0.0/+0.0
        ki = rng.choice(np.array([0.0, -0.0, 1.5, 2.25, -7.0, 3e-8, 1e30], np.float32), size=total)
        ki = np.where(rng.random(total) < 0.5, ki, rng.standard_normal(total).astype(np.float32))
        ks = rng.choice(np.array([-1.0, -0.0, 0.0, 0.5, 0.25, 1.0], np.float32), size=total)
        ks = np.where(rng.random(total) < 0.5, ks, rng.uniform(-1, 1, total).astype(np.float32))
    elif shape == "const":
        ki = np.full(total, 0.75, np.float32)
        ks = np.full(total, -0.125, np.float32)
    elif shape == "outlier":
        ki = (0.57 + 1e-4 * rng.standard_normal(total)).astype(np.float32)
        ki[total // 2] = 4095.0
        ks = (0.3 + 1e-3 * rng.standard_normal(total)).astype(np.float32)
        ks[total // 3] = -1.0
    elif shape == "denormal":
        # subnormal keys (and zeros) of both signs: a key range too narrow for
        # the value buckets' arithmetic, so the integer fallbacks decide
        ki = rng.integers(0, 3000, total).astype(np.uint32).view(np.float32).copy()
        ks = rng.integers(0, 500, total).astype(np.uint32).view(np.float32).copy()
        ks = np.where(rng.random(total) < 0.5, -ks, ks).astype(np.float32)
    else:
        ki = (1.0 + 1e-6 * rng.integers(0, 40, total)).astype(np.float32)
        ks = (0.5 + 1e-7 * rng.integers(0, 300, total)).astype(np.float32)
    return ki, ks


def _at_offset(a, off):
    """a on the device, starting `off` floats past a 256-byte aligned base."""
    buf = torch.zeros(a.size + off + 4, dtype=torch.float32, device=DEV)
    v = buf[off:off + a.size]
    v.copy_(torch.from_numpy(a))
    return v


def _select_against_oracle(cases, rng, stride_real, offsets=(0, 0)):
    import paper_2607_13500_amd as tr
    for ci, (N, K, lam, shape) in enumerate(cases):
        say("select keys case", ci, "B", len(N), "lam", lam, "shape", shape, "stride_real", stride_real,
            "key offsets", offsets)
        total = sum(N)
        ki, ks = _select_keys(rng, shape, total)
        r = tr.Reducer(8, 8, torch.bfloat16, lam=lam, max_images=len(N), max_tokens=total,
                       max_N=max(N), stride_real=stride_real)
        idx, src = r.select(_at_offset(ki, offsets[0]), _at_offset(ks, offsets[1]), N, K)
        idx, src = idx.cpu().numpy(), src.cpu().numpy()
        r0 = o0 = 0
        for n, k in zip(N, K):
            # Stage I key: smaller is more important, so the oracle ranks -key.
            wi, ws = oracle.select(-ki[r0:r0 + n].astype(np.float64), ks[r0:r0 + n].astype(np.float64),
                                   k, lam, stride_mode=1 if stride_real else 0)
            assert np.array_equal(idx[o0:o0 + k], wi), (ci, n, k, lam)
            assert np.array_equal(src[o0:o0 + k], ws), (ci, n, k, lam)
            r0 += n
            o0 += k
        r.close()


def test_select_bit_exact_on_given_keys():
    """Integer work: with the same fp32 keys, the GPU selection equals the oracle's exactly."""
    rng = np.random.default_rng(11)
    _select_against_oracle(_select_cases(rng), rng, stride_real=False)


@pytest.mark.parametrize("offsets", [(1, 3), (2, 0), (3, 1)])
def test_select_bit_exact_on_misaligned_keys(offsets):
    """Key arrays whose bases are 4, 8 or 12 bytes past a 16-byte boundary
    (each kind its own offset): tr_select takes any 4-byte aligned key array
    and still equals the oracle's selection."""
    rng = np.random.default_rng(13 + offsets[0])
    _select_against_oracle(_select_cases(rng, trials=12), rng, stride_real=False, offsets=offsets)


def test_select_bit_exact_stride_real():
    """The real-interval stride variant, on every selection path, equals the oracle's."""
    rng = np.random.default_rng(12)
    _select_against_oracle(_select_cases(rng, trials=30), rng, stride_real=True)


def test_score_then_select_equals_reduce():
    say("score+select == reduce, qwen ragged B=3")
    w = synth.qwen_ragged(device=DEV, B=3, n_lo=256, n_hi=2000, D=3584)
    r = reducer_for(w)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)
    cv2, s, _ = r.score(w.X, w.Xpre, w.Xpost)
    idx, src = r.select(cv2, s, w.N, w.K)
    torch.cuda.synchronize()
    assert torch.equal(idx, res.idx) and torch.equal(src, res.src)
    r.close()


def test_empty_batch_and_errors():
    import paper_2607_13500_amd as tr
    say("empty batch / invalid calls")
    r = tr.Reducer(64, 64, torch.bfloat16, max_images=4, max_tokens=1000, max_N=500)
    X = torch.zeros(0, 64, dtype=torch.bfloat16, device=DEV)
    res = r.reduce(X, X, X, [], [])
    assert res.out.shape == (0, 64) and res.idx.numel() == 0
    X = torch.randn(10, 64, device=DEV).to(torch.bfloat16)
    with pytest.raises(tr.TRError):
        r.reduce(X, X, X, [10], [11])                                    # K > N
    with pytest.raises(tr.TRError):
        r.reduce(X, X, X, [5, 5], [0, 2])                                # K < 1
    big = torch.randn(1000, 64, device=DEV).to(torch.bfloat16)
    with pytest.raises(tr.TRError):
        r.reduce(big[:600], big[:600], big[:600], [600], [10])          # N > max_N
    with pytest.raises(tr.TRError):
        tr.Reducer(64, 64, torch.bfloat16, max_N=tr.capacity_N() + 1)   # beyond LDS capacity
    r.close()


def test_create_reports_enomem_and_keeps_nothing(monkeypatch):
    """A device allocation failing inside tr_create (forced by the library's
    TR_FAIL_ALLOC hook, for each of a bf16 context's six allocations) gives
    TR_ENOMEM with *out == NULL, and frees what was already allocated."""
    import ctypes
    from paper_2607_13500_amd import _lib
    say("tr_create allocation failures")
    lib = _lib.load()
    p = _lib.Params(D=4096, Dc=4096, dtype=_lib.TR_BF16, max_images=64, max_tokens=4_000_000, max_N=576,
                    flags=0, lam=1.0 / 3.0, keep_ratio=0.0)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for k in range(1, 7):
        monkeypatch.setenv("TR_FAIL_ALLOC", str(k))
        for _ in range(4):
            ctx = ctypes.c_void_p(1234)
            st = lib.tr_create(ctypes.byref(p), ctypes.byref(ctx))
            assert st == _lib.TR_ENOMEM, (k, st)
            assert ctx.value is None
            assert b"failed" in lib.tr_last_error()
    monkeypatch.delenv("TR_FAIL_ALLOC")
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    # 24 failed creates; a leak of the allocations made before the failing one
    # would keep at least 16 MB each (4M tokens x 4 B)
    assert free0 - free1 < 32 << 20, (free0, free1)
    ctx = ctypes.c_void_p()
    assert lib.tr_create(ctypes.byref(p), ctypes.byref(ctx)) == _lib.TR_OK and ctx.value
    lib.tr_destroy(ctx)


def test_capacity_and_max_n():
    import paper_2607_13500_amd as tr
    cap = tr.capacity_N()
    say("max N", cap)
    assert cap >= 18432          # the longest workload (a 32-frame clip) fits
    w = synth.video(device=DEV, B=1, frames=1, positions=cap, D=256, K=cap // 7)
    run_and_check(w)
    # K = N and lambda extremes at the maximum size
    w.K = [cap]
    run_and_check(w)
    for lam in (0.0, 1.0):
        w.lam, w.K = lam, [cap // 5]
        run_and_check(w)


@pytest.mark.parametrize("variant", ["algorithm-1", "stride-real", "shannon"])
def test_batching_and_order_do_not_change_any_image(variant):
    """Every image's kept indices, sources, kept rows and scores are the same
    bit for bit whether it is reduced alone, in a ragged batch or in a
    permuted batch.  The paths differ between these: alone, an image of at
    most 1024 tokens takes the one-token-per-thread selection with the copy
    fused into it, in the batch the general selection; an image with a large
    remainder is shared by more or fewer workgroups depending on how many
    such images its launch holds."""
    import paper_2607_13500_amd as tr
    w = synth.qwen_ragged(device=DEV, seed=11, B=7, n_lo=64, n_hi=9000, D=256)
    say("ragged batch N", w.N, "K", w.K, variant)
    offs = np.concatenate([[0], np.cumsum(w.N)]).tolist()
    flags = dict(stride_real=variant == "stride-real", shannon=variant == "shannon")

    def run(order):
        Ns = [w.N[b] for b in order]
        Ks = [w.K[b] for b in order]
        cut = lambda t: torch.cat([t[offs[b]:offs[b + 1]] for b in order]).contiguous()
        r = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=len(order), max_tokens=sum(Ns), max_N=max(Ns),
                       **flags)
        res = r.reduce(cut(w.X), cut(w.Xpre), cut(w.Xpost), Ns, Ks, want_scores=True)
        torch.cuda.synchronize()
        per, ko, to = {}, 0, 0
        for b, n, k in zip(order, Ns, Ks):
            per[b] = (res.idx[ko:ko + k].cpu(), res.src[ko:ko + k].cpu(),
                      res.out[ko:ko + k].view(torch.int16).cpu(), res.h2[to:to + n].cpu(), res.s[to:to + n].cpu())
            ko += k
            to += n
        r.close()
        return per

    base = run(list(range(w.B)))
    others = [("permuted", run([3, 6, 0, 5, 1, 4, 2]))]
    others += [("alone", run([b])) for b in range(w.B)]
    for what, got in others:
        for b, v in got.items():
            for name, x, y in zip(("idx", "src", "out", "h2", "s"), base[b], v):
                assert torch.equal(x, y), (what, b, w.N[b], name)


def test_many_large_images_one_workgroup_each():
    """More images with large remainders than half the compute units: the
    launch gives each image one workgroup, which ranks all of its buckets a
    bucket per wavefront (the workgroup count per image is picked per launch
    from the device's compute units; the result does not depend on it)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    B = cus // 2 + 1
    say("uniform batch of", B, "x 4160 tokens, D 64, K 64 (remainder 4139)")
    w = synth.video(device=DEV, B=B, frames=1, positions=4160, D=64, K=64)
    run_and_check(w)


def test_ragged_batch_beyond_one_selection_launch():
    """A ragged batch of more images than one selection launch describes (the
    per-image descriptors travel in the launch's arguments, 32 to a launch):
    the batch is selected in three launches, and every image matches the
    oracle, long ones shared by several workgroups in the later launches
    included."""
    w = synth.qwen_ragged(device=DEV, seed=21, B=70, n_lo=16, n_hi=9000, D=128)
    say("ragged batch of", w.B, "images, N", min(w.N), "..", max(w.N), "tokens", sum(w.N))
    rep, _ = run_and_check(w, use_keep_ratio=True)
    assert rep.images == 70


def test_many_tiny_images():
    """Thousands of images of 1 to 40 tokens (a ragged batch selected in 32
    launches, then a uniform batch of 4096 one-token images in one launch):
    every image against the oracle, K from 1 to N."""
    import random
    rng = random.Random(77)
    N = [rng.randint(1, 40) for _ in range(1000)]
    K = [rng.randint(1, n) for n in N]
    g = torch.Generator(device="cpu").manual_seed(77)
    rows = sum(N)
    X = (torch.randn(rows, 48, generator=g) * torch.exp(torch.randn(rows, 1, generator=g))).to(torch.bfloat16)
    P = torch.randn(rows, 40, generator=g).to(torch.bfloat16)
    Q = (P.float() + torch.randn(rows, 40, generator=g)).to(torch.bfloat16)
    w = synth.Workload("tiny", X.to(DEV), P.to(DEV), Q.to(DEV), N, K, synth.LAMBDA)
    say("ragged batch of", w.B, "images of 1..40 tokens")
    rep, _ = run_and_check(w)
    assert rep.images == 1000
    w = synth.Workload("tiny", X[:4096].to(DEV), P[:4096].to(DEV), Q[:4096].to(DEV), [1] * 4096, [1] * 4096,
                       synth.LAMBDA)
    say("uniform batch of 4096 one-token images")
    rep, res = run_and_check(w)
    assert torch.count_nonzero(res.idx) == 0


def test_batch_beyond_4_gib_per_tensor():
    """A batch whose tensors pass 4 GiB (1100 images of 576 x 4096 bf16, 5.2 GB
    each of X, X_pre, X_post): every byte offset is 64-bit.  Images at the
    start, the middle and the end of the batch match the oracle run on those
    images alone (an image's result depends on its own rows only), and the
    fused projection over this X equals the GEMM on the gathered copy."""
    import paper_2607_13500_amd as tr
    w = synth.llava(device=DEV, B=1100, N=576, D=4096, K=64)
    assert w.X.numel() * w.X.element_size() > 4 << 30
    say("batch of", w.B, "images,", sum(w.N), "tokens,", w.X.numel() * 2 / 1e9, "GB per tensor")
    r = reducer_for(w)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    torch.cuda.synchronize()
    for b in (0, 1, 550, 1098, 1099):
        t0, t1, k0, k1 = 576 * b, 576 * (b + 1), 64 * b, 64 * (b + 1)
        sub = synth.Workload(w.name, w.X[t0:t1], w.Xpre[t0:t1], w.Xpost[t0:t1], [576], [64], w.lam)
        got = tr.ReduceResult(res.out[k0:k1], res.idx[k0:k1], res.src[k0:k1], res.h2[t0:t1], res.s[t0:t1])
        assert torch.equal(got.out.view(torch.int16), sub.X[got.idx.long()].view(torch.int16)), b
        rep = parity.check(sub, got, parity.oracle_reference(sub))
        print("    image", b, rep.summary(), flush=True)
        assert rep.ok(), (b, rep.failures[:5])
    # the projection reading the kept rows straight from this X (past 31-bit
    # offsets: the GEMM's register-prefetch tiling) equals the GEMM on the
    # gathered copy (the LDS-destination tiling) bit for bit
    g = torch.Generator(device=DEV).manual_seed(5)
    W = (torch.randn(1024, 4096, device=DEV, generator=g) / 64).to(torch.bfloat16)
    proj = r.reduce_project(w.X, w.Xpre, w.Xpost, w.N, w.K, W)
    ref = r.gemm(res.out, W)
    torch.cuda.synchronize()
    assert torch.equal(proj.idx, res.idx)
    assert torch.equal(proj.out.view(torch.int16), ref.view(torch.int16))
    r.close()


# ------------------------------------------------------ non-finite inputs

@pytest.mark.parametrize("N,dtype", [(600, torch.bfloat16), (5000, torch.bfloat16), (300, torch.float32)])
def test_non_finite_inputs_give_well_formed_output(N, dtype):
    """NaN and infinite inputs make the scores unspecified, but the selection
    falls back to its integer paths (a non-finite key range is never
    bucketed), so the output is still K distinct ascending in-range indices
    with the stage split of Algorithm 1, and out is the gathered rows."""
    say("non-finite inputs", N, dtype)
    g = torch.Generator().manual_seed(N)
    D = Dc = 256
    X = torch.randn(N, D, generator=g)
    P = torch.randn(N, Dc, generator=g)
    Q = torch.randn(N, Dc, generator=g)
    X[3, 5] = float("nan")
    X[7] = float("inf")
    X[11, :10] = float("-inf")
    X[13] = float("nan")
    P[17, 0] = float("nan")
    Q[19] = float("inf")
    P[23] = 3.0e38
    cast = lambda t: t.to(dtype).to(DEV).contiguous()
    K = N // 7
    w = synth.Workload("nonfinite", cast(X), cast(P), cast(Q), [N], [K], synth.LAMBDA)
    r = reducer_for(w)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    # NaN keys straight into the selection
    ki = torch.randn(N, generator=g)
    ki[::9] = float("nan")
    ks = torch.randn(N, generator=g)
    ks[::5] = float("-inf")
    ks[1::11] = float("nan")
    idx2, src2 = r.select(ki.to(DEV), ks.to(DEV), [N], [K])
    torch.cuda.synchronize()
    K1, K2, _ = oracle.budget(N, K, synth.LAMBDA)
    for idx, src in ((res.idx.cpu().numpy(), res.src.cpu().numpy()), (idx2.cpu().numpy(), src2.cpu().numpy())):
        assert idx.size == K and np.all(np.diff(idx) > 0) and idx.min() >= 0 and idx.max() < N
        assert int((src == 0).sum()) == K1 and int((src == 1).sum()) == K2
    rows = res.idx.long()
    assert torch.equal(res.out.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                       w.X.index_select(0, rows).view(torch.int16 if dtype == torch.bfloat16 else torch.int32))
    r.close()


@pytest.mark.parametrize("shannon", [False, True])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_check_finite_counts_the_nonfinite_rows(dtype, shannon):
    """TR_FLAG_CHECK_FINITE: the context counts every scored row that holds a
    NaN or an infinite element, once per row, among the tensors the call
    reads (X when H2 is computed, X_pre / X_post when s is); huge finite
    values are not counted.  The count accumulates over calls until read with
    reset.  On finite rows nothing is counted and every result equals that of
    a context without the flag, bit for bit."""
    import ctypes
    import paper_2607_13500_amd as tr
    from paper_2607_13500_amd import _lib
    say("check finite", dtype, "shannon", shannon)
    g = torch.Generator().manual_seed(77)
    N, D, Dc, K = 600, 256, 200, 60
    X = torch.randn(N, D, generator=g)
    P = torch.randn(N, Dc, generator=g)
    Q = torch.randn(N, Dc, generator=g)
    X[3, 5] = float("nan")
    X[7] = float("inf")
    X[11, :10] = float("-inf")
    X[13] = float("nan")
    X[40, 100] = float("nan")
    X[29, 0] = 3.0e38                  # finite
    P[17, 0] = float("nan")
    P[40, 3] = float("inf")            # the same row as an X entry: counted once
    Q[19] = float("inf")
    P[23] = 3.0e38                     # finite
    x_rows, c_rows = {3, 7, 11, 13, 40}, {17, 19, 40}
    cast = lambda t: t.to(dtype).to(DEV).contiguous()
    Xd, Pd, Qd = cast(X), cast(P), cast(Q)

    def ctx(lam):
        return tr.Reducer(D, Dc, dtype, lam=lam, max_images=1, max_tokens=N, max_N=N, shannon=shannon,
                          check_finite=True)

    r = ctx(synth.LAMBDA)
    r.reduce(Xd, Pd, Qd, [N], [K])
    assert r.nonfinite_rows() == len(x_rows | c_rows)
    r.reduce(Xd, Pd, Qd, [N], [K], want_scores=True)
    assert r.nonfinite_rows(reset=True) == 2 * len(x_rows | c_rows)
    assert r.nonfinite_rows() == 0
    r.score(Xd, Pd, Qd)
    assert r.nonfinite_rows(reset=True) == len(x_rows | c_rows)
    r.close()
    r = ctx(1.0)                                   # s decides nothing: the states are not read
    r.reduce(Xd, Pd, Qd, [N], [K])
    assert r.nonfinite_rows() == len(x_rows)
    r.close()
    r = ctx(0.0)                                   # H2 decides nothing: X is only gathered
    r.reduce(Xd, Pd, Qd, [N], [K])
    assert r.nonfinite_rows() == len(c_rows)
    r.close()
    # finite rows: no count, and the same bits as without the flag
    w = synth.llava(device=DEV, B=3, N=577, D=520, K=100, dtype=dtype)
    a = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=3, max_tokens=sum(w.N), max_N=577, shannon=shannon,
                   check_finite=True)
    b = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=3, max_tokens=sum(w.N), max_N=577, shannon=shannon)
    ra = a.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    rb = b.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    assert a.nonfinite_rows() == 0
    assert torch.equal(ra.idx, rb.idx) and torch.equal(ra.src, rb.src)
    assert torch.equal(ra.h2.view(torch.int32), rb.h2.view(torch.int32))
    assert torch.equal(ra.s.view(torch.int32), rb.s.view(torch.int32))
    assert torch.equal(ra.out.view(torch.uint8), rb.out.view(torch.uint8))
    with pytest.raises(tr.TRError) as e:           # only a context holds the count
        b.nonfinite_rows()
    assert e.value.status == _lib.TR_EUNSUPPORTED
    a.close()
    b.close()
    p = _lib.Params(D=w.D, Dc=w.Dc, dtype=_lib.TR_BF16 if dtype == torch.bfloat16 else _lib.TR_FP32, max_images=0,
                    max_tokens=0, max_N=0, flags=_lib.TR_FLAG_CHECK_FINITE, lam=w.lam, keep_ratio=0.0)
    out = torch.empty(sum(w.K), w.D, dtype=dtype, device=DEV)
    idx = torch.empty(sum(w.K), dtype=torch.int32, device=DEV)
    Nh = (ctypes.c_int32 * 3)(*w.N)
    Kh = (ctypes.c_int32 * 3)(*w.K)
    st = _lib.load().tr_reduce_noalloc(ctypes.byref(p), w.X.data_ptr(), w.Xpre.data_ptr(), w.Xpost.data_ptr(), 3,
                                       Nh, Kh, out.data_ptr(), idx.data_ptr(), None, None, None, None)
    assert st == _lib.TR_EUNSUPPORTED
    torch.cuda.synchronize()


# ------------------------------------------------------ stream ordering

ORDER_CASES = [
    ("llava", dict(B=64, N=576, D=4096, K=64)),
    ("qwen_ragged", dict(B=9, n_lo=256, n_hi=9000, D=1024)),
    ("video", dict(B=3, frames=8, positions=576, D=512, K=288)),       # split selection
]


@pytest.mark.parametrize("name,kw", ORDER_CASES, ids=[n for n, _ in ORDER_CASES])
def test_reduce_is_ordered_on_the_callers_stream(name, kw):
    """Work the caller enqueues on its stream right after tr_reduce, with no
    host synchronisation, sees the finished outputs: on the null stream and on
    a stream of the caller's own, for back-to-back calls, and equal to the run
    with the per-stage timing events."""
    import paper_2607_13500_amd as tr
    say("stream order", name, kw)
    w = synth.make(name, device=DEV, **kw)
    say("   rows", sum(w.N), "images", w.B)
    r = reducer_for(w)
    r.timing(True)
    ref_run = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    with pytest.raises(tr.TRError):   # rejected before any launch: not timed
        r.reduce(w.X, w.Xpre, w.Xpost, w.N, [n + 1 for n in w.N], want_scores=True)
    torch.cuda.synchronize()
    ms, calls = r.timing_read()
    # score and select each run a kernel; the gather stage is empty when the
    # selection copies the kept rows itself
    assert calls == 1 and ms[0] > 0 and ms[1] > 0 and ms[2] >= 0, (ms, calls)
    assert r.timing_read()[1] == 0
    r.timing(False)
    for stream in (torch.cuda.current_stream(), torch.cuda.Stream()):
        with torch.cuda.stream(stream):
            copies = []
            for _ in range(3):
                res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
                copies.append([t.clone() for t in res])
        torch.cuda.synchronize()
        for c in copies:
            for u, v in zip(ref_run, c):
                assert torch.equal(u, v)
    rep = parity.check(w, ref_run, parity.oracle_reference(w))
    print("   ", w.name, rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    r.close()


def _bytes(t):
    return t.contiguous().view(torch.uint8)


@pytest.mark.parametrize("name,kw", ORDER_CASES, ids=[n for n, _ in ORDER_CASES])
def test_reduce_replays_from_a_hip_graph(name, kw):
    """tr_reduce allocates nothing, copies nothing from the host and clears its
    scratch with kernels (per-image metadata travels in kernel arguments), so
    a call can be captured in a HIP graph.  Every replay, with eager calls of
    the same context between replays, gives the eager result bit for bit."""
    say("graph replay", name, kw)
    w = synth.make(name, device=DEV, **kw)
    r = reducer_for(w)
    eager = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)
    torch.cuda.synchronize()
    out, idx, src = torch.empty_like(eager.out), torch.empty_like(eager.idx), torch.empty_like(eager.src)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up on the capture stream
        r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src)
    torch.cuda.synchronize()
    for rep in range(3):
        out.zero_()
        idx.fill_(-1)
        src.fill_(7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(_bytes(out), _bytes(eager.out)), "replay %d: out differs" % rep
        assert torch.equal(idx, eager.idx) and torch.equal(src, eager.src), "replay %d: indices differ" % rep
        between = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)   # eager work of the same context
        torch.cuda.synchronize()
        assert torch.equal(between.idx, eager.idx)
    del graph
    r.close()


def test_two_contexts_run_concurrently_from_two_threads():
    """Distinct contexts are independent: two of them, each driven from its own
    host thread on its own stream (the library call releases Python's lock),
    reproduce their single-threaded results bit for bit."""
    import threading
    say("two contexts, two threads")
    cases = [synth.make("llava", device=DEV, B=8, N=576, D=4096, K=64),
             synth.make("qwen_ragged", device=DEV, B=5, n_lo=256, n_hi=6000, D=1024)]
    reducers = [reducer_for(w) for w in cases]
    ref = [r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K) for r, w in zip(reducers, cases)]
    torch.cuda.synchronize()
    got = [[], []]
    errors = []

    def worker(k):
        try:
            s = torch.cuda.Stream()
            w, r = cases[k], reducers[k]
            with torch.cuda.stream(s):
                for _ in range(20):
                    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)
                    got[k].append((res.out.clone(), res.idx.clone(), res.src.clone()))
            s.synchronize()
        except Exception as e:   # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k in range(2):
        assert len(got[k]) == 20
        for out, idx, src in got[k]:
            assert torch.equal(_bytes(out), _bytes(ref[k].out))
            assert torch.equal(idx, ref[k].idx) and torch.equal(src, ref[k].src)
    for r in reducers:
        r.close()


# ------------------------------------------- lambda extremes and stride variant

LAM_CASES = [
    ("llava", dict(B=4, N=576, D=4096, K=64)),
    ("llava_fp32", dict()),
    ("qwen_ragged", dict(B=4, n_lo=256, n_hi=6000, D=3584)),
]


@pytest.mark.parametrize("lam", [0.0, 1.0])
@pytest.mark.parametrize("name,kw", LAM_CASES, ids=[n for n, _ in LAM_CASES])
def test_lambda_extremes_skip_unused_scores(name, kw, lam):
    """lambda = 1 never reads X_pre/X_post (passed as NULL); lambda = 0 never
    scores X.  The kept set equals both the oracle's and that of a call that
    computes both scores."""
    say("lambda fast path", name, kw, "lam", lam)
    w = synth.make(name, device=DEV, **kw)
    w.lam = lam
    r = reducer_for(w)
    full = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    states = (None, None) if lam == 1.0 else (w.Xpre, w.Xpost)
    fast = r.reduce(w.X, *states, w.N, w.K)
    torch.cuda.synchronize()
    assert fast.h2 is None and fast.s is None
    assert torch.equal(full.idx, fast.idx) and torch.equal(full.src, fast.src)
    assert torch.equal(full.out, fast.out)
    rep = parity.check(w, fast, parity.oracle_reference(w))
    print("   ", w.name, "lam", lam, rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    if lam == 1.0:
        assert rep.picks == 0
    r.close()


@pytest.mark.parametrize("D,Dc,dtype", [(4096, 4096, torch.bfloat16), (37, 45, torch.float32),
                                        (3584, 1024, torch.bfloat16)])
def test_partial_scores_are_bit_identical(D, Dc, dtype):
    import paper_2607_13500_amd as tr
    from paper_2607_13500_amd import _lib
    say("partial scores", D, Dc, dtype)
    w = _edge_workload(D, Dc, dtype, EDGE_KINDS, 300)
    r = reducer_for(w)
    cv2, s, h2 = r.score(w.X, w.Xpre, w.Xpost, want_h2=True)
    cv2a, sa, h2a = r.score(w.X, None, None, want_h2=True)
    cv2b, sb, h2b = r.score(None, w.Xpre, w.Xpost, want_h2=True)
    torch.cuda.synchronize()
    assert sa is None and cv2b is None and h2b is None
    assert torch.equal(cv2, cv2a) and torch.equal(h2, h2a) and torch.equal(s, sb)
    # a group given in part is rejected before anything is enqueued
    lib = _lib.load()
    p = lambda t: None if t is None else t.data_ptr()
    for args in ((w.X, None, w.Xpost, cv2, s), (w.X, w.Xpre, w.Xpost, None, s),
                 (None, w.Xpre, w.Xpost, cv2, s), (None, None, None, None, None)):
        st = lib.tr_score(r._ctx, *[p(a) for a in args[:3]], w.X.shape[0], p(args[3]), p(args[4]),
                          None, None)
        assert st == _lib.TR_EINVAL, args
    # lambda = 1/3 needs the MLP states: NULL is an argument error
    with pytest.raises(tr.TRError):
        r.reduce(w.X, None, None, w.N, w.K)
    # asking for s needs them too, whatever lambda is
    r1 = tr.Reducer(D, Dc, dtype, lam=1.0, max_images=1, max_tokens=300, max_N=300)
    with pytest.raises(tr.TRError):
        r1.reduce(w.X, None, None, w.N, w.K, want_scores=True)
    r1.close()
    r.close()


SHANNON_CASES = [
    ("llava_fp32", dict()),                                            # 10 % near-constant rows
    ("llava", dict(B=6, N=576, D=4096)),
    ("llava", dict(B=3, N=577, D=520, K=100)),
    ("qwen_ragged", dict(B=4, n_lo=256, n_hi=5000, D=3584)),
    ("video", dict(B=1, frames=8, positions=576, D=1024, K=288)),
]


@pytest.mark.parametrize("name,kw", SHANNON_CASES, ids=[f"{n}-{i}" for i, (n, _) in enumerate(SHANNON_CASES)])
def test_shannon_variant_parity(name, kw):
    say("shannon", name, kw)
    w = synth.make(name, device=DEV, **kw)
    r = reducer_for(w, shannon=True)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    key, s2, h1 = r.score(w.X, w.Xpre, w.Xpost, want_h2=True)
    key_only, _, h1_only = r.score(w.X, None, None, want_h2=True)
    torch.cuda.synchronize()
    assert torch.equal(h1, res.h2) and torch.equal(s2, res.s)
    assert torch.equal(key, key_only) and torch.equal(h1, h1_only)
    rep = parity.check(w, res, parity.oracle_reference(w, entropy=1), cv2_gpu=key, entropy=1)
    print("   ", w.name, "shannon", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    assert rep.stage1_swaps <= max(1, rep.images // 10)
    r.close()


@pytest.mark.parametrize("D,Dc,dtype", [(4096, 4096, torch.bfloat16), (1024, 1024, torch.float32),
                                        (37, 45, torch.bfloat16), (5, 3, torch.float32),
                                        (1, 1, torch.bfloat16)])
def test_shannon_degenerate_rows(D, Dc, dtype):
    say("shannon degenerate rows", D, Dc, dtype)
    w = _edge_workload(D, Dc, dtype, EDGE_KINDS, 150)
    r = reducer_for(w, shannon=True)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    key, _, _ = r.score(w.X, None, None)
    rep = parity.check(w, res, parity.oracle_reference(w, entropy=1), cv2_gpu=key, entropy=1)
    print("   ", "edge shannon", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    h1 = res.h2.cpu().numpy()
    if D > 1:
        assert h1[0] == 0.0 and h1[8] == 0.0                       # all-zero rows
        assert abs(h1[1]) < 1e-5                                    # one-hot (log D - KL in fp32)
        assert abs(h1[2] - math.log(D)) < 1e-5 * math.log(D)        # uniform magnitude
        assert key[2].item() == 0.0 and key[10].item() == 0.0       # ... ties exactly: KL = 0
    r.close()


STRIDE_CASES = [
    ("llava", dict(B=4, N=576, D=4096, K=64)),
    ("llava_next", dict(B=2, D=4096, K=320)),
    ("qwen_ragged", dict(B=4, n_lo=256, n_hi=9000, D=3584)),
    ("video", dict(B=1, frames=8, positions=576, D=1024, K=288)),     # N = 4608: split selection
]


@pytest.mark.parametrize("name,kw", STRIDE_CASES, ids=[n for n, _ in STRIDE_CASES])
def test_stride_real_variant_parity(name, kw):
    say("stride real", name, kw)
    w = synth.make(name, device=DEV, **kw)
    r = reducer_for(w, stride_real=True)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    cv2, _, _ = r.score(w.X, None, None)
    ref = parity.oracle_reference(w, stride_mode=1)
    rep = parity.check(w, res, ref, cv2_gpu=cv2, stride_mode=1)
    print("   ", w.name, "stride real", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    assert rep.stage2_near <= max(4, rep.picks // 100)
    # the variant differs from Algorithm 1 wherever R / K2 is not an integer
    base = reducer_for(w).reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)
    torch.cuda.synchronize()
    assert not torch.equal(base.idx, res.idx)
    r.close()


# ---------------------------------------------------------------- full sizes

FULL = [
    ("llava_fp32", dict(), False),
    ("llava", dict(K=64), False),
    ("llava", dict(K=128), False),
    ("llava", dict(K=192), False),
    ("llava_next", dict(), False),
    ("qwen_ragged", dict(), True),
    ("video", dict(), False),
]

FULL_SHANNON = [("llava", dict(K=64), False), ("qwen_ragged", dict(), True)]


@pytest.mark.parametrize("name,kw,ratio", FULL, ids=[f"{n}-{kw.get('K', '')}" for n, kw, _ in FULL])
def test_reduce_parity_full(name, kw, ratio):
    say("full", name, kw)
    w = synth.make(name, device=DEV, **kw)
    say("   rows", sum(w.N), "D", w.D, "images", w.B)
    rep, _ = run_and_check(w, use_keep_ratio=ratio)
    # near-tie excusals must stay rare
    assert rep.stage1_swaps <= max(2, rep.images // 10)
    assert rep.stage2_near <= max(4, rep.picks // 100)


@pytest.mark.parametrize("name,kw,ratio", FULL_SHANNON, ids=[n for n, _, _ in FULL_SHANNON])
def test_shannon_parity_full(name, kw, ratio):
    say("full shannon", name, kw)
    w = synth.make(name, device=DEV, **kw)
    r = reducer_for(w, shannon=True)
    res = r.reduce(w.X, w.Xpre, w.Xpost, w.N, None if ratio else w.K, want_scores=True)
    key, _, _ = r.score(w.X, None, None)
    rep = parity.check(w, res, parity.oracle_reference(w, entropy=1), cv2_gpu=key, entropy=1)
    print("   ", w.name, "shannon", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    assert rep.stage1_swaps <= max(2, rep.images // 10)
    r.close()


FULL_VARIANTS = [("lambda0", dict(lam=0.0)), ("lambda1", dict(lam=1.0)), ("stride_real", dict(stride_real=True))]


@pytest.mark.parametrize("name,opt", FULL_VARIANTS, ids=[n for n, _ in FULL_VARIANTS])
def test_variants_parity_full_llava(name, opt):
    """The variants at the benchmark size (64 x 576 x 4096 bf16 -> 64), in the
    launch configuration bench.py times for them."""
    say("full variant", name)
    w = synth.llava(device=DEV, B=64, N=576, D=4096, K=64)
    stride_real = opt.get("stride_real", False)
    if "lam" in opt:
        w.lam = opt["lam"]
    r = reducer_for(w, stride_real=stride_real)
    states = (None, None) if w.lam == 1.0 else (w.Xpre, w.Xpost)
    res = r.reduce(w.X, *states, w.N, w.K)
    ref = parity.oracle_reference(w, stride_mode=1 if stride_real else 0)
    rep = parity.check(w, res, ref, stride_mode=1 if stride_real else 0)
    print("   ", name, rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    assert rep.stage1_swaps <= 2 and rep.stage2_near <= max(4, rep.picks // 100)
    r.close()


def test_read_bandwidth_hook():
    import ctypes
    import paper_2607_13500_amd as tr
    from paper_2607_13500_amd import _lib
    say("read bandwidth hook")
    buf = torch.ones(1 << 20, dtype=torch.float32, device=DEV)
    other = torch.ones(3000, dtype=torch.bfloat16, device=DEV)   # 6000 B: a partial last span
    tr.read_bandwidth([buf, buf[: (1 << 19)], other])
    torch.cuda.synchronize()
    lib = _lib.load()
    sink = torch.empty(16, dtype=torch.int32, device=DEV)

    def call(ptrs, sizes, words=16):
        n = len(ptrs)
        p = (ctypes.c_void_p * n)(*ptrs)
        b = (ctypes.c_int64 * n)(*sizes)
        return lib.tr_read_bandwidth(ctypes.cast(p, ctypes.c_void_p), ctypes.cast(b, ctypes.c_void_p), n,
                                     sink.data_ptr(), words, None)

    assert call([buf.data_ptr()], [100]) == _lib.TR_EINVAL              # not a multiple of 16
    assert call([buf.data_ptr() + 4], [64]) == _lib.TR_EINVAL           # misaligned
    assert call([buf.data_ptr()], [64], words=0) == _lib.TR_EINVAL      # no sink
    assert call([buf.data_ptr()], [0]) == _lib.TR_OK                    # nothing to read
    assert call([buf.data_ptr(), other.data_ptr()], [64, 5984]) == _lib.TR_OK
    torch.cuda.synchronize()