"""GPU parity of the matrix-core GEMM and of the two fusions built on it.

* tr_gemm_bf16 against the oracle's float64 product (oracle.matmul_bt) of the
  same bf16 inputs: each output is the fp32 sum rounded once to bf16, so
  |C - C64| <= 2^-8 |C64| + 2 K 2^-24 sum_k |a_k b_k| (rounding to bf16 plus
  a bound on fp32 accumulation), on ragged M, padded strides and gathered
  rows (out-of-range indices read as zero rows).
* tr_mlp_out_cos (Eq. 6 fused into the encoder MLP's second layer): X_post
  as above and s against the oracle's cosine of x' and the float64 x''
  within 1e-5 (floor 1), then the whole module with that key against the
  oracle's selection (parity protocol of tests/parity.py).
* tr_reduce_project (projection fused with the gather): the kept indices
  equal tr_reduce's, and the projected rows equal tr_gemm_bf16 applied to
  tr_reduce's gathered output bit for bit, and the float64 product within the
  bound above.
"""
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


def reducer(D=4096, Dc=1024, max_tokens=40000, max_images=64, max_N=4096, lam=synth.LAMBDA):
    import paper_2607_13500_amd as tr
    return tr.Reducer(D, Dc, torch.bfloat16, lam=lam, max_images=max_images, max_tokens=max_tokens,
                      max_N=max_N)


def randn_bf16(g, *shape, scale=1.0):
    return (scale * torch.randn(*shape, generator=g)).to(torch.bfloat16)


def check_gemm(C, A_rows, B):
    """C (device bf16) against the float64 product of the given (host) rows."""
    ref = oracle.matmul_bt(A_rows, B)
    K = ref.shape[1] and oracle.as_f64(B).shape[1]
    mag = oracle.matmul_bt(np.abs(oracle.as_f64(A_rows)), np.abs(oracle.as_f64(B)))
    bound = 2.0 ** -8 * np.abs(ref) + 2 * K * 2.0 ** -24 * mag + 1e-30
    got = oracle.as_f64(C.cpu())
    bad = np.abs(got - ref) > bound
    assert not bad.any(), "%d outputs outside the bound, first at %s" % (bad.sum(), np.argwhere(bad)[:3])


# N % 256 == 0 with K % 128 == 0 runs the wide tiling (256 x 256, LDS-destination
# loads), every other shape the narrow one (256 x 128, register prefetch).
@pytest.mark.parametrize("M,N,K,pad", [(1, 128, 64, 0), (300, 256, 128, 0), (257, 384, 512, 8),
                                       (130, 256, 192, 0), (257, 512, 512, 8), (1000, 1024, 4096, 0),
                                       (4096, 4096, 4096, 0)])
def test_gemm_matches_fp64(M, N, K, pad):
    say("gemm", M, N, K, "pad", pad)
    g = torch.Generator().manual_seed(M + N + K)
    A = randn_bf16(g, M, K + pad)
    B = randn_bf16(g, N, K + pad)
    r = reducer()
    Ad, Bd = A.to(DEV), B.to(DEV)
    C = r.gemm(Ad[:, :K], Bd[:, :K])
    torch.cuda.synchronize()
    check_gemm(C, A[:, :K].contiguous(), B[:, :K].contiguous())
    r.close()


@pytest.mark.parametrize("N", [384, 512])
def test_gemm_gathered_rows(N):
    say("gemm gather 777 x %d x 512" % N)
    g = torch.Generator().manual_seed(3)
    A = randn_bf16(g, 900, 512)
    B = randn_bf16(g, N, 512)
    rows = torch.randint(-3, 905, (777,), generator=g, dtype=torch.int32)   # duplicates and out-of-range
    r = reducer()
    C = r.gemm(A.to(DEV), B.to(DEV), rows=rows.to(DEV))
    torch.cuda.synchronize()
    ok = (rows >= 0) & (rows < A.shape[0])
    Ag = torch.zeros(777, 512, dtype=torch.bfloat16)
    Ag[ok] = A[rows[ok].long()]
    check_gemm(C, Ag, B)
    assert torch.count_nonzero(C[~ok.to(DEV)]) == 0
    r.close()


@pytest.mark.parametrize("tile_rows", [None, 128, 192, 256])
def test_gemm_tilings_agree_bit_for_bit(tile_rows, monkeypatch):
    """The wide (N % 256 == 0) and narrow (N % 256 == 128) tilings run the same
    MFMA sequence for every output element, so the columns they share are
    bit-identical, plain and gathered, at every tile height of the wide one
    (TR_GEMM_TILE_ROWS pins it; None leaves it to the model)."""
    if tile_rows is not None:
        monkeypatch.setenv("TR_GEMM_TILE_ROWS", str(tile_rows))
    say("gemm wide vs narrow 1000 x 512/384 x 1024, tile rows", tile_rows)
    g = torch.Generator().manual_seed(11)
    A = randn_bf16(g, 1000, 1024).to(DEV)
    B = randn_bf16(g, 512, 1024).to(DEV)
    rows = torch.randint(-2, 1003, (600,), generator=g, dtype=torch.int32).to(DEV)
    r = reducer()
    wide, narrow = r.gemm(A, B), r.gemm(A, B[:384])
    gw, gn = r.gemm(A, B, rows=rows), r.gemm(A, B[:384], rows=rows)
    torch.cuda.synchronize()
    assert torch.equal(wide[:, :384].view(torch.int16), narrow.view(torch.int16))
    assert torch.equal(gw[:, :384].view(torch.int16), gn.view(torch.int16))
    r.close()


def test_gemm_rejects_unsupported_shapes():
    import paper_2607_13500_amd as tr
    say("gemm shape errors")
    r = reducer()
    A = torch.zeros(10, 96, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(tr.TRError):
        r.gemm(A, torch.zeros(128, 96, dtype=torch.bfloat16, device=DEV))      # K % 64 != 0
    with pytest.raises(tr.TRError):
        r.gemm(A[:, :64], torch.zeros(100, 64, dtype=torch.bfloat16, device=DEV))   # N % 128 != 0
    r.close()


def mlp_inputs(M, Dc, Hd, seed):
    g = torch.Generator().manual_seed(seed)
    Xpre = randn_bf16(g, M, Dc)
    # hidden activations of a GELU-like MLP: mostly positive, some zeros
    H = torch.relu(torch.randn(M, Hd, generator=g) + 0.3).to(torch.bfloat16)
    W2 = randn_bf16(g, Dc, Hd, scale=1.0 / np.sqrt(Hd))
    return Xpre, H, W2


@pytest.mark.parametrize("M,Dc,Hd", [(1000, 1024, 4096), (333, 256, 512), (64, 128, 64)])
def test_mlp_out_cos_parity(M, Dc, Hd):
    run_mlp_out_cos_parity(M, Dc, Hd)


@pytest.mark.parametrize("tile_rows", [128, 192, 256])
def test_mlp_out_cos_parity_each_tile_height(tile_rows, monkeypatch):
    """The cosine epilogue stages P through LDS by 128-row halves; 192-row
    tiles split a wavefront's rows across both stages."""
    monkeypatch.setenv("TR_GEMM_TILE_ROWS", str(tile_rows))
    run_mlp_out_cos_parity(1000, 512, 256)


def run_mlp_out_cos_parity(M, Dc, Hd):
    say("mlp_out_cos", M, Dc, Hd)
    Xpre, H, W2 = mlp_inputs(M, Dc, Hd, M + Dc)
    Xpre[5] = 0                                                   # zero-norm x': s = 0
    r = reducer(D=Dc, Dc=Dc, max_tokens=M)
    Xpost, s = r.mlp_out_cos(H.to(DEV), W2.to(DEV), Xpre.to(DEV))
    torch.cuda.synchronize()
    check_gemm(Xpost, H, W2)
    # Eq. (6) on the x'' the caller receives (the stored bf16 X_post, itself
    # within the GEMM bound of the fp64 product above)
    xp = oracle.as_f64(Xpre)
    xq = oracle.as_f64(Xpost.cpu())
    s_ref = np.array([oracle.cosine(xp[m], xq[m]) for m in range(M)])
    sg = s.double().cpu().numpy()
    err = np.abs(sg - s_ref)
    print("    max |s - s_oracle(stored x'')| = %.2e" % err.max(), flush=True)
    assert np.all(err <= parity.TOL * np.maximum(parity.S_FLOOR, np.abs(s_ref)))
    assert sg[5] == 0.0
    # the same s an unfused scoring pass computes from the stored states
    _, s_unfused, _ = r.score(None, Xpre.to(DEV), Xpost)
    torch.cuda.synchronize()
    du = (s - s_unfused).abs().max().item()
    print("    max |s_fused - s_unfused| = %.2e" % du, flush=True)
    assert du <= 2e-6
    r.close()


def test_fused_mlp_module_parity():
    """Stage II key from the fused epilogue, Stage I from X: the module's
    selection against the oracle's (H2 of X, cos(x', x'') on the stored x''),
    and against the unfused module on the same stored states."""
    B, N, D, Dc, Hd, K = 6, 576, 1024, 1024, 4096, 64
    say("fused mlp module", B, N, D, Dc, Hd, K)
    w = synth.llava(device="cpu", B=B, N=N, D=D, K=K)
    Xpre, H, W2 = mlp_inputs(B * N, Dc, Hd, 17)
    r = reducer(D=D, Dc=Dc, max_tokens=B * N, max_images=B, max_N=N)
    Xd = w.X.to(DEV)
    Xpost, s = r.mlp_out_cos(H.to(DEV), W2.to(DEV), Xpre.to(DEV))
    res = r.reduce_given_s(Xd, s, w.N, w.K)
    torch.cuda.synchronize()
    h2, _ = oracle.scores(w.X, w.Xpre, w.Xpost)
    xp = oracle.as_f64(Xpre)
    xq = oracle.as_f64(Xpost.cpu())
    s_ref = np.array([oracle.cosine(xp[m], xq[m]) for m in range(B * N)])
    idx, src = [], []
    for b in range(B):
        i, sr = oracle.select(h2[b * N:(b + 1) * N], s_ref[b * N:(b + 1) * N], K, w.lam)
        idx.append(i)
        src.append(sr)
    ref = {"h2": h2, "s": s_ref, "idx": np.concatenate(idx), "src": np.concatenate(src)}
    wd = synth.Workload(w.name, Xd, None, None, w.N, w.K, w.lam)
    res = res._replace(s=s)
    rep = parity.check(wd, res, ref)
    print("   ", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    # the unfused module on the stored X_pre / X_post keeps the same tokens
    # (the two s differ only in fp32 summation order)
    unf = r.reduce(Xd, Xpre.to(DEV), Xpost, w.N, w.K)
    torch.cuda.synchronize()
    differ = int((unf.idx != res.idx).sum().item())
    print("    fused vs unfused kept tokens differing: %d of %d" % (differ, unf.idx.numel()), flush=True)
    assert differ <= 2
    r.close()


@pytest.mark.parametrize("name,kw,nout", [("llava", dict(B=8, N=576, D=4096, K=64), 1024),
                                          ("qwen_ragged", dict(B=3, n_lo=256, n_hi=3000, D=3584), 512)])
def test_reduce_project_parity(name, kw, nout):
    say("reduce_project", name, kw, nout)
    w = synth.make(name, device=DEV, **kw)
    import paper_2607_13500_amd as tr
    r = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=w.B, max_tokens=sum(w.N), max_N=max(w.N))
    g = torch.Generator().manual_seed(nout)
    W = randn_bf16(g, nout, w.D, scale=1.0 / np.sqrt(w.D))
    Wd = W.to(DEV)
    base = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K)
    proj = r.reduce_project(w.X, w.Xpre, w.Xpost, w.N, w.K, Wd)
    two_step = r.gemm(base.out, Wd)
    torch.cuda.synchronize()
    assert torch.equal(base.idx, proj.idx) and torch.equal(base.src, proj.src)
    assert torch.equal(proj.out.view(torch.int16), two_step.view(torch.int16))
    rows = []
    o0 = r0 = 0
    idx = proj.idx.cpu().numpy()
    for n, k in zip(w.N, w.K):
        rows.append(idx[o0:o0 + k] + r0)
        o0 += k
        r0 += n
    rows = np.concatenate(rows)
    check_gemm(proj.out, w.X.cpu()[torch.from_numpy(rows).long()], W)
    # the selection itself against the oracle (the gather path's parity)
    rep = parity.check(w, base, parity.oracle_reference(w))
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    r.close()


def test_reduce_project_lambda_one_without_states():
    """lambda = 1 never reads X_pre / X_post, also when the kept rows are projected."""
    import paper_2607_13500_amd as tr
    say("reduce_project lambda=1, NULL states")
    w = synth.llava(device=DEV, B=4, N=576, D=1024, K=64)
    r = tr.Reducer(w.D, w.Dc, w.dtype, lam=1.0, max_images=w.B, max_tokens=sum(w.N), max_N=576)
    g = torch.Generator().manual_seed(2)
    W = randn_bf16(g, 256, w.D, scale=1.0 / np.sqrt(w.D)).to(DEV)
    a = r.reduce_project(w.X, None, None, w.N, w.K, W)
    b = r.reduce_project(w.X, w.Xpre, w.Xpost, w.N, w.K, W)
    torch.cuda.synchronize()
    assert torch.equal(a.idx, b.idx) and torch.equal(a.out.view(torch.int16), b.out.view(torch.int16))
    assert int(a.src.sum()) == 0                                   # every kept token from Stage I
    r.close()


def test_mlp_out_cos_rejects_bad_requests():
    import paper_2607_13500_amd as tr
    say("mlp_out_cos errors")
    H = torch.zeros(100, 64, dtype=torch.bfloat16, device=DEV)
    P = torch.zeros(100, 192, dtype=torch.bfloat16, device=DEV)
    r = tr.Reducer(192, 192, torch.bfloat16, max_images=1, max_tokens=100, max_N=100)
    with pytest.raises(tr.TRError):                                # Dc = 192 is not a multiple of 128
        r.mlp_out_cos(H, torch.zeros(192, 64, dtype=torch.bfloat16, device=DEV), P)
    r.close()
    r = tr.Reducer(128, 128, torch.bfloat16, max_images=1, max_tokens=50, max_N=50)
    with pytest.raises(tr.TRError):                                # M = 100 > max_tokens = 50
        r.mlp_out_cos(H, torch.zeros(128, 64, dtype=torch.bfloat16, device=DEV),
                      torch.zeros(100, 128, dtype=torch.bfloat16, device=DEV))
    r.close()
    r = tr.Reducer(128, 128, torch.float32, max_images=1, max_tokens=100, max_N=100)
    with pytest.raises((tr.TRError, ValueError, TypeError)):        # fp32 context
        r.mlp_out_cos(H, torch.zeros(128, 64, dtype=torch.bfloat16, device=DEV),
                      torch.zeros(100, 128, dtype=torch.float32, device=DEV))
    r.close()


@pytest.mark.parametrize("c", range(24))
def test_gemm_random_shapes(c, monkeypatch):
    """Seeded random shapes: M from 1 to 5000, N and K over their allowed
    multiples, padded row strides, gathered rows with duplicates and
    out-of-range indices, each tile height; against the float64 product."""
    import random
    rng = random.Random(7000 + c)
    tile = rng.choice([None, 128, 192, 256])
    if tile is not None:
        monkeypatch.setenv("TR_GEMM_TILE_ROWS", str(tile))
    M = rng.choice([1, 31, 64, 200, 257, 1000, 2049, 5000])
    N = 128 * rng.choice([1, 2, 3, 4, 8, 12])
    K = 64 * rng.choice([1, 2, 3, 4, 8, 16])
    pad = rng.choice([0, 0, 8, 24])
    gather = rng.random() < 0.4
    say("gemm random", c, M, N, K, "pad", pad, "gather", gather, "tile rows", tile)
    g = torch.Generator().manual_seed(7000 + c)
    R = M + rng.choice([0, 7, 300]) if gather else M
    A = randn_bf16(g, R, K + pad)
    B = randn_bf16(g, N, K + pad)
    r = reducer()
    Ad, Bd = A.to(DEV), B.to(DEV)
    if gather:
        rows = torch.randint(-2, R + 3, (M,), generator=g, dtype=torch.int32)
        C = r.gemm(Ad[:, :K], Bd[:, :K], rows=rows.to(DEV))
        ok = (rows >= 0) & (rows < R)
        Ag = torch.zeros(M, K, dtype=torch.bfloat16)
        Ag[ok] = A[rows[ok].long(), :K]
        torch.cuda.synchronize()
        check_gemm(C, Ag, B[:, :K].contiguous())
        assert torch.count_nonzero(C[~ok.to(DEV)]) == 0
    else:
        C = r.gemm(Ad[:, :K], Bd[:, :K])
        torch.cuda.synchronize()
        check_gemm(C, A[:, :K].contiguous(), B[:, :K].contiguous())
    r.close()
