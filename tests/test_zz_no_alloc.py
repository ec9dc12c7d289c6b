"""tr_reduce_noalloc against tr_reduce (GPU, through the C ABI).

The entry point that allocates nothing works in the library's static device
scratch.  It must give tr_reduce's results bit for bit: on two calls in a row,
the second with a smaller input (so the scratch still holds the first call's
contents), again on the first input (the split selection's bitmaps were left
clean), and under a variant.  Calls beyond the scratch are rejected before
anything is enqueued.
"""
import pytest
import torch

import parity
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(*a):
    print("[case]", *a, flush=True)


def _bits(t):
    return t.contiguous().view(torch.uint8)


def _both(w, **kw):
    """(tr_reduce result, tr_reduce_noalloc result) on the same inputs."""
    import paper_2607_13500_amd as tr
    r = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=w.B, max_tokens=sum(w.N), max_N=max(w.N), **kw)
    ref = r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, want_scores=True)
    sk, rows = sum(w.K), sum(w.N)
    out = torch.full((sk, w.D), 7.0, dtype=w.dtype, device=DEV)
    idx = torch.full((sk,), -1, dtype=torch.int32, device=DEV)
    src = torch.full((sk,), 9, dtype=torch.uint8, device=DEV)
    h2 = torch.full((rows,), float("nan"), device=DEV)
    s = torch.full((rows,), float("nan"), device=DEV)
    got = tr.reduce_noalloc(w.X, w.Xpre, w.Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src, out_h2=h2,
                            out_s=s, lam=w.lam, **kw)
    torch.cuda.synchronize()
    r.close()
    return ref, got


def _same(ref, got, what):
    assert torch.equal(_bits(ref.out), _bits(got.out)), what + ": out differs"
    assert torch.equal(ref.idx, got.idx) and torch.equal(ref.src, got.src), what + ": indices differ"
    assert torch.equal(_bits(ref.h2), _bits(got.h2)) and torch.equal(_bits(ref.s), _bits(got.s)), \
        what + ": scores differ"


def test_noalloc_equals_reduce_on_consecutive_calls():
    # first call: two 4608-token clips (the selection of each is shared by
    # several workgroups through the scratch's bitmaps) and a 576-token image
    say("no-alloc call 1: 2 clips of 8 x 576 tokens + 1 image, D 1024 bf16")
    big = synth.video(device=DEV, B=2, frames=8, positions=576, D=1024, K=288)
    ref, got = _both(big)
    _same(ref, got, "call 1")
    # second call, smaller: 3 LLaVA images of 576 x 4096
    say("no-alloc call 2: 3 x 576 x 4096 bf16 -> 64")
    small = synth.llava(device=DEV, B=3, N=576, D=4096, K=64)
    ref2, got2 = _both(small)
    _same(ref2, got2, "call 2")
    rep = parity.check(small, got2, parity.oracle_reference(small))
    print("   ", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    assert rep.near_ties_rare(), rep.summary()
    # the first input again, and a variant on the second
    say("no-alloc call 3: call 1 again")
    ref3, got3 = _both(big)
    _same(ref3, got3, "call 3")
    assert torch.equal(got3.idx, got.idx)
    say("no-alloc call 4: Shannon entropy, real-interval stride, fp32 image")
    w4 = synth.make("llava_fp32", device=DEV)
    ref4, got4 = _both(w4, shannon=True, stride_real=True)
    _same(ref4, got4, "call 4")


def test_noalloc_replays_from_a_hip_graph():
    """Work under HIP graph capture is one of the callers the entry point is
    for: a captured call (including a split selection, whose bitmaps live in
    the shared static array) replays bit for bit like tr_reduce, with eager
    calls of the entry point on other inputs between the replays."""
    import paper_2607_13500_amd as tr
    say("no-alloc under graph capture: 1 clip of 8 x 576 tokens + 3 images of 576, D 1024 bf16")
    clip = synth.video(device=DEV, B=1, frames=8, positions=576, D=1024, K=288)
    imgs = synth.llava(device=DEV, B=3, N=576, D=1024, K=64)
    ref, _ = _both(clip)
    sk, rows = sum(clip.K), sum(clip.N)
    out = torch.empty(sk, clip.D, dtype=clip.dtype, device=DEV)
    idx = torch.empty(sk, dtype=torch.int32, device=DEV)
    src = torch.empty(sk, dtype=torch.uint8, device=DEV)
    h2 = torch.empty(rows, device=DEV)
    s = torch.empty(rows, device=DEV)

    def call():
        tr.reduce_noalloc(clip.X, clip.Xpre, clip.Xpost, clip.N, clip.K, out=out, out_idx=idx, out_src=src,
                          out_h2=h2, out_s=s, lam=clip.lam)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up on the capture stream (the array is set up by now)
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        out.zero_()
        idx.fill_(-1)
        src.fill_(7)
        h2.fill_(float("nan"))
        s.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _same(ref, tr.ReduceResult(out, idx, src, h2, s), "replay %d" % rep)
        # eager use of the same static array on other inputs between replays
        ref2, got2 = _both(imgs)
        _same(ref2, got2, "eager call between replays %d" % rep)
    del graph


def test_noalloc_at_its_limits():
    """Calls at the scratch's limits: the largest image count (a ragged batch,
    selected in several launches, long images shared by several workgroups)
    and the largest token count, each equal to tr_reduce and to the oracle."""
    from paper_2607_13500_amd import _lib
    B = _lib.TR_NOALLOC_MAX_IMAGES
    say("no-alloc at the image limit:", B, "ragged images, D 64 bf16")
    w = synth.qwen_ragged(device=DEV, seed=31, B=B, n_lo=16, n_hi=3000, D=64)
    assert sum(w.N) <= _lib.TR_NOALLOC_MAX_TOKENS
    ref, got = _both(w)
    _same(ref, got, "image limit")
    rep = parity.check(w, got, parity.oracle_reference(w))
    print("   ", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]
    n = _lib.TR_NOALLOC_MAX_TOKENS // B
    say("no-alloc at the token limit:", B, "x", n, "tokens, D 64 bf16")
    w = synth.video(device=DEV, B=B, frames=1, positions=n, D=64, K=n // 8)
    assert sum(w.N) == _lib.TR_NOALLOC_MAX_TOKENS
    ref, got = _both(w)
    _same(ref, got, "token limit")
    rep = parity.check(w, got, parity.oracle_reference(w))
    print("   ", rep.summary(), flush=True)
    assert rep.ok(), rep.failures[:5]


def test_noalloc_rejects_calls_beyond_its_scratch():
    import paper_2607_13500_amd as tr
    from paper_2607_13500_amd import _lib
    say("no-alloc limits")
    X = torch.zeros(4, 64, dtype=torch.bfloat16, device=DEV)
    idx = torch.zeros(4, dtype=torch.int32, device=DEV)
    n_over = _lib.TR_NOALLOC_MAX_TOKENS // 60000 + 1
    with pytest.raises(tr.TRError, match="no-allocation") as e:
        tr.reduce_noalloc(X, X, X, [60000] * n_over, [1] * n_over, out=X, out_idx=idx)
    assert e.value.status == _lib.TR_EINVAL
    B = _lib.TR_NOALLOC_MAX_IMAGES + 1
    with pytest.raises(tr.TRError, match="no-allocation") as e:
        tr.reduce_noalloc(X, X, X, [1] * B, [1] * B, out=X, out_idx=idx)
    assert e.value.status == _lib.TR_EINVAL
    # an ordinary argument error, as tr_reduce reports it
    with pytest.raises(tr.TRError) as e:
        tr.reduce_noalloc(X, X, X, [4], [5], out=X, out_idx=idx)
    assert e.value.status == _lib.TR_EINVAL
    torch.cuda.synchronize()
