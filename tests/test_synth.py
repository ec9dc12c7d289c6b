"""Shapes, determinism and planted structure of the synthetic workloads."""
import torch

import synth


def test_recipes_small_shapes_and_determinism():
    cases = [
        ("llava_fp32", dict(N=96, D=64)),
        ("llava", dict(B=3, N=80, D=128)),
        ("llava_next", dict(B=2, tiles=3, tile_tokens=40, D=64, K=30)),
        ("qwen_ragged", dict(B=4, n_lo=20, n_hi=90, D=72)),
        ("video", dict(B=2, frames=4, positions=30, D=64, K=20)),
    ]
    for name, kw in cases:
        a = synth.make(name, **kw)
        b = synth.make(name, **kw)
        assert a.X.shape[0] == sum(a.N) == a.Xpre.shape[0] == a.Xpost.shape[0]
        assert len(a.N) == len(a.K) and all(1 <= k <= n for n, k in zip(a.N, a.K))
        for t, u in ((a.X, b.X), (a.Xpre, b.Xpre), (a.Xpost, b.Xpost)):
            assert t.is_contiguous() and torch.equal(t, u)
        assert torch.isfinite(a.X.float()).all() and torch.isfinite(a.Xpost.float()).all()
        assert a.algorithmic_bytes() > 0


def test_llava_duplicates_are_byte_copies():
    w = synth.llava(B=2, N=100, D=64)
    assert w.dtype == torch.bfloat16
    for b in range(2):
        x = w.X[b * 100:(b + 1) * 100].view(torch.int16)
        uniq = torch.unique(x, dim=0).shape[0]
        assert uniq == 100 - 5          # 5 % of 100 tokens are exact copies
        p = w.Xpre[b * 100:(b + 1) * 100].view(torch.int16)
        assert torch.unique(p, dim=0).shape[0] == 95


def test_qwen_keep_ratio():
    w = synth.qwen_ragged(B=5, n_lo=256, n_hi=400, D=32)
    assert w.keep_ratio == 0.11
    assert w.K == [int(0.11 * n) for n in w.N]
