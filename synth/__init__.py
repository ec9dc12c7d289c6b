"""Seeded synthetic inputs shaped like the paper's VLM workloads.

This module holds no arithmetic of the token-reduction method: it only draws
random tensors.  Both the oracle side and the HIP side of every test, and the
benchmark, take their inputs from here.

A workload is three row-aligned packed tensors, all of one dtype:

* ``X``     [sum N, D]   final visual tokens (scored by entropy and gathered);
* ``Xpre``  [sum N, Dc]  input of the vision encoder's last MLP;
* ``Xpost`` [sum N, Dc]  output of that MLP, ``Xpost = W2 gelu(W1 Xpre)``.

The pre-/post-MLP pair mimics Eq. (5): ``Xpre`` is a per-channel rescale of the
standardised token and ``Xpost`` is a random two-layer GELU MLP of it (width
256, fp32, drawn once per workload).  Exact duplicate tokens copy all three
rows byte for byte.  Values are drawn in fp32 and rounded to the workload dtype
(round to nearest even for bfloat16).

The five named recipes are the benchmark's workloads (B = images or clips):

1. ``llava_fp32``: B=1, N=576 (24x24), D=1024 fp32, K=64; 8-cluster Gaussian
   mixture, per-token scale LogNormal(0, 0.5), 10 % near-constant rows.
2. ``llava``: B=64, N=576, D=4096 bf16, K=64 (128, 192); 16 clusters per image,
   5 % exact duplicate tokens, 10 % low-variance rows around a per-image
   background.
3. ``llava_next``: B=16, N=2880 = 5 tiles x 576, D=4096 bf16, K=320; 8 clusters
   per tile, 20 % near-duplicates of tokens in other tiles.
4. ``qwen_ragged``: 32 images, N ~ U{256..16384}, D=3584 bf16, 11 % kept;
   16 clusters per image, per-token norms |t|*sqrt(D) with t ~ Student-t(3).
5. ``video``: 4 clips x 32 frames x 576 tokens (N=18432), D=4096 bf16, K=1152;
   shared per-position base + AR(1) temporal drift (rho = 0.95) + noise.

The random streams come from ``torch.Generator`` on the target device, so a
workload is reproducible per (recipe, seed, device); tests hand the very same
tensors to both implementations.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import torch

LAMBDA = 1.0 / 3.0   # 64 importance + 128 diversity of 192 (the paper's efficiency setting)
MLP_WIDTH = 256


@dataclasses.dataclass
class Workload:
    name: str
    X: torch.Tensor
    Xpre: torch.Tensor
    Xpost: torch.Tensor
    N: List[int]
    K: List[int]
    lam: float
    keep_ratio: Optional[float] = None

    @property
    def D(self) -> int:
        return self.X.shape[1]

    @property
    def Dc(self) -> int:
        return self.Xpre.shape[1]

    @property
    def B(self) -> int:
        return len(self.N)

    @property
    def dtype(self) -> torch.dtype:
        return self.X.dtype

    def algorithmic_bytes(self, score_x: bool = True, score_states: bool = True) -> int:
        """Compulsory HBM bytes of one reduction: read X (every row when it is
        scored, else only the kept rows), Xpre and Xpost (when s is scored),
        write out."""
        e = self.X.element_size()
        return sum(e * ((n if score_x else k) * self.D + (2 * n * self.Dc if score_states else 0)
                        + k * self.D) for n, k in zip(self.N, self.K))


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _randn(g, *shape, device):
    return torch.randn(*shape, generator=g, device=device, dtype=torch.float32)


def _randint(g, lo, hi, shape, device):
    return torch.randint(lo, hi, shape, generator=g, device=device)


def _lognormal(g, sigma, *shape, device):
    return torch.exp(sigma * _randn(g, *shape, device=device))


def _mlp_pair(g, Xr: torch.Tensor, Dc: int, dtype, device, chunk_rows: int = 1 << 15):
    """Xpre = gamma * standardize(X) (per row), Xpost = W2 gelu(W1 Xpre).

    ``Xr`` is the rounded token block in fp32.  When Dc differs from D the
    standardised token is cut or tiled to Dc channels.
    """
    D = Xr.shape[1]
    gamma = _lognormal(g, 0.25, Dc, device=device)
    W1 = _randn(g, MLP_WIDTH, Dc, device=device) / math.sqrt(Dc)
    W2 = _randn(g, Dc, MLP_WIDTH, device=device) / math.sqrt(MLP_WIDTH)
    rows = Xr.shape[0]
    pre = torch.empty(rows, Dc, dtype=dtype, device=device)
    post = torch.empty(rows, Dc, dtype=dtype, device=device)
    for r0 in range(0, rows, chunk_rows):
        xb = Xr[r0:r0 + chunk_rows]
        mu = xb.mean(dim=1, keepdim=True)
        sd = xb.std(dim=1, unbiased=False, keepdim=True).clamp_min(1e-12)
        z = (xb - mu) / sd
        if Dc != D:
            reps = (Dc + D - 1) // D
            z = z.repeat(1, reps)[:, :Dc]
        p = (z * gamma).to(dtype)
        pf = p.float()
        h = torch.nn.functional.gelu(pf @ W1.t())
        q = (h @ W2.t()).to(dtype)
        pre[r0:r0 + chunk_rows] = p
        post[r0:r0 + chunk_rows] = q
    return pre, post


def _cluster_tokens(g, n, D, n_clusters, device):
    """z_i = (mu_c(i) + eps_i) / sqrt(2): unit-variance marginals, clustered."""
    centres = _randn(g, n_clusters, D, device=device)
    lab = _randint(g, 0, n_clusters, (n,), device)
    return (centres[lab] + _randn(g, n, D, device=device)) / math.sqrt(2.0)


def _copy_rows(tensors, dst: torch.Tensor, src: torch.Tensor):
    for t in tensors:
        t[dst] = t[src]


def _finish(name, g, X32, N, K, dtype, device, Dc=None, dups=None, keep_ratio=None):
    Xr = X32.to(dtype)
    pre, post = _mlp_pair(g, Xr.float(), Dc or X32.shape[1], dtype, device)
    if dups is not None:
        dst, src = dups
        _copy_rows((Xr, pre, post), dst, src)
    return Workload(name, Xr.contiguous(), pre.contiguous(), post.contiguous(),
                    [int(n) for n in N], [int(k) for k in K], LAMBDA, keep_ratio)


def llava_fp32(device="cpu", seed=1001, B=1, N=576, D=1024, K=64, Dc=None):
    g = _gen(device, seed)
    blocks = []
    for b in range(B):
        z = _cluster_tokens(g, N, D, 8, device)
        a = _lognormal(g, 0.5, N, 1, device=device)
        x = a * z
        n_flat = max(1, round(0.10 * N))
        rows = torch.randperm(N, generator=g, device=device)[:n_flat]
        c = _randn(g, n_flat, 1, device=device)
        eps = _randn(g, n_flat, D, device=device)
        x[rows] = a[rows] * (c + 1e-3 * c.abs() * eps)
        blocks.append(x)
    return _finish("llava_fp32", g, torch.cat(blocks), [N] * B, [K] * B, torch.float32, device, Dc)


def llava(device="cpu", seed=1002, B=64, N=576, D=4096, K=64, Dc=None, dtype=torch.bfloat16):
    g = _gen(device, seed)
    blocks, dst_all, src_all = [], [], []
    n_low = round(0.10 * N)
    n_dup = round(0.05 * N)
    for b in range(B):
        x = _cluster_tokens(g, N, D, 16, device)
        perm = torch.randperm(N, generator=g, device=device)
        low = perm[:n_low]
        beta = _randn(g, 1, D, device=device)
        x[low] = beta + 0.05 * _randn(g, n_low, D, device=device)
        dst = perm[n_low:n_low + n_dup]
        pool = torch.cat([perm[:n_low], perm[n_low + n_dup:]])
        src = pool[_randint(g, 0, pool.numel(), (n_dup,), device)]
        dst_all.append(dst + b * N)
        src_all.append(src + b * N)
        blocks.append(x)
    dups = (torch.cat(dst_all), torch.cat(src_all)) if n_dup else None
    return _finish("llava", g, torch.cat(blocks), [N] * B, [K] * B, dtype, device, Dc, dups)


def llava_next(device="cpu", seed=1003, B=16, tiles=5, tile_tokens=576, D=4096, K=320, Dc=None):
    g = _gen(device, seed)
    N = tiles * tile_tokens
    blocks = []
    n_near = round(0.20 * N)
    for b in range(B):
        x = torch.cat([_cluster_tokens(g, tile_tokens, D, 8, device) for _ in range(tiles)])
        dst = torch.randperm(N, generator=g, device=device)[:n_near]
        tile_of = dst // tile_tokens
        other = (tile_of + _randint(g, 1, tiles, (n_near,), device)) % tiles
        src = other * tile_tokens + _randint(g, 0, tile_tokens, (n_near,), device)
        x[dst] = x[src] + 0.01 * _randn(g, n_near, D, device=device)
        blocks.append(x)
    return _finish("llava_next", g, torch.cat(blocks), [N] * B, [K] * B, torch.bfloat16, device, Dc)


def qwen_ragged(device="cpu", seed=1004, B=32, n_lo=256, n_hi=16384, D=3584, keep_ratio=0.11, Dc=None):
    g = _gen(device, seed)
    Ns = _randint(g, n_lo, n_hi + 1, (B,), device).tolist()
    blocks = []
    for n in Ns:
        z = _cluster_tokens(g, n, D, 16, device)
        # Student-t(3) = N(0,1) / sqrt(chi2_3 / 3)
        chi2 = (_randn(g, n, 3, device=device) ** 2).sum(dim=1, keepdim=True)
        tau = _randn(g, n, 1, device=device) / torch.sqrt(chi2 / 3.0)
        x = tau.abs() * math.sqrt(D) * z / z.norm(dim=1, keepdim=True)
        blocks.append(x)
    Ks = [min(n, max(1, math.floor(keep_ratio * n))) for n in Ns]
    return _finish("qwen_ragged", g, torch.cat(blocks), Ns, Ks, torch.bfloat16, device, Dc,
                   keep_ratio=keep_ratio)


def video(device="cpu", seed=1005, B=4, frames=32, positions=576, D=4096, K=1152, rho=0.95, Dc=None):
    g = _gen(device, seed)
    N = frames * positions
    blocks = []
    for b in range(B):
        base = _randn(g, positions, D, device=device)
        d = _randn(g, positions, D, device=device)
        clip = torch.empty(N, D, device=device)
        for f in range(frames):
            if f:
                d = rho * d + math.sqrt(1 - rho * rho) * _randn(g, positions, D, device=device)
            clip[f * positions:(f + 1) * positions] = base + 0.5 * d + 0.1 * _randn(g, positions, D, device=device)
        blocks.append(clip)
    return _finish("video", g, torch.cat(blocks), [N] * B, [K] * B, torch.bfloat16, device, Dc)


RECIPES = {
    "llava_fp32": llava_fp32,
    "llava": llava,
    "llava_next": llava_next,
    "qwen_ragged": qwen_ragged,
    "video": video,
}


def make(name: str, device="cpu", **kw) -> Workload:
    return RECIPES[name](device=device, **kw)
