"""Exact brute-force reference for tiny inputs (pure Python, rational arithmetic).

A third implementation of the selection, independent of both the fp64 oracle
and the HIP path, used only as a pin for the oracle on tiny N:

* Stage I order (Eq. (3)-(4)): H2 = -log(sum_j p_j^2) is strictly decreasing in
  q = sum_j p_j^2 = sum_j x_j^2 / (sum_j |x_j|)^2, so tokens are compared on the
  exact rational q (ascending), ties to the lower index.  An all-zero row has
  H2 = 0, i.e. q = 1.
* Stage II order (Eq. (6)): s = sign(dot) * sqrt(dot^2 / (|x'|^2 |x''|^2)); the
  order of s equals the lexicographic order of (sign, sign * dot^2/(n1 n2)),
  compared exactly as fractions; a zero norm gives s = 0.
* X^imp is found by enumerating every K1-subset and keeping the one whose
  members all precede all non-members (it must be unique).
* The stride picks are found by rank counting: rank_i = #{j in rem : j before
  i}; token i is picked when rank_i = j*t for some j < K2 (Algorithm 1).

Every float converts to a Fraction exactly, so for any float32 or bfloat16
input these orders are the exact mathematical ones.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction


def _frac(v) -> Fraction:
    return Fraction(float(v))


def stage1_key(row):
    """Exact q = sum p^2 for a row (smaller q = larger H2)."""
    mags = [abs(_frac(v)) for v in row]
    s1 = sum(mags, Fraction(0))
    if s1 == 0:
        return Fraction(1)
    return sum((m * m for m in mags), Fraction(0)) / (s1 * s1)


def stage2_key(a, b):
    """Exact sort key of s = cos(a, b)."""
    fa = [_frac(v) for v in a]
    fb = [_frac(v) for v in b]
    dot = sum((u * w for u, w in zip(fa, fb)), Fraction(0))
    n1 = sum((u * u for u in fa), Fraction(0))
    n2 = sum((w * w for w in fb), Fraction(0))
    if n1 == 0 or n2 == 0 or dot == 0:
        return (0, Fraction(0))
    sign = 1 if dot > 0 else -1
    return (sign, sign * dot * dot / (n1 * n2))


def budget(N: int, K: int, lam: float):
    k1 = math.floor(lam * K)
    k2 = K - k1
    t = max(1, (N - k1) // k2) if k2 > 0 else 0
    return k1, k2, t


def select(q, skey, K: int, lam: float, given_imp=None, stride_mode: int = 0):
    """Brute-force Algorithm 1 on exact keys; returns (idx list, src list)."""
    N = len(q)
    k1, k2, t = budget(N, K, lam)
    if given_imp is None:
        found = []
        for sub in itertools.combinations(range(N), k1):
            ss = set(sub)
            ok = all((q[i], i) < (q[j], j) for i in ss for j in range(N) if j not in ss)
            if ok:
                found.append(ss)
        assert len(found) == 1, "Stage I subset not unique"
        imp = found[0]
    else:
        imp = {i for i in range(N) if given_imp[i]}
        assert len(imp) == k1
    rem = [i for i in range(N) if i not in imp]
    div = set()
    R = len(rem)
    if k2 > 0:
        if stride_mode == 0:
            wanted = {j * t for j in range(k2)}
        else:
            wanted = {(j * R) // k2 for j in range(k2)}
        for i in rem:
            rank = sum(1 for j in rem if (skey[j], j) < (skey[i], i))
            if rank in wanted:
                div.add(i)
    idx = sorted(imp | div)
    src = [1 if i in div else 0 for i in idx]
    return idx, src


def reduce_rows(X, Xpre, Xpost, K: int, lam: float, given_imp=None, stride_mode: int = 0):
    q = [stage1_key(r) for r in X]
    sk = [stage2_key(a, b) for a, b in zip(Xpre, Xpost)]
    return select(q, sk, K, lam, given_imp, stride_mode)
