"""fp64 CPU oracle for the ALTR token-reduction path (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never loads it and shares no code with it.

The arithmetic lives in ``altr_oracle.c`` (plain C, double precision, one loop
per definition):

* Eq. (3)-(4): per-token second-order Renyi entropy of normalised magnitudes.
* Eq. (6): cosine between the pre- and post-MLP states of a token.
* Algorithm 1 / Eq. (7): budget split, top-K1 by entropy, ascending sort of
  the remainder by the cosine, stride picks, union in ascending token index.
* Variants: Shannon entropy of the same distribution as the Stage I score;
  the real-valued stride interval of the method's prose.

This module only marshals numpy arrays into that library and builds it with
gcc when it is missing.  Parity pins: ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "altr_oracle.c")
_LIB = os.path.join(_HERE, "libaltr_oracle.so")

DTYPE_F32 = 0
DTYPE_BF16 = 1
DTYPE_F64 = 2

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math) into libaltr_oracle.so."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # ALTR_ORACLE_LIB names another build of altr_oracle.c to load instead;
    # the mutation test uses it to run the pins against deliberately broken
    # copies of the oracle.
    path = os.environ.get("ALTR_ORACLE_LIB") or _LIB
    if path == _LIB and not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(path)
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
    lib.altr_oracle_renyi2.argtypes = [vp, i32, i32]
    lib.altr_oracle_renyi2.restype = dbl
    lib.altr_oracle_renyi2_cv.argtypes = [vp, i32, i32]
    lib.altr_oracle_renyi2_cv.restype = dbl
    lib.altr_oracle_cosine.argtypes = [vp, vp, i32, i32]
    lib.altr_oracle_cosine.restype = dbl
    lib.altr_oracle_shannon.argtypes = [vp, i32, i32]
    lib.altr_oracle_shannon.restype = dbl
    lib.altr_oracle_scores.argtypes = [vp, vp, vp, i32, i64, i32, i32, i32, vp, vp]
    lib.altr_oracle_scores.restype = None
    lib.altr_oracle_budget.argtypes = [i32, i32, dbl, vp, vp, vp]
    lib.altr_oracle_budget.restype = i32
    lib.altr_oracle_select.argtypes = [i32, i32, dbl, vp, vp, vp, i32, vp, vp]
    lib.altr_oracle_select.restype = i32
    lib.altr_oracle_reduce.argtypes = [vp, vp, vp, i32, i32, vp, vp, i32, i32, dbl,
                                       i32, i32, vp, vp, vp, vp, vp, vp]
    lib.altr_oracle_reduce.restype = i32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def as_raw(t) -> tuple[np.ndarray, int]:
    """Return (contiguous numpy array of the stored bits, dtype code).

    Accepts numpy float32 arrays, numpy uint16 arrays holding bfloat16 bit
    patterns, and CPU torch tensors of dtype float32 or bfloat16.
    """
    try:
        import torch
        if isinstance(t, torch.Tensor):
            t = t.detach().cpu().contiguous()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16), DTYPE_BF16
            if t.dtype == torch.float32:
                return t.numpy(), DTYPE_F32
            raise TypeError("oracle takes float32 or bfloat16, got %s" % t.dtype)
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(t)
    if a.dtype == np.float32:
        return a, DTYPE_F32
    if a.dtype == np.uint16:
        return a, DTYPE_BF16
    if a.dtype == np.float64:
        return a, DTYPE_F64
    raise TypeError("unsupported dtype %s" % a.dtype)


def as_f64(t) -> np.ndarray:
    """The values of float32 / bfloat16 / float64 rows (numpy or CPU torch) as float64, exactly."""
    a, dt = as_raw(t)
    if dt == DTYPE_BF16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def matmul_bt(A, B) -> np.ndarray:
    """A . B^T in float64 (numpy) from exactly widened inputs: the linear layers
    around the path (the encoder MLP's second layer, the projector)."""
    return as_f64(A) @ as_f64(B).T


def renyi2(row) -> float:
    """Eq. (3)-(4) for one row (natural log; all-zero row -> 0)."""
    a, dt = as_raw(row)
    return _load().altr_oracle_renyi2(_ptr(a), dt, a.size)


def renyi2_cv(row) -> float:
    """log D - log1p(Var|x| / mean|x|^2): the same value as renyi2, other form."""
    a, dt = as_raw(row)
    return _load().altr_oracle_renyi2_cv(_ptr(a), dt, a.size)


def shannon(row) -> float:
    """Shannon entropy -sum p log p of the Eq. (3) distribution (variant; all-zero row -> 0)."""
    a, dt = as_raw(row)
    return _load().altr_oracle_shannon(_ptr(a), dt, a.size)


def cosine(a, b) -> float:
    """Eq. (6) for one token (zero norm -> 0)."""
    ra, dt = as_raw(a)
    rb, dt2 = as_raw(b)
    assert dt == dt2 and ra.size == rb.size
    return _load().altr_oracle_cosine(_ptr(ra), _ptr(rb), dt, ra.size)


def scores(X, Xpre, Xpost, entropy: int = 2):
    """Per-row (H, s) in float64 for packed [rows, D] / [rows, Dc] inputs.

    H is the Renyi-2 entropy (entropy=2, the method) or the Shannon entropy
    (entropy=1, the variant).
    """
    x, dt = as_raw(X)
    p, dt1 = as_raw(Xpre)
    q, dt2 = as_raw(Xpost)
    assert dt == dt1 == dt2
    rows, D = x.shape
    Dc = p.shape[1]
    assert p.shape == q.shape == (rows, Dc)
    h2 = np.empty(rows, np.float64)
    s = np.empty(rows, np.float64)
    _load().altr_oracle_scores(_ptr(x), _ptr(p), _ptr(q), dt, rows, D, Dc, int(entropy),
                               _ptr(h2), _ptr(s))
    return h2, s


def budget(N: int, K: int, lam: float):
    """Algorithm 1 budget: (K1, K2, t); raises ValueError outside 1<=K<=N, 0<=lam<=1."""
    k1, k2, t = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    rc = _load().altr_oracle_budget(int(N), int(K), float(lam), ctypes.byref(k1),
                                    ctypes.byref(k2), ctypes.byref(t))
    if rc != 0:
        raise ValueError("invalid budget N=%r K=%r lambda=%r" % (N, K, lam))
    return k1.value, k2.value, t.value


def select(h2, s, K: int, lam: float, given_imp=None, stride_mode: int = 0):
    """Algorithm 1 selection for one image from its scores.

    ``h2`` ranks Stage I (higher kept first, ties to the lower index), ``s``
    orders Stage II (ascending, ties in index order).  ``given_imp`` (bool
    array) replaces Stage I by a supplied X^imp (the conditional form).
    Returns (idx int32 ascending, src uint8: 0 = X^imp, 1 = X^div).
    """
    h2 = np.ascontiguousarray(h2, dtype=np.float64)
    s = np.ascontiguousarray(s, dtype=np.float64)
    N = h2.size
    gi = None if given_imp is None else np.ascontiguousarray(given_imp, dtype=np.uint8)
    idx = np.empty(K, np.int32)
    src = np.empty(K, np.uint8)
    rc = _load().altr_oracle_select(N, int(K), float(lam), _ptr(h2), _ptr(s), _ptr(gi),
                                    int(stride_mode), _ptr(idx), _ptr(src))
    if rc != 0:
        raise ValueError("oracle select rejected N=%d K=%d lambda=%r" % (N, K, lam))
    return idx, src


def reduce(X, Xpre, Xpost, N, K, lam: float, *, given_imp=None, stride_mode: int = 0,
           entropy: int = 2, want_out: bool = True, want_scores: bool = True):
    """The whole module over a packed batch (Algorithm 1 per image).

    Returns a dict with ``idx`` (int32 [sum K], image-local), ``src``
    (uint8 [sum K]), ``out`` (kept rows of X, same raw dtype, or None),
    ``h2`` / ``s`` (float64 [sum N], or None; ``h2`` holds H1 when
    ``entropy`` = 1, the Shannon variant).
    """
    x, dt = as_raw(X)
    p, _ = as_raw(Xpre)
    q, _ = as_raw(Xpost)
    rows, D = x.shape
    Dc = p.shape[1]
    Na = np.ascontiguousarray(N, dtype=np.int32)
    Ka = np.ascontiguousarray(K, dtype=np.int32)
    assert int(Na.sum()) == rows
    sk = int(Ka.sum())
    idx = np.empty(sk, np.int32)
    src = np.empty(sk, np.uint8)
    out = np.empty((sk, D), x.dtype) if want_out else None
    h2 = np.empty(rows, np.float64) if want_scores else None
    s = np.empty(rows, np.float64) if want_scores else None
    gi = None if given_imp is None else np.ascontiguousarray(given_imp, dtype=np.uint8)
    rc = _load().altr_oracle_reduce(_ptr(x), _ptr(p), _ptr(q), dt, Na.size, _ptr(Na),
                                    _ptr(Ka), D, Dc, float(lam), int(stride_mode), int(entropy),
                                    _ptr(gi),
                                    _ptr(idx), _ptr(src), _ptr(out), _ptr(h2), _ptr(s))
    if rc != 0:
        raise ValueError("oracle reduce failed on image %d" % (-rc - 1))
    return {"idx": idx, "src": src, "out": out, "h2": h2, "s": s}
