"""MI355X-native ALTR visual-token reduction (Python binding of include/tr.h).

Every step of the path runs in the HIP library libaltr.so (gfx950):

* score  - Eq. (3)-(4) Renyi-2 entropy and Eq. (6) MLP-consistency cosine,
           one HBM pass, one wavefront per token;
* select - Algorithm 1: top-K1 by entropy, ascending sort of the remainder by
           the cosine, stride picks, union in token order (LDS-resident);
* gather - byte copies of the kept rows into a compact [sum K, D] output.

This module only marshals torch tensors (device memory) and the current torch
stream into the C ABI; it computes nothing itself.  If the library is missing
or the tensors are not on a ROCm device, calls raise.
"""
from __future__ import annotations

import ctypes
from typing import NamedTuple, Optional, Sequence

import torch

from . import _lib
from ._lib import Params

__all__ = ["Reducer", "ReduceResult", "TRError", "plan", "capacity_N", "reduce_noalloc", "LAMBDA_PAPER"]

LAMBDA_PAPER = 1.0 / 3.0   # 64 importance + 128 diversity of 192 (efficiency setting)

_DTYPES = {torch.float32: _lib.TR_FP32, torch.bfloat16: _lib.TR_BF16}


class TRError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = _lib.load()
        msg = lib.tr_last_error().decode() or lib.tr_strerror(status).decode()
        super().__init__("%s failed (%s): %s" % (where, lib.tr_strerror(status).decode(), msg))
        self.status = status


def _check(status: int, where: str):
    if status != _lib.TR_OK:
        raise TRError(status, where)


def _i32(seq) -> ctypes.Array:
    arr = (ctypes.c_int32 * len(seq))(*[int(v) for v in seq])
    return arr


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _params(D, Dc, dtype, lam, keep_ratio, max_images, max_tokens, max_N, flags=0) -> Params:
    if dtype not in _DTYPES:
        raise TypeError("dtype must be torch.float32 or torch.bfloat16")
    return Params(D=int(D), Dc=int(Dc or 0), dtype=_DTYPES[dtype], max_images=int(max_images),
                  max_tokens=int(max_tokens), max_N=int(max_N), flags=int(flags), lam=float(lam),
                  keep_ratio=float(keep_ratio or 0.0))


def plan(N: Sequence[int], K: Optional[Sequence[int]] = None, lam: float = LAMBDA_PAPER,
         keep_ratio: Optional[float] = None):
    """Host-only budget plan of the library: lists (K, K1, K2, t) per image."""
    lib = _lib.load()
    B = len(N)
    p = _params(1, 0, torch.float32, lam, keep_ratio, 0, 0, 0)
    outs = [(ctypes.c_int32 * max(B, 1))() for _ in range(4)]
    st = lib.tr_plan(ctypes.byref(p), B, _i32(N), None if K is None else _i32(K), *outs)
    _check(st, "tr_plan")
    return tuple([list(o[:B]) for o in outs])


def read_bandwidth(buffers, stream=None) -> None:
    """Measurement hook: read the (16-byte aligned, contiguous) device tensors
    once, in one kernel launch (the streaming-read ceiling of the device)."""
    lib = _lib.load()
    if not 1 <= len(buffers) <= 8:
        raise ValueError("read_bandwidth takes 1 to 8 tensors")
    sink = torch.empty(4096, dtype=torch.int32, device=buffers[0].device)
    st = stream if stream is not None else torch.cuda.current_stream(buffers[0].device)
    n = len(buffers)
    ptrs = (ctypes.c_void_p * n)(*[b.data_ptr() for b in buffers])
    sizes = (ctypes.c_int64 * n)(*[(b.numel() * b.element_size()) // 16 * 16 for b in buffers])
    _check(lib.tr_read_bandwidth(ctypes.cast(ptrs, ctypes.c_void_p), ctypes.cast(sizes, ctypes.c_void_p), n,
                                 _ptr(sink), sink.numel(), ctypes.c_void_p(st.cuda_stream)), "tr_read_bandwidth")


def capacity_N() -> int:
    """Largest per-image N the selection handles on the current device."""
    return int(_lib.load().tr_capacity_N())


class ReduceResult(NamedTuple):
    out: torch.Tensor              # [sum K, D] kept rows of X
    idx: torch.Tensor              # [sum K] int32, image-local, ascending per image
    src: Optional[torch.Tensor]    # [sum K] uint8, 0 = Stage I, 1 = Stage II
    h2: Optional[torch.Tensor]     # [sum N] float32
    s: Optional[torch.Tensor]      # [sum N] float32


def _flags(stride_real: bool, shannon: bool) -> int:
    return (_lib.TR_FLAG_STRIDE_REAL if stride_real else 0) | (_lib.TR_FLAG_SHANNON if shannon else 0)


def reduce_noalloc(X: torch.Tensor, Xpre: Optional[torch.Tensor], Xpost: Optional[torch.Tensor],
                   N: Sequence[int], K: Optional[Sequence[int]] = None, *, out: torch.Tensor,
                   out_idx: torch.Tensor, out_src: Optional[torch.Tensor] = None,
                   out_h2: Optional[torch.Tensor] = None, out_s: Optional[torch.Tensor] = None,
                   lam: float = LAMBDA_PAPER, keep_ratio: Optional[float] = None,
                   stride_real: bool = False, shannon: bool = False, stream=None) -> ReduceResult:
    """tr_reduce_noalloc: the module without a context, working in the
    library's static device scratch (at most TR_NOALLOC_MAX_TOKENS tokens in
    TR_NOALLOC_MAX_IMAGES images).  Every output is the caller's: nothing is
    allocated here or in the library.  D, Dc and the dtype come from X and
    Xpre."""
    if X.dtype not in _DTYPES or not X.is_cuda or X.dim() != 2 or not X.is_contiguous():
        raise ValueError("X must be a contiguous [rows, D] float32 or bfloat16 tensor on a ROCm device")
    if (Xpre is None) != (Xpost is None):
        raise ValueError("Xpre and Xpost must both be given or both be None")
    Dc = Xpre.shape[1] if Xpre is not None else X.shape[1]
    p = _params(X.shape[1], Dc, X.dtype, lam, keep_ratio, 0, 0, 0, _flags(stride_real, shannon))
    lib = _lib.load()
    st = stream if stream is not None else torch.cuda.current_stream(X.device)
    with torch.cuda.device(X.device):
        status = lib.tr_reduce_noalloc(ctypes.byref(p), _ptr(X), _ptr(Xpre), _ptr(Xpost), len(N), _i32(N),
                                       None if K is None else _i32(K), _ptr(out), _ptr(out_idx),
                                       _ptr(out_src), _ptr(out_h2), _ptr(out_s),
                                       ctypes.c_void_p(st.cuda_stream))
    _check(status, "tr_reduce_noalloc")
    return ReduceResult(out, out_idx, out_src, out_h2, out_s)


class Reducer:
    """A library context bound to one device, row widths, dtype and lambda.

    stride_real selects the real-interval variant of the diversity stride
    (positions floor(j R / K2) of the sorted remainder instead of j t);
    shannon ranks Stage I by Shannon entropy instead of Renyi-2 (the key is
    then log D - H1 and the returned h2 holds H1); check_finite makes the
    context count the scored rows that hold a NaN or infinite element
    (nonfinite_rows reads the count).
    """

    def __init__(self, D: int, Dc: Optional[int] = None, dtype: torch.dtype = torch.bfloat16,
                 lam: float = LAMBDA_PAPER, keep_ratio: Optional[float] = None,
                 max_images: int = 256, max_tokens: int = 1 << 20, max_N: Optional[int] = None,
                 device=None, stride_real: bool = False, shannon: bool = False, check_finite: bool = False):
        if not torch.cuda.is_available():
            raise RuntimeError("paper_2607_13500_amd needs a ROCm GPU (gfx950)")
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else torch.device(device).index or 0)
        self.lib = _lib.load()
        self.D, self.Dc, self.dtype = int(D), int(Dc or D), dtype
        self.lam, self.keep_ratio = float(lam), keep_ratio
        if max_N is None:
            max_N = min(capacity_N_on(self.device), int(max_tokens))
        self.max_images, self.max_tokens, self.max_N = int(max_images), int(max_tokens), int(max_N)
        self.stride_real, self.shannon = bool(stride_real), bool(shannon)
        flags = _flags(stride_real, shannon) | (_lib.TR_FLAG_CHECK_FINITE if check_finite else 0)
        p = _params(D, Dc, dtype, lam, keep_ratio, max_images, max_tokens, max_N, flags)
        ctx = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(self.lib.tr_create(ctypes.byref(p), ctypes.byref(ctx)), "tr_create")
        self._ctx = ctx

    # -- helpers ----------------------------------------------------------
    def _stream(self, stream):
        st = stream if stream is not None else torch.cuda.current_stream(self.device)
        return ctypes.c_void_p(st.cuda_stream)

    def _check_rows(self, name, t, width):
        if not isinstance(t, torch.Tensor) or t.device != self.device:
            raise ValueError("%s must be a tensor on %s" % (name, self.device))
        if t.dtype != self.dtype:
            raise TypeError("%s must be %s, got %s" % (name, self.dtype, t.dtype))
        if t.dim() != 2 or t.shape[1] != width or not t.is_contiguous():
            raise ValueError("%s must be a contiguous [rows, %d] tensor, got %s"
                             % (name, width, tuple(t.shape)))

    def kept_counts(self, N: Sequence[int], K: Optional[Sequence[int]] = None):
        Kb, _, _, _ = plan(N, K, self.lam, self.keep_ratio)
        return Kb

    # -- the module ---------------------------------------------------------
    def reduce(self, X: torch.Tensor, Xpre: Optional[torch.Tensor], Xpost: Optional[torch.Tensor],
               N: Sequence[int], K: Optional[Sequence[int]] = None, *,
               out: Optional[torch.Tensor] = None, out_idx: Optional[torch.Tensor] = None,
               out_src: Optional[torch.Tensor] = None, want_src: bool = True,
               want_scores: bool = False, stream=None) -> ReduceResult:
        """Run score -> select -> gather on a packed batch (asynchronous).

        Xpre and Xpost may be None when no image's Stage II ranks tokens
        (lambda = 1) and want_scores is False; the library then never reads
        them.  Likewise H2 is not computed when no Stage I ranks (lambda = 0).
        """
        self._check_rows("X", X, self.D)
        if (Xpre is None) != (Xpost is None):
            raise ValueError("Xpre and Xpost must both be given or both be None")
        rows = X.shape[0]
        if Xpre is not None:
            self._check_rows("Xpre", Xpre, self.Dc)
            self._check_rows("Xpost", Xpost, self.Dc)
            if Xpre.shape[0] != rows or Xpost.shape[0] != rows:
                raise ValueError("X, Xpre, Xpost must have the same number of rows")
        if sum(int(n) for n in N) != rows:
            raise ValueError("X must have sum(N) = %d rows" % sum(int(n) for n in N))
        sk = sum(self.kept_counts(N, K)) if len(N) else 0
        dev = self.device
        if out is None:
            out = torch.empty(sk, self.D, dtype=self.dtype, device=dev)
        if out_idx is None:
            out_idx = torch.empty(sk, dtype=torch.int32, device=dev)
        if out_src is None and want_src:
            out_src = torch.empty(sk, dtype=torch.uint8, device=dev)
        h2 = torch.empty(rows, dtype=torch.float32, device=dev) if want_scores else None
        s = torch.empty(rows, dtype=torch.float32, device=dev) if want_scores else None
        for name, t, shape, dt in (("out", out, (sk, self.D), self.dtype),
                                   ("out_idx", out_idx, (sk,), torch.int32),
                                   ("out_src", out_src, (sk,), torch.uint8)):
            if t is not None and (t.device != dev or tuple(t.shape) != shape or t.dtype != dt
                                  or not t.is_contiguous()):
                raise ValueError("%s must be a contiguous %s tensor of shape %s on %s"
                                 % (name, dt, shape, dev))
        st = self.lib.tr_reduce(self._ctx, _ptr(X), _ptr(Xpre), _ptr(Xpost), len(N), _i32(N),
                                None if K is None else _i32(K), _ptr(out), _ptr(out_idx),
                                _ptr(out_src), _ptr(h2), _ptr(s), self._stream(stream))
        _check(st, "tr_reduce")
        return ReduceResult(out, out_idx, out_src, h2, s)

    # -- the steps around the path (bf16) ------------------------------------
    def _check_mat(self, name, t, cols=None):
        if not isinstance(t, torch.Tensor) or t.device != self.device or t.dtype != torch.bfloat16 \
                or t.dim() != 2 or t.stride(1) != 1 or (cols is not None and t.shape[1] != cols):
            raise ValueError("%s must be a bf16 [rows, %s] tensor with unit column stride on %s"
                             % (name, cols, self.device))

    def gemm(self, A: torch.Tensor, B: torch.Tensor, rows: Optional[torch.Tensor] = None,
             out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """C = A[rows] . B^T (bf16, fp32 accumulation) on the matrix cores.

        A [R, K], B [N, K]; rows (int32 [M], indices into A; out-of-range rows
        read as zeros) or None for all rows of A.
        """
        self._check_mat("A", A)
        self._check_mat("B", B, A.shape[1])
        M = A.shape[0] if rows is None else rows.numel()
        N, K = B.shape
        if rows is not None and (rows.dtype != torch.int32 or rows.device != self.device
                                 or not rows.is_contiguous()):
            raise ValueError("rows must be a contiguous int32 tensor on %s" % self.device)
        if out is None:
            out = torch.empty(M, N, dtype=torch.bfloat16, device=self.device)
        self._check_mat("out", out, N)
        st = self.lib.tr_gemm_bf16(self._ctx, _ptr(A), A.stride(0), _ptr(rows), A.shape[0], _ptr(B),
                                   B.stride(0), _ptr(out), out.stride(0), M, N, K, self._stream(stream))
        _check(st, "tr_gemm_bf16")
        return out

    def mlp_out_cos(self, Hact: torch.Tensor, W2: torch.Tensor, Xpre: torch.Tensor, *,
                    out: Optional[torch.Tensor] = None, stream=None):
        """(X_post, s): X_post = Hact . W2^T with s = cos(X_pre, X_post) fused in."""
        self._check_mat("Hact", Hact)
        self._check_mat("W2", W2, Hact.shape[1])
        self._check_rows("Xpre", Xpre, self.Dc)
        M, Hd = Hact.shape
        if W2.shape[0] != self.Dc or Xpre.shape[0] != M:
            raise ValueError("W2 must be [Dc, Hd] and Xpre [M, Dc]")
        if out is None:
            out = torch.empty(M, self.Dc, dtype=torch.bfloat16, device=self.device)
        self._check_rows("out", out, self.Dc)
        s = torch.empty(M, dtype=torch.float32, device=self.device)
        st = self.lib.tr_mlp_out_cos(self._ctx, _ptr(Hact), Hact.stride(0), _ptr(W2), W2.stride(0),
                                     _ptr(Xpre), _ptr(out), M, Hd, _ptr(s), self._stream(stream))
        _check(st, "tr_mlp_out_cos")
        return out, s

    def reduce_given_s(self, X: torch.Tensor, key_s: torch.Tensor, N: Sequence[int],
                       K: Optional[Sequence[int]] = None, *, out=None, out_idx=None, out_src=None,
                       want_src: bool = True, stream=None) -> ReduceResult:
        """The module with the Stage II key supplied (e.g. by mlp_out_cos)."""
        self._check_rows("X", X, self.D)
        rows = X.shape[0]
        if key_s.dtype != torch.float32 or key_s.device != self.device or key_s.numel() != rows \
                or not key_s.is_contiguous() or sum(int(n) for n in N) != rows:
            raise ValueError("key_s must be a contiguous float32 [sum N] tensor")
        sk = sum(self.kept_counts(N, K)) if len(N) else 0
        dev = self.device
        out = torch.empty(sk, self.D, dtype=self.dtype, device=dev) if out is None else out
        out_idx = torch.empty(sk, dtype=torch.int32, device=dev) if out_idx is None else out_idx
        if out_src is None and want_src:
            out_src = torch.empty(sk, dtype=torch.uint8, device=dev)
        st = self.lib.tr_reduce_given_s(self._ctx, _ptr(X), _ptr(key_s), len(N), _i32(N),
                                        None if K is None else _i32(K), _ptr(out), _ptr(out_idx),
                                        _ptr(out_src), None, self._stream(stream))
        _check(st, "tr_reduce_given_s")
        return ReduceResult(out, out_idx, out_src, None, None)

    def reduce_project(self, X: torch.Tensor, Xpre: Optional[torch.Tensor], Xpost: Optional[torch.Tensor],
                       N: Sequence[int], K: Optional[Sequence[int]], W: torch.Tensor, *, out=None,
                       out_idx=None, out_src=None, want_src: bool = True, stream=None) -> ReduceResult:
        """The module with its gather replaced by the projection X[kept] . W^T (W [Nout, D])."""
        self._check_rows("X", X, self.D)
        self._check_mat("W", W, self.D)
        if (Xpre is None) != (Xpost is None):
            raise ValueError("Xpre and Xpost must both be given or both be None")
        if Xpre is not None:
            self._check_rows("Xpre", Xpre, self.Dc)
            self._check_rows("Xpost", Xpost, self.Dc)
        sk = sum(self.kept_counts(N, K)) if len(N) else 0
        dev, nout = self.device, W.shape[0]
        out = torch.empty(sk, nout, dtype=torch.bfloat16, device=dev) if out is None else out
        out_idx = torch.empty(sk, dtype=torch.int32, device=dev) if out_idx is None else out_idx
        if out_src is None and want_src:
            out_src = torch.empty(sk, dtype=torch.uint8, device=dev)
        st = self.lib.tr_reduce_project(self._ctx, _ptr(X), _ptr(Xpre), _ptr(Xpost), len(N), _i32(N),
                                        None if K is None else _i32(K), _ptr(W), W.stride(0), nout,
                                        _ptr(out), _ptr(out_idx), _ptr(out_src), self._stream(stream))
        _check(st, "tr_reduce_project")
        return ReduceResult(out, out_idx, out_src, None, None)

    def score(self, X: Optional[torch.Tensor], Xpre: Optional[torch.Tensor],
              Xpost: Optional[torch.Tensor], *, want_h2: bool = False, out=None, stream=None):
        """Scoring kernel alone: (CV^2 key, s, H2), float32 [rows] each.

        X = None skips the Stage I key (CV^2 and H2 come back None); Xpre =
        Xpost = None skips s.  ``out`` may pass preallocated (CV^2, s)
        tensors (None for a skipped one).
        """
        if X is None and Xpre is None:
            raise ValueError("nothing to score")
        if (Xpre is None) != (Xpost is None):
            raise ValueError("Xpre and Xpost must both be given or both be None")
        rows = None
        for name, t, width in (("X", X, self.D), ("Xpre", Xpre, self.Dc), ("Xpost", Xpost, self.Dc)):
            if t is None:
                continue
            self._check_rows(name, t, width)
            if rows is None:
                rows = t.shape[0]
            elif t.shape[0] != rows:
                raise ValueError("X, Xpre and Xpost must have the same number of rows")
        f32 = dict(dtype=torch.float32, device=self.device)
        if out is not None:
            cv2, s = out
        else:
            cv2 = torch.empty(rows, **f32) if X is not None else None
            s = torch.empty(rows, **f32) if Xpre is not None else None
        for t, given in ((cv2, X), (s, Xpre)):
            if (t is None) != (given is None):
                raise ValueError("score outputs must match the inputs given")
            if t is not None and (t.dtype != torch.float32 or t.device != self.device or t.dim() != 1
                                  or t.numel() != rows or not t.is_contiguous()):
                raise ValueError("score outputs must be contiguous float32 [rows] tensors")
        h2 = torch.empty(rows, **f32) if want_h2 and X is not None else None
        st = self.lib.tr_score(self._ctx, _ptr(X), _ptr(Xpre), _ptr(Xpost), rows, _ptr(cv2),
                               _ptr(s), _ptr(h2), self._stream(stream))
        _check(st, "tr_score")
        return cv2, s, h2

    def select(self, key_imp: torch.Tensor, key_s: torch.Tensor, N: Sequence[int],
               K: Optional[Sequence[int]] = None, *, want_src: bool = True, stream=None):
        """Algorithm 1 selection from given fp32 keys (Stage I key: smaller first)."""
        for name, t in (("key_imp", key_imp), ("key_s", key_s)):
            if t.device != self.device or t.dtype != torch.float32 or t.dim() != 1 \
                    or not t.is_contiguous() or t.numel() != sum(int(n) for n in N):
                raise ValueError("%s must be a contiguous float32 [sum N] tensor on %s"
                                 % (name, self.device))
        sk = sum(self.kept_counts(N, K)) if len(N) else 0
        idx = torch.empty(sk, dtype=torch.int32, device=self.device)
        src = torch.empty(sk, dtype=torch.uint8, device=self.device) if want_src else None
        st = self.lib.tr_select(self._ctx, _ptr(key_imp), _ptr(key_s), len(N), _i32(N),
                                None if K is None else _i32(K), _ptr(idx), _ptr(src),
                                self._stream(stream))
        _check(st, "tr_select")
        return idx, src

    # -- measurement --------------------------------------------------------
    def nonfinite_rows(self, reset: bool = False, stream=None) -> int:
        """The context's count of scored rows holding a NaN or infinite element
        (a context created with check_finite=True); waits for the stream."""
        out = torch.zeros(1, dtype=torch.int32, device=self.device)
        _check(self.lib.tr_nonfinite_rows(self._ctx, _ptr(out), 1 if reset else 0, self._stream(stream)),
               "tr_nonfinite_rows")
        return int(out.item())

    def timing(self, enable: bool = True):
        _check(self.lib.tr_timing_enable(self._ctx, 1 if enable else 0), "tr_timing_enable")

    def timing_read(self):
        """(ms per stage [score, select, gather] summed over calls, calls)."""
        ms = (ctypes.c_double * 3)()
        calls = ctypes.c_int64()
        _check(self.lib.tr_timing_read(self._ctx, ms, ctypes.byref(calls)), "tr_timing_read")
        return list(ms), int(calls.value)

    def close(self):
        if getattr(self, "_ctx", None):
            self.lib.tr_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def capacity_N_on(device) -> int:
    with torch.cuda.device(device):
        return capacity_N()
