"""Thin ctypes binding of ``librelaxkv.so`` (the C ABI in include/relaxkv.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  PyTorch supplies device memory (tensors) and streams.  There is
no fallback: if the library is missing or a call fails, an exception is raised.
"""

from __future__ import annotations

import ctypes
import math
import os
from ctypes import (POINTER, Structure, c_char_p, c_double, c_float, c_int32, c_int64,
                    c_size_t, c_void_p)

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librelaxkv.so")

OK, EINVAL, ENOSPACE, EUNSUPPORTED, EDEVICE = 0, -1, -2, -3, -4
ERR_NAN_SCORE, ERR_BAD_TARGETS, ERR_ROWS = 1, 2, 4      # bits of the device error word
DTYPE_F32, DTYPE_BF16 = 0, 1
CONTEXT_UNION, CONTEXT_FULL = 0, 1
CONTEXT_SETS_UNION, CONTEXT_SETS_GLOBAL, CONTEXT_SETS_LAYERWISE = 0, 1, 2

EXPORTS = ("relaxkv_status_string", "relaxkv_anchor_count", "relaxkv_validate",
           "relaxkv_score_workspace_bytes", "relaxkv_sets_bytes", "relaxkv_sets_bind",
           "relaxkv_score", "relaxkv_select", "relaxkv_build_sets", "relaxkv_build_sets_context",
           "relaxkv_select_global",
           "relaxkv_build_sets_global", "relaxkv_sparse_attn", "relaxkv_update_cache",
           "relaxkv_query_attn_workspace_bytes", "relaxkv_query_attn",
           "relaxkv_query_attn_noalloc", "relaxkv_counts_to_host")
QUERY_ATTN_NOALLOC_MAX_BYTES = 32 << 20


class RelaxKVError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {_status_text(status)} ({status})")


class Problem(Structure):
    _fields_ = [("L", c_int32), ("T_c", c_int32), ("n_query", c_int32), ("H", c_int32),
                ("H_kv", c_int32), ("d", c_int32), ("dtype", c_int32),
                ("softmax_scale", c_float), ("anchor_ratio", c_double),
                ("q", c_void_p), ("k_cache", c_void_p), ("v_cache", c_void_p),
                ("q_lse", c_void_p), ("kv_stride_layer", c_int64), ("kv_stride_head", c_int64),
                ("kv_stride_token", c_int64)]


class Sets(Structure):
    _fields_ = [("L", c_int32), ("T_c", c_int32), ("k", c_int32),
                ("anchors", c_void_p), ("h", c_void_p), ("U", c_void_p), ("cidx", c_void_p),
                ("R_off", c_void_p), ("R_idx", c_void_p), ("R_u", c_void_p),
                ("src", c_void_p), ("rank", c_void_p), ("counts", c_void_p),
                ("edges", c_void_p), ("ctx", c_void_p), ("g", c_void_p), ("tiles", c_void_p),
                ("global_targets", c_int32), ("context_sets", c_int32)]


_lib = None


def load(path=None):
    """Load the library (once).  Raises if it has not been built, or if the
    in-tree library was not built from the sources in the tree (its build
    record, written by ``build.py``, must match them)."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or _LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2609_33503_amd.build`")
    if path is None:
        from . import build
        build.verify(p)
    lib = ctypes.CDLL(p)
    lib.relaxkv_status_string.restype = c_char_p
    lib.relaxkv_status_string.argtypes = [c_int32]
    lib.relaxkv_anchor_count.restype = c_int32
    lib.relaxkv_anchor_count.argtypes = [c_double, c_int32]
    lib.relaxkv_validate.restype = c_int32
    lib.relaxkv_validate.argtypes = [POINTER(Problem)]
    lib.relaxkv_score_workspace_bytes.restype = c_size_t
    lib.relaxkv_score_workspace_bytes.argtypes = [POINTER(Problem)]
    lib.relaxkv_sets_bytes.restype = c_size_t
    lib.relaxkv_sets_bytes.argtypes = [POINTER(Problem)]
    lib.relaxkv_sets_bind.restype = c_int32
    lib.relaxkv_sets_bind.argtypes = [POINTER(Problem), c_void_p, c_size_t, POINTER(Sets)]
    lib.relaxkv_score.restype = c_int32
    lib.relaxkv_score.argtypes = [POINTER(Problem), c_void_p, c_size_t, c_void_p, c_void_p]
    lib.relaxkv_select.restype = c_int32
    lib.relaxkv_select.argtypes = [POINTER(Problem), c_void_p, POINTER(Sets), c_void_p]
    lib.relaxkv_build_sets.restype = c_int32
    lib.relaxkv_build_sets.argtypes = [POINTER(Problem), POINTER(Sets), c_void_p]
    lib.relaxkv_build_sets_context.restype = c_int32
    lib.relaxkv_build_sets_context.argtypes = [POINTER(Problem), c_void_p, c_int32, POINTER(Sets),
                                               c_void_p]
    lib.relaxkv_select_global.restype = c_int32
    lib.relaxkv_select_global.argtypes = [POINTER(Problem), c_void_p, c_double, POINTER(Sets),
                                          c_void_p, c_void_p, c_void_p, c_void_p]
    lib.relaxkv_build_sets_global.restype = c_int32
    lib.relaxkv_build_sets_global.argtypes = [POINTER(Problem), POINTER(Sets), c_void_p, c_void_p,
                                              c_void_p]
    lib.relaxkv_sparse_attn.restype = c_int32
    lib.relaxkv_sparse_attn.argtypes = [POINTER(Problem), POINTER(Sets), c_int32, c_void_p,
                                        c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                        c_int32, c_void_p]
    lib.relaxkv_update_cache.restype = c_int32
    lib.relaxkv_update_cache.argtypes = [POINTER(Problem), POINTER(Sets), c_int32, c_void_p,
                                         c_void_p, c_int32, c_void_p, c_void_p, c_void_p]
    lib.relaxkv_query_attn_workspace_bytes.restype = c_size_t
    lib.relaxkv_query_attn_workspace_bytes.argtypes = [POINTER(Problem)]
    lib.relaxkv_query_attn.restype = c_int32
    lib.relaxkv_query_attn.argtypes = [POINTER(Problem), c_int32, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.relaxkv_query_attn_noalloc.restype = c_int32
    lib.relaxkv_query_attn_noalloc.argtypes = [POINTER(Problem), c_int32, c_void_p, c_void_p,
                                               c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
    lib.relaxkv_counts_to_host.restype = c_int32
    lib.relaxkv_counts_to_host.argtypes = [POINTER(Sets), POINTER(c_int32), POINTER(c_int64),
                                           c_void_p]
    _lib = lib
    return lib


def _status_text(s):
    try:
        return load().relaxkv_status_string(s).decode()
    except Exception:  # pragma: no cover - only when the library itself is missing
        return "status"


def _check(status, what):
    if status != OK:
        raise RelaxKVError(status, what)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, name, dtype, shape, device):
    """Raise ValueError unless t is a contiguous tensor on `device` with this dtype
    and shape (None in `shape` matches any size).  Every pointer the library
    gets passes through here, so a host tensor, a tensor on another device or
    one too small never reaches a kernel."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the problem's tensors are on {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    _need_shape(t, name, shape)


def _need_shape(t, name, shape):
    if t.dim() != len(shape) or any(want is not None and got != want
                                    for got, want in zip(t.shape, shape)):
        want = tuple("*" if x is None else x for x in shape)
        raise ValueError(f"{name} must have shape {want}, got {tuple(t.shape)}")


def _need_cache(t, name, dtype, shape, device, strides=None):
    """A [L][H_kv][T_c][d] cache tensor: like _need, but any strides of the first
    three dimensions are passed on (the library checks them); d must be
    contiguous, and with `strides` given the tensor must have exactly those."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the problem's tensors are on {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    _need_shape(t, name, shape)
    if t.stride(3) != 1:
        raise ValueError(f"{name} must have contiguous rows (stride 1 in d)")
    if strides is not None and _cache_strides(t) != tuple(strides):
        raise ValueError(f"{name} must have the strides {tuple(strides)} of the request's "
                         f"cache, got {_cache_strides(t)}")


def _cache_strides(t):
    """The layer, KV-head and token strides of a cache tensor for the descriptor
    (0, the dense value, for a dimension of size 1, whose stride torch leaves
    arbitrary and the library never uses)."""
    return tuple(st if n > 1 else 0 for st, n in zip(t.stride()[:3], t.shape[:3]))


def _nbytes(t):
    return t.numel() * t.element_size()


def anchor_count(ratio, T_c):
    k = load().relaxkv_anchor_count(float(ratio), int(T_c))
    _check(OK if k > 0 else k, "relaxkv_anchor_count")
    return k


class Request:
    """One problem: the descriptor plus the tensors it points at (kept alive).

    q        [L][n_query][H][d]   bf16 or f32, CUDA, contiguous
    k_cache  [L][H_kv][T_c][d]    any strides with contiguous rows (e.g. a slice of a
                                  cache allocated for more tokens); the library checks them
    v_cache  [L][H_kv][T_c][d]    the same strides as k_cache
    q_lse    optional [L][n_query][H] f32 (natural log)
    """

    def __init__(self, q, k_cache, v_cache, anchor_ratio, softmax_scale=0.0, q_lse=None):
        lib = load()
        if not isinstance(q, torch.Tensor) or not q.is_cuda or q.dim() != 4:
            raise ValueError("q must be a [L][n_query][H][d] device tensor")
        dt = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}.get(q.dtype)
        if dt is None:
            raise ValueError("dtype must be bfloat16 or float32")
        L, Qn, H, d = q.shape
        if not isinstance(k_cache, torch.Tensor) or k_cache.dim() != 4:
            raise ValueError("k_cache must be a [L][H_kv][T_c][d] tensor")
        H_kv, T_c = k_cache.shape[1], k_cache.shape[2]
        self.device = q.device
        _need(q, "q", q.dtype, (L, Qn, H, d), self.device)
        _need_cache(k_cache, "k_cache", q.dtype, (L, H_kv, T_c, d), self.device)
        self.kv_strides = _cache_strides(k_cache)
        _need_cache(v_cache, "v_cache", q.dtype, (L, H_kv, T_c, d), self.device, self.kv_strides)
        if q_lse is not None:
            _need(q_lse, "q_lse", torch.float32, (L, Qn, H), self.device)
        self.dtype = q.dtype
        self.tensors = (q, k_cache, v_cache, q_lse)
        self.p = Problem(L, T_c, Qn, H, H_kv, d, dt, float(softmax_scale), float(anchor_ratio),
                         _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(q_lse), *self.kv_strides)
        _check(lib.relaxkv_validate(ctypes.byref(self.p)), "relaxkv_validate")
        self.L, self.T_c, self.n_query, self.H, self.H_kv, self.d = L, T_c, Qn, H, H_kv, d
        self.k = anchor_count(anchor_ratio, T_c)

    # ---- sizes and buffers (device memory comes from torch)
    def workspace_bytes(self):
        return load().relaxkv_score_workspace_bytes(ctypes.byref(self.p))

    def sets_bytes(self):
        return load().relaxkv_sets_bytes(ctypes.byref(self.p))

    def alloc_workspace(self):
        return torch.empty(self.workspace_bytes(), dtype=torch.uint8, device=self.device)

    # ---- argument checks shared by the calls
    def _scores(self, scores):
        _need(scores, "scores", torch.float32, (self.L, self.T_c), self.device)

    def _sets(self, sets):
        if not isinstance(sets, SetsBuffer) or sets.buf.device != self.device or \
                (sets.s.L, sets.s.T_c, sets.s.k) != (self.L, self.T_c, self.k):
            raise ValueError("sets must come from alloc_sets() of a request of this shape")

    def _ws(self, ws, name="ws"):
        if not isinstance(ws, torch.Tensor) or ws.device != self.device or not ws.is_contiguous():
            raise ValueError(f"{name} must be a contiguous tensor on {self.device}")

    def alloc_sets(self):
        """A device buffer for the sets and its bound descriptor."""
        nbytes = self.sets_bytes()
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = buf.data_ptr()
        pad = (-base) % 256
        s = Sets()
        _check(load().relaxkv_sets_bind(ctypes.byref(self.p), ctypes.c_void_p(base + pad),
                                        nbytes, ctypes.byref(s)), "relaxkv_sets_bind")
        return SetsBuffer(self, buf, s, pad)

    # ---- the four calls
    def score(self, ws, scores, stream=None):
        self._ws(ws)
        self._scores(scores)
        _check(load().relaxkv_score(ctypes.byref(self.p), _ptr(ws), _nbytes(ws), _ptr(scores),
                                    _stream(stream)), "relaxkv_score")

    def select(self, scores, sets, stream=None):
        self._scores(scores)
        self._sets(sets)
        _check(load().relaxkv_select(ctypes.byref(self.p), _ptr(scores), ctypes.byref(sets.s),
                                     _stream(stream)), "relaxkv_select")

    def build_sets(self, sets, stream=None):
        self._sets(sets)
        _check(load().relaxkv_build_sets(ctypes.byref(self.p), ctypes.byref(sets.s),
                                         _stream(stream)), "relaxkv_build_sets")

    def build_sets_context(self, scores, construction, sets, stream=None):
        """RelaxKV's anchors and targets with the context set replaced
        (CONTEXT_SETS_UNION / _GLOBAL / _LAYERWISE); scores [L][T_c] f32."""
        self._scores(scores)
        self._sets(sets)
        _check(load().relaxkv_build_sets_context(ctypes.byref(self.p), _ptr(scores),
                                                 int(construction), ctypes.byref(sets.s),
                                                 _stream(stream)), "relaxkv_build_sets_context")

    # ---- matched-target variants: one global target list for every layer
    def select_global(self, scores, target_ratio, sets, g, targets, n_targets, stream=None):
        """g [T_c] f32, targets [T_c] int32 and n_targets [1] int32 are outputs."""
        self._scores(scores)
        self._sets(sets)
        _need(g, "g", torch.float32, (self.T_c,), self.device)
        _need(targets, "targets", torch.int32, (self.T_c,), self.device)
        _need(n_targets, "n_targets", torch.int32, (1,), self.device)
        _check(load().relaxkv_select_global(ctypes.byref(self.p), _ptr(scores),
                                            float(target_ratio), ctypes.byref(sets.s), _ptr(g),
                                            _ptr(targets), _ptr(n_targets), _stream(stream)),
               "relaxkv_select_global")

    def build_sets_global(self, sets, targets, n_targets, stream=None):
        """targets: int32 device [T_c], ascending in its first n_targets entries;
        n_targets: int32 device [1]."""
        self._sets(sets)
        _need(targets, "targets", torch.int32, (self.T_c,), self.device)
        _need(n_targets, "n_targets", torch.int32, (1,), self.device)
        _check(load().relaxkv_build_sets_global(ctypes.byref(self.p), ctypes.byref(sets.s),
                                                _ptr(targets), _ptr(n_targets), _stream(stream)),
               "relaxkv_build_sets_global")

    def sparse_attn(self, sets, layer, q_new, k_new, v_new, out, lse_out=None,
                    context_mode=CONTEXT_UNION, stream=None):
        """q_new/out [n][H][d], k_new/v_new [n][H_kv][d], lse_out [n][H] f32, with n
        rows allocated (normally |R_l|; targets past n are not computed and set the
        device error word)."""
        self._sets(sets)
        n = q_new.shape[0] if isinstance(q_new, torch.Tensor) and q_new.dim() == 3 else -1
        _need(q_new, "q_new", self.dtype, (n, self.H, self.d), self.device)
        _need(k_new, "k_new", self.dtype, (n, self.H_kv, self.d), self.device)
        _need(v_new, "v_new", self.dtype, (n, self.H_kv, self.d), self.device)
        _need(out, "out", self.dtype, (n, self.H, self.d), self.device)
        if lse_out is not None:
            _need(lse_out, "lse_out", torch.float32, (n, self.H), self.device)
        _check(load().relaxkv_sparse_attn(ctypes.byref(self.p), ctypes.byref(sets.s), int(layer),
                                          _ptr(q_new), _ptr(k_new), _ptr(v_new), int(n),
                                          _ptr(out), _ptr(lse_out), int(context_mode),
                                          _stream(stream)),
               "relaxkv_sparse_attn")

    def update_cache(self, sets, layer, k_new, v_new, k_cache, v_cache, stream=None):
        """Fresh rows of R_l (k_new/v_new [n][H_kv][d]) into the cache
        (k_cache/v_cache: [L][H_kv][T_c][d] with the request's cache strides)."""
        self._sets(sets)
        n = k_new.shape[0] if isinstance(k_new, torch.Tensor) and k_new.dim() == 3 else -1
        _need(k_new, "k_new", self.dtype, (n, self.H_kv, self.d), self.device)
        _need(v_new, "v_new", self.dtype, (n, self.H_kv, self.d), self.device)
        cache = (self.L, self.H_kv, self.T_c, self.d)
        _need_cache(k_cache, "k_cache", self.dtype, cache, self.device, self.kv_strides)
        _need_cache(v_cache, "v_cache", self.dtype, cache, self.device, self.kv_strides)
        _check(load().relaxkv_update_cache(ctypes.byref(self.p), ctypes.byref(sets.s), int(layer),
                                           _ptr(k_new), _ptr(v_new), int(n), _ptr(k_cache),
                                           _ptr(v_cache), _stream(stream)),
               "relaxkv_update_cache")


    # ---- query-side completion (the query prefill after repair)
    def query_attn_workspace_bytes(self):
        return load().relaxkv_query_attn_workspace_bytes(ctypes.byref(self.p))

    def alloc_query_workspace(self):
        n = self.query_attn_workspace_bytes()
        return None if n == 0 else torch.empty(n, dtype=torch.uint8, device=self.device)

    def query_attn(self, layer, k_cache, v_cache, k_q, v_q, out, lse_out=None, ws=None,
                   stream=None):
        """k_cache/v_cache [L][H_kv][T_c][d] (the request's cache strides); k_q/v_q
        [n_query][H_kv][d]; out [n_query][H][d];
        lse_out [n_query][H] f32."""
        cache = (self.L, self.H_kv, self.T_c, self.d)
        _need_cache(k_cache, "k_cache", self.dtype, cache, self.device, self.kv_strides)
        _need_cache(v_cache, "v_cache", self.dtype, cache, self.device, self.kv_strides)
        _need(k_q, "k_q", self.dtype, (self.n_query, self.H_kv, self.d), self.device)
        _need(v_q, "v_q", self.dtype, (self.n_query, self.H_kv, self.d), self.device)
        _need(out, "out", self.dtype, (self.n_query, self.H, self.d), self.device)
        if lse_out is not None:
            _need(lse_out, "lse_out", torch.float32, (self.n_query, self.H), self.device)
        if ws is not None:
            self._ws(ws)
        _check(load().relaxkv_query_attn(ctypes.byref(self.p), int(layer), _ptr(k_cache),
                                         _ptr(v_cache), _ptr(k_q), _ptr(v_q), _ptr(out),
                                         _ptr(lse_out), _ptr(ws), 0 if ws is None else _nbytes(ws),
                                         _stream(stream)), "relaxkv_query_attn")


    def query_attn_noalloc(self, layer, k_cache, v_cache, k_q, v_q, out, lse_out=None,
                           stream=None):
        """query_attn through the allocation-free entry point (the library's own
        per-GPU scratch; calls that overlap on one GPU race)."""
        cache = (self.L, self.H_kv, self.T_c, self.d)
        _need_cache(k_cache, "k_cache", self.dtype, cache, self.device, self.kv_strides)
        _need_cache(v_cache, "v_cache", self.dtype, cache, self.device, self.kv_strides)
        _need(k_q, "k_q", self.dtype, (self.n_query, self.H_kv, self.d), self.device)
        _need(v_q, "v_q", self.dtype, (self.n_query, self.H_kv, self.d), self.device)
        _need(out, "out", self.dtype, (self.n_query, self.H, self.d), self.device)
        if lse_out is not None:
            _need(lse_out, "lse_out", torch.float32, (self.n_query, self.H), self.device)
        _check(load().relaxkv_query_attn_noalloc(ctypes.byref(self.p), int(layer), _ptr(k_cache),
                                                 _ptr(v_cache), _ptr(k_q), _ptr(v_q), _ptr(out),
                                                 _ptr(lse_out), _stream(stream)),
               "relaxkv_query_attn_noalloc")


class SetsBuffer:
    """Device arrays of relaxkv_sets (views into one torch buffer)."""

    def __init__(self, req, buf, s, pad):
        self.req, self.buf, self.s = req, buf, s
        L, T, k = req.L, req.T_c, req.k
        base = buf.data_ptr() + pad

        def view(ptr, n, dtype):
            off = ptr - base + pad
            esz = 8 if dtype == torch.int64 else 4
            return buf[off:off + n * esz].view(dtype)

        self.anchors = view(s.anchors, L * k, torch.int32).view(L, k)
        self.h = view(s.h, T, torch.int32)
        self.U = view(s.U, T, torch.int32)
        self.cidx = view(s.cidx, T, torch.int32)
        self.R_off = view(s.R_off, L + 1, torch.int32)
        self.R_idx = view(s.R_idx, L * T, torch.int32)
        self.R_u = view(s.R_u, L * T, torch.int32)
        self.src = view(s.src, L * T, torch.int32).view(L, T)
        self.rank = view(s.rank, L * T, torch.int32).view(L, T)
        self.counts = view(s.counts, L + 2, torch.int32)
        self.edges = view(s.edges, 2 * L, torch.int64)
        self.ctx = view(s.ctx, L * T, torch.int32).view(L, T)
        self.g = view(s.g, T, torch.float32)
        self.tiles = view(s.tiles, 2 * L * (req.H_kv + 1), torch.int32).view(2, L, req.H_kv + 1)

    def counts_to_host(self, stream=None, check=True):
        """(counts [L+2], edges [2L]) on the host; synchronises the stream.  With
        check=True a set device error word (counts[L+1], ERR_* bits) raises
        RelaxKVError; with check=False the counts are returned as they are."""
        L = self.req.L
        c = (c_int32 * (L + 2))()
        e = (c_int64 * (2 * L))()
        st = load().relaxkv_counts_to_host(ctypes.byref(self.s), c, e, _stream(stream))
        if check or st not in (OK, EINVAL):
            _check(st, "relaxkv_counts_to_host")
        return list(c), list(e)


def default_scale(d):
    return 1.0 / math.sqrt(d)
