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
DTYPE_F32, DTYPE_BF16 = 0, 1
CONTEXT_UNION, CONTEXT_FULL = 0, 1
CONTEXT_SETS_UNION, CONTEXT_SETS_GLOBAL, CONTEXT_SETS_LAYERWISE = 0, 1, 2

EXPORTS = ("relaxkv_status_string", "relaxkv_anchor_count", "relaxkv_validate",
           "relaxkv_score_workspace_bytes", "relaxkv_sets_bytes", "relaxkv_sets_bind",
           "relaxkv_score", "relaxkv_select", "relaxkv_build_sets", "relaxkv_build_sets_context",
           "relaxkv_select_global",
           "relaxkv_build_sets_global", "relaxkv_sparse_attn", "relaxkv_update_cache",
           "relaxkv_query_attn_workspace_bytes", "relaxkv_query_attn", "relaxkv_counts_to_host")


class RelaxKVError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {_status_text(status)} ({status})")


class Problem(Structure):
    _fields_ = [("L", c_int32), ("T_c", c_int32), ("n_query", c_int32), ("H", c_int32),
                ("H_kv", c_int32), ("d", c_int32), ("dtype", c_int32),
                ("softmax_scale", c_float), ("anchor_ratio", c_double),
                ("q", c_void_p), ("k_cache", c_void_p), ("v_cache", c_void_p),
                ("q_lse", c_void_p)]


class Sets(Structure):
    _fields_ = [("L", c_int32), ("T_c", c_int32), ("k", c_int32),
                ("anchors", c_void_p), ("h", c_void_p), ("U", c_void_p), ("cidx", c_void_p),
                ("R_off", c_void_p), ("R_idx", c_void_p), ("R_u", c_void_p),
                ("src", c_void_p), ("rank", c_void_p), ("counts", c_void_p),
                ("edges", c_void_p), ("ctx", c_void_p), ("g", c_void_p),
                ("global_targets", c_int32), ("context_sets", c_int32)]


_lib = None


def load(path=None):
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or _LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2609_33503_amd.build`")
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
                                        c_void_p, c_void_p, c_void_p, c_void_p, c_int32,
                                        c_void_p]
    lib.relaxkv_update_cache.restype = c_int32
    lib.relaxkv_update_cache.argtypes = [POINTER(Problem), POINTER(Sets), c_int32, c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_void_p]
    lib.relaxkv_query_attn_workspace_bytes.restype = c_size_t
    lib.relaxkv_query_attn_workspace_bytes.argtypes = [POINTER(Problem)]
    lib.relaxkv_query_attn.restype = c_int32
    lib.relaxkv_query_attn.argtypes = [POINTER(Problem), c_int32, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
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


def anchor_count(ratio, T_c):
    k = load().relaxkv_anchor_count(float(ratio), int(T_c))
    _check(OK if k > 0 else k, "relaxkv_anchor_count")
    return k


class Request:
    """One problem: the descriptor plus the tensors it points at (kept alive).

    q        [L][n_query][H][d]   bf16 or f32, CUDA, contiguous
    k_cache  [L][H_kv][T_c][d]
    v_cache  [L][H_kv][T_c][d]
    q_lse    optional [L][n_query][H] f32 (natural log)
    """

    def __init__(self, q, k_cache, v_cache, anchor_ratio, softmax_scale=0.0, q_lse=None):
        lib = load()
        for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache)):
            if not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous device tensor")
        if q.dtype != k_cache.dtype or v_cache.dtype != k_cache.dtype:
            raise ValueError("q, k_cache and v_cache must share a dtype")
        if q_lse is not None and (q_lse.dtype != torch.float32 or not q_lse.is_contiguous()):
            raise ValueError("q_lse must be contiguous float32")
        L, Qn, H, d = q.shape
        _, H_kv, T_c, d2 = k_cache.shape
        if k_cache.shape[0] != L or d2 != d or tuple(v_cache.shape) != tuple(k_cache.shape):
            raise ValueError("inconsistent shapes")
        dt = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}.get(q.dtype)
        if dt is None:
            raise ValueError("dtype must be bfloat16 or float32")
        self.dtype = q.dtype
        self.tensors = (q, k_cache, v_cache, q_lse)
        self.p = Problem(L, T_c, Qn, H, H_kv, d, dt, float(softmax_scale), float(anchor_ratio),
                         _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(q_lse))
        _check(lib.relaxkv_validate(ctypes.byref(self.p)), "relaxkv_validate")
        self.L, self.T_c, self.n_query, self.H, self.H_kv, self.d = L, T_c, Qn, H, H_kv, d
        self.k = anchor_count(anchor_ratio, T_c)

    # ---- sizes and buffers (device memory comes from torch)
    def workspace_bytes(self):
        return load().relaxkv_score_workspace_bytes(ctypes.byref(self.p))

    def sets_bytes(self):
        return load().relaxkv_sets_bytes(ctypes.byref(self.p))

    def alloc_workspace(self):
        return torch.empty(self.workspace_bytes(), dtype=torch.uint8,
                           device=self.tensors[1].device)

    def alloc_sets(self):
        """A device buffer for the sets and its bound descriptor."""
        nbytes = self.sets_bytes()
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.tensors[1].device)
        base = buf.data_ptr()
        pad = (-base) % 256
        s = Sets()
        _check(load().relaxkv_sets_bind(ctypes.byref(self.p), ctypes.c_void_p(base + pad),
                                        nbytes, ctypes.byref(s)), "relaxkv_sets_bind")
        return SetsBuffer(self, buf, s, pad)

    # ---- the four calls
    def score(self, ws, scores, stream=None):
        _check(load().relaxkv_score(ctypes.byref(self.p), _ptr(ws), ws.numel(), _ptr(scores),
                                    _stream(stream)), "relaxkv_score")

    def select(self, scores, sets, stream=None):
        _check(load().relaxkv_select(ctypes.byref(self.p), _ptr(scores), ctypes.byref(sets.s),
                                     _stream(stream)), "relaxkv_select")

    def build_sets(self, sets, stream=None):
        _check(load().relaxkv_build_sets(ctypes.byref(self.p), ctypes.byref(sets.s),
                                         _stream(stream)), "relaxkv_build_sets")

    def build_sets_context(self, scores, construction, sets, stream=None):
        """RelaxKV's anchors and targets with the context set replaced
        (CONTEXT_SETS_UNION / _GLOBAL / _LAYERWISE); scores [L][T_c] f32."""
        _check(load().relaxkv_build_sets_context(ctypes.byref(self.p), _ptr(scores),
                                                 int(construction), ctypes.byref(sets.s),
                                                 _stream(stream)), "relaxkv_build_sets_context")

    # ---- matched-target variants: one global target list for every layer
    def select_global(self, scores, target_ratio, sets, g, targets, n_targets, stream=None):
        """g [T_c] f32, targets [T_c] int32 and n_targets [1] int32 are outputs."""
        for t, dt, n in ((g, torch.float32, self.T_c), (targets, torch.int32, self.T_c),
                         (n_targets, torch.int32, 1)):
            if t.dtype != dt or not t.is_contiguous() or t.numel() < n:
                raise ValueError("select_global outputs: g f32 [T_c], targets int32 [T_c], "
                                 "n_targets int32 [1]")
        _check(load().relaxkv_select_global(ctypes.byref(self.p), _ptr(scores),
                                            float(target_ratio), ctypes.byref(sets.s), _ptr(g),
                                            _ptr(targets), _ptr(n_targets), _stream(stream)),
               "relaxkv_select_global")

    def build_sets_global(self, sets, targets, n_targets, stream=None):
        """targets: int32 device, ascending; n_targets: int32 device [1]."""
        for t in (targets, n_targets):
            if t.dtype != torch.int32 or not t.is_contiguous() or not t.is_cuda:
                raise ValueError("targets and n_targets must be contiguous int32 device tensors")
        _check(load().relaxkv_build_sets_global(ctypes.byref(self.p), ctypes.byref(sets.s),
                                                _ptr(targets), _ptr(n_targets), _stream(stream)),
               "relaxkv_build_sets_global")

    def sparse_attn(self, sets, layer, q_new, k_new, v_new, out, lse_out=None,
                    context_mode=CONTEXT_UNION, stream=None):
        for t in (q_new, k_new, v_new, out):
            if not t.is_contiguous() or t.dtype != self.dtype:
                raise ValueError("fresh rows and out must be contiguous, in the problem dtype")
        _check(load().relaxkv_sparse_attn(ctypes.byref(self.p), ctypes.byref(sets.s), int(layer),
                                          _ptr(q_new), _ptr(k_new), _ptr(v_new), _ptr(out),
                                          _ptr(lse_out), int(context_mode), _stream(stream)),
               "relaxkv_sparse_attn")


    def update_cache(self, sets, layer, k_new, v_new, k_cache, v_cache, stream=None):
        """Fresh rows of R_l into the cache (k_cache/v_cache: [L][H_kv][T_c][d])."""
        for t in (k_new, v_new, k_cache, v_cache):
            if not t.is_contiguous() or t.dtype != self.dtype:
                raise ValueError("rows and caches must be contiguous, in the problem dtype")
        if tuple(k_cache.shape) != tuple(self.tensors[1].shape) or \
                tuple(v_cache.shape) != tuple(self.tensors[2].shape):
            raise ValueError("caches must have the problem's cache shape")
        _check(load().relaxkv_update_cache(ctypes.byref(self.p), ctypes.byref(sets.s), int(layer),
                                           _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                           _ptr(v_cache), _stream(stream)),
               "relaxkv_update_cache")


    # ---- query-side completion (the query prefill after repair)
    def query_attn_workspace_bytes(self):
        return load().relaxkv_query_attn_workspace_bytes(ctypes.byref(self.p))

    def alloc_query_workspace(self):
        n = self.query_attn_workspace_bytes()
        return None if n == 0 else torch.empty(n, dtype=torch.uint8, device=self.tensors[1].device)

    def query_attn(self, layer, k_cache, v_cache, k_q, v_q, out, lse_out=None, ws=None,
                   stream=None):
        """k_cache/v_cache [L][H_kv][T_c][d]; k_q/v_q [n_query][H_kv][d]; out [n_query][H][d]."""
        for t in (k_cache, v_cache, k_q, v_q, out):
            if not t.is_contiguous() or t.dtype != self.dtype:
                raise ValueError("caches, query keys/values and out must be contiguous, "
                                 "in the problem dtype")
        _check(load().relaxkv_query_attn(ctypes.byref(self.p), int(layer), _ptr(k_cache),
                                         _ptr(v_cache), _ptr(k_q), _ptr(v_q), _ptr(out),
                                         _ptr(lse_out), _ptr(ws), 0 if ws is None else ws.numel(),
                                         _stream(stream)), "relaxkv_query_attn")


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

    def counts_to_host(self, stream=None):
        """(counts [L+2], edges [2L]) on the host; synchronises the stream."""
        L = self.req.L
        c = (c_int32 * (L + 2))()
        e = (c_int64 * (2 * L))()
        st = load().relaxkv_counts_to_host(ctypes.byref(self.s), c, e, _stream(stream))
        _check(st, "relaxkv_counts_to_host")
        return list(c), list(e)


def default_scale(d):
    return 1.0 / math.sqrt(d)
