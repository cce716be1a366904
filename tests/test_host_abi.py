"""Host-side checks of the C ABI (no GPU): the library loads and exports every
symbol include/relaxkv.h declares; argument validation, anchor budget, and
buffer sizing/carving behave as documented.  No call here reaches a kernel:
every call either fails validation before anything is enqueued or is a
host-only function."""

import ctypes
import os
import re
import subprocess

import pytest

from oracle import anchor_count as oracle_anchor_count

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "relaxkv.h")


def _declared():
    txt = open(HEADER).read()
    decl = r"^(?:const char\*|int32_t|size_t|relaxkv_status)\s+(relaxkv_[a-z_]+)\("
    return sorted(set(re.findall(decl, txt, re.M)))


def test_exports_match_header(rk):
    declared = _declared()
    assert set(declared) == set(rk.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", rk._LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (relaxkv_[a-z_]+)$", out, re.M))
    assert exported == set(declared)
    lib = rk.load()
    for name in declared:
        assert hasattr(lib, name)


def test_status_strings(rk):
    lib = rk.load()
    for s in (0, -1, -2, -3, -4):
        assert lib.relaxkv_status_string(s).decode()
    assert lib.relaxkv_status_string(12345) == b"unknown status"


@pytest.mark.parametrize("r,T", [(0.15, 1024), (0.15, 8192), (0.05, 16384), (0.15, 16384),
                                 (0.30, 16384), (0.15, 32768), (0.125, 20), (0.375, 4),
                                 (0.625, 4), (0.5, 1), (0.0, 50), (1.0, 77), (0.5, 3),
                                 (0.3, 5), (1e-9, 10), (0.999999, 1000)])
def test_anchor_count_matches_oracle(rk, r, T):
    assert rk.load().relaxkv_anchor_count(r, T) == oracle_anchor_count(r, T)


@pytest.mark.parametrize("r,T", [(-0.1, 10), (1.5, 10), (float("nan"), 10), (float("inf"), 10),
                                 (0.2, 0), (0.2, -5)])
def test_anchor_count_rejects(rk, r, T):
    assert rk.load().relaxkv_anchor_count(r, T) == rk.EINVAL


def _problem(rk, **kw):
    base = dict(L=4, T_c=2048, n_query=16, H=8, H_kv=2, d=128, dtype=rk.DTYPE_BF16,
                softmax_scale=0.0, anchor_ratio=0.15, q=0x1000, k_cache=0x2000, v_cache=0x3000,
                q_lse=None, sL=0, sH=0, sT=0)
    base.update(kw)
    return rk.Problem(base["L"], base["T_c"], base["n_query"], base["H"], base["H_kv"],
                      base["d"], base["dtype"], base["softmax_scale"], base["anchor_ratio"],
                      base["q"], base["k_cache"], base["v_cache"], base["q_lse"],
                      base["sL"], base["sH"], base["sT"])


@pytest.mark.parametrize("kw,status", [
    ({}, 0),
    ({"L": 0}, -1), ({"T_c": 0}, -1), ({"n_query": 0}, -1), ({"H": 6, "H_kv": 4}, -1),
    ({"H_kv": 0}, -1), ({"L": 1025}, -1), ({"T_c": (1 << 22) + 1}, -1),
    ({"q": None}, -1), ({"k_cache": None}, -1), ({"v_cache": None}, -1),
    ({"anchor_ratio": -0.5}, -1), ({"anchor_ratio": float("nan")}, -1),
    ({"softmax_scale": float("nan")}, -1), ({"softmax_scale": float("inf")}, -1),
    ({"d": 96}, -3), ({"d": 256}, -3), ({"dtype": 7}, -3),
    ({"H": 512, "H_kv": 1}, -3),                      # a GQA group wider than the bf16 tile
    ({"H": 512, "H_kv": 1, "dtype": 0}, 0),           # fp32 kernels have no such limit
    ({"d": 64, "dtype": 0}, 0),
    # one layer's bf16 cache slab must stay below 2^31 elements (32-bit row offsets)
    ({"L": 1, "T_c": 1 << 21, "H": 8, "H_kv": 8}, -3),
    ({"L": 1, "T_c": (1 << 21) - 1, "H": 8, "H_kv": 8}, 0),
    ({"L": 1, "T_c": 1 << 21, "H": 8, "H_kv": 8, "dtype": 0}, 0),
])
def test_validate(rk, kw, status):
    p = _problem(rk, **kw)
    assert rk.load().relaxkv_validate(ctypes.byref(p)) == status


# The cache strides (base problem: L 4, H_kv 2, T_c 2048, d 128; dense strides
# 524288, 262144, 128).  0 is the dense value; rows may not overlap; rows and
# pointers 16-byte aligned; bf16 token strides below 2^24 with (T_c - 1) * stride
# + d < 2^31.
@pytest.mark.parametrize("kw,status", [
    ({"sL": 524288, "sH": 262144, "sT": 128}, 0),               # the dense values spelled out
    ({"sH": 2100 * 128}, 0),                                    # room for 2100 tokens per head
    ({"sH": 2100 * 128, "sL": 2 * 2100 * 128 + 64}, 0),         # and padding between layers
    ({"sT": 2 * 128, "sH": 128, "sL": 2048 * 256}, 0),          # [L][T_c][H_kv][d]
    ({"sT": 2 * 128}, 0),                                       # every other row (K/V interleaved)
    ({"sL": 128, "sH": 4 * 128, "sT": 8 * 128}, 0),             # [T_c][H_kv][L][d]
    ({"sT": 64}, -1),                                           # rows overlap
    ({"sH": 2047 * 128}, -1),                                   # heads overlap
    ({"sH": 2048 * 128 + 64, "sL": 2 * 2048 * 128}, -1),        # layers overlap
    ({"sT": 128, "sH": 128, "sL": 2048 * 256}, -1),             # two strides alike
    ({"sL": -1}, -1), ({"sH": -128}, -1), ({"sT": -128}, -1),
    ({"sT": 132}, -3),                                          # rows not 16-byte aligned
    ({"sT": 132, "dtype": 0}, 0),                               # 528 bytes: aligned in fp32
    ({"sH": 2048 * 128 + 4}, -3),
    ({"k_cache": 0x2008}, -3), ({"v_cache": 0x3004}, -3), ({"q": 0x1002}, -3),
    ({"L": 1, "T_c": 2, "sT": 1 << 24}, -3),                    # bf16: 24-bit token offsets
    ({"L": 1, "T_c": 2, "sT": 1 << 24, "dtype": 0}, 0),
    ({"L": 1, "T_c": 1 << 14, "sT": (1 << 17) + 8}, -3),        # (T_c - 1) * stride + d >= 2^31
    ({"L": 1, "T_c": 1 << 14, "sT": 1 << 17}, 0),               # 2^31 - 2^17 + 128
    ({"L": 1, "H_kv": 1, "H": 1, "sH": 8}, 0),                  # a dimension of size 1 is free
    ({"L": 1, "sL": 3}, 0),                                     # even unaligned
    ({"L": 1, "T_c": 1, "sT": (1 << 24) + 8}, 0),               # one token: its stride is unused
    ({"L": 2, "sL": 1 << 40}, 0),                               # far apart is fine
    ({"L": 2, "sL": 1 << 48}, -3),                              # but not past 2^48 elements
    ({"L": 3, "sL": 1 << 62}, -3),                              # nor past int64
    ({"sT": 1 << 62}, -3),                                      # dense head stride T_c * 2^62
    ({"sH": 1 << 62}, -3),                                      # dense layer stride H_kv * 2^62
])
def test_validate_cache_strides(rk, kw, status):
    p = _problem(rk, **kw)
    lib = rk.load()
    assert lib.relaxkv_validate(ctypes.byref(p)) == status
    if status != 0:
        assert lib.relaxkv_sets_bytes(ctypes.byref(p)) == 0


@pytest.mark.parametrize("kw,n_split", [
    # one round of 256 workgroups: 256 / H_kv splits of at least 256 keys (at 32K, 40q/8kv:
    # 32 splits of 1024 keys, which have a merge kernel of their own; the GPU test shapes
    # "splits32" and "many-splits" take 32 and 34)
    (dict(T_c=32768, H=40, H_kv=8, n_query=64), 32),
    (dict(T_c=8500, H=4, H_kv=2, n_query=8), 34),
    (dict(T_c=8192, H=32, H_kv=8, n_query=8), 32),
    (dict(T_c=1040, H=40, H_kv=8, n_query=64), 5),     # the last split holds 16 keys
    (dict(T_c=1500, H=32, H_kv=8, n_query=64), 6),
])
def test_query_workspace_split_count(rk, kw, n_split):
    p = _problem(rk, L=1, **kw)
    G = kw["H"] // kw["H_kv"]
    rows_pad = (kw["n_query"] * G + 31) // 32 * 32
    rows = n_split * kw["H_kv"] * rows_pad
    al = lambda x: (x + 255) // 256 * 256          # noqa: E731
    assert rk.load().relaxkv_query_attn_workspace_bytes(ctypes.byref(p)) == \
        al(rows * 128 * 2) + al(rows * 4)


def test_validate_null(rk):
    assert rk.load().relaxkv_validate(None) == rk.EINVAL


def test_sizes(rk):
    lib = rk.load()
    p = _problem(rk)
    ws = lib.relaxkv_score_workspace_bytes(ctypes.byref(p))
    sb = lib.relaxkv_sets_bytes(ctypes.byref(p))
    L, T, k = 4, 2048, oracle_anchor_count(0.15, 2048)
    assert ws >= L * 2 * T * 4                      # per-KV-head partial sums
    assert sb >= 4 * (L * k + 3 * T + (L + 1) + 4 * L * T + (L + 2)) + 8 * 2 * L
    assert sb % 256 == 0 and ws % 256 == 0
    bad = _problem(rk, d=96)
    assert lib.relaxkv_score_workspace_bytes(ctypes.byref(bad)) == 0
    assert lib.relaxkv_sets_bytes(ctypes.byref(bad)) == 0


def test_sets_bind_carves_buffer(rk):
    lib = rk.load()
    p = _problem(rk)
    nbytes = lib.relaxkv_sets_bytes(ctypes.byref(p))
    base = 0x7f0000000000                            # never dereferenced: host-only arithmetic
    s = rk.Sets()
    assert lib.relaxkv_sets_bind(ctypes.byref(p), ctypes.c_void_p(base), nbytes,
                                 ctypes.byref(s)) == 0
    assert (s.L, s.T_c, s.k) == (4, 2048, oracle_anchor_count(0.15, 2048))
    ptrs = [s.anchors, s.h, s.U, s.cidx, s.R_off, s.R_idx, s.R_u, s.src, s.rank, s.counts,
            s.edges, s.ctx, s.g, s.tiles]
    assert ptrs[0] == base and ptrs == sorted(ptrs)
    assert all(x % 256 == 0 for x in ptrs)
    L, T, k = s.L, s.T_c, s.k
    sizes = [L * k * 4, T * 4, T * 4, T * 4, (L + 1) * 4, L * T * 4, L * T * 4, L * T * 4,
             L * T * 4, (L + 2) * 4, 2 * L * 8, L * T * 4, T * 4, 2 * L * (p.H_kv + 1) * 4]
    for a, b, n in zip(ptrs, ptrs[1:] + [base + nbytes], sizes):
        assert b - a >= n
    assert lib.relaxkv_sets_bind(ctypes.byref(p), ctypes.c_void_p(base), nbytes - 1,
                                 ctypes.byref(s)) == rk.ENOSPACE
    assert lib.relaxkv_sets_bind(ctypes.byref(p), ctypes.c_void_p(base + 4), nbytes,
                                 ctypes.byref(s)) == rk.EINVAL
    assert lib.relaxkv_sets_bind(ctypes.byref(p), None, nbytes, ctypes.byref(s)) == rk.EINVAL


def _bound_sets(rk, p):
    lib = rk.load()
    s = rk.Sets()
    nbytes = lib.relaxkv_sets_bytes(ctypes.byref(p))
    assert lib.relaxkv_sets_bind(ctypes.byref(p), ctypes.c_void_p(0x7f0000000000), nbytes,
                                 ctypes.byref(s)) == 0
    return s


def test_compute_calls_reject_before_launch(rk):
    lib = rk.load()
    p = _problem(rk)
    s = _bound_sets(rk, p)
    fake = ctypes.c_void_p(0x7e0000000000)
    ws = lib.relaxkv_score_workspace_bytes(ctypes.byref(p))
    bp = _problem(rk, H=6, H_kv=4)
    # score
    assert lib.relaxkv_score(ctypes.byref(p), None, ws, fake, None) == rk.EINVAL
    assert lib.relaxkv_score(ctypes.byref(p), fake, ws, None, None) == rk.EINVAL
    assert lib.relaxkv_score(ctypes.byref(p), fake, ws - 1, fake, None) == rk.ENOSPACE
    assert lib.relaxkv_score(ctypes.byref(bp), fake, ws, fake, None) == rk.EINVAL
    # select / build_sets: sets bound for another problem are refused
    other = _problem(rk, T_c=4096)
    assert lib.relaxkv_select(ctypes.byref(other), fake, ctypes.byref(s), None) == rk.EINVAL
    assert lib.relaxkv_select(ctypes.byref(p), None, ctypes.byref(s), None) == rk.EINVAL
    assert lib.relaxkv_select(ctypes.byref(p), fake, None, None) == rk.EINVAL
    assert lib.relaxkv_build_sets(ctypes.byref(other), ctypes.byref(s), None) == rk.EINVAL
    s2 = _bound_sets(rk, p)
    s2.src = None
    assert lib.relaxkv_build_sets(ctypes.byref(p), ctypes.byref(s2), None) == rk.EINVAL
    # sparse_attn: (q_new, k_new, v_new, n_rows, out, lse_out, context_mode, stream)
    args = (fake, fake, fake, 100, fake, None)
    for layer in (-1, 4):
        assert lib.relaxkv_sparse_attn(ctypes.byref(p), ctypes.byref(s), layer, *args, 0,
                                       None) == rk.EINVAL
    assert lib.relaxkv_sparse_attn(ctypes.byref(p), ctypes.byref(s), 0, *args, 2,
                                   None) == rk.EINVAL
    assert lib.relaxkv_sparse_attn(ctypes.byref(p), ctypes.byref(s), 0, None, fake, fake, 100,
                                   fake, None, 0, None) == rk.EINVAL
    assert lib.relaxkv_sparse_attn(ctypes.byref(p), ctypes.byref(s), 0, fake, fake, fake, -1,
                                   fake, None, 0, None) == rk.EINVAL
    assert lib.relaxkv_sparse_attn(ctypes.byref(_problem(rk, d=96)), ctypes.byref(s), 0, *args,
                                   0, None) == rk.EUNSUPPORTED
    # update_cache: (k_new, v_new, n_rows, k_cache, v_cache, stream)
    for layer in (-1, 4):
        assert lib.relaxkv_update_cache(ctypes.byref(p), ctypes.byref(s), layer, fake, fake, 100,
                                        fake, fake, None) == rk.EINVAL
    assert lib.relaxkv_update_cache(ctypes.byref(p), ctypes.byref(s), 0, fake, fake, 100, None,
                                    fake, None) == rk.EINVAL
    assert lib.relaxkv_update_cache(ctypes.byref(p), ctypes.byref(s), 0, fake, fake, -1, fake,
                                    fake, None) == rk.EINVAL
    assert lib.relaxkv_update_cache(ctypes.byref(other), ctypes.byref(s), 0, fake, fake, 100,
                                    fake, fake, None) == rk.EINVAL
    # select_global / build_sets_global (matched-target variants)
    sg = lib.relaxkv_select_global
    for r in (-0.1, 1.5, float("nan"), float("inf")):
        assert sg(ctypes.byref(p), fake, r, ctypes.byref(s), fake, fake, fake, None) == rk.EINVAL
    for i in range(4):
        args_g = [fake, fake, fake, fake]
        args_g[i] = None
        scores_, g_, t_, n_ = args_g
        assert sg(ctypes.byref(p), scores_, 0.2, ctypes.byref(s), g_, t_, n_, None) == rk.EINVAL
    assert sg(ctypes.byref(other), fake, 0.2, ctypes.byref(s), fake, fake, fake, None) == rk.EINVAL
    bg = lib.relaxkv_build_sets_global
    assert bg(ctypes.byref(p), ctypes.byref(s), None, fake, None) == rk.EINVAL
    assert bg(ctypes.byref(p), ctypes.byref(s), fake, None, None) == rk.EINVAL
    assert bg(ctypes.byref(other), ctypes.byref(s), fake, fake, None) == rk.EINVAL
    assert bg(ctypes.byref(p), None, fake, fake, None) == rk.EINVAL
    assert s.global_targets == 0                     # unchanged by rejected calls
    # build_sets_context (context-construction variants)
    bc = lib.relaxkv_build_sets_context
    for c in (-1, 3):
        assert bc(ctypes.byref(p), fake, c, ctypes.byref(s), None) == rk.EINVAL
    assert bc(ctypes.byref(p), None, 1, ctypes.byref(s), None) == rk.EINVAL
    assert bc(ctypes.byref(other), fake, 1, ctypes.byref(s), None) == rk.EINVAL
    assert bc(ctypes.byref(p), fake, 1, None, None) == rk.EINVAL
    s3 = _bound_sets(rk, p)
    s3.ctx = None
    assert bc(ctypes.byref(p), fake, 1, ctypes.byref(s3), None) == rk.EINVAL
    s3 = _bound_sets(rk, p)
    s3.context_sets = 7                              # a corrupted flag is refused
    assert lib.relaxkv_sparse_attn(ctypes.byref(p), ctypes.byref(s3), 0, *args, 0,
                                   None) == rk.EINVAL
    assert s.context_sets == 0
    # query_attn (query-side completion)
    qws = lib.relaxkv_query_attn_workspace_bytes(ctypes.byref(p))
    assert qws > 0 and qws % 256 == 0
    qa = lib.relaxkv_query_attn
    for layer in (-1, 4):
        assert qa(ctypes.byref(p), layer, fake, fake, fake, fake, fake, None, fake, qws,
                  None) == rk.EINVAL
    for i in range(5):
        ptrs = [fake] * 5
        ptrs[i] = None
        assert qa(ctypes.byref(p), 0, *ptrs, None, fake, qws, None) == rk.EINVAL
    assert qa(ctypes.byref(p), 0, fake, fake, fake, fake, fake, None, None, qws, None) == rk.EINVAL
    assert qa(ctypes.byref(p), 0, fake, fake, fake, fake, fake, None, fake, qws - 1,
              None) == rk.ENOSPACE
    assert qa(ctypes.byref(_problem(rk, d=96)), 0, fake, fake, fake, fake, fake, None, fake, qws,
              None) == rk.EUNSUPPORTED
    assert lib.relaxkv_query_attn_workspace_bytes(ctypes.byref(_problem(rk, d=96))) == 0
    # counts_to_host
    c = (ctypes.c_int32 * 6)()
    assert lib.relaxkv_counts_to_host(None, c, None, None) == rk.EINVAL
    assert lib.relaxkv_counts_to_host(ctypes.byref(s), None, None, None) == rk.EINVAL


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: any other count exits with status 2 and says so
    (before touching a device)."""
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_library_refused_when_sources_change(tmp_path):
    """The build record ties the library to its sources: a touched source, a
    touched header or a swapped library makes verification (and so
    relaxkv.load()) fail."""
    import shutil

    from paper_2609_33503_amd import build
    for sub in ("paper_2609_33503_amd/csrc", "include"):
        shutil.copytree(os.path.join(ROOT, sub), tmp_path / sub)
    lib = tmp_path / "librelaxkv.so"
    lib.write_bytes(b"stand-in library bytes")
    rec = tmp_path / "librelaxkv.build.json"
    import json
    rec.write_text(json.dumps({"sources_sha256": build.source_digest(str(tmp_path)),
                               "library_sha256": build.file_digest(str(lib))}))
    build.verify(str(lib), str(rec), str(tmp_path))            # matching record: accepted
    src = tmp_path / "paper_2609_33503_amd/csrc/attn.hip"
    src.write_text(src.read_text() + "\n// touched\n")
    with pytest.raises(RuntimeError, match="other sources"):
        build.verify(str(lib), str(rec), str(tmp_path))
    src.write_text(src.read_text()[:-len("\n// touched\n")])
    build.verify(str(lib), str(rec), str(tmp_path))
    hdr = tmp_path / "include/relaxkv.h"
    hdr.write_text(hdr.read_text() + " ")
    with pytest.raises(RuntimeError, match="other sources"):
        build.verify(str(lib), str(rec), str(tmp_path))
    hdr.write_text(hdr.read_text()[:-1])
    lib.write_bytes(b"another library")
    with pytest.raises(RuntimeError, match="not the library"):
        build.verify(str(lib), str(rec), str(tmp_path))
    rec.unlink()
    with pytest.raises(RuntimeError, match="no build record"):
        build.verify(str(lib), str(rec), str(tmp_path))


def test_binding_checks_tensors_before_any_call(rk):
    """The binding's tensor checks (device, dtype, contiguity, shape) run before
    a pointer reaches the library; here on CPU tensors, so nothing is called."""
    import torch
    cpu = torch.device("cpu")
    t = torch.zeros(4, 8, 16, dtype=torch.bfloat16)
    rk._need(t, "x", torch.bfloat16, (4, 8, 16), cpu)
    rk._need(t, "x", torch.bfloat16, (None, 8, 16), cpu)
    for args, msg in [((torch.float32, (4, 8, 16), cpu), "must be torch.float32"),
                      ((torch.bfloat16, (4, 8, 17), cpu), "shape"),
                      ((torch.bfloat16, (4, 8), cpu), "shape"),
                      ((torch.bfloat16, (4, 8, 16), torch.device("cuda", 0)), "is on cpu")]:
        with pytest.raises(ValueError, match=msg):
            rk._need(t, "x", *args)
    with pytest.raises(ValueError, match="contiguous"):
        rk._need(t.transpose(0, 1), "x", torch.bfloat16, (8, 4, 16), cpu)
    with pytest.raises(ValueError, match="tensor"):
        rk._need(None, "x", torch.bfloat16, (4, 8, 16), cpu)
    q = torch.zeros(2, 4, 8, 64, dtype=torch.bfloat16)
    kc = torch.zeros(2, 2, 32, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        rk.Request(q, kc, kc.clone(), 0.15)


def test_query_attn_noalloc_rejects_before_any_device_call(rk):
    """The allocation-free query-side completion validates like relaxkv_query_attn
    and refuses a problem whose scratch exceeds what it holds, before it touches
    a device (every call here is refused)."""
    lib = rk.load()
    fake = ctypes.c_void_p(0x7e0000000000)
    cap = rk.QUERY_ATTN_NOALLOC_MAX_BYTES
    big = _problem(rk, T_c=1 << 19, n_query=64, H=40, H_kv=8)
    assert lib.relaxkv_query_attn_workspace_bytes(ctypes.byref(big)) > cap
    qn = lib.relaxkv_query_attn_noalloc
    assert qn(ctypes.byref(big), 0, fake, fake, fake, fake, fake, None, None) == rk.ENOSPACE
    p = _problem(rk)
    for layer in (-1, 4):
        assert qn(ctypes.byref(p), layer, fake, fake, fake, fake, fake, None, None) == rk.EINVAL
    for i in range(5):
        ptrs = [fake] * 5
        ptrs[i] = None
        assert qn(ctypes.byref(p), 0, *ptrs, None, None) == rk.EINVAL
    assert qn(ctypes.byref(_problem(rk, d=96)), 0, fake, fake, fake, fake, fake, None,
              None) == rk.EUNSUPPORTED
    assert qn(None, 0, fake, fake, fake, fake, fake, None, None) == rk.EINVAL
    # the bound the header states: 40q/8kv heads, 64 query tokens, T_c up to 131072
    for T in (4096, 32768, 131072):
        fits = _problem(rk, T_c=T, n_query=64, H=40, H_kv=8)
        assert 0 < lib.relaxkv_query_attn_workspace_bytes(ctypes.byref(fits)) <= cap
