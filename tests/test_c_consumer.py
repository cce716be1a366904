"""A plain C11 program as the library's caller (tests/c_consumer): it compiles
against include/relaxkv.h with -std=c11 -pedantic -Werror, and its results
match the Python binding's (host calls) and the oracle's (the GPU path: scores,
selection, sets and attention of every layer, run from C with its own HIP
allocations and stream)."""

from __future__ import annotations

import ctypes
import os
import subprocess
import sys
import tempfile

import numpy as np
import pytest
import torch

import oracle
from harness import assert_close
from paper_2609_33503_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c_consumer"))
import build_consumer as c_build  # noqa: E402


def test_c_consumer_compiles_and_host_calls_agree(rk):
    with tempfile.TemporaryDirectory() as d:
        exe = c_build.build(os.path.join(d, "consumer"))
        r = subprocess.run([exe, "host"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    got = dict(line.split(" ", 1) for line in r.stdout.strip().splitlines())
    lib = rk.load()
    p = rk.Problem(4, 2048, 16, 8, 2, 128, rk.DTYPE_BF16, 0.0, 0.15, 0x1000, 0x2000, 0x3000, None)
    assert int(got["anchor_count_0.15_2048"]) == oracle.anchor_count(0.15, 2048)
    assert int(got["anchor_count_0.125_20"]) == oracle.anchor_count(0.125, 20) == 2
    assert int(got["anchor_count_bad"]) == rk.EINVAL
    assert int(got["validate_ok"]) == 0
    assert int(got["validate_d96"]) == rk.EUNSUPPORTED
    assert int(got["validate_gqa"]) == rk.EINVAL
    assert int(got["sets_bytes"]) == lib.relaxkv_sets_bytes(ctypes.byref(p))
    assert int(got["score_ws_bytes"]) == lib.relaxkv_score_workspace_bytes(ctypes.byref(p))
    assert int(got["sets_bind"]) == 0 and int(got["sets_bind_short"]) == rk.ENOSPACE
    assert int(got["sets_k"]) == oracle.anchor_count(0.15, 2048)
    s = rk.Sets()
    base = 0x7f0000000000
    assert lib.relaxkv_sets_bind(ctypes.byref(p), ctypes.c_void_p(base),
                                 lib.relaxkv_sets_bytes(ctypes.byref(p)), ctypes.byref(s)) == 0
    assert int(got["sets_tiles_offset"]) == s.tiles - base
    assert int(got["score_null_ws"]) == rk.EINVAL
    assert int(got["attn_bad_layer"]) == rk.EINVAL and int(got["attn_neg_rows"]) == rk.EINVAL
    assert got["status_string"] == "buffer too small"


def _bf16_bytes(t):
    return t.contiguous().view(torch.int16).cpu().numpy().tobytes()


def _read(d, name, dtype):
    return np.fromfile(os.path.join(d, name), dtype=dtype)


@pytest.mark.gpu
def test_c_consumer_pipeline_matches_oracle(gpu_lib):
    exe = c_build.OUT
    if not os.path.exists(exe):          # normally built by build(); a host-side gcc step
        c_build.build()
    w = synth.shrink(synth.WORKLOADS["qwen14b-32k-planted"], L=3, T_c=1500)
    q, kc, vc = synth.make_cache(w, "cpu")
    with tempfile.TemporaryDirectory() as d:
        with open(os.path.join(d, "params.txt"), "w") as f:
            f.write(f"{w.L} {w.T_c} {w.Qn} {w.H} {w.H_kv} {w.d} {w.ratio!r}\n")
        for name, t in (("q.bin", q), ("kc.bin", kc), ("vc.bin", vc)):
            with open(os.path.join(d, name), "wb") as f:
                f.write(_bf16_bytes(t))
        fresh_all = []
        for l in range(w.L):
            fq, fk, fv = synth.make_fresh_layer(w, l, kc[l], vc[l], "cpu")
            fresh_all.append((fq, fk, fv))
            for name, t in ((f"fq_{l}.bin", fq), (f"fk_{l}.bin", fk), (f"fv_{l}.bin", fv)):
                with open(os.path.join(d, name), "wb") as f:
                    f.write(_bf16_bytes(t))
        r = subprocess.run([exe, "run", d], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stdout + r.stderr
        k = oracle.anchor_count(w.ratio, w.T_c)
        scores = _read(d, "scores.bin", np.float32).reshape(w.L, w.T_c)
        anchors = _read(d, "anchors.bin", np.int32).reshape(w.L, k)
        counts = _read(d, "counts.bin", np.int32)
        r_off = _read(d, "r_off.bin", np.int32)
        r_idx = _read(d, "r_idx.bin", np.int32)
        outs = []
        for l in range(w.L):
            n = int(counts[1 + l])
            outs.append((
                torch.from_numpy(_read(d, f"out_{l}.bin", np.int16).reshape(n, w.H, w.d)
                                 .copy()).view(torch.bfloat16),
                _read(d, f"lse_{l}.bin", np.float32).reshape(n, w.H)))
    a_ref, _, _ = oracle.score(synth.to_f64(q), synth.to_f64(kc))
    assert_close(scores, a_ref, w, "scores (C caller)")
    anchors_ref = oracle.select(scores.astype(np.float64), k)
    assert np.array_equal(anchors, anchors_ref)
    sets_ref = oracle.build_sets(anchors_ref, w.T_c)
    assert counts[0] == len(sets_ref.U) and counts[w.L + 1] == 0
    for l in range(w.L):
        R = r_idx[r_off[l]:r_off[l + 1]]
        assert np.array_equal(R, sets_ref.R[l])
        fresh = tuple(synth.to_f64(synth.gather_rows(t, R)) for t in fresh_all[l])
        O_ref, lse_ref = oracle.sparse_attn(l, sets_ref, *fresh, synth.to_f64(kc[l]),
                                            synth.to_f64(vc[l]))
        assert_close(outs[l][0].float().numpy(), O_ref, w, f"O layer {l} (C caller)",
                     rel_gate=1e-2)
        assert_close(outs[l][1], lse_ref, w, f"lse layer {l} (C caller)")
