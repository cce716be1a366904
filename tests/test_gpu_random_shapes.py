"""Seeded random problem shapes through the whole path against the oracle:
scores, selection and sets (bit-exact on shared fp32 scores), the attention of
every layer (union context, and the full prefix for every other shape), and
the query-side completion.  The shapes are drawn once from a fixed seed over
the ranges the kernels handle (1-4 layers, 1-4000 context positions, 1-8 KV
heads, GQA groups of 1-16, head dim 64 or 128, 1-160 query tokens, anchor
ratios from 1% to 100%, bf16 and fp32), so ragged tails, tiny contexts,
tiles that split a target's heads, several query row chunks and single-row
cases all occur."""

from __future__ import annotations

import numpy as np
import pytest

from harness import Case, assert_close
from paper_2609_33503_amd import synth

from test_gpu_parity import _pipeline
from test_gpu_query_attn import oracle_query, run_query

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


def _shapes(n=32, seed=2026):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        fp32 = i % 4 == 3
        H_kv = int(rng.choice([1, 2, 3, 4, 8]))
        G = int(rng.integers(1, 17))
        base = W["tiny-2L-1k-fp32"] if fp32 else W["llama8b-8k"]
        kw = dict(L=int(rng.integers(1, 5)), T_c=int(rng.integers(1, 4001)), H=H_kv * G, H_kv=H_kv,
                  d=int(rng.choice([64, 128])), Qn=int(rng.integers(1, 161)),
                  ratio=float(rng.choice([0.01, 0.05, 0.15, 0.3, 0.6, 1.0])))
        if kw["H"] > 32:                    # keeps the oracle's per-head loops to seconds
            kw["H"], kw["H_kv"] = 4 * G if G <= 8 else 2 * G, 4 if G <= 8 else 2
        out.append((f"s{i}-" + "-".join(f"{k}{v}" for k, v in kw.items()) + ("-f32" if fp32 else ""),
                    synth.shrink(base, **kw)))
    return out


SHAPES = _shapes()


@pytest.mark.parametrize("name,w", SHAPES, ids=[s[0] for s in SHAPES])
def test_random_shape_pipeline(gpu_lib, name, w):
    _pipeline(Case(w))
    if SHAPES.index((name, w)) % 2 == 0:
        _pipeline(Case(w), mode="full")
    case = Case(w)
    for l in range(case.L):
        kq, vq, out, lse = run_query(case, l)
        O_ref, lse_ref = oracle_query(case, l, kq, vq)
        assert_close(out.float().cpu().numpy(), O_ref, w, f"{name} query O layer {l}",
                     rel_gate=1e-2 if w.dtype == "bf16" else None)
        assert_close(lse.cpu().numpy(), lse_ref, w, f"{name} query lse layer {l}")
