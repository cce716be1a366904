"""Seeded random problem shapes through the whole path against the oracle:
scores, selection and sets (bit-exact on shared fp32 scores), the attention of
every layer (union context, and the full prefix for every other shape), and
the query-side completion.  The shapes are drawn once from a fixed seed over
the ranges the kernels handle (1-4 layers, 1-4000 context positions, 1-8 KV
heads, GQA groups of 1-16, head dim 64 or 128, 1-160 query tokens, anchor
ratios from 1% to 100%, bf16 and fp32), so ragged tails, tiny contexts,
tiles that split a target's heads, several query row chunks and single-row
cases all occur.  A third of the shapes also run the matched-target lists and
another third the Global and Layerwise Sparse contexts."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from harness import Case, assert_close, synthetic_scores
from paper_2609_33503_amd import relaxkv, synth

from test_gpu_context_variants import build_both, compare_context_sets
from test_gpu_context_variants import _compare_attn as _compare_variant_attn
from test_gpu_matched_targets import compare_global_sets, gpu_global_sets
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


# The matched-target and context-construction variants over a third of the
# shapes each, on seeded fp32 scores (the selection is bit-exact on them).
MATCHED = [s for i, s in enumerate(SHAPES) if i % 3 == 1]
CONTEXT = [s for i, s in enumerate(SHAPES) if i % 3 == 2]


@pytest.mark.parametrize("name,w", MATCHED, ids=[s[0] for s in MATCHED])
def test_random_shape_matched_targets(gpu_lib, name, w):
    """A random global target list (with every position up to the first union
    position, so some targets have empty contexts): sets bit-exact, attention
    of every layer in both modes against the oracle."""
    case = Case(w)
    a32 = synthetic_scores(case.L, case.T, seed=SHAPES.index((name, w)))
    anchors = oracle.select(a32.astype(np.float64), case.k)
    assert np.array_equal(case.gpu_select(torch.from_numpy(a32).cuda()), anchors)
    U = oracle.build_sets(anchors, case.T).U
    rng = np.random.default_rng(SHAPES.index((name, w)) + 100)
    P = set(rng.choice(case.T, size=max(1, case.T // 4), replace=False).tolist())
    P |= set(range(0, int(U[0]) + 1))
    P = np.array(sorted(P), dtype=np.int64)
    ref = oracle.build_sets_global(anchors, case.T, P)
    compare_global_sets(gpu_global_sets(case, P), ref)
    for mode, cm in (("union", relaxkv.CONTEXT_UNION), ("full", relaxkv.CONTEXT_FULL)):
        for l in range(case.L):
            fresh = case.fresh(l, P)
            out, lse = case.gpu_attn(l, fresh, len(P), cm)
            O_ref, lse_ref = case.oracle_attn(l, ref, fresh, mode=mode)
            _compare_variant_attn(case, out, lse, O_ref, lse_ref, f"{name} {mode} layer {l}")


@pytest.mark.parametrize("construction", ["global", "layerwise"])
@pytest.mark.parametrize("name,w", CONTEXT, ids=[s[0] for s in CONTEXT])
def test_random_shape_context_variants(gpu_lib, name, w, construction):
    """Global and Layerwise Sparse contexts: sets bit-exact, attention of every
    layer (union mode) against the oracle."""
    case = Case(w)
    a32 = synthetic_scores(case.L, case.T, seed=SHAPES.index((name, w)) + 200)
    _, ref = build_both(case, a32, construction)
    compare_context_sets(case, ref, construction)
    for l in range(case.L):
        R_l = ref.R[l]
        fresh = case.fresh(l, R_l)
        out, lse = case.gpu_attn(l, fresh, len(R_l), relaxkv.CONTEXT_UNION)
        O_ref, lse_ref = case.oracle_attn(l, ref, fresh)
        _compare_variant_attn(case, out, lse, O_ref, lse_ref, f"{name} {construction} layer {l}")
