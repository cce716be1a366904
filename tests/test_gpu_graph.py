"""The whole hot path under HIP stream capture: scoring, selection, set
construction and the attention of every layer (both context modes) recorded
into one graph and replayed.  Every call enqueues kernels only (no memset, no
host synchronisation, no allocation), and the attention's per-layer work
counters return to zero at the end of each launch, so every replay must give
the eager results bit for bit.  Replays are separated by the program's own
eager work (another attention launch, torch ops) and synchronisations, and
the graph's attention is checked against the oracle once."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from harness import Case, assert_close, compare_sets
from paper_2609_33503_amd import relaxkv, synth

pytestmark = pytest.mark.gpu

W = synth.shrink(synth.WORKLOADS["qwen14b-32k-planted"], L=4, T_c=2600)


def _step(case, scores, fresh, outs, lses):
    case.req.score(case.ws, scores)
    case.req.select(scores, case.sets)
    case.req.build_sets(case.sets)
    for (l, cm), (qn, kn, vn) in fresh.items():
        case.req.sparse_attn(case.sets, l, qn, kn, vn, outs[(l, cm)], lses[(l, cm)],
                             context_mode=cm)


def test_hot_path_graph_replays_match_eager(gpu_lib):
    case = Case(W)
    scores = torch.empty(case.L, case.T, dtype=torch.float32, device="cuda")
    # eager: the sets give each layer's targets, whose fresh rows the graph reuses
    case.req.score(case.ws, scores)
    case.req.select(scores, case.sets)
    got = case.gpu_sets()
    modes = (relaxkv.CONTEXT_UNION, relaxkv.CONTEXT_FULL)
    fresh = {(l, cm): case.fresh(l, got["R"][l]) for l in range(case.L) for cm in modes}
    n = {l: len(got["R"][l]) for l in range(case.L)}
    eager_o = {k: torch.empty(n[k[0]], W.H, W.d, dtype=case.q.dtype, device="cuda") for k in fresh}
    eager_l = {k: torch.empty(n[k[0]], W.H, dtype=torch.float32, device="cuda") for k in fresh}
    eager_s = torch.empty_like(scores)
    _step(case, eager_s, fresh, eager_o, eager_l)
    torch.cuda.synchronize()

    outs = {k: torch.empty_like(v) for k, v in eager_o.items()}
    lses = {k: torch.empty_like(v) for k, v in eager_l.items()}
    g_scores = torch.empty_like(scores)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                   # one warm pass on the capture stream
        _step(case, g_scores, fresh, outs, lses)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(case, g_scores, fresh, outs, lses)
    torch.cuda.synchronize()

    other = fresh[(1, relaxkv.CONTEXT_UNION)]
    other_o = torch.empty_like(eager_o[(1, relaxkv.CONTEXT_UNION)])
    for rep in range(4):
        g_scores.fill_(float("nan"))
        for k in outs:
            outs[k].fill_(float("nan"))
            lses[k].fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(g_scores, eager_s), rep
        for k in outs:
            assert torch.equal(outs[k], eager_o[k]), (rep, k)
            assert torch.equal(lses[k], eager_l[k]), (rep, k)
        assert int(case.sets.tiles.abs().sum()) == 0, rep
        # the program's own eager work between replays
        case.req.sparse_attn(case.sets, 1, *other, other_o)
        torch.cuda.synchronize()
        assert torch.equal(other_o, eager_o[(1, relaxkv.CONTEXT_UNION)]), rep
        _ = (g_scores * 2).sum().item()

    # the graph's results against the oracle (sets bit-exact, attention of two layers)
    a_ref, _, _ = case.oracle_scores()
    assert_close(g_scores.cpu().numpy(), a_ref, W, "scores (graph)")
    a32 = g_scores.cpu().numpy()
    sets_ref = oracle.build_sets(oracle.select(a32.astype(np.float64), case.k), case.T)
    compare_sets(case.gpu_sets(), sets_ref)
    for l in (0, case.L - 1):
        for cm, mode in zip(modes, ("union", "full")):
            O_ref, lse_ref = case.oracle_attn(l, sets_ref, fresh[(l, cm)], mode=mode)
            assert_close(outs[(l, cm)].float().cpu().numpy(), O_ref, W, f"O layer {l} {mode}",
                         rel_gate=1e-2)
            assert_close(lses[(l, cm)].cpu().numpy(), lse_ref, W, f"lse layer {l} {mode}")
