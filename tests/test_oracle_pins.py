"""Pins of the float64 oracle against things other than itself.

Closed forms, the hand-worked example under tests/golden/, brute force on tiny
inputs, torch's scaled_dot_product_attention in float64, and the set
invariants the method implies (Sec. 3.2 - 3.4, App. A).  No GPU needed.
"""

import json
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import anchor_count, attention_flops, build_sets, score, select, sparse_attn

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# anchor budget k = max(1, round(r T_c))
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("r,T,k", [
    (0.15, 1024, 154), (0.15, 8192, 1229), (0.05, 16384, 819), (0.15, 16384, 2458),
    (0.30, 16384, 4915), (0.15, 32768, 4915),
    # exact halves go to the even neighbour; k never drops below 1 or above T_c
    (0.125, 20, 2), (0.375, 4, 2), (0.625, 4, 2), (0.5, 1, 1), (0.0, 50, 1), (1.0, 77, 77),
])
def test_anchor_count_closed_forms(r, T, k):
    assert anchor_count(r, T) == k


@pytest.mark.parametrize("r", [-0.01, 1.01, float("nan"), float("inf")])
def test_anchor_count_rejects(r):
    with pytest.raises(ValueError):
        anchor_count(r, 100)


# ----------------------------------------------------------------------------
# hand-worked example (select, sets, attention)
# ----------------------------------------------------------------------------

def _hand():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        return json.load(f)


def test_hand_example_select_and_sets():
    ex = _hand()
    k = anchor_count(ex["ratio"], ex["T_c"])
    assert k == ex["k"]
    S = select(np.array(ex["a"]), k)
    assert S.tolist() == ex["anchors"]
    s = build_sets(S, ex["T_c"])
    assert s.h.tolist() == ex["h"]
    assert s.U.tolist() == ex["U"]
    assert [r.tolist() for r in s.R] == ex["R"]
    assert [x.tolist() for x in s.src] == ex["src"]
    assert s.edges.tolist() == ex["edges"]
    assert s.edges_full.tolist() == ex["edges_full"]


def test_hand_example_attention():
    ex = _hand()
    T = ex["T_c"]
    s = build_sets(np.array(ex["anchors"]), T)
    kc = np.zeros((1, T, 1))
    vc = np.arange(T, dtype=np.float64).reshape(1, T, 1)
    for case in ex["attention"]:
        l = case["layer"]
        R_l = s.R[l]
        qn = np.ones((len(R_l), 1, 1))
        kn = np.zeros((len(R_l), 1, 1))
        vn = (R_l.astype(np.float64) + 100.0).reshape(-1, 1, 1)
        t = int(np.flatnonzero(R_l == case["position"])[0])
        O, _ = sparse_attn(l, s, qn, kn, vn, kc, vc, softmax_scale=1.0,
                           mode=case["mode"], targets=[t])
        assert O[0, 0, 0] == pytest.approx(case["out"], abs=1e-12)


def _count_attention_flops(sets, H, d, mode="union"):
    """Operation count of a naive evaluation, enumerated from the mask itself
    (not from the edge counts): for every layer, target p in R_l, query head
    and context key j (j in U and j <= p, or j <= p for the full prefix) one
    d-long dot product (d multiplies, d adds) and one d-long scaled
    accumulation of V_j (d multiplies, d adds)."""
    n = 0
    union = set(sets.U.tolist())
    for l in range(sets.L):
        for p in sets.R[l].tolist():
            for _h in range(H):
                for j in range(p + 1):
                    if mode == "full" or j in union:
                        n += (d + d) + (d + d)
    return n


def test_attention_flops_hand_example():
    # 10 + 9 + 5 = 24 unmasked edges (App. A.2 edge count); with one head and
    # d = 1 each edge is one multiply-add for the logit and one for the output.
    ex = _hand()
    s = build_sets(np.array(ex["anchors"]), ex["T_c"])
    assert attention_flops(1, 1, s.edges) == 96.0
    assert attention_flops(1, 1, s.edges_full) == 4 * (18 + 16 + 8)
    assert attention_flops(3, 5, s.edges) == _count_attention_flops(s, 3, 5)
    assert attention_flops(3, 5, s.edges_full) == _count_attention_flops(s, 3, 5, "full")


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 4), st.integers(1, 40), st.integers(1, 4), st.integers(1, 9),
       st.integers(0, 2**31 - 1), st.data())
def test_attention_flops_brute_force(L, T, H, d, seed, data):
    k = data.draw(st.integers(1, T))
    rng = np.random.default_rng(seed)
    S = np.stack([np.sort(rng.choice(T, size=k, replace=False)) for _ in range(L)])
    s = build_sets(S, T)
    assert attention_flops(H, d, s.edges) == _count_attention_flops(s, H, d)
    assert attention_flops(H, d, s.edges_full) == _count_attention_flops(s, H, d, "full")


# ----------------------------------------------------------------------------
# score: closed forms, invariants, independent library routine
# ----------------------------------------------------------------------------

def test_score_closed_form_logs():
    # one head, one query token, d = 1, sigma = 1, q = 1, keys = log(1..4):
    # softmax = (1,2,3,4)/10, MinMax -> (0, 1/3, 2/3, 1).
    q = np.ones((1, 1, 1, 1))
    k = np.log(np.arange(1, 5, dtype=np.float64)).reshape(1, 1, 4, 1)
    a, p, lse = score(q, k, softmax_scale=1.0)
    np.testing.assert_allclose(p[0], [0.1, 0.2, 0.3, 0.4], atol=1e-15)
    np.testing.assert_allclose(a[0], [0, 1 / 3, 2 / 3, 1], atol=1e-15)
    assert lse[0, 0, 0] == pytest.approx(math.log(10.0), abs=1e-15)


def test_score_degenerate_minmax_and_gqa_sharing():
    # Two query heads share one KV head (G = 2) with q = (+1, -1) and keys
    # (0, log 2): the rows are (1/3, 2/3) and (2/3, 1/3), the pooled score is
    # (1/2, 1/2) -> constant -> a = 0 -> the tie rule picks position 0.
    q = np.array([1.0, -1.0]).reshape(1, 1, 2, 1)
    k = np.array([0.0, math.log(2.0)]).reshape(1, 1, 2, 1)
    a, p, _ = score(q, k, softmax_scale=1.0)
    np.testing.assert_allclose(p[0], [0.5, 0.5], atol=1e-15)
    assert a[0].tolist() == [0.0, 0.0]
    kk = anchor_count(0.2, 2)
    assert kk == 1
    assert select(a, kk).tolist() == [[0]]


def test_score_equal_keys_select_first_k():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((2, 3, 4, 8))
    k = np.broadcast_to(rng.standard_normal((1, 2, 1, 8)), (2, 2, 30, 8)).copy()
    a, _, _ = score(q, k)
    assert np.all(a == 0.0)
    assert select(a, 5).tolist() == [list(range(5))] * 2


def _rand_score_inputs(seed, L=2, Qn=3, H=4, H_kv=2, T=37, d=8):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((L, Qn, H, d)), rng.standard_normal((L, H_kv, T, d))


def test_score_pooled_mass_is_one():
    # every softmax row sums to 1, so the pooled mean over H*Qn rows sums to 1
    q, k = _rand_score_inputs(1)
    _, p, _ = score(q, k)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-13)


def test_score_matches_brute_force_loops():
    q, k = _rand_score_inputs(2, L=1, Qn=2, H=4, H_kv=2, T=9, d=3)
    a, p, _ = score(q, k)
    L, Qn, H, d = q.shape
    T = k.shape[2]
    pb = [0.0] * T
    for h in range(H):
        g = h // 2
        for t in range(Qn):
            logits = [sum(q[0, t, h, e] * k[0, g, i, e] for e in range(d)) / math.sqrt(d)
                      for i in range(T)]
            z = sum(math.exp(x) for x in logits)
            for i in range(T):
                pb[i] += math.exp(logits[i]) / z / (H * Qn)
    np.testing.assert_allclose(p[0], pb, rtol=1e-12)
    lo, hi = min(pb), max(pb)
    np.testing.assert_allclose(a[0], [(x - lo) / (hi - lo) for x in pb], atol=1e-12)


def test_score_matches_sdpa_attention_weights():
    # scaled_dot_product_attention with V = identity returns the attention
    # weights themselves; enable_gqa maps query head h to KV head h // G.
    q, k = _rand_score_inputs(3, L=2, Qn=5, H=6, H_kv=2, T=23, d=16)
    _, p, _ = score(q, k)
    for l in range(q.shape[0]):
        qt = torch.from_numpy(q[l]).permute(1, 0, 2)[None]            # [1][H][Qn][d]
        kt = torch.from_numpy(k[l])[None]                               # [1][H_kv][T][d]
        eye = torch.eye(k.shape[2], dtype=torch.float64).expand(1, k.shape[1], -1, -1)
        A = torch.nn.functional.scaled_dot_product_attention(qt, kt, eye, enable_gqa=True)
        np.testing.assert_allclose(p[l], A.mean(dim=(0, 1, 2)).numpy(), atol=1e-14)


def test_score_supplied_lse():
    q, k = _rand_score_inputs(4)
    a, p, lse = score(q, k)
    a2, p2, _ = score(q, k, row_lse=lse)
    np.testing.assert_allclose(p2, p, rtol=1e-12)
    # a larger normaliser (the query's own tokens in a real forward) scales p
    # by exp(-c) and leaves the MinMax-normalised score unchanged
    a3, p3, _ = score(q, k, row_lse=lse + 0.7)
    np.testing.assert_allclose(p3, p * math.exp(-0.7), rtol=1e-12)
    np.testing.assert_allclose(a3, a, atol=1e-12)


def test_score_permutation_equivariance():
    q, k = _rand_score_inputs(5)
    perm = np.random.default_rng(9).permutation(k.shape[2])
    a, p, _ = score(q, k)
    a2, p2, _ = score(q, k[:, :, perm, :])
    np.testing.assert_allclose(p2, p[:, perm], rtol=1e-12)


# ----------------------------------------------------------------------------
# select: brute force, ties, -0.0, NaN, invariance
# ----------------------------------------------------------------------------

def _brute_topk(row, k):
    order = sorted(range(len(row)), key=lambda i: (-row[i], i))
    return sorted(order[:k])


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 4), st.integers(1, 40), st.data())
def test_select_brute_force_with_ties(L, T, data):
    vals = data.draw(st.lists(st.sampled_from([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, 0.1]),
                              min_size=L * T, max_size=L * T))
    a = np.array(vals).reshape(L, T)
    k = data.draw(st.integers(1, T))
    S = select(a, k)
    for l in range(L):
        assert S[l].tolist() == _brute_topk([0.0 if x == 0 else x for x in a[l]], k)


def test_select_negative_zero_ties_positive_zero():
    a = np.array([[-0.0, 0.0, -0.0, 0.0]])
    assert select(a, 2).tolist() == [[0, 1]]


def test_select_rejects_nan():
    with pytest.raises(ValueError):
        select(np.array([[0.1, float("nan")]]), 1)


def test_select_positive_affine_invariance():
    rng = np.random.default_rng(6)
    a = rng.integers(0, 16, size=(3, 50)) / 8.0          # exact under x -> 2x + 0.5
    for k in (1, 7, 25, 50):
        assert np.array_equal(select(a, k), select(2.0 * a + 0.5, k))


# ----------------------------------------------------------------------------
# sets: invariants of h, U, R_l and the edge counts
# ----------------------------------------------------------------------------

def _random_anchors(rng, L, T, k):
    return np.stack([np.sort(rng.choice(T, size=k, replace=False)) for _ in range(L)])


@settings(max_examples=80, deadline=None)
@given(st.integers(1, 5), st.integers(1, 60), st.integers(0, 2**31 - 1), st.data())
def test_sets_invariants(L, T, seed, data):
    k = data.draw(st.integers(1, T))
    S = _random_anchors(np.random.default_rng(seed), L, T, k)
    s = build_sets(S, T)
    union = set()
    for l in range(L):
        union |= set(S[l].tolist())
    assert s.U.tolist() == sorted(union)                          # U = union of S_l
    assert len(s.R) == L
    for i in range(T):                                            # active exactly up to h_i
        for l in range(L):
            assert (i in set(s.R[l].tolist())) == (s.h[i] >= 0 and l <= s.h[i])
    assert s.R[0].tolist() == s.U.tolist()                        # R_0 = U
    assert s.R[L - 1].tolist() == S[L - 1].tolist()               # R_{L-1} = S_{L-1}
    for l in range(L):
        assert len(S[l]) == k
        assert set(S[l].tolist()) <= set(s.R[l].tolist())          # S_l within R_l
        if l + 1 < L:
            assert set(s.R[l + 1].tolist()) <= set(s.R[l].tolist())   # nested
        assert np.all(np.diff(s.R[l]) > 0)
        # src: rank of U[c] in R_l, or -1
        for c, pos in enumerate(s.U.tolist()):
            hits = np.flatnonzero(s.R[l] == pos)
            assert s.src[l][c] == (hits[0] if len(hits) else -1)
        # edges by counting |C_l(p)| directly
        e = sum(sum(1 for j in s.U.tolist() if j <= p) for p in s.R[l].tolist())
        assert s.edges[l] == e
        assert s.edges_full[l] == sum(p + 1 for p in s.R[l].tolist())
        assert s.edges[l] <= s.edges_full[l]
        full_prefix_in_U = all(set(range(p + 1)) <= union for p in s.R[l].tolist())
        assert (s.edges[l] == s.edges_full[l]) == full_prefix_in_U
    assert sum(len(r) for r in s.R) == int(np.sum(s.h[s.U] + 1))   # state count


# ----------------------------------------------------------------------------
# sparse attention: brute force with an explicit dense mask, causal reduction
# ----------------------------------------------------------------------------

def _brute_attention(l, S, T, qn, kn, vn, kc, vc, sigma, mode):
    """Dense masked attention over all T positions, evaluating the context and
    the mixed fresh/cached rule literally for every (target, position) pair."""
    L = len(S)
    U = set()
    for x in S:
        U |= set(int(i) for i in x)
    h = {i: max(ll for ll in range(L) if i in set(S[ll].tolist())) for i in U}
    R = sorted(i for i in U if h[i] >= l)
    rank = {p: t for t, p in enumerate(R)}
    H, d = qn.shape[1], qn.shape[2]
    G = H // kc.shape[0]
    O = np.zeros((len(R), H, d))
    lse = np.zeros((len(R), H))
    for t, p in enumerate(R):
        for hh in range(H):
            g = hh // G
            logits = np.full(T, -np.inf)
            vals = np.zeros((T, d))
            for j in range(T):
                in_ctx = (j in U and j <= p) if mode == "union" else (j <= p)
                if not in_ctx:
                    continue
                fresh = j in rank                    # j in R_l (and in the context)
                kj = kn[rank[j], g] if fresh else kc[g, j]
                vals[j] = vn[rank[j], g] if fresh else vc[g, j]
                logits[j] = sigma * float(np.dot(qn[t, hh], kj))
            m = logits.max()
            w = np.exp(logits - m)
            O[t, hh] = (w / w.sum()) @ vals
            lse[t, hh] = m + math.log(w.sum())
    return np.array(R), O, lse


@pytest.mark.parametrize("seed,L,T,k,mode", [(0, 3, 40, 6, "union"), (1, 2, 33, 3, "union"),
                                             (2, 3, 40, 6, "full"), (3, 4, 25, 1, "union")])
def test_attention_brute_force(seed, L, T, k, mode):
    rng = np.random.default_rng(seed)
    H, H_kv, d = 4, 2, 8
    S = _random_anchors(rng, L, T, k)
    s = build_sets(S, T)
    for l in range(L):
        n = len(s.R[l])
        qn = rng.standard_normal((n, H, d))
        kn = rng.standard_normal((n, H_kv, d))
        vn = rng.standard_normal((n, H_kv, d))
        kc = rng.standard_normal((H_kv, T, d))
        vc = rng.standard_normal((H_kv, T, d))
        O, lse = sparse_attn(l, s, qn, kn, vn, kc, vc, mode=mode)
        R, Ob, lseb = _brute_attention(l, S, T, qn, kn, vn, kc, vc, 1 / math.sqrt(d), mode)
        assert R.tolist() == s.R[l].tolist()
        np.testing.assert_allclose(O, Ob, atol=1e-12)
        np.testing.assert_allclose(lse, lseb, atol=1e-12)
        # softmax rows sum to 1: exp(logits - lse) over the context
        t = n - 1
        p = s.R[l][t]
        ctx = s.U[s.U <= p] if mode == "union" else np.arange(p + 1)
        rank = {int(x): i for i, x in enumerate(s.R[l])}
        Krows = np.stack([kn[rank[j]] if j in rank else kc[:, j] for j in ctx.tolist()])
        for hh in range(H):
            w = np.exp(Krows[:, hh // 2] @ qn[t, hh] / math.sqrt(d) - lse[t, hh])
            assert w.sum() == pytest.approx(1.0, abs=1e-12)


def test_attention_full_union_is_causal_sdpa():
    # every position an anchor of every layer -> U = R_l = all positions, and
    # sparse-context attention is ordinary causal GQA self-attention on the
    # fresh rows.
    rng = np.random.default_rng(7)
    L, T, H, H_kv, d = 2, 29, 6, 2, 16
    S = np.tile(np.arange(T), (L, 1))
    s = build_sets(S, T)
    qn = rng.standard_normal((T, H, d))
    kn = rng.standard_normal((T, H_kv, d))
    vn = rng.standard_normal((T, H_kv, d))
    kc = rng.standard_normal((H_kv, T, d))          # never read
    vc = rng.standard_normal((H_kv, T, d))
    for mode in ("union", "full"):
        O, _ = sparse_attn(1, s, qn, kn, vn, kc, vc, mode=mode)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(qn).permute(1, 0, 2)[None],
            torch.from_numpy(kn).permute(1, 0, 2)[None],
            torch.from_numpy(vn).permute(1, 0, 2)[None], is_causal=True, enable_gqa=True)
        np.testing.assert_allclose(O, ref[0].permute(1, 0, 2).numpy(), atol=1e-12)


def test_attention_union_equals_full_prefix_when_union_covers_all():
    # S_0, S_1, S_2 partition the positions: U = everything, but R_l shrinks.
    rng = np.random.default_rng(8)
    T, H, H_kv, d = 12, 2, 1, 4
    S = np.arange(T).reshape(3, 4)
    s = build_sets(S, T)
    assert s.U.tolist() == list(range(T))
    kc = rng.standard_normal((H_kv, T, d))
    vc = rng.standard_normal((H_kv, T, d))
    for l in range(3):
        n = len(s.R[l])
        qn, kn, vn = (rng.standard_normal((n, hh, d)) for hh in (H, H_kv, H_kv))
        Ou, lu = sparse_attn(l, s, qn, kn, vn, kc, vc, mode="union")
        Of, lf = sparse_attn(l, s, qn, kn, vn, kc, vc, mode="full")
        np.testing.assert_allclose(Ou, Of, atol=1e-14)
        np.testing.assert_allclose(lu, lf, atol=1e-14)


def test_chunk_size_does_not_change_inputs():
    # Chunking only affects how a real cache is built; the 2048-token chunking of
    # the matched-target control has identical inputs to the 512-token one.
    from paper_2609_33503_amd import synth
    a = synth.shrink(synth.WORKLOADS["qwen14b-32k-control"], T_c=700, L=2, Qn=4)
    b = synth.shrink(synth.WORKLOADS["qwen14b-32k-control-c2048"], T_c=700, L=2, Qn=4)
    import dataclasses
    assert a.wid == b.wid and a.chunk != b.chunk
    for l in range(2):
        for x, y in zip(synth.make_cache_layer(a, l), synth.make_cache_layer(b, l)):
            assert torch.equal(x, y)
    assert dataclasses.replace(b, chunk=a.chunk, name=a.name) == a


# ----------------------------------------------------------------------------
# cache update
# ----------------------------------------------------------------------------

def test_update_cache_hand_example():
    from oracle import update_cache
    ex = _hand()
    T = ex["T_c"]
    s = build_sets(np.array(ex["anchors"]), T)
    kc = np.arange(T, dtype=np.float64).reshape(1, T, 1)
    vc = -kc
    for l, R_l in enumerate(ex["R"]):
        kn = (np.array(R_l, dtype=np.float64) + 100.0).reshape(-1, 1, 1)
        k2, v2 = update_cache(l, s, kn, -kn, kc, vc)
        # exactly the positions of R_l change, to their fresh rows
        expect = [p + 100.0 if p in R_l else float(p) for p in range(T)]
        assert k2[0, :, 0].tolist() == expect
        assert v2[0, :, 0].tolist() == [-x for x in expect]
        assert kc[0, :, 0].tolist() == list(range(T))          # input untouched


def test_update_cache_then_full_prefix_attention_reads_fresh_rows():
    # After the update, the layer's cache holds the fresh rows at R_l, so the
    # Full-Prefix Control over the updated cache with every row "cached" gives
    # the same output as the mixed rule over the naive cache.
    from oracle import update_cache
    rng = np.random.default_rng(12)
    L, T, H, H_kv, d = 2, 30, 4, 2, 8
    S = _random_anchors(rng, L, T, 5)
    s = build_sets(S, T)
    l = 0
    n = len(s.R[l])
    qn, kn, vn = (rng.standard_normal((n, hh, d)) for hh in (H, H_kv, H_kv))
    kc = rng.standard_normal((H_kv, T, d))
    vc = rng.standard_normal((H_kv, T, d))
    O1, _ = sparse_attn(l, s, qn, kn, vn, kc, vc, mode="full")
    k2, v2 = update_cache(l, s, kn, vn, kc, vc)
    O2, _ = sparse_attn(l, s, qn, kn, vn, k2, v2, mode="full")
    np.testing.assert_allclose(O1, O2, atol=1e-14)
    # positions outside R_l keep their naive values
    outside = np.setdiff1d(np.arange(T), s.R[l])
    assert np.array_equal(k2[:, outside], kc[:, outside])


# ----------------------------------------------------------------------------
# matched-target variants: RelaxKV^G and the global repair target sweep
# ----------------------------------------------------------------------------

def test_global_scores_closed_form_and_loops():
    from oracle import global_scores
    a = np.array([[0.0, 1.0, 0.5, 0.25], [1.0, 0.0, 0.5, 0.75]])
    assert global_scores(a).tolist() == [0.5, 0.5, 0.5, 0.5]
    rng = np.random.default_rng(21)
    a = rng.random((7, 31))
    g = global_scores(a)
    for i in range(31):
        assert g[i] == pytest.approx(math.fsum(a[l, i] for l in range(7)) / 7, abs=1e-15)


@pytest.mark.parametrize("r,T,nU,n", [
    (0.2, 1000, 500, 200), (0.2, 1000, 150, 150), (0.15, 1001, 999, 150),   # floor(150.15)
    (0.0, 64, 10, 0), (1.0, 64, 40, 40), (0.7, 10, 10, 7), (0.05, 19, 19, 0),
])
def test_global_target_count_floor_and_cap(r, T, nU, n):
    from oracle import global_target_count
    assert global_target_count(r, T, nU) == n


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 50), st.integers(0, 2**31 - 1), st.data())
def test_select_global_brute_force_with_ties(T, seed, data):
    from oracle import select_global
    rng = np.random.default_rng(seed)
    g = rng.integers(0, 4, size=T) / 4.0                      # many equal values
    n = data.draw(st.integers(0, T))
    order = sorted(range(T), key=lambda i: (-g[i], i))        # larger g first, then lower i
    assert select_global(g, n).tolist() == sorted(order[:n])


def test_build_sets_global_equals_relaxkv_sets_for_identical_layers():
    # When every layer selects the same anchors S, RelaxKV's targets are R_l = S = U
    # for every layer, which is the matched-target variant with P = S.
    from oracle import build_sets_global
    rng = np.random.default_rng(22)
    L, T, k = 4, 50, 9
    S1 = np.sort(rng.choice(T, size=k, replace=False))
    S = np.tile(S1, (L, 1))
    a, b = build_sets(S, T), build_sets_global(S, T, S1)
    assert a.U.tolist() == b.U.tolist() and a.h.tolist() == b.h.tolist()
    assert a.cidx.tolist() == b.cidx.tolist()
    for l in range(L):
        for f in ("R", "R_u", "src"):
            assert getattr(a, f)[l].tolist() == getattr(b, f)[l].tolist()
    assert a.edges.tolist() == b.edges.tolist() and a.edges_full.tolist() == b.edges_full.tolist()


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 4), st.integers(1, 40), st.integers(0, 2**31 - 1), st.data())
def test_build_sets_global_brute_force(L, T, seed, data):
    from oracle import build_sets_global
    rng = np.random.default_rng(seed)
    k = data.draw(st.integers(1, T))
    S = _random_anchors(rng, L, T, k)
    n = data.draw(st.integers(0, T))
    P = np.sort(rng.choice(T, size=n, replace=False))
    s = build_sets_global(S, T, P)
    U = sorted(set(int(x) for row in S for x in row))
    assert s.U.tolist() == U
    for l in range(L):
        assert s.R[l].tolist() == P.tolist()
        for t, p in enumerate(P.tolist()):
            assert s.R_u[l][t] == sum(1 for j in U if j <= p) - 1     # -1: empty context
        for c, pos in enumerate(U):
            assert s.src[l][c] == (P.tolist().index(pos) if pos in P.tolist() else -1)
        assert s.edges[l] == sum(sum(1 for j in U if j <= p) for p in P.tolist())
        assert s.edges_full[l] == sum(p + 1 for p in P.tolist())
    for i in range(T):
        assert s.h[i] == (L - 1 if i in P.tolist() else -1)
    with pytest.raises(ValueError):
        build_sets_global(S, T, np.array([1, 1]) if T > 1 else np.array([0, 0]))


def _brute_attention_global(P, U, T, qn, kn, vn, kc, vc, sigma, mode):
    """Dense masked attention for a global target list: target p sees
    j in U with j <= p (union) or j <= p (full); fresh row iff j in P."""
    rank = {p: t for t, p in enumerate(P)}
    H, d = qn.shape[1], qn.shape[2]
    G = H // kc.shape[0]
    O = np.zeros((len(P), H, d))
    lse = np.full((len(P), H), -np.inf)
    for t, p in enumerate(P):
        for hh in range(H):
            g = hh // G
            terms = []
            for j in range(T):
                if not ((j in U and j <= p) if mode == "union" else (j <= p)):
                    continue
                kj = kn[rank[j], g] if j in rank else kc[g, j]
                vj = vn[rank[j], g] if j in rank else vc[g, j]
                terms.append((sigma * float(np.dot(qn[t, hh], kj)), vj))
            if not terms:
                continue                                  # empty sum: O = 0, lse = -inf
            m = max(x for x, _ in terms)
            w = [math.exp(x - m) for x, _ in terms]
            z = math.fsum(w)
            O[t, hh] = sum(wi * vj for wi, (_, vj) in zip(w, terms)) / z
            lse[t, hh] = m + math.log(z)
    return O, lse


@pytest.mark.parametrize("seed,mode", [(0, "union"), (1, "full"), (2, "union")])
def test_attention_global_targets_brute_force(seed, mode):
    from oracle import build_sets_global
    rng = np.random.default_rng(30 + seed)
    L, T, H, H_kv, d = 3, 36, 4, 2, 8
    S = 1 + _random_anchors(rng, L, T - 1, 5)          # position 0 is never in U
    U = sorted(set(int(x) for row in S for x in row))
    # targets inside and outside U, including position 0 (empty context)
    P = sorted(set([0] + rng.choice(T, size=10, replace=False).tolist()))
    s = build_sets_global(S, T, np.array(P))
    assert s.R_u[0][0] == -1
    n = len(P)
    qn = rng.standard_normal((n, H, d))
    kn = rng.standard_normal((n, H_kv, d))
    vn = rng.standard_normal((n, H_kv, d))
    kc = rng.standard_normal((H_kv, T, d))
    vc = rng.standard_normal((H_kv, T, d))
    for l in range(L):
        O, lse = sparse_attn(l, s, qn, kn, vn, kc, vc, mode=mode)
        Ob, lseb = _brute_attention_global(P, set(U), T, qn, kn, vn, kc, vc, 1 / math.sqrt(d), mode)
        np.testing.assert_allclose(O, Ob, atol=1e-12)
        np.testing.assert_array_equal(np.isinf(lse), np.isinf(lseb))
        fin = np.isfinite(lseb)
        np.testing.assert_allclose(lse[fin], lseb[fin], atol=1e-12)


def test_attention_empty_context_is_empty_sum():
    from oracle import build_sets_global
    T, H, H_kv, d = 10, 2, 1, 4
    S = np.array([[4, 7], [5, 7]])                 # U = {4, 5, 7}
    s = build_sets_global(S, T, np.array([1, 3, 6]))
    assert s.R_u[0].tolist() == [-1, -1, 1]
    rng = np.random.default_rng(5)
    qn, kn, vn = (rng.standard_normal((3, hh, d)) for hh in (H, H_kv, H_kv))
    kc, vc = (rng.standard_normal((H_kv, T, d)) for _ in range(2))
    O, lse = sparse_attn(0, s, qn, kn, vn, kc, vc)
    assert np.all(O[:2] == 0.0) and np.all(lse[:2] == -np.inf)
    # target 6 sees positions 4 and 5 (cached rows: neither is a target)
    for hh in range(H):
        x = kc[0, [4, 5]] @ qn[2, hh] / math.sqrt(d)
        w = np.exp(x - x.max())
        np.testing.assert_allclose(O[2, hh], (w / w.sum()) @ vc[0, [4, 5]], atol=1e-13)


def test_global_scores_f32_rounding():
    from oracle import global_scores, global_scores_f32
    a = np.array([[0.5, 0.25, 1.0], [0.125, 0.75, 0.0], [0.375, 0.0, 0.5]], dtype=np.float32)
    # sums of multiples of 1/8 are exact in fp32; only the division rounds
    assert global_scores_f32(a).tolist() == np.float32([1.0 / 3, 1.0 / 3, 0.5]).tolist()
    rng = np.random.default_rng(23)
    a = rng.random((40, 500)).astype(np.float32)
    g32 = global_scores_f32(a).astype(np.float64)
    g64 = global_scores(a.astype(np.float64))
    ulp = np.spacing(np.float32(1.0)).astype(np.float64)
    assert np.max(np.abs(g32 - g64)) <= 40 * ulp                 # L roundings of values <= 1
    assert global_scores_f32(a[:1]).tolist() == a[0].tolist()      # L = 1: the row itself


# ----------------------------------------------------------------------------
# context-construction variants (Global Sparse, Layerwise Sparse)
# ----------------------------------------------------------------------------

@settings(max_examples=50, deadline=None)
@given(st.integers(1, 4), st.integers(1, 40), st.integers(0, 2**31 - 1), st.data(),
       st.sampled_from(["union", "global", "layerwise"]))
def test_build_sets_context_brute_force(L, T, seed, data, construction):
    from oracle import build_sets_context
    rng = np.random.default_rng(seed)
    k = data.draw(st.integers(1, T))
    a = rng.integers(0, 5, size=(L, T)) / 4.0                   # ties across positions
    S = select(a, k)
    base = build_sets(S, T)
    s = build_sets_context(S, T, a, construction)
    n = len(base.U)
    for l in range(L):
        if construction == "union":
            want = base.U.tolist()
        else:
            sc = a.mean(axis=0) if construction == "global" else a[l]
            want = sorted(sorted(range(T), key=lambda i: (-sc[i], i))[:n])
        assert s.context(l).tolist() == want
        assert len(want) == n                                     # same set size |U|
        assert s.R[l].tolist() == base.R[l].tolist()              # targets unchanged
        for t, p in enumerate(s.R[l].tolist()):
            assert s.R_u[l][t] == sum(1 for j in want if j <= p) - 1
        rank = {p: t for t, p in enumerate(s.R[l].tolist())}
        assert s.src[l].tolist() == [rank.get(j, -1) for j in want]
        assert s.edges[l] == sum(sum(1 for j in want if j <= p) for p in s.R[l].tolist())
    assert s.edges_full.tolist() == base.edges_full.tolist()
    assert s.U.tolist() == base.U.tolist() and s.h.tolist() == base.h.tolist()
    if construction == "union":
        for l in range(L):
            assert s.R_u[l].tolist() == base.R_u[l].tolist()
            assert s.src[l].tolist() == base.src[l].tolist()
        assert s.edges.tolist() == base.edges.tolist()


def test_context_constructions_hand_example():
    # Worked by hand from the definitions (Sec. 4.4; ties to the lower position):
    # a_0 = [1, 0, .7, 0, 0, 0], a_1 = [0, .9, 0, 0, 1, 0], k = 1 -> S_0 = {0},
    # S_1 = {4}, U = {0, 4}, h = (0 at 0, 1 at 4), R_0 = {0, 4}, R_1 = {4}.
    # Global Sparse: g = [.5, .45, .35, 0, .5, 0], top-2 = {0, 4} (0 and 4 tie at
    # .5, both taken).  Layerwise Sparse: layer 0 top-2 of a_0 = {0, 2}; layer 1
    # top-2 of a_1 = {1, 4}.  R_u = |U_l cap {j <= p}| - 1, src = rank in R_l.
    from oracle import build_sets_context
    a = np.array([[1, 0, 0.7, 0, 0, 0], [0, 0.9, 0, 0, 1, 0]])
    S = np.array([[0], [4]])
    g = build_sets_context(S, 6, a, "global")
    assert [c.tolist() for c in g.ctx] == [[0, 4], [0, 4]]
    assert [r.tolist() for r in g.R_u] == [[0, 1], [1]]
    assert [x.tolist() for x in g.src] == [[0, 1], [-1, 0]]
    assert g.edges.tolist() == [3, 2]
    lw = build_sets_context(S, 6, a, "layerwise")
    assert [c.tolist() for c in lw.ctx] == [[0, 2], [1, 4]]
    assert [r.tolist() for r in lw.R_u] == [[0, 1], [1]]
    assert [x.tolist() for x in lw.src] == [[0, -1], [-1, 0]]
    assert lw.edges.tolist() == [3, 2]
    assert [r.tolist() for r in lw.R] == [[0, 4], [4]] and lw.U.tolist() == [0, 4]


def test_context_global_equals_layerwise_for_identical_layers():
    from oracle import build_sets_context
    rng = np.random.default_rng(24)
    L, T = 3, 60
    a = np.tile(rng.random(T), (L, 1))
    S = select(a, 7)
    g, lw = build_sets_context(S, T, a, "global"), build_sets_context(S, T, a, "layerwise")
    for l in range(L):
        assert g.context(l).tolist() == lw.context(l).tolist()
        assert g.R_u[l].tolist() == lw.R_u[l].tolist()


@pytest.mark.parametrize("construction,mode", [("global", "union"), ("layerwise", "union"),
                                               ("layerwise", "full")])
def test_attention_context_variants_brute_force(construction, mode):
    from oracle import build_sets_context
    rng = np.random.default_rng(40)
    L, T, H, H_kv, d = 3, 40, 4, 2, 8
    a = rng.random((L, T))
    S = select(a, 5)
    s = build_sets_context(S, T, a, construction)
    kc = rng.standard_normal((H_kv, T, d))
    vc = rng.standard_normal((H_kv, T, d))
    sigma = 1 / math.sqrt(d)
    for l in range(L):
        R = s.R[l].tolist()
        n = len(R)
        qn, kn, vn = (rng.standard_normal((n, hh, d)) for hh in (H, H_kv, H_kv))
        O, lse = sparse_attn(l, s, qn, kn, vn, kc, vc, mode=mode)
        ctx = set(s.context(l).tolist())
        rank = {p: t for t, p in enumerate(R)}
        for t, p in enumerate(R):
            for hh in range(H):
                g = hh // (H // H_kv)
                terms = []
                for j in range(T):
                    if not ((j in ctx and j <= p) if mode == "union" else j <= p):
                        continue
                    kj = kn[rank[j], g] if j in rank else kc[g, j]
                    vj = vn[rank[j], g] if j in rank else vc[g, j]
                    terms.append((sigma * float(qn[t, hh] @ kj), vj))
                if not terms:
                    assert np.all(O[t, hh] == 0) and lse[t, hh] == -np.inf
                    continue
                m = max(x for x, _ in terms)
                w = [math.exp(x - m) for x, _ in terms]
                ref = sum(wi * vj for wi, (_, vj) in zip(w, terms)) / math.fsum(w)
                np.testing.assert_allclose(O[t, hh], ref, atol=1e-12)
                assert lse[t, hh] == pytest.approx(m + math.log(math.fsum(w)), abs=1e-12)


# ----------------------------------------------------------------------------
# query-side completion: query tokens over the cache and causally over themselves
# ----------------------------------------------------------------------------

def test_query_attn_matches_sdpa_with_offset_causal_mask():
    from oracle import query_attn
    rng = np.random.default_rng(60)
    T, Qn, H, H_kv, d = 23, 6, 6, 2, 16
    q = rng.standard_normal((Qn, H, d))
    kc, vc = rng.standard_normal((H_kv, T, d)), rng.standard_normal((H_kv, T, d))
    kq, vq = rng.standard_normal((Qn, H_kv, d)), rng.standard_normal((Qn, H_kv, d))
    O, lse = query_attn(q, kc, vc, kq, vq)
    K = torch.cat([torch.from_numpy(kc), torch.from_numpy(kq).permute(1, 0, 2)], dim=1)   # [H_kv][T+Qn][d]
    V = torch.cat([torch.from_numpy(vc), torch.from_numpy(vq).permute(1, 0, 2)], dim=1)
    mask = torch.arange(T + Qn)[None, :] <= (T + torch.arange(Qn))[:, None]               # [Qn][T+Qn]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2)[None], K[None], V[None], attn_mask=mask,
        enable_gqa=True)
    np.testing.assert_allclose(O, ref[0].permute(1, 0, 2).numpy(), atol=1e-12)
    Kh = K.repeat_interleave(H // H_kv, dim=0)                                             # [H][T+Qn][d]
    logits = torch.einsum("htd,hkd->htk", torch.from_numpy(q).permute(1, 0, 2), Kh) / math.sqrt(d)
    logits = logits.masked_fill(~mask[None], float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(logits, -1).permute(1, 0).numpy(), atol=1e-12)


def test_query_attn_brute_force_and_normalisation():
    from oracle import query_attn
    rng = np.random.default_rng(61)
    T, Qn, H, H_kv, d = 9, 4, 2, 1, 4
    q = rng.standard_normal((Qn, H, d))
    kc, vc = rng.standard_normal((H_kv, T, d)), rng.standard_normal((H_kv, T, d))
    kq, vq = rng.standard_normal((Qn, H_kv, d)), rng.standard_normal((Qn, H_kv, d))
    O, lse = query_attn(q, kc, vc, kq, vq, softmax_scale=0.3)
    for t in range(Qn):
        for h in range(H):
            keys = [kc[0, j] for j in range(T)] + [kq[u, 0] for u in range(t + 1)]
            vals = [vc[0, j] for j in range(T)] + [vq[u, 0] for u in range(t + 1)]
            x = [0.3 * float(np.dot(q[t, h], k)) for k in keys]
            z = math.fsum(math.exp(v) for v in x)
            assert lse[t, h] == pytest.approx(math.log(z), abs=1e-12)
            ref = sum(math.exp(xi) / z * vi for xi, vi in zip(x, vals))
            np.testing.assert_allclose(O[t, h], ref, atol=1e-12)
            # the cache keys' share plus the query prefix's share is 1
            cache_mass = math.fsum(math.exp(xi - lse[t, h]) for xi in x[:T])
            prefix_mass = math.fsum(math.exp(xi - lse[t, h]) for xi in x[T:])
            assert cache_mass + prefix_mass == pytest.approx(1.0, abs=1e-12)
