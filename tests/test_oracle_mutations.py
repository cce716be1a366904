"""The oracle's pins catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of the oracle's source (a dropped
scale, a flipped tie-break, an off-by-one causal limit, a fresh/cached swap,
...), loads the copy as a module of its own, points the pin tests of
test_oracle_pins at it, and requires the case's first named pin (a
deterministic one) to fail.
The oracle itself is never modified; every planted mistake must match its
site in the source exactly once, so an edit of the oracle cannot turn a case
into a silent no-op.  CPU only.
"""

from __future__ import annotations

import os
import sys
import types

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "relaxkv_oracle.py")
EXPORTS = ("anchor_count", "attention_flops", "build_sets", "build_sets_context",
           "build_sets_global", "global_scores", "global_scores_f32", "global_target_count",
           "query_attn", "score", "select", "select_global", "sparse_attn", "update_cache")

# (name, text in the oracle, planted text, pins).  A pin is a test function of
# test_oracle_pins, or (function, kwargs).  The first pin of every case is
# deterministic (no hypothesis draw) and must fail; the others are further
# pins that bear on the same definition (they run on the real oracle below).
MUTANTS = [
    ("score: softmax scale dropped",
     "s = sigma * (q[l, :, h, :] @ k_cache[l, g].T)",
     "s = (q[l, :, h, :] @ k_cache[l, g].T)",
     ["test_score_matches_sdpa_attention_weights", "test_score_closed_form_logs"]),
    ("score: query head h read against KV head h mod H_kv",
     "            g = h // G\n            s = sigma * (q[l, :, h, :]",
     "            g = h % H_kv\n            s = sigma * (q[l, :, h, :]",
     ["test_score_matches_brute_force_loops", "test_score_degenerate_minmax_and_gqa_sharing"]),
    ("score: MinMax normalisation dropped",
     "a[l] = (p[l] - lo) / (hi - lo)", "a[l] = p[l]",
     ["test_score_closed_form_logs", "test_score_matches_brute_force_loops"]),
    ("score: pooled mass divided by H only",
     "p /= H * Qn", "p /= H",
     ["test_score_pooled_mass_is_one", "test_score_matches_brute_force_loops"]),
    ("score: supplied row normaliser ignored",
     "A = np.exp(s - np.asarray(row_lse, np.float64)[l, :, h][:, None])",
     "A = np.exp(s - m) / z",
     ["test_score_supplied_lse"]),
    ("anchor_count: round half up",
     "k = max(1, int(round(ratio * T_c)))",
     "k = max(1, int(np.floor(ratio * T_c + 0.5)))",
     [("test_anchor_count_closed_forms", dict(r=0.125, T=20, k=2)),
      ("test_anchor_count_closed_forms", dict(r=0.625, T=4, k=2))]),
    ("anchor_count: no floor of one anchor",
     "k = max(1, int(round(ratio * T_c)))", "k = max(0, int(round(ratio * T_c)))",
     [("test_anchor_count_closed_forms", dict(r=0.0, T=50, k=1))]),
    ("select: highest position wins a tie",
     "order = np.lexsort((pos, -a[l]))", "order = np.lexsort((-pos, -a[l]))",
     ["test_score_equal_keys_select_first_k", "test_select_brute_force_with_ties"]),
    ("select: lowest scores taken",
     "order = np.lexsort((pos, -a[l]))", "order = np.lexsort((pos, a[l]))",
     ["test_hand_example_select_and_sets", "test_select_brute_force_with_ties"]),
    ("build_sets: h is the lowest selecting layer",
     "h[anchors[l]] = np.maximum(h[anchors[l]], l)",
     "h[anchors[l]] = np.where(h[anchors[l]] < 0, l, np.minimum(h[anchors[l]], l))",
     ["test_hand_example_select_and_sets", "test_sets_invariants"]),
    ("build_sets: R_l drops the targets whose highest layer is l",
     "R_l = U[h[U] >= l]", "R_l = U[h[U] > l]",
     ["test_hand_example_select_and_sets", "test_sets_invariants"]),
    ("build_sets: edge count one short per target",
     "edges[l] = int(np.sum(u_l + 1))", "edges[l] = int(np.sum(u_l))",
     ["test_hand_example_select_and_sets", "test_sets_invariants"]),
    ("sparse_attn: a target does not see its own key",
     'm = int(np.searchsorted(ctx_all, p, side="right"))',
     'm = int(np.searchsorted(ctx_all, p, side="left"))',
     ["test_hand_example_attention", "test_attention_full_union_is_causal_sdpa",
      ("test_attention_brute_force", dict(seed=0, L=3, T=40, k=6, mode="union"))]),
    ("sparse_attn: cached keys and values for the active targets",
     "    Kt[:, fresh, :] = np.transpose(k_new[rank[ctx_all[fresh]]], (1, 0, 2))\n"
     "    Vt[:, fresh, :] = np.transpose(v_new[rank[ctx_all[fresh]]], (1, 0, 2))\n",
     "",
     ["test_hand_example_attention", "test_attention_full_union_is_causal_sdpa",
      ("test_attention_brute_force", dict(seed=0, L=3, T=40, k=6, mode="union"))]),
    ("sparse_attn: fresh values but cached keys",
     "    Kt[:, fresh, :] = np.transpose(k_new[rank[ctx_all[fresh]]], (1, 0, 2))\n", "",
     ["test_attention_full_union_is_causal_sdpa", "test_hand_example_attention",
      ("test_attention_brute_force", dict(seed=0, L=3, T=40, k=6, mode="union"))]),
    ("sparse_attn: query head h read against KV head h mod H_kv",
     "            g = h // G\n            s = sigma * (Kt[g, :m, :] @ q_new[t, h])",
     "            g = h % H_kv\n            s = sigma * (Kt[g, :m, :] @ q_new[t, h])",
     ["test_attention_full_union_is_causal_sdpa",
      ("test_attention_brute_force", dict(seed=0, L=3, T=40, k=6, mode="union"))]),
    ("sparse_attn: the full-prefix mode attends over the union",
     'ctx_all = np.arange(sets.T_c)', 'ctx_all = sets.context(layer)',
     [("test_attention_brute_force", dict(seed=2, L=3, T=40, k=6, mode="full")),
      "test_attention_full_union_is_causal_sdpa"]),
    ("attention_flops: one product per edge instead of two",
     "return 4.0 * H * d * float(np.sum(edges))", "return 2.0 * H * d * float(np.sum(edges))",
     ["test_attention_flops_hand_example", "test_attention_flops_brute_force"]),
    ("query_attn: no causal mask among the query tokens",
     "m = T_c + t + 1", "m = T_c + Qn",
     ["test_query_attn_matches_sdpa_with_offset_causal_mask",
      "test_query_attn_brute_force_and_normalisation"]),
    ("query_attn: a query token does not see its own key",
     "m = T_c + t + 1", "m = T_c + t",
     ["test_query_attn_matches_sdpa_with_offset_causal_mask",
      "test_query_attn_brute_force_and_normalisation"]),
    ("update_cache: values not written",
     "        v[:, p, :] = v_new[t]\n", "",
     ["test_update_cache_hand_example",
      "test_update_cache_then_full_prefix_attention_reads_fresh_rows"]),
    ("global_scores: layer sum instead of layer mean",
     "return a.sum(axis=0) / a.shape[0]", "return a.sum(axis=0)",
     ["test_global_scores_closed_form_and_loops", "test_global_scores_f32_rounding"]),
    ("global_target_count: rounded instead of floored",
     "return min(int(np.floor(ratio * T_c)), int(n_union))",
     "return min(int(np.round(ratio * T_c)), int(n_union))",
     [("test_global_target_count_floor_and_cap", dict(r=0.05, T=19, nU=19, n=0)),
      ("test_global_target_count_floor_and_cap", dict(r=0.2, T=1000, nU=500, n=200))]),
    ("global_target_count: not capped by |U|",
     "return min(int(np.floor(ratio * T_c)), int(n_union))",
     "return int(np.floor(ratio * T_c))",
     [("test_global_target_count_floor_and_cap", dict(r=0.2, T=1000, nU=150, n=150)),
      ("test_global_target_count_floor_and_cap", dict(r=1.0, T=64, nU=40, n=40))]),
    ("build_sets_global: a target does not see its own key",
     "n_le = np.array([int(np.count_nonzero(U <= p)) for p in P], dtype=np.int64)",
     "n_le = np.array([int(np.count_nonzero(U < p)) for p in P], dtype=np.int64)",
     ["test_build_sets_global_equals_relaxkv_sets_for_identical_layers",
      "test_build_sets_global_brute_force"]),
    ("build_sets_global: targets marked active at layer 0 only",
     "h[P] = L - 1", "h[P] = 0",
     ["test_build_sets_global_equals_relaxkv_sets_for_identical_layers",
      "test_build_sets_global_brute_force"]),
    ("build_sets_context: Global Sparse ranks by layer 0 instead of the layer mean",
     "shared = select_global(global_scores(a) if g is None else g, n)",
     "shared = select_global(a[0] if g is None else g, n)",
     ["test_context_constructions_hand_example", "test_build_sets_context_brute_force"]),
    ("build_sets_context: Layerwise Sparse uses layer 0 for every layer",
     "ctx = [select(a[l:l + 1], n)[0] for l in range(L)]",
     "ctx = [select(a[0:1], n)[0] for l in range(L)]",
     ["test_context_constructions_hand_example", "test_build_sets_context_brute_force"]),
]


def _mutant(monkeypatch, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, f"planted site matches {text.count(old)} times: {old!r}"
    mod = types.ModuleType("relaxkv_oracle_mutant")
    mod.__file__ = SRC
    monkeypatch.setitem(sys.modules, mod.__name__, mod)   # dataclasses look their module up
    exec(compile(text.replace(old, new), SRC + " (mutant)", "exec"), mod.__dict__)
    return mod


def _run(pin):
    name, kw = (pin, {}) if isinstance(pin, str) else pin
    getattr(pins, name)(**kw)


@pytest.mark.parametrize("name,old,new,catchers", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, old, new, catchers):
    first = catchers[0] if isinstance(catchers[0], str) else catchers[0][0]
    assert not hasattr(getattr(pins, first), "hypothesis"), "the first pin must be deterministic"
    mod = _mutant(monkeypatch, old, new)
    for sym in EXPORTS:
        monkeypatch.setattr(oracle, sym, getattr(mod, sym))      # `from oracle import` inside pins
        if hasattr(pins, sym):
            monkeypatch.setattr(pins, sym, getattr(mod, sym))    # names bound at import
    try:
        _run(catchers[0])
    except Exception:                # the pin failed (an assertion, or an error inside the mutant)
        return
    pytest.fail(f"the pin {catchers[0]} did not catch the planted mistake {name!r}")


@pytest.mark.parametrize("pin", sorted({p if isinstance(p, str) else (p[0], tuple(sorted(p[1].items())))
                                        for m in MUTANTS for p in m[3]}, key=str),
                         ids=str)
def test_named_pins_pass_on_the_oracle(pin):
    """Every pin named above passes on the unmodified oracle, so a catch above
    is the planted mistake's doing."""
    _run(pin if isinstance(pin, str) else (pin[0], dict(pin[1])))
