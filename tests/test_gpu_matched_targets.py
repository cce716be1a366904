"""GPU parity of the matched-target variants against the float64 oracle:
RelaxKV^G (a global target list P for every layer with the union context,
Sec. 4.1 / App. A.3 table) and the global repair target sweep (App. B:
g = layer mean of a, P = TopK(g, min(floor(r_g T_c), |U|))).

Bars as for the main path: g within fp32 rounding of the oracle's mean of the
same fp32 scores; P and every set array bit-exact; attention outputs within
2e-2 max-abs (bf16) / 1e-5 relative (fp32); targets with an empty context give
O = 0 and lse = -inf exactly; the cache update is bit-exact.
"""

import numpy as np
import pytest
import torch

import oracle
from harness import assert_close, Case, every_target_property, synthetic_scores
from paper_2609_33503_amd import relaxkv, synth

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
SMALL = {
    "tiny": W["tiny-2L-1k-fp32"],
    "qwen-planted": synth.shrink(W["qwen14b-32k-planted"], L=4, T_c=2600),
    "d64-bf16": synth.shrink(W["llama8b-8k"], L=2, T_c=777, H=8, H_kv=2, d=64, Qn=24),
}


def _dev_i32(x):
    return torch.as_tensor(np.asarray(x, dtype=np.int32)).cuda()


def gpu_global_sets(case, P, n=None):
    """Build the global-target sets on the GPU from a host list P."""
    T = case.T
    t = torch.zeros(T, dtype=torch.int32, device="cuda")
    t[:len(P)] = _dev_i32(P) if len(P) else t[:0]
    nt = _dev_i32([len(P) if n is None else n])
    case.req.build_sets_global(case.sets, t, nt)
    counts, edges = case.sets.counts_to_host()
    L = case.L
    nU = counts[0]
    R_off = case.sets.R_off.cpu().numpy()
    R_idx = case.sets.R_idx.cpu().numpy()
    R_u = case.sets.R_u.cpu().numpy()
    src = case.sets.src.cpu().numpy()
    return dict(counts=counts, edges=edges, h=case.sets.h.cpu().numpy(),
                U=case.sets.U.cpu().numpy()[:nU], cidx=case.sets.cidx.cpu().numpy(),
                R=[R_idx[R_off[l]:R_off[l + 1]] for l in range(L)],
                R_u=[R_u[R_off[l]:R_off[l + 1]] for l in range(L)],
                src=[src[l, :nU] for l in range(L)], rank=case.sets.rank.cpu().numpy())


def compare_global_sets(got, ref):
    L = len(ref.R)
    assert got["h"].tolist() == ref.h.tolist()
    assert got["U"].tolist() == ref.U.tolist()
    assert got["cidx"].tolist() == ref.cidx.tolist()
    assert got["counts"][0] == len(ref.U)
    for l in range(L):
        assert got["counts"][1 + l] == len(ref.R[l])
        assert got["R"][l].tolist() == ref.R[l].tolist()
        assert got["R_u"][l].tolist() == ref.R_u[l].tolist()
        assert got["src"][l].tolist() == ref.src[l].tolist()
        rank = np.full(ref.T_c, -1)
        rank[ref.R[l]] = np.arange(len(ref.R[l]))
        assert got["rank"][l].tolist() == rank.tolist()
        assert got["edges"][l] == int(ref.edges[l])
        assert got["edges"][L + l] == int(ref.edges_full[l])
    assert got["counts"][L + 1] == 0


def _anchors_and_sets(case, seed):
    """Oracle anchors of seeded fp32 scores; the GPU selects the same anchors."""
    a = synthetic_scores(case.L, case.T, seed=seed)
    anchors = oracle.select(a.astype(np.float64), case.k)
    got = case.gpu_select(torch.from_numpy(a).cuda())
    assert np.array_equal(got, anchors)
    return a, anchors


def _compare_attn(case, out, lse, O_ref, lse_ref, what):
    empty = np.isneginf(lse_ref[:, 0])
    got_O = out.float().cpu().numpy()
    got_lse = lse.cpu().numpy()
    assert np.all(got_O[empty] == 0.0), what
    assert np.all(np.isneginf(got_lse[empty])), what
    if (~empty).any():
        assert_close(got_O[~empty], O_ref[~empty], case.w, what,
                     rel_gate=1e-2 if case.w.dtype == "bf16" else None)
        assert_close(got_lse[~empty], lse_ref[~empty], case.w, what + " lse")


@pytest.mark.parametrize("name", list(SMALL))
def test_select_global_matches_oracle(gpu_lib, name):
    case = Case(SMALL[name])
    a, anchors = _anchors_and_sets(case, seed=41)
    case.req.build_sets(case.sets)
    nU = len(oracle.build_sets(anchors, case.T).U)
    assert case.sets.counts_to_host()[0][0] == nU
    g = torch.empty(case.T, dtype=torch.float32, device="cuda")
    P = torch.empty(case.T, dtype=torch.int32, device="cuda")
    n = torch.empty(1, dtype=torch.int32, device="cuda")
    g_ref = oracle.global_scores(a.astype(np.float64))
    g32 = oracle.global_scores_f32(a)                    # the ranking precision
    for r in (0.2, 0.5, 1.0, 1e-4):
        case.req.select_global(torch.from_numpy(a).cuda(), r, case.sets, g, P, n)
        torch.cuda.synchronize()
        g_gpu = g.cpu().numpy()
        np.testing.assert_allclose(g_gpu, g_ref, rtol=0, atol=4e-7 * case.L)
        assert np.array_equal(g_gpu, g32)                # same fp32 operations in the same order
        n_ref = oracle.global_target_count(r, case.T, nU)
        assert int(n.item()) == n_ref
        P_ref = oracle.select_global(g32.astype(np.float64), n_ref)
        assert P.cpu().numpy()[:n_ref].tolist() == P_ref.tolist()


@pytest.mark.parametrize("name", list(SMALL))
def test_global_sets_and_attention(gpu_lib, name):
    """A caller's target list (RelaxKV^G) with positions inside and outside U,
    including positions before the first union position (empty contexts)."""
    case = Case(SMALL[name])
    _, anchors = _anchors_and_sets(case, seed=42)
    sref0 = oracle.build_sets(anchors, case.T)
    U = sref0.U
    rng = np.random.default_rng(43)
    P = set(rng.choice(case.T, size=max(1, case.T // 5), replace=False).tolist())
    P |= set(range(0, min(int(U[0]) + 1, case.T)))          # up to and including U[0]
    P = np.array(sorted(P), dtype=np.int64)
    ref = oracle.build_sets_global(anchors, case.T, P)
    compare_global_sets(gpu_global_sets(case, P), ref)
    for mode, cm in (("union", relaxkv.CONTEXT_UNION), ("full", relaxkv.CONTEXT_FULL)):
        for l in range(case.L):
            fresh = case.fresh(l, P)
            out, lse = case.gpu_attn(l, fresh, len(P), cm)
            O_ref, lse_ref = case.oracle_attn(l, ref, fresh, mode=mode)
            _compare_attn(case, out, lse, O_ref, lse_ref, f"{name} {mode} layer {l}")


def test_global_sets_empty_list_and_all_targets(gpu_lib):
    case = Case(SMALL["qwen-planted"])
    _, anchors = _anchors_and_sets(case, seed=44)
    for P in (np.zeros(0, dtype=np.int64), np.arange(case.T)):
        ref = oracle.build_sets_global(anchors, case.T, P)
        compare_global_sets(gpu_global_sets(case, P), ref)
    # every position a target: union attention equals the oracle's on all rows
    fresh = case.fresh(1, np.arange(case.T))
    out, lse = case.gpu_attn(1, fresh, case.T)
    O_ref, lse_ref = case.oracle_attn(1, ref, fresh)
    _compare_attn(case, out, lse, O_ref, lse_ref, "all targets")


def test_global_sets_reject_invalid_lists(gpu_lib):
    case = Case(SMALL["tiny"])
    _, anchors = _anchors_and_sets(case, seed=45)
    T = case.T
    for P, n in (([5, 3, 9], None), ([1, 1, 2], None), ([0, T], None), ([-1, 4], None),
                 ([1, 2], T + 1), ([1, 2], -1)):
        with pytest.raises(relaxkv.RelaxKVError) as e:
            gpu_global_sets(case, P, n)
        assert e.value.status == relaxkv.EINVAL
        # every index written stays in range
        n_written = int(case.sets.R_off.cpu().numpy()[case.L])
        R_idx = case.sets.R_idx.cpu().numpy()[:n_written]
        assert n_written <= case.L * T
        assert R_idx.size == 0 or (R_idx.min() >= 0 and R_idx.max() < T)
    # the error word clears at the next selection; a valid list then builds
    case.gpu_select(torch.from_numpy(synthetic_scores(case.L, T, seed=45)).cuda())
    ref = oracle.build_sets_global(anchors, T, np.array([2, 7, 40]))
    compare_global_sets(gpu_global_sets(case, [2, 7, 40]), ref)
    # back to RelaxKV's own targets
    case.req.build_sets(case.sets)
    assert case.sets.s.global_targets == 0
    case.sets.counts_to_host()


@pytest.mark.parametrize("name", ["qwen-planted", "tiny"])
def test_global_update_cache_bit_exact(gpu_lib, name):
    case = Case(SMALL[name])
    _, anchors = _anchors_and_sets(case, seed=46)
    P = np.sort(np.random.default_rng(47).choice(case.T, size=case.T // 3, replace=False))
    ref = oracle.build_sets_global(anchors, case.T, P)
    compare_global_sets(gpu_global_sets(case, P), ref)
    k_out, v_out = case.kc.clone(), case.vc.clone()
    for l in range(case.L):
        _, kn, vn = case.fresh(l, P)
        case.req.update_cache(case.sets, l, kn, vn, k_out, v_out)
        torch.cuda.synchronize()
        kr, vr = oracle.update_cache(l, ref, synth.to_f64(kn), synth.to_f64(vn),
                                     synth.to_f64(case.kc[l]), synth.to_f64(case.vc[l]))
        assert np.array_equal(synth.to_f64(k_out[l]), kr)
        assert np.array_equal(synth.to_f64(v_out[l]), vr)


def test_full_size_global_target_sweep(gpu_lib):
    """The 32K planted workload: seeded fp32 scores drive both sides, anchors at
    r = 0.15, P_{r_g} at r_g = 0.2 and the Target-Union cap (r_g = 1), sets
    bit-exact and attention on sampled targets of sampled layers, as the
    benchmark runs it."""
    w = W["qwen14b-32k-planted"]
    case = Case(w)
    a_np = synthetic_scores(w.L, w.T_c, seed=49)
    a = torch.from_numpy(a_np).cuda()
    anchors = oracle.select(a_np.astype(np.float64), case.k)
    assert np.array_equal(case.gpu_select(a), anchors)
    case.req.build_sets(case.sets)
    nU = len(oracle.build_sets(anchors, case.T).U)
    assert case.sets.counts_to_host()[0][0] == nU
    g32 = oracle.global_scores_f32(a_np)
    g = torch.empty(case.T, dtype=torch.float32, device="cuda")
    P = torch.empty(case.T, dtype=torch.int32, device="cuda")
    n = torch.empty(1, dtype=torch.int32, device="cuda")
    rng = np.random.default_rng(48)
    for r in (0.2, 1.0):
        case.req.select_global(a, r, case.sets, g, P, n)
        torch.cuda.synchronize()
        g_gpu = g.cpu().numpy()
        np.testing.assert_allclose(g_gpu, oracle.global_scores(a_np.astype(np.float64)),
                                   rtol=0, atol=4e-7 * case.L)
        assert np.array_equal(g_gpu, g32)
        n_ref = oracle.global_target_count(r, case.T, nU)
        P_ref = oracle.select_global(g32.astype(np.float64), n_ref)
        assert int(n.item()) == n_ref
        assert P.cpu().numpy()[:n_ref].tolist() == P_ref.tolist()
        case.req.build_sets_global(case.sets, P, n)
        ref = oracle.build_sets_global(anchors, case.T, P_ref)
        got = gpu_global_sets(case, P_ref)
        compare_global_sets(got, ref)
        for l in (0, w.L - 1):
            fresh = case.fresh(l, P_ref)
            out, lse = case.gpu_attn(l, fresh, n_ref)
            ts = sorted(set([0, 1, n_ref // 2, n_ref - 1] + rng.integers(0, n_ref, size=6).tolist()))
            O_ref, lse_ref = case.oracle_attn(l, ref, fresh, targets=ts)
            _compare_attn(case, out[ts], lse[ts], O_ref, lse_ref, f"32K r_g={r} layer {l}")
        every_target_property(case, ref, w.L - 1, "union")     # every target of the last layer
