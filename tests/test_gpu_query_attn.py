"""GPU parity of the query-side completion (the query prefill after repair,
App. C.4) against the float64 oracle: the query tokens attend to every cache
position and causally to themselves; outputs within 2e-2 max-abs (bf16) or
1e-5 relative (fp32), the row log-sum-exp likewise, at small sizes with ragged
splits and at the 32K workload in the launch configuration the benchmark
times.  The emitted log-sum-exp then drives the one-pass scoring mode.
"""

import numpy as np
import pytest
import torch

import oracle
from harness import Case, assert_close, synthetic_scores
from paper_2609_33503_amd import relaxkv, synth

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
SMALL = {
    "tiny": W["tiny-2L-1k-fp32"],
    "llama-shape": synth.shrink(W["llama8b-8k"], L=2, T_c=1500),
    "qwen-shape": synth.shrink(W["qwen14b-16k"], L=2, T_c=2100),
    "d64-bf16": synth.shrink(W["llama8b-8k"], L=2, T_c=777, H=8, H_kv=2, d=64, Qn=24),
    "mha-bf16": synth.shrink(W["llama8b-8k"], L=2, T_c=640, H=4, H_kv=4, Qn=8),
    "big-group": synth.shrink(W["llama8b-8k"], L=2, T_c=900, H=32, H_kv=2, Qn=40),   # 640 rows
    # 288 rows (nine 32-row blocks: the twelve-wave kernel with a padding block among
    # its key-half waves) and 320 rows at d = 64 (the twelve-wave kernel's d = 64 form)
    "rows288": synth.shrink(W["llama8b-8k"], L=2, T_c=1100, Qn=72),
    "rows320-d64": synth.shrink(W["qwen14b-16k"], L=2, T_c=1000, d=64),
    "fp32-d128": synth.shrink(W["tiny-2L-1k-fp32"], L=2, T_c=300, d=128, H=6, H_kv=3, Qn=5),
    # 320 rows (key-half waves) with a last split of 16 cache keys and 64 query tokens:
    # the key-half waves meet fully masked tiles before their first visible key
    "half-tail": synth.shrink(W["qwen14b-16k"], L=1, T_c=1040),
    # 32 key splits (the merge kernel for exactly 32) and 34 (the general merge)
    "splits32": synth.shrink(W["llama8b-8k"], L=1, T_c=8192, Qn=8),
    "many-splits": synth.shrink(W["llama8b-8k"], L=1, T_c=8500, H=4, H_kv=2, Qn=8),
}


def run_query(case, layer, kc=None, vc=None):
    w = case.w
    kq, vq = synth.make_query_kv(w, layer, "cuda")
    out = torch.empty(w.Qn, w.H, w.d, dtype=case.q.dtype, device="cuda")
    lse = torch.empty(w.Qn, w.H, dtype=torch.float32, device="cuda")
    ws = case.req.alloc_query_workspace()
    case.req.query_attn(layer, case.kc if kc is None else kc, case.vc if vc is None else vc,
                        kq, vq, out, lse, ws)
    torch.cuda.synchronize()
    return kq, vq, out, lse


def oracle_query(case, layer, kq, vq, kc=None, vc=None):
    kc = case.kc if kc is None else kc
    vc = case.vc if vc is None else vc
    return oracle.query_attn(synth.to_f64(case.q[layer]), synth.to_f64(kc[layer]),
                             synth.to_f64(vc[layer]), synth.to_f64(kq), synth.to_f64(vq))


@pytest.mark.parametrize("name", list(SMALL))
def test_query_attn_small(gpu_lib, name):
    case = Case(SMALL[name])
    for l in range(case.L):
        kq, vq, out, lse = run_query(case, l)
        O_ref, lse_ref = oracle_query(case, l, kq, vq)
        bf16 = case.w.dtype == "bf16"
        assert_close(out.float().cpu().numpy(), O_ref, case.w, f"{name} O layer {l}",
                     rel_gate=1e-2 if bf16 else None)
        assert_close(lse.cpu().numpy(), lse_ref, case.w, f"{name} lse layer {l}")


def test_query_attn_over_repaired_cache(gpu_lib):
    """After every layer's cache update, the query prefill reads the repaired
    rows (the oracle's repaired cache from the same fresh rows)."""
    case = Case(synth.shrink(W["qwen14b-32k-planted"], L=3, T_c=2600))
    a = synthetic_scores(case.L, case.T, seed=61)
    anchors = oracle.select(a.astype(np.float64), case.k)
    sets_ref = oracle.build_sets(anchors, case.T)
    case.req.select(torch.from_numpy(a).cuda(), case.sets)
    case.req.build_sets(case.sets)
    k_out, v_out = case.kc.clone(), case.vc.clone()
    k_ref, v_ref = {}, {}
    for l in range(case.L):
        _, kn, vn = case.fresh(l, sets_ref.R[l])
        case.req.update_cache(case.sets, l, kn, vn, k_out, v_out)
        k_ref[l], v_ref[l] = oracle.update_cache(l, sets_ref, synth.to_f64(kn), synth.to_f64(vn),
                                                 synth.to_f64(case.kc[l]), synth.to_f64(case.vc[l]))
    torch.cuda.synchronize()
    for l in range(case.L):
        kq, vq, out, lse = run_query(case, l, k_out, v_out)
        O_ref, lse_ref = oracle.query_attn(synth.to_f64(case.q[l]), k_ref[l], v_ref[l],
                                           synth.to_f64(kq), synth.to_f64(vq))
        assert_close(out.float().cpu().numpy(), O_ref, case.w, f"repaired O layer {l}",
                     rel_gate=1e-2)
        assert_close(lse.cpu().numpy(), lse_ref, case.w, f"repaired lse layer {l}")


def test_query_lse_drives_one_pass_scoring(gpu_lib):
    """The query prefill's row LSE as q_lse: one-pass scores match the oracle's
    scores with the oracle's own query-prefill LSE."""
    w = synth.shrink(W["qwen14b-16k"], L=2, T_c=2100)
    base = Case(w)
    lse_gpu = torch.empty(w.L, w.Qn, w.H, dtype=torch.float32, device="cuda")
    lse_ref = np.zeros((w.L, w.Qn, w.H))
    for l in range(w.L):
        kq, vq, _, lse = run_query(base, l)
        lse_gpu[l] = lse
        lse_ref[l] = oracle_query(base, l, kq, vq)[1]
    case = Case(w, q_lse=lse_gpu)
    a_gpu = case.gpu_scores().cpu().numpy()
    a_ref, _, _ = oracle.score(synth.to_f64(case.q), synth.to_f64(case.kc), row_lse=lse_ref)
    assert_close(a_gpu, a_ref, w, "scores from the query prefill's lse")


def test_query_attn_full_size(gpu_lib):
    """The 32K planted workload: two layers, every (token, head) checked."""
    w = W["qwen14b-32k-planted"]
    case = Case(w, layers=[0, w.L - 1])
    for i in range(case.L):
        kq, vq, out, lse = run_query(case, i)
        O_ref, lse_ref = oracle_query(case, i, kq, vq)
        assert_close(out.float().cpu().numpy(), O_ref, w, f"32K O {i}", rel_gate=1e-2)
        assert_close(lse.cpu().numpy(), lse_ref, w, f"32K lse {i}")
