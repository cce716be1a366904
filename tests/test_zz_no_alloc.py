"""The allocation-free query-side completion (relaxkv_query_attn_noalloc, for
callers that cannot allocate device memory) against the allocating entry point
(relaxkv_query_attn) and the float64 oracle: two calls in a row through the
library's per-GPU scratch, the second with a smaller problem, each equal bit for
bit to the allocating call and within the parity bar of the oracle."""

import pytest
import torch

import oracle
from harness import Case, assert_close
from paper_2609_33503_amd import relaxkv, synth

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
# the first problem uses more scratch than the second (more key splits, more rows)
BIG = synth.shrink(W["qwen14b-32k-planted"], L=2, T_c=5000)
SMALL = synth.shrink(W["llama8b-8k"], L=2, T_c=1300, H=16, H_kv=4, Qn=12)
FP32 = W["tiny-2L-1k-fp32"]


def _both(case, layer):
    w = case.w
    kq, vq = synth.make_query_kv(w, layer, "cuda")
    out_a = torch.empty(w.Qn, w.H, w.d, dtype=case.q.dtype, device="cuda")
    lse_a = torch.empty(w.Qn, w.H, dtype=torch.float32, device="cuda")
    case.req.query_attn(layer, case.kc, case.vc, kq, vq, out_a, lse_a,
                        case.req.alloc_query_workspace())
    out_n = torch.full_like(out_a, 3.0)
    lse_n = torch.full_like(lse_a, 3.0)
    case.req.query_attn_noalloc(layer, case.kc, case.vc, kq, vq, out_n, lse_n)
    torch.cuda.synchronize()
    return kq, vq, out_a, lse_a, out_n, lse_n


def _check(case, layer):
    w = case.w
    assert case.req.query_attn_workspace_bytes() <= relaxkv.QUERY_ATTN_NOALLOC_MAX_BYTES
    kq, vq, out_a, lse_a, out_n, lse_n = _both(case, layer)
    assert torch.equal(out_n, out_a)
    assert torch.equal(lse_n, lse_a)
    O_ref, lse_ref = oracle.query_attn(synth.to_f64(case.q[layer]), synth.to_f64(case.kc[layer]),
                                       synth.to_f64(case.vc[layer]), synth.to_f64(kq),
                                       synth.to_f64(vq))
    bf16 = w.dtype == "bf16"
    assert_close(out_n.float().cpu().numpy(), O_ref, w, f"{w.name} O layer {layer}",
                 rel_gate=1e-2 if bf16 else None)
    assert_close(lse_n.cpu().numpy(), lse_ref, w, f"{w.name} lse layer {layer}")


def test_noalloc_matches_allocating_entry_point_twice(gpu_lib):
    big, small = Case(BIG), Case(SMALL)
    assert big.req.query_attn_workspace_bytes() > small.req.query_attn_workspace_bytes() > 0
    _check(big, 1)
    _check(small, 1)          # the smaller problem after the larger one, same scratch
    _check(big, 0)            # and back


def test_noalloc_fp32_needs_no_scratch(gpu_lib):
    case = Case(FP32)
    assert case.req.query_attn_workspace_bytes() == 0
    _check(case, 1)
