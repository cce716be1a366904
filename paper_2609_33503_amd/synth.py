"""Seeded synthetic workloads shaped like the paper's long-context RAG settings.

This module only draws and lays out inputs: it holds none of the method's
arithmetic (no scoring, selection, set construction or attention).  Both the
HIP path and the float64 oracle take their inputs from here.

Every tensor of every layer has its own stream: its 64-bit seed is derived
from numpy's SeedSequence(42, spawn_key=(workload id, layer, tensor id)), so a
single layer can be regenerated alone; the draws themselves come from a
``torch.Generator`` on the requested device (Philox on the GPU, Mersenne
Twister on the CPU), so values depend on the device the inputs are made on.

Shapes follow the paper's setting: contexts made of 512-token chunks encoded
at their global positions (Sec. 2.1, App. C.1), 8K to 32K contexts (Sec. 4,
App. C.2), grouped-query attention with the head layouts of Llama-3-8B and
Qwen3-14B, bfloat16 caches.  Chunking only affects how a real cache would be
built, so the generator is chunk-agnostic; ``chunk`` is carried as metadata.
The paper's datasets (RULER-MV, LongBench, LV-Eval) are not used; these seeded
Gaussian inputs stand in for them.

Layouts (row-major, last index contiguous):
  q         [Qn][H][d]        user-query rows of one layer (already rotated)
  k_cache   [H_kv][T_c][d]    naive cached keys of one layer (already rotated)
  v_cache   [H_kv][T_c][d]
  q_new     [T_c][H][d]       fresh queries for every context position
  k_new     [T_c][H_kv][d]    fresh keys   = cached + sigma_p * N(0, 1)
  v_new     [T_c][H_kv][d]    fresh values = cached + sigma_p * N(0, 1)
  k_q, v_q  [Qn][H_kv][d]     the query tokens' own keys and values (law of K, V)
The harness gathers the rows of the active targets out of the fresh tensors
(``gather_rows``); in a real model they would be the projections' outputs.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np
import torch

BASE_SEED = 42                 # the paper's random seed (App. C.1)
_GLOBAL = 65535                # spawn-key "layer" slot for per-workload streams
_T_Q, _T_K, _T_V, _T_QN, _T_KN, _T_VN, _T_PLANT, _T_QK, _T_QV, _T_LAT = range(10)


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int                   # stream id
    L: int
    T_c: int
    chunk: int
    Qn: int
    H: int
    H_kv: int
    d: int
    dtype: str                 # "f32" or "bf16"
    std: float                 # std of K, V, Q, Q_new draws
    sigma_p: float             # std of the fresh-K/V perturbation
    ratio: float               # anchor ratio r
    planted_frac: float = 0.0  # fraction of positions shifted toward the query
    beta: float = 1.0          # size of that shift
    latent_gamma: float = 0.0  # strength of a per-position latent shared by all layers

    @property
    def G(self):
        return self.H // self.H_kv

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


_S128 = 1.0 / math.sqrt(128.0)

WORKLOADS = {
    # 2 layers, 1K context in 4 chunks of 256, 16 query tokens, 4q/2kv heads, d 64, fp32.
    "tiny-2L-1k-fp32": Workload("tiny-2L-1k-fp32", 0, L=2, T_c=1024, chunk=256, Qn=16,
                                 H=4, H_kv=2, d=64, dtype="f32", std=1.0, sigma_p=0.1,
                                 ratio=0.15),
    # Llama-3-8B-shaped layer stack: 32 layers, 32q/8kv, d 128, 8K context in 16x512.
    "llama8b-8k": Workload("llama8b-8k", 1, L=32, T_c=8192, chunk=512, Qn=64, H=32,
                           H_kv=8, d=128, dtype="bf16", std=_S128, sigma_p=0.05,
                           ratio=0.15),
    # Qwen3-14B-shaped: 40 layers, 40q/8kv, d 128, 16K context in 32x512 (ratio sweep).
    "qwen14b-16k": Workload("qwen14b-16k", 2, L=40, T_c=16384, chunk=512, Qn=64, H=40,
                            H_kv=8, d=128, dtype="bf16", std=_S128, sigma_p=0.05,
                            ratio=0.15),
    # Qwen3-14B-shaped at 32K (64x512) with 2% planted relevant tokens.
    "qwen14b-32k-planted": Workload("qwen14b-32k-planted", 3, L=40, T_c=32768, chunk=512,
                                    Qn=64, H=40, H_kv=8, d=128, dtype="bf16", std=_S128,
                                    sigma_p=0.05, ratio=0.15, planted_frac=0.02,
                                    beta=1.0),
}
# The 32K planted inputs plus a per-position latent shared by all layers, of
# strength 0.038: calibrated so that the union is about 63% of the context, the
# realized union reported for Qwen3-14B at r = 0.15 (Sec. 4.5).  The draws are
# otherwise those of the planted workload.  Not one of the benchmark's named
# configurations: it shows the attention when the union, and with it every
# context, is well below T_c.
WORKLOADS["qwen14b-32k-latent"] = replace(WORKLOADS["qwen14b-32k-planted"],
                                          name="qwen14b-32k-latent", latent_gamma=0.038)
# The matched-target control runs on the 32K planted inputs; the 2048-token
# chunking has identical inputs because the generator is chunk-agnostic.
WORKLOADS["qwen14b-32k-control"] = replace(WORKLOADS["qwen14b-32k-planted"],
                                           name="qwen14b-32k-control")
WORKLOADS["qwen14b-32k-control-c2048"] = replace(WORKLOADS["qwen14b-32k-planted"],
                                                 name="qwen14b-32k-control-c2048",
                                                 chunk=2048)
SWEEP_RATIOS_16K = (0.05, 0.15, 0.30)


def shrink(w: Workload, **kw) -> Workload:
    """A smaller workload with the same laws (for parity runs that the oracle
    finishes in seconds)."""
    return replace(w, name=w.name + "-" + "-".join(f"{k}{v}" for k, v in sorted(kw.items())),
                   **kw)


def _seed(wid, layer, tid):
    ss = np.random.SeedSequence(BASE_SEED, spawn_key=(wid, layer, tid))
    return int(ss.generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def _normal(shape, wid, layer, tid, device):
    g = torch.Generator(device=device)
    g.manual_seed(_seed(wid, layer, tid))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def planted_positions(w: Workload, device="cpu"):
    """The first round(planted_frac * T_c) entries of a seeded permutation of the
    context positions (the same in every layer), sorted."""
    n = int(round(w.planted_frac * w.T_c))
    if n == 0:
        return torch.empty(0, dtype=torch.long, device=device)
    g = torch.Generator(device="cpu")
    g.manual_seed(_seed(w.wid, _GLOBAL, _T_PLANT))
    perm = torch.randperm(w.T_c, generator=g)
    return torch.sort(perm[:n]).values.to(device)


def make_cache_layer(w: Workload, layer: int, device="cpu"):
    """(q [Qn][H][d], k_cache [H_kv][T_c][d], v_cache [H_kv][T_c][d]) of one layer,
    in the workload's dtype."""
    dt = w.torch_dtype
    q = (_normal((w.Qn, w.H, w.d), w.wid, layer, _T_Q, device) * w.std).to(dt)
    k = _normal((w.H_kv, w.T_c, w.d), w.wid, layer, _T_K, device) * w.std
    v = _normal((w.H_kv, w.T_c, w.d), w.wid, layer, _T_V, device) * w.std
    if w.planted_frac > 0.0 or w.latent_gamma > 0.0:
        # Unit mean direction of the group's Qn x G query vectors (after rounding).
        qg = q.float().reshape(w.Qn, w.H_kv, w.G, w.d).mean(dim=(0, 2))      # [H_kv][d]
        u = qg / qg.norm(dim=1, keepdim=True)
        if w.planted_frac > 0.0:
            pos = planted_positions(w, device)
            k[:, pos, :] += w.beta * u[:, None, :]
        if w.latent_gamma > 0.0:
            # z_i ~ N(0, 1), one value per position shared by every layer, so the
            # layers' scores are correlated and their top-k sets overlap.
            z = _normal((w.T_c,), w.wid, _GLOBAL, _T_LAT, device)
            k += w.latent_gamma * z[None, :, None] * u[:, None, :]
    return q, k.to(dt), v.to(dt)


def make_fresh_layer(w: Workload, layer: int, k_cache, v_cache, device="cpu"):
    """(q_new [T_c][H][d], k_new [T_c][H_kv][d], v_new [T_c][H_kv][d]) of one layer:
    fresh queries with the law of Q and fresh K/V = cached + sigma_p * N(0, 1),
    for every context position (the harness gathers the targets' rows)."""
    dt = w.torch_dtype
    qn = (_normal((w.T_c, w.H, w.d), w.wid, layer, _T_QN, device) * w.std).to(dt)
    kc = k_cache.float().transpose(0, 1)                                      # [T_c][H_kv][d]
    vc = v_cache.float().transpose(0, 1)
    kn = (kc + w.sigma_p * _normal((w.T_c, w.H_kv, w.d), w.wid, layer, _T_KN, device)).to(dt)
    vn = (vc + w.sigma_p * _normal((w.T_c, w.H_kv, w.d), w.wid, layer, _T_VN, device)).to(dt)
    return qn, kn.contiguous(), vn.contiguous()


def make_query_kv(w: Workload, layer: int, device="cpu"):
    """(k_q, v_q) [Qn][H_kv][d] of one layer: the user-query tokens' own keys and
    values, drawn with the law of the cached K and V."""
    dt = w.torch_dtype
    kq = (_normal((w.Qn, w.H_kv, w.d), w.wid, layer, _T_QK, device) * w.std).to(dt)
    vq = (_normal((w.Qn, w.H_kv, w.d), w.wid, layer, _T_QV, device) * w.std).to(dt)
    return kq.contiguous(), vq.contiguous()


def gather_rows(t, rows):
    """Rows of a position-major tensor, in the given (ascending) order."""
    idx = torch.as_tensor(np.asarray(rows, dtype=np.int64), device=t.device)
    return t.index_select(0, idx).contiguous()


def make_cache(w: Workload, device="cpu", layers=None):
    """Stacked (q [L][Qn][H][d], k_cache [L][H_kv][T_c][d], v_cache [L][H_kv][T_c][d])."""
    layers = range(w.L) if layers is None else layers
    qs, ks, vs = zip(*(make_cache_layer(w, l, device) for l in layers))
    return torch.stack(qs), torch.stack(ks), torch.stack(vs)


def to_f64(t):
    """Exact float64 numpy copy of a float32 / bfloat16 tensor (on the host)."""
    return t.detach().to("cpu").to(torch.float64).numpy()
