"""Properties of the seeded input generator that the workloads rely on (CPU).

The generator holds none of the method's arithmetic; these tests run the
float64 oracle on its outputs to check that each workload has the structure its
recipe promises.
"""

import numpy as np

import oracle
from paper_2609_33503_amd import synth

W = synth.WORKLOADS


def _sets(w):
    q, k, _ = synth.make_cache(w)
    a, _, _ = oracle.score(synth.to_f64(q), synth.to_f64(k))
    k_sel = max(1, int(round(w.ratio * w.T_c)))
    anchors = oracle.select(a, k_sel)
    return oracle.build_sets(anchors, w.T_c)


def test_latent_shrinks_the_union():
    # Same draws, one shared per-position latent: the layers' top-k sets overlap,
    # so the union and the active ratio fall well below those of iid layers.
    kw = dict(L=8, T_c=2048)                  # the 32K workloads' heads and query length
    # measured: union 0.69 (iid layers, ~1 - 0.85^8) against 0.42 with the latent
    s_iid = _sets(synth.shrink(W["qwen14b-32k-planted"], **kw))
    s_lat = _sets(synth.shrink(W["qwen14b-32k-latent"], **kw))
    u_iid, u_lat = len(s_iid.U) / 2048, len(s_lat.U) / 2048
    assert u_iid > 0.6
    assert u_lat < 0.7 * u_iid
    a_lat = sum(len(r) for r in s_lat.R) / (8 * 2048)
    a_iid = sum(len(r) for r in s_iid.R) / (8 * 2048)
    assert a_lat < a_iid


def test_latent_is_shared_across_layers():
    # The latent term is the same per-position scalar in every layer: the key
    # shift along each group's mean query direction correlates across layers.
    w = synth.shrink(W["qwen14b-32k-latent"], L=2, T_c=1024, H=8, H_kv=2, Qn=16)
    base = synth.shrink(W["qwen14b-32k-planted"], L=2, T_c=1024, H=8, H_kv=2, Qn=16)
    proj = []
    for l in range(2):
        q, k, _ = synth.make_cache_layer(w, l)
        _, k0, _ = synth.make_cache_layer(base, l)
        qg = q.float().reshape(w.Qn, w.H_kv, w.G, w.d).mean(dim=(0, 2))
        u = (qg / qg.norm(dim=1, keepdim=True)).numpy()
        dk = (k.float() - k0.float()).numpy()                 # [H_kv][T_c][d]
        proj.append(np.einsum("gtd,gd->gt", dk, u)[0])
    c = np.corrcoef(proj[0], proj[1])[0, 1]
    assert c > 0.95
