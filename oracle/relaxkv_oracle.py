"""Float64 CPU oracle for the RelaxKV selective-repair hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers, tables or pre/post-processing) and
imports nothing from the product package.

Every function is a plain, slow restatement of the paper's definitions in
numpy float64 (arXiv 2609.33503, "RelaxKV: Recomputation Guided by the Query
with Sparse Context Attention for Efficient KV Cache Reuse"):

* ``score``        -- Sec. 3.2, layer-wise query-attention score a_{l,i}
                      (pooled attention, MinMax-normalised per layer);
                      first step of Algorithm 1.
* ``anchor_count`` -- App. A.1, first equation: k = max(1, round(r T_c)).
* ``select``       -- Sec. 3.2 / App. A.1 second equation: S_l = TopK_i(a_{l,i}, k),
                      ties to the lowest position.
* ``build_sets``   -- Sec. 3.2 / App. A.1 set equations: h_i, U, R_l; the compact
                      index of App. A.2 ("compact execution"); the edge count
                      E_unmasked and state cost of App. A.2.
* ``sparse_attn``  -- Sec. 3.3 (C_l(p) = U cap {j <= p}) and Sec. 3.4 / App. A.2
                      (mixed fresh/cached K~, V~ rule); the Full-Prefix Control
                      of App. A.3 (Table "Controlled configurations") with
                      ``mode="full"``.
* ``update_cache`` -- Sec. 3.4 cache-update semantics, Algorithm 1 update step:
                      fresh rows of R_l overwrite their cache positions.
* ``query_attn``   -- the query prefill after repair (App. C.4, cache-ready TTFT
                      protocol): query tokens attend to the cache and causally
                      to themselves; its row log-sum-exp is the normaliser of
                      the supplied-LSE scoring mode.
* ``build_sets_context`` -- the context-construction variants of Sec. 4.4
                      (Global Sparse, Layerwise Sparse): the same anchors and
                      targets with the context set U_l replaced.
* ``global_scores``, ``global_target_count``, ``select_global``,
  ``build_sets_global`` -- the matched-target variants: RelaxKV^G (Sec. 4.1
                      comparison setup; App. A.3 table "Controlled
                      configurations") keeps a global target set P for every
                      layer with the context C_l(p); the global repair target
                      sweep (App. B equation) ranks g_i = (1/L) sum_l a_{l,i}.

Readings where the paper is silent (each also listed in the design notes):

* softmax domain of the scoring attention: the T_c cached keys only, unless
  the caller supplies each query row's log-sum-exp (``row_lse``), in which case
  A = exp(s - lse) with that normaliser;
* softmax scale 1/sqrt(d) unless given;
* GQA map: query head h reads KV head floor(h / (H / H_kv));
* MinMax of a constant row is the all-zero row;
* round() is round-half-to-even in IEEE double (Python's ``round``), then k is
  clamped to [1, T_c];
* equal scores are ordered by ascending position; -0.0 equals +0.0; a NaN
  score is an error;
* layers are 0-based, positions are context positions 0..T_c-1 only;
* a global target p need not lie in U; its context U cap {j <= p} may then be
  empty, and attention over an empty context is the empty sum: O = 0 and
  log-sum-exp = -inf.

Pins: every function is checked in ``tests/test_oracle_pins.py`` against
something other than itself (closed forms, a hand-worked example, brute force
on tiny inputs, torch's scaled_dot_product_attention in float64, and set
invariants).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


# ----------------------------------------------------------------------------
# Scoring: Sec. 3.2 equation for a_{l,i}; Algorithm 1, scoring step.
# ----------------------------------------------------------------------------

def score(q, k_cache, softmax_scale=None, row_lse=None):
    """Layer-wise pooled query attention over the cached context.

    q        [L][Qn][H][d]     user-query rows per layer (already rotated).
    k_cache  [L][H_kv][T_c][d] naive cached keys (already rotated).
    row_lse  optional [L][Qn][H] natural-log normaliser of each query row.

    For each layer l, head h and query token t the attention row is
    A_l[h,t,:] = softmax_i(sigma <q_{l,t,h}, k_{l,g(h),i}>) over the T_c cached
    keys (or exp(s - row_lse) when a normaliser is supplied).  The pooled score
    is p_{l,i} = (1/(H Qn)) sum_h sum_t A_l[h,t,i] and a_{l,i} = MinMax_i(p_{l,i}).

    Returns (a [L][T_c], p [L][T_c], lse [L][Qn][H]) in float64, where lse is
    the log-sum-exp of each row's logits over the cached keys.
    """
    q = np.asarray(q, dtype=np.float64)
    k_cache = np.asarray(k_cache, dtype=np.float64)
    L, Qn, H, d = q.shape
    H_kv, T_c = k_cache.shape[1], k_cache.shape[2]
    if H % H_kv:
        raise ValueError("H must be a multiple of H_kv")
    G = H // H_kv
    sigma = 1.0 / np.sqrt(d) if softmax_scale is None else float(softmax_scale)

    p = np.zeros((L, T_c))
    lse = np.zeros((L, Qn, H))
    for l in range(L):
        for h in range(H):
            g = h // G
            s = sigma * (q[l, :, h, :] @ k_cache[l, g].T)          # [Qn][T_c]
            m = s.max(axis=1, keepdims=True)
            z = np.exp(s - m).sum(axis=1, keepdims=True)
            lse[l, :, h] = (m + np.log(z))[:, 0]
            if row_lse is None:
                A = np.exp(s - m) / z                               # softmax rows
            else:
                A = np.exp(s - np.asarray(row_lse, np.float64)[l, :, h][:, None])
            p[l] += A.sum(axis=0)
    p /= H * Qn

    a = np.zeros_like(p)
    for l in range(L):
        lo, hi = p[l].min(), p[l].max()
        if hi > lo:
            a[l] = (p[l] - lo) / (hi - lo)
        # else: constant row -> all zeros (MinMax of a constant)
    return a, p, lse


# ----------------------------------------------------------------------------
# Selection: App. A.1, k and TopK equations; Algorithm 1, selection steps.
# ----------------------------------------------------------------------------

def anchor_count(ratio, T_c):
    """k = max(1, round(r T_c)), clamped to T_c (Sec. 3.2, App. A.1)."""
    ratio = float(ratio)
    if not np.isfinite(ratio) or ratio < 0.0 or ratio > 1.0:
        raise ValueError("anchor ratio must be a finite number in [0, 1]")
    k = max(1, int(round(ratio * T_c)))
    return min(k, int(T_c))


def select(a, k):
    """S_l = TopK_i(a_{l,i}, k) for every layer, returned sorted ascending.

    Order is by descending score, then ascending position (lowest index wins
    a tie).  -0.0 and +0.0 compare equal.  NaN is rejected.
    """
    a = np.asarray(a, dtype=np.float64)
    if np.isnan(a).any():
        raise ValueError("NaN score")
    L, T_c = a.shape
    out = np.empty((L, k), dtype=np.int64)
    pos = np.arange(T_c)
    for l in range(L):
        # np.lexsort sorts by the last key first: primary -a (descending a),
        # secondary the position (ascending).
        order = np.lexsort((pos, -a[l]))
        out[l] = np.sort(order[:k])
    return out


# ----------------------------------------------------------------------------
# Sets: h_i, U, R_l (Sec. 3.2 / App. A.1), compact indices and accounting
# (App. A.2).
# ----------------------------------------------------------------------------

@dataclass
class Sets:
    T_c: int
    k: int
    anchors: np.ndarray                 # [L][k] sorted ascending
    h: np.ndarray                       # [T_c] highest selected layer, -1 if none
    U: np.ndarray                       # sorted union of anchors
    cidx: np.ndarray                    # [T_c] compact index in U, -1 if not in U
    R: list = field(default_factory=list)       # R[l]: sorted positions
    R_u: list = field(default_factory=list)     # R_u[l][t]: compact index of R[l][t]
    src: list = field(default_factory=list)     # src[l][c]: rank of context[l][c] in R[l] or -1
    edges: np.ndarray = None            # [L] sum_{p in R_l} |C_l(p)|
    edges_full: np.ndarray = None       # [L] sum_{p in R_l} (p + 1)
    ctx: list = None                    # ctx[l]: sorted context set U_l; None: U at every layer

    @property
    def L(self):
        return len(self.R)

    def context(self, layer):
        """The context set U_l of a layer (the union U unless a construction
        variant replaced it)."""
        return self.U if self.ctx is None else self.ctx[layer]


def build_sets(anchors, T_c):
    """Highest selected layer, union, active targets and compact maps.

    h_i = max{l : i in S_l}; U = union_l S_l; R_l = {i in U : h_i >= l}.
    U is kept sorted and each position gets its compact index (App. A.2);
    src[l][c] is the rank of U[c] within R_l (the row of the freshly
    recomputed K/V), or -1 when U[c] is not active at layer l.
    edges[l] = sum_{p in R_l} |C_l(p)| with C_l(p) = U cap {j <= p}
    (App. A.2 edge count); edges_full[l] is the same count for the full causal
    prefix, sum_{p in R_l} (p + 1).
    """
    anchors = np.asarray(anchors, dtype=np.int64)
    L, k = anchors.shape
    h = np.full(T_c, -1, dtype=np.int64)
    for l in range(L):
        h[anchors[l]] = np.maximum(h[anchors[l]], l)
    U = np.flatnonzero(h >= 0)
    cidx = np.full(T_c, -1, dtype=np.int64)
    cidx[U] = np.arange(len(U))

    R, R_u, src = [], [], []
    edges = np.zeros(L, dtype=np.int64)
    edges_full = np.zeros(L, dtype=np.int64)
    for l in range(L):
        R_l = U[h[U] >= l]
        u_l = cidx[R_l]
        s_l = np.full(len(U), -1, dtype=np.int64)
        s_l[u_l] = np.arange(len(R_l))
        R.append(R_l)
        R_u.append(u_l)
        src.append(s_l)
        # |C_l(p)| = number of union positions <= p = compact index of p + 1.
        edges[l] = int(np.sum(u_l + 1))
        edges_full[l] = int(np.sum(R_l + 1))
    return Sets(T_c=T_c, k=k, anchors=anchors, h=h, U=U, cidx=cidx,
                R=R, R_u=R_u, src=src, edges=edges, edges_full=edges_full)


# ----------------------------------------------------------------------------
# Matched-target variants: RelaxKV^G (App. A.3 table) and the global repair
# target sweep (App. B equation).
# ----------------------------------------------------------------------------

def global_scores(a):
    """g_i = (1/L) sum_l a_{l,i}: the layer mean of the normalised scores (App. B)."""
    a = np.asarray(a, dtype=np.float64)
    return a.sum(axis=0) / a.shape[0]


def global_scores_f32(a32):
    """g in float32, the precision in which the GPU takes the TopK decision over
    g: a float32 running sum over layers in layer order, then one float32
    division by L (each step an IEEE-754 single operation)."""
    a32 = np.asarray(a32, dtype=np.float32)
    g = np.zeros(a32.shape[1], dtype=np.float32)
    for l in range(a32.shape[0]):
        g = (g + a32[l]).astype(np.float32)
    return (g / np.float32(a32.shape[0])).astype(np.float32)


def global_target_count(ratio, T_c, n_union):
    """|P_{r_g}| = min(floor(r_g T_c), |U|) (App. B equation)."""
    ratio = float(ratio)
    if not np.isfinite(ratio) or ratio < 0.0 or ratio > 1.0:
        raise ValueError("target ratio must be a finite number in [0, 1]")
    return min(int(np.floor(ratio * T_c)), int(n_union))


def select_global(g, n_targets):
    """P = TopK_i(g_i, n_targets), lowest position first among equal g,
    returned ascending (App. B equation)."""
    g = np.asarray(g, dtype=np.float64)
    if n_targets == 0:
        return np.zeros(0, dtype=np.int64)
    return select(g[None, :], int(n_targets))[0]


def build_sets_global(anchors, T_c, P):
    """Sets of a matched-target variant: the context is still the union U of
    the layer-wise anchors, but every layer repairs the same global target
    list P (sorted, distinct positions).

    R_l = P for every l; the compact limit of a target p is
    |U cap {j <= p}| - 1, which is -1 (empty context) when p precedes every
    union position; src[l][c] is the rank of U[c] in P or -1; h_i = L - 1 for
    targets (active at every layer) and -1 otherwise.
    """
    anchors = np.asarray(anchors, dtype=np.int64)
    P = np.asarray(P, dtype=np.int64)
    if P.ndim != 1 or (len(P) > 0 and (P.min() < 0 or P.max() >= T_c)):
        raise ValueError("targets must be positions in [0, T_c)")
    if np.any(np.diff(P) <= 0):
        raise ValueError("targets must be strictly ascending")
    L = anchors.shape[0]
    in_union = np.zeros(T_c, dtype=bool)
    for l in range(L):
        in_union[anchors[l]] = True
    U = np.flatnonzero(in_union)
    cidx = np.full(T_c, -1, dtype=np.int64)
    cidx[U] = np.arange(len(U))
    h = np.full(T_c, -1, dtype=np.int64)
    h[P] = L - 1
    # |U cap {j <= p}| for every target, counted directly.
    n_le = np.array([int(np.count_nonzero(U <= p)) for p in P], dtype=np.int64)
    u = n_le - 1
    rank = np.full(T_c, -1, dtype=np.int64)
    rank[P] = np.arange(len(P))
    s_l = rank[U]
    R, R_u, src = [], [], []
    for _ in range(L):
        R.append(P.copy())
        R_u.append(u.copy())
        src.append(s_l.copy())
    edges = np.full(L, int(np.sum(n_le)), dtype=np.int64)
    edges_full = np.full(L, int(np.sum(P + 1)), dtype=np.int64)
    return Sets(T_c=T_c, k=anchors.shape[1], anchors=anchors, h=h, U=U, cidx=cidx,
                R=R, R_u=R_u, src=src, edges=edges, edges_full=edges_full)


# ----------------------------------------------------------------------------
# Context-construction variants: Sec. 4.4 (Global Sparse, Layerwise Sparse).
# ----------------------------------------------------------------------------

def build_sets_context(anchors, T_c, a, construction, g=None):
    """RelaxKV's anchors and targets R_l with the context set replaced by a
    construction variant of the same size |U| (Sec. 4.4):

    "union"      U_l = U, the union of the anchors (RelaxKV itself);
    "global"     U_l = TopK_i(g_i, |U|) for every layer, g the layer mean of a
                 (Global Sparse: one set shared across layers);
    "layerwise"  U_l = TopK_i(a_{l,i}, |U|) (Layerwise Sparse).

    g (optional) replaces the layer mean for "global", e.g. the float32 mean
    in which a GPU ranks.  Ties go to the lower position.
    C_l(p) = U_l cap {j <= p}: a target need not
    lie in U_l (it then does not see its own key, and its context may be
    empty).  R_u[l][t] = |U_l cap {j <= p}| - 1; src[l][c] = rank of U_l[c] in R_l
    or -1; edges count |C_l(p)| over R_l; U, cidx and h stay those of the
    anchor union.
    """
    base = build_sets(anchors, T_c)
    a = np.asarray(a, dtype=np.float64)
    L = len(base.R)
    n = len(base.U)
    if construction == "union":
        ctx = [base.U.copy() for _ in range(L)]
    elif construction == "global":
        shared = select_global(global_scores(a) if g is None else g, n)
        ctx = [shared.copy() for _ in range(L)]
    elif construction == "layerwise":
        ctx = [select(a[l:l + 1], n)[0] for l in range(L)]
    else:
        raise ValueError("construction must be 'union', 'global' or 'layerwise'")
    R_u, src = [], []
    edges = np.zeros(L, dtype=np.int64)
    for l in range(L):
        U_l = ctx[l]
        n_le = np.array([int(np.count_nonzero(U_l <= p)) for p in base.R[l]], dtype=np.int64)
        R_u.append(n_le - 1)
        rank = np.full(T_c, -1, dtype=np.int64)
        rank[base.R[l]] = np.arange(len(base.R[l]))
        src.append(rank[U_l])
        edges[l] = int(np.sum(n_le))
    return Sets(T_c=T_c, k=base.k, anchors=base.anchors, h=base.h, U=base.U, cidx=base.cidx,
                R=base.R, R_u=R_u, src=src, edges=edges, edges_full=base.edges_full, ctx=ctx)


# ----------------------------------------------------------------------------
# Sparse-context attention: Sec. 3.3, Sec. 3.4 equation, App. A.2.
# ----------------------------------------------------------------------------

def sparse_attn(layer, sets, q_new, k_new, v_new, k_cache_l, v_cache_l,
                softmax_scale=None, mode="union", targets=None):
    """Attention of the active targets of one layer over their context.

    q_new      [|R_l|][H][d]    fresh queries of the targets, rows in R_l order.
    k_new/v_new[|R_l|][H_kv][d] fresh keys/values of the targets.
    k_cache_l/v_cache_l [H_kv][T_c][d] naive cache of this layer.
    mode       "union": target p attends to C_l(p) = U cap {j <= p} (RelaxKV);
               "full":  target p attends to {j <= p} (Full-Prefix Control).
    targets    optional iterable of ranks t in R_l to evaluate (default: all).

    For every context position j the key/value is the fresh row when j is an
    active target of this layer (j in R_l) and the naive cached row otherwise
    (Sec. 3.4).  With O_{t,h} = sum_j softmax_j(sigma <q_{t,h}, K~_{j,g(h)}>) V~_{j,g(h)}.

    Returns (O [n][H][d], lse [n][H]) in float64 for the requested targets.
    """
    q_new = np.asarray(q_new, dtype=np.float64)
    k_new = np.asarray(k_new, dtype=np.float64)
    v_new = np.asarray(v_new, dtype=np.float64)
    k_cache_l = np.asarray(k_cache_l, dtype=np.float64)
    v_cache_l = np.asarray(v_cache_l, dtype=np.float64)
    R_l = sets.R[layer]
    n_R = len(R_l)
    if q_new.shape[0] != n_R or k_new.shape[0] != n_R or v_new.shape[0] != n_R:
        raise ValueError("fresh rows must number |R_l|")
    H, d = q_new.shape[1], q_new.shape[2]
    H_kv = k_cache_l.shape[0]
    G = H // H_kv
    sigma = 1.0 / np.sqrt(d) if softmax_scale is None else float(softmax_scale)

    # Rank of every position within R_l (-1 when not active at this layer).
    rank = np.full(sets.T_c, -1, dtype=np.int64)
    rank[R_l] = np.arange(n_R)

    if mode == "union":
        ctx_all = sets.context(layer)
    elif mode == "full":
        ctx_all = np.arange(sets.T_c)
    else:
        raise ValueError("mode must be 'union' or 'full'")

    # K~, V~ over the candidate context positions, [H_kv][n_ctx][d]: fresh
    # rows where the position is in R_l, naive cached rows elsewhere.
    fresh = rank[ctx_all] >= 0
    Kt = k_cache_l[:, ctx_all, :].copy()
    Vt = v_cache_l[:, ctx_all, :].copy()
    Kt[:, fresh, :] = np.transpose(k_new[rank[ctx_all[fresh]]], (1, 0, 2))
    Vt[:, fresh, :] = np.transpose(v_new[rank[ctx_all[fresh]]], (1, 0, 2))

    ts = range(n_R) if targets is None else list(targets)
    O = np.zeros((len(ts), H, d))
    lse = np.zeros((len(ts), H))
    for n, t in enumerate(ts):
        p = R_l[t]
        m = int(np.searchsorted(ctx_all, p, side="right"))   # |{j in ctx : j <= p}|
        if m == 0:                       # empty context: the empty sum
            lse[n, :] = -np.inf
            continue
        for h in range(H):
            g = h // G
            s = sigma * (Kt[g, :m, :] @ q_new[t, h])           # [m]
            mx = s.max()
            e = np.exp(s - mx)
            z = e.sum()
            O[n, h] = (e / z) @ Vt[g, :m, :]
            lse[n, h] = mx + np.log(z)
    return O, lse


def attention_flops(H, d, edges):
    """Algorithmic attention FLOPs for a number of unmasked causal edges:
    per edge and query head one d-long dot product (2d) and one d-long
    weighted sum (2d)."""
    return 4.0 * H * d * float(np.sum(edges))


# ----------------------------------------------------------------------------
# Query-side completion: the query prefill of the cache-ready TTFT protocol
# (App. C.4): the query tokens attend to the (repaired) cache and causally to
# themselves.
# ----------------------------------------------------------------------------

def query_attn(q_l, k_cache_l, v_cache_l, k_q, v_q, softmax_scale=None):
    """Attention of the n_query query tokens of one layer, placed after the T_c
    context positions: token t attends to every cache position 0..T_c-1 and to
    the query tokens 0..t.

    q_l [n_query][H][d]; k_cache_l / v_cache_l [H_kv][T_c][d] (the layer's cache,
    naive or repaired); k_q / v_q [n_query][H_kv][d] (the query tokens' own keys
    and values).  Returns (O [n_query][H][d], lse [n_query][H]) in float64; lse
    is the natural-log normaliser over all keys a row sees, the value the
    supplied-LSE scoring mode takes as q_lse.
    """
    q_l = np.asarray(q_l, dtype=np.float64)
    k_cache_l = np.asarray(k_cache_l, dtype=np.float64)
    v_cache_l = np.asarray(v_cache_l, dtype=np.float64)
    k_q = np.asarray(k_q, dtype=np.float64)
    v_q = np.asarray(v_q, dtype=np.float64)
    Qn, H, d = q_l.shape
    H_kv, T_c, _ = k_cache_l.shape
    G = H // H_kv
    sigma = 1.0 / np.sqrt(d) if softmax_scale is None else float(softmax_scale)
    O = np.zeros((Qn, H, d))
    lse = np.zeros((Qn, H))
    for h in range(H):
        g = h // G
        K = np.concatenate([k_cache_l[g], k_q[:, g, :]], axis=0)    # [T_c + Qn][d]
        V = np.concatenate([v_cache_l[g], v_q[:, g, :]], axis=0)
        for t in range(Qn):
            m = T_c + t + 1                                          # keys visible to token t
            s = sigma * (K[:m] @ q_l[t, h])
            mx = s.max()
            e = np.exp(s - mx)
            z = e.sum()
            O[t, h] = (e / z) @ V[:m]
            lse[t, h] = mx + np.log(z)
    return O, lse


# ----------------------------------------------------------------------------
# Cache update: Sec. 3.4 cache-update semantics; Algorithm 1, update step.
# ----------------------------------------------------------------------------

def update_cache(layer, sets, k_new, v_new, k_cache_l, v_cache_l):
    """The layer's cache after repair: the fresh rows of the active targets R_l
    overwrite their positions; every other entry keeps its value.

    k_new/v_new [|R_l|][H_kv][d] in R_l order; k_cache_l/v_cache_l [H_kv][T_c][d].
    Returns new (k, v) arrays; the inputs are not modified."""
    R_l = sets.R[layer]
    k = np.array(k_cache_l, copy=True)
    v = np.array(v_cache_l, copy=True)
    for t, p in enumerate(R_l):
        k[:, p, :] = k_new[t]
        v[:, p, :] = v_new[t]
    return k, v
