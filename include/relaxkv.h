/*
 * relaxkv.h -- C ABI of the RelaxKV selective-repair hot path on MI355X (gfx950).
 *
 * RelaxKV (arXiv 2609.33503) repairs a position-independent chunk KV cache for
 * one user query.  Its problem statement (Sec. 3.1): given the naive cache
 * K^naive, a query q and an anchor ratio r, choose per-layer repair targets and
 * a shared recomputation context, and recompute the targets' attention over
 * that context.  This library implements the per-layer hot path of that
 * repair as four calls, in order:
 *
 *   relaxkv_score       pooled, MinMax-normalised query attention a_{l,i}  (Sec. 3.2)
 *   relaxkv_select      S_l = TopK_i(a_{l,i}, k), k = max(1, round(r T_c)) (Sec. 3.2, App. A.1)
 *   relaxkv_build_sets  h_i, U, R_l, compact maps, edge counts          (Sec. 3.2, App. A.1-A.2)
 *   relaxkv_sparse_attn attention of R_l over C_l(p) = U cap {j <= p}
 *                       with the mixed fresh/cached K~, V~ rule          (Sec. 3.3, 3.4, App. A.2)
 *
 * plus the cache update of the repaired rows (relaxkv_update_cache, Sec. 3.4)
 * the matched-target variants, where one global target list replaces R_l
 * (relaxkv_select_global, relaxkv_build_sets_global; Sec. 4.1, App. A.3, App. B),
 * the context-construction variants, where another context set of the same
 * size replaces U (relaxkv_build_sets_context; Sec. 4.4), and the query-side
 * completion: the query tokens' attention over the repaired cache, whose row
 * log-sum-exp feeds the one-pass scoring mode (relaxkv_query_attn; App. C.4).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Device pointers are HIP device memory of the current device; host
 *   pointers are marked "host".  The caller owns every buffer: the library
 *   never allocates, frees or retains a pointer past the call.
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *   stream) unless it says it synchronises.  Inputs must stay valid and
 *   unmodified until the stream reaches the call.
 * - Arguments are validated on the host before anything is enqueued.  On any
 *   error code nothing is enqueued and no output is touched.
 * - Arrays are row-major with the last index contiguous and no padding.
 *   Element types: int32 for indices and counts, int64 for edge counts,
 *   float32 for scores and log-sum-exp values, and `dtype` (bfloat16 or
 *   float32) for Q/K/V and attention outputs.
 * - Layers are 0-based; positions are context positions 0 .. T_c-1 (the
 *   query tokens are never targets or context).
 * - The library keeps no host state between calls (besides the per-device
 *   address of relaxkv_query_attn_noalloc's scratch array, looked up once per
 *   device) and calls are reentrant; two calls that write the same buffers must
 *   be ordered by the caller.
 *   Device state lives in caller-owned buffers: the sets buffer holds the bf16
 *   attention's work counters (each launch returns its slot to zero), so two
 *   relaxkv_sparse_attn launches with the same sets, layer and context mode
 *   must not overlap in time; relaxkv_query_attn_noalloc uses a device array
 *   of the library instead (see there).
 * - Compute calls enqueue kernels only (no allocation, memset or host
 *   synchronisation; relaxkv_counts_to_host is the one synchronising call),
 *   so a sequence of them can be captured into a HIP graph and replayed.
 * - The one piece of request state on the host is in relaxkv_sets: the set-building
 *   calls record in it which kind of target and context lists they built
 *   (global_targets, context_sets), so pass the struct the last of them
 *   filled, not an older copy.  A stale copy cannot make a kernel overrun:
 *   the attention and cache-update kernels clamp the device row count to the
 *   row capacity they were given and to the bound the host sized their grid
 *   from, and set RELAXKV_ERR_ROWS when they had to clamp.
 * - Device error word (counts[L+1] of relaxkv_sets, cleared by relaxkv_select):
 *   bits RELAXKV_ERR_*; relaxkv_counts_to_host returns RELAXKV_EINVAL while it
 *   is nonzero.
 */
#ifndef RELAXKV_H
#define RELAXKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t relaxkv_status;
#define RELAXKV_OK            0
#define RELAXKV_EINVAL       -1  /* null pointer, bad dimension, ratio not in [0,1], layer out of range, NaN score */
#define RELAXKV_ENOSPACE     -2  /* caller buffer smaller than the size query reports */
#define RELAXKV_EUNSUPPORTED -3  /* head_dim, dtype or head layout this build has no kernel for */
#define RELAXKV_EDEVICE      -4  /* a HIP runtime call or kernel launch failed */

/* Bits of the device error word counts[L+1]. */
#define RELAXKV_ERR_NAN_SCORE   1  /* a NaN score reached a selection */
#define RELAXKV_ERR_BAD_TARGETS 2  /* relaxkv_build_sets_global got an invalid target list */
#define RELAXKV_ERR_ROWS        4  /* |R_l| on the device exceeded the rows an attention or
                                      cache-update call could process (its n_rows, or the
                                      bound of the target lists the host was told about) */

#define RELAXKV_DTYPE_F32  0
#define RELAXKV_DTYPE_BF16 1

#define RELAXKV_CONTEXT_UNION 0  /* C_l(p) = U_l cap {j <= p} (RelaxKV, Sec. 3.3) */
#define RELAXKV_CONTEXT_FULL  1  /* {j <= p}: Full-Prefix Control (App. A.3) */

/* Context set U_l of relaxkv_build_sets_context (Sec. 4.4). */
#define RELAXKV_CONTEXT_SETS_UNION     0  /* U_l = U, the anchor union (RelaxKV) */
#define RELAXKV_CONTEXT_SETS_GLOBAL    1  /* U_l = TopK(g, |U|) for every layer (Global Sparse) */
#define RELAXKV_CONTEXT_SETS_LAYERWISE 2  /* U_l = TopK(a_l, |U|) per layer (Layerwise Sparse) */

/* Limits of this build (checked by relaxkv_validate).  The bf16 path also
 * needs one layer's cache slab, T_c * H_kv * d elements, below
 * RELAXKV_MAX_BF16_LAYER_ELEMS (its attention addresses rows with 32-bit
 * element offsets); larger bf16 problems get RELAXKV_EUNSUPPORTED. */
#define RELAXKV_MAX_LAYERS 1024
#define RELAXKV_MAX_TC     (1 << 22)
#define RELAXKV_MAX_BF16_LAYER_ELEMS ((int64_t)1 << 31)

/*
 * The problem every call describes.
 *   L, T_c     layers and context tokens; n_query query tokens; H query heads,
 *              H_kv key/value heads (H % H_kv == 0; query head h reads KV head
 *              h / (H / H_kv)); d head dimension (64 or 128).
 *   softmax_scale  sigma in softmax(sigma q.k); <= 0 selects 1/sqrt(d).
 *   anchor_ratio   r in [0, 1].
 *   q          device [L][n_query][H][d]  the user query's rows (already rotated
 *              at their global positions).
 *   k_cache    device [L][H_kv][T_c][d]   naive cached keys (already rotated).
 *   v_cache    device [L][H_kv][T_c][d]   naive cached values.
 *   q_lse      optional device [L][n_query][H] float32: natural-log normaliser of
 *              each query row from the caller's own query forward.  When NULL
 *              the scoring softmax runs over the T_c cached keys only and
 *              relaxkv_score computes the normaliser itself (two passes over K);
 *              when given, relaxkv_score reads K once.
 *   kv_stride_layer, kv_stride_head, kv_stride_token
 *              element strides of k_cache and v_cache (both laid out alike, and
 *              so are the cache arguments of relaxkv_update_cache and
 *              relaxkv_query_attn): the d contiguous elements of token i of KV
 *              head g of layer l start at element l * kv_stride_layer +
 *              g * kv_stride_head + i * kv_stride_token.  0 selects the dense
 *              value (d, T_c * token stride, H_kv * head stride), so a zeroed
 *              descriptor describes [L][H_kv][T_c][d]; a cache allocated for
 *              more tokens than T_c, or laid out [L][T_c][H_kv][d], is passed
 *              with its own strides.  Every other array (q, q_lse, the fresh
 *              rows, the outputs) is dense row-major.
 * Pointers: q, k_cache and v_cache 16-byte aligned, and every cache row too
 * (strides times the element size a multiple of 16 bytes).
 */
typedef struct relaxkv_problem {
    int32_t L, T_c, n_query, H, H_kv, d;
    int32_t dtype;
    float softmax_scale;
    double anchor_ratio;
    const void* q;
    const void* k_cache;
    const void* v_cache;
    const float* q_lse;
    int64_t kv_stride_layer, kv_stride_head, kv_stride_token;
} relaxkv_problem;

/*
 * The index sets of one request, carved by relaxkv_sets_bind out of one
 * caller-owned device buffer.  All pointers are device pointers.
 *   anchors  [L][k]        S_l, ascending positions.
 *   h        [T_c]         highest selected layer h_i, -1 when i is in no S_l.
 *   U        [T_c]         U sorted ascending in the first |U| entries.
 *   cidx     [T_c]         compact index of position i in U, -1 if i not in U.
 *   R_off    [L+1]         R_l occupies entries R_off[l] .. R_off[l+1]-1 of R_idx/R_u.
 *   R_idx    [L*T_c]       positions of R_l, ascending (CSR over layers).
 *   R_u      [L*T_c]       compact limit of each R_idx entry: |U_l cap {j <= p}| - 1
 *                          (its compact index when p is in U_l; -1 for an empty context).
 *   src      [L][T_c]      src[l*T_c + c] = rank of U_l[c] within R_l (its row in the
 *                          fresh K/V of layer l), or -1 (cached row), c < |U|; U_l is
 *                          the layer's context list (U unless a construction variant
 *                          replaced it, see ctx).
 *   rank     [L][T_c]      rank[l*T_c + j] = rank of position j within R_l, or -1 when j is
 *                          not an active target of layer l (position-indexed view of src).
 *   counts   [L+2]         counts[0] = |U|; counts[1+l] = |R_l|; counts[L+1] = error
 *                          word (RELAXKV_ERR_* bits; cleared by relaxkv_select).
 *   edges    [2L]          edges[l] = sum_{p in R_l} |C_l(p)| (App. A.2 edge count);
 *                          edges[L+l] = sum_{p in R_l} (p+1), the full-prefix count.
 *   ctx      [L][T_c]      context lists of the construction variants (first |U| entries
 *                          of a row, ascending): row 0 for every layer (Global Sparse) or
 *                          row l for layer l (Layerwise Sparse); unused for the union.
 *   g        [T_c]         float32 layer-mean scores of the last Global Sparse build.
 *   tiles    [2][L][H_kv+1] uint32 work counters of the bf16 attention, one slot per
 *                          context mode (0: the layer's context list, 1: Full-Prefix
 *                          Control) and layer: a next-tile counter per KV head and a
 *                          count of the launch's workgroups.  Zeroed by every set build;
 *                          each relaxkv_sparse_attn launch returns its slot to zero.
 *   k        the anchor budget k = max(1, round(r T_c)), computed on the host.
 *   global_targets  host flag: 0 after relaxkv_sets_bind and relaxkv_build_sets
 *                   (targets R_l of RelaxKV, |R_l| <= min(T_c, (L-l) k)), 1 after
 *                   relaxkv_build_sets_global (one target list for every layer,
 *                   |R_l| <= T_c); the attention and cache-update calls size their
 *                   grids from it.
 *   context_sets    host flag: the RELAXKV_CONTEXT_SETS_* construction of U_l of the
 *                   last set build (0 after relaxkv_sets_bind, relaxkv_build_sets and
 *                   relaxkv_build_sets_global); relaxkv_sparse_attn reads U_l from
 *                   U or ctx accordingly.
 */
typedef struct relaxkv_sets {
    int32_t L, T_c, k;
    int32_t* anchors;
    int32_t* h;
    int32_t* U;
    int32_t* cidx;
    int32_t* R_off;
    int32_t* R_idx;
    int32_t* R_u;
    int32_t* src;
    int32_t* rank;
    int32_t* counts;
    int64_t* edges;
    int32_t* ctx;
    float* g;
    uint32_t* tiles;
    int32_t global_targets;
    int32_t context_sets;
} relaxkv_sets;

/* Text of a status code (static storage). */
const char* relaxkv_status_string(relaxkv_status s);

/* Host only.  k = max(1, round(r T_c)) with round-half-to-even in double,
 * clamped to T_c (Sec. 3.2, App. A.1).  Returns k >= 1, or RELAXKV_EINVAL when
 * r is not a finite number in [0, 1] or T_c < 1. */
int32_t relaxkv_anchor_count(double anchor_ratio, int32_t T_c);

/* Host only.  Checks dimensions, pointers, dtype, strides and the ratio of `p`:
 * RELAXKV_EINVAL for a bad dimension, pointer, scale or ratio, a negative
 * stride, or cache strides that do not nest: taken from the smallest, the
 * stride of each dimension with more than one entry must step past the whole
 * extent of the dimensions inside it, so that no two rows overlap (dimensions
 * of size 1 are ignored),
 * RELAXKV_EUNSUPPORTED for a head_dim, dtype, GQA group or bf16 layer size
 * (see the limits above) this build has no kernel for, a pointer or cache row
 * that is not 16-byte aligned, cache strides spanning 2^48 elements or more,
 * or (bf16, T_c > 1) a token stride of 2^24 elements or more or with
 * (T_c - 1) * stride + d >= RELAXKV_MAX_BF16_LAYER_ELEMS.  The stride of a
 * cache dimension of size 1 is never used and not checked. */
relaxkv_status relaxkv_validate(const relaxkv_problem* p);

/* Host only.  Device scratch bytes relaxkv_score needs (0 when p is invalid). */
size_t relaxkv_score_workspace_bytes(const relaxkv_problem* p);

/* Host only.  Device bytes of the set arrays of relaxkv_sets (0 when p is invalid). */
size_t relaxkv_sets_bytes(const relaxkv_problem* p);

/* Host only.  Fills *out with L, T_c, k and pointers carved out of the device
 * buffer `dev_buf` of `bytes` bytes (256-byte aligned sub-arrays).
 * RELAXKV_ENOSPACE when bytes < relaxkv_sets_bytes(p). */
relaxkv_status relaxkv_sets_bind(const relaxkv_problem* p, void* dev_buf, size_t bytes,
                                 relaxkv_sets* out);

/*
 * Layer-wise query-attention score (Sec. 3.2 equation; first step of
 * Algorithm 1).  For every layer l, query head h and query token t the row
 * A_l[h,t,:] = softmax_i(sigma <q_{l,t,h}, k_{l,h/G,i}>) over the T_c cached keys
 * (or exp(s - q_lse) with a supplied normaliser); then
 *   p_{l,i} = (1/(H n_query)) sum_{h,t} A_l[h,t,i],  a_{l,i} = MinMax_i(p_{l,i}),
 * and a constant row maps to all zeros.
 *   ws       device scratch of ws_bytes >= relaxkv_score_workspace_bytes(p).
 *   scores   device out [L][T_c] float32, a_{l,i} in [0, 1].
 * Reads q, k_cache and (optionally) q_lse of `p`; never reads v_cache.
 */
relaxkv_status relaxkv_score(const relaxkv_problem* p, void* ws, size_t ws_bytes,
                             float* scores, void* stream);

/*
 * Per-layer top-k anchor selection (Sec. 3.2, App. A.1 TopK equation).
 * S_l holds the k positions with the largest scores[l][i]; equal scores go to
 * the lower position; -0.0 equals +0.0.  Writes s->anchors[l][0..k-1]
 * ascending and clears s->counts[L+1]; a NaN score sets that error word
 * (read it with relaxkv_counts_to_host) and leaves that layer's anchors
 * unspecified.
 *   scores   device [L][T_c] float32 (any finite values).
 *   s        sets bound for the same problem (s->k from relaxkv_sets_bind).
 */
relaxkv_status relaxkv_select(const relaxkv_problem* p, const float* scores,
                              const relaxkv_sets* s, void* stream);

/*
 * Repair schedule and compact context (Sec. 3.2 set equations, App. A.1-A.2):
 *   h_i = max{l : i in S_l},  U = union_l S_l,  R_l = {i in U : h_i >= l},
 * the compact index of every position in U, the per-layer source map src, the
 * CSR lists R_idx/R_u, counts and edge counts.  Reads s->anchors (ascending
 * rows, entries in [0, T_c)); writes every other array of `s` and sets
 * s->global_targets = 0.
 */
relaxkv_status relaxkv_build_sets(const relaxkv_problem* p, relaxkv_sets* s, void* stream);

/*
 * Context-construction variants (Sec. 4.4): RelaxKV's anchors S_l (s->anchors)
 * and active targets R_l, with the context set U_l replaced by one of the same
 * size |U| (the anchor union's size):
 *   RELAXKV_CONTEXT_SETS_UNION      U_l = U (the same sets as relaxkv_build_sets);
 *   RELAXKV_CONTEXT_SETS_GLOBAL     U_l = TopK_i(g_i, |U|) for every layer, with
 *                                   g_i = (1/L) sum_l a_{l,i} (Global Sparse);
 *   RELAXKV_CONTEXT_SETS_LAYERWISE  U_l = TopK_i(a_{l,i}, |U|) (Layerwise Sparse);
 * larger scores first, equal scores to the lower position.  C_l(p) = U_l cap
 * {j <= p}; K~/V~ are fresh for j in R_l.  A target need not lie in U_l (it then
 * does not see its own key; an empty context gives O = 0, lse = -inf).  h, U,
 * cidx, R_idx and the full-prefix edge counts are those of relaxkv_build_sets;
 * R_u, src and edges[0..L-1] refer to U_l; the lists go to s->ctx and g to s->g.
 *   scores        device [L][T_c] float32 (a_{l,i}); a NaN sets bit 0 of the error word.
 *   construction  one of RELAXKV_CONTEXT_SETS_*.
 * Sets s->context_sets = construction and s->global_targets = 0.
 */
relaxkv_status relaxkv_build_sets_context(const relaxkv_problem* p, const float* scores,
                                          int32_t construction, relaxkv_sets* s,
                                          void* stream);

/*
 * Global repair targets of the target-capacity sweep (App. B equation):
 *   g_i = (1/L) sum_l a_{l,i},   P = TopK_i(g_i, min(floor(r_g T_c), |U|)),
 * larger g first, equal g to the lower position, P written ascending.
 *   scores        device [L][T_c] float32: a_{l,i} from relaxkv_score.
 *   target_ratio  r_g, a finite number in [0, 1] (floor(r_g T_c) in double).
 *   s             sets after relaxkv_build_sets: |U| is read from s->counts[0]
 *                 on the device.
 *   g             device out [T_c] float32: g_i (float32 sum over layers in layer
 *                 order, then divided by L).
 *   targets       device out [T_c] int32: P in entries 0 .. |P|-1.
 *   n_targets     device out [1] int32: |P| (0 when floor(r_g T_c) = 0).
 * A NaN in g sets bit 0 of the error word of s.
 */
relaxkv_status relaxkv_select_global(const relaxkv_problem* p, const float* scores,
                                     double target_ratio, const relaxkv_sets* s, float* g,
                                     int32_t* targets, int32_t* n_targets, void* stream);

/*
 * Sets of the matched-target variants: RelaxKV^G (Sec. 4.1; App. A.3 table
 * "Controlled configurations") and the global repair target sweep (App. B).
 * The context is still the union U of the layer-wise anchors in s->anchors,
 * but every layer repairs the same global target list P:
 *   R_l = P for every l,  C_l(p) = U cap {j <= p},  K~/V~ fresh exactly for j in P.
 * A target need not lie in U: its compact limit R_u = |U cap {j <= p}| - 1 is
 * -1 when no union position precedes it, and relaxkv_sparse_attn returns the
 * empty sum (O = 0, lse = -inf) for it in the union context.  h_i = L-1 for
 * targets (active at every layer), -1 otherwise; U, cidx as in
 * relaxkv_build_sets.
 *   targets    device [T_c] int32: P, strictly ascending positions in [0, T_c).
 *   n_targets  device [1] int32: |P| in [0, T_c].
 * A list that is not strictly ascending within [0, T_c), or a count outside
 * [0, T_c], sets bit 1 of the error word (relaxkv_counts_to_host then returns
 * RELAXKV_EINVAL); the arrays are then unspecified but every index in them is
 * in range.  Sets s->global_targets = 1.
 */
relaxkv_status relaxkv_build_sets_global(const relaxkv_problem* p, relaxkv_sets* s,
                                         const int32_t* targets, const int32_t* n_targets,
                                         void* stream);

/*
 * Sparse-context causal attention of layer `layer` (Sec. 3.3-3.4, App. A.2;
 * Algorithm 1, attention step).  For every active target t (position
 * p = R_idx[R_off[l] + t]) and query head h:
 *   O_{t,h} = sum_{j in C} softmax_j(sigma <q_new_{t,h}, K~_j>) V~_j
 * over C = C_l(p) = U cap {j <= p} (context_mode RELAXKV_CONTEXT_UNION) or
 * {j <= p} (RELAXKV_CONTEXT_FULL), where K~_j, V~_j are the fresh row of j when
 * j is in R_l and the naive cached row of j otherwise, read from KV head
 * h / (H / H_kv).
 *   q_new    device [n_rows][H][d]     fresh queries, rows in R_l order.
 *   k_new    device [n_rows][H_kv][d]  fresh keys, rows in R_l order.
 *   v_new    device [n_rows][H_kv][d]  fresh values, rows in R_l order.
 *   n_rows   rows the caller allocated in each of q_new, k_new, v_new, out and
 *            lse_out (>= 0; normally |R_l|, which the caller learns from
 *            relaxkv_counts_to_host or bounds by min(T_c, (L - layer) k)); the
 *            row pointers may be NULL when n_rows is 0.
 *   out      device out [n_rows][H][d] dtype: attention output before o_proj.
 *   lse_out  optional device out [n_rows][H] float32: natural-log normaliser.
 * |R_l| is read on the device from s->counts.  Targets t < min(|R_l|, n_rows)
 * are computed; when |R_l| exceeds n_rows (or the bound of the lists s says it
 * holds) the surplus targets are not computed and RELAXKV_ERR_ROWS is set in
 * the error word, so no row past the caller's buffers is read or written.  The
 * naive cache of the layer is read from p->k_cache / p->v_cache.  A target
 * whose context is empty (only with the lists of relaxkv_build_sets_global or
 * relaxkv_build_sets_context, union context) gets O = 0 and lse = -inf.
 * The bf16 kernel's workgroups take their tiles from the s->tiles slot of this
 * layer and context mode (dynamic balancing across XCDs whose clocks differ):
 * two launches with the same sets, layer and context mode must not overlap in
 * time (stream-ordered calls are fine); launches for other layers or modes may.
 */
relaxkv_status relaxkv_sparse_attn(const relaxkv_problem* p, const relaxkv_sets* s,
                                   int32_t layer, const void* q_new, const void* k_new,
                                   const void* v_new, int32_t n_rows, void* out,
                                   float* lse_out, int32_t context_mode, void* stream);

/*
 * Cache update of layer `layer` (Sec. 3.4 cache-update semantics; Algorithm 1,
 * cache-update step; App. A.2): the fresh K/V rows of the active targets R_l
 * overwrite the layer's cache entries at their positions; every other entry
 * keeps its value.
 *   k_new, v_new      device [n_rows][H_kv][d] in dtype, R_l order (the rows given
 *                     to relaxkv_sparse_attn).
 *   n_rows            rows allocated in k_new and v_new (>= 0); as in
 *                     relaxkv_sparse_attn, only targets t < min(|R_l|, n_rows) are
 *                     written and RELAXKV_ERR_ROWS is set when |R_l| is larger.
 *   k_cache, v_cache  device [L][H_kv][T_c][d] in dtype: the cache to update in
 *                     place.  It may be p->k_cache / p->v_cache themselves, or an
 *                     output cache the caller initialised from them.
 * Reads s->R_off, s->R_idx and s->counts on the device.  Rows written (positions
 * in R_l) are never read by relaxkv_sparse_attn of the same layer, which reads
 * cached rows only outside R_l, so the two calls need no mutual ordering.
 */
relaxkv_status relaxkv_update_cache(const relaxkv_problem* p, const relaxkv_sets* s,
                                    int32_t layer, const void* k_new, const void* v_new,
                                    int32_t n_rows, void* k_cache, void* v_cache,
                                    void* stream);

/* Host only.  Device scratch bytes relaxkv_query_attn needs (0 for float32
 * problems, which need none; 0 when p is invalid). */
size_t relaxkv_query_attn_workspace_bytes(const relaxkv_problem* p);

/*
 * Query-side completion of layer `layer` (the query prefill of App. C.4's
 * cache-ready TTFT protocol, after repair): the n_query query tokens, placed
 * after the T_c context positions, attend to every cache position and causally
 * to themselves:
 *   O_{t,h} = sum_j softmax_j(sigma <q_{l,t,h}, K_j>) V_j,  j over the cache
 *   positions 0..T_c-1 and then the query tokens 0..t, KV head h / (H / H_kv).
 * The queries are the layer's rows of p->q.
 *   k_cache, v_cache  device [L][H_kv][T_c][d] in dtype: the cache to attend to (the
 *                     naive cache, or one repaired by relaxkv_update_cache); layer
 *                     `layer` is read.
 *   k_q, v_q          device [n_query][H_kv][d] in dtype: the query tokens' own keys
 *                     and values at this layer.
 *   out               device out [n_query][H][d] in dtype.
 *   lse_out           optional device out [n_query][H] float32: the natural-log
 *                     normaliser of each row over all keys it sees, the value
 *                     relaxkv_score takes as q_lse (layer row l).
 *   ws                device scratch of ws_bytes >= relaxkv_query_attn_workspace_bytes(p)
 *                     (may be NULL when that is 0).
 */
relaxkv_status relaxkv_query_attn(const relaxkv_problem* p, int32_t layer, const void* k_cache,
                                  const void* v_cache, const void* k_q, const void* v_q,
                                  void* out, float* lse_out, void* ws, size_t ws_bytes,
                                  void* stream);

/* Scratch that relaxkv_query_attn_noalloc holds on each GPU (a problem whose
 * relaxkv_query_attn_workspace_bytes exceeds it is refused). */
#define RELAXKV_QUERY_ATTN_NOALLOC_MAX_BYTES ((size_t)32 << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph or
 * stream capture, serving loops and harnesses that forbid hipMalloc):
 * relaxkv_query_attn without a workspace argument.  Same arguments, kernels and
 * results as relaxkv_query_attn; its scratch is a device array of
 * RELAXKV_QUERY_ATTN_NOALLOC_MAX_BYTES inside the library, which each GPU it runs
 * on holds until the process ends.  It calls no allocating routine.
 * RELAXKV_ENOSPACE when relaxkv_query_attn_workspace_bytes(p) exceeds
 * RELAXKV_QUERY_ATTN_NOALLOC_MAX_BYTES (e.g. bf16, H_kv 8, 64 query tokens x 5
 * heads: 21 MB at any T_c up to 131072).  Every call on one GPU shares that GPU's
 * scratch: calls that overlap on one device (other streams or threads) race and
 * must be ordered by the caller.  Nothing in the scratch needs clearing: each
 * call writes every element it reads.
 */
relaxkv_status relaxkv_query_attn_noalloc(const relaxkv_problem* p, int32_t layer,
                                          const void* k_cache, const void* v_cache,
                                          const void* k_q, const void* v_q, void* out,
                                          float* lse_out, void* stream);

/*
 * Synchronising.  Copies s->counts ([L+2] int32) to host_counts and, when
 * host_edges is not NULL, s->edges ([2L] int64) to host_edges, after all work
 * queued on `stream`.  Returns RELAXKV_EINVAL when the device error word is
 * set (RELAXKV_ERR_* bits: a NaN score, an invalid global target list, or more
 * active targets than an attention or cache-update call could process; the
 * counts are still copied), RELAXKV_EDEVICE on a HIP error.
 */
relaxkv_status relaxkv_counts_to_host(const relaxkv_sets* s, int32_t* host_counts,
                                      int64_t* host_edges, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RELAXKV_H */
