// Host side of the C ABI: validation, buffer sizing and carving, launches.
// Nothing here allocates device memory; every buffer belongs to the caller.

#include <math.h>
#include <stdint.h>
#include <string.h>

#include "internal.h"

using namespace relaxkv;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool dims_ok(const relaxkv_problem* p) {
    return p->L >= 1 && p->L <= RELAXKV_MAX_LAYERS && p->T_c >= 1 && p->T_c <= RELAXKV_MAX_TC &&
           p->n_query >= 1 && p->n_query <= 4096 && p->H >= 1 && p->H <= 1024 &&
           p->H_kv >= 1 && p->H % p->H_kv == 0 &&
           (int64_t)p->L * p->T_c <= INT32_MAX;          // CSR offsets over layers are int32
}

// Byte sizes of the set arrays, in carving order.
struct SetsLayout {
    size_t anchors, h, U, cidx, R_off, R_idx, R_u, src, rank, counts, edges, ctx, g, tiles, total;
};

SetsLayout sets_layout(const relaxkv_problem* p, int32_t k) {
    SetsLayout s;
    const size_t L = (size_t)p->L, T = (size_t)p->T_c;
    s.anchors = align_up(L * (size_t)k * 4);
    s.h = align_up(T * 4);
    s.U = align_up(T * 4);
    s.cidx = align_up(T * 4);
    s.R_off = align_up((L + 1) * 4);
    s.R_idx = align_up(L * T * 4);
    s.R_u = align_up(L * T * 4);
    s.src = align_up(L * T * 4);
    s.rank = align_up(L * T * 4);
    s.counts = align_up((L + 2) * 4);
    s.edges = align_up(2 * L * 8);
    s.ctx = align_up(L * T * 4);
    s.g = align_up(T * 4);
    s.tiles = align_up(attn_tile_words(*p) * 4);
    s.total = s.anchors + s.h + s.U + s.cidx + s.R_off + s.R_idx + s.R_u + s.src + s.rank + s.counts +
              s.edges + s.ctx + s.g + s.tiles;
    return s;
}

bool sets_match(const relaxkv_problem* p, const relaxkv_sets* s) {
    return s && s->L == p->L && s->T_c == p->T_c &&
           s->k == relaxkv_anchor_count(p->anchor_ratio, p->T_c) && s->anchors && s->h &&
           s->U && s->cidx && s->R_off && s->R_idx && s->R_u && s->src && s->rank && s->counts &&
           s->edges && s->ctx && s->g && s->tiles &&
           s->context_sets >= RELAXKV_CONTEXT_SETS_UNION &&
           s->context_sets <= RELAXKV_CONTEXT_SETS_LAYERWISE;
}

// The cache strides: none negative; no two rows overlap, i.e. taken from the
// smallest, each stride of a dimension with more than one entry steps past the
// whole extent of the dimensions inside it; an extent below 2^48 elements (no
// device holds more, and every offset the kernels form then fits in 64 bits);
// 16-byte aligned rows and pointers (the kernels move rows in 16-byte pieces);
// and, for bf16, cached-row offsets within a head that fit the attention's
// 32-bit element offsets.  The stride of a dimension with one entry is never
// used and is not checked.
relaxkv_status strides_status(const relaxkv_problem* p) {
    if (p->kv_stride_layer < 0 || p->kv_stride_head < 0 || p->kv_stride_token < 0)
        return RELAXKV_EINVAL;
    constexpr int64_t kMaxExtent = (int64_t)1 << 48;
    // The dense defaults (as kv_strides forms them), with overflow checks.
    int64_t sT = p->kv_stride_token ? p->kv_stride_token : p->d, sH, sL;
    if (p->kv_stride_head) sH = p->kv_stride_head;
    else if (__builtin_mul_overflow((int64_t)p->T_c, sT, &sH)) return RELAXKV_EUNSUPPORTED;
    if (p->kv_stride_layer) sL = p->kv_stride_layer;
    else if (__builtin_mul_overflow((int64_t)p->H_kv, sH, &sL)) return RELAXKV_EUNSUPPORTED;
    struct Dim { int64_t stride, n; } dims[3] = {{sT, p->T_c}, {sH, p->H_kv}, {sL, p->L}};
    for (int i = 1; i < 3; ++i)                          // ascending strides (insertion sort)
        for (int j = i; j > 0 && dims[j].stride < dims[j - 1].stride; --j) {
            const Dim t = dims[j];
            dims[j] = dims[j - 1];
            dims[j - 1] = t;
        }
    const int64_t align = p->dtype == RELAXKV_DTYPE_BF16 ? 8 : 4;   // elements per 16 bytes
    int64_t extent = p->d;                               // elements spanned by the inner dimensions
    for (const Dim& dm : dims) {
        if (dm.n <= 1) continue;
        if (dm.stride < extent) return RELAXKV_EINVAL;
        if (dm.stride % align) return RELAXKV_EUNSUPPORTED;
        // extent += (n - 1) * stride, kept below 2^48
        if (dm.stride > (kMaxExtent - extent) / (dm.n - 1)) return RELAXKV_EUNSUPPORTED;
        extent += (dm.n - 1) * dm.stride;
    }
    if ((uintptr_t)p->q % 16 || (uintptr_t)p->k_cache % 16 || (uintptr_t)p->v_cache % 16)
        return RELAXKV_EUNSUPPORTED;
    // (the bf16 attention forms the offset with a 24-bit multiply)
    if (p->dtype == RELAXKV_DTYPE_BF16 && p->T_c > 1 &&
        (sT >= ((int64_t)1 << 24) ||
         (int64_t)(p->T_c - 1) * sT + p->d >= RELAXKV_MAX_BF16_LAYER_ELEMS))
        return RELAXKV_EUNSUPPORTED;
    return RELAXKV_OK;
}

relaxkv_status from_hip(hipError_t e) { return e == hipSuccess ? RELAXKV_OK : RELAXKV_EDEVICE; }

}  // namespace

extern "C" {

const char* relaxkv_status_string(relaxkv_status s) {
    switch (s) {
        case RELAXKV_OK: return "ok";
        case RELAXKV_EINVAL: return "invalid argument";
        case RELAXKV_ENOSPACE: return "buffer too small";
        case RELAXKV_EUNSUPPORTED: return "unsupported shape or dtype";
        case RELAXKV_EDEVICE: return "HIP runtime error";
        default: return "unknown status";
    }
}

int32_t relaxkv_anchor_count(double r, int32_t T_c) {
    if (!isfinite(r) || r < 0.0 || r > 1.0 || T_c < 1) return RELAXKV_EINVAL;
    // round-half-to-even in double (the default rounding mode of nearbyint)
    double k = nearbyint(r * (double)T_c);
    if (k < 1.0) k = 1.0;
    if (k > (double)T_c) k = (double)T_c;
    return (int32_t)k;
}

relaxkv_status relaxkv_validate(const relaxkv_problem* p) {
    if (!p) return RELAXKV_EINVAL;
    if (!dims_ok(p)) return RELAXKV_EINVAL;
    if (!p->q || !p->k_cache || !p->v_cache) return RELAXKV_EINVAL;
    if (isnan(p->softmax_scale) || isinf(p->softmax_scale)) return RELAXKV_EINVAL;
    if (relaxkv_anchor_count(p->anchor_ratio, p->T_c) < 1) return RELAXKV_EINVAL;
    if (p->dtype != RELAXKV_DTYPE_F32 && p->dtype != RELAXKV_DTYPE_BF16)
        return RELAXKV_EUNSUPPORTED;
    if (p->d != 64 && p->d != 128) return RELAXKV_EUNSUPPORTED;
    // The bf16 attention counts (target, head) rows of a KV head in 32-bit
    // integers: |R_l| * G < 2^22 * kAttnRows < 2^31.
    if (p->dtype == RELAXKV_DTYPE_BF16 && p->H / p->H_kv > kAttnRows) return RELAXKV_EUNSUPPORTED;
    // The bf16 attention's fills address fresh and cached rows with 32-bit
    // element offsets (below T_c * H_kv * d).
    if (p->dtype == RELAXKV_DTYPE_BF16 &&
        (int64_t)p->T_c * p->H_kv * p->d >= RELAXKV_MAX_BF16_LAYER_ELEMS)
        return RELAXKV_EUNSUPPORTED;
    return strides_status(p);
}

size_t relaxkv_score_workspace_bytes(const relaxkv_problem* p) {
    if (relaxkv_validate(p) != RELAXKV_OK) return 0;
    return score_workspace_layout(*p).total;
}

size_t relaxkv_sets_bytes(const relaxkv_problem* p) {
    if (relaxkv_validate(p) != RELAXKV_OK) return 0;
    return sets_layout(p, relaxkv_anchor_count(p->anchor_ratio, p->T_c)).total;
}

relaxkv_status relaxkv_sets_bind(const relaxkv_problem* p, void* dev_buf, size_t bytes,
                                 relaxkv_sets* out) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!dev_buf || !out) return RELAXKV_EINVAL;
    if (((uintptr_t)dev_buf) % kAlign) return RELAXKV_EINVAL;
    const int32_t k = relaxkv_anchor_count(p->anchor_ratio, p->T_c);
    SetsLayout l = sets_layout(p, k);
    if (bytes < l.total) return RELAXKV_ENOSPACE;
    char* b = (char*)dev_buf;
    relaxkv_sets s;
    s.L = p->L;
    s.T_c = p->T_c;
    s.k = k;
    s.anchors = (int32_t*)b; b += l.anchors;
    s.h = (int32_t*)b; b += l.h;
    s.U = (int32_t*)b; b += l.U;
    s.cidx = (int32_t*)b; b += l.cidx;
    s.R_off = (int32_t*)b; b += l.R_off;
    s.R_idx = (int32_t*)b; b += l.R_idx;
    s.R_u = (int32_t*)b; b += l.R_u;
    s.src = (int32_t*)b; b += l.src;
    s.rank = (int32_t*)b; b += l.rank;
    s.counts = (int32_t*)b; b += l.counts;
    s.edges = (int64_t*)b; b += l.edges;
    s.ctx = (int32_t*)b; b += l.ctx;
    s.g = (float*)b; b += l.g;
    s.tiles = (uint32_t*)b;
    s.global_targets = 0;
    s.context_sets = RELAXKV_CONTEXT_SETS_UNION;
    *out = s;
    return RELAXKV_OK;
}

relaxkv_status relaxkv_score(const relaxkv_problem* p, void* ws, size_t ws_bytes,
                             float* scores, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!ws || !scores) return RELAXKV_EINVAL;
    ScoreWorkspace w = score_workspace_layout(*p);
    if (ws_bytes < w.total) return RELAXKV_ENOSPACE;
    return from_hip(launch_score(*p, w, (char*)ws, scores, (hipStream_t)stream));
}

relaxkv_status relaxkv_select(const relaxkv_problem* p, const float* scores,
                              const relaxkv_sets* s, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!scores || !sets_match(p, s)) return RELAXKV_EINVAL;
    return from_hip(launch_select(*p, scores, *s, (hipStream_t)stream));
}

relaxkv_status relaxkv_build_sets(const relaxkv_problem* p, relaxkv_sets* s, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!sets_match(p, s)) return RELAXKV_EINVAL;
    st = from_hip(launch_build_sets(*p, *s, (hipStream_t)stream));
    if (st == RELAXKV_OK) {
        s->global_targets = 0;
        s->context_sets = RELAXKV_CONTEXT_SETS_UNION;
    }
    return st;
}

relaxkv_status relaxkv_build_sets_context(const relaxkv_problem* p, const float* scores,
                                          int32_t construction, relaxkv_sets* s, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!scores || !sets_match(p, s)) return RELAXKV_EINVAL;
    if (construction < RELAXKV_CONTEXT_SETS_UNION || construction > RELAXKV_CONTEXT_SETS_LAYERWISE)
        return RELAXKV_EINVAL;
    st = from_hip(launch_build_sets_context(*p, scores, construction, *s, (hipStream_t)stream));
    if (st == RELAXKV_OK) {
        s->global_targets = 0;
        s->context_sets = construction;
    }
    return st;
}

relaxkv_status relaxkv_select_global(const relaxkv_problem* p, const float* scores,
                                     double target_ratio, const relaxkv_sets* s, float* g,
                                     int32_t* targets, int32_t* n_targets, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!scores || !g || !targets || !n_targets || !sets_match(p, s)) return RELAXKV_EINVAL;
    if (!isfinite(target_ratio) || target_ratio < 0.0 || target_ratio > 1.0) return RELAXKV_EINVAL;
    double kt = floor(target_ratio * (double)p->T_c);           // floor(r_g T_c) in double
    if (kt > (double)p->T_c) kt = (double)p->T_c;
    return from_hip(launch_select_global(*p, scores, (int)kt, *s, g, targets, n_targets,
                                         (hipStream_t)stream));
}

relaxkv_status relaxkv_build_sets_global(const relaxkv_problem* p, relaxkv_sets* s,
                                         const int32_t* targets, const int32_t* n_targets,
                                         void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!targets || !n_targets || !sets_match(p, s)) return RELAXKV_EINVAL;
    st = from_hip(launch_build_sets_global(*p, *s, targets, n_targets, (hipStream_t)stream));
    if (st == RELAXKV_OK) {
        s->global_targets = 1;
        s->context_sets = RELAXKV_CONTEXT_SETS_UNION;
    }
    return st;
}

relaxkv_status relaxkv_sparse_attn(const relaxkv_problem* p, const relaxkv_sets* s,
                                   int32_t layer, const void* q_new, const void* k_new,
                                   const void* v_new, int32_t n_rows, void* out,
                                   float* lse_out, int32_t context_mode, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!sets_match(p, s)) return RELAXKV_EINVAL;
    if (layer < 0 || layer >= p->L || n_rows < 0) return RELAXKV_EINVAL;
    if (n_rows > 0 && (!q_new || !k_new || !v_new || !out)) return RELAXKV_EINVAL;
    if (context_mode != RELAXKV_CONTEXT_UNION && context_mode != RELAXKV_CONTEXT_FULL)
        return RELAXKV_EINVAL;
    return from_hip(launch_sparse_attn(*p, *s, layer, q_new, k_new, v_new, n_rows, out,
                                       lse_out, context_mode, (hipStream_t)stream));
}

relaxkv_status relaxkv_update_cache(const relaxkv_problem* p, const relaxkv_sets* s,
                                    int32_t layer, const void* k_new, const void* v_new,
                                    int32_t n_rows, void* k_cache, void* v_cache,
                                    void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (!sets_match(p, s)) return RELAXKV_EINVAL;
    if (layer < 0 || layer >= p->L || n_rows < 0) return RELAXKV_EINVAL;
    if ((n_rows > 0 && (!k_new || !v_new)) || !k_cache || !v_cache) return RELAXKV_EINVAL;
    return from_hip(launch_update_cache(*p, *s, layer, k_new, v_new, n_rows, k_cache, v_cache,
                                        (hipStream_t)stream));
}

size_t relaxkv_query_attn_workspace_bytes(const relaxkv_problem* p) {
    if (relaxkv_validate(p) != RELAXKV_OK) return 0;
    return query_attn_workspace_layout(*p).total;
}

relaxkv_status relaxkv_query_attn(const relaxkv_problem* p, int32_t layer, const void* k_cache,
                                  const void* v_cache, const void* k_q, const void* v_q,
                                  void* out, float* lse_out, void* ws, size_t ws_bytes,
                                  void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (layer < 0 || layer >= p->L) return RELAXKV_EINVAL;
    if (!k_cache || !v_cache || !k_q || !v_q || !out) return RELAXKV_EINVAL;
    const QueryAttnWorkspace w = query_attn_workspace_layout(*p);
    if (w.total && !ws) return RELAXKV_EINVAL;
    if (ws_bytes < w.total) return RELAXKV_ENOSPACE;
    return from_hip(launch_query_attn(*p, layer, k_cache, v_cache, k_q, v_q, out, lse_out,
                                      (char*)ws, (hipStream_t)stream));
}

relaxkv_status relaxkv_counts_to_host(const relaxkv_sets* s, int32_t* host_counts,
                                      int64_t* host_edges, void* stream) {
    if (!s || !s->counts || !s->edges || !host_counts || s->L < 1) return RELAXKV_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e = hipMemcpyAsync(host_counts, s->counts, sizeof(int32_t) * (s->L + 2),
                                  hipMemcpyDeviceToHost, st);
    if (e == hipSuccess && host_edges)
        e = hipMemcpyAsync(host_edges, s->edges, sizeof(int64_t) * 2 * s->L,
                           hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return RELAXKV_EDEVICE;
    return host_counts[s->L + 1] != 0 ? RELAXKV_EINVAL : RELAXKV_OK;
}

}  // extern "C"
