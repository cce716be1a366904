// Internal declarations shared by the host C ABI and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_config.h"
#include "relaxkv.h"

namespace relaxkv {

// Element strides of k_cache and v_cache (layer, KV head, token), the
// descriptor's zeros replaced by the dense values.
struct KvStrides {
    int64_t layer, head, token;
};

inline KvStrides kv_strides(const relaxkv_problem& p) {
    KvStrides s;
    s.token = p.kv_stride_token ? p.kv_stride_token : p.d;
    s.head = p.kv_stride_head ? p.kv_stride_head : (int64_t)p.T_c * s.token;
    s.layer = p.kv_stride_layer ? p.kv_stride_layer : (int64_t)p.H_kv * s.head;
    return s;
}

// Scratch layout of relaxkv_score (offsets in bytes from the workspace base).
struct ScoreWorkspace {
    size_t part_off;    // float [L][n_part][T_c]   per-KV-head pooled partial sums
    size_t stats_off;   // float2 [L][H_kv][n_split][rows_pad] (max, sum) per key split, log2 units
    size_t lse_off;     // float [L][H_kv][rows_pad] row log2-sum-exp
    size_t mm_off;      // float2 [L][n_blk] (min, max) of p per finaliser block
    size_t total;
    int n_blk;          // finaliser blocks per layer
    int n_part;         // partial slices summed by the finaliser
    int n_split;        // key splits of the row-statistics pass
    int rows_pad;       // n_query * G rounded up to a multiple of 32
};

ScoreWorkspace score_workspace_layout(const relaxkv_problem& p);

// Scratch layout of relaxkv_query_attn (bf16 path; the fp32 path needs none).
struct QueryAttnWorkspace {
    size_t part_o_off;  // bf16 [n_split][H_kv][rows_pad][d] normalised partial outputs
    size_t part_l_off;  // float [n_split][H_kv][rows_pad] log2-sum-exp of each partial
    size_t total;
    int n_split;        // cache-key splits (the last also takes the query tokens' keys)
    int kps;            // cache keys per split (a multiple of 64)
    int n_chunks;       // row chunks of up to 320 rows per KV head
    int rows_pad;       // n_query * G rounded up to a multiple of 32
};

QueryAttnWorkspace query_attn_workspace_layout(const relaxkv_problem& p);

// Kernel launchers (each returns hipSuccess or the launch error).
hipError_t launch_score(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                        float* scores, hipStream_t st);
hipError_t launch_select(const relaxkv_problem& p, const float* scores,
                         const relaxkv_sets& s, hipStream_t st);
hipError_t launch_select_global(const relaxkv_problem& p, const float* scores, int k_target,
                                const relaxkv_sets& s, float* g, int32_t* targets,
                                int32_t* n_targets, hipStream_t st);
hipError_t launch_build_sets_context(const relaxkv_problem& p, const float* scores,
                                     int construction, const relaxkv_sets& s, hipStream_t st);
hipError_t launch_select_rows(const float* scores, int n_rows, int T, int k, const int32_t* k_cap,
                              int32_t* out, int out_stride, int32_t* counts, int L,
                              hipStream_t st);
hipError_t launch_global_mean(const float* scores, int L, int T, float* g, hipStream_t st);
hipError_t launch_build_sets_global(const relaxkv_problem& p, const relaxkv_sets& s,
                                    const int32_t* targets, const int32_t* n_targets,
                                    hipStream_t st);
hipError_t launch_build_sets(const relaxkv_problem& p, const relaxkv_sets& s,
                             hipStream_t st);
hipError_t launch_update_cache(const relaxkv_problem& p, const relaxkv_sets& s, int layer,
                               const void* k_new, const void* v_new, int n_rows, void* k_cache,
                               void* v_cache, hipStream_t st);
hipError_t launch_query_attn(const relaxkv_problem& p, int layer, const void* k_cache,
                             const void* v_cache, const void* k_q, const void* v_q, void* out,
                             float* lse_out, char* ws, hipStream_t st);
hipError_t launch_sparse_attn(const relaxkv_problem& p, const relaxkv_sets& s, int layer,
                              const void* q_new, const void* k_new, const void* v_new,
                              int n_rows, void* out, float* lse_out, int context_mode,
                              hipStream_t st);

// Words of relaxkv_sets::tiles: per context mode and layer, one next-tile
// counter per KV head and one workgroup count.
inline size_t attn_tile_words(const relaxkv_problem& p) {
    return 2 * (size_t)p.L * (size_t)(p.H_kv + 1);
}

// Rows an attention or cache-update launch may process for layer `layer`: the
// caller's row capacity, and the bound on |R_l| of the lists the sets hold
// (min(T_c, (L - l) k) for RelaxKV's targets: R_l lies in the union of S_l'
// for l' >= l; T_c for a global target list).  Kernels clamp the device count
// to it and set RELAXKV_ERR_ROWS when they have to.
inline int row_cap(const relaxkv_problem& p, const relaxkv_sets& s, int layer, int n_rows) {
    const long kb = s.global_targets ? (long)p.T_c : (long)(p.L - layer) * s.k;
    long cap = kb < p.T_c ? kb : p.T_c;
    if (n_rows < cap) cap = n_rows;
    return (int)cap;
}


}  // namespace relaxkv
