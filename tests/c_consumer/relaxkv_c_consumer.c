/*
 * A plain C11 consumer of the library: it includes only include/relaxkv.h and
 * the HIP runtime API, owns its device memory, and runs the per-request path
 * (relaxkv_score -> relaxkv_select -> relaxkv_build_sets ->
 * relaxkv_counts_to_host -> relaxkv_sparse_attn for every layer) the way a
 * serving engine written in C would.  Test infrastructure: the Python tests
 * write its seeded inputs, run it, and compare what it writes with the oracle.
 *
 *   relaxkv_c_consumer host
 *       Host-only calls (no device work): prints "key value" lines.
 *   relaxkv_c_consumer run DIR
 *       DIR/params.txt "L T_c n_query H H_kv d anchor_ratio"; DIR/q.bin,
 *       kc.bin, vc.bin (bf16 [L][n_query][H][d], [L][H_kv][T_c][d] x 2);
 *       DIR/fq_<l>.bin, fk_<l>.bin, fv_<l>.bin (bf16 fresh rows of every
 *       position, [T_c][H][d] and [T_c][H_kv][d] x 2).  Writes scores.bin
 *       (f32 [L][T_c]), anchors.bin (i32 [L][k]), counts.bin (i32 [L+2]),
 *       r_off.bin, r_idx.bin (i32) and out_<l>.bin (bf16 [|R_l|][H][d]),
 *       lse_<l>.bin (f32 [|R_l|][H]).
 * Exit status 0 on success; any failed call prints its name and status.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "relaxkv.h"

#define CHECK_RK(call)                                                                   \
    do {                                                                                 \
        relaxkv_status st_ = (call);                                                     \
        if (st_ != RELAXKV_OK) {                                                         \
            fprintf(stderr, "%s: %s (%d)\n", #call, relaxkv_status_string(st_), (int)st_); \
            exit(1);                                                                     \
        }                                                                                \
    } while (0)

#define CHECK_HIP(call)                                                              \
    do {                                                                             \
        hipError_t e_ = (call);                                                      \
        if (e_ != hipSuccess) {                                                      \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));               \
            exit(1);                                                                 \
        }                                                                            \
    } while (0)

static void* read_file(const char* dir, const char* name, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "rb");
    if (!f) {
        fprintf(stderr, "cannot open %s\n", path);
        exit(1);
    }
    void* buf = malloc(bytes ? bytes : 1);
    if (!buf || fread(buf, 1, bytes, f) != bytes) {
        fprintf(stderr, "short read %s\n", path);
        exit(1);
    }
    fclose(f);
    return buf;
}

static void write_file(const char* dir, const char* name, const void* buf, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(buf, 1, bytes, f) != bytes) {
        fprintf(stderr, "cannot write %s\n", path);
        exit(1);
    }
    fclose(f);
}

static void* to_device(const void* host, size_t bytes) {
    void* d = NULL;
    CHECK_HIP(hipMalloc(&d, bytes ? bytes : 1));
    if (bytes) CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
    return d;
}

static relaxkv_problem problem(int L, int T, int Qn, int H, int Hkv, int d, double r) {
    relaxkv_problem p;
    memset(&p, 0, sizeof p);
    p.L = L;
    p.T_c = T;
    p.n_query = Qn;
    p.H = H;
    p.H_kv = Hkv;
    p.d = d;
    p.dtype = RELAXKV_DTYPE_BF16;
    p.softmax_scale = 0.0f;
    p.anchor_ratio = r;
    return p;
}

/* Host-only calls: sizes, validation and argument checks that reject before
 * anything is enqueued (no device is touched). */
static int run_host(void) {
    relaxkv_problem p = problem(4, 2048, 16, 8, 2, 128, 0.15);
    p.q = (const void*)(uintptr_t)0x1000;
    p.k_cache = (const void*)(uintptr_t)0x2000;
    p.v_cache = (const void*)(uintptr_t)0x3000;
    printf("anchor_count_0.15_2048 %d\n", (int)relaxkv_anchor_count(0.15, 2048));
    printf("anchor_count_0.125_20 %d\n", (int)relaxkv_anchor_count(0.125, 20));
    printf("anchor_count_bad %d\n", (int)relaxkv_anchor_count(1.5, 10));
    printf("validate_ok %d\n", (int)relaxkv_validate(&p));
    relaxkv_problem bad = p;
    bad.d = 96;
    printf("validate_d96 %d\n", (int)relaxkv_validate(&bad));
    bad = p;
    bad.H = 6;
    bad.H_kv = 4;
    printf("validate_gqa %d\n", (int)relaxkv_validate(&bad));
    const size_t sb = relaxkv_sets_bytes(&p);
    printf("sets_bytes %zu\n", sb);
    printf("score_ws_bytes %zu\n", relaxkv_score_workspace_bytes(&p));
    relaxkv_sets s;
    void* fake = (void*)(uintptr_t)0x7f0000000000ull;         /* never dereferenced */
    printf("sets_bind %d\n", (int)relaxkv_sets_bind(&p, fake, sb, &s));
    printf("sets_bind_short %d\n", (int)relaxkv_sets_bind(&p, fake, sb - 1, &s));
    printf("sets_k %d\n", (int)s.k);
    printf("sets_tiles_offset %zu\n", (size_t)((char*)s.tiles - (char*)fake));
    printf("score_null_ws %d\n", (int)relaxkv_score(&p, NULL, 0, (float*)fake, NULL));
    printf("attn_bad_layer %d\n",
           (int)relaxkv_sparse_attn(&p, &s, 4, fake, fake, fake, 1, fake, NULL,
                                    RELAXKV_CONTEXT_UNION, NULL));
    printf("attn_neg_rows %d\n",
           (int)relaxkv_sparse_attn(&p, &s, 0, fake, fake, fake, -1, fake, NULL,
                                    RELAXKV_CONTEXT_UNION, NULL));
    printf("status_string %s\n", relaxkv_status_string(RELAXKV_ENOSPACE));
    return 0;
}

static int run_pipeline(const char* dir) {
    int L, T, Qn, H, Hkv, d;
    double r;
    {
        char path[4096];
        snprintf(path, sizeof path, "%s/params.txt", dir);
        FILE* f = fopen(path, "r");
        if (!f || fscanf(f, "%d %d %d %d %d %d %lf", &L, &T, &Qn, &H, &Hkv, &d, &r) != 7) {
            fprintf(stderr, "bad %s\n", path);
            return 1;
        }
        fclose(f);
    }
    const size_t e2 = 2;                                       /* bf16 bytes */
    const size_t q_bytes = (size_t)L * Qn * H * d * e2;
    const size_t c_bytes = (size_t)L * Hkv * T * d * e2;
    void* hq = read_file(dir, "q.bin", q_bytes);
    void* hk = read_file(dir, "kc.bin", c_bytes);
    void* hv = read_file(dir, "vc.bin", c_bytes);
    relaxkv_problem p = problem(L, T, Qn, H, Hkv, d, r);
    p.q = to_device(hq, q_bytes);
    p.k_cache = to_device(hk, c_bytes);
    p.v_cache = to_device(hv, c_bytes);
    free(hq);
    free(hk);
    free(hv);
    CHECK_RK(relaxkv_validate(&p));

    hipStream_t st;
    CHECK_HIP(hipStreamCreate(&st));
    const size_t ws_bytes = relaxkv_score_workspace_bytes(&p);
    const size_t sets_bytes = relaxkv_sets_bytes(&p);
    void *ws = NULL, *sets_buf = NULL;
    float* scores = NULL;
    CHECK_HIP(hipMalloc(&ws, ws_bytes));
    CHECK_HIP(hipMalloc(&sets_buf, sets_bytes));
    CHECK_HIP(hipMalloc((void**)&scores, (size_t)L * T * sizeof(float)));
    relaxkv_sets s;
    CHECK_RK(relaxkv_sets_bind(&p, sets_buf, sets_bytes, &s));

    CHECK_RK(relaxkv_score(&p, ws, ws_bytes, scores, st));
    CHECK_RK(relaxkv_select(&p, scores, &s, st));
    CHECK_RK(relaxkv_build_sets(&p, &s, st));
    int32_t* counts = (int32_t*)malloc((size_t)(L + 2) * sizeof(int32_t));
    int64_t* edges = (int64_t*)malloc((size_t)2 * L * sizeof(int64_t));
    CHECK_RK(relaxkv_counts_to_host(&s, counts, edges, st));

    float* h_scores = (float*)malloc((size_t)L * T * sizeof(float));
    int32_t* h_anchors = (int32_t*)malloc((size_t)L * s.k * sizeof(int32_t));
    int32_t* r_off = (int32_t*)malloc((size_t)(L + 1) * sizeof(int32_t));
    CHECK_HIP(hipMemcpy(h_scores, scores, (size_t)L * T * sizeof(float), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(h_anchors, s.anchors, (size_t)L * s.k * sizeof(int32_t),
                        hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(r_off, s.R_off, (size_t)(L + 1) * sizeof(int32_t), hipMemcpyDeviceToHost));
    const int32_t n_all = r_off[L];
    int32_t* r_idx = (int32_t*)malloc((size_t)(n_all ? n_all : 1) * sizeof(int32_t));
    if (n_all)
        CHECK_HIP(hipMemcpy(r_idx, s.R_idx, (size_t)n_all * sizeof(int32_t), hipMemcpyDeviceToHost));
    write_file(dir, "scores.bin", h_scores, (size_t)L * T * sizeof(float));
    write_file(dir, "anchors.bin", h_anchors, (size_t)L * s.k * sizeof(int32_t));
    write_file(dir, "counts.bin", counts, (size_t)(L + 2) * sizeof(int32_t));
    write_file(dir, "r_off.bin", r_off, (size_t)(L + 1) * sizeof(int32_t));
    write_file(dir, "r_idx.bin", r_idx, (size_t)n_all * sizeof(int32_t));

    const size_t qrow = (size_t)H * d * e2, kvrow = (size_t)Hkv * d * e2;
    for (int l = 0; l < L; ++l) {
        const int n = counts[1 + l];
        const int32_t* R = r_idx + r_off[l];
        char name[64];
        snprintf(name, sizeof name, "fq_%d.bin", l);
        unsigned char* fq = (unsigned char*)read_file(dir, name, (size_t)T * qrow);
        snprintf(name, sizeof name, "fk_%d.bin", l);
        unsigned char* fk = (unsigned char*)read_file(dir, name, (size_t)T * kvrow);
        snprintf(name, sizeof name, "fv_%d.bin", l);
        unsigned char* fv = (unsigned char*)read_file(dir, name, (size_t)T * kvrow);
        /* the active targets' fresh rows, in R_l order */
        unsigned char* gq = (unsigned char*)malloc((size_t)(n ? n : 1) * qrow);
        unsigned char* gk = (unsigned char*)malloc((size_t)(n ? n : 1) * kvrow);
        unsigned char* gv = (unsigned char*)malloc((size_t)(n ? n : 1) * kvrow);
        for (int t = 0; t < n; ++t) {
            memcpy(gq + (size_t)t * qrow, fq + (size_t)R[t] * qrow, qrow);
            memcpy(gk + (size_t)t * kvrow, fk + (size_t)R[t] * kvrow, kvrow);
            memcpy(gv + (size_t)t * kvrow, fv + (size_t)R[t] * kvrow, kvrow);
        }
        void* dq = to_device(gq, (size_t)n * qrow);
        void* dk = to_device(gk, (size_t)n * kvrow);
        void* dv = to_device(gv, (size_t)n * kvrow);
        void* dout = NULL;
        float* dlse = NULL;
        CHECK_HIP(hipMalloc(&dout, (size_t)(n ? n : 1) * qrow));
        CHECK_HIP(hipMalloc((void**)&dlse, (size_t)(n ? n : 1) * H * sizeof(float)));
        CHECK_RK(relaxkv_sparse_attn(&p, &s, l, dq, dk, dv, n, dout, dlse, RELAXKV_CONTEXT_UNION,
                                     st));
        CHECK_HIP(hipStreamSynchronize(st));
        CHECK_HIP(hipMemcpy(gq, dout, (size_t)n * qrow, hipMemcpyDeviceToHost));
        float* hl = (float*)malloc((size_t)(n ? n : 1) * H * sizeof(float));
        CHECK_HIP(hipMemcpy(hl, dlse, (size_t)n * H * sizeof(float), hipMemcpyDeviceToHost));
        snprintf(name, sizeof name, "out_%d.bin", l);
        write_file(dir, name, gq, (size_t)n * qrow);
        snprintf(name, sizeof name, "lse_%d.bin", l);
        write_file(dir, name, hl, (size_t)n * H * sizeof(float));
        CHECK_HIP(hipFree(dq));
        CHECK_HIP(hipFree(dk));
        CHECK_HIP(hipFree(dv));
        CHECK_HIP(hipFree(dout));
        CHECK_HIP(hipFree(dlse));
        free(fq);
        free(fk);
        free(fv);
        free(gq);
        free(gk);
        free(gv);
        free(hl);
    }
    /* the error word must be clear after the whole path */
    CHECK_RK(relaxkv_counts_to_host(&s, counts, edges, st));
    CHECK_HIP(hipStreamDestroy(st));
    CHECK_HIP(hipFree(ws));
    CHECK_HIP(hipFree(sets_buf));
    CHECK_HIP(hipFree(scores));
    CHECK_HIP(hipFree((void*)p.q));
    CHECK_HIP(hipFree((void*)p.k_cache));
    CHECK_HIP(hipFree((void*)p.v_cache));
    free(counts);
    free(edges);
    free(h_scores);
    free(h_anchors);
    free(r_off);
    free(r_idx);
    printf("ok\n");
    return 0;
}

int main(int argc, char** argv) {
    if (argc == 2 && strcmp(argv[1], "host") == 0) return run_host();
    if (argc == 3 && strcmp(argv[1], "run") == 0) return run_pipeline(argv[2]);
    fprintf(stderr, "usage: %s host | run DIR\n", argv[0]);
    return 2;
}
