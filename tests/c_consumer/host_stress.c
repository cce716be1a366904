/*
 * Host-side stress of the library for the sanitizer build (test
 * infrastructure): over a grid of problem shapes, from tiny to the limits the
 * header states, it calls every host-only function (validation, size queries,
 * binding, the anchor count, the cache-stride rules) and every compute entry point with an argument
 * that must be rejected before anything is enqueued, and checks the results
 * against the header's rules.  No call reaches a device: every compute call
 * here fails validation.  Built with AddressSanitizer and UndefinedBehavior-
 * Sanitizer (tests/c_consumer/build_sanitized.py); any finding aborts.
 * Prints "ok <checks>" and exits 0 when every check holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "relaxkv.h"

static long n_checks = 0;

#define EXPECT(cond, ...)                                                  \
    do {                                                                   \
        ++n_checks;                                                        \
        if (!(cond)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s: ", __LINE__, #cond); \
            fprintf(stderr, __VA_ARGS__);                                  \
            fprintf(stderr, "\n");                                         \
            exit(1);                                                       \
        }                                                                  \
    } while (0)

static relaxkv_problem make(int L, int T, int Qn, int H, int Hkv, int d, int dtype, double r) {
    relaxkv_problem p;
    memset(&p, 0, sizeof p);
    p.L = L;
    p.T_c = T;
    p.n_query = Qn;
    p.H = H;
    p.H_kv = Hkv;
    p.d = d;
    p.dtype = dtype;
    p.softmax_scale = 0.0f;
    p.anchor_ratio = r;
    p.q = (const void*)(uintptr_t)0x1000;
    p.k_cache = (const void*)(uintptr_t)0x2000;
    p.v_cache = (const void*)(uintptr_t)0x3000;
    p.q_lse = NULL;
    return p;
}

/* Every pointer of a bound sets struct lies inside [base, base + bytes) and is
 * 256-byte aligned. */
static void check_bound(const relaxkv_sets* s, uintptr_t base, size_t bytes) {
    const void* ptrs[] = {s->anchors, s->h, s->U, s->cidx, s->R_off, s->R_idx, s->R_u,
                          s->src, s->rank, s->counts, s->edges, s->ctx, s->g, s->tiles};
    for (size_t i = 0; i < sizeof ptrs / sizeof ptrs[0]; ++i) {
        const uintptr_t a = (uintptr_t)ptrs[i];
        EXPECT(a >= base && a < base + bytes, "pointer %zu outside the buffer", i);
        EXPECT(a % 256 == 0, "pointer %zu not 256-byte aligned", i);
    }
}

static void stress_problem(const relaxkv_problem* p0) {
    relaxkv_problem p = *p0;
    const relaxkv_status v = relaxkv_validate(&p);
    const size_t sb = relaxkv_sets_bytes(&p);
    const size_t wb = relaxkv_score_workspace_bytes(&p);
    const size_t qb = relaxkv_query_attn_workspace_bytes(&p);
    if (v != RELAXKV_OK) {
        EXPECT(sb == 0 && wb == 0 && qb == 0, "sizes of an invalid problem must be 0");
        EXPECT(v == RELAXKV_EINVAL || v == RELAXKV_EUNSUPPORTED, "status %d", (int)v);
        return;
    }
    EXPECT(sb > 0 && sb % 256 == 0, "sets bytes %zu", sb);
    EXPECT(wb % 256 == 0, "score workspace bytes %zu", wb);
    EXPECT(qb % 256 == 0, "query workspace bytes %zu", qb);
    const int32_t k = relaxkv_anchor_count(p.anchor_ratio, p.T_c);
    EXPECT(k >= 1 && k <= p.T_c, "k %d", (int)k);

    const uintptr_t base = (uintptr_t)0x7f0000000000ull;       /* never dereferenced */
    void* fake = (void*)base;
    relaxkv_sets s;
    memset(&s, 0, sizeof s);
    EXPECT(relaxkv_sets_bind(&p, fake, sb - 1, &s) == RELAXKV_ENOSPACE, "short buffer");
    EXPECT(relaxkv_sets_bind(&p, (void*)(base + 16), sb, &s) == RELAXKV_EINVAL, "misaligned");
    EXPECT(relaxkv_sets_bind(&p, fake, sb, &s) == RELAXKV_OK, "bind");
    EXPECT(s.L == p.L && s.T_c == p.T_c && s.k == k, "bound dims");
    check_bound(&s, base, sb);

    /* Each compute call with one argument that must be refused. */
    float* fscores = (float*)fake;
    if (wb)
        EXPECT(relaxkv_score(&p, fake, wb - 1, fscores, NULL) == RELAXKV_ENOSPACE,
               "score short workspace");
    EXPECT(relaxkv_score(&p, NULL, wb, fscores, NULL) == RELAXKV_EINVAL, "score null ws");
    EXPECT(relaxkv_select(&p, NULL, &s, NULL) == RELAXKV_EINVAL, "select null scores");
    relaxkv_sets other = s;
    other.L = p.L + 1;
    EXPECT(relaxkv_build_sets(&p, &other, NULL) == RELAXKV_EINVAL, "build_sets other L");
    EXPECT(relaxkv_build_sets_context(&p, fscores, 7, &s, NULL) == RELAXKV_EINVAL,
           "context construction 7");
    int32_t* ifake = (int32_t*)fake;
    EXPECT(relaxkv_select_global(&p, fscores, NAN, &s, fscores, ifake, ifake, NULL) ==
               RELAXKV_EINVAL, "select_global NaN ratio");
    EXPECT(relaxkv_select_global(&p, fscores, 1.5, &s, fscores, ifake, ifake, NULL) ==
               RELAXKV_EINVAL, "select_global ratio 1.5");
    EXPECT(relaxkv_build_sets_global(&p, &s, NULL, ifake, NULL) == RELAXKV_EINVAL,
           "build_sets_global null targets");
    EXPECT(relaxkv_sparse_attn(&p, &s, p.L, fake, fake, fake, 1, fake, NULL,
                               RELAXKV_CONTEXT_UNION, NULL) == RELAXKV_EINVAL, "attn layer L");
    EXPECT(relaxkv_sparse_attn(&p, &s, -1, fake, fake, fake, 1, fake, NULL,
                               RELAXKV_CONTEXT_UNION, NULL) == RELAXKV_EINVAL, "attn layer -1");
    EXPECT(relaxkv_sparse_attn(&p, &s, 0, fake, fake, fake, -1, fake, NULL,
                               RELAXKV_CONTEXT_UNION, NULL) == RELAXKV_EINVAL, "attn rows -1");
    EXPECT(relaxkv_sparse_attn(&p, &s, 0, fake, fake, fake, 1, fake, NULL, 2, NULL) ==
               RELAXKV_EINVAL, "attn mode 2");
    EXPECT(relaxkv_sparse_attn(&p, &s, 0, NULL, fake, fake, 1, fake, NULL,
                               RELAXKV_CONTEXT_UNION, NULL) == RELAXKV_EINVAL, "attn null q");
    EXPECT(relaxkv_update_cache(&p, &s, 0, fake, fake, 1, NULL, fake, NULL) == RELAXKV_EINVAL,
           "update null cache");
    EXPECT(relaxkv_update_cache(&p, &s, p.L, fake, fake, 1, fake, fake, NULL) ==
               RELAXKV_EINVAL, "update layer L");
    EXPECT(relaxkv_query_attn(&p, p.L, fake, fake, fake, fake, fake, NULL, fake, qb, NULL) ==
               RELAXKV_EINVAL, "query layer L");
    if (qb) {
        EXPECT(relaxkv_query_attn(&p, 0, fake, fake, fake, fake, fake, NULL, fake, qb - 1,
                                  NULL) == RELAXKV_ENOSPACE, "query short workspace");
        EXPECT(relaxkv_query_attn(&p, 0, fake, fake, fake, fake, fake, NULL, NULL, qb, NULL) ==
                   RELAXKV_EINVAL, "query null workspace");
    }
    EXPECT(relaxkv_query_attn_noalloc(&p, -1, fake, fake, fake, fake, fake, NULL, NULL) ==
               RELAXKV_EINVAL, "noalloc layer -1");
    EXPECT(relaxkv_query_attn_noalloc(&p, 0, NULL, fake, fake, fake, fake, NULL, NULL) ==
               RELAXKV_EINVAL, "noalloc null cache");
    if (qb > RELAXKV_QUERY_ATTN_NOALLOC_MAX_BYTES)
        EXPECT(relaxkv_query_attn_noalloc(&p, 0, fake, fake, fake, fake, fake, NULL, NULL) ==
                   RELAXKV_ENOSPACE, "noalloc too large");
    EXPECT(relaxkv_counts_to_host(NULL, ifake, NULL, NULL) == RELAXKV_EINVAL, "counts null");
}

/* The cache strides on tiny shapes, against two independent checks: the
 * header's nesting rule tried over every order of the three dimensions (brute
 * force instead of the library's sort), and, for every accepted layout, that no
 * two of the L * H_kv * T_c rows share an element. */
static void stress_strides(void) {
    const int64_t cand[] = {0, 64, 128, 192, 256, 320, 384, 448, 512, 768, 1024};
    const int nc = (int)(sizeof cand / sizeof cand[0]);
    const int d = 64;
    long accepted = 0, rejected = 0;
    for (int L = 1; L <= 3; ++L)
        for (int Hkv = 1; Hkv <= 3; ++Hkv)
            for (int T = 1; T <= 3; ++T)
                for (int a = 0; a < nc; ++a)
                    for (int b = 0; b < nc; ++b)
                        for (int c = 0; c < nc; ++c) {
                            relaxkv_problem p = make(L, T, 4, Hkv, Hkv, d, RELAXKV_DTYPE_BF16, 0.5);
                            p.kv_stride_layer = cand[a];
                            p.kv_stride_head = cand[b];
                            p.kv_stride_token = cand[c];
                            const int64_t sT = cand[c] ? cand[c] : d;
                            const int64_t sH = cand[b] ? cand[b] : (int64_t)T * sT;
                            const int64_t sL = cand[a] ? cand[a] : (int64_t)Hkv * sH;
                            const int64_t st[3] = {sL, sH, sT}, n[3] = {L, Hkv, T};
                            static const int perm[6][3] = {{0, 1, 2}, {0, 2, 1}, {1, 0, 2},
                                                           {1, 2, 0}, {2, 0, 1}, {2, 1, 0}};
                            int nests = 0;
                            for (int q = 0; q < 6 && !nests; ++q) {   /* perm[q][0] innermost */
                                int64_t ext = d;
                                int ok = 1;
                                for (int i = 0; i < 3; ++i) {
                                    const int k = perm[q][i];
                                    if (n[k] <= 1) continue;
                                    if (st[k] < ext) { ok = 0; break; }
                                    ext += (n[k] - 1) * st[k];
                                }
                                nests = ok;
                            }
                            const relaxkv_status v = relaxkv_validate(&p);
                            EXPECT(v == (nests ? RELAXKV_OK : RELAXKV_EINVAL),
                                   "strides %lld %lld %lld at L %d H_kv %d T %d: status %d",
                                   (long long)cand[a], (long long)cand[b], (long long)cand[c], L,
                                   Hkv, T, (int)v);
                            if (v != RELAXKV_OK) { ++rejected; continue; }
                            ++accepted;
                            int64_t starts[27];
                            int m = 0;
                            for (int l = 0; l < L; ++l)
                                for (int g = 0; g < Hkv; ++g)
                                    for (int i = 0; i < T; ++i) starts[m++] = l * sL + g * sH + i * sT;
                            for (int i = 0; i < m; ++i)
                                for (int j = i + 1; j < m; ++j) {
                                    const int64_t gap = starts[i] > starts[j] ? starts[i] - starts[j]
                                                                              : starts[j] - starts[i];
                                    EXPECT(gap >= d, "accepted strides %lld %lld %lld overlap",
                                           (long long)sL, (long long)sH, (long long)sT);
                                }
                        }
    EXPECT(accepted > 1000 && rejected > 1000, "stride sweep %ld / %ld", accepted, rejected);
    /* Strides near the int64 range: refused, with no overflow along the way (UBSan). */
    const int64_t huge[] = {(int64_t)1 << 47, (int64_t)1 << 48, (int64_t)1 << 62, INT64_MAX - 7,
                            INT64_MAX};
    for (int i = 0; i < 5; ++i)
        for (int which = 0; which < 3; ++which) {
            relaxkv_problem p = make(40, 32768, 64, 40, 8, 128, RELAXKV_DTYPE_BF16, 0.15);
            if (which == 0) p.kv_stride_layer = huge[i];
            if (which == 1) p.kv_stride_head = huge[i];
            if (which == 2) p.kv_stride_token = huge[i];
            const relaxkv_status v = relaxkv_validate(&p);
            EXPECT(v == RELAXKV_EUNSUPPORTED || v == RELAXKV_EINVAL, "huge stride %d/%d: %d", i,
                   which, (int)v);
        }
}

int main(void) {
    const int Ls[] = {1, 2, 40, 1024, 1025};
    const int Ts[] = {1, 2, 63, 64, 65, 1000, 32768, 1 << 20, (1 << 21) - 1, 1 << 21, 1 << 22,
                      (1 << 22) + 1};
    const int heads[][2] = {{1, 1}, {8, 2}, {40, 8}, {32, 8}, {14, 2}, {384, 1}, {385, 1},
                            {1024, 8}, {1024, 1024}, {6, 4}, {8, 0}};
    const int ds[] = {64, 96, 128, 256};
    const int dts[] = {RELAXKV_DTYPE_F32, RELAXKV_DTYPE_BF16, 7};
    const int Qns[] = {1, 64, 4096, 4097};
    const double rs[] = {0.0, 1e-9, 0.125, 0.15, 0.5, 1.0, 1.01, -0.01, NAN, INFINITY};
    long problems = 0;
    for (size_t a = 0; a < sizeof Ls / sizeof Ls[0]; ++a)
        for (size_t b = 0; b < sizeof Ts / sizeof Ts[0]; ++b)
            for (size_t c = 0; c < sizeof heads / sizeof heads[0]; ++c)
                for (size_t e = 0; e < sizeof ds / sizeof ds[0]; ++e)
                    for (size_t f = 0; f < sizeof dts / sizeof dts[0]; ++f) {
                        const int Qn = Qns[(a + b + c + e + f) % 4];
                        const double r = rs[(a * 7 + b * 3 + c + e + f) % 10];
                        relaxkv_problem p = make(Ls[a], Ts[b], Qn, heads[c][0], heads[c][1],
                                                 ds[e], dts[f], r);
                        stress_problem(&p);
                        ++problems;
                    }
    stress_strides();
    /* Pointer and descriptor checks. */
    EXPECT(relaxkv_validate(NULL) == RELAXKV_EINVAL, "validate NULL");
    relaxkv_problem p = make(2, 100, 4, 8, 2, 64, RELAXKV_DTYPE_BF16, 0.15);
    p.q = NULL;
    EXPECT(relaxkv_validate(&p) == RELAXKV_EINVAL, "null q");
    p = make(2, 100, 4, 8, 2, 64, RELAXKV_DTYPE_BF16, 0.15);
    p.softmax_scale = NAN;
    EXPECT(relaxkv_validate(&p) == RELAXKV_EINVAL, "NaN scale");
    for (int r = -8; r <= 1; ++r) EXPECT(relaxkv_status_string(r) != NULL, "status string");
    for (int T = 1; T <= 300; ++T)
        for (int i = 0; i <= 16; ++i) {
            const int32_t k = relaxkv_anchor_count(i / 16.0, T);
            EXPECT(k >= 1 && k <= T, "k(%d/16, %d) = %d", i, T, (int)k);
        }
    printf("ok %ld problems, %ld checks\n", problems, n_checks);
    return 0;
}
