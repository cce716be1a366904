// Query-side completion (the query prefill of the cache-ready TTFT protocol,
// App. C.4): the n_query query tokens of a layer, placed after the T_c context
// positions, attend to every cache position and causally to themselves.  The
// row log-sum-exp it emits is the normaliser relaxkv_score takes as q_lse.
//
// bf16 path, split over keys (the row set is small: n_query * G rows per KV
// head against T_c keys):
// - a workgroup owns one KV head g, one chunk of up to NB 32-row blocks of
//   (token, head) rows (token t, head g*G + hh -> row t*G + hh) and one split
//   of consecutive cache keys (sized on the host so that one round of
//   workgroups covers the layer); the last split also takes the query tokens'
//   own keys;
// - ten blocks run as twelve waves (two blocks in key halves whose partial
//   results are combined through LDS at the end), so the four SIMDs of a CU
//   (waves w and w+4 share one) carry equal work;
// - K and V tiles of 64 keys stream into a 4-deep ring of swizzled LDS buffers
//   by direct global->LDS loads (see tile_swz), three tiles ahead of the MFMAs;
// - each wave computes S^T = K Q^T for its 32 rows (one row per lane), a
//   flash-style online softmax in the exp2 domain with lazy rescaling, and
//   O^T += V^T P^T with transposing LDS reads of V;
// - every split writes its normalised partial output (bf16) and its row
//   log2-sum-exp; qattn_merge combines the splits with weights
//   exp2(lse_s - max) in a fixed order and writes O and the natural-log LSE.
// fp32 path: one wave per (token, head), VALU dot products over all keys.

#include <math.h>

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

constexpr int kQaKeys = 64;            // keys per tile
#ifndef RELAXKV_QA_STAGES
#define RELAXKV_QA_STAGES 4
#endif
#ifndef RELAXKV_QA_WGS
#define RELAXKV_QA_WGS 256                     // workgroups the key splits aim for (one per CU)
#endif
#ifndef QA_NH
#define QA_NH 2
#endif
constexpr int kQaStages = RELAXKV_QA_STAGES;   // LDS ring depth (a K and a V tile per stage)
constexpr int kQaMinSplit = 256;       // fewest cache keys per split
constexpr int kQaMaxSplit = 4096;      // most cache keys per split
constexpr int kQaRing = 4;             // K fragments read ahead of their MFMA
constexpr float kQaSlack = 8.0f;       // log2 units the running max may lag the true max

template <int N> struct Int { static constexpr int value = N; };

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

struct QaArgs {
    const uint16_t* q;       // this layer's query rows [Qn][H][D]
    const uint16_t* kc;      // this layer's cache: row i of KV head g at element g * kv_sh + i * kv_st
    const uint16_t* vc;
    const uint16_t* kq;      // the query tokens' keys/values [Qn][Hkv][D]
    const uint16_t* vq;
    uint16_t* part_o;        // [n_split][Hkv][rows_pad][D] bf16 normalised partial outputs
    float* part_l;           // [n_split][Hkv][rows_pad] log2-sum-exp of each partial
    int64_t kv_sh, kv_st;    // element strides of the cache's KV heads and tokens
    int T, Qn, H, Hkv, G, n_rows, rows_pad, n_split, kps;   // kps: cache keys per split
    float sl2;               // softmax scale * log2(e)
};

__device__ __forceinline__ float qa_pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float qa_pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D, int NB, int NH>
__global__ __launch_bounds__((NB + NH) * 64) void qattn_bf16(QaArgs a) {
    constexpr int NW = NB + NH;            // waves: NB - NH whole row blocks, 2 NH half blocks
    constexpr int TK = kQaKeys;
    constexpr int KS = D / 16;             // k-steps of QK^T
    constexpr int DB = D / 32;             // 32-wide d blocks of O^T
    constexpr int ROWB = 2 * D;            // tile row bytes
    constexpr int CH = D / 8;              // 16-byte chunks per row
    constexpr int RPI = 64 / CH;           // rows per wave-wide load
    constexpr int NL = TK / RPI;           // wave-wide loads per tile and tensor
    constexpr int NL2 = 2 * NL;            // K and V
    constexpr int LPW = NL2 / NW;          // loads per tile every wave issues (some one more)
    constexpr int NI = (NL2 + NW - 1) / NW;
    static_assert(LPW >= 1 && (kQaStages == 3 || kQaStages == 4), "loader shape");
    __shared__ __attribute__((aligned(1024))) uint16_t Kt[kQaStages][TK * D];
    __shared__ __attribute__((aligned(1024))) uint16_t Vt[kQaStages][TK * D];

    const int split = blockIdx.x, g = blockIdx.y, chunk = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, r32 = lane & 31, hf = lane >> 5;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    // Tiles: ntc over this split's cache keys, then (last split only) ntq over
    // the query tokens' own keys.
    const int key0 = split * a.kps;
    const int nkc = min(a.kps, a.T - key0);
    const int ntc = (nkc + TK - 1) / TK;
    const int ntq = split == a.n_split - 1 ? (a.Qn + TK - 1) / TK : 0;
    const int ntile = ntc + ntq;

    // The wave's row block: waves below NB - NH own a whole block; the other
    // 2 NH waves take the last NH blocks in halves (half 0: keys 0-31 of every
    // tile, half 1: keys 32-63), so the waves of the four SIMDs carry equal work.
    constexpr int NHD = NH > 0 ? NH : 1;   // (no half waves when NH = 0: halfw is never true)
    const int hw = w - (NB - NH);
    const bool halfw = hw >= 0;
    const int hsel = halfw ? hw / NHD : 0;                // the half this wave takes
    const int blk = halfw ? NB - NH + hw % NHD : w;
    // This lane's (token, head) row.  Within a tile, key index > lim is masked:
    // the cache tail of the split, or the causal future in the query tiles.
    const int rho = (chunk * NB + blk) * 32 + r32;
    const bool valid = rho < a.n_rows;
    const int t_row = valid ? rho / a.G : 0;
    const int hh = valid ? rho - t_row * a.G : 0;
    const int lim_q = valid ? t_row : a.Qn - 1;
    bf16x8 qf[KS];
    {
        const uint16_t* qrow = a.q + ((size_t)t_row * a.H + g * a.G + hh) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8*)(qrow + ks * 16 + hf * 8);
        // Consumed here, so the compiler's waits for these loads stay before the loop.
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(qf[ks]));
    }
    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    // Loader: load j < NL fills K rows, j >= NL V rows; lane l of a load writes
    // (row (j % NL)*RPI + l/CH, chunk l%CH) and fetches the chunk that belongs
    // there.  Rows past the tile's keys re-read its last key (masked).
    const int lrow = lane / CH, pchunk = lane % CH;
    auto issue_tile = [&](int tt) {
        // Lane indices made opaque per call, so that the addresses derived from
        // them are recomputed here instead of being kept live across the loop.
        int lr = lrow, pc = pchunk;
        asm volatile("" : "+v"(lr), "+v"(pc));
        const int st = tt % kQaStages;
        const bool qt = tt >= ntc;                      // a tile of the query tokens' keys
        const int k0 = qt ? (tt - ntc) * TK : tt * TK;
        const int kmax = qt ? a.Qn - 1 : nkc - 1;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int j = w + i * NW;
            if (i < LPW || j < NL2) {
                const bool isv = j >= NL;
                const int jj = isv ? j - NL : j;
                const int row = jj * RPI + lr;
                const int kk = min(k0 + row, kmax);
                const size_t e = qt ? ((size_t)kk * a.Hkv + g) * D
                                    : (size_t)(g * a.kv_sh + (key0 + kk) * a.kv_st);
                const uint16_t* base = qt ? (isv ? a.vq : a.kq) : (isv ? a.vc : a.kc);
                uint16_t* dst = (isv ? Vt[st] : Kt[st]) + jj * RPI * D;
                load_lds16(base + e + ((pc ^ tile_swz<D>(row)) << 3), dst);
            }
        }
    };
    // Full cache tiles (all but the split's tail tile and the query tiles): the
    // lane's source of load i is a loop-invariant base plus the tile offset.
    const uint16_t* cbase[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int j = w + i * NW;
        const bool isv = j >= NL;
        const int jj = isv ? j - NL : j;
        const int row = jj * RPI + lrow;
        cbase[i] = (isv ? a.vc : a.kc) + g * a.kv_sh + (key0 + row) * a.kv_st +
                   ((pchunk ^ tile_swz<D>(row)) << 3);
    }
    auto issue_full = [&](int tt) {
        const int st = tt % kQaStages;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int j = w + i * NW;
            if (i < LPW || j < NL2) {
                const bool isv = j >= NL;
                const int jj = isv ? j - NL : j;
                uint16_t* dst = (isv ? Vt[st] : Kt[st]) + jj * RPI * D;
                load_lds16(cbase[i] + tt * TK * a.kv_st, dst);
            }
        }
    };
    auto issue = [&](int tt) {
        if ((tt + 1) * TK <= nkc) issue_full(tt);
        else issue_tile(tt);
    };
    // rem = tiles issued after the one needed now: each wave issued at least
    // LPW loads per tile after it (in-order completion).
    auto wait_tile = [&](int rem) {
        if (kQaStages > 3 && rem >= 2) wait_loads_barrier<2 * LPW>();
        else if (rem >= 1) wait_loads_barrier<LPW>();
        else wait_loads_barrier<0>();
    };

    // Fragment byte offsets (see attn_bf16 for the transposing-read layout).
    const int k_base = r32 * ROWB | ((hf ^ tile_swz<D>(r32)) << 4);
    const int rl = 4 * (lane >> 5) + ((lane & 15) >> 2);
    const int cl = ((lane >> 4) & 1) * 2 + ((lane & 3) >> 1);
    const int v_base0 = rl * ROWB | ((cl ^ tile_swz<D>(rl)) << 4) | ((lane & 1) << 3);
    const int v_base1 = (rl + 8) * ROWB | ((cl ^ tile_swz<D>(rl + 8)) << 4) | ((lane & 1) << 3);

    // One tile for NKB 32-key blocks (2: the whole tile; 1: the wave's half,
    // whose rows start hoff bytes into the tile and whose keys start at c0).
    auto step = [&](auto nkb_t, const char* kst, uint32_t stage, uint32_t vstage, int c0, int lim,
                    bool masked, uint32_t hoff) {
        constexpr int NKB = decltype(nkb_t)::value;
        int kbo = k_base + (int)stage + (int)hoff;
        uint32_t vb0 = v_base0 + vstage + hoff, vb1 = v_base1 + vstage + hoff;
        asm volatile("" : "+v"(kbo), "+v"(vb0), "+v"(vb1));
        // S^T = K Q^T: s[kb][v] = S[row][key c0 + 32kb + 8(v/4) + 4hf + v%4]
        f32x16 s[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) s[kb] = f32x16{};
        auto frag = [&](int x) {                       // x = NKB ks + kb
            return *(const bf16x8*)(kst + (x % NKB) * 32 * ROWB + (kbo ^ ((x / NKB) << 5)));
        };
        bf16x8 kf[kQaRing];
#pragma unroll
        for (int i = 0; i < kQaRing; ++i) kf[i] = frag(i);
#pragma unroll
        for (int x = 0; x < NKB * KS; ++x) {
            const bf16x8 cur = kf[x % kQaRing];
            if (x + kQaRing < NKB * KS) kf[x % kQaRing] = frag(x + kQaRing);
            s[x % NKB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur, qf[x / NKB], s[x % NKB], 0, 0, 0);
        }
        if (masked) {                                  // cache tail or causal tile
            const int e = lim - c0 - 4 * hf;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (32 * kb + 8 * (v >> 2) + (v & 3) > e) s[kb][v] = -INFINITY;
        }
        // Chains of 3-input maxima (two new values per instruction).
        float mk[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            mk[kb] = fmaxf(s[kb][0], s[kb][1]);
#pragma unroll
            for (int v = 2; v < 16; v += 2) mk[kb] = fmaxf(fmaxf(mk[kb], s[kb][v]), s[kb][v + 1]);
        }
        const float mx = qa_pair_max(NKB == 2 ? fmaxf(mk[0], mk[NKB - 1]) : mk[0]) * a.sl2;
        if (__any(mx > m_run + kQaSlack)) {
            const float m_new = mx > m_run + kQaSlack ? mx : m_run;
            // (a row whose max stays -inf keeps its zero sum and output)
            const float alpha = m_new == m_run ? 1.f : fast_exp2(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
            m_run = m_new;
        }
        // The row sum adds the bf16 probabilities that the PV product uses, two
        // per dot2 instruction, in four chains.
        // A key-half wave can meet tiles whose keys are all masked before its
        // first visible key (the last split's cache tail when it holds at most
        // 32 keys, the causal query tiles): its running max is still -inf
        // there, and exp2 of -inf - (-inf) would be NaN.  Those tiles use a
        // reference of 0 instead, so they add exact zeros.
        const float m_ref = m_run == -INFINITY ? 0.f : m_run;
        bf16x8 pb[NKB][2];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                pb[kb][v >> 3][v & 7] = (__bf16)fast_exp2(fmaf(s[kb][v], a.sl2, -m_ref));
        {
            typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
            const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
            float ls0 = 0.f, ls1 = 0.f, ls2 = 0.f, ls3 = 0.f;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const bf16x8 q8 = pb[kb][k2];
                    ls0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(q8, q8, 0, 1), one2, ls0, false);
                    ls1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(q8, q8, 2, 3), one2, ls1, false);
                    ls2 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(q8, q8, 4, 5), one2, ls2, false);
                    ls3 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(q8, q8, 6, 7), one2, ls3, false);
                }
            l_run += (ls0 + ls1) + (ls2 + ls3);
        }
        // O^T += V^T P^T
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const uint32_t rowo = (kb * 32 + k2 * 16) * ROWB;
                    const v4i16 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_v4i16*)(uintptr_t)((vb0 ^ (db << 6)) + rowo));
                    const v4i16 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (lds_v4i16*)(uintptr_t)((vb1 ^ (db << 6)) + rowo));
                    const bf16x8 vv = __builtin_bit_cast(
                        bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
                    o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pb[kb][k2], o[db], 0, 0, 0);
                }
    };

#pragma unroll
    for (int tt = 0; tt < kQaStages - 1; ++tt)
        if (tt < ntile) issue(tt);
    // The tile loop, once per wave kind (so each is allocated on its own).
    auto run = [&](auto nkb_t) {
        constexpr int NKB = decltype(nkb_t)::value;
        for (int tt = 0; tt < ntile; ++tt) {
            wait_tile(min(kQaStages - 2, ntile - 1 - tt));
            if (tt + kQaStages - 1 < ntile) issue(tt + kQaStages - 1);
            const char* kst = (const char*)Kt[0];
            const uint32_t stage = (uint32_t)(tt % kQaStages) * (TK * D * 2);
            const uint32_t vstage = lds_addr(Vt[0]) + stage;
            const bool qt = tt >= ntc;
            const int c0 = qt ? (tt - ntc) * TK : tt * TK;
            const int lim = qt ? lim_q : nkc - 1;
            if (NKB == 1)
                step(nkb_t, kst, stage, vstage, c0 + 32 * hsel, lim, qt || c0 + TK > nkc,
                     (uint32_t)hsel * (32 * ROWB));
            else
                step(nkb_t, kst, stage, vstage, c0, lim, qt || c0 + TK > nkc, 0u);
        }
    };
    if (NH > 0 && halfw) run(Int<1>{});
    else run(Int<2>{});

    float l_tot = qa_pair_sum(l_run);
    if constexpr (NH > 0) {
        // The half-1 wave of each split block hands (O, m, l) to its half-0 wave
        // through LDS (the ring is free once every wave is past the last tile);
        // the half-0 wave combines them like two key splits.
        float* mo = (float*)&Kt[0][0];                     // [NH][DB * 16][64]
        float* ml = mo + NH * DB * 16 * 64;                // [NH][2][64]
        __syncthreads();
        const int pr = hw % NH;
        if (halfw && hsel == 1) {
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) mo[((pr * DB + db) * 16 + v) * 64 + lane] = o[db][v];
            ml[(pr * 2) * 64 + lane] = m_run;
            ml[(pr * 2 + 1) * 64 + lane] = l_tot;
        }
        __syncthreads();
        if (halfw && hsel == 1) return;
        if (halfw) {
            const float mB = ml[(pr * 2) * 64 + lane], lB = ml[(pr * 2 + 1) * 64 + lane];
            const float m = fmaxf(m_run, mB);
            const float wA = m_run == -INFINITY ? 0.f : fast_exp2(m_run - m);
            const float wB = mB == -INFINITY ? 0.f : fast_exp2(mB - m);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    o[db][v] = o[db][v] * wA + mo[((pr * DB + db) * 16 + v) * 64 + lane] * wB;
            l_tot = l_tot * wA + lB * wB;
            m_run = m;
        }
    }
    if (!valid) return;
    const float inv = 1.0f / l_tot;
    const size_t prow = ((size_t)split * a.Hkv + g) * a.rows_pad + rho;
    uint16_t* po = a.part_o + prow * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int d0 = db * 32 + 8 * j + 4 * hf;
            const uint32_t lo = (uint32_t)f32_to_bf16_bits(o[db][4 * j] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * j + 1] * inv) << 16);
            const uint32_t hi = (uint32_t)f32_to_bf16_bits(o[db][4 * j + 2] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * j + 3] * inv) << 16);
            *(u32x2*)(po + d0) = u32x2{lo, hi};
        }
    }
    if (hf == 0) a.part_l[prow] = m_run + __log2f(l_tot);
}

// One workgroup of D threads per (token, head): the splits' partial outputs
// combined with weights exp2(lse_s - max_s lse_s), in split order.  The split
// weights are staged in LDS; each thread then sums its d element with several
// partial loads in flight.
constexpr int kQaMergeSplits = 1024;   // splits per LDS pass
constexpr int kQaFixedSplits = 32;     // split count with its own merge kernel

template <int D>
__global__ __launch_bounds__(D) void qattn_merge(const uint16_t* __restrict__ part_o,
                                                 const float* __restrict__ part_l, int n_split,
                                                 int Hkv, int G, int H, int rows_pad,
                                                 uint16_t* __restrict__ out,
                                                 float* __restrict__ lse) {
    __shared__ float wl[kQaMergeSplits];
    __shared__ float red[D / 64];
    const int th = blockIdx.x;                      // t * H + h
    const int t = th / H, h = th - t * H;
    const int g = h / G, rho = t * G + (h - g * G);
    const int e = threadIdx.x;
    const size_t stride = (size_t)Hkv * rows_pad;   // between splits
    const size_t row0 = (size_t)g * rows_pad + rho;
    float M = -INFINITY;
    for (int s = e; s < n_split; s += D) M = fmaxf(M, part_l[s * stride + row0]);
    M = wave_max(M);
    if ((e & 63) == 0) red[e >> 6] = M;
    __syncthreads();
    M = red[0];
#pragma unroll
    for (int i = 1; i < D / 64; ++i) M = fmaxf(M, red[i]);
    float z = 0.f, acc = 0.f;
    for (int s0 = 0; s0 < n_split; s0 += kQaMergeSplits) {
        const int ns = min(kQaMergeSplits, n_split - s0);
        __syncthreads();
        for (int s = e; s < ns; s += D) wl[s] = fast_exp2(part_l[(s0 + s) * stride + row0] - M);
        __syncthreads();
        int s = 0;
        for (; s + 8 <= ns; s += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                v[u] = bf16_bits_to_f32(part_o[((s0 + s + u) * stride + row0) * D + e]);
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                z += wl[s + u];
                acc = fmaf(wl[s + u], v[u], acc);
            }
        }
        for (; s < ns; ++s) {
            z += wl[s];
            acc = fmaf(wl[s], bf16_bits_to_f32(part_o[((s0 + s) * stride + row0) * D + e]), acc);
        }
    }
    out[(size_t)th * D + e] = f32_to_bf16_bits(acc / z);
    if (lse && e == 0) lse[th] = (M + __log2f(z)) * kLn2;
}

// The same combination for exactly NS splits (the split count one round of
// workgroups gives at 8 KV heads): every split's partial element and its
// log-sum-exp are loaded before any of them is used, with no predication, so
// a thread waits for memory once instead of once per batch.  Same operations
// in the same order as qattn_merge, so the results are the same bits.
template <int D, int NS>
__global__ __launch_bounds__(D) void qattn_merge_fixed(const uint16_t* __restrict__ part_o,
                                                       const float* __restrict__ part_l,
                                                       int Hkv, int G, int H, int rows_pad,
                                                       uint16_t* __restrict__ out,
                                                       float* __restrict__ lse) {
    static_assert(NS <= 64, "one wave holds the splits' log-sum-exps");
    __shared__ float wl[NS];
    __shared__ float red[D / 64];
    const int th = blockIdx.x;                      // t * H + h
    const int t = th / H, h = th - t * H;
    const int g = h / G, rho = t * G + (h - g * G);
    const int e = threadIdx.x;
    const size_t stride = (size_t)Hkv * rows_pad;   // between splits
    const uint16_t* po = part_o + ((size_t)g * rows_pad + rho) * D + e;
    uint16_t raw[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) raw[s] = po[s * stride * D];
    const int el = e < NS ? e : NS - 1;
    const float ls = part_l[el * stride + (size_t)g * rows_pad + rho];
    float M = wave_max(e < NS ? ls : -INFINITY);
    if ((e & 63) == 0) red[e >> 6] = M;
    __syncthreads();
    M = red[0];
#pragma unroll
    for (int i = 1; i < D / 64; ++i) M = fmaxf(M, red[i]);
    if (e < NS) wl[e] = fast_exp2(ls - M);
    __syncthreads();
    float z = 0.f, acc = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        z += wl[s];
        acc = fmaf(wl[s], bf16_bits_to_f32(raw[s]), acc);
    }
    out[(size_t)th * D + e] = f32_to_bf16_bits(acc / z);
    if (lse && e == 0) lse[th] = (M + __log2f(z)) * kLn2;
}

// fp32: one wave per (token, head) over all T + t + 1 keys.
template <int D>
__global__ __launch_bounds__(64) void qattn_f32(const float* __restrict__ q,
                                                const float* __restrict__ kc,
                                                const float* __restrict__ vc,
                                                const float* __restrict__ kq,
                                                const float* __restrict__ vq, KvStrides ks,
                                                int T, int H, int Hkv, int G, float scale,
                                                float* __restrict__ out, float* __restrict__ lse) {
    constexpr int DPL = D / 64;
    __shared__ float qs[D];
    const int t = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    const int g = h / G;
    for (int e = lane; e < D; e += 64) qs[e] = q[((size_t)t * H + h) * D + e];
    __syncthreads();
    float o[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;
    const int nk = T + t + 1;
    for (int c0 = 0; c0 < nk; c0 += 64) {
        const int c = c0 + lane;
        float s = -INFINITY;
        const float* vrow = nullptr;
        if (c < nk) {
            const int64_t ce = g * ks.head + c * ks.token;          // cache row element offset
            const float* krow = c < T ? kc + ce : kq + ((size_t)(c - T) * Hkv + g) * D;
            vrow = c < T ? vc + ce : vq + ((size_t)(c - T) * Hkv + g) * D;
            float acc = 0.f;
            for (int e = 0; e < D; ++e) acc = fmaf(qs[e], krow[e], acc);
            s = acc * scale;
        }
        const float m_new = fmaxf(m_run, wave_max(s));
        const float alpha = expf(m_run - m_new);
        const float p = c < nk ? expf(s - m_new) : 0.f;
        l_run = l_run * alpha + wave_sum(p);
#pragma unroll
        for (int i = 0; i < DPL; ++i) o[i] *= alpha;
        const int cnt = min(64, nk - c0);
        for (int j = 0; j < cnt; ++j) {
            const float pj = __shfl(p, j, 64);
            const float* vj = (const float*)__shfl((long long)vrow, j, 64);
#pragma unroll
            for (int i = 0; i < DPL; ++i) o[i] = fmaf(pj, vj[lane + 64 * i], o[i]);
        }
        m_run = m_new;
    }
    float* orow = out + ((size_t)t * H + h) * D;
#pragma unroll
    for (int i = 0; i < DPL; ++i) orow[lane + 64 * i] = o[i] / l_run;
    if (lse && lane == 0) lse[(size_t)t * H + h] = m_run + logf(l_run);
}

int qa_waves(int rows_pad) {
    const int nrb = rows_pad / 32;
    return nrb <= 4 ? 4 : (nrb <= 8 || nrb > 10) ? 8 : 10;
}

template <int D, int NB, int NH>
void launch_qattn_bf16(const QaArgs& a, int n_chunks, hipStream_t st, void* out, float* lse) {
    hipLaunchKernelGGL((qattn_bf16<D, NB, NH>), dim3(a.n_split, a.Hkv, n_chunks),
                       dim3((NB + NH) * 64), 0, st, a);
    if (a.n_split == kQaFixedSplits)
        hipLaunchKernelGGL((qattn_merge_fixed<D, kQaFixedSplits>), dim3(a.Qn * a.H), dim3(D), 0, st,
                           (const uint16_t*)a.part_o, (const float*)a.part_l, a.Hkv, a.G, a.H,
                           a.rows_pad, (uint16_t*)out, lse);
    else
        hipLaunchKernelGGL((qattn_merge<D>), dim3(a.Qn * a.H), dim3(D), 0, st,
                           (const uint16_t*)a.part_o, (const float*)a.part_l, a.n_split, a.Hkv,
                           a.G, a.H, a.rows_pad, (uint16_t*)out, lse);
}

}  // namespace

QueryAttnWorkspace query_attn_workspace_layout(const relaxkv_problem& p) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    QueryAttnWorkspace w;
    const int G = p.H / p.H_kv;
    w.rows_pad = (p.n_query * G + 31) / 32 * 32;
    const int nw = qa_waves(w.rows_pad);
    w.n_chunks = (w.rows_pad + nw * 32 - 1) / (nw * 32);
    // One round of workgroups over the CUs: about 256 / (H_kv * chunks) splits,
    // each a multiple of the 64-key tile.
    const long groups = (long)p.H_kv * w.n_chunks;
    const long want = groups >= RELAXKV_QA_WGS ? 1 : RELAXKV_QA_WGS / groups;
    long kps = ((long)p.T_c + want - 1) / want;
    kps = (kps + kQaKeys - 1) / kQaKeys * kQaKeys;
    kps = kps < kQaMinSplit ? kQaMinSplit : kps > kQaMaxSplit ? kQaMaxSplit : kps;
    w.kps = (int)kps;
    w.n_split = (int)(((long)p.T_c + kps - 1) / kps);
    w.part_o_off = 0;
    w.part_l_off = 0;
    w.total = 0;
    if (p.dtype == RELAXKV_DTYPE_BF16) {
        const size_t rows = (size_t)w.n_split * p.H_kv * w.rows_pad;
        w.part_l_off = al(rows * p.d * 2);
        w.total = w.part_l_off + al(rows * 4);
    }
    return w;
}

hipError_t launch_query_attn(const relaxkv_problem& p, int layer, const void* k_cache,
                             const void* v_cache, const void* k_q, const void* v_q, void* out,
                             float* lse_out, char* ws, hipStream_t st) {
    const int G = p.H / p.H_kv;
    const float scale = p.softmax_scale > 0.f ? p.softmax_scale : 1.0f / sqrtf((float)p.d);
    const KvStrides ks = kv_strides(p);
    const size_t cache_layer = (size_t)(layer * ks.layer);     // this layer's first element
    const size_t q_layer = (size_t)p.n_query * p.H * p.d;
    if (p.dtype == RELAXKV_DTYPE_F32) {
        const float* q = (const float*)p.q + (size_t)layer * q_layer;
        const float* kc = (const float*)k_cache + cache_layer;
        const float* vc = (const float*)v_cache + cache_layer;
        if (p.d == 128)
            hipLaunchKernelGGL(qattn_f32<128>, dim3(p.n_query, p.H), dim3(64), 0, st, q, kc, vc,
                               (const float*)k_q, (const float*)v_q, ks, p.T_c, p.H, p.H_kv, G, scale,
                               (float*)out, lse_out);
        else
            hipLaunchKernelGGL(qattn_f32<64>, dim3(p.n_query, p.H), dim3(64), 0, st, q, kc, vc,
                               (const float*)k_q, (const float*)v_q, ks, p.T_c, p.H, p.H_kv, G, scale,
                               (float*)out, lse_out);
        return hipGetLastError();
    }
    const QueryAttnWorkspace w = query_attn_workspace_layout(p);
    QaArgs a;
    a.q = (const uint16_t*)p.q + (size_t)layer * q_layer;
    a.kc = (const uint16_t*)k_cache + cache_layer;
    a.vc = (const uint16_t*)v_cache + cache_layer;
    a.kv_sh = ks.head;
    a.kv_st = ks.token;
    a.kq = (const uint16_t*)k_q;
    a.vq = (const uint16_t*)v_q;
    a.part_o = (uint16_t*)(ws + w.part_o_off);
    a.part_l = (float*)(ws + w.part_l_off);
    a.T = p.T_c;
    a.Qn = p.n_query;
    a.H = p.H;
    a.Hkv = p.H_kv;
    a.G = G;
    a.n_rows = p.n_query * G;
    a.rows_pad = w.rows_pad;
    a.n_split = w.n_split;
    a.kps = w.kps;
    a.sl2 = scale * kLog2e;
    const int nw = qa_waves(w.rows_pad);
    const int n_chunks = w.n_chunks;
    // Ten row blocks run as 12 waves (two blocks in key halves), so that each of the
    // four SIMDs carries two and a half blocks.
    if (p.d == 128) {
        if (nw == 4) launch_qattn_bf16<128, 4, 0>(a, n_chunks, st, out, lse_out);
        else if (nw == 8) launch_qattn_bf16<128, 8, 0>(a, n_chunks, st, out, lse_out);
        else launch_qattn_bf16<128, 10, QA_NH>(a, n_chunks, st, out, lse_out);
    } else {
        if (nw == 4) launch_qattn_bf16<64, 4, 0>(a, n_chunks, st, out, lse_out);
        else if (nw == 8) launch_qattn_bf16<64, 8, 0>(a, n_chunks, st, out, lse_out);
        else launch_qattn_bf16<64, 10, QA_NH>(a, n_chunks, st, out, lse_out);
    }
    return hipGetLastError();
}

}  // namespace relaxkv
