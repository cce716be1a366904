// Layer-wise query-attention score (Sec. 3.2 equation; first step of Algorithm 1):
//   A_l[h,t,i] = softmax_i(sigma <q_{l,t,h}, k_{l,g(h),i}>),
//   p_{l,i} = (1/(H Qn)) sum_{h,t} A_l[h,t,i],   a_{l,i} = MinMax_i(p_{l,i}).
//
// bf16 path (bf16 MFMA, fp32 accumulation), per layer l and KV head g the
// Qn*G query rows that share g form one row set; each workgroup takes a split
// of 2048 contiguous keys, each wave holds one 32-row block of the row set's
// queries in registers, and 16 KB tiles of K stream through a 4-deep ring of
// LDS buffers filled by direct global->LDS loads (two workgroups per CU):
//   1. score_pass<STATS> -- S^T = K Q^T (one query row per lane) and each
//      row's (max, sum of exp2) over the split.          [skipped with q_lse]
//   2. score_merge  -- per row, merge the splits into a log2-sum-exp.
//   3. score_pass<colsum> -- the same tiles as S = Q K^T (one key per lane):
//      every lane sums exp2(s - lse) over its rows, the waves' partial sums are
//      added in a fixed order, giving the pooled mass of each key for this KV
//      head.  K is read once more (from the last-level cache when the layer's
//      K fits there).
//   4. score_pool / score_minmax -- the fixed-order sum over KV heads and the
//      1/(H Qn) factor with per-block extrema, then the MinMax normalisation.
// float32 path: plain VALU kernels with the same four steps (used for fp32
// inputs, where bf16 MFMA would not meet fp32 accuracy).
// Every reduction has a fixed order and no float atomics: results are
// bit-identical run to run.

#include <math.h>

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

constexpr int kTileBytes = 16384;             // bytes of K per LDS tile (64 keys at d = 128)
constexpr int kKeysPerSplit = 2048;           // keys per workgroup
constexpr int kMaxWaves = 10;                 // row blocks per workgroup (one per wave)
constexpr int kStages = 4;                    // LDS ring of K tiles
constexpr int kRing = 4;                      // K fragments read ahead of their MFMA

template <int D>
constexpr int tile_keys() { return kTileBytes / (2 * D); }

// Two workgroups share a CU (LDS ~70 KB each), so the waves of one overlap the
// barrier waits and vector phases of the other, and 2 x 10 waves spread evenly
// over the 4 SIMDs.
template <int NW>
constexpr int score_waves_per_simd() { return (2 * NW + 3) / 4; }

__host__ __device__ inline int round_up32(int x) { return (x + 31) / 32 * 32; }

// The copy of a value held by the lane 32 away.  v_permlane32_swap with both
// operands x returns, in each lane, x and its partner's x in its two results;
// xor-ing both results with x leaves the partner's bits whichever result holds
// which.
__device__ __forceinline__ float pair_other(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(r[0] ^ r[1] ^ u);
}

// One pass over the keys of a 2048-key split for the row set (l, g).  NW waves
// each hold one 32-row block of the row set's queries in registers (row rho =
// t*G + hh reads q[l][t][g*G + hh][:]); 16 KB tiles of K stream into a ring of
// kStages swizzled LDS buffers by direct global->LDS loads, kStages-1 tiles
// ahead of the MFMAs.
//   STATS: S^T = K Q^T (one query row per lane): per-lane online (max, sum of
//          exp2) over its keys, merged with the lane 32 away at the end ->
//          stats[l][g][split][row] in log2 units.
//   else:  S = Q K^T (one key per lane): per-lane sum of exp2(s - lse) over its
//          16 rows, the two half-waves added, then a fixed-order sum over the
//          waves in LDS -> part[l][g][key].
template <int D, int NW, bool STATS>
__global__ __launch_bounds__(NW * 64, score_waves_per_simd<NW>()) void score_pass_bf16(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, int T, int Qn, int H,
    int Hkv, int G, int n_rows, int rows_pad, int n_split, float sl2,
    float2* __restrict__ stats, const float* __restrict__ lse2, const float* __restrict__ q_lse,
    float* __restrict__ part) {
    constexpr int TK = tile_keys<D>();              // keys per tile
    constexpr int NT = kKeysPerSplit / TK;          // tiles per split
    constexpr int KS = D / 16;
    constexpr int NB = TK / 32;                     // 32-key MFMA blocks per tile
    constexpr int ROWB = 2 * D;                     // tile row bytes
    constexpr int CH = D / 8;                       // 16-byte chunks per row
    constexpr int RPI = 64 / CH;                    // rows per wave-wide load
    constexpr int NL = TK / RPI;                    // wave-wide loads per tile (16)
    constexpr int LPW = NL / NW;                    // loads per tile every wave issues (some one more)
    constexpr int NI = (NL + NW - 1) / NW;
    static_assert(LPW >= 1 && kStages == 4 && TK % 64 == 0, "pipeline shape");
    __shared__ __attribute__((aligned(1024))) uint16_t Ks[kStages][TK * D];
    __shared__ float colp[2][STATS ? 1 : NW][TK];
    __shared__ __attribute__((aligned(16))) float lrs[STATS ? 1 : NW][32];

    const int split = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, r32 = lane & 31, hf = lane >> 5;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint16_t* Kg = kc + ((size_t)l * Hkv + g) * (size_t)T * D;
    const int key0 = split * kKeysPerSplit;
    const int ntile = min(NT, (T - key0 + TK - 1) / TK);

    // Tile tt into stage tt % kStages.  Wave w issues loads j = w, w+NW, ...;
    // lane l of load j fills (row j*RPI + l/CH, chunk l%CH).  Rows past T re-read
    // row T-1: their logits are masked (STATS) or their sums never stored.
    const int lrow = lane / CH, pchunk = lane % CH;
    uint32_t loff[NI];                              // byte offset of this lane's chunk in a tile
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int row = (w + i * NW) * RPI + lrow;
        loff[i] = (uint32_t)(row * ROWB + ((pchunk ^ tile_swz<D>(row)) << 4));
    }
    auto issue_tile = [&](int tt) {
        uint16_t* st = Ks[tt % kStages];
        const int kb = key0 + tt * TK;
        const char* tb = (const char*)(Kg + (size_t)kb * D);
        const bool tail = kb + TK > T;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int j = w + i * NW;
            if (i < LPW || j < NL) {
                uint32_t o = loff[i];
                if (tail) {                                  // clamp the row to T-1
                    const int row = j * RPI + lrow;
                    o = (uint32_t)((min(kb + row, T - 1) - kb) * ROWB) + (o & (ROWB - 1));
                }
                load_lds16(tb + o, st + j * RPI * D);
            }
        }
    };
    // Wait for tile tt (rem tiles were issued after it), then barrier.
    auto wait_tile = [&](int rem) {
        if (rem >= 2) wait_loads_barrier<2 * LPW>();
        else if (rem == 1) wait_loads_barrier<LPW>();
        else wait_loads_barrier<0>();
    };
    auto reduce_cols = [&](int tt, bool first_chunk) {   // colsum: fixed-order sum over waves
        const int key = key0 + tt * TK + tid;
        if (tid < TK && key < T) {
            float v = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) v += colp[tt & 1][STATS ? 0 : ww][tid];
            float* dst = part + ((size_t)l * Hkv + g) * T + key;
            *dst = first_chunk ? v : *dst + v;
        }
    };
    // K fragment (tile row 32b + r32, logical chunk 2ks + hf) byte offset.
    const int k_base = r32 * ROWB | ((hf ^ tile_swz<D>(r32)) << 4);

    for (int rc0 = 0; rc0 < rows_pad; rc0 += NW * 32) {
        const int rho = rc0 + w * 32 + r32;
        bf16x8 qf[KS];
        if (rho < n_rows) {
            const int t = rho / G, hh = rho % G;
            const uint16_t* qrow = q + (((size_t)l * Qn + t) * H + g * G + hh) * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8*)(qrow + ks * 16 + hf * 8);
        } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) qf[ks] = bf16x8{};
        }
        // Colsum: log2-sum-exp of the wave's 32 rows, kept in LDS (padding rows
        // get +inf); the lane that accumulates rows 8j + 4hf + i reads
        // lrs[w][8j + 4hf .. +3] as one 16-byte broadcast.
        if constexpr (!STATS) {
            if (lane < 32) {
                const int row = rc0 + w * 32 + lane;
                float x = INFINITY;
                if (row < n_rows) {
                    x = q_lse ? q_lse[((size_t)l * Qn + row / G) * H + g * G + row % G] * kLog2e
                              : lse2[((size_t)l * Hkv + g) * rows_pad + row];
                }
                lrs[w][lane] = x;
            }
        }
        float m_run = -INFINITY, z_run = 0.f;

        __syncthreads();                                // LDS free from the previous row chunk
#pragma unroll
        for (int tt = 0; tt < kStages - 1; ++tt)
            if (tt < ntile) issue_tile(tt);
        for (int tt = 0; tt < ntile; ++tt) {
            wait_tile(min(kStages - 2, ntile - 1 - tt));
            if (!STATS && tt > 0) reduce_cols(tt - 1, rc0 == 0);
            if (tt + kStages - 1 < ntile) issue_tile(tt + kStages - 1);
            const char* kt = (const char*)Ks[tt % kStages];
            const int kbase = key0 + tt * TK;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                // 32-key block: KS MFMAs, K fragments read kRing ahead.
                const char* kp = kt + b * 32 * ROWB;
                bf16x8 kf[kRing];
#pragma unroll
                for (int i = 0; i < kRing; ++i) kf[i] = *(const bf16x8*)(kp + (k_base ^ (i << 5)));
                f32x16 acc = f32x16{};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 cur = kf[ks % kRing];
                    if (ks + kRing < KS) kf[ks % kRing] = *(const bf16x8*)(kp + (k_base ^ ((ks + kRing) << 5)));
                    if constexpr (STATS)
                        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur, qf[ks], acc, 0, 0, 0);
                    else
                        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ks], cur, acc, 0, 0, 0);
                }
                const int kb0 = kbase + 32 * b;
                if constexpr (STATS) {
                    // acc[v] = S[row r32][key kb0 + 8(v/4) + 4hf + v%4]
                    if (kb0 + 32 > T) {
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            if (kb0 + 8 * (v >> 2) + 4 * hf + (v & 3) >= T) acc[v] = -INFINITY;
                    }
                    float mt = acc[0];
#pragma unroll
                    for (int v = 1; v < 16; ++v) mt = fmaxf(mt, acc[v]);
                    const float m_new = fmaxf(m_run, mt * sl2);
                    const float mref = m_new == -INFINITY ? 0.f : m_new;
                    float z = z_run * fast_exp2(m_run - mref);
#pragma unroll
                    for (int v = 0; v < 16; ++v) z += fast_exp2(fmaf(acc[v], sl2, -mref));
                    z_run = z;
                    m_run = m_new;
                } else {
                    // acc[v] = S[row rc0 + w*32 + 8(v/4) + 4hf + v%4][key kb0 + r32]
                    float cs = 0.f;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const f32x4 lr = *(const f32x4*)&lrs[w][8 * j + 4 * hf];
#pragma unroll
                        for (int i = 0; i < 4; ++i) cs += fast_exp2(fmaf(acc[4 * j + i], sl2, -lr[i]));
                    }
                    const float other = pair_other(cs);
                    if (hf == 0) colp[tt & 1][w][32 * b + r32] = cs + other;
                }
            }
        }
        if constexpr (STATS) {
            // merge with the lane 32 away (same row, the other half of the keys)
            const float m2 = pair_other(m_run), z2 = pair_other(z_run);
            const float M = fmaxf(m_run, m2);
            float Z = 0.f;
            if (M != -INFINITY)
                Z = (m_run == -INFINITY ? 0.f : z_run * fast_exp2(m_run - M)) +
                    (m2 == -INFINITY ? 0.f : z2 * fast_exp2(m2 - M));
            if (hf == 0 && rho < rows_pad)
                stats[(((size_t)l * Hkv + g) * n_split + split) * rows_pad + rho] = make_float2(M, Z);
        } else {
            __syncthreads();
            reduce_cols(ntile - 1, rc0 == 0);
        }
    }
}

__global__ void score_merge(const float2* __restrict__ stats, int n_groups, int n_split,
                            int rows_pad, int n_rows, float* __restrict__ lse2) {
    const long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
    if (i >= (long)n_groups * rows_pad) return;
    const long lg = i / rows_pad;
    const int row = (int)(i % rows_pad);
    if (row >= n_rows) {
        lse2[i] = INFINITY;     // padding rows contribute exp2(-inf) = 0
        return;
    }
    const float2* s = stats + lg * n_split * rows_pad + row;
    float M = -INFINITY;
    for (int j = 0; j < n_split; ++j) M = fmaxf(M, s[(size_t)j * rows_pad].x);
    float Z = 0.f;
    for (int j = 0; j < n_split; ++j) {
        const float2 v = s[(size_t)j * rows_pad];
        if (v.x != -INFINITY) Z += v.y * fast_exp2(v.x - M);
    }
    lse2[i] = M + __log2f(Z);
}

// ---------------------------------------------------------------- float32 path

template <int D>
__global__ __launch_bounds__(256) void score_stats_f32(const float* __restrict__ q,
                                                       const float* __restrict__ kc, int T,
                                                       int Qn, int H, int Hkv, int G,
                                                       int rows_pad, float scale,
                                                       float* __restrict__ lse_nat) {
    __shared__ float qs[D];
    __shared__ float red_m[4], red_z[4];
    const int th = blockIdx.x;                 // t * H + h
    const int l = blockIdx.y;
    const int t = th / H, h = th % H, g = h / G;
    const int tid = threadIdx.x;
    for (int e = tid; e < D; e += 256) qs[e] = q[((size_t)l * Qn + t) * H * D + (size_t)h * D + e];
    __syncthreads();
    const float* Kg = kc + ((size_t)l * Hkv + g) * (size_t)T * D;
    float m = -INFINITY, z = 0.f;
    for (int i = tid; i < T; i += 256) {
        const float* kr = Kg + (size_t)i * D;
        float s = 0.f;
        for (int e = 0; e < D; ++e) s = fmaf(qs[e], kr[e], s);
        s *= scale;
        if (s > m) {
            z = z * expf(m - s) + 1.f;
            m = s;
        } else {
            z += expf(s - m);
        }
    }
    // combine (m, z) over the block
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o, 64), z2 = __shfl_xor(z, o, 64);
        const float M = fmaxf(m, m2);
        z = (m == -INFINITY ? 0.f : z * expf(m - M)) + (m2 == -INFINITY ? 0.f : z2 * expf(m2 - M));
        m = M;
    }
    if ((tid & 63) == 0) {
        red_m[tid >> 6] = m;
        red_z[tid >> 6] = z;
    }
    __syncthreads();
    if (tid == 0) {
        float M = -INFINITY;
        for (int i = 0; i < 4; ++i) M = fmaxf(M, red_m[i]);
        float Z = 0.f;
        for (int i = 0; i < 4; ++i)
            if (red_m[i] != -INFINITY) Z += red_z[i] * expf(red_m[i] - M);
        lse_nat[((size_t)l * Hkv + g) * rows_pad + t * G + (h % G)] = M + logf(Z);
    }
}

template <int D>
__global__ __launch_bounds__(256) void score_colsum_f32(const float* __restrict__ q,
                                                        const float* __restrict__ kc, int T,
                                                        int Qn, int H, int Hkv, int G,
                                                        int rows_pad, float scale,
                                                        const float* __restrict__ lse_nat,
                                                        const float* __restrict__ q_lse,
                                                        float* __restrict__ part) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int l = blockIdx.y;
    if (i >= T) return;
    float acc = 0.f;
    for (int g = 0; g < Hkv; ++g) {
        float kr[D];
        const float* kp = kc + (((size_t)l * Hkv + g) * T + i) * D;
#pragma unroll
        for (int e = 0; e < D; ++e) kr[e] = kp[e];
        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh;
            for (int t = 0; t < Qn; ++t) {
                const float* qr = q + (((size_t)l * Qn + t) * H + h) * D;
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < D; ++e) s = fmaf(qr[e], kr[e], s);
                const float lse = q_lse ? q_lse[((size_t)l * Qn + t) * H + h]
                                        : lse_nat[((size_t)l * Hkv + g) * rows_pad + t * G + hh];
                acc += expf(s * scale - lse);
            }
        }
    }
    part[(size_t)l * T + i] = acc;
}

// ---------------------------------------------------------------- finaliser

// Finaliser, two launches over (key block, layer):
//   score_pool: p_i = (1/(H Qn)) * sum over the n_part partial slices (fixed
//     order), written to scores, plus each block's (min, max) of p;
//   score_minmax: every block reduces its layer's block extrema (fixed order)
//     and rescales its keys to a = (p - min) / (max - min), or 0 when flat.
constexpr int kFinKeys = 1024;                 // keys per finaliser block (256 threads x 4)

__global__ __launch_bounds__(256) void score_pool(const float* __restrict__ part, int n_part,
                                                  int T, float inv_hq, float* __restrict__ scores,
                                                  float2* __restrict__ mm, int n_blk) {
    __shared__ float red_lo[4], red_hi[4];
    const int blk = blockIdx.x, l = blockIdx.y, tid = threadIdx.x;
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = blk * kFinKeys + e * 256 + tid;
        if (i < T) {
            float p = 0.f;
            for (int j = 0; j < n_part; ++j) p += part[((size_t)l * n_part + j) * T + i];
            p *= inv_hq;
            scores[(size_t)l * T + i] = p;
            lo = fminf(lo, p);
            hi = fmaxf(hi, p);
        }
    }
    lo = -wave_max(-lo);
    hi = wave_max(hi);
    if ((tid & 63) == 0) {
        red_lo[tid >> 6] = lo;
        red_hi[tid >> 6] = hi;
    }
    __syncthreads();
    if (tid == 0) {
        float a = red_lo[0], b = red_hi[0];
        for (int i = 1; i < 4; ++i) {
            a = fminf(a, red_lo[i]);
            b = fmaxf(b, red_hi[i]);
        }
        mm[(size_t)l * n_blk + blk] = make_float2(a, b);
    }
}

__global__ __launch_bounds__(256) void score_minmax(const float2* __restrict__ mm, int n_blk, int T,
                                                    float* __restrict__ scores) {
    __shared__ float red_lo[4], red_hi[4];
    const int blk = blockIdx.x, l = blockIdx.y, tid = threadIdx.x;
    float lo = INFINITY, hi = -INFINITY;
    for (int b = tid; b < n_blk; b += 256) {
        const float2 v = mm[(size_t)l * n_blk + b];
        lo = fminf(lo, v.x);
        hi = fmaxf(hi, v.y);
    }
    lo = -wave_max(-lo);
    hi = wave_max(hi);
    if ((tid & 63) == 0) {
        red_lo[tid >> 6] = lo;
        red_hi[tid >> 6] = hi;
    }
    __syncthreads();
    lo = fminf(fminf(red_lo[0], red_lo[1]), fminf(red_lo[2], red_lo[3]));
    hi = fmaxf(fmaxf(red_hi[0], red_hi[1]), fmaxf(red_hi[2], red_hi[3]));
    const bool flat = !(hi > lo);
    const float span = hi - lo;
    float* a = scores + (size_t)l * T;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = blk * kFinKeys + e * 256 + tid;
        if (i < T) a[i] = flat ? 0.f : (a[i] - lo) / span;
    }
}

void launch_finalize(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws, float* scores,
                     hipStream_t st) {
    const dim3 grid(w.n_blk, p.L);
    float2* mm = (float2*)(ws + w.mm_off);
    hipLaunchKernelGGL(score_pool, grid, dim3(256), 0, st, (const float*)(ws + w.part_off), w.n_part,
                       p.T_c, 1.0f / ((float)p.H * (float)p.n_query), scores, mm, w.n_blk);
    hipLaunchKernelGGL(score_minmax, grid, dim3(256), 0, st, (const float2*)mm, w.n_blk, p.T_c, scores);
}

template <int D, int NW>
void launch_passes_bf16(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                        hipStream_t st, float sl2) {
    const int G = p.H / p.H_kv;
    const int n_rows = p.n_query * G;
    const uint16_t* q = (const uint16_t*)p.q;
    const uint16_t* kc = (const uint16_t*)p.k_cache;
    float* part = (float*)(ws + w.part_off);
    float* lse2 = (float*)(ws + w.lse_off);
    float2* stats = (float2*)(ws + w.stats_off);
    const dim3 grid(w.n_split, p.H_kv, p.L);
    if (!p.q_lse) {
        hipLaunchKernelGGL((score_pass_bf16<D, NW, true>), grid, dim3(NW * 64), 0, st, q, kc,
                           p.T_c, p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, w.n_split, sl2,
                           stats, (const float*)nullptr, (const float*)nullptr, part);
        const long n = (long)p.L * p.H_kv * w.rows_pad;
        hipLaunchKernelGGL(score_merge, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                           (const float2*)stats, p.L * p.H_kv, w.n_split, w.rows_pad, n_rows, lse2);
    }
    hipLaunchKernelGGL((score_pass_bf16<D, NW, false>), grid, dim3(NW * 64), 0, st, q, kc, p.T_c,
                       p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, w.n_split, sl2, stats,
                       (const float*)lse2, p.q_lse, part);
}

template <int D>
hipError_t launch_score_bf16(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                             float* scores, hipStream_t st, float scale) {
    const float sl2 = scale * kLog2e;
    // One wave per 32-row block of the row set, up to kMaxWaves; larger row sets
    // loop over row chunks of 8 blocks.
    const int nrb = w.rows_pad / 32;
    if (nrb <= 4) launch_passes_bf16<D, 4>(p, w, ws, st, sl2);
    else if (nrb <= 8 || nrb > kMaxWaves) launch_passes_bf16<D, 8>(p, w, ws, st, sl2);
    else launch_passes_bf16<D, kMaxWaves>(p, w, ws, st, sl2);
    launch_finalize(p, w, ws, scores, st);
    return hipGetLastError();
}

template <int D>
hipError_t launch_score_f32(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                            float* scores, hipStream_t st, float scale) {
    const int G = p.H / p.H_kv;
    const float* q = (const float*)p.q;
    const float* kc = (const float*)p.k_cache;
    float* part = (float*)(ws + w.part_off);
    float* lse = (float*)(ws + w.lse_off);
    if (!p.q_lse)
        hipLaunchKernelGGL(score_stats_f32<D>, dim3(p.n_query * p.H, p.L), dim3(256), 0, st, q, kc,
                           p.T_c, p.n_query, p.H, p.H_kv, G, w.rows_pad, scale, lse);
    hipLaunchKernelGGL(score_colsum_f32<D>, dim3((p.T_c + 255) / 256, p.L), dim3(256), 0, st, q,
                       kc, p.T_c, p.n_query, p.H, p.H_kv, G, w.rows_pad, scale, lse, p.q_lse,
                       part);
    launch_finalize(p, w, ws, scores, st);
    return hipGetLastError();
}

}  // namespace

ScoreWorkspace score_workspace_layout(const relaxkv_problem& p) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    ScoreWorkspace w;
    const int G = p.H / p.H_kv;
    const bool bf = p.dtype == RELAXKV_DTYPE_BF16;
    w.rows_pad = round_up32(p.n_query * G);
    w.n_split = (p.T_c + kKeysPerSplit - 1) / kKeysPerSplit;
    w.n_part = bf ? p.H_kv : 1;
    w.part_off = 0;
    size_t off = al((size_t)p.L * w.n_part * p.T_c * sizeof(float));
    w.stats_off = off;
    if (bf) off += al((size_t)p.L * p.H_kv * w.n_split * w.rows_pad * sizeof(float2));
    w.lse_off = off;
    off += al((size_t)p.L * p.H_kv * w.rows_pad * sizeof(float));
    w.n_blk = (p.T_c + kFinKeys - 1) / kFinKeys;
    w.mm_off = off;
    off += al((size_t)p.L * w.n_blk * sizeof(float2));
    w.total = off;
    return w;
}

hipError_t launch_score(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                        float* scores, hipStream_t st) {
    const float scale = p.softmax_scale > 0.f ? p.softmax_scale : 1.0f / sqrtf((float)p.d);
    if (p.dtype == RELAXKV_DTYPE_BF16) {
        return p.d == 128 ? launch_score_bf16<128>(p, w, ws, scores, st, scale)
                          : launch_score_bf16<64>(p, w, ws, scores, st, scale);
    }
    return p.d == 128 ? launch_score_f32<128>(p, w, ws, scores, st, scale)
                      : launch_score_f32<64>(p, w, ws, scores, st, scale);
}

}  // namespace relaxkv
