// Layer-wise query-attention score (Sec. 3.2 equation; first step of Algorithm 1):
//   A_l[h,t,i] = softmax_i(sigma <q_{l,t,h}, k_{l,g(h),i}>),
//   p_{l,i} = (1/(H Qn)) sum_{h,t} A_l[h,t,i],   a_{l,i} = MinMax_i(p_{l,i}).
//
// bf16 path (bf16 MFMA, fp32 accumulation), per layer l and KV head g the
// Qn*G query rows that share g form one row set:
//   1. score_stats  -- key splits of 512 keys; each of 8 waves keeps 64 keys
//      of K in registers and streams the row set's Q through LDS, computing
//      S^T = K Q^T (one query row per lane) and each row's (max, sum of exp2)
//      over its keys.                                    [skipped with q_lse]
//   2. score_merge  -- per row, merge the splits into a log2-sum-exp.
//   3. score_colsum -- the same tiles as S = Q K^T (one key per lane): every
//      lane sums exp2(s - lse) over its rows, giving the pooled mass of its key
//      for this KV head.  K is read once more (from the last-level cache when
//      the layer's K fits there).
//   4. score_finalize -- per layer, the fixed-order sum over KV heads, the
//      1/(H Qn) factor and the MinMax normalisation.
// float32 path: plain VALU kernels with the same four steps (used for fp32
// inputs, where bf16 MFMA would not meet fp32 accuracy).
// Every reduction has a fixed order and no float atomics: results are
// bit-identical run to run.

#include <math.h>

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

constexpr int kScoreWaves = 8;
constexpr int kScoreThreads = kScoreWaves * 64;
constexpr int kKeysPerWave = 64;
constexpr int kKeysPerSplit = kScoreWaves * kKeysPerWave;   // 512
constexpr int kRowChunk = 384;                              // query rows staged in LDS at once

__host__ __device__ inline int round_up32(int x) { return (x + 31) / 32 * 32; }

template <int D>
__device__ __forceinline__ void load_k_frags(const uint16_t* __restrict__ Kg, int c0, int T,
                                             int r32, int hf, bf16x8 (&kf)[2][D / 16]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int key = c0 + kb * 32 + r32;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
            if (key < T)
                kf[kb][ks] = *(const bf16x8*)(Kg + (size_t)key * D + ks * 16 + hf * 8);
            else
                kf[kb][ks] = bf16x8{};
        }
    }
}

// Stage rows rc0 .. rc0+nrows-1 of the row set (row rho = t*G + hh reads
// q[l][t][g*G + hh][:]) into LDS with a padded stride; rows >= n_rows are zero.
template <int D>
__device__ __forceinline__ void stage_q(const uint16_t* __restrict__ q, uint16_t* Qs, int l,
                                        int g, int rc0, int nrows, int n_rows, int Qn, int H,
                                        int G) {
    constexpr int QSTR = D + 8;
    constexpr int P = D / 8;
    for (int idx = threadIdx.x; idx < nrows * P; idx += blockDim.x) {
        const int rr = idx / P, part = idx % P;
        const int rho = rc0 + rr;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (rho < n_rows) {
            const int t = rho / G, hh = rho % G;
            v = *(const u32x4*)(q + (((size_t)l * Qn + t) * H + g * G + hh) * D + part * 8);
        }
        *(u32x4*)(Qs + rr * QSTR + part * 8) = v;
    }
}

template <int D>
__global__ __launch_bounds__(kScoreThreads) void score_stats_bf16(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, int T, int Qn, int H,
    int Hkv, int G, int n_rows, int rows_pad, int n_split, float scale_log2,
    float2* __restrict__ stats) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int KS = D / 16, QSTR = D + 8;
    uint16_t* Qs = (uint16_t*)smem;
    const int chunk_cap = rows_pad < kRowChunk ? rows_pad : kRowChunk;
    float2* wst = (float2*)(smem + (size_t)chunk_cap * QSTR * 2);   // [waves][chunk_cap]

    const int split = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, r32 = lane & 31, hf = lane >> 5;
    const int c0 = split * kKeysPerSplit + w * kKeysPerWave;
    const uint16_t* Kg = kc + ((size_t)l * Hkv + g) * (size_t)T * D;

    bf16x8 kf[2][KS];
    load_k_frags<D>(Kg, c0, T, r32, hf, kf);

    for (int rc0 = 0; rc0 < rows_pad; rc0 += kRowChunk) {
        const int nrows = rows_pad - rc0 < kRowChunk ? rows_pad - rc0 : kRowChunk;
        __syncthreads();
        stage_q<D>(q, Qs, l, g, rc0, nrows, n_rows, Qn, H, G);
        __syncthreads();
        for (int rb = 0; rb < nrows / 32; ++rb) {
            f32x16 acc0 = {}, acc1 = {};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 qf = *(const bf16x8*)(Qs + (rb * 32 + r32) * QSTR + ks * 16 + hf * 8);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0][ks], qf, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[1][ks], qf, acc1, 0, 0, 0);
            }
            // acc_kb[v] = S[row rb*32 + r32][key c0 + kb*32 + 8(v/4) + 4hf + v%4]
            float x[32];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = c0 + 8 * (v >> 2) + 4 * hf + (v & 3);
                x[v] = key < T ? acc0[v] * scale_log2 : -INFINITY;
                x[16 + v] = key + 32 < T ? acc1[v] * scale_log2 : -INFINITY;
            }
            float m = -INFINITY;
#pragma unroll
            for (int v = 0; v < 32; ++v) m = fmaxf(m, x[v]);
            float z = 0.f;
            if (m != -INFINITY) {
#pragma unroll
                for (int v = 0; v < 32; ++v) z += fast_exp2(x[v] - m);
            }
            const float m2 = swap_half(m), z2 = swap_half(z);
            const float M = fmaxf(m, m2);
            float Z = 0.f;
            if (M != -INFINITY) {
                Z = (m == -INFINITY ? 0.f : z * fast_exp2(m - M)) +
                    (m2 == -INFINITY ? 0.f : z2 * fast_exp2(m2 - M));
            }
            if (hf == 0) wst[w * chunk_cap + rb * 32 + r32] = make_float2(M, Z);
        }
        __syncthreads();
        for (int rr = tid; rr < nrows; rr += kScoreThreads) {
            float M = -INFINITY;
            for (int ww = 0; ww < kScoreWaves; ++ww) M = fmaxf(M, wst[ww * chunk_cap + rr].x);
            float Z = 0.f;
            if (M != -INFINITY) {
                for (int ww = 0; ww < kScoreWaves; ++ww) {
                    const float2 s = wst[ww * chunk_cap + rr];
                    if (s.x != -INFINITY) Z += s.y * fast_exp2(s.x - M);
                }
            }
            stats[(((size_t)l * Hkv + g) * n_split + split) * rows_pad + rc0 + rr] =
                make_float2(M, Z);
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

template <int D>
__global__ __launch_bounds__(kScoreThreads) void score_colsum_bf16(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, int T, int Qn, int H,
    int Hkv, int G, int n_rows, int rows_pad, float scale_log2, const float* __restrict__ lse2,
    const float* __restrict__ q_lse, float* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int KS = D / 16, QSTR = D + 8;
    uint16_t* Qs = (uint16_t*)smem;
    const int chunk_cap = rows_pad < kRowChunk ? rows_pad : kRowChunk;
    float* ls = (float*)(smem + (size_t)chunk_cap * QSTR * 2);     // [chunk_cap]

    const int split = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, r32 = lane & 31, hf = lane >> 5;
    const int c0 = split * kKeysPerSplit + w * kKeysPerWave;
    const uint16_t* Kg = kc + ((size_t)l * Hkv + g) * (size_t)T * D;

    bf16x8 kf[2][KS];
    load_k_frags<D>(Kg, c0, T, r32, hf, kf);
    float cs0 = 0.f, cs1 = 0.f;

    for (int rc0 = 0; rc0 < rows_pad; rc0 += kRowChunk) {
        const int nrows = rows_pad - rc0 < kRowChunk ? rows_pad - rc0 : kRowChunk;
        __syncthreads();
        stage_q<D>(q, Qs, l, g, rc0, nrows, n_rows, Qn, H, G);
        for (int rr = tid; rr < nrows; rr += kScoreThreads) {
            const int rho = rc0 + rr;
            float v;
            if (rho >= n_rows) v = INFINITY;
            else if (q_lse) v = q_lse[((size_t)l * Qn + rho / G) * H + g * G + rho % G] * kLog2e;
            else v = lse2[((size_t)l * Hkv + g) * rows_pad + rho];
            ls[rr] = v;
        }
        __syncthreads();
        for (int rb = 0; rb < nrows / 32; ++rb) {
            f32x16 acc0 = {}, acc1 = {};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 qf = *(const bf16x8*)(Qs + (rb * 32 + r32) * QSTR + ks * 16 + hf * 8);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf, kf[0][ks], acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf, kf[1][ks], acc1, 0, 0, 0);
            }
            // acc_kb[v] = S[row rb*32 + 8(v/4) + 4hf + v%4][key c0 + kb*32 + r32]
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x4 lr = *(const f32x4*)(ls + rb * 32 + 8 * j + 4 * hf);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    cs0 += fast_exp2(acc0[4 * j + i] * scale_log2 - lr[i]);
                    cs1 += fast_exp2(acc1[4 * j + i] * scale_log2 - lr[i]);
                }
            }
        }
    }
    cs0 += swap_half(cs0);
    cs1 += swap_half(cs1);
    if (hf == 0) {
        float* out = part + ((size_t)l * Hkv + g) * T;
        if (c0 + r32 < T) out[c0 + r32] = cs0;
        if (c0 + 32 + r32 < T) out[c0 + 32 + r32] = cs1;
    }
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

__global__ __launch_bounds__(1024) void score_finalize(const float* __restrict__ part, int n_part,
                                                       int T, float inv_hq,
                                                       float* __restrict__ scores) {
    __shared__ float red_lo[16], red_hi[16];
    const int l = blockIdx.x, tid = threadIdx.x;
    float* a = scores + (size_t)l * T;
    float lo = INFINITY, hi = -INFINITY;
    for (int i = tid; i < T; i += 1024) {
        float p = 0.f;
        for (int j = 0; j < n_part; ++j) p += part[((size_t)l * n_part + j) * T + i];
        p *= inv_hq;
        a[i] = p;
        lo = fminf(lo, p);
        hi = fmaxf(hi, p);
    }
    for (int o = 32; o > 0; o >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, o, 64));
        hi = fmaxf(hi, __shfl_xor(hi, o, 64));
    }
    if ((tid & 63) == 0) {
        red_lo[tid >> 6] = lo;
        red_hi[tid >> 6] = hi;
    }
    __syncthreads();
    lo = red_lo[0];
    hi = red_hi[0];
    for (int i = 1; i < 16; ++i) {
        lo = fminf(lo, red_lo[i]);
        hi = fmaxf(hi, red_hi[i]);
    }
    const bool flat = !(hi > lo);
    const float span = hi - lo;
    for (int i = tid; i < T; i += 1024) a[i] = flat ? 0.f : (a[i] - lo) / span;
}

template <int D>
hipError_t launch_score_bf16(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                             float* scores, hipStream_t st, float scale) {
    const int G = p.H / p.H_kv;
    const int n_rows = p.n_query * G;
    const int chunk_cap = w.rows_pad < kRowChunk ? w.rows_pad : kRowChunk;
    const size_t qbytes = (size_t)chunk_cap * (D + 8) * 2;
    const float sl2 = scale * kLog2e;
    const uint16_t* q = (const uint16_t*)p.q;
    const uint16_t* kc = (const uint16_t*)p.k_cache;
    float* part = (float*)(ws + w.part_off);
    float* lse2 = (float*)(ws + w.lse_off);
    const dim3 grid(w.n_split, p.H_kv, p.L);
    if (!p.q_lse) {
        const size_t lds = qbytes + (size_t)kScoreWaves * chunk_cap * sizeof(float2);
        hipFuncSetAttribute((const void*)score_stats_bf16<D>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(score_stats_bf16<D>, grid, dim3(kScoreThreads), lds, st, q, kc, p.T_c,
                           p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, w.n_split, sl2,
                           (float2*)(ws + w.stats_off));
        const long n = (long)p.L * p.H_kv * w.rows_pad;
        hipLaunchKernelGGL(score_merge, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                           (const float2*)(ws + w.stats_off), p.L * p.H_kv, w.n_split,
                           w.rows_pad, n_rows, lse2);
    }
    const size_t lds = qbytes + (size_t)chunk_cap * sizeof(float);
    hipFuncSetAttribute((const void*)score_colsum_bf16<D>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(score_colsum_bf16<D>, grid, dim3(kScoreThreads), lds, st, q, kc, p.T_c,
                       p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, sl2, lse2, p.q_lse, part);
    hipLaunchKernelGGL(score_finalize, dim3(p.L), dim3(1024), 0, st, part, w.n_part, p.T_c,
                       1.0f / ((float)p.H * (float)p.n_query), scores);
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
    hipLaunchKernelGGL(score_finalize, dim3(p.L), dim3(1024), 0, st, part, w.n_part, p.T_c,
                       1.0f / ((float)p.H * (float)p.n_query), scores);
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
