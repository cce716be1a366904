// Layer-wise query-attention score (Sec. 3.2 equation; first step of Algorithm 1):
//   A_l[h,t,i] = softmax_i(sigma <q_{l,t,h}, k_{l,g(h),i}>),
//   p_{l,i} = (1/(H Qn)) sum_{h,t} A_l[h,t,i],   a_{l,i} = MinMax_i(p_{l,i}).
//
// bf16 path (bf16 MFMA, fp32 accumulation).  Per layer l and KV head g the
// Qn*G query rows that share g form one row set.  A workgroup takes one
// (l, g, split of contiguous keys: 4096 in the statistics pass, 4096 or 8192 in
// the column-sum pass): it stages the row set into LDS once (fragment-major),
// and each of its waves loads its own 32-key blocks from HBM straight into
// registers and runs every 32-row block against them, so K never passes
// through LDS (in the column-sum pass a wave holds two key blocks, so a query
// fragment read from LDS feeds two MFMAs):
//   1. score_stats_kreg -- S^T = K Q^T (one query row per lane): each row's
//      (reference, sum of exp2) over the split.           [skipped with q_lse]
//   2. score_merge  -- per row, merge the splits into a log2-sum-exp.
//   3. score_colsum_kreg -- S = Q K^T - lse (one key per lane; each
//      accumulator starts at its row's -lse), summing exp2 over the rows: the
//      pooled mass of each key for this KV head.
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

#ifndef RELAXKV_SCORE_SPLIT
#define RELAXKV_SCORE_SPLIT 4096              // keys per statistics workgroup
#endif
#ifndef RELAXKV_SCORE_KREG_NW
#define RELAXKV_SCORE_KREG_NW 16              // waves per workgroup (four per SIMD)
#endif
#ifndef RELAXKV_SCORE_KREG_NKB
#define RELAXKV_SCORE_KREG_NKB 1              // 32-key blocks per wave and round (statistics pass)
#endif
#ifndef RELAXKV_SCORE_COLSUM_NW
#define RELAXKV_SCORE_COLSUM_NW 16            // waves per column-sum workgroup
#endif
#ifndef RELAXKV_SCORE_COLSUM_NKB
#define RELAXKV_SCORE_COLSUM_NKB 2            // 32-key blocks per wave and round (column-sum pass)
#endif
constexpr int kKeysPerSplit = RELAXKV_SCORE_SPLIT;
constexpr int kKregRowBlocks = 10;            // 32-row blocks staged per row chunk

// Range a block's sum of exp2(s - m) may take before the statistics pass moves
// its reference m (see score_stats_kreg).
constexpr float kRefHi = 18446744073709551616.0f;     // 2^64
constexpr float kRefLo = 5.42101086242752217e-20f;    // 2^-64

__host__ __device__ inline int round_up32(int x) { return (x + 31) / 32 * 32; }

// x plus the copy of x held by the lane 32 away (v_permlane32_swap with both
// operands x returns x and the partner's x, in some order, in its two results).
__device__ __forceinline__ float pair_add(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// The copy of x held by the lane 32 away (xor of both results with x leaves the
// partner's bits whichever result holds which).
__device__ __forceinline__ float pair_other(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(r[0] ^ r[1] ^ u);
}

// Stage rows rc0 .. rc0 + 32 nrb - 1 of the row set (l, g) into Qs, fragment-major:
// fragment (rb, j) holds the MFMA operand of 32-row block rb and k-step j (lane
// l: row 32 rb + l % 32, 16-byte chunk 2j + l / 32; padding rows are zero).
template <int D, int NW>
__device__ __forceinline__ void stage_rows(bf16x8* Qs, const uint16_t* __restrict__ q, int l,
                                           int g, int Qn, int H, int G, int n_rows, int rc0,
                                           int nrb) {
    constexpr int KS = D / 16;
    for (int f = threadIdx.x; f < nrb * KS * 64; f += NW * 64) {
        const int ln = f & 63, fj = f >> 6, rb = fj / KS, j = fj - rb * KS;
        const int row = rc0 + rb * 32 + (ln & 31), h2 = ln >> 5;
        bf16x8 v = {};
        if (row < n_rows) {
            const int t = row / G, hh = row - t * G;
            v = *(const bf16x8*)(q + (((size_t)l * Qn + t) * H + g * G + hh) * D + 16 * j + 8 * h2);
        }
        Qs[f] = v;
    }
}

// The accumulator start values of the column-sum pass: Ls[rb][hf][i] = -lse2 / sl2
// of row rc0 + 32 rb + 8 (i / 4) + 4 hf + i % 4, the row that element i of an
// S = Q K^T accumulator of row block rb holds in lane half hf; -inf for padding
// rows (their probabilities are then exp2(-inf) = 0).
__device__ __forceinline__ void stage_lse(float (*Ls)[2][16], int nt, int l, int g, int Qn,
                                          int H, int Hkv, int G, int n_rows, int rows_pad,
                                          int rc0, int nrb, float sl2,
                                          const float* __restrict__ lse2,
                                          const float* __restrict__ q_lse) {
    for (int f = threadIdx.x; f < nrb * 32; f += nt) {
        const int rb = f >> 5, hh = (f >> 4) & 1, i = f & 15;
        const int row = rc0 + 32 * rb + 8 * (i >> 2) + 4 * hh + (i & 3);
        const float x = row >= n_rows ? INFINITY
                        : q_lse ? q_lse[((size_t)l * Qn + row / G) * H + g * G + row % G] * kLog2e
                                : lse2[((size_t)l * Hkv + g) * rows_pad + row];
        Ls[rb][hh][i] = -x / sl2;
    }
}

// The 32-key blocks kr + 32 kb (kb < NKB) of K into registers, as MFMA operands
// (lane l: key kr + 32 kb + l % 32, 16-byte chunk 2j + l / 32 of k-step j); keys
// past T re-read key T-1 (their results are masked or never stored).
template <int D, int NKB>
__device__ __forceinline__ void load_keys(bf16x8 (&dst)[NKB][D / 16], const uint16_t* Kg, int T,
                                          int64_t sT, int kr, int r32, int hf) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        const int key = min(kr + 32 * kb + r32, T - 1);
        const bf16x8* kp = (const bf16x8*)(Kg + key * sT + hf * 8);
#pragma unroll
        for (int j = 0; j < D / 16; ++j) dst[kb][j] = kp[2 * j];
    }
}

// Column-sum pass with the keys in registers (rows known by their log2-sum-exp).
// A workgroup takes one (layer l, KV head g, key split).  The query rows of the
// group are staged once into LDS, fragment-major: fragment (rb, j) is the MFMA A
// operand of 32-row block rb and k-step j, lane l's 16 bytes at 16 l, so every
// read is one conflict-free ds_read_b128 at a fixed offset from the lane's base.
// Each accumulator starts at its rows' -lse2 / sl2 (the C operand of the first
// MFMA, read from a small LDS table; the lanes of a half read the same 64
// bytes), so it ends at s - lse2 / sl2 and exp2(sl2 * acc) is the probability.
// Each wave owns NKB blocks of 32 keys per round, loads them from HBM straight
// into registers (the B operand of S = Q K^T: lane l holds key l % 32, the
// 16-byte chunk 2j + l / 32 of k-step j) and runs every row block against them,
// so a query fragment read from LDS feeds NKB MFMAs and K needs no LDS at all.
// Per lane the 16 rows of a block are summed in fp32 in a fixed order, then the
// two half-waves are added: part[l][g][key] (added to the earlier row chunks'
// sum when the row set takes several chunks).  The next round's keys are
// loaded while the last row block's exp2 work runs.  Waves never wait for one
// another inside a row chunk.
template <int D, int NW, int NKB>
__global__ __launch_bounds__(NW * 64) void score_colsum_kreg(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, KvStrides ks, int T, int Qn, int H,
    int Hkv, int G, int n_rows, int rows_pad, int keys_per_split, float sl2,
    const float* __restrict__ lse2, const float* __restrict__ q_lse, float* __restrict__ part) {
    constexpr int KS = D / 16;                      // k-steps of the dot product
    constexpr int NRB = kKregRowBlocks;             // row blocks per chunk
    constexpr int KPW = NKB * 32;                   // keys of a wave per round
    constexpr int KPR = NW * KPW;                   // keys of the workgroup per round
    __shared__ bf16x8 Qs[NRB * KS * 64];
    __shared__ __attribute__((aligned(64))) float Ls[NRB][2][16];

    const int split = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, r32 = lane & 31, hf = lane >> 5;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint16_t* Kg = kc + l * ks.layer + g * ks.head;
    float* part_g = part + ((size_t)l * Hkv + g) * T;
    const int key0 = split * keys_per_split;
    const int key1 = min(T, key0 + keys_per_split);

    bf16x8 kf[NKB][KS];
    auto load_k = [&](bf16x8 (&dst)[NKB][KS], int kr) { load_keys<D, NKB>(dst, Kg, T, ks.token, kr, r32, hf); };

    for (int rc0 = 0; rc0 < rows_pad; rc0 += NRB * 32) {
        const int nrb = min(NRB, (rows_pad - rc0) / 32);
        __syncthreads();                             // the previous chunk's reads are done
        stage_rows<D, NW>(Qs, q, l, g, Qn, H, G, n_rows, rc0, nrb);
        stage_lse(Ls, NW * 64, l, g, Qn, H, Hkv, G, n_rows, rows_pad, rc0, nrb, sl2, lse2, q_lse);
        __syncthreads();

        // One round: the wave's NKB key blocks (in kfr) against every row block;
        // hook(rb) runs after the MFMAs of row block rb (before its exp2 work).
        auto round = [&](const bf16x8 (&kfr)[NKB][KS], int kr, auto&& hook) {
            float cs[NKB][2];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) cs[kb][0] = cs[kb][1] = 0.f;
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                if (rb >= nrb) break;
                f32x16 acc[NKB];
                const f32x16 init = *(const f32x16*)&Ls[rb][hf][0];
                const bf16x8* qb = Qs + rb * KS * 64 + lane;
#pragma unroll
                for (int j = 0; j < KS; ++j) {
                    const bf16x8 qj = qb[j * 64];
#pragma unroll
                    for (int kb = 0; kb < NKB; ++kb)
                        acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            qj, kfr[kb][j], j == 0 ? init : acc[kb], 0, 0, 0);
                }
                hook(rb);
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) cs[kb][v & 1] += fast_exp2(acc[kb][v] * sl2);
            }
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const float s = pair_add(cs[kb][0] + cs[kb][1]);
                const int key = kr + 32 * kb + r32;
                if (hf == 0 && key < key1) part_g[key] = rc0 == 0 ? s : part_g[key] + s;
            }
        };

        int kr = key0 + w * KPW;
        if (kr < key1) load_k(kf, kr);
        for (; kr < key1; kr += KPR)
            round(kf, kr, [&](int rb) { if (rb == nrb - 1 && kr + KPR < key1) load_k(kf, kr + KPR); });
    }
}

// Row statistics with the keys in registers: the same workgroup shape, staging
// and key rounds as score_colsum_kreg, with S^T = K Q^T (K the A operand from
// registers, the staged query fragment the B operand), so lane l holds row
// 32 rb + l % 32 and 16 keys of each 32-key block.  Per row block each lane
// keeps (m, z) = (reference, sum of exp2(s - m)) in log2 units over its keys,
// with a lazy reference: m starts at 0 and moves only when a block's sum
// leaves [2^-64, 2^64], to the larger of the block maximum and log2 of the
// running sum (so no term and no running sum exceeds 16 * 2^m); until some lane
// of the wave moves, m = 0 costs no subtraction.  Logits hundreds of log2 units
// from 0 (either sign) stay exact.  At the end of a row chunk the two
// half-waves and then the NW waves are merged in a fixed order (through LDS)
// into stats[l][g][split][row].
template <int D, int NW, int NKB>
__global__ __launch_bounds__(NW * 64) void score_stats_kreg(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, KvStrides ks, int T, int Qn, int H,
    int Hkv, int G, int n_rows, int rows_pad, int keys_per_split, int n_split, float sl2,
    float2* __restrict__ stats) {
    constexpr int KS = D / 16;
    constexpr int NRB = kKregRowBlocks;
    constexpr int KPW = NKB * 32;
    constexpr int KPR = NW * KPW;
    __shared__ bf16x8 Qs[NRB * KS * 64];
    __shared__ float2 red[NW][NRB * 32];

    const int split = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, r32 = lane & 31, hf = lane >> 5;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint16_t* Kg = kc + l * ks.layer + g * ks.head;
    const int key0 = split * keys_per_split;
    const int key1 = min(T, key0 + keys_per_split);
    bf16x8 kf[NKB][KS];

    for (int rc0 = 0; rc0 < rows_pad; rc0 += NRB * 32) {
        const int nrb = min(NRB, (rows_pad - rc0) / 32);
        __syncthreads();                             // the previous chunk's reads are done
        stage_rows<D, NW>(Qs, q, l, g, Qn, H, G, n_rows, rc0, nrb);
        __syncthreads();

        float m_ref[NRB], z_run[NRB];
        bool moved[NRB];                             // some lane of the wave left reference 0
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            m_ref[rb] = 0.f;
            z_run[rb] = 0.f;
            moved[rb] = false;
        }
        int kr = key0 + w * KPW;
        if (kr < key1) load_keys<D, NKB>(kf, Kg, T, ks.token, kr, r32, hf);
        for (; kr < key1; kr += KPR) {
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) {
                if (rb < nrb) {
                    f32x16 acc[NKB];
                    const bf16x8* qb = Qs + rb * KS * 64 + lane;
#pragma unroll
                    for (int j = 0; j < KS; ++j) {
                        const bf16x8 qj = qb[j * 64];
#pragma unroll
                        for (int kb = 0; kb < NKB; ++kb)
                            acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                kf[kb][j], qj, j == 0 ? f32x16{} : acc[kb], 0, 0, 0);
                    }
                    if (rb == nrb - 1 && kr + KPR < key1)
                        load_keys<D, NKB>(kf, Kg, T, ks.token, kr + KPR, r32, hf);
#pragma unroll
                    for (int kb = 0; kb < NKB; ++kb) {
                        // acc[kb][v] is key kr + 32 kb + 8(v/4) + 4 hf + v%4 of the row.
                        const int kb0 = kr + 32 * kb;
                        if (kb0 + 32 > key1) {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (kb0 + 8 * (v >> 2) + 4 * hf + (v & 3) >= key1)
                                    acc[kb][v] = -INFINITY;
                        }
                        float z0 = 0.f, z1 = 0.f;
                        if (moved[rb]) {
                            const float m = m_ref[rb];
#pragma unroll
                            for (int v = 0; v < 16; v += 2) {
                                z0 += fast_exp2(fmaf(acc[kb][v], sl2, -m));
                                z1 += fast_exp2(fmaf(acc[kb][v + 1], sl2, -m));
                            }
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; v += 2) {
                                z0 += fast_exp2(acc[kb][v] * sl2);
                                z1 += fast_exp2(acc[kb][v + 1] * sl2);
                            }
                        }
                        float zb = z0 + z1;
                        const bool out = !(zb <= kRefHi) || z_run[rb] + zb < kRefLo;
                        if (__builtin_expect(out, 0)) {
                            // New reference: the larger of the block maximum and the
                            // log2 of what the row has summed so far.
                            float mt = acc[kb][0];
#pragma unroll
                            for (int v = 1; v < 16; ++v) mt = fmaxf(mt, acc[kb][v]);
                            mt *= sl2;
                            const float lz =
                                z_run[rb] > 0.f ? m_ref[rb] + __log2f(z_run[rb]) : -INFINITY;
                            mt = fmaxf(mt, lz);
                            if (mt > -INFINITY) {
                                zb = 0.f;
#pragma unroll
                                for (int v = 0; v < 16; ++v)
                                    zb += fast_exp2(fmaf(acc[kb][v], sl2, -mt));
                                z_run[rb] = fast_exp2(lz - mt);
                                m_ref[rb] = mt;
                            }
                        }
                        moved[rb] = moved[rb] || __any(out);
                        z_run[rb] += zb;
                    }
                }
            }
        }
        // Each half-wave's (m, z) per row; a half that met no key holds (0, 0)
        // and becomes (-inf, 0), so no merge takes its 0 as the reference.
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            if (rb < nrb) {
                const float m = z_run[rb] > 0.f ? m_ref[rb] : -INFINITY, z = z_run[rb];
                const float m2 = pair_other(m), z2 = pair_other(z);
                const float M = fmaxf(m, m2);
                const float Z = M == -INFINITY ? 0.f : z * fast_exp2(m - M) + z2 * fast_exp2(m2 - M);
                if (hf == 0) red[w][rb * 32 + r32] = make_float2(M, Z);
            }
        }
        __syncthreads();
        for (int row = tid; row < nrb * 32; row += NW * 64) {
            float M = -INFINITY;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, red[ww][row].x);
            float Z = 0.f;
            if (M > -INFINITY) {
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) Z += red[ww][row].y * fast_exp2(red[ww][row].x - M);
            }
            stats[(((size_t)l * Hkv + g) * n_split + split) * rows_pad + rc0 + row] = make_float2(M, Z);
        }
    }
}

// Per row: merge the splits' (m, sum) pairs into a log2-sum-exp.
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
        Z += v.y * fast_exp2(v.x - M);
    }
    lse2[i] = M + __log2f(Z);
}

// ---------------------------------------------------------------- float32 path

template <int D>
__global__ __launch_bounds__(256) void score_stats_f32(const float* __restrict__ q,
                                                       const float* __restrict__ kc, KvStrides ks, int T,
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
    const float* Kg = kc + l * ks.layer + g * ks.head;
    float m = -INFINITY, z = 0.f;
    for (int i = tid; i < T; i += 256) {
        const float* kr = Kg + i * ks.token;
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
                                                        const float* __restrict__ kc, KvStrides ks, int T,
                                                        int Qn, int H, int Hkv, int G,
                                                        int rows_pad, float scale,
                                                        const float* __restrict__ lse_nat,
                                                        const float* __restrict__ q_lse,
                                                        float* __restrict__ part) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int l = blockIdx.y;
    if (i >= T) return;
    // Summed in double: a key's column takes H * Qn terms (thousands for long
    // queries and wide GQA groups), and a float running sum of that many terms
    // drifts by more than the 1e-5 the fp32 path has to meet after MinMax.
    double acc = 0.0;
    for (int g = 0; g < Hkv; ++g) {
        float kr[D];
        const float* kp = kc + l * ks.layer + g * ks.head + i * ks.token;
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
                acc += (double)expf(s * scale - lse);
            }
        }
    }
    part[(size_t)l * T + i] = (float)acc;
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

// Keys per column-sum workgroup: 4096 or 8192, whichever needs fewer key-steps
// per CU on the chip's 256 CUs (ceil(workgroups / 256) * split), the larger one
// on a tie (fewer query stagings and workgroup starts).  Each key's column sum
// does not depend on the split, so neither do the scores.
int colsum_split(const relaxkv_problem& p) {
    constexpr long kCUs = 256;
    auto cost = [&](long split) {
        const long wg = (p.T_c + split - 1) / split * (long)p.H_kv * p.L;
        return (wg + kCUs - 1) / kCUs * split;
    };
    return cost(2 * kKeysPerSplit) <= cost(kKeysPerSplit) ? 2 * kKeysPerSplit : kKeysPerSplit;
}

template <int D>
void launch_passes_bf16(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                        hipStream_t st, float sl2) {
    const int G = p.H / p.H_kv;
    const int n_rows = p.n_query * G;
    const uint16_t* q = (const uint16_t*)p.q;
    const uint16_t* kc = (const uint16_t*)p.k_cache;
    float* part = (float*)(ws + w.part_off);
    float* lse2 = (float*)(ws + w.lse_off);
    float2* stats = (float2*)(ws + w.stats_off);
    constexpr int KNW = RELAXKV_SCORE_KREG_NW, KNKB = RELAXKV_SCORE_KREG_NKB;
    constexpr int CNW = RELAXKV_SCORE_COLSUM_NW, CNKB = RELAXKV_SCORE_COLSUM_NKB;
    static_assert(kKeysPerSplit % (KNW * KNKB * 32) == 0 && kKeysPerSplit % (CNW * CNKB * 32) == 0,
                  "a split is whole rounds of both passes (the statistics splits are the workspace's n_split)");
    const int kps = kKeysPerSplit;
    const dim3 kgrid((p.T_c + kps - 1) / kps, p.H_kv, p.L);
    if (!p.q_lse) {
        hipLaunchKernelGGL((score_stats_kreg<D, KNW, KNKB>), kgrid, dim3(KNW * 64), 0, st, q, kc,
                           kv_strides(p), p.T_c, p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, kps, w.n_split,
                           sl2, stats);
        const long n = (long)p.L * p.H_kv * w.rows_pad;
        hipLaunchKernelGGL(score_merge, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                           (const float2*)stats, p.L * p.H_kv, w.n_split, w.rows_pad, n_rows, lse2);
    }
    const int cps = colsum_split(p);
    const dim3 cgrid((p.T_c + cps - 1) / cps, p.H_kv, p.L);
    hipLaunchKernelGGL((score_colsum_kreg<D, CNW, CNKB>), cgrid, dim3(CNW * 64), 0, st, q, kc,
                       kv_strides(p), p.T_c, p.n_query, p.H, p.H_kv, G, n_rows, w.rows_pad, cps, sl2,
                       (const float*)lse2, p.q_lse, part);
}

template <int D>
hipError_t launch_score_bf16(const relaxkv_problem& p, const ScoreWorkspace& w, char* ws,
                             float* scores, hipStream_t st, float scale) {
    launch_passes_bf16<D>(p, w, ws, st, scale * kLog2e);
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
                           kv_strides(p), p.T_c, p.n_query, p.H, p.H_kv, G, w.rows_pad, scale, lse);
    hipLaunchKernelGGL(score_colsum_f32<D>, dim3((p.T_c + 255) / 256, p.L), dim3(256), 0, st, q,
                       kc, kv_strides(p), p.T_c, p.n_query, p.H, p.H_kv, G, w.rows_pad, scale, lse, p.q_lse,
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
