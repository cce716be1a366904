// Sparse-context causal attention (Sec. 3.3-3.4, App. A.2; the attention step of
// Algorithm 1).  Target t of layer l (position p, compact index u_t in U)
// attends to the compact context c = 0 .. u_t (C_l(p) = U cap {j <= p}) or, for
// the Full-Prefix Control, to positions j = 0 .. p.  Key/value row j is the
// fresh row of j when j is in R_l (src[l][c] >= 0) and the naive cached row
// otherwise.
//
// bf16 kernel (bf16 MFMA 32x32x16, fp32 accumulation, flash-style online
// softmax in the exp2 domain):
// - a workgroup of 4 waves owns 128 (target, head) rows of one KV head g:
//   floor(128/G) consecutive targets times the G query heads that share g, so
//   every gathered K/V tile is used by all G heads;
// - per tile of 64 context keys the 256 threads gather the K and V rows into
//   LDS, choosing per key between the fresh rows (k_new/v_new) and the cached
//   layer (k_cache/v_cache); K is stored row-major, V transposed so the PV
//   product reads it as an MFMA A operand;
// - each wave computes S^T = K Q^T with one query row per lane (Q stays in
//   registers), so row max and row sum are lane-local plus one exchange with
//   the lane 32 away; P^T stays in registers as the B operand of O^T = V^T P^T;
// - the mask is the staircase of the targets' limits: tiles below the first
//   target's limit run unmasked, the rest compare each key with its row's limit;
// - tiles are taken heaviest-first (the last targets have the longest
//   contexts) and consecutive workgroups cycle through the KV heads, so the
//   workgroups that land on one XCD share a KV head and its L2 working set;
// - the global loads of the next tile are issued before the current tile's
//   MFMAs.
// fp32 kernel: one wave per (target, head), VALU dot products and an online
// softmax across the wave; used for fp32 inputs where bf16 MFMA would not meet
// fp32 accuracy.

#include <math.h>

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

struct AttnArgs {
    const void* q_new;
    const void* k_new;
    const void* v_new;
    const void* kc;          // layer base [H_kv][T][d]
    const void* vc;
    const int32_t* U;
    const int32_t* cidx;
    const int32_t* src_l;    // src + layer * T
    const int32_t* rank_l;   // rank + layer * T
    const int32_t* R_off;
    const int32_t* R_idx;
    const int32_t* R_u;
    const int32_t* counts;
    void* out;
    float* lse;
    int H, Hkv, G, T, layer, BT;
    float scale;             // softmax scale (natural units)
};

// Row of key index c for KV head g: returns the element offset of that row in
// either the fresh tensor (fresh = true) or the cached layer.
template <bool FULL>
__device__ __forceinline__ size_t kv_row(const AttnArgs& a, int c, int g, bool& fresh) {
    int pos, r;
    if (FULL) {
        pos = c;
        r = a.rank_l[c];
    } else {
        pos = a.U[c];
        r = a.src_l[c];
    }
    fresh = r >= 0;
    return fresh ? ((size_t)r * a.Hkv + g) : ((size_t)g * a.T + pos);
}

// ----------------------------------------------------------------- bf16 MFMA

constexpr float kRescaleSlack = 8.0f;      // log2 units the running max may lag the true max

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// max / sum of a value and its copy in the lane 32 away (one VALU swap).
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// NW waves x RB*32 rows per workgroup; LDS tiles of BN keys, computed in
// 64-key steps of two 32-key MFMA blocks.  With RB = 2 every K and V fragment
// read from LDS feeds two MFMAs (one per 32-row block).
template <int D, bool FULL, int NW, int BN, int RB>
__global__ __launch_bounds__(NW * 64, RB == 1 ? 8 / NW : 4 / NW) void attn_bf16(AttnArgs a) {
    constexpr int NT = NW * 64;            // threads
    constexpr int KS = D / 16;             // k-steps of the QK^T contraction
    constexpr int DB = D / 32;             // 32-wide d blocks of O^T
    constexpr int KSTR = D + 8;            // K tile row stride (elements)
    constexpr int VSTR = D + RELAXKV_ATTN_VPAD;   // V tile row stride (elements)
    constexpr int P = D / 8;               // 16-byte parts per row
    constexpr int KPT = BN * P / NT;       // keys per thread in the loader
    static_assert(KPT >= 1 && BN * P == KPT * NT, "loader shape");
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][BN * KSTR];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[2][BN * VSTR];

    const int Hkv = a.Hkv;
    const int g = blockIdx.x % Hkv;
    const int tile_rev = blockIdx.x / Hkv;
    const int nR = a.counts[1 + a.layer];
    const int ntiles = (nR + a.BT - 1) / a.BT;
    if (tile_rev >= ntiles) return;
    const int tile = ntiles - 1 - tile_rev;          // heaviest tiles first
    const int t0 = tile * a.BT;
    const int t1 = min(t0 + a.BT, nR);
    const int off = a.R_off[a.layer];
    const int32_t* lim_of = FULL ? a.R_idx + off : a.R_u + off;
    // Limits are compact indices (union) or positions (full prefix).  A global
    // target that precedes every union position has limit -1 (empty context):
    // its row masks every key and is written as the empty sum at the end.
    const int cmin = lim_of[t0];
    const int cmax = max(lim_of[t1 - 1], 0);

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r32 = lane & 31, hf = lane >> 5;
    const uint16_t* qn = (const uint16_t*)a.q_new;
    const float sl2 = a.scale * kLog2e;              // > 0

    // This lane's (target, head) rows, one per 32-row block.
    int t_of[RB], head_of[RB], lim[RB];
    bool valid[RB];
    bf16x8 qf[RB][KS];
    f32x16 o[RB][DB];
    float m_run[RB], l_run[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int rho = (w * RB + rb) * 32 + r32;
        const int tl = rho / a.G, hh = rho - tl * a.G;
        t_of[rb] = t0 + tl;
        valid[rb] = tl < a.BT && t_of[rb] < t1;
        lim[rb] = valid[rb] ? lim_of[t_of[rb]] : cmax;   // padding rows: finite, never stored
        head_of[rb] = g * a.G + hh;
        const uint16_t* qrow =
            qn + ((size_t)(valid[rb] ? t_of[rb] : t0) * a.H + (valid[rb] ? head_of[rb] : 0)) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[rb][ks] = *(const bf16x8*)(qrow + ks * 16 + hf * 8);
#pragma unroll
        for (int db = 0; db < DB; ++db) o[rb][db] = f32x16{};
        m_run[rb] = lim[rb] < 0 ? 0.f : -INFINITY;     // empty context: every p is exp2(-inf) = 0
        l_run[rb] = 0.f;
    }

    // Loader: thread -> (key group kq, 16-byte part); keys kq*KPT .. kq*KPT+KPT-1.
    // Two-stage pipeline: the row indices of tile kt+2 are loaded while tile kt
    // is computed; the K/V rows of tile kt+1 are loaded from them one step later.
    const int kq = tid / P, part = tid % P;
    const uint16_t* kn = (const uint16_t*)a.k_new;
    const uint16_t* vn = (const uint16_t*)a.v_new;
    const uint16_t* kc = (const uint16_t*)a.kc;
    const uint16_t* vc = (const uint16_t*)a.vc;
    const int32_t* srcmap = FULL ? a.rank_l : a.src_l;
    // Per-workgroup bases of KV head g; per key only a row offset is added.
    const uint16_t* kng = kn + (size_t)g * D;                    // fresh rows: stride Hkv*D
    const uint16_t* kcg = kc + (size_t)g * a.T * D;              // cached rows: stride D
    const long dv_fresh = vn - kn;                               // V address = K address + delta
    const long dv_cached = vc - kc;
    int ipos[KPT], irow[KPT];                        // position, fresh rank (-1: cached row)
    u32x4 kr[KPT], vr[KPT];

    // Keys past cmax re-read the row of cmax: their logits are masked (every
    // 64-key step that holds such a key is a staircase step), so only
    // finiteness matters.
    auto load_idx = [&](int c0) {
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk) {
            const int c = min(c0 + kq * KPT + kk, cmax);
            ipos[kk] = FULL ? c : a.U[c];
            irow[kk] = srcmap[c];
        }
    };
    auto load_rows = [&]() {
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk) {
            const bool fresh = irow[kk] >= 0;
            const uint16_t* kp = fresh ? kng + (size_t)irow[kk] * (Hkv * D) : kcg + (size_t)ipos[kk] * D;
            kp += part * 8;
            kr[kk] = *(const u32x4*)kp;
            vr[kk] = *(const u32x4*)(kp + (fresh ? dv_fresh : dv_cached));
        }
    };

    // Transposing V reads: lane (group G = lane/16, j = lane%16) points at key row
    // 4*(G/2) + j/4 and d column (G%2)*16 + 4*(j%4) of each 16-key, 32-d block.
    // ds_read_b64_tr_b16 gives lane i of a 16-lane group element i%4 of the
    // 8-byte chunks read by lanes 4m + i/4 (m = 0..3), so lane i receives 4 keys
    // at one d: element e of the k-index block hf*8 .. hf*8+7 of half k2 is key
    // 16*k2 + 8(e/4) + 4hf + e%4 of the 32-key block, the S^T lane layout.
    const int vtr_off = (4 * (lane >> 5) + ((lane & 15) >> 2)) * VSTR + ((lane >> 4) & 1) * 16 +
                        4 * (lane & 3);

    const int nkt = cmax / BN + 1;
    load_idx(0);
    load_rows();
    if (nkt > 1) load_idx(BN);
    for (int kt = 0; kt < nkt; ++kt) {
        uint16_t* ks_b = Ks[kt & 1];
        uint16_t* vs_b = Vs[kt & 1];
        // Store tile kt.  The buffer was last read in step kt-2, which every wave
        // finished before the barrier of step kt-1.
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk) {
            *(u32x4*)(ks_b + (kq * KPT + kk) * KSTR + part * 8) = kr[kk];
            *(u32x4*)(vs_b + (kq * KPT + kk) * VSTR + part * 8) = vr[kk];
        }
        __syncthreads();
        if (kt + 1 < nkt) {
            load_rows();                                   // tile kt+1
            if (kt + 2 < nkt) load_idx((kt + 2) * BN);     // indices of tile kt+2
        }
#pragma unroll
        for (int sub = 0; sub < BN / 64; ++sub) {
            const int c0 = kt * BN + sub * 64;
            if (c0 > cmax) break;
            const uint16_t* kst = ks_b + sub * 64 * KSTR;
            const uint16_t* vst = vs_b + sub * 64 * VSTR;
            // S^T = K Q^T: s[rb][kb][v] = S[row rb][key c0 + kb*32 + 8(v/4) + 4hf + v%4]
            f32x16 s[RB][2];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) s[rb][0] = s[rb][1] = f32x16{};
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(2);
#endif
            // K fragments are read ahead of the MFMAs that use them: with one row
            // block all 2*KS fragments are issued first; with two row blocks (each
            // fragment feeds two MFMAs) a ring of two k-steps keeps registers low.
            if constexpr (RB == 1) {
                bf16x8 kf[KS][2];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    kf[ks][0] = *(const bf16x8*)(kst + r32 * KSTR + ks * 16 + hf * 8);
                    kf[ks][1] = *(const bf16x8*)(kst + (32 + r32) * KSTR + ks * 16 + hf * 8);
                }
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    s[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][0], qf[0][ks], s[0][0], 0, 0, 0);
                    s[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][1], qf[0][ks], s[0][1], 0, 0, 0);
                }
#if RELAXKV_ATTN_SCHED
                __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);      // 4 LDS reads
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // 2 MFMAs
                    if (ks + 2 < KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                }
#endif
            } else {
                bf16x8 ka[2], kb[2];
                ka[0] = *(const bf16x8*)(kst + r32 * KSTR + hf * 8);
                ka[1] = *(const bf16x8*)(kst + (32 + r32) * KSTR + hf * 8);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    if (ks + 1 < KS) {
                        kb[0] = *(const bf16x8*)(kst + r32 * KSTR + (ks + 1) * 16 + hf * 8);
                        kb[1] = *(const bf16x8*)(kst + (32 + r32) * KSTR + (ks + 1) * 16 + hf * 8);
                    }
#pragma unroll
                    for (int rb = 0; rb < RB; ++rb) {
                        s[rb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qf[rb][ks], s[rb][0], 0, 0, 0);
                        s[rb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qf[rb][ks], s[rb][1], 0, 0, 0);
                    }
                    ka[0] = kb[0];
                    ka[1] = kb[1];
                }
            }
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(0);
#endif
            if (c0 + 63 > cmin) {                          // staircase step: mask
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int key = c0 + 8 * (v >> 2) + 4 * hf + (v & 3);
                        if (key > lim[rb]) s[rb][0][v] = -INFINITY;
                        if (key + 32 > lim[rb]) s[rb][1][v] = -INFINITY;
                    }
            }
            // Row max over the step in log2 units.  Lazy rescaling: the running
            // max only moves when the step's max exceeds it by more than
            // kRescaleSlack, so p <= 2^kRescaleSlack and most steps skip the O
            // rescale.  Both halves of a row take the same decision.
            float mx[RB];
            bool need = false;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                float m = fmaxf(s[rb][0][0], s[rb][1][0]);
#pragma unroll
                for (int v = 1; v < 16; ++v) m = fmaxf(m, fmaxf(s[rb][0][v], s[rb][1][v]));
                mx[rb] = pair_max(m) * sl2;
                need |= mx[rb] > m_run[rb] + kRescaleSlack;
            }
            if (__any(need)) {
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    const float m_new = mx[rb] > m_run[rb] + kRescaleSlack ? mx[rb] : m_run[rb];
                    const float alpha = fast_exp2(m_run[rb] - m_new);
                    l_run[rb] *= alpha;
#pragma unroll
                    for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
                    m_run[rb] = m_new;
                }
            }
            // P^T as bf16 B operands: pb[rb][kb][k2] holds values 8*k2 .. 8*k2+7.
            bf16x8 pb[RB][2][2];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                float ls = 0.f;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const float p = fast_exp2(fmaf(s[rb][kb][v], sl2, -m_run[rb]));
                        ls += p;
                        pb[rb][kb][v >> 3][v & 7] = (__bf16)p;
                    }
                l_run[rb] += ls;
            }
            // O^T += V^T P^T
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(2);
#endif
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int db = 0; db < DB; ++db) {
#pragma unroll
                    for (int k2 = 0; k2 < 2; ++k2) {
                        const uint16_t* p0 = vst + vtr_off + (kb * 32 + k2 * 16) * VSTR + db * 32;
                        const v4i16 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p0);
                        const v4i16 a1 =
                            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 8 * VSTR));
                        const bf16x8 vv = __builtin_bit_cast(
                            bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                        for (int rb = 0; rb < RB; ++rb)
                            o[rb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pb[rb][kb][k2],
                                                                                o[rb][db], 0, 0, 0);
                    }
                }
            }
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(0);
#endif
        }
    }

#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const float l_tot = pair_sum(l_run[rb]);
        if (!valid[rb]) continue;
        const bool empty = lim[rb] < 0;
        const float inv = empty ? 0.f : 1.0f / l_tot;
        uint16_t* out = (uint16_t*)a.out + ((size_t)t_of[rb] * a.H + head_of[rb]) * D;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d0 = db * 32 + 8 * j + 4 * hf;
                const uint32_t lo = (uint32_t)f32_to_bf16_bits(o[rb][db][4 * j] * inv) |
                                    ((uint32_t)f32_to_bf16_bits(o[rb][db][4 * j + 1] * inv) << 16);
                const uint32_t hi = (uint32_t)f32_to_bf16_bits(o[rb][db][4 * j + 2] * inv) |
                                    ((uint32_t)f32_to_bf16_bits(o[rb][db][4 * j + 3] * inv) << 16);
                *(u32x2*)(out + d0) = u32x2{lo, hi};
            }
        }
        if (a.lse && hf == 0)
            a.lse[(size_t)t_of[rb] * a.H + head_of[rb]] =
                empty ? -INFINITY : (m_run[rb] + __log2f(l_tot)) * kLn2;
    }
}

// ----------------------------------------------------------------- fp32 VALU

template <int D, bool FULL>
__global__ __launch_bounds__(64) void attn_f32(AttnArgs a) {
    constexpr int DPL = D / 64;            // d values owned per lane
    __shared__ float qs[D];
    const int t = blockIdx.x, head = blockIdx.y;
    const int nR = a.counts[1 + a.layer];
    if (t >= nR) return;
    const int lane = threadIdx.x;
    const int g = head / a.G;
    const int off = a.R_off[a.layer];
    const int lim = FULL ? a.R_idx[off + t] : a.R_u[off + t];
    if (lim < 0) {                                     // empty context: the empty sum
        float* out = (float*)a.out + ((size_t)t * a.H + head) * D;
        for (int e = lane; e < D; e += 64) out[e] = 0.f;
        if (a.lse && lane == 0) a.lse[(size_t)t * a.H + head] = -INFINITY;
        return;
    }
    const float* qn = (const float*)a.q_new;
    const float* kn = (const float*)a.k_new;
    const float* vn = (const float*)a.v_new;
    const float* kc = (const float*)a.kc;
    const float* vc = (const float*)a.vc;
    for (int e = lane; e < D; e += 64) qs[e] = qn[((size_t)t * a.H + head) * D + e];
    __syncthreads();

    float o[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;
    for (int c0 = 0; c0 <= lim; c0 += 64) {
        const int c = c0 + lane;
        float s = -INFINITY;
        const float* vrow = nullptr;
        if (c <= lim) {
            bool fresh;
            const size_t row = kv_row<FULL>(a, c, g, fresh);
            const float* kr = (fresh ? kn : kc) + row * D;
            vrow = (fresh ? vn : vc) + row * D;
            float acc = 0.f;
            for (int e = 0; e < D; ++e) acc = fmaf(qs[e], kr[e], acc);
            s = acc * a.scale;
        }
        const float m_new = fmaxf(m_run, wave_max(s));
        const float alpha = expf(m_run - m_new);
        const float p = c <= lim ? expf(s - m_new) : 0.f;
        l_run = l_run * alpha + wave_sum(p);
#pragma unroll
        for (int i = 0; i < DPL; ++i) o[i] *= alpha;
        const int nk = min(64, lim - c0 + 1);
        for (int j = 0; j < nk; ++j) {
            const float pj = __shfl(p, j, 64);
            const float* vj = (const float*)__shfl((long long)vrow, j, 64);
#pragma unroll
            for (int i = 0; i < DPL; ++i) o[i] = fmaf(pj, vj[lane + 64 * i], o[i]);
        }
        m_run = m_new;
    }
    float* out = (float*)a.out + ((size_t)t * a.H + head) * D;
#pragma unroll
    for (int i = 0; i < DPL; ++i) out[lane + 64 * i] = o[i] / l_run;
    if (a.lse && lane == 0) a.lse[(size_t)t * a.H + head] = m_run + logf(l_run);
}

constexpr int kNW = RELAXKV_ATTN_WAVES;
constexpr int kBN = RELAXKV_ATTN_TILE;
constexpr int kRB = RELAXKV_ATTN_ROWBLOCKS;
static_assert(kAttnRows == kNW * kRB * 32, "rows per workgroup");

template <int D, bool FULL>
void launch_one(const AttnArgs& a, bool bf16, int n_bound, hipStream_t st) {
    if (bf16) {
        const int ntiles = (n_bound + a.BT - 1) / a.BT;
        hipLaunchKernelGGL((attn_bf16<D, FULL, kNW, kBN, kRB>), dim3(ntiles * a.Hkv), dim3(kNW * 64),
                           0, st, a);
    } else {
        hipLaunchKernelGGL((attn_f32<D, FULL>), dim3(n_bound, a.H), dim3(64), 0, st, a);
    }
}

}  // namespace

hipError_t launch_sparse_attn(const relaxkv_problem& p, const relaxkv_sets& s, int layer,
                              const void* q_new, const void* k_new, const void* v_new,
                              void* out, float* lse_out, int context_mode, hipStream_t st) {
    const bool bf16 = p.dtype == RELAXKV_DTYPE_BF16;
    const size_t esz = bf16 ? 2 : 4;
    const size_t layer_elems = (size_t)p.H_kv * p.T_c * p.d;
    AttnArgs a;
    a.q_new = q_new;
    a.k_new = k_new;
    a.v_new = v_new;
    a.kc = (const char*)p.k_cache + (size_t)layer * layer_elems * esz;
    a.vc = (const char*)p.v_cache + (size_t)layer * layer_elems * esz;
    // The layer's context list: the union, or a construction variant's list.
    a.U = s.context_sets == RELAXKV_CONTEXT_SETS_GLOBAL      ? s.ctx
          : s.context_sets == RELAXKV_CONTEXT_SETS_LAYERWISE ? s.ctx + (size_t)layer * p.T_c
                                                             : s.U;
    a.cidx = s.cidx;
    a.src_l = s.src + (size_t)layer * p.T_c;
    a.rank_l = s.rank + (size_t)layer * p.T_c;
    a.R_off = s.R_off;
    a.R_idx = s.R_idx;
    a.R_u = s.R_u;
    a.counts = s.counts;
    a.out = out;
    a.lse = lse_out;
    a.H = p.H;
    a.Hkv = p.H_kv;
    a.G = p.H / p.H_kv;
    a.T = p.T_c;
    a.layer = layer;
    a.BT = bf16 ? kNW * kRB * 32 / a.G : 1;
    a.scale = p.softmax_scale > 0.f ? p.softmax_scale : 1.0f / sqrtf((float)p.d);
    // |R_l| <= |union of S_l' for l' >= l| <= min(T_c, (L - l) k) for RelaxKV's
    // targets, <= T_c for a global target list; the device count decides which
    // workgroups run.
    const long kb = s.global_targets ? (long)p.T_c : (long)(p.L - layer) * s.k;
    const int n_bound = (int)(kb < p.T_c ? kb : p.T_c);
    const bool full = context_mode == RELAXKV_CONTEXT_FULL;
    if (p.d == 128) {
        full ? launch_one<128, true>(a, bf16, n_bound, st) : launch_one<128, false>(a, bf16, n_bound, st);
    } else {
        full ? launch_one<64, true>(a, bf16, n_bound, st) : launch_one<64, false>(a, bf16, n_bound, st);
    }
    return hipGetLastError();
}

}  // namespace relaxkv
