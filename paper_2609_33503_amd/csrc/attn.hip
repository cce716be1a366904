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
        const int ci = a.cidx[c];
        r = ci >= 0 ? a.src_l[ci] : -1;
    } else {
        pos = a.U[c];
        r = a.src_l[c];
    }
    fresh = r >= 0;
    return fresh ? ((size_t)r * a.Hkv + g) : ((size_t)g * a.T + pos);
}

// ----------------------------------------------------------------- bf16 MFMA

constexpr int BN = kAttnKeys;              // 64 keys per tile

template <int D, bool FULL>
__global__ __launch_bounds__(256, 2) void attn_bf16(AttnArgs a) {
    constexpr int KS = D / 16;             // k-steps of the QK^T contraction
    constexpr int DB = D / 32;             // 32-wide d blocks of O^T
    constexpr int KSTR = D + 8;            // K tile row stride (elements)
    constexpr int VSTR = BN + 4;           // V^T tile row stride (elements)
    constexpr int P = D / 8;               // 16-byte parts per row
    constexpr int KPT = BN * P / 256;      // keys per thread in the loader (4 or 2)
    __shared__ __attribute__((aligned(16))) uint16_t Ks[BN * KSTR];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VSTR];

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
    const int cmin = lim_of[t0];
    const int cmax = lim_of[t1 - 1];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r32 = lane & 31, hf = lane >> 5;
    const int rho = w * 32 + r32;                    // this lane's (target, head) row
    const int tl = rho / a.G, hh = rho - tl * a.G;
    const int t = t0 + tl;
    const bool valid = tl < a.BT && t < t1;
    const int lim = valid ? lim_of[t] : cmax;        // padding rows: finite, never stored
    const int head = g * a.G + hh;

    const uint16_t* qn = (const uint16_t*)a.q_new;
    bf16x8 qf[KS];
    {
        const uint16_t* qrow = qn + ((size_t)(valid ? t : t0) * a.H + (valid ? head : 0)) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8*)(qrow + ks * 16 + hf * 8);
    }
    const float sl2 = a.scale * kLog2e;

    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    // loader: thread -> (key group kq, 16-byte part) ; keys kq*KPT .. kq*KPT+KPT-1
    const int kq = tid / P, part = tid % P;
    const uint16_t* kn = (const uint16_t*)a.k_new;
    const uint16_t* vn = (const uint16_t*)a.v_new;
    const uint16_t* kc = (const uint16_t*)a.kc;
    const uint16_t* vc = (const uint16_t*)a.vc;
    u32x4 kr[KPT], vr[KPT];

    auto load_tile = [&](int c0) {
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk) {
            const int c = c0 + kq * KPT + kk;
            if (c <= cmax) {
                bool fresh;
                const size_t row = kv_row<FULL>(a, c, g, fresh);
                const uint16_t* kb = fresh ? kn : kc;
                const uint16_t* vb = fresh ? vn : vc;
                kr[kk] = *(const u32x4*)(kb + row * D + part * 8);
                vr[kk] = *(const u32x4*)(vb + row * D + part * 8);
            } else {
                kr[kk] = u32x4{0u, 0u, 0u, 0u};
                vr[kk] = u32x4{0u, 0u, 0u, 0u};
            }
        }
    };

    const int nkt = cmax / BN + 1;
    load_tile(0);
    for (int kt = 0; kt < nkt; ++kt) {
        const int c0 = kt * BN;
        __syncthreads();                              // previous tile fully consumed
#pragma unroll
        for (int kk = 0; kk < KPT; ++kk)
            *(u32x4*)(Ks + (kq * KPT + kk) * KSTR + part * 8) = kr[kk];
        // V transposed: Vt[d][key]; this thread holds KPT keys x 8 d values.
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sh = (e & 1) * 16;
            const int wd = e >> 1;
            if constexpr (KPT == 4) {
                const uint32_t lo = ((vr[0][wd] >> sh) & 0xffffu) | (((vr[1][wd] >> sh) & 0xffffu) << 16);
                const uint32_t hi = ((vr[2][wd] >> sh) & 0xffffu) | (((vr[3][wd] >> sh) & 0xffffu) << 16);
                *(u32x2*)(Vt + (part * 8 + e) * VSTR + kq * KPT) = u32x2{lo, hi};
            } else {
                const uint32_t lo = ((vr[0][wd] >> sh) & 0xffffu) | (((vr[1][wd] >> sh) & 0xffffu) << 16);
                *(uint32_t*)(Vt + (part * 8 + e) * VSTR + kq * KPT) = lo;
            }
        }
        __syncthreads();
        if (kt + 1 < nkt) load_tile(c0 + BN);

        // S^T = K Q^T for two 32-key blocks
        f32x16 s0 = {}, s1 = {};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 k0 = *(const bf16x8*)(Ks + r32 * KSTR + ks * 16 + hf * 8);
            const bf16x8 k1 = *(const bf16x8*)(Ks + (32 + r32) * KSTR + ks * 16 + hf * 8);
            s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[ks], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[ks], s1, 0, 0, 0);
        }
        // s_kb[v] = S[row][key c0 + kb*32 + 8(v/4) + 4hf + v%4], in log2 units below
        const bool masked = c0 + BN - 1 > cmin;
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int kc0 = c0 + 8 * (v >> 2) + 4 * hf + (v & 3);
            float x0 = s0[v] * sl2, x1 = s1[v] * sl2;
            if (masked) {
                if (kc0 > lim) x0 = -INFINITY;
                if (kc0 + 32 > lim) x1 = -INFINITY;
            }
            s0[v] = x0;
            s1[v] = x1;
            mx = fmaxf(mx, fmaxf(x0, x1));
        }
        mx = fmaxf(mx, swap_half(mx));
        const float m_new = fmaxf(m_run, mx);        // finite: key 0 is in every row's context
        const float alpha = fast_exp2(m_run - m_new);
        float ls = 0.f;
        bf16x8 pb[2][2];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const float p0 = fast_exp2(s0[v] - m_new);
            const float p1 = fast_exp2(s1[v] - m_new);
            ls += p0 + p1;
            pb[0][v >> 3][v & 7] = (__bf16)p0;
            pb[1][v >> 3][v & 7] = (__bf16)p1;
        }
        l_run = l_run * alpha + ls;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;

        // O^T += V^T P^T ; k-index hf*8+e of step (kb, k2) is key
        // kb*32 + k2*16 + 8(e/4) + 4hf + e%4, matching the S^T lane layout.
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const uint16_t* vrow = Vt + (db * 32 + r32) * VSTR;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const int ko = kb * 32 + k2 * 16 + 4 * hf;
                    const bf16x4 va = *(const bf16x4*)(vrow + ko);
                    const bf16x4 vb = *(const bf16x4*)(vrow + ko + 8);
                    const bf16x8 vv = {va[0], va[1], va[2], va[3], vb[0], vb[1], vb[2], vb[3]};
                    o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pb[kb][k2], o[db], 0, 0, 0);
                }
            }
        }
    }

    const float l_tot = l_run + swap_half(l_run);
    if (!valid) return;
    const float inv = 1.0f / l_tot;
    uint16_t* out = (uint16_t*)a.out + ((size_t)t * a.H + head) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int d0 = db * 32 + 8 * j + 4 * hf;
            const uint32_t lo = (uint32_t)f32_to_bf16_bits(o[db][4 * j] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * j + 1] * inv) << 16);
            const uint32_t hi = (uint32_t)f32_to_bf16_bits(o[db][4 * j + 2] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * j + 3] * inv) << 16);
            *(u32x2*)(out + d0) = u32x2{lo, hi};
        }
    }
    if (a.lse && hf == 0) a.lse[(size_t)t * a.H + head] = (m_run + __log2f(l_tot)) * kLn2;
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

template <int D, bool FULL>
void launch_one(const AttnArgs& a, bool bf16, int n_bound, hipStream_t st) {
    if (bf16) {
        const int ntiles = (n_bound + a.BT - 1) / a.BT;
        hipLaunchKernelGGL((attn_bf16<D, FULL>), dim3(ntiles * a.Hkv), dim3(256), 0, st, a);
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
    a.U = s.U;
    a.cidx = s.cidx;
    a.src_l = s.src + (size_t)layer * p.T_c;
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
    a.BT = kAttnRows / a.G;
    a.scale = p.softmax_scale > 0.f ? p.softmax_scale : 1.0f / sqrtf((float)p.d);
    // |R_l| <= |union of S_l' for l' >= l| <= min(T_c, (L - l) k); the device
    // count decides which workgroups run.
    const long kb = (long)(p.L - layer) * s.k;
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
