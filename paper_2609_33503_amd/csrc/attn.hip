// Sparse-context causal attention (Sec. 3.3-3.4, App. A.2; the attention step of
// Algorithm 1).  Target t of layer l (position p, compact index u_t in U)
// attends to the compact context c = 0 .. u_t (C_l(p) = U cap {j <= p}) or, for
// the Full-Prefix Control, to positions j = 0 .. p.  Key/value row j is the
// fresh row of j when j is in R_l (src[l][c] >= 0) and the naive cached row
// otherwise.
//
// bf16 kernel (bf16 MFMA 32x32x16, fp32 accumulation, flash-style online
// softmax in the exp2 domain):
// - a workgroup of NW = 12 waves owns NW*32 consecutive (target, head) rows of
//   one KV head g (row t*G + hh: target t, the hh-th of the G query heads that
//   share g), so every K/V row brought into LDS is used by NW*32 rows; a tile
//   may begin or end inside a target's group of heads, so no row is idle when
//   G does not divide NW*32;
// - context keys go in steps of 64 through a 4-deep ring of LDS buffers (a K
//   and a V tile per step, unpadded rows with an XOR swizzle), filled by direct
//   global->LDS loads that choose per key between the fresh rows
//   (k_new/v_new) and the cached layer; the keys' indices (U and src, or rank)
//   are staged into LDS the same way one step earlier, so the only vector
//   loads in flight are LDS fills, waited for by in-order counts;
// - each wave computes S^T = K Q^T with one query row per lane (Q stays in
//   registers), so row max and row sum are lane-local plus one exchange with
//   the lane 32 away; P^T stays in registers as the B operand of
//   O^T = V^T P^T, whose V^T operand comes from transposing LDS reads;
// - the mask is the staircase of the targets' limits: steps below the first
//   target's limit run unmasked, the rest compare each key with its row's limit,
//   and a wave skips the arithmetic of steps past all of its rows' limits;
// - tiles are taken heaviest-first (the last targets have the longest
//   contexts) from per-KV-head counters; a workgroup starts with the head tied
//   to its XCD, so the workgroups of one XCD share a KV head and its L2
//   working set, and takes the next head's tiles once its own are gone (the
//   XCDs run at different clocks, and a fixed map would wait for the slowest).
// fp32 kernel: one wave per (target, head), VALU dot products and an online
// softmax across the wave; used for fp32 inputs, where bf16 MFMA would not meet
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
    const void* kc;          // layer base: row i of KV head g at element g * kv_sh + i * kv_st
    const void* vc;
    const int32_t* U;
    const int32_t* cidx;
    const int32_t* src_l;    // src + layer * T
    const int32_t* rank_l;   // rank + layer * T
    const int32_t* R_off;
    const int32_t* R_idx;
    const int32_t* R_u;
    const int32_t* counts;
    int32_t* err;            // the error word counts[L+1]
    uint32_t* tiles;         // this layer's and mode's work counters: [Hkv] next tile, [Hkv] workgroups
    void* out;
    float* lse;
    int64_t kv_sh, kv_st;    // element strides of the cache's KV heads and tokens
    int H, Hkv, G, T, layer;
    int cap;                 // rows this launch may process (row capacity, host bound)
    float scale;             // softmax scale (natural units)
};

// Row of key index c for KV head g: returns the element offset of that row in
// either the fresh tensor (fresh = true) or the cached layer.
template <int D, bool FULL>
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
    return fresh ? ((size_t)r * a.Hkv + g) * D : (size_t)(g * a.kv_sh + pos * a.kv_st);
}

// ----------------------------------------------------------------- bf16 MFMA

constexpr float kRescaleSlack = 8.0f;      // log2 units the running max may lag the true max
constexpr int kXcds = 8;                   // XCDs of an MI355X (workgroup i runs on XCD i mod 8)
constexpr int kHwRegXccId = 20;            // hardware register holding the wave's XCD index

typedef short v4i16 __attribute__((ext_vector_type(4)));
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

// NW waves of 32 rows, 64-key steps, one barrier per step.  The fills of step
// j+3 and the indices of step j+4 are issued right after the barrier of step j,
// so every fill has two steps of compute to land.
template <int D, bool FULL, int NW>
__global__ __launch_bounds__(NW * 64, 1) void attn_bf16(AttnArgs a) {
    constexpr int TK = 64, NST = 4;
    constexpr int KS = D / 16;             // k-steps of the QK^T contraction
    constexpr int DB = D / 32;             // 32-wide d blocks of O^T
    constexpr int ROWB = 2 * D;            // tile row bytes
    constexpr int CH = D / 8;              // 16-byte chunks per row
    constexpr int RPI = 64 / CH;           // rows per wave-wide load
    constexpr int NL = TK / RPI;           // wave-wide loads per step and tensor
    constexpr int PPW = (NL + NW - 1) / NW;   // K/V load pairs of the busiest wave
    constexpr int NWAIT = 2 * PPW;         // its fills per step
    constexpr int NWAIT_TAIL = 2 * (NL / NW);  // fills per step of the least busy wave
    __shared__ __attribute__((aligned(1024))) uint16_t Kt[NST][TK * D];
    __shared__ __attribute__((aligned(1024))) uint16_t Vt[NST][TK * D];
    __shared__ __attribute__((aligned(256))) int32_t Ix[NST][2][TK];   // [U or rank, src]

    __shared__ int s_pick;

    const int Hkv = a.Hkv;
    const int nR_dev = a.counts[1 + a.layer];
    const int nR = min(nR_dev, a.cap);
    if (nR_dev > a.cap && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(a.err, RELAXKV_ERR_ROWS);
    constexpr int TR = NW * 32;            // (target, head) rows per tile
    const int nrows = nR * a.G;            // rows of one KV head (< 2^31: T_c <= 2^22, G <= TR)
    const int ntiles = (nrows + TR - 1) / TR;
    // Tile choice.  Each KV head's tiles are handed out heaviest first from its
    // counter; a workgroup starts with a head tied to its XCD (so the
    // workgroups of one XCD share that head's K/V in their L2) and moves on to
    // the next head once that one is exhausted.  The XCDs run at different
    // clocks, so a fixed blockIdx -> tile map would make every launch wait for
    // the slowest; the grid carries spare workgroups for the faster ones.  The
    // last workgroup to take its pick returns the counters to zero for the
    // next launch of this layer and mode.
    if (threadIdx.x == 0) {
        const int xcc = (int)__builtin_amdgcn_s_getreg(kHwRegXccId | ((4 - 1) << 11));
        int h = (xcc + kXcds * (int)((blockIdx.x / kXcds) % ((Hkv + kXcds - 1) / kXcds))) % Hkv;
        int pick = -1;
        for (int tried = 0; tried < Hkv; ++tried) {
            const int t = (int)atomicAdd(a.tiles + h, 1u);
            if (t < ntiles) {
                pick = t * Hkv + h;
                break;
            }
            h = h + 1 == Hkv ? 0 : h + 1;
        }
        s_pick = pick;
        __threadfence();
        if (atomicAdd(a.tiles + Hkv, 1u) == gridDim.x - 1) {
            __threadfence();                       // every other pick happens before the resets
            for (int i = 0; i < Hkv; ++i) atomicExch(a.tiles + i, 0u);
            atomicExch(a.tiles + Hkv, 0u);
        }
    }
    __syncthreads();
    const int pick = s_pick;
    if (pick < 0) return;
    const int g = pick % Hkv;
    const int tile = ntiles - 1 - pick / Hkv;        // heaviest tiles first
    const int r0 = tile * TR;                        // the tile's rows [r0, r1)
    const int r1 = min(r0 + TR, nrows);
    const int t0 = r0 / a.G, t1 = (r1 - 1) / a.G + 1;  // the targets they belong to
    const int off = a.R_off[a.layer];
    const int32_t* lim_of = FULL ? a.R_idx + off : a.R_u + off;
    const int cmin = lim_of[t0];
    const int cmax = max(lim_of[t1 - 1], 0);

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r32 = lane & 31, hf = lane >> 5;
    const float sl2 = a.scale * kLog2e;

    const int row = r0 + w * 32 + r32;
    const bool valid = row < r1;
    const int t_row = valid ? row / a.G : t0;
    const int hh = valid ? row - t_row * a.G : 0;
    const int lim_v = lim_of[t_row];                 // value select: no pointer to cmax
    const int lim = valid ? lim_v : cmax;
    // The largest limit among the wave's rows (limits ascend with the row), -1
    // for a wave without rows: steps past it are masked for every row of the wave.
    const int w_first = r0 + w * 32, w_last = min(w_first + 31, r1 - 1);
    const int wlim = __builtin_amdgcn_readfirstlane(w_last < w_first ? -1 : lim_of[w_last / a.G]);
    const int head = g * a.G + hh;
    bf16x8 qf[KS];
    {
        const uint16_t* qrow = (const uint16_t*)a.q_new + ((size_t)t_row * a.H + head) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8*)(qrow + ks * 16 + hf * 8);
        // Consumed here, so the compiler's waits for these loads stay before the
        // loop: inside it they would also wait for the K/V fills just issued.
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(qf[ks]));
    }
    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x16{};
    float m_run = lim < 0 ? 0.f : -INFINITY;       // empty context: every p is exp2(-inf) = 0
    float l_run = 0.f;

    // Row bases of the fresh rows (stride Hkv*D) and of the cached layer (stride D).
    const uint16_t* kng = (const uint16_t*)a.k_new + (size_t)g * D;
    const uint16_t* vng = (const uint16_t*)a.v_new + (size_t)g * D;
    const uint16_t* kcg = (const uint16_t*)a.kc + g * a.kv_sh;
    const uint16_t* vcg = (const uint16_t*)a.vc + g * a.kv_sh;
    const uint32_t kst = (uint32_t)a.kv_st;              // < 2^24 (checked on the host)
    const int32_t* srcmap = FULL ? a.rank_l : a.src_l;
    const int S = cmax / TK + 1;                     // 64-key steps

    auto issue_idx = [&](int m) {
        if (w < (FULL ? 1 : 2)) {
            int ww = w;
            asm volatile("" : "+s"(ww));
            const int c = min(m * TK + lane, cmax);
            const int32_t* src = FULL ? srcmap + c : (ww == 0 ? a.U + c : srcmap + c);
            fill_lds4(src, lds_addr(&Ix[m & 3][ww][0]));
        }
    };
    // The lane's tile row and swizzled chunk offset (elements) in each of its
    // fills: loop invariant.
    int f_row[PPW];
    uint32_t f_choff[PPW];
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        f_row[i] = (w + i * NW) * RPI + lane / CH;
        f_choff[i] = (uint32_t)(((lane % CH) ^ tile_swz<D>(f_row[i])) << 3);
    }
    auto issue_rows = [&](int m) {
        const int st = m & 3;
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const int j = w + i * NW;
            if (NL % NW == 0 || j < NL) {
                int row = f_row[i];
                uint32_t choff = f_choff[i];
                asm volatile("" : "+v"(row), "+v"(choff));
                const int c = m * TK + row;
                int pos = FULL ? min(c, cmax) : Ix[st][0][row];
                int r = Ix[st][FULL ? 0 : 1][row];
                asm volatile("" : "+v"(pos), "+v"(r));      // both read, then selected
                // (the empty asm statements keep the compiler from turning the
                // fresh/cached choice into a divergent branch)
                const bool fresh = r >= 0;
                // element offset of the row's chunk (< 2^31: (T_c - 1) * kst + D and
                // |R_l| * Hkv * D, both checked on the host, so 24-bit multiplies do)
                const uint32_t off = (fresh ? __umul24((uint32_t)r, (uint32_t)(Hkv * D))
                                            : __umul24((uint32_t)pos, kst)) + choff;
                const uint64_t kb = fresh ? (uint64_t)kng : (uint64_t)kcg;
                const uint64_t vb = fresh ? (uint64_t)vng : (uint64_t)vcg;
                const uint16_t* kp = (const uint16_t*)kb + off;
                const uint16_t* vp = (const uint16_t*)vb + off;
                fill_lds16(kp, lds_addr(Kt[st] + j * RPI * D));
                fill_lds16(vp, lds_addr(Vt[st] + j * RPI * D));
            }
        }
    };

    const int k_base = r32 * ROWB | ((hf ^ tile_swz<D>(r32)) << 4);
    const int rl = 4 * (lane >> 5) + ((lane & 15) >> 2);
    const int cl = ((lane >> 4) & 1) * 2 + ((lane & 3) >> 1);
    const int v_base0 = rl * ROWB | ((cl ^ tile_swz<D>(rl)) << 4) | ((lane & 1) << 3);
    const int v_base1 = (rl + 8) * ROWB | ((cl ^ tile_swz<D>(rl + 8)) << 4) | ((lane & 1) << 3);

#pragma unroll
    for (int m = 0; m < NST; ++m)
        if (m < S) issue_idx(m);
    wait_loads_barrier<0>();
#pragma unroll
    for (int m = 0; m < NST - 1; ++m)
        if (m < S) issue_rows(m);

    for (int j = 0; j < S; ++j) {
        // The fills of step j and the indices of step j+3 are complete (only the
        // fills of step j+2 may be in flight), and every wave is done with step
        // j-1, whose buffers the fills of step j+3 reuse.  Loads complete in
        // order, so a wave's fills of step j are done once at most as many of
        // its loads are outstanding as it issued after them: the fills of steps
        // j+1 and j+2 (at least NWAIT loads while both steps exist), only those
        // of step j+1 near the end (at least NWAIT_TAIL), none in the last step.
        if (j + 2 < S) wait_loads_barrier<NWAIT>();
        else if (j + 1 < S) wait_loads_barrier<NWAIT_TAIL>();
        else wait_loads_barrier<0>();
        if (j + NST < S) issue_idx(j + NST);
        if (j + NST - 1 < S) issue_rows(j + NST - 1);
        // A step whose keys all lie past every limit of the wave's rows adds
        // exact zeros to them (p = 0): the wave only keeps the ring moving.
        if (j * TK > wlim) continue;
        // S^T = K Q^T: s[kb][v] = S[row][key 64 j + 32 kb + 8(v/4) + 4 hf + v%4]
        f32x16 s[2];
        {
            int kbo = k_base + (j & 3) * (TK * D * 2);    // the stage offset leaves the swizzled bits alone
            asm volatile("" : "+v"(kbo));
            const char* kst = (const char*)Kt[0];
            s[0] = s[1] = f32x16{};
            // K fragments x = 2 ks + kb, read KA ahead of their MFMA.
            constexpr int KA = RELAXKV_ATTN_KAHEAD < 2 * KS ? RELAXKV_ATTN_KAHEAD : 2 * KS;
            auto frag = [&](int x) {
                return *(const bf16x8*)(kst + (x & 1) * 32 * ROWB + (kbo ^ ((x >> 1) << 5)));
            };
            bf16x8 kf[KA];
#pragma unroll
            for (int x = 0; x < KA; ++x) kf[x] = frag(x);
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(2);
#endif
#pragma unroll
            for (int x = 0; x < 2 * KS; ++x) {
                const bf16x8 cur = kf[x % KA];
                if (x + KA < 2 * KS) kf[x % KA] = frag(x + KA);
                s[x & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur, qf[x >> 1], s[x & 1], 0, 0, 0);
            }
#if RELAXKV_ATTN_SCHED
            __builtin_amdgcn_sched_group_barrier(0x100, KA, 0);
#pragma unroll
            for (int x = 0; x < 2 * KS; ++x) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (x + KA < 2 * KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
#endif
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(0);
#endif
        }
        const int c0 = j * TK;
        if (c0 + TK - 1 > cmin) {                      // staircase step: mask
            const int ex = lim - c0 - 4 * hf;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                if (8 * (v >> 2) + (v & 3) > ex) s[0][v] = -INFINITY;
                if (32 + 8 * (v >> 2) + (v & 3) > ex) s[1][v] = -INFINITY;
            }
        }
#if RELAXKV_ATTN_LEAN
        // Two chains of 3-input maxima (two new values per instruction).
        float m0 = fmaxf(s[0][0], s[0][1]), m1 = fmaxf(s[1][0], s[1][1]);
#pragma unroll
        for (int v = 2; v < 16; v += 2) {
            m0 = fmaxf(fmaxf(m0, s[0][v]), s[0][v + 1]);
            m1 = fmaxf(fmaxf(m1, s[1][v]), s[1][v + 1]);
        }
        const float mx = pair_max(fmaxf(m0, m1)) * sl2;
#else
        float m = fmaxf(s[0][0], s[1][0]);
#pragma unroll
        for (int v = 1; v < 16; ++v) m = fmaxf(m, fmaxf(s[0][v], s[1][v]));
        const float mx = pair_max(m) * sl2;
#endif
        const bool need = mx > m_run + kRescaleSlack;
        if (__any(need)) {
            const float m_new = need ? mx : m_run;
            const float alpha = fast_exp2(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[db] *= alpha;
            m_run = m_new;
        }
        bf16x8 pb[2][2];
#if RELAXKV_ATTN_LEAN
        // The row sum adds the bf16 probabilities that the PV product uses, two
        // per dot2 instruction, in four chains.
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                pb[kb][v >> 3][v & 7] = (__bf16)fast_exp2(fmaf(s[kb][v], sl2, -m_run));
        {
            typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
            const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
            float ls0 = 0.f, ls1 = 0.f, ls2 = 0.f, ls3 = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
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
#else
        float ls = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = fast_exp2(fmaf(s[kb][v], sl2, -m_run));
                ls += p;
                pb[kb][v >> 3][v & 7] = (__bf16)p;
            }
        l_run += ls;
#endif
        // O^T += V^T P^T
        {
            // LDS byte addresses of the lane's two V rows in this step's tile: the
            // tile base and stage only set bits above the swizzled chunk bits.
            const uint32_t vstage = lds_addr(Vt[0]) + (uint32_t)(j & 3) * (TK * D * 2);
            uint32_t vb0 = v_base0 + vstage, vb1 = v_base1 + vstage;
            asm volatile("" : "+v"(vb0), "+v"(vb1));
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(2);
#endif
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int k2 = 0; k2 < 2; ++k2) {
                        const uint32_t rowo = (kb * 32 + k2 * 16) * ROWB;
                        const v4i16 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_v4i16*)(uintptr_t)((vb0 ^ (db << 6)) + rowo));
                        const v4i16 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_v4i16*)(uintptr_t)((vb1 ^ (db << 6)) + rowo));
                        const bf16x8 vv =
                            __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
                        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pb[kb][k2], o[db], 0, 0, 0);
                    }
#if RELAXKV_ATTN_SETPRIO
            __builtin_amdgcn_s_setprio(0);
#endif
        }
    }

    const float l_tot = pair_sum(l_run);
    if (!valid) return;
    const bool empty = lim < 0;
    const float inv = empty ? 0.f : 1.0f / l_tot;
    // (t, head) row index: below T_c * H <= 2^32, and one register where a 64-bit
    // product held across the loop would take two
    const uint32_t orow = (uint32_t)t_row * (uint32_t)a.H + (uint32_t)head;
    uint16_t* out = (uint16_t*)a.out + (size_t)orow * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int d0 = db * 32 + 8 * jj + 4 * hf;
            const uint32_t lo = (uint32_t)f32_to_bf16_bits(o[db][4 * jj] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * jj + 1] * inv) << 16);
            const uint32_t hi = (uint32_t)f32_to_bf16_bits(o[db][4 * jj + 2] * inv) |
                                ((uint32_t)f32_to_bf16_bits(o[db][4 * jj + 3] * inv) << 16);
            *(u32x2*)(out + d0) = u32x2{lo, hi};
        }
    }
    if (a.lse && hf == 0)
        a.lse[orow] = empty ? -INFINITY : (m_run + __log2f(l_tot)) * kLn2;
}


// ----------------------------------------------------------------- fp32 VALU

template <int D, bool FULL>
__global__ __launch_bounds__(64) void attn_f32(AttnArgs a) {
    constexpr int DPL = D / 64;            // d values owned per lane
    __shared__ float qs[D];
    const int t = blockIdx.x, head = blockIdx.y;
    const int nR_dev = a.counts[1 + a.layer];
    if (nR_dev > a.cap && t == 0 && head == 0 && threadIdx.x == 0) atomicOr(a.err, RELAXKV_ERR_ROWS);
    if (t >= min(nR_dev, a.cap)) return;
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
            const size_t row = kv_row<D, FULL>(a, c, g, fresh);
            const float* kr = (fresh ? kn : kc) + row;
            vrow = (fresh ? vn : vc) + row;
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
static_assert(kAttnRows == kNW * 32, "rows per workgroup");

template <int D, bool FULL>
void launch_one(const AttnArgs& a, bool bf16, int n_bound, hipStream_t st) {
    n_bound = n_bound > 0 ? n_bound : 1;                 // workgroup 0 still checks the count
    if (bf16) {
        const long rows = (long)n_bound * a.G;
        const int ntiles = (int)((rows + kAttnRows - 1) / kAttnRows);
        const int nwg = ntiles * a.Hkv;
        // One workgroup per tile of the bound plus an eighth spare (they exit
        // once every counter is exhausted).
        hipLaunchKernelGGL((attn_bf16<D, FULL, kNW>), dim3(nwg + nwg / 8), dim3(kNW * 64), 0, st, a);
    } else {
        hipLaunchKernelGGL((attn_f32<D, FULL>), dim3(n_bound, a.H), dim3(64), 0, st, a);
    }
}

}  // namespace

hipError_t launch_sparse_attn(const relaxkv_problem& p, const relaxkv_sets& s, int layer,
                              const void* q_new, const void* k_new, const void* v_new,
                              int n_rows, void* out, float* lse_out, int context_mode,
                              hipStream_t st) {
    const bool bf16 = p.dtype == RELAXKV_DTYPE_BF16;
    const size_t esz = bf16 ? 2 : 4;
    const KvStrides ks = kv_strides(p);
    AttnArgs a;
    a.q_new = q_new;
    a.k_new = k_new;
    a.v_new = v_new;
    a.kc = (const char*)p.k_cache + (size_t)(layer * ks.layer) * esz;
    a.vc = (const char*)p.v_cache + (size_t)(layer * ks.layer) * esz;
    a.kv_sh = ks.head;
    a.kv_st = ks.token;
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
    a.err = s.counts + p.L + 1;
    a.tiles = s.tiles + ((size_t)(context_mode == RELAXKV_CONTEXT_FULL ? p.L : 0) + layer) *
                            (size_t)(p.H_kv + 1);
    a.out = out;
    a.lse = lse_out;
    a.H = p.H;
    a.Hkv = p.H_kv;
    a.G = p.H / p.H_kv;
    a.T = p.T_c;
    a.layer = layer;
    a.scale = p.softmax_scale > 0.f ? p.softmax_scale : 1.0f / sqrtf((float)p.d);
    // The grid covers the row cap; the device count (clamped to it) decides
    // which workgroups run.
    a.cap = row_cap(p, s, layer, n_rows);
    const int n_bound = a.cap;
    const bool full = context_mode == RELAXKV_CONTEXT_FULL;
    if (p.d == 128) {
        full ? launch_one<128, true>(a, bf16, n_bound, st) : launch_one<128, false>(a, bf16, n_bound, st);
    } else {
        full ? launch_one<64, true>(a, bf16, n_bound, st) : launch_one<64, false>(a, bf16, n_bound, st);
    }
    return hipGetLastError();
}

}  // namespace relaxkv
