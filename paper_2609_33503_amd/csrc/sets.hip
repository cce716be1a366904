// Repair schedule and compact context (Sec. 3.2 set equations, App. A.1-A.2):
//   h_i = max{l : i in S_l},  U = union_l S_l (sorted),  R_l = {i in U : h_i >= l},
// the compact index of every union position, the per-layer source map
// (rank within R_l, or -1 for a cached row), the CSR lists of R_l and the
// edge counts sum_{p in R_l} |C_l(p)| and sum_{p in R_l} (p + 1).
//
// Four launches: reset h; integer atomicMax of each anchor's layer into h;
// one workgroup that compacts U in position order and counts |R_l| from the
// histogram of h; one workgroup per layer that compacts R_l out of U.  All
// compactions are block prefix scans, so every output is deterministic.
//
// Matched-target variants (RelaxKV^G, Sec. 4.1 / App. A.3; the global target
// sweep of App. B): U is built the same way from the anchors, then every layer
// takes the same caller-given target list P.  A prefix maximum of the compact
// map gives each target its compact limit |U cap {j <= p}| - 1 without any
// search; targets need not lie in U.
//
// Context-construction variants (Sec. 4.4): the same anchors and targets R_l;
// the context list of a layer is replaced by a top-|U| list (of the layer-mean
// score, shared, or of the layer's score), written to ctx; the compact limits,
// source map and edge counts are recomputed against it.

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

constexpr int kSetThreads = 1024;
constexpr int kSetPerThread = 8;

__global__ void sets_reset(int32_t* __restrict__ h, int T, int32_t* __restrict__ rank, long n_rank,
                           uint32_t* __restrict__ tiles, int n_tiles) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < T; i += gridDim.x * blockDim.x)
        h[i] = -1;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_tiles; i += gridDim.x * blockDim.x)
        tiles[i] = 0u;
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_rank;
         i += (long)gridDim.x * blockDim.x)
        rank[i] = -1;
}

__global__ void sets_mark(const int32_t* __restrict__ anchors, int L, int k, int T,
                          int32_t* __restrict__ h) {
    const long n = (long)L * k;
    for (long j = blockIdx.x * (long)blockDim.x + threadIdx.x; j < n;
         j += (long)gridDim.x * blockDim.x) {
        const int pos = anchors[j];
        if (pos >= 0 && pos < T) atomicMax(&h[pos], (int)(j / k));
    }
}

// Single workgroup: U, cidx, |U|, |R_l| and R_off.
__global__ __launch_bounds__(kSetThreads) void sets_union(const int32_t* __restrict__ h, int T,
                                                          int L, int32_t* __restrict__ U,
                                                          int32_t* __restrict__ cidx,
                                                          int32_t* __restrict__ R_off,
                                                          int32_t* __restrict__ counts) {
    __shared__ int hist[RELAXKV_MAX_LAYERS];
    __shared__ int scan_scratch[kSetThreads / 64];
    const int tid = threadIdx.x;
    for (int l = tid; l < L; l += kSetThreads) hist[l] = 0;
    __syncthreads();

    int c_base = 0;
    for (int base = 0; base < T; base += kSetThreads * kSetPerThread) {
        const int i0 = base + tid * kSetPerThread;
        int hv[kSetPerThread];
        int n = 0;
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e) {
            const int i = i0 + e;
            hv[e] = i < T ? h[i] : -1;
            n += hv[e] >= 0;
        }
        int tot;
        int c = block_exclusive_scan<kSetThreads>(n, scan_scratch, tot) + c_base;
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e) {
            const int i = i0 + e;
            if (i >= T) break;
            if (hv[e] >= 0) {
                U[c] = i;
                cidx[i] = c;
                ++c;
                atomicAdd(&hist[hv[e]], 1);
            } else {
                cidx[i] = -1;
            }
        }
        c_base += tot;
    }
    __syncthreads();

    // |R_l| = #{i : h_i >= l}: suffix sums of the histogram, then R_off is the
    // exclusive prefix of |R_l| over layers.  L <= 1024 = one layer per thread.
    const int rl = tid < L ? hist[L - 1 - tid] : 0;
    int tot1;
    const int sfx = block_exclusive_scan<kSetThreads>(rl, scan_scratch, tot1) + rl;  // layer L-1-tid
    __syncthreads();
    if (tid < L) hist[L - 1 - tid] = sfx;     // hist[l] now holds |R_l|
    __syncthreads();
    const int nr = tid < L ? hist[tid] : 0;
    int tot2;
    const int off = block_exclusive_scan<kSetThreads>(nr, scan_scratch, tot2);
    if (tid < L) {
        R_off[tid] = off;
        counts[1 + tid] = nr;
    }
    if (tid == 0) {
        R_off[L] = tot2;
        counts[0] = c_base;
    }
}

// One workgroup per layer: R_l in position order, its compact indices, the
// source map and the edge counts.
__global__ __launch_bounds__(kSetThreads) void sets_layers(
    const int32_t* __restrict__ h, const int32_t* __restrict__ U, int T,
    const int32_t* __restrict__ R_off, const int32_t* __restrict__ counts,
    int32_t* __restrict__ R_idx, int32_t* __restrict__ R_u, int32_t* __restrict__ src,
    int32_t* __restrict__ rank, int64_t* __restrict__ edges, int L) {
    __shared__ int scan_scratch[kSetThreads / 64];
    __shared__ long long red[2][kSetThreads / 64];
    const int l = blockIdx.x;
    const int tid = threadIdx.x;
    const int nU = counts[0];
    const int off = R_off[l];
    int32_t* src_l = src + (size_t)l * T;
    int32_t* rank_l = rank + (size_t)l * T;
    long long e_sum = 0, ef_sum = 0;
    int r_base = 0;
    for (int base = 0; base < nU; base += kSetThreads * kSetPerThread) {
        const int c0 = base + tid * kSetPerThread;
        int pos[kSetPerThread];
        bool act[kSetPerThread];
        int n = 0;
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e) {
            const int c = c0 + e;
            pos[e] = c < nU ? U[c] : 0;
            act[e] = c < nU && h[pos[e]] >= l;
            n += act[e];
        }
        int tot;
        int r = block_exclusive_scan<kSetThreads>(n, scan_scratch, tot) + r_base;
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e) {
            const int c = c0 + e;
            if (c >= nU) break;
            if (act[e]) {
                R_idx[off + r] = pos[e];
                R_u[off + r] = c;
                src_l[c] = r;
                rank_l[pos[e]] = r;
                ++r;
                e_sum += c + 1;          // |C_l(p)| = compact index of p + 1
                ef_sum += pos[e] + 1;    // full causal prefix
            } else {
                src_l[c] = -1;
            }
        }
        r_base += tot;
    }
    e_sum = wave_sum(e_sum);
    ef_sum = wave_sum(ef_sum);
    const int lane = tid & 63, w = tid >> 6;
    if (lane == 0) {
        red[0][w] = e_sum;
        red[1][w] = ef_sum;
    }
    __syncthreads();
    if (tid == 0) {
        long long a = 0, b = 0;
        for (int i = 0; i < kSetThreads / 64; ++i) {
            a += red[0][i];
            b += red[1][i];
        }
        edges[l] = a;
        edges[L + l] = b;
    }
}

// ------------------------------------------------------ global target lists

__device__ __forceinline__ int wave_inclusive_max(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x = max(x, y);
    }
    return x;
}

// Single workgroup.  last[i] = max_{j <= i} cidx[j] = |U cap {j <= i}| - 1
// (written into h, which the last launch overwrites); checks the target list;
// |R_l| = |P| and R_off for every layer.
__global__ __launch_bounds__(kSetThreads) void gt_prefix(const int32_t* __restrict__ cidx, int T,
                                                         int L, const int32_t* __restrict__ P,
                                                         const int32_t* __restrict__ n_P,
                                                         int32_t* __restrict__ last,
                                                         int32_t* __restrict__ R_off,
                                                         int32_t* __restrict__ counts) {
    __shared__ int wmax[kSetThreads / 64];
    __shared__ int bad_sh;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    if (tid == 0) bad_sh = 0;
    int carry = -1;
    for (int base = 0; base < T; base += kSetThreads * kSetPerThread) {
        const int i0 = base + tid * kSetPerThread;
        int v[kSetPerThread];
        int m = -1;
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e) {
            v[e] = i0 + e < T ? cidx[i0 + e] : -1;
            m = max(m, v[e]);
            v[e] = m;                                  // running max within the thread
        }
        const int incl = wave_inclusive_max(m);
        if (lane == 63) wmax[w] = incl;
        __syncthreads();
        int before = carry;                            // max over earlier chunks and waves
        for (int ww = 0; ww < w; ++ww) before = max(before, wmax[ww]);
        int prev = __shfl_up(incl, 1, 64);             // earlier lanes of this wave
        if (lane == 0) prev = -1;
        const int excl = max(before, prev);
        int blk = carry;
        for (int ww = 0; ww < kSetThreads / 64; ++ww) blk = max(blk, wmax[ww]);
#pragma unroll
        for (int e = 0; e < kSetPerThread; ++e)
            if (i0 + e < T) last[i0 + e] = max(excl, v[e]);
        carry = blk;
        __syncthreads();
    }
    // Target list checks: 0 <= |P| <= T, strictly ascending within [0, T).
    const int n_raw = n_P[0];
    const int n = min(max(n_raw, 0), T);
    int bad = n_raw < 0 || n_raw > T;
    for (int t = tid; t < n; t += kSetThreads) {
        const int p = P[t];
        bad |= p < 0 || p >= T || (t > 0 && P[t - 1] >= p);
    }
    if (bad) bad_sh = 1;                               // benign race: every writer stores 1
    for (int l = tid; l <= L; l += kSetThreads) {
        R_off[l] = l * n;
        if (l < L) counts[1 + l] = n;
    }
    __syncthreads();
    if (tid == 0 && bad_sh) atomicOr(&counts[L + 1], 2);
}

// One workgroup per layer: R_l = P, compact limits, the rank and source maps,
// and the edge counts.
__global__ __launch_bounds__(kSetThreads) void gt_layers(
    const int32_t* __restrict__ last, const int32_t* __restrict__ U, int T,
    const int32_t* __restrict__ P, const int32_t* __restrict__ R_off,
    const int32_t* __restrict__ counts, int32_t* __restrict__ R_idx, int32_t* __restrict__ R_u,
    int32_t* __restrict__ src, int32_t* __restrict__ rank, int64_t* __restrict__ edges, int L) {
    __shared__ long long red[2][kSetThreads / 64];
    const int l = blockIdx.x, tid = threadIdx.x;
    const int nU = counts[0], n = counts[1 + l], off = R_off[l];
    int32_t* src_l = src + (size_t)l * T;
    int32_t* rank_l = rank + (size_t)l * T;
    long long e_sum = 0, ef_sum = 0;
    for (int t = tid; t < n; t += kSetThreads) {
        const int p = min(max(P[t], 0), T - 1);        // in range even for a rejected list
        const int u = last[p];
        R_idx[off + t] = p;
        R_u[off + t] = u;
        rank_l[p] = t;
        e_sum += u + 1;                                // |C_l(p)| = |U cap {j <= p}|
        ef_sum += p + 1;
    }
    __syncthreads();                                   // rank_l complete for this layer
    for (int c = tid; c < nU; c += kSetThreads) src_l[c] = rank_l[U[c]];
    e_sum = wave_sum(e_sum);
    ef_sum = wave_sum(ef_sum);
    const int lane = tid & 63, w = tid >> 6;
    if (lane == 0) {
        red[0][w] = e_sum;
        red[1][w] = ef_sum;
    }
    __syncthreads();
    if (tid == 0) {
        long long a = 0, b = 0;
        for (int i = 0; i < kSetThreads / 64; ++i) {
            a += red[0][i];
            b += red[1][i];
        }
        edges[l] = a;
        edges[L + l] = b;
    }
}

// h_i = L - 1 for targets, -1 otherwise (after gt_layers read the prefix maxima).
__global__ void gt_h(const int32_t* __restrict__ rank0, int T, int L, int32_t* __restrict__ h) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < T; i += gridDim.x * blockDim.x)
        h[i] = rank0[i] >= 0 ? L - 1 : -1;
}

// ------------------------------------------------ context-construction variants

// One workgroup per layer: compact limits of RelaxKV's targets R_l within the
// layer's context list U_l (upper bound by binary search: both are ascending),
// the source map over U_l and the edge counts.
__global__ __launch_bounds__(kSetThreads) void ctx_layers(
    const int32_t* __restrict__ ctx, int ctx_stride, int T, const int32_t* __restrict__ R_off,
    const int32_t* __restrict__ R_idx, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ rank, int32_t* __restrict__ R_u, int32_t* __restrict__ src,
    int64_t* __restrict__ edges) {
    __shared__ long long red[kSetThreads / 64];
    const int l = blockIdx.x, tid = threadIdx.x;
    const int32_t* ctx_l = ctx + (size_t)l * ctx_stride;
    const int n = counts[0];                           // every context list has |U| entries
    const int off = R_off[l], nR = counts[1 + l];
    const int32_t* rank_l = rank + (size_t)l * T;
    int32_t* src_l = src + (size_t)l * T;
    long long e_sum = 0;
    for (int t = tid; t < nR; t += kSetThreads) {
        const int p = R_idx[off + t];
        int lo = 0, hi = n;                            // first entry > p
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (ctx_l[mid] <= p) lo = mid + 1;
            else hi = mid;
        }
        R_u[off + t] = lo - 1;
        e_sum += lo;                                   // |U_l cap {j <= p}|
    }
    for (int c = tid; c < n; c += kSetThreads) src_l[c] = rank_l[ctx_l[c]];
    e_sum = wave_sum(e_sum);
    if ((tid & 63) == 0) red[tid >> 6] = e_sum;
    __syncthreads();
    if (tid == 0) {
        long long a = 0;
        for (int i = 0; i < kSetThreads / 64; ++i) a += red[i];
        edges[l] = a;
    }
}

void launch_union(const relaxkv_problem& p, const relaxkv_sets& s, hipStream_t st) {
    const int T = p.T_c, L = p.L;
    const long n_rank = (long)L * T;
    const long rb = (n_rank + 255) / 256;
    hipLaunchKernelGGL(sets_reset, dim3(rb < 2048 ? (int)rb : 2048), dim3(256), 0, st, s.h, T,
                       s.rank, n_rank, s.tiles, (int)attn_tile_words(p));
    const long nm = (long)L * s.k;
    const long mb = (nm + 255) / 256;
    hipLaunchKernelGGL(sets_mark, dim3(mb < 2048 ? (int)mb : 2048), dim3(256), 0, st, s.anchors,
                       L, s.k, T, s.h);
    hipLaunchKernelGGL(sets_union, dim3(1), dim3(kSetThreads), 0, st, s.h, T, L, s.U, s.cidx,
                       s.R_off, s.counts);
}

}  // namespace

hipError_t launch_build_sets_context(const relaxkv_problem& p, const float* scores,
                                     int construction, const relaxkv_sets& s, hipStream_t st) {
    const int T = p.T_c, L = p.L;
    hipError_t e = launch_build_sets(p, s, st);       // anchors -> h, U, R_l, rank (+ union maps)
    if (e != hipSuccess || construction == RELAXKV_CONTEXT_SETS_UNION) return e;
    // Top-|U| context lists, ascending (the k cap |U| is read on the device).
    if (construction == RELAXKV_CONTEXT_SETS_GLOBAL) {
        e = launch_global_mean(scores, L, T, s.g, st);
        if (e == hipSuccess) e = launch_select_rows(s.g, 1, T, T, s.counts, s.ctx, 0, s.counts, L, st);
    } else {
        e = launch_select_rows(scores, L, T, T, s.counts, s.ctx, T, s.counts, L, st);
    }
    if (e != hipSuccess) return e;
    const int stride = construction == RELAXKV_CONTEXT_SETS_GLOBAL ? 0 : T;
    hipLaunchKernelGGL(ctx_layers, dim3(L), dim3(kSetThreads), 0, st, (const int32_t*)s.ctx, stride,
                       T, s.R_off, s.R_idx, s.counts, s.rank, s.R_u, s.src, s.edges);
    return hipGetLastError();
}

hipError_t launch_build_sets_global(const relaxkv_problem& p, const relaxkv_sets& s,
                                    const int32_t* targets, const int32_t* n_targets,
                                    hipStream_t st) {
    const int T = p.T_c, L = p.L;
    launch_union(p, s, st);
    hipLaunchKernelGGL(gt_prefix, dim3(1), dim3(kSetThreads), 0, st, s.cidx, T, L, targets,
                       n_targets, s.h, s.R_off, s.counts);
    hipLaunchKernelGGL(gt_layers, dim3(L), dim3(kSetThreads), 0, st, (const int32_t*)s.h, s.U, T,
                       targets, s.R_off, s.counts, s.R_idx, s.R_u, s.src, s.rank, s.edges, L);
    const int hb = (T + 255) / 256;
    hipLaunchKernelGGL(gt_h, dim3(hb < 2048 ? hb : 2048), dim3(256), 0, st, (const int32_t*)s.rank,
                       T, L, s.h);
    return hipGetLastError();
}

hipError_t launch_build_sets(const relaxkv_problem& p, const relaxkv_sets& s, hipStream_t st) {
    const int T = p.T_c, L = p.L;
    launch_union(p, s, st);
    hipLaunchKernelGGL(sets_layers, dim3(L), dim3(kSetThreads), 0, st, s.h, s.U, T, s.R_off,
                       s.counts, s.R_idx, s.R_u, s.src, s.rank, s.edges, L);
    return hipGetLastError();
}

}  // namespace relaxkv
