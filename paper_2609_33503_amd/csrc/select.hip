// Per-layer top-k anchor selection (Sec. 3.2 / App. A.1: S_l = TopK_i(a_{l,i}, k)),
// and the global target list of the target-capacity sweep (App. B equation:
// g_i = (1/L) sum_l a_{l,i}, P = TopK_i(g_i, min(floor(r_g T_c), |U|))), which
// runs the same selection on the single row g with the count capped on the
// device by |U|.
//
// One 1024-thread workgroup per selected row.  Scores are mapped to order-preserving
// unsigned keys (-0.0 folded onto +0.0), a 4 x 8-bit MSB-first radix select
// finds the k-th largest key T and how many keys equal to T must be taken,
// and a stable prefix-scan compaction in position order writes the anchors:
// every key above T, plus the lowest-position keys equal to T.  Because the
// compaction walks positions in ascending order, each S_l comes out sorted.
// Histograms use integer LDS atomics and every reduction is a scan, so the
// result is deterministic and unique.

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelPerThread = 8;   // contiguous elements per thread per compaction chunk

__device__ __forceinline__ uint32_t order_key(float f, int& nan_seen) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) nan_seen = 1;
    if (u == 0x80000000u) u = 0u;                       // -0.0 ties +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // ascending key == ascending value
}

__global__ void clear_error_word(int32_t* counts, int L) {
    if (threadIdx.x == 0 && blockIdx.x == 0) counts[L + 1] = 0;
}

// Row blockIdx.x of `scores` [rows][T]: its k largest entries (k capped by
// *k_cap when given), ascending positions into out + row * out_stride; the
// count taken into *n_out when given.
__global__ __launch_bounds__(kSelThreads) void select_topk(const float* __restrict__ scores,
                                                           int T, int k,
                                                           const int32_t* __restrict__ k_cap,
                                                           int32_t* __restrict__ out_base,
                                                           int out_stride,
                                                           int32_t* __restrict__ n_out,
                                                           int32_t* __restrict__ counts, int L) {
    __shared__ int hist[256];
    __shared__ int scan_scratch[kSelThreads / 64];
    __shared__ int digit_sh, above_sh, nan_sh;
    const int l = blockIdx.x;
    const int tid = threadIdx.x;
    const float* a = scores + (size_t)l * T;
    if (k_cap) k = min(k, k_cap[0]);
    if (n_out && tid == 0) n_out[0] = max(k, 0);
    if (k <= 0) return;                                  // nothing to select

    if (tid == 0) nan_sh = 0;
    int nan_seen = 0;
    uint32_t prefix = 0, mask = 0;
    int k_rem = k;

    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for (int i = tid; i < T; i += kSelThreads) {
            uint32_t key = order_key(a[i], nan_seen);
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        // Suffix sums over digits: threads 0..255 take digit 255 - tid, so an
        // inclusive prefix scan gives sum_{b' >= b} hist[b'].  The first four
        // waves hold those 256 threads; the other waves add zeros.
        const int b = 255 - tid;
        const int cnt = tid < 256 ? hist[b] : 0;
        int tot;
        const int excl = block_exclusive_scan<kSelThreads>(cnt, scan_scratch, tot);
        if (tid < 256) {
            const int above = excl;                 // keys whose digit exceeds b
            if (above < k_rem && k_rem <= above + cnt) {
                digit_sh = b;
                above_sh = above;
            }
        }
        __syncthreads();
        prefix |= (uint32_t)digit_sh << shift;
        mask |= 255u << shift;
        k_rem -= above_sh;
        __syncthreads();
    }
    if (nan_seen) nan_sh = 1;   // benign race: every writer stores 1

    // prefix = the k-th largest key; k_rem = how many keys equal to it to take.
    const uint32_t thr = prefix;
    int eq_base = 0, sel_base = 0;
    int32_t* out = out_base + (size_t)l * out_stride;
    for (int base = 0; base < T; base += kSelThreads * kSelPerThread) {
        const int i0 = base + tid * kSelPerThread;
        uint32_t keys[kSelPerThread];
        int n_eq = 0;
#pragma unroll
        for (int e = 0; e < kSelPerThread; ++e) {
            const int i = i0 + e;
            keys[e] = i < T ? order_key(a[i], nan_seen) : 0u;
            n_eq += (i < T && keys[e] == thr);
        }
        int eq_tot;
        int eq_rank = block_exclusive_scan<kSelThreads>(n_eq, scan_scratch, eq_tot) + eq_base;
        bool sel[kSelPerThread];
        int n_sel = 0;
#pragma unroll
        for (int e = 0; e < kSelPerThread; ++e) {
            const int i = i0 + e;
            bool s = false;
            if (i < T) {
                if (keys[e] > thr) s = true;
                else if (keys[e] == thr) s = (eq_rank++ < k_rem);
            }
            sel[e] = s;
            n_sel += s;
        }
        int sel_tot;
        int pos = block_exclusive_scan<kSelThreads>(n_sel, scan_scratch, sel_tot) + sel_base;
#pragma unroll
        for (int e = 0; e < kSelPerThread; ++e)
            if (sel[e] && pos < k) out[pos++] = i0 + e;
        eq_base += eq_tot;
        sel_base += sel_tot;
    }
    __syncthreads();
    if (tid == 0 && nan_sh) atomicOr(&counts[L + 1], 1);
}

// g_i = (sum_l a_{l,i}) / L, the sum in layer order.
__global__ void global_mean(const float* __restrict__ scores, int L, int T, float* __restrict__ g) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T) return;
    float acc = 0.f;
    for (int l = 0; l < L; ++l) acc += scores[(size_t)l * T + i];
    g[i] = acc / (float)L;
}

}  // namespace

hipError_t launch_select(const relaxkv_problem& p, const float* scores, const relaxkv_sets& s,
                         hipStream_t st) {
    hipLaunchKernelGGL(clear_error_word, dim3(1), dim3(64), 0, st, s.counts, p.L);
    hipLaunchKernelGGL(select_topk, dim3(p.L), dim3(kSelThreads), 0, st, scores, p.T_c, s.k,
                       (const int32_t*)nullptr, s.anchors, s.k, (int32_t*)nullptr, s.counts, p.L);
    return hipGetLastError();
}

hipError_t launch_select_rows(const float* scores, int n_rows, int T, int k, const int32_t* k_cap,
                              int32_t* out, int out_stride, int32_t* counts, int L,
                              hipStream_t st) {
    hipLaunchKernelGGL(select_topk, dim3(n_rows), dim3(kSelThreads), 0, st, scores, T, k, k_cap,
                       out, out_stride, (int32_t*)nullptr, counts, L);
    return hipGetLastError();
}

hipError_t launch_global_mean(const float* scores, int L, int T, float* g, hipStream_t st) {
    hipLaunchKernelGGL(global_mean, dim3((T + 255) / 256), dim3(256), 0, st, scores, L, T, g);
    return hipGetLastError();
}

hipError_t launch_select_global(const relaxkv_problem& p, const float* scores, int k_target,
                                const relaxkv_sets& s, float* g, int32_t* targets,
                                int32_t* n_targets, hipStream_t st) {
    hipLaunchKernelGGL(global_mean, dim3((p.T_c + 255) / 256), dim3(256), 0, st, scores, p.L,
                       p.T_c, g);
    // |P| = min(floor(r_g T_c), |U|) with |U| = counts[0] on the device.
    hipLaunchKernelGGL(select_topk, dim3(1), dim3(kSelThreads), 0, st, (const float*)g, p.T_c,
                       k_target, (const int32_t*)s.counts, targets, 0, n_targets, s.counts, p.L);
    return hipGetLastError();
}

}  // namespace relaxkv
