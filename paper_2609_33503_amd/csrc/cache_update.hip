// Cache update (Sec. 3.4 cache-update semantics; Algorithm 1, cache-update step):
// after layer l is recomputed, the fresh K/V rows of R_l overwrite the layer's
// cache entries at their positions; every other entry keeps its value.
//
// One pass of 16-byte copies: thread -> (target t, KV head g, 16-byte part), so
// consecutive threads read consecutive bytes of the fresh rows and write whole
// d-long rows of the cache.  |R_l| is read on the device and clamped to the
// launch's row cap (the caller's row capacity and the host bound on |R_l|); the
// grid is sized from that cap and surplus threads exit.  A clamped count sets
// RELAXKV_ERR_ROWS.

#include "dev_common.h"
#include "internal.h"

namespace relaxkv {
namespace {

__global__ __launch_bounds__(256) void update_cache_rows(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, u32x4* __restrict__ k_cache,
    u32x4* __restrict__ v_cache, const int32_t* __restrict__ R_off,
    const int32_t* __restrict__ R_idx, const int32_t* __restrict__ counts,
    int32_t* __restrict__ err, int layer, int Hkv, int64_t head_parts, int64_t token_parts,
    int parts, int cap) {
    const int nR_dev = counts[1 + layer];
    const int nR = min(nR_dev, cap);
    if (nR_dev > cap && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, RELAXKV_ERR_ROWS);
    const long n = (long)nR * Hkv * parts;
    const int32_t* pos = R_idx + R_off[layer];
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n;
         i += (long)gridDim.x * blockDim.x) {
        const int part = (int)(i % parts);
        const long tg = i / parts;                       // t * Hkv + g
        const int g = (int)(tg % Hkv);
        const int t = (int)(tg / Hkv);
        const int64_t dst = g * head_parts + pos[t] * token_parts + part;
        k_cache[dst] = k_new[i];
        v_cache[dst] = v_new[i];
    }
}

}  // namespace

hipError_t launch_update_cache(const relaxkv_problem& p, const relaxkv_sets& s, int layer,
                               const void* k_new, const void* v_new, int n_rows, void* k_cache,
                               void* v_cache, hipStream_t st) {
    const size_t esz = p.dtype == RELAXKV_DTYPE_BF16 ? 2 : 4;
    const int parts = (int)(p.d * esz / 16);             // 16-byte parts per row
    const KvStrides ks = kv_strides(p);                   // 16-byte multiples (checked on the host)
    u32x4* kc = (u32x4*)((char*)k_cache + (size_t)(layer * ks.layer) * esz);
    u32x4* vc = (u32x4*)((char*)v_cache + (size_t)(layer * ks.layer) * esz);
    const int cap = row_cap(p, s, layer, n_rows);
    const long n_bound = (long)cap * p.H_kv * parts;
    long blocks = (n_bound + 255) / 256;
    if (blocks < 1) blocks = 1;                          // block 0 still checks the count
    hipLaunchKernelGGL(update_cache_rows, dim3((unsigned)(blocks < 8192 ? blocks : 8192)),
                       dim3(256), 0, st, (const u32x4*)k_new, (const u32x4*)v_new, kc, vc,
                       s.R_off, s.R_idx, s.counts, s.counts + p.L + 1, layer, p.H_kv,
                       (int64_t)(ks.head * esz / 16), (int64_t)(ks.token * esz / 16), parts, cap);
    return hipGetLastError();
}

}  // namespace relaxkv
