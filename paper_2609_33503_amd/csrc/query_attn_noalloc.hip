// Allocation-free variant of the query-side completion (relaxkv_query_attn_noalloc).
//
// relaxkv_query_attn's bf16 path needs scratch for its key splits (normalised
// partial outputs and their log2-sum-exp).  Callers that cannot allocate device
// memory (code under stream capture, tight serving loops) call this variant
// instead: the scratch is a file-scope device array of kScratchBytes that every
// GPU the library runs on holds until the process ends.  Host code never uses
// the array's name as a device address (in host code it names a host-side
// stand-in); it uses the address hipGetSymbolAddress returns, looked up once per
// device with that device current.  The kernels are the ones relaxkv_query_attn
// launches and take that address as their workspace.
//
// Every scratch element the merge reads is written earlier in the same call
// (each split writes its partial rows before the merge kernel reads them), so
// nothing needs clearing between calls.  Calls on one GPU share the array:
// calls that overlap in time on one device (two streams, or two threads) race.

#include <mutex>

#include "internal.h"

namespace relaxkv {
namespace {

constexpr size_t kScratchBytes = RELAXKV_QUERY_ATTN_NOALLOC_MAX_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of this device's copy of `scratch` (looked up on the first call
// on each device, with that device current).
hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace relaxkv

using namespace relaxkv;

extern "C" relaxkv_status relaxkv_query_attn_noalloc(const relaxkv_problem* p, int32_t layer,
                                                      const void* k_cache, const void* v_cache,
                                                      const void* k_q, const void* v_q, void* out,
                                                      float* lse_out, void* stream) {
    relaxkv_status st = relaxkv_validate(p);
    if (st != RELAXKV_OK) return st;
    if (layer < 0 || layer >= p->L) return RELAXKV_EINVAL;
    if (!k_cache || !v_cache || !k_q || !v_q || !out) return RELAXKV_EINVAL;
    const QueryAttnWorkspace w = query_attn_workspace_layout(*p);
    if (w.total > kScratchBytes) return RELAXKV_ENOSPACE;
    void* ws = nullptr;
    if (w.total && scratch_address(&ws) != hipSuccess) return RELAXKV_EDEVICE;
    const hipError_t e = launch_query_attn(*p, layer, k_cache, v_cache, k_q, v_q, out, lse_out,
                                           (char*)ws, (hipStream_t)stream);
    return e == hipSuccess ? RELAXKV_OK : RELAXKV_EDEVICE;
}
