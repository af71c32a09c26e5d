// pcpp_partial_attention_noalloc: the partially conditioned attention (Sec.
// 3.3 of arXiv 2412.02962) for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  It runs the same kernels as pcpp_partial_attention; their
// workspace (work counters and float32 partials of split key ranges) is a
// file-scope device array of fixed size instead of a caller buffer.
//
// The array's name is a host-side stand-in in host code: its device address
// on each GPU comes from hipGetSymbolAddress, taken once per device (with
// that device current) at the entry point's first call there, and only that
// address is handed to kernels.  Every call on one GPU shares that GPU's
// array: calls that overlap on one GPU (on different streams, or from
// different threads) race.  The counters must be zero at every launch; the
// set-up clears them with a fill kernel on the caller's stream, and every
// launch leaves them at zero again.  The float32 partials need no clearing.

#include <atomic>

#include "../../include/pcpp.h"
#include "api_internal.h"
#include "kernels.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

constexpr size_t kScratchBytes = (size_t)PCPP_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

// Per-device address of `scratch` (null until the device's set-up).
std::atomic<void*> g_scratch[kMaxDevices];

__global__ void zero_ints(int* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// The current device's scratch address; on the first call on a device, look
// it up and clear the attention's work counters (the first `counter_bytes`).
int scratch_for_current_device(hipStream_t stream, size_t counter_bytes, void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PCPP_EHIP;
    void* ptr = g_scratch[dev].load(std::memory_order_acquire);
    if (ptr == nullptr) {
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return PCPP_EHIP;
        const int n = (int)(counter_bytes / sizeof(int));
        zero_ints<<<(n + 255) / 256, 256, 0, stream>>>((int*)ptr, n);
        if (hipGetLastError() != hipSuccess) return PCPP_EHIP;
        g_scratch[dev].store(ptr, std::memory_order_release);
    }
    *out = ptr;
    return PCPP_OK;
}

}  // namespace

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT int pcpp_partial_attention_noalloc(const pcpp_geom_t* g, const void* q, const void* k_fresh,
                                               const void* v_fresh, const void* k_up, const void* v_up,
                                               const void* k_dn, const void* v_dn, void* out, void* stream) {
    Geo r;
    int st = check_attention(g, &r, q, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, out);
    if (st != PCPP_OK) return st;
    KvSource kv = make_kv_source(g, r, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn);
    AttnParams p = make_attn_params(g, r, q, out, kv);
    hipStream_t s = (hipStream_t)stream;
    if (g->dtype != PCPP_DTYPE_BF16) return launch_attention_f32(p, s) == hipSuccess ? PCPP_OK : PCPP_EHIP;
    const size_t need = attention_bf16_ws_bytes(p);
    if (need > kScratchBytes) return PCPP_EWORKSPACE;
    void* ws = nullptr;
    st = scratch_for_current_device(s, attention_bf16_counter_bytes(), &ws);
    if (st != PCPP_OK) return st;
    return launch_attention_bf16(p, ws, kScratchBytes, s) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}
