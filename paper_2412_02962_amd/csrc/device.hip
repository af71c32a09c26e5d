// Device layout queries shared by the launches that merge split work through
// one XCD's L2 (the bf16 attention's key pieces, the split-K GEMMs).
//
// On gfx950 the hardware deals the workgroups of a launch round-robin over
// the device's XCDs (32 compute units each): workgroup w runs on XCD
// w % n_xcd.  A launch that keeps all pieces of one tile on one XCD can then
// merge them with plain stores and a workgroup-scope counter in that XCD's
// L2.  That holds only when the launch may use every compute unit: a stream
// with a CU mask, or a device whose compute units are not whole XCDs, gets
// n_xcd = 1 and no merging, and the launches fall back to unsplit work.

#include <atomic>

#include "kernels.h"

namespace pcpp {

namespace {

constexpr int kCusPerXcd = 32;
constexpr int kMaxDevices = 64;
constexpr uint32_t kMaskWords = 32;  // up to 1024 compute units

// Per-device compute-unit count, asked once (0 = not asked yet).  Relaxed
// atomics: every thread that asks stores the same value.
std::atomic<int> g_cus[kMaxDevices];

}  // namespace

DeviceLayout layout_for(int cus, int cus_enabled) {
    DeviceLayout d;
    d.cus = cus > 0 ? cus : 256;
    d.xcd_merge = cus > 0 && cus % kCusPerXcd == 0 && cus_enabled >= cus;
    d.n_xcd = d.xcd_merge ? cus / kCusPerXcd : 1;
    return d;
}

int device_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (dev >= 0 && dev < kMaxDevices) {
        const int c = g_cus[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 0;
    if (dev >= 0 && dev < kMaxDevices) g_cus[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

// Compute units among the device's first `cus` that `stream` may use; 0 when
// the runtime cannot say (then nothing is merged across workgroups).
int stream_cus(hipStream_t stream, int cus) {
    uint32_t mask[kMaskWords] = {};
    if (cus <= 0 || cus > (int)(32 * kMaskWords)) return 0;
    if (hipExtStreamGetCUMask(stream, kMaskWords, mask) != hipSuccess) return 0;
    int n = 0;
    for (int c = 0; c < cus; ++c) n += (mask[c >> 5] >> (c & 31)) & 1u;
    return n;
}

DeviceLayout device_layout(hipStream_t stream) {
    const int cus = device_cus();
    return layout_for(cus, stream_cus(stream, cus));
}

// Workspace sizing: every compute unit usable; an MI355X's 256 when the
// device cannot be asked (sizes are then upper bounds for that device).
DeviceLayout device_layout_unmasked() {
    int cus = device_cus();
    if (cus <= 0) cus = 256;
    return layout_for(cus, cus);
}

}  // namespace pcpp
