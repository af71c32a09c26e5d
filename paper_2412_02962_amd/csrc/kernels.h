// Internal launch interfaces of the PCPP kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pcpp {

// Key/value rows of one attention call as up to three contiguous token
// ranges: [0, end0) from segment 0, [end0, end1) from segment 1 and
// [end1, n_kv) from segment 2.  Each segment pointer already points at the
// first token it contributes; tokens are `C` elements apart; images are
// bstride[s] elements apart.  For partially conditioned attention the
// segments are the stale rows above, the fresh band and the stale rows below.
struct KvSource {
    const void* k[3];
    const void* v[3];
    int64_t bstride[3];
    int32_t end0;
    int32_t end1;
    int32_t n_kv;
};

struct AttnParams {
    const void* q;        // [B, nq, C]
    void* out;            // [B, nq, C]
    int64_t q_bstride;    // elements between images of q / out
    int32_t nq;
    int32_t C;
    int32_t heads;
    int32_t batch;
    KvSource kv;
    float scale_log2;     // log2(e) / sqrt(head_dim)
    float scale;          // 1 / sqrt(head_dim)
};

// Where the workgroups of a launch run (device.hip).  n_xcd > 1 only when
// workgroup w of a launch is known to run on XCD w % n_xcd: a device whose
// compute units are whole XCDs (32 each) and a stream without a CU mask.
// Only then may a launch merge the pieces of one tile through an XCD's L2.
struct DeviceLayout {
    int32_t cus;       // compute units of the device
    int32_t n_xcd;     // XCDs the workgroups are dealt over, or 1
    bool xcd_merge;    // pieces of a tile may be merged through one XCD's L2
};
DeviceLayout layout_for(int cus, int cus_enabled);  // pure: for planning and tests
int device_cus();                                    // current device, cached per device; 0 if unknown
DeviceLayout device_layout(hipStream_t stream);      // current device, the stream's CU mask
DeviceLayout device_layout_unmasked();               // current device, every compute unit (workspace sizing)

// bf16 path: workspace bytes it needs (work counters and float32 partial
// results of query blocks split across workgroups; sized for a launch that
// may use every compute unit) and the launch.
size_t attention_bf16_ws_bytes(const AttnParams& p);
// Bytes at the start of every bf16 attention workspace that hold its work
// counters (the same for every geometry).
size_t attention_bf16_counter_bytes();
hipError_t launch_attention_bf16(const AttnParams& p, void* ws, size_t ws_bytes, hipStream_t stream);
// Launch plan for a device layout: queries per block, pieces per block,
// workgroups, and the work counters a launch uses (they must be zero at the
// launch and are left zero).
struct AttnPlanInfo {
    int32_t block_queries, pieces, workgroups, counters;
};
AttnPlanInfo attention_bf16_plan(const AttnParams& p, const DeviceLayout& d);
hipError_t launch_attention_f32(const AttnParams& p, hipStream_t stream);

// Context assembly: contiguous segment copies plus the index set.
struct GatherParams {
    KvSource src;         // as above; k/v element type from esize
    void* k_ctx;          // [B, n_kv, C] or null
    void* v_ctx;
    int32_t* idx;         // [n_kv] or null
    int32_t idx_base;     // global token id of context token 0
    int32_t C;
    int32_t batch;
    int32_t esize;        // bytes per element (2 or 4)
};
hipError_t launch_gather(const GatherParams& p, hipStream_t stream);

// Up to four contiguous runs of `bytes` per image, image b's run starting at
// src + b * src_bstride and going to dst + b * dst_bstride (bytes).  Runs
// must not overlap each other's destinations or any source.
struct CopySeg {
    const char* src;
    char* dst;
    int64_t src_bstride;
    int64_t dst_bstride;
    int64_t bytes;
};
struct CopyParams {
    CopySeg seg[4];
    int32_t n_seg;
    int32_t batch;
};
hipError_t launch_seg_copy(const CopyParams& p, int esize, hipStream_t stream);

}  // namespace pcpp
