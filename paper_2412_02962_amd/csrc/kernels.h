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

// bf16 path: workspace bytes it needs (work counters and float32 partial
// results of query blocks split across workgroups) and the launch.
size_t attention_bf16_ws_bytes(const AttnParams& p);
hipError_t launch_attention_bf16(const AttnParams& p, void* ws, size_t ws_bytes, hipStream_t stream);
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
