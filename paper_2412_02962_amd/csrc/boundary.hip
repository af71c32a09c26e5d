// p-aware boundary messages of the neighbour exchange (Sec. 3.2 with Eq. 1
// of arXiv 2412.02962).
//
// A band's neighbours read only r rows of its fresh keys and values at the
// next step: the band above its first r rows, the band below its last r
// rows.  Packing gathers those rows of K and V of every image into one
// contiguous message per neighbour, [B][K rows, V rows][r*W][C]; unpacking
// places a received message at the rows of the stale buffers the attention
// reads.  Both are a handful of contiguous runs (rows of one image are
// contiguous in [B, h*W, C]), copied with the widest vector every run
// allows, all loads of a thread issued before its stores.

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

template <typename V>
__global__ __launch_bounds__(kThreads) void seg_copy(CopyParams p) {
    const int s = blockIdx.y;
    const int b = blockIdx.z;
    const CopySeg sg = p.seg[s];
    const int64_t nvec = sg.bytes / (int64_t)sizeof(V);
    if (nvec == 0) return;
    const V* src = (const V*)(sg.src + (int64_t)b * sg.src_bstride);
    V* dst = (V*)(sg.dst + (int64_t)b * sg.dst_bstride);
    const int64_t stride = (int64_t)gridDim.x * kThreads * kUnroll;
    for (int64_t v0 = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; v0 < nvec; v0 += stride) {
        V buf[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + (int64_t)u * kThreads;
            if (v < nvec) buf[u] = src[v];
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + (int64_t)u * kThreads;
            if (v < nvec) dst[v] = buf[u];
        }
    }
}

}  // namespace

hipError_t launch_seg_copy(const CopyParams& p, int esize, hipStream_t stream) {
    if (p.n_seg < 1 || p.n_seg > 4 || p.batch < 1 || p.batch > 65535) return hipErrorInvalidValue;
    int64_t most = 0;
    bool v16 = true;
    for (int s = 0; s < p.n_seg; ++s) {
        const CopySeg& g = p.seg[s];
        if (g.bytes > most) most = g.bytes;
        v16 = v16 && g.bytes % 16 == 0 && g.src_bstride % 16 == 0 && g.dst_bstride % 16 == 0 &&
              (uintptr_t)g.src % 16 == 0 && (uintptr_t)g.dst % 16 == 0;
    }
    if (most == 0) return hipSuccess;
    const int vbytes = v16 ? 16 : esize;
    int64_t blocks = (most / vbytes + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    const dim3 grid((unsigned)blocks, (unsigned)p.n_seg, (unsigned)p.batch);
    if (v16)
        seg_copy<u32x4><<<grid, kThreads, 0, stream>>>(p);
    else if (esize == 4)
        seg_copy<uint32_t><<<grid, kThreads, 0, stream>>>(p);
    else
        seg_copy<uint16_t><<<grid, kThreads, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace pcpp
