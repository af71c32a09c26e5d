// Key/value context assembly (Eq. 1, Fig. 3 of arXiv 2412.02962).
//
// The context of band i is the row range [i*h - up, (i+1)*h + dn) of the
// token grid, every column.  In each source buffer those rows are one
// contiguous run of tokens (the last `up` rows of the band above, the whole
// local band, the first `dn` rows of the band below), so assembly is three
// contiguous streaming copies per tensor and image, and the index set is the
// contiguous range of global token ids starting at (i*h - up) * W.
//
// HBM-bound: every byte is read once and written once with 16-byte vector
// accesses; each thread moves UNROLL chunks with all loads issued before the
// stores so several requests per lane are in flight.

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// One tensor's three source runs.  The kernel turns them into three
// per-image base pointers held in scalar registers before the copy loop; a
// run picked per lane by indexing an array (or a local struct) would make
// the compiler keep the struct in per-lane private memory, whose stores
// reach HBM.
struct Seg3 {
    const char* base0;
    const char* base1;
    const char* base2;
    int64_t bstride0, bstride1, bstride2;  // bytes between images
    int64_t end0;  // byte offsets of the run boundaries within one image
    int64_t end1;
};

// Source address of byte `off` of the context: run 0 below e0, run 1 below
// e1, run 2 after (p0..p2 already point at this image's runs).
__device__ __forceinline__ const char* seg_addr(const char* p0, const char* p1, const char* p2, int64_t e0,
                                                int64_t e1, int64_t off) {
    return off < e0 ? p0 + off : (off < e1 ? p1 + (off - e0) : p2 + (off - e1));
}

template <typename V>
__global__ __launch_bounds__(kThreads) void gather_copy(Seg3 ks, Seg3 vs, char* kdst, char* vdst,
                                                         int64_t image_bytes, int32_t* idx,
                                                         int32_t idx_base, int32_t n_kv) {
    const int b = blockIdx.z;
    const bool is_v = blockIdx.y == 1;
    const Seg3& s = is_v ? vs : ks;
    const char* p0 = s.base0 + (int64_t)b * s.bstride0;
    const char* p1 = s.base1 + (int64_t)b * s.bstride1;
    const char* p2 = s.base2 + (int64_t)b * s.bstride2;
    const int64_t e0 = ks.end0, e1 = ks.end1;
    char* dst = (is_v ? vdst : kdst);
    if (dst != nullptr) {
        dst += (int64_t)b * image_bytes;
        const int64_t nvec = image_bytes / (int64_t)sizeof(V);
        const int64_t chunk = (int64_t)kThreads * kUnroll;
        for (int64_t c = (int64_t)blockIdx.x * chunk; c < nvec; c += (int64_t)gridDim.x * chunk) {
            const int64_t v0 = c + threadIdx.x;
            V buf[kUnroll];
            if (c + chunk <= nvec) {
                // whole chunk: every load issued before the first store
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    buf[u] = *(const V*)seg_addr(p0, p1, p2, e0, e1, (v0 + (int64_t)u * kThreads) * (int64_t)sizeof(V));
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    *(V*)(dst + (v0 + (int64_t)u * kThreads) * (int64_t)sizeof(V)) = buf[u];
            } else {
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int64_t v = v0 + (int64_t)u * kThreads;
                    if (v < nvec) buf[u] = *(const V*)seg_addr(p0, p1, p2, e0, e1, v * (int64_t)sizeof(V));
                }
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int64_t v = v0 + (int64_t)u * kThreads;
                    if (v < nvec) *(V*)(dst + v * (int64_t)sizeof(V)) = buf[u];
                }
            }
        }
    }
    if (idx != nullptr && b == 0 && !is_v) {
        for (int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x; j < n_kv;
             j += (int64_t)gridDim.x * kThreads)
            idx[j] = idx_base + (int32_t)j;
    }
}

}  // namespace

hipError_t launch_gather(const GatherParams& p, hipStream_t stream) {
    const int64_t row = (int64_t)p.C * p.esize;
    const int64_t image = row * p.src.n_kv;
    Seg3 ks, vs;
    ks.base0 = (const char*)p.src.k[0];
    ks.base1 = (const char*)p.src.k[1];
    ks.base2 = (const char*)p.src.k[2];
    vs.base0 = (const char*)p.src.v[0];
    vs.base1 = (const char*)p.src.v[1];
    vs.base2 = (const char*)p.src.v[2];
    ks.bstride0 = vs.bstride0 = p.src.bstride[0] * p.esize;
    ks.bstride1 = vs.bstride1 = p.src.bstride[1] * p.esize;
    ks.bstride2 = vs.bstride2 = p.src.bstride[2] * p.esize;
    ks.end0 = vs.end0 = row * p.src.end0;
    ks.end1 = vs.end1 = row * p.src.end1;

    bool vec16 = (row % 16) == 0;
    for (int k = 0; k < 3; ++k) {
        vec16 = vec16 && ((uintptr_t)p.src.k[k] % 16 == 0) && ((uintptr_t)p.src.v[k] % 16 == 0) &&
                ((p.src.bstride[k] * p.esize) % 16 == 0);
    }
    vec16 = vec16 && ((uintptr_t)p.k_ctx % 16 == 0) && ((uintptr_t)p.v_ctx % 16 == 0);
    const int vbytes = vec16 ? 16 : p.esize;
    const bool copy = p.k_ctx != nullptr;
    int64_t nvec = copy ? image / vbytes : 0;
    int64_t want = (nvec + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
    int64_t want_idx = (p.src.n_kv + kThreads - 1) / kThreads;
    if (want_idx > want) want = want_idx;
    if (want < 1) want = 1;
    if (want > 4096) want = 4096;
    dim3 grid((unsigned)want, 2, (unsigned)p.batch);
    if (vec16)
        gather_copy<u32x4><<<grid, kThreads, 0, stream>>>(ks, vs, (char*)p.k_ctx, (char*)p.v_ctx, image,
                                                          p.idx, p.idx_base, p.src.n_kv);
    else if (p.esize == 4)
        gather_copy<uint32_t><<<grid, kThreads, 0, stream>>>(ks, vs, (char*)p.k_ctx, (char*)p.v_ctx, image,
                                                             p.idx, p.idx_base, p.src.n_kv);
    else
        gather_copy<uint16_t><<<grid, kThreads, 0, stream>>>(ks, vs, (char*)p.k_ctx, (char*)p.v_ctx, image,
                                                             p.idx, p.idx_base, p.src.n_kv);
    return hipGetLastError();
}

}  // namespace pcpp
