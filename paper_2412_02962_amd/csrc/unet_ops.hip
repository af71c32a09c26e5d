// Small pieces of a U-Net step around the library's layers:
//   pcpp_concat_channels  [rows, ca] and [rows, cb] (or zeros) side by side
//                         into [rows, ca + cb]: the up path's concatenation
//                         with the skip connection, and the zero padding of
//                         the 4 latent channels to the convolution's 64
//   pcpp_group_norm       GroupNorm (optionally with SiLU; band-local or
//                         synchronized statistics): the U-Net's output head
//                         before conv_out
//   pcpp_layer_norm       the transformer block's LayerNorm on its own
// All are bandwidth-bound; the copy moves 16-byte vectors, all loads of a
// thread issued before its stores.

#include <stdint.h>

#include "../../include/pcpp.h"
#include "common.h"
#include "gemm.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

__global__ __launch_bounds__(kThreads) void concat_channels(bf16* out, const bf16* a, const bf16* b, int64_t rows,
                                                            int ca, int cb) {
    const int va = ca / 8, vo = (ca + cb) / 8;
    const int64_t total = rows * vo;
    const int64_t stride = (int64_t)gridDim.x * kThreads * kUnroll;
    for (int64_t i0 = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; i0 < total; i0 += stride) {
        u32x4 buf[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = i0 + (int64_t)u * kThreads;
            buf[u] = u32x4{0u, 0u, 0u, 0u};
            if (i < total) {
                const int64_t r = i / vo;
                const int v = (int)(i - r * vo);
                if (v < va)
                    buf[u] = *(const u32x4*)(a + r * ca + 8 * v);
                else if (b != nullptr)
                    buf[u] = *(const u32x4*)(b + r * cb + 8 * (v - va));
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = i0 + (int64_t)u * kThreads;
            if (i < total) *(u32x4*)(out + i * 8) = buf[u];
        }
    }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool ranges_overlap(const void* a, int64_t na, const void* b, int64_t nb) {
    if (!a || !b) return false;
    return (uintptr_t)a < (uintptr_t)b + (uintptr_t)nb && (uintptr_t)b < (uintptr_t)a + (uintptr_t)na;
}

}  // namespace

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT int pcpp_concat_channels(int64_t rows, const void* a, int32_t ca, const void* b, int32_t cb, void* out,
                                     void* stream) {
    if (rows < 0 || ca < 8 || cb < 8 || ca % 8 != 0 || cb % 8 != 0) return PCPP_EINVAL;
    if (rows == 0) return PCPP_OK;
    if (!a || !out || !aligned16(a) || !aligned16(out) || (b && !aligned16(b))) return PCPP_EINVAL;
    const int64_t bytes_out = rows * (ca + cb) * 2;
    if (ranges_overlap(out, bytes_out, a, rows * ca * 2) || ranges_overlap(out, bytes_out, b, rows * cb * 2))
        return PCPP_EINVAL;
    const int64_t units = rows * ((ca + cb) / 8);
    int64_t blocks = (units + kThreads * kUnroll - 1) / (kThreads * kUnroll);
    if (blocks > 4096) blocks = 4096;
    concat_channels<<<(unsigned)blocks, kThreads, 0, (hipStream_t)stream>>>((bf16*)out, (const bf16*)a,
                                                                            (const bf16*)b, rows, ca, cb);
    return hipGetLastError() == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT int pcpp_layer_norm(int64_t rows, int32_t channels, float eps, const float* x, const void* gamma,
                                const void* beta, void* y, void* stream) {
    if (rows < 1 || rows > ((int64_t)1 << 24) || !(eps > 0.f)) return PCPP_EINVAL;
    if (channels < 4 || channels % 4 != 0 || channels > 2048) return PCPP_ENOTSUP;
    const void* ptrs[] = {x, gamma, beta, y};
    for (const void* p : ptrs)
        if (!p || !aligned16(p)) return PCPP_EINVAL;
    const char* xb = (const char*)x;
    const char* yb = (const char*)y;
    if (yb < xb + rows * channels * 4 && xb < yb + rows * channels * 2) return PCPP_EINVAL;
    LayerNormParams lp;
    lp.x = x;
    lp.y = (__bf16*)y;
    lp.gamma = (const __bf16*)gamma;
    lp.beta = (const __bf16*)beta;
    lp.rows = (int32_t)rows;
    lp.C = channels;
    lp.eps = eps;
    return launch_layer_norm(lp, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT size_t pcpp_group_norm_workspace_size(int32_t batch, int32_t tokens, int32_t channels, int32_t groups) {
    if (batch < 1 || batch > 65535 || tokens < 1 || !gn_shapes_ok(channels, groups)) return 0;
    return group_norm_ws_bytes(batch, groups, tokens);
}

PCPP_EXPORT int pcpp_group_norm(int32_t batch, int32_t tokens, int32_t channels, int32_t groups, float eps,
                                int32_t silu, const void* x, const void* gamma, const void* beta,
                                const float* bands, int32_t n_bands, int32_t band, float* own_out, void* y,
                                void* workspace, size_t ws_bytes, void* stream) {
    if (batch < 1 || batch > 65535 || tokens < 1 || !(eps > 0.f) || (silu != 0 && silu != 1)) return PCPP_EINVAL;
    if (bands != nullptr && (n_bands < 1 || band < 0 || band >= n_bands || ((uintptr_t)bands & 3u) != 0))
        return PCPP_EINVAL;
    if (own_out != nullptr && ((uintptr_t)own_out & 3u) != 0) return PCPP_EINVAL;
    if (!gn_shapes_ok(channels, groups)) return PCPP_ENOTSUP;
    if ((int64_t)batch * tokens * channels > ((int64_t)1 << 40)) return PCPP_EINVAL;
    const void* ptrs[] = {x, gamma, beta, y};
    for (const void* p : ptrs)
        if (!p || !aligned16(p)) return PCPP_EINVAL;
    const size_t need = group_norm_ws_bytes(batch, groups, tokens);
    if (!workspace || ws_bytes < need) return PCPP_EWORKSPACE;
    if (!aligned16(workspace)) return PCPP_EINVAL;
    GroupNormParams gp;
    gp.x = (const __bf16*)x;
    gp.y = (__bf16*)y;
    gp.gamma = (const __bf16*)gamma;
    gp.beta = (const __bf16*)beta;
    gp.stats = (float*)workspace;
    gp.B = batch;
    gp.N = tokens;
    gp.C = channels;
    gp.G = groups;
    gp.eps = eps;
    gp.bands = bands;
    gp.n_bands = bands ? n_bands : 1;
    gp.band = bands ? band : 0;
    gp.own_out = own_out;
    gp.silu = silu;
    return launch_group_norm(gp, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}
