// GroupNorm and LayerNorm of the transformer block (bandwidth-bound).
//
// GroupNorm uses the statistics of the band's own tokens (each image, each
// group of C/G consecutive channels): a first kernel reduces token chunks to
// (count, mean, M2) with a two-pass sum per chunk, the apply kernel merges
// the chunk statistics (Chan et al.'s pairwise update) and writes
// (x - mean) / sqrt(var + eps) * gamma + beta with the biased variance.
// LayerNorm: one wavefront per fp32 row, two passes over registers.

#include <math.h>

#include "common.h"
#include "gemm.h"

namespace pcpp {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float s = 0.f;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
    return s;
}

__global__ __launch_bounds__(256) void gn_partial(GroupNormParams p) {
    __shared__ float red[4];
    const int g = blockIdx.x, b = blockIdx.y, ch = blockIdx.z;
    const int cg = p.C / p.G;
    const int t0 = (int)((int64_t)p.N * ch / p.chunks);
    const int t1 = (int)((int64_t)p.N * (ch + 1) / p.chunks);
    const int64_t cnt = (int64_t)(t1 - t0) * cg;
    const bf16* xb = p.x + (int64_t)b * p.N * p.C + (int64_t)g * cg;
    float s = 0.f;
    for (int64_t e = threadIdx.x; e < cnt; e += 256) {
        const int tok = t0 + (int)(e / cg), c = (int)(e % cg);
        s += bf16_to_f32(xb[(int64_t)tok * p.C + c]);
    }
    const float mean = cnt > 0 ? block_sum(s, red) / (float)cnt : 0.f;
    float q = 0.f;
    for (int64_t e = threadIdx.x; e < cnt; e += 256) {
        const int tok = t0 + (int)(e / cg), c = (int)(e % cg);
        const float d = bf16_to_f32(xb[(int64_t)tok * p.C + c]) - mean;
        q += d * d;
    }
    const float m2 = block_sum(q, red);
    if (threadIdx.x == 0) {
        float* st = p.stats + (((int64_t)b * p.G + g) * p.chunks + ch) * 3;
        st[0] = (float)cnt;
        st[1] = mean;
        st[2] = m2;
    }
}

__global__ __launch_bounds__(256) void gn_apply(GroupNormParams p) {
    const int64_t pairs = (int64_t)p.B * p.N * (p.C / 2);
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= pairs) return;
    const int cp = (int)(i % (p.C / 2));
    const int64_t bt = i / (p.C / 2);
    const int b = (int)(bt / p.N);
    const int cg = p.C / p.G;
    float y[2];
    const bf16* xr = p.x + bt * p.C + 2 * cp;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int c = 2 * cp + e;
        const int g = c / cg;
        const float* st = p.stats + ((int64_t)b * p.G + g) * p.chunks * 3;
        float n = st[0], mean = st[1], m2 = st[2];
        for (int k = 1; k < p.chunks; ++k) {
            const float nb = st[3 * k], mb = st[3 * k + 1], m2b = st[3 * k + 2];
            const float nn = n + nb;
            if (nn <= 0.f) continue;
            const float d = mb - mean;
            mean += d * (nb / nn);
            m2 += m2b + d * d * (n * nb / nn);
            n = nn;
        }
        const float rstd = rsqrtf(m2 / n + p.eps);
        y[e] = (bf16_to_f32(xr[e]) - mean) * rstd * bf16_to_f32(p.gamma[c]) + bf16_to_f32(p.beta[c]);
    }
    bf16* yr = p.y + bt * p.C + 2 * cp;
    yr[0] = f32_to_bf16(y[0]);
    yr[1] = f32_to_bf16(y[1]);
}

constexpr int LN_MAX_PER_LANE = 32;  // C <= 2048

__global__ __launch_bounds__(256) void ln_kernel(LayerNormParams p) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= p.rows) return;
    const float* xr = p.x + (int64_t)row * p.C;
    float v[LN_MAX_PER_LANE];
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < LN_MAX_PER_LANE; ++k) {
        const int c = lane + 64 * k;
        v[k] = c < p.C ? xr[c] : 0.f;
        s += v[k];
    }
    const float mean = wave_sum(s) / (float)p.C;
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < LN_MAX_PER_LANE; ++k) {
        const int c = lane + 64 * k;
        const float d = c < p.C ? v[k] - mean : 0.f;
        q += d * d;
    }
    const float rstd = rsqrtf(wave_sum(q) / (float)p.C + p.eps);
    bf16* yr = p.y + (int64_t)row * p.C;
#pragma unroll
    for (int k = 0; k < LN_MAX_PER_LANE; ++k) {
        const int c = lane + 64 * k;
        if (c < p.C)
            yr[c] = f32_to_bf16((v[k] - mean) * rstd * bf16_to_f32(p.gamma[c]) + bf16_to_f32(p.beta[c]));
    }
}

}  // namespace

size_t group_norm_ws_bytes(int B, int G) { return (size_t)B * G * 8 * 3 * sizeof(float); }

hipError_t launch_group_norm(GroupNormParams p, hipStream_t s) {
    p.chunks = 8;
    gn_partial<<<dim3(p.G, p.B, p.chunks), 256, 0, s>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t pairs = (int64_t)p.B * p.N * (p.C / 2);
    gn_apply<<<(unsigned)((pairs + 255) / 256), 256, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_layer_norm(const LayerNormParams& p, hipStream_t s) {
    ln_kernel<<<(p.rows + 3) / 4, 256, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace pcpp
