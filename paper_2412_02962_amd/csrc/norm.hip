// GroupNorm and LayerNorm of the transformer block (bandwidth-bound).
//
// GroupNorm uses the statistics of the band's own tokens (each image, each
// group of C/G consecutive channels).  gn_stats: a workgroup holds a chunk of
// 16 whole token rows in registers (coalesced channel pairs) and reduces them
// to per-group (count, mean, M2) with two passes over the registers (sum,
// then squared deviations from the chunk mean).  gn_finalize (one workgroup
// per image) merges the chunk statistics of every group with Chan et al.'s
// pairwise update in a fixed order and stores mean and 1/sqrt(var + eps)
// (biased variance).  Synchronized GroupNorm (the whole image's statistics,
// Sec. 3.3 of arXiv 2412.02962) merges every band's (count, mean, M2) in
// band order, this band's own in its place, before that.  gn_apply: per-channel scale and shift in LDS, 16-byte
// vectors.
// LayerNorm: one wavefront per fp32 row, 16-byte loads, two passes over
// registers, 8-byte bf16 stores.

#include <math.h>

#include "common.h"
#include "gemm.h"

namespace pcpp {

namespace {

constexpr int GN_THREADS = 256;
constexpr int GN_MAX_C = 2048;     // channels (registers of gn_stats, LDS tables of gn_apply)
constexpr int GN_MAX_G = 256;
constexpr int GN_TOKENS_PER_APPLY = 8;
constexpr int GN_CHUNK_TOKENS = 16;  // tokens per statistics workgroup

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Workspace of GroupNorm, per image: [chunks][G] x (count, mean, M2), then
// [G] x (mean, rstd).
struct GnLayout {
    size_t part, fin, total;
};
__host__ __device__ inline GnLayout gn_layout(int B, int G, int chunks) {
    GnLayout l;
    l.part = 0;
    l.fin = l.part + (size_t)B * G * chunks * 3 * sizeof(float);
    l.total = l.fin + (size_t)B * G * 2 * sizeof(float);
    return l;
}

// Chan et al.'s pairwise update of (n, mean, M2) with (nb, mb, m2b).
__device__ __forceinline__ void chan_merge(float& n, float& mean, float& m2, float nb, float mb, float m2b) {
    if (nb <= 0.f) return;
    const float nn = n + nb;
    const float r = __builtin_amdgcn_rcpf(nn);  // statistics: a 1-ulp reciprocal is plenty
    const float d = mb - mean;
    mean += d * (nb * r);
    m2 += m2b + d * d * (n * nb * r);
    n = nn;
}

__global__ __launch_bounds__(GN_THREADS) void gn_stats(GroupNormParams p) {
    __shared__ float chan_acc[GN_MAX_C];
    __shared__ float g_mean[GN_MAX_G];
    const int ch = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x;
    const int C = p.C, G = p.G, cg = C / G, np = C / 2;
    const int t0 = (int)((int64_t)p.N * ch / p.chunks);
    const int t1 = (int)((int64_t)p.N * (ch + 1) / p.chunks);
    const bf16* xb = p.x + (int64_t)b * p.N * C;
    const GnLayout L = gn_layout(p.B, G, p.chunks);
    char* ws = (char*)p.stats;
    float* part = (float*)(ws + L.part);

    // The chunk's rows, channel pairs per lane, held in registers for both
    // passes (at most GN_CHUNK_TOKENS tokens and GN_MAX_C / 2 / GN_THREADS
    // pairs per thread).
    constexpr int PP = GN_MAX_C / 2 / GN_THREADS;
    bf16x2 xv[PP][GN_CHUNK_TOKENS];
#pragma unroll
    for (int k = 0; k < PP; ++k) {
        const int cp = tid + GN_THREADS * k;
#pragma unroll
        for (int t = 0; t < GN_CHUNK_TOKENS; ++t) {
            bf16x2 v = {};
            if (cp < np && t0 + t < t1) v = *(const bf16x2*)(xb + (int64_t)(t0 + t) * C + 2 * cp);
            xv[k][t] = v;
        }
    }
    // Pass 1: per channel, the sum over the chunk's tokens.
#pragma unroll
    for (int k = 0; k < PP; ++k) {
        const int cp = tid + GN_THREADS * k;
        if (cp >= np) break;
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int t = 0; t < GN_CHUNK_TOKENS; ++t) {
            s0 += (float)xv[k][t][0];
            s1 += (float)xv[k][t][1];
        }
        chan_acc[2 * cp] = s0;
        chan_acc[2 * cp + 1] = s1;
    }
    __syncthreads();
    const int nt = t1 - t0;
    const float n_chunk = (float)nt * (float)cg;
    for (int g = tid; g < G; g += GN_THREADS) {
        float s = 0.f;
        for (int c = g * cg; c < (g + 1) * cg; ++c) s += chan_acc[c];
        g_mean[g] = n_chunk > 0.f ? s / n_chunk : 0.f;
    }
    __syncthreads();
    // Pass 2: squared deviations from the chunk mean of the channel's group.
#pragma unroll
    for (int k = 0; k < PP; ++k) {
        const int cp = tid + GN_THREADS * k;
        if (cp >= np) break;
        const float m0 = g_mean[2 * cp / cg], m1 = g_mean[(2 * cp + 1) / cg];
        float q0 = 0.f, q1 = 0.f;
#pragma unroll
        for (int t = 0; t < GN_CHUNK_TOKENS; ++t) {
            if (t < nt) {
                const float d0 = (float)xv[k][t][0] - m0, d1 = (float)xv[k][t][1] - m1;
                q0 += d0 * d0;
                q1 += d1 * d1;
            }
        }
        chan_acc[2 * cp] = q0;
        chan_acc[2 * cp + 1] = q1;
    }
    __syncthreads();
    for (int g = tid; g < G; g += GN_THREADS) {
        float q = 0.f;
        for (int c = g * cg; c < (g + 1) * cg; ++c) q += chan_acc[c];
        float* st = part + (((int64_t)b * p.chunks + ch) * G + g) * 3;
        st[0] = n_chunk;
        st[1] = g_mean[g];
        st[2] = q;
    }
}

__global__ __launch_bounds__(GN_THREADS) void gn_finalize(GroupNormParams p) {
    __shared__ float mrg[GN_THREADS][3];
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    float* fin = (float*)((char*)p.stats + gn_layout(p.B, p.G, p.chunks).fin);
    // Group statistics of the image from the chunk statistics, in a fixed
    // order: thread (g, j) of S = GN_THREADS / G per group (consecutive
    // threads take consecutive groups: coalesced loads) merges chunks j,
    // j + S, ... (sixteen loads in flight), then thread (g, 0) merges the S
    // results in order j = 0, 1, ...
    const float* part = (const float*)((const char*)p.stats + gn_layout(p.B, p.G, p.chunks).part);
    for (int g0 = 0; g0 < p.G; g0 += GN_THREADS) {
        const int ng = min(p.G - g0, GN_THREADS);
        const int S = GN_THREADS / ng;
        const int g = g0 + tid % ng, j = tid / ng;
        float n = 0.f, mean = 0.f, m2 = 0.f;
        if (tid < ng * S) {
            const float* st = part + ((int64_t)b * p.chunks * p.G + g) * 3;
            for (int k0 = j; k0 < p.chunks; k0 += 16 * S) {
                float cn[16], cm[16], cq[16];
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int k = k0 + u * S;
                    const bool ok = k < p.chunks;
                    const float* r = st + (int64_t)k * p.G * 3;
                    cn[u] = ok ? r[0] : 0.f;
                    cm[u] = ok ? r[1] : 0.f;
                    cq[u] = ok ? r[2] : 0.f;
                }
#pragma unroll
                for (int u = 0; u < 16; ++u) chan_merge(n, mean, m2, cn[u], cm[u], cq[u]);
            }
        }
        mrg[tid][0] = n;
        mrg[tid][1] = mean;
        mrg[tid][2] = m2;
        __syncthreads();
        if (tid < ng) {
            for (int k = 1; k < S; ++k)
                chan_merge(n, mean, m2, mrg[tid + k * ng][0], mrg[tid + k * ng][1], mrg[tid + k * ng][2]);
            if (p.own_out != nullptr) {
                float* o = p.own_out + ((int64_t)b * p.G + g) * 3;
                o[0] = n;
                o[1] = mean;
                o[2] = m2;
            }
            if (p.bands != nullptr) {
                // whole-image statistics: every band's, in band order, this
                // band's own in its place
                float tn = 0.f, tm = 0.f, tq = 0.f;
                for (int j = 0; j < p.n_bands; ++j) {
                    if (j == p.band) {
                        chan_merge(tn, tm, tq, n, mean, m2);
                    } else {
                        const float* o = p.bands + (((int64_t)j * p.B + b) * p.G + g) * 3;
                        chan_merge(tn, tm, tq, o[0], o[1], o[2]);
                    }
                }
                n = tn;
                mean = tm;
                m2 = tq;
            }
            fin[((int64_t)b * p.G + g) * 2] = mean;
            fin[((int64_t)b * p.G + g) * 2 + 1] = n > 0.f ? rsqrtf(m2 / n + p.eps) : 0.f;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(GN_THREADS) void gn_apply(GroupNormParams p) {
    __shared__ float sc[GN_MAX_C];
    __shared__ float sh[GN_MAX_C];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int C = p.C, cg = C / p.G;
    const int tok0 = blockIdx.x * GN_TOKENS_PER_APPLY;
    const int ntok = min(GN_TOKENS_PER_APPLY, p.N - tok0);
    const int vpr = C / 8;  // 16-byte vectors per token row
    const int64_t base = ((int64_t)b * p.N + tok0) * C;
    // The tile's vectors are loaded first, the scale/shift tables meanwhile.
    constexpr int VPT = GN_TOKENS_PER_APPLY * GN_MAX_C / 8 / GN_THREADS;
    bf16x8 xv[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
        const int i = tid + GN_THREADS * k;
        if (i < ntok * vpr) {
            const int t = i / vpr, c = (i - t * vpr) * 8;
            xv[k] = *(const bf16x8*)(p.x + base + (int64_t)t * C + c);
        }
    }
    const GnLayout L = gn_layout(p.B, p.G, p.chunks);
    const float* fin = (const float*)((const char*)p.stats + L.fin) + (int64_t)b * p.G * 2;
    for (int c = tid; c < C; c += GN_THREADS) {
        const int g = c / cg;
        const float a = fin[2 * g + 1] * bf16_to_f32(p.gamma[c]);
        sc[c] = a;
        sh[c] = bf16_to_f32(p.beta[c]) - fin[2 * g] * a;
    }
    __syncthreads();
    const int pad_rows = p.pad_W > 0 ? p.N / p.pad_W : 0;
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
        const int i = tid + GN_THREADS * k;
        if (i < ntok * vpr) {
            const int t = i / vpr, c = (i - t * vpr) * 8;
            bf16x8 y;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float v = __builtin_fmaf((float)xv[k][e], sc[c + e], sh[c + e]);
                if (p.silu) v = v * __builtin_amdgcn_rcpf(1.f + __expf(-v));
                y[e] = f32_to_bf16(v);
            }
            int64_t dst = base + (int64_t)t * C;
            if (p.pad_W > 0) {  // token (row, col) of image b at framed (row + 1, col + 1)
                const int tok = tok0 + t, row = tok / p.pad_W, col = tok - row * p.pad_W;
                dst = ((int64_t)(b * (pad_rows + 2) + row + 1) * (p.pad_W + 2) + col + 1) * C;
            }
            *(bf16x8*)(p.y + dst + c) = y;
        }
    }
}

constexpr int LN_MAX_VEC = 8;  // 16-byte fp32 vectors per lane: C <= 2048

template <int NV>  // 16-byte vectors per lane: C <= 256 * NV
__global__ __launch_bounds__(256) void ln_kernel(LayerNormParams p) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= p.rows) return;
    const int nv = p.C / 4;
    const f32x4* xr = (const f32x4*)(p.x + (int64_t)row * p.C);
    f32x4 v[NV];
    bf16x4 gm[NV], bt[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int j = lane + 64 * k;
        v[k] = j < nv ? xr[j] : f32x4{0.f, 0.f, 0.f, 0.f};
        if (j < nv) {
            gm[k] = *(const bf16x4*)(p.gamma + 4 * j);
            bt[k] = *(const bf16x4*)(p.beta + 4 * j);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) s += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
    float t = s;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o);
    const float mean = t / (float)p.C;
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int j = lane + 64 * k;
        if (j < nv) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float d = v[k][e] - mean;
                q += d * d;
            }
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o);
    const float rstd = rsqrtf(q / (float)p.C + p.eps);
    bf16* yr = p.y + (int64_t)row * p.C;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int j = lane + 64 * k;
        if (j < nv) {
            bf16x4 y;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                y[e] = f32_to_bf16((v[k][e] - mean) * rstd * (float)gm[k][e] + (float)bt[k][e]);
            *(bf16x4*)(yr + 4 * j) = y;
        }
    }
}

int gn_chunks(int N) { return N > 0 ? (N + GN_CHUNK_TOKENS - 1) / GN_CHUNK_TOKENS : 1; }

}  // namespace

size_t group_norm_ws_bytes(int B, int G, int N) { return gn_layout(B, G, gn_chunks(N)).total; }

bool norm_shapes_ok(int C, int G) {
    return C > 0 && C % 8 == 0 && C <= GN_MAX_C && C <= 4 * 64 * LN_MAX_VEC && G > 0 && G <= GN_MAX_G && C % G == 0;
}

hipError_t launch_group_norm(GroupNormParams p, hipStream_t s) {
    if (!norm_shapes_ok(p.C, p.G)) return hipErrorInvalidValue;
    if (p.pad_W < 0 || (p.pad_W > 0 && p.N % p.pad_W != 0)) return hipErrorInvalidValue;
    p.chunks = gn_chunks(p.N);
    gn_stats<<<dim3(p.chunks, p.B), GN_THREADS, 0, s>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    gn_finalize<<<p.B, GN_THREADS, 0, s>>>(p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    gn_apply<<<dim3((p.N + GN_TOKENS_PER_APPLY - 1) / GN_TOKENS_PER_APPLY, p.B), GN_THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_layer_norm(const LayerNormParams& p, hipStream_t s) {
    if (p.C % 4 != 0 || p.C > 4 * 64 * LN_MAX_VEC) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)((p.rows + 3) / 4);
    switch ((p.C + 255) / 256) {
        case 1: ln_kernel<1><<<grid, 256, 0, s>>>(p); break;
        case 2: ln_kernel<2><<<grid, 256, 0, s>>>(p); break;
        case 3: ln_kernel<3><<<grid, 256, 0, s>>>(p); break;
        case 4: ln_kernel<4><<<grid, 256, 0, s>>>(p); break;
        case 5: ln_kernel<5><<<grid, 256, 0, s>>>(p); break;
        case 6: ln_kernel<6><<<grid, 256, 0, s>>>(p); break;
        case 7: ln_kernel<7><<<grid, 256, 0, s>>>(p); break;
        default: ln_kernel<8><<<grid, 256, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

}  // namespace pcpp
