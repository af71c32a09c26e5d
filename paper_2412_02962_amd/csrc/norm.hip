// GroupNorm and LayerNorm (bandwidth-bound).
//
// GroupNorm uses the statistics of the band's own tokens (each image, each
// group of C/G consecutive channels), or with `bands` the whole image's
// (synchronized GroupNorm, Sec. 3.3 of arXiv 2412.02962: every band's
// (count, mean, M2) merged in band order, this band's own in its place).
// Two kernels:
//   gn_stats  one workgroup per chunk of 32 tokens (8 for bands under 2048
//             tokens), held in registers
//             (coalesced channel pairs), reduced to per-group (count, mean,
//             M2) with two passes over the registers (sum, then squared
//             deviations from the chunk mean).
//   gn_apply  every workgroup first merges its image's chunk records with
//             Chan et al.'s pairwise update in a fixed order (so all of them
//             get the same statistics), then the bands, then applies the
//             per-channel scale and shift to 2, 4 or 8 tokens with 16-byte
//             vectors (optionally SiLU).  Workgroup 0 of an image writes the band's
//             own statistics.  In framed mode (the input of a 3x3
//             convolution) it writes into [B][rows+2][W+2][C], and the
//             workgroups also fill the frame (neighbour edge rows or zeros)
//             and export the band's own first and last rows.
// LayerNorm: one wavefront per fp32 row, 16-byte loads, two passes over
// registers (wavefront sums by DPP and lane swaps), 8-byte bf16 stores.

#include <math.h>

#include "common.h"
#include "gemm.h"
#include "gn_merge.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int GN_THREADS = 256;
constexpr int GN_MAX_C = 2560;     // channels (LDS tables of gn_apply; the U-Net's widest concatenation)
constexpr int GN_MAX_G = 256;
// Tokens per statistics workgroup: 32, or 8 when a band has fewer than
// 2048 tokens (so that it still gives about 64 or more workgroups per image
// while the apply merges few chunk records).
constexpr int GN_CHUNK_LONG = 32;
constexpr int GN_CHUNK_SHORT = 8;
__host__ __device__ inline int gn_chunk_tokens(int N) { return N >= 64 * GN_CHUNK_LONG ? GN_CHUNK_LONG : GN_CHUNK_SHORT; }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Lanes that sum one group's channel totals in gn_stats: the largest power of
// two with G of them in the workgroup, at most a wavefront.
__host__ __device__ inline int gn_group_lanes(int G) {
    int t = 1;
    while (2 * t * G <= GN_THREADS && 2 * t <= 64) t *= 2;
    return t;
}

// Workspace of GroupNorm: [B][chunks][G] x (count, mean, M2).
size_t gn_part_bytes(int B, int G, int chunks) { return (size_t)B * G * chunks * 3 * sizeof(float); }

template <int GN_CHUNK_TOKENS, int PP>  // PP: channel pairs per thread, ceil(C / 2 / GN_THREADS)
__global__ __launch_bounds__(GN_THREADS) void gn_stats(GroupNormParams p) {
    __shared__ float chan_acc[GN_MAX_C];
    __shared__ float g_mean[GN_MAX_G];
    const int ch = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x;
    if (ch == 0 && b == 0) {
        if (p.zero != nullptr)
            for (int i = tid; i < p.n_zero; i += GN_THREADS) p.zero[i] = 0;
        if (p.zero2 != nullptr)
            for (int i = tid; i < p.n_zero2; i += GN_THREADS) p.zero2[i] = 0;
    }
    const int C = p.C, G = p.G, cg = C / G, np = C / 2;
    const int t0 = ch * GN_CHUNK_TOKENS;
    const int nt = min(GN_CHUNK_TOKENS, p.N - t0);
    const bf16* xb = p.x + ((int64_t)b * p.N + t0) * C;

    // The chunk's rows, channel pairs per lane, held in registers for both
    // passes (GN_CHUNK_TOKENS tokens, PP pairs per thread): all loads of a
    // thread in flight together.
    bf16x2 xv[PP][GN_CHUNK_TOKENS];
#pragma unroll
    for (int k = 0; k < PP; ++k) {
        const int cp = tid + GN_THREADS * k;
#pragma unroll
        for (int t = 0; t < GN_CHUNK_TOKENS; ++t) {
            bf16x2 v = {};
            if (cp < np && t < nt) v = *(const bf16x2*)(xb + (int64_t)t * C + 2 * cp);
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
    // Per group: T consecutive lanes (a power of two, within one wavefront)
    // each add every T-th channel of the group, then a fixed shuffle tree.
    const int T = gn_group_lanes(G);
    const int gg = tid / T, gu = tid % T;
    auto group_sum = [&]() {
        float v = 0.f;
        if (gg < G)
            for (int c = gg * cg + gu; c < (gg + 1) * cg; c += T) v += chan_acc[c];
        for (int o = 1; o < T; o <<= 1) v += __shfl_xor(v, o);
        return v;
    };
    const float n_chunk = (float)nt * (float)cg;
    {
        const float v = group_sum();
        if (gg < G && gu == 0) g_mean[gg] = v / n_chunk;
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
    {
        const float q = group_sum();
        if (gg < G && gu == 0) {
            float* st = p.stats + (((int64_t)b * p.chunks + ch) * G + gg) * 3;
            st[0] = n_chunk;
            st[1] = g_mean[gg];
            st[2] = q;
        }
    }
}

template <int TPW>  // tokens per workgroup
__global__ __launch_bounds__(GN_THREADS) void gn_apply(GroupNormParams p) {
    __shared__ float sc[GN_MAX_C];
    __shared__ float sh[GN_MAX_C];
    __shared__ float mrg[GN_THREADS][3];
    __shared__ float g_mean[GN_MAX_G], g_rstd[GN_MAX_G];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int C = p.C, G = p.G, cg = C / G;
    const int tok0 = blockIdx.x * TPW;
    const int ntok = min(TPW, p.N - tok0);
    const int vpr = C / 8;  // 16-byte vectors per token row
    const int64_t base = ((int64_t)b * p.N + tok0) * C;
    // The tile's vectors are loaded first, the statistics merged meanwhile.
    constexpr int VPT = (TPW * GN_MAX_C / 8 + GN_THREADS - 1) / GN_THREADS;
    bf16x8 xv[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
        const int i = tid + GN_THREADS * k;
        if (i < ntok * vpr) {
            const int t = i / vpr, c = (i - t * vpr) * 8;
            xv[k] = *(const bf16x8*)(p.x + base + (int64_t)t * C + c);
        }
    }
    // The image's statistics (chunks, then bands), the same code as the GEMM
    // that applies GroupNorm while staging its operand.
    {
        GnStatsSrc src;
        src.stats = p.stats;
        src.chunks = p.chunks;
        src.G = G;
        src.B = p.B;
        src.eps = p.eps;
        src.bands = p.bands;
        src.n_bands = p.n_bands;
        src.band = p.band;
        src.own_out = p.own_out;
        gn_group_stats(src, b, blockIdx.x == 0, &mrg[0][0], g_mean, g_rstd);
    }
    for (int c = tid; c < C; c += GN_THREADS) {
        const int g = c / cg;
        const float a = g_rstd[g] * bf16_to_f32(p.gamma[c]);
        sc[c] = a;
        sh[c] = bf16_to_f32(p.beta[c]) - g_mean[g] * a;
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
            if (p.pad_W > 0) {  // token (row, col) of image b at framed (row + 1, col + 1)
                const int tok = tok0 + t, row = tok / p.pad_W, col = tok - row * p.pad_W;
                const int64_t dst = ((int64_t)(b * (pad_rows + 2) + row + 1) * (p.pad_W + 2) + col + 1) * C;
                *(bf16x8*)(p.y + dst + c) = y;
                if (p.edges_out != nullptr) {  // the band's first and last rows, for its neighbours
                    if (row == 0) *(bf16x8*)(p.edges_out + ((int64_t)(2 * b) * p.pad_W + col) * C + c) = y;
                    if (row == pad_rows - 1)
                        *(bf16x8*)(p.edges_out + ((int64_t)(2 * b + 1) * p.pad_W + col) * C + c) = y;
                }
            } else {
                *(bf16x8*)(p.y + base + (int64_t)t * C + c) = y;
            }
        }
    }
    // Framed mode: the frame of image b, spread over the image's workgroups:
    // framed row 0 (columns 1..W) from row 1 of frame_up [B][2][W][C] or
    // zeros, framed row rows+1 from row 0 of frame_dn or zeros, and zero
    // columns 0 and W+1 of every framed row.
    if (p.pad_W > 0) {
        const int W = p.pad_W;
        const int64_t halo = 2LL * W * vpr;
        const int64_t total = halo + 2LL * (pad_rows + 2) * vpr;
        bf16* fb = p.y + (int64_t)b * (pad_rows + 2) * (W + 2) * C;
        for (int64_t u = (int64_t)blockIdx.x * GN_THREADS + tid; u < total; u += (int64_t)gridDim.x * GN_THREADS) {
            u32x4 v = {0u, 0u, 0u, 0u};
            int64_t dst;
            if (u < halo) {
                const int side = (int)(u / ((int64_t)W * vpr));
                const int64_t jj = u - (int64_t)side * W * vpr;
                const int x = (int)(jj / vpr), c = (int)(jj - (int64_t)x * vpr) * 8;
                const bf16* src = side == 0 ? p.frame_up : p.frame_dn;
                if (src != nullptr) v = *(const u32x4*)(src + ((int64_t)(2 * b + (side == 0 ? 1 : 0)) * W + x) * C + c);
                dst = ((int64_t)(side == 0 ? 0 : pad_rows + 1) * (W + 2) + x + 1) * C + c;
            } else {
                const int64_t jj = u - halo;
                const int row = (int)(jj / (2 * vpr));
                const int rem = (int)(jj - (int64_t)row * 2 * vpr);
                const int col = rem < vpr ? 0 : W + 1;
                const int c = (rem < vpr ? rem : rem - vpr) * 8;
                dst = ((int64_t)row * (W + 2) + col) * C + c;
            }
            *(u32x4*)(fb + dst) = v;
        }
    }
}

constexpr int LN_MAX_VEC = 8;  // 16-byte fp32 vectors per lane: C <= 2048

// Sum over the 64 lanes of a wavefront, the same bits in every lane:
// quad permutes, the half-row and row mirrors (DPP), then the 16- and
// 32-lane swaps; no LDS round trip.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
    v = dpp_add<0xB1>(v);   // quad_perm [1, 0, 3, 2]
    v = dpp_add<0x4E>(v);   // quad_perm [2, 3, 0, 1]
    v = dpp_add<0x141>(v);  // row_half_mirror
    v = dpp_add<0x140>(v);  // row_mirror
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
    const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

template <int NV>  // 16-byte vectors per lane: C <= 256 * NV
__global__ __launch_bounds__(256) void ln_kernel(LayerNormParams p) {
    const int row = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= p.rows) return;
    const int nv = p.C / 4;
    const f32x4* xr = (const f32x4*)(p.x + (int64_t)row * p.C);
    // The row's loads first (all in flight together), then gamma and beta.
    f32x4 v[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int j = lane + 64 * k;
        v[k] = j < nv ? xr[j] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    bf16x4 gm[NV], bt[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int j = lane + 64 * k;
        if (j < nv) {
            gm[k] = *(const bf16x4*)(p.gamma + 4 * j);
            bt[k] = *(const bf16x4*)(p.beta + 4 * j);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) s += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
    const float mean = wave_sum(s) / (float)p.C;
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
    const float rstd = rsqrtf(wave_sum(q) / (float)p.C + p.eps);
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

int gn_chunks(int N) {
    const int ct = gn_chunk_tokens(N);
    return N > 0 ? (N + ct - 1) / ct : 1;
}

}  // namespace

size_t group_norm_ws_bytes(int B, int G, int N) { return gn_part_bytes(B, G, gn_chunks(N)); }

bool gn_shapes_ok(int C, int G) {
    return C > 0 && C % 8 == 0 && C <= GN_MAX_C && G > 0 && G <= GN_MAX_G && C % G == 0;
}

bool norm_shapes_ok(int C, int G) { return gn_shapes_ok(C, G) && C <= 4 * 64 * LN_MAX_VEC; }

hipError_t launch_group_norm_stats(GroupNormParams& p, hipStream_t s) {
    if (!gn_shapes_ok(p.C, p.G)) return hipErrorInvalidValue;
    if (p.pad_W < 0 || (p.pad_W > 0 && p.N % p.pad_W != 0)) return hipErrorInvalidValue;
    p.chunks = gn_chunks(p.N);
    const dim3 grid(p.chunks, p.B);
    const bool lng = gn_chunk_tokens(p.N) == GN_CHUNK_LONG;
    switch ((p.C / 2 + GN_THREADS - 1) / GN_THREADS) {
#define PCPP_GN_STATS(PP)                                                                      \
    case PP:                                                                                   \
        if (lng)                                                                               \
            gn_stats<GN_CHUNK_LONG, PP><<<grid, GN_THREADS, 0, s>>>(p);                         \
        else                                                                                   \
            gn_stats<GN_CHUNK_SHORT, PP><<<grid, GN_THREADS, 0, s>>>(p);                        \
        break;
        PCPP_GN_STATS(1)
        PCPP_GN_STATS(2)
        PCPP_GN_STATS(3)
        PCPP_GN_STATS(4)
        PCPP_GN_STATS(5)
#undef PCPP_GN_STATS
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_group_norm(GroupNormParams p, hipStream_t s) {
    const hipError_t e = launch_group_norm_stats(p, s);
    if (e != hipSuccess) return e;
    // Tokens per apply workgroup: the most of 8, 4 and 2 that still give four
    // workgroups per compute unit over the images (each workgroup merges the
    // statistics records itself, so larger tiles where there are enough of
    // them).  2048 x 640 and 512 x 1280: 2 tokens (the ResNets 2-5 us faster
    // than with 8); 8192 x 320: 8.
    const int cus = device_layout(s).cus;
    int tpw = 8;
    while (tpw > 2 && (int64_t)((p.N + tpw - 1) / tpw) * p.B < 4 * (int64_t)cus) tpw /= 2;
    const dim3 grid((unsigned)((p.N + tpw - 1) / tpw), (unsigned)p.B);
    if (tpw == 8)
        gn_apply<8><<<grid, GN_THREADS, 0, s>>>(p);
    else if (tpw == 4)
        gn_apply<4><<<grid, GN_THREADS, 0, s>>>(p);
    else
        gn_apply<2><<<grid, GN_THREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_layer_norm(const LayerNormParams& p, hipStream_t s) {
    if (p.C % 4 != 0 || p.C > 4 * 64 * LN_MAX_VEC) return hipErrorInvalidValue;
    // One row per wavefront; one wavefront per workgroup, so that short
    // launches still spread over every compute unit.
    const unsigned grid = (unsigned)p.rows;
    switch ((p.C + 255) / 256) {
        case 1: ln_kernel<1><<<grid, 64, 0, s>>>(p); break;
        case 2: ln_kernel<2><<<grid, 64, 0, s>>>(p); break;
        case 3: ln_kernel<3><<<grid, 64, 0, s>>>(p); break;
        case 4: ln_kernel<4><<<grid, 64, 0, s>>>(p); break;
        case 5: ln_kernel<5><<<grid, 64, 0, s>>>(p); break;
        case 6: ln_kernel<6><<<grid, 64, 0, s>>>(p); break;
        case 7: ln_kernel<7><<<grid, 64, 0, s>>>(p); break;
        default: ln_kernel<8><<<grid, 64, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

}  // namespace pcpp
