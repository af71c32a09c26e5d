// pcpp_resnet_block: one SDXL-shaped ResNet block on one row band, the
// U-Net's convolution layers around the partially conditioned attention
// (Sec. 3.3 of arXiv 2412.02962: convolutions keep the exchange of boundary
// pixels, so a band's 3x3 convolution reads its neighbours' edge rows of
// the convolution input from the previous step).
//
// Data flow (all images of the batch stacked as GEMM rows):
//   F1 = frame(SiLU(GroupNorm(x)))        bf16, [B][h+2][W+2][C_in]
//   tb = SiLU(temb) Wt^T + bt             fp32, [B][C_out]
//   h1 = conv3x3(F1) + b1 + tb            bf16  (implicit GEMM, K = 9 C_in)
//   F2 = frame(SiLU(GroupNorm(h1)))       bf16
//   s  = x Ws^T + bs  (C_in != C_out)     fp32, else s = x
//   y  = conv3x3(F2) + b2 + s             bf16  (epilogue residual)
// frame(): GroupNorm's apply writes the band inside a frame one token wide:
// the top frame row takes the band above's last edge row, the bottom one the
// band below's first (zeros at the image's edges), the side columns zeros, so
// every tap of the convolution is one constant offset from a token's framed
// position.  The same kernel exports the band's own first and last rows of
// each convolution input for its neighbours.

#include <math.h>
#include <stdint.h>

#include "../../include/pcpp.h"
#include "common.h"
#include "gemm.h"
#include "kernels.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

constexpr int kThreads = 256;

// tb[b][n] = bt[n] + sum_k SiLU(temb[b][k]) Wt[n][k]: one wavefront per
// output, 16-byte chunks of k per lane.
// Block 0 also clears the convolutions' split counters (n_zero ints), so the
// workspace needs no clearing by the caller.
__global__ __launch_bounds__(kThreads) void temb_proj(float* tb, const bf16* temb, const bf16* wt, const bf16* bt,
                                                      int B, int N, int T, int* zero, int n_zero) {
    if (blockIdx.x == 0 && zero != nullptr)
        for (int i = threadIdx.x; i < n_zero; i += kThreads) zero[i] = 0;
    const int o = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (o >= B * N) return;
    const int b = o / N, n = o - b * N;
    float acc = 0.f;
    for (int k8 = lane; k8 < T / 8; k8 += 64) {
        const bf16x8 e = *(const bf16x8*)(temb + (int64_t)b * T + 8 * k8);
        const bf16x8 w = *(const bf16x8*)(wt + (int64_t)n * T + 8 * k8);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float v = (float)e[j];
            acc += v * __builtin_amdgcn_rcpf(1.f + __expf(-v)) * (float)w[j];
        }
    }
#pragma unroll
    for (int s = 32; s > 0; s >>= 1) acc += __shfl_xor(acc, s);
    if (lane == 0) tb[o] = acc + (bt ? (float)bt[n] : 0.f);
}

struct ResLayout {
    size_t f1, h1, f2, skip, tb, gn, split, split_bytes, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

ResLayout res_layout(const pcpp_resnet_geom_t* g) {
    const size_t B = g->batch, h = g->H / g->n_patches, W = g->W;
    const size_t framed = B * (h + 2) * (W + 2);
    ResLayout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    L.f1 = take(framed * g->c_in * 2);
    L.h1 = take(B * h * W * g->c_out * 2);
    L.f2 = take(framed * g->c_out * 2);
    L.skip = g->c_in != g->c_out ? take(B * h * W * g->c_out * 4) : 0;
    L.tb = take(B * g->c_out * 4);
    L.gn = take(group_norm_ws_bytes(g->batch, g->groups, (int)(h * W)));
    const int M = (int)(B * h * W);
    const size_t s1 = gemm_split_ws_bytes(M, g->c_out, 9 * g->c_in), s2 = gemm_split_ws_bytes(M, g->c_out, 9 * g->c_out);
    L.split_bytes = s1 > s2 ? s1 : s2;
    L.split = L.split_bytes ? take(L.split_bytes) : 0;
    L.total = off;
    return L;
}

int validate_resnet(const pcpp_resnet_geom_t* g) {
    if (g == nullptr || g->reserved != 0) return PCPP_EINVAL;
    if (g->n_patches < 1 || g->H < 1 || g->W < 1 || g->H % g->n_patches != 0) return PCPP_EINVAL;
    if (g->patch_idx < 0 || g->patch_idx >= g->n_patches) return PCPP_EINVAL;
    if (g->batch < 1 || g->batch > 65535) return PCPP_EINVAL;
    if (g->c_in < 1 || g->c_out < 1 || g->groups < 1 || g->temb_dim < 8 || g->temb_dim % 8 != 0)
        return PCPP_EINVAL;
    if (g->c_in % g->groups != 0 || g->c_out % g->groups != 0) return PCPP_EINVAL;
    if (!(g->eps > 0.f) || !isfinite(g->eps)) return PCPP_EINVAL;
    if ((int64_t)(g->H + 2) * (g->W + 2) > INT32_MAX / 4) return PCPP_EINVAL;
    if ((int64_t)g->batch * (g->H / g->n_patches) * g->W > INT32_MAX / 4) return PCPP_EINVAL;
    // the convolution's k-tiles hold 64 channels of one tap
    if (g->c_in % 64 != 0 || g->c_out % 64 != 0) return PCPP_ENOTSUP;
    if (!gn_shapes_ok(g->c_in, g->groups) || !gn_shapes_ok(g->c_out, g->groups)) return PCPP_ENOTSUP;
    return PCPP_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

GemmParams conv_params(const void* framed, const void* w, const void* bias, int M, int N, int K, int h, int W,
                       void* out) {
    GemmParams p;
    p.a = framed;
    p.lda = 0;
    p.a_f32 = 0;
    p.w = (const __bf16*)w;
    p.bias = (const __bf16*)bias;
    p.M = M;
    p.N = N;
    p.K = K;
    p.geglu = 0;
    p.F = 0;
    p.resid = nullptr;
    p.ldr = 0;
    p.resid_f32 = 0;
    p.out[0] = out;
    p.out[1] = p.out[2] = nullptr;
    p.seg = N;
    p.ldo = N;
    p.out_f32 = 0;
    p.out_bf16 = nullptr;
    p.conv_W = W;
    p.conv_rows = h;
    return p;
}

}  // namespace

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT size_t pcpp_resnet_block_workspace_size(const pcpp_resnet_geom_t* g) {
    if (validate_resnet(g) != PCPP_OK) return 0;
    return res_layout(g).total;
}

PCPP_EXPORT int pcpp_resnet_block(const pcpp_resnet_geom_t* g, const pcpp_resnet_weights_t* w, const void* x,
                                  const void* temb, const void* edges1_up, const void* edges1_dn,
                                  const void* edges2_up, const void* edges2_dn, const float* gn1_bands,
                                  float* gn1_own, const float* gn2_bands, float* gn2_own, void* y,
                                  void* edges1_out, void* edges2_out, void* workspace, size_t ws_bytes,
                                  void* stream) {
    int st = validate_resnet(g);
    if (st != PCPP_OK) return st;
    if (w == nullptr) return PCPP_EINVAL;
    const bool proj_skip = g->c_in != g->c_out;
    const void* wptrs[] = {w->gn1_gamma, w->gn1_beta, w->conv1_w, w->conv1_b, w->temb_w, w->temb_b,
                           w->gn2_gamma, w->gn2_beta, w->conv2_w, w->conv2_b};
    for (const void* p : wptrs)
        if (p == nullptr || !aligned16(p)) return PCPP_EINVAL;
    if (proj_skip && (!w->skip_w || !w->skip_b || !aligned16(w->skip_w) || !aligned16(w->skip_b)))
        return PCPP_EINVAL;
    const bool has_up = g->patch_idx > 0, has_dn = g->patch_idx < g->n_patches - 1;
    if (!x || !temb || !y) return PCPP_EINVAL;
    if (has_up && (!edges1_up || !edges2_up)) return PCPP_EINVAL;
    if (has_dn && (!edges1_dn || !edges2_dn)) return PCPP_EINVAL;
    const void* aptrs[] = {x, temb, y, edges1_up, edges1_dn, edges2_up, edges2_dn, edges1_out, edges2_out};
    for (const void* p : aptrs)
        if (p && !aligned16(p)) return PCPP_EINVAL;
    const void* fptrs[] = {gn1_bands, gn1_own, gn2_bands, gn2_own};
    for (const void* p : fptrs)
        if (p && ((uintptr_t)p & 3u) != 0) return PCPP_EINVAL;
    // the exports are written while the neighbours' rows are read: no overlap
    auto overlap = [](const void* a, const void* b, int64_t n) {
        return a && b && (uintptr_t)a < (uintptr_t)b + (uintptr_t)n && (uintptr_t)b < (uintptr_t)a + (uintptr_t)n;
    };
    const int64_t e1 = 4LL * g->batch * g->W * g->c_in, e2 = 4LL * g->batch * g->W * g->c_out;
    if (overlap(edges1_out, edges1_up, e1) || overlap(edges1_out, edges1_dn, e1) ||
        overlap(edges2_out, edges2_up, e2) || overlap(edges2_out, edges2_dn, e2) ||
        (edges1_out && edges2_out && (uintptr_t)edges1_out < (uintptr_t)edges2_out + (uintptr_t)e2 &&
         (uintptr_t)edges2_out < (uintptr_t)edges1_out + (uintptr_t)e1))
        return PCPP_EINVAL;
    const ResLayout L = res_layout(g);
    if (workspace == nullptr || ws_bytes < L.total) return PCPP_EWORKSPACE;
    if (!aligned16(workspace)) return PCPP_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const int B = g->batch, h = g->H / g->n_patches, W = g->W, N = h * W;
    const int Ci = g->c_in, Co = g->c_out, rows = B * N;
    bf16* f1 = (bf16*)(ws + L.f1);
    bf16* h1 = (bf16*)(ws + L.h1);
    bf16* f2 = (bf16*)(ws + L.f2);
    float* skip = proj_skip ? (float*)(ws + L.skip) : nullptr;
    float* tb = (float*)(ws + L.tb);
#define PCPP_CHECK(call)                                   \
    do {                                                   \
        if ((call) != hipSuccess) return PCPP_EHIP;        \
    } while (0)

    auto norm = [&](const void* in, int C, const void* gamma, const void* beta, const float* bands, float* own,
                    bf16* framed, const void* up, const void* dn, void* edges_out) {
        GroupNormParams gp;
        gp.x = (const __bf16*)in;
        gp.y = framed;
        gp.gamma = (const __bf16*)gamma;
        gp.beta = (const __bf16*)beta;
        gp.stats = (float*)(ws + L.gn);
        gp.B = B;
        gp.N = N;
        gp.C = C;
        gp.G = g->groups;
        gp.eps = g->eps;
        gp.bands = bands;
        gp.n_bands = g->n_patches;
        gp.band = g->patch_idx;
        gp.own_out = own;
        gp.silu = 1;
        gp.pad_W = W;
        gp.frame_up = has_up ? (const bf16*)up : nullptr;
        gp.frame_dn = has_dn ? (const bf16*)dn : nullptr;
        gp.edges_out = (bf16*)edges_out;
        return launch_group_norm(gp, s);
    };

    PCPP_CHECK(norm(x, Ci, w->gn1_gamma, w->gn1_beta, gn1_bands, gn1_own, f1, edges1_up, edges1_dn, edges1_out));
    void* split_ws = L.split_bytes ? ws + L.split : nullptr;
    temb_proj<<<(B * Co + 3) / 4, kThreads, 0, s>>>(tb, (const bf16*)temb, (const bf16*)w->temb_w,
                                                   (const bf16*)w->temb_b, B, Co, g->temb_dim, (int*)split_ws,
                                                   split_ws ? GEMM_SPLIT_COUNTERS : 0);
    PCPP_CHECK(hipGetLastError());
    GemmParams c1 = conv_params(f1, w->conv1_w, w->conv1_b, rows, Co, 9 * Ci, h, W, h1);
    c1.bias2 = tb;
    c1.bias2_rows = N;
    c1.split_ws = split_ws;
    c1.split_ws_bytes = L.split_bytes;
    PCPP_CHECK(launch_gemm(c1, s));
    PCPP_CHECK(norm(h1, Co, w->gn2_gamma, w->gn2_beta, gn2_bands, gn2_own, f2, edges2_up, edges2_dn, edges2_out));
    if (proj_skip) {
        GemmParams sp = conv_params(x, w->skip_w, w->skip_b, rows, Co, Ci, 0, 0, skip);
        sp.lda = Ci;
        sp.out_f32 = 1;
        PCPP_CHECK(launch_gemm(sp, s));
    }
    GemmParams c2 = conv_params(f2, w->conv2_w, w->conv2_b, rows, Co, 9 * Co, h, W, y);
    c2.resid = proj_skip ? (const void*)skip : x;
    c2.ldr = Co;
    c2.resid_f32 = proj_skip ? 1 : 0;
    c2.split_ws = split_ws;
    c2.split_ws_bytes = L.split_bytes;
    PCPP_CHECK(launch_gemm(c2, s));
#undef PCPP_CHECK
    return PCPP_OK;
}
