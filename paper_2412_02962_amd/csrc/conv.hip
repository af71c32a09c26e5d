// pcpp_conv3x3: the U-Net's 3x3 convolutions on one row band, with the row
// above and the row below the band taken from the neighbours (Sec. 3.3 of
// arXiv 2412.02962: convolutions keep the exchange of boundary pixels).
//   PCPP_CONV_SAME  stride 1 (conv_in, conv_out, ResNet convolutions)
//   PCPP_CONV_DOWN  stride 2, padding 1 (SDXL's downsampler): reads only the
//                   row above
//   PCPP_CONV_UP    nearest 2x upsampling, then stride 1 (SDXL's upsampler)
// frame_copy writes the band (upsampled for UP) into a [B][Hf+2][Wf+2][C]
// buffer with the neighbour rows on top and bottom (upsampled for UP; zeros
// at the image's edges) and zero side columns; the implicit-GEMM convolution
// of gemm_dma_kernel then reads every tap at one constant offset from a
// token's framed position (stride 2: from (2y, 2x)).

#include <stdint.h>

#include "../../include/pcpp.h"
#include "common.h"
#include "gemm.h"
#include "kernels.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

constexpr int kThreads = 256;

// One 16-byte vector per thread-iteration over the framed buffer of image b:
// framed (fy, fx) with 1 <= fy <= Hf, 1 <= fx <= Wf takes the band's token
// ((fy - 1) / u, (fx - 1) / u) (u = 2 when upsampling, else 1); framed row 0
// takes row_up [B][W][C] at column (fx - 1) / u, row Hf + 1 row_dn (zeros
// when null); columns 0 and Wf + 1 are zeros.  Block 0 also clears the
// convolution's split counters (n_zero ints).  first_out / last_out [B][W][C]
// (if not null) receive the band's first and last rows, what its neighbours
// read as row_dn and row_up at the next step.
__global__ __launch_bounds__(kThreads) void frame_copy(bf16* f, const bf16* x, const bf16* row_up, const bf16* row_dn,
                                                       int h, int W, int C, int u, int* zero, int n_zero,
                                                       bf16* first_out, bf16* last_out) {
    if (blockIdx.x == 0 && blockIdx.y == 0 && zero != nullptr)
        for (int i = threadIdx.x; i < n_zero; i += kThreads) zero[i] = 0;
    const int b = blockIdx.y;
    const int Hf = h * u, Wf = W * u, vpt = C / 8;
    const int64_t total = (int64_t)(Hf + 2) * (Wf + 2) * vpt;
    bf16* fb = f + (int64_t)b * (Hf + 2) * (Wf + 2) * C;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
        const int64_t cell = i / vpt;
        const int c = (int)(i - cell * vpt) * 8;
        const int fy = (int)(cell / (Wf + 2)), fx = (int)(cell - (int64_t)fy * (Wf + 2));
        u32x4 v = {0u, 0u, 0u, 0u};
        if (fx >= 1 && fx <= Wf) {
            const int col = (fx - 1) / u;
            const bf16* src = nullptr;
            if (fy == 0)
                src = row_up ? row_up + ((int64_t)b * W + col) * C : nullptr;
            else if (fy == Hf + 1)
                src = row_dn ? row_dn + ((int64_t)b * W + col) * C : nullptr;
            else
                src = x + (((int64_t)b * h + (fy - 1) / u) * W + col) * C;
            if (src != nullptr) v = *(const u32x4*)(src + c);
            if ((fx - 1) % u == 0) {  // once per band token
                const int64_t o = ((int64_t)b * W + col) * C + c;
                if (fy == 1 && first_out != nullptr) *(u32x4*)(first_out + o) = v;
                if (fy == Hf && last_out != nullptr) *(u32x4*)(last_out + o) = v;
            }
        }
        *(u32x4*)(fb + cell * C + c) = v;
    }
}

struct ConvLayout {
    size_t framed, split, split_bytes, total;
    int h, Hf, Wf, ho, wo;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

ConvLayout conv_layout(const pcpp_conv_geom_t* g) {
    ConvLayout L;
    L.h = g->H / g->n_patches;
    const int u = g->mode == PCPP_CONV_UP ? 2 : 1;
    L.Hf = L.h * u;
    L.Wf = g->W * u;
    const int st = g->mode == PCPP_CONV_DOWN ? 2 : 1;
    L.ho = L.Hf / st;
    L.wo = L.Wf / st;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    L.framed = take((size_t)g->batch * (L.Hf + 2) * (L.Wf + 2) * g->c_in * 2);
    L.split_bytes = gemm_split_ws_bytes(g->batch * L.ho * L.wo, g->c_out, 9 * g->c_in);
    L.split = L.split_bytes ? take(L.split_bytes) : 0;
    L.total = off;
    return L;
}

int validate_conv(const pcpp_conv_geom_t* g) {
    if (g == nullptr || g->reserved != 0) return PCPP_EINVAL;
    if (g->n_patches < 1 || g->H < 1 || g->W < 1 || g->H % g->n_patches != 0) return PCPP_EINVAL;
    if (g->patch_idx < 0 || g->patch_idx >= g->n_patches) return PCPP_EINVAL;
    if (g->batch < 1 || g->batch > 65535 || g->c_in < 1 || g->c_out < 1) return PCPP_EINVAL;
    if (g->mode != PCPP_CONV_SAME && g->mode != PCPP_CONV_DOWN && g->mode != PCPP_CONV_UP) return PCPP_EINVAL;
    const int h = g->H / g->n_patches;
    if (g->mode == PCPP_CONV_DOWN && (h % 2 != 0 || g->W % 2 != 0)) return PCPP_EINVAL;
    if ((int64_t)(2 * g->H + 2) * (2 * g->W + 2) > INT32_MAX / 8) return PCPP_EINVAL;
    if ((int64_t)g->batch * 4 * h * g->W > INT32_MAX / 4) return PCPP_EINVAL;
    // the convolution's k-tiles hold 64 channels of one tap; 64-wide output tiles
    if (g->c_in % 64 != 0 || g->c_out % 64 != 0) return PCPP_ENOTSUP;
    return PCPP_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void* a, int64_t na, const void* b, int64_t nb) {
    if (!a || !b) return false;
    return (uintptr_t)a < (uintptr_t)b + (uintptr_t)nb && (uintptr_t)b < (uintptr_t)a + (uintptr_t)na;
}

}  // namespace

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT size_t pcpp_conv3x3_workspace_size(const pcpp_conv_geom_t* g) {
    if (validate_conv(g) != PCPP_OK) return 0;
    return conv_layout(g).total;
}

PCPP_EXPORT int pcpp_conv3x3_export(const pcpp_conv_geom_t* g, const void* x, const void* row_up,
                                    const void* row_dn, const void* w, const void* bias, void* y, void* first_out,
                                    void* last_out, void* workspace, size_t ws_bytes, void* stream) {
    int st = validate_conv(g);
    if (st != PCPP_OK) return st;
    const bool need_up = g->patch_idx > 0;
    const bool need_dn = g->patch_idx < g->n_patches - 1 && g->mode != PCPP_CONV_DOWN;
    if (!x || !w || !y || (need_up && !row_up) || (need_dn && !row_dn)) return PCPP_EINVAL;
    const void* ptrs[] = {x, row_up, row_dn, w, bias, y, first_out, last_out};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return PCPP_EINVAL;
    {  // the exported rows must not overlap the inputs, the output or each other
        const int hb = g->H / g->n_patches;
        const int64_t row_b = (int64_t)g->batch * g->W * g->c_in * 2;
        const int64_t x_b = row_b * hb;
        const int st_o = g->mode == PCPP_CONV_DOWN ? 2 : 1, u_o = g->mode == PCPP_CONV_UP ? 2 : 1;
        const int64_t y_b = (int64_t)g->batch * (hb * u_o / st_o) * (g->W * u_o / st_o) * g->c_out * 2;
        for (void* e : {first_out, last_out}) {
            if (!e) continue;
            if (overlap(e, row_b, x, x_b) || overlap(e, row_b, row_up, need_up ? row_b : 0) ||
                overlap(e, row_b, row_dn, need_dn ? row_b : 0) || overlap(e, row_b, y, y_b))
                return PCPP_EINVAL;
        }
        if (overlap(first_out, row_b, last_out, row_b)) return PCPP_EINVAL;
    }
    const ConvLayout L = conv_layout(g);
    if (workspace == nullptr || ws_bytes < L.total) return PCPP_EWORKSPACE;
    if (!aligned16(workspace)) return PCPP_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    bf16* framed = (bf16*)(ws + L.framed);
    void* split_ws = L.split_bytes ? ws + L.split : nullptr;
    const int u = g->mode == PCPP_CONV_UP ? 2 : 1;
    const int64_t units = (int64_t)(L.Hf + 2) * (L.Wf + 2) * (g->c_in / 8);
    int64_t blocks = (units + kThreads - 1) / kThreads;
    if (blocks > 2048) blocks = 2048;
    frame_copy<<<dim3((unsigned)blocks, (unsigned)g->batch), kThreads, 0, s>>>(
        framed, (const bf16*)x, need_up ? (const bf16*)row_up : nullptr, need_dn ? (const bf16*)row_dn : nullptr,
        L.h, g->W, g->c_in, u, (int*)split_ws, split_ws ? GEMM_SPLIT_COUNTERS : 0, (bf16*)first_out,
        (bf16*)last_out);
    if (hipGetLastError() != hipSuccess) return PCPP_EHIP;

    GemmParams p;
    p.a = framed;
    p.lda = 0;
    p.a_f32 = 0;
    p.w = (const __bf16*)w;
    p.bias = (const __bf16*)bias;
    p.M = g->batch * L.ho * L.wo;
    p.N = g->c_out;
    p.K = 9 * g->c_in;
    p.geglu = 0;
    p.F = 0;
    p.resid = nullptr;
    p.ldr = 0;
    p.resid_f32 = 0;
    p.out[0] = y;
    p.out[1] = p.out[2] = nullptr;
    p.seg = g->c_out;
    p.ldo = g->c_out;
    p.out_f32 = 0;
    p.out_bf16 = nullptr;
    p.conv_W = L.Wf;
    p.conv_rows = L.Hf;
    p.conv_stride = g->mode == PCPP_CONV_DOWN ? 2 : 1;
    p.split_ws = split_ws;
    p.split_ws_bytes = L.split_bytes;
    return launch_gemm(p, s) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT int pcpp_conv3x3(const pcpp_conv_geom_t* g, const void* x, const void* row_up, const void* row_dn,
                             const void* w, const void* bias, void* y, void* workspace, size_t ws_bytes,
                             void* stream) {
    return pcpp_conv3x3_export(g, x, row_up, row_dn, w, bias, y, nullptr, nullptr, workspace, ws_bytes, stream);
}
