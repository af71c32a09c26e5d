// Internal interface of the block's GEMM and normalisation kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gn_merge.h"

namespace pcpp {

constexpr int GEMM_MAX_WSEG = 16;

// Y[m, n] = X[m, :] . W[n, :] (+ bias[n]) (+ resid[m, n]), optionally
// value * GELU(gate) with the gate taken from W rows F + n.
struct GemmParams {
    const void* a;        // X [M, K], row stride lda (bf16, or fp32 if a_f32)
    int64_t lda;
    int32_t a_f32;
    const __bf16* w;      // W [rows, K] bf16, nn.Linear layout
    const __bf16* bias;   // [rows] or null
    int32_t M, N, K;      // N = output columns
    int32_t geglu;        // 1: output n = (acc_n + b_n) * GELU(acc_{F+n} + b_{F+n})
    int32_t F;            // gate row offset for geglu
    const void* resid;    // [M, N] row stride ldr, or null
    int64_t ldr;
    int32_t resid_f32;
    void* out[3];         // output segments: column n goes to out[n / seg] column n % seg
    int32_t seg;
    int64_t ldo;          // row stride of each output segment
    int32_t out_f32;
    void* out_bf16;       // optional bf16 copy of the output [M, N] (row stride ldo), or null
    // Implicit 3x3 convolution when conv_W > 0 (bf16 a, pipelined kernel
    // only): a is the framed band [B][conv_rows + 2][conv_W + 2][K / 9] (lda
    // unused), token m is (b, y, x) of [B][conv_rows][conv_W], and
    // K = 9 * C_in with k = (3 ky + kx) * C_in + c; C_in % 64 == 0.
    int32_t conv_W = 0, conv_rows = 0;
    // 2: stride 2 (conv_rows and conv_W even): output token (b, y, x) of
    // [B][conv_rows / 2][conv_W / 2] has its tap (0, 0) at framed (2y, 2x).
    int32_t conv_stride = 1;
    // Optional per-image float bias added to output n of token m:
    // bias2[(m / bias2_rows) * N + n] (16-byte aligned), or null.
    const float* bias2 = nullptr;
    int32_t bias2_rows = 1;
    // Workspace that lets the GEMM split K over several workgroups
    // (gemm_split_ws_bytes; its first bytes are counters that must be zero
    // before the first use and are left zero), or null.
    void* split_ws = nullptr;
    size_t split_ws_bytes = 0;
    // Several W matrices sharing X (plain bf16 GEMMs on the pipelined kernel
    // only): W rows [j * w_seg_rows, (j + 1) * w_seg_rows) are the rows of
    // w_seg[j] (w_seg_rows % 128 == 0, N / w_seg_rows <= GEMM_MAX_WSEG);
    // w_seg_rows = 0: w alone.
    const __bf16* w_seg[GEMM_MAX_WSEG] = {};
    int32_t w_seg_rows = 0;
    // > 0: output segment s at out[0] + s * seg_stride elements (out[1..2]
    // unused), for any number of segments.
    int64_t seg_stride = 0;
    // a_mode 1: GroupNorm of X applied while X is staged (bf16 X; K = C <=
    // GEMM_GN_MAXC channels, G <= 256 groups; gn_N tokens per image, a
    // multiple of 64): channel k of token m becomes X * sc + sh with the
    // scale and shift of m's image, from the statistics launch's records in
    // gn (and the other bands' for the synchronized form), in the arithmetic
    // of the GroupNorm apply kernel (the same bits).  Runs on the 64 x 64
    // pipelined kernel; the workgroup holding image b's first token tile and
    // the first W tile writes the band's own statistics to gn.own_out.
    int32_t a_mode = 0;
    GnStatsSrc gn = {};
    const __bf16* gn_gamma = nullptr;
    const __bf16* gn_beta = nullptr;
    int32_t gn_N = 0;
    // a_mode 2: cross-attention in the epilogue (bf16 X and output, N = heads
    // x 64, xa_N tokens per image, a multiple of 64; no bias, residual or
    // copy): the product is the attention's Q, and the workgroup of token
    // tile m and head h goes on to softmax(Q K_h^T / 8) V_h over the xa_T <=
    // 96 keys of its image (xa_k, xa_v: [B][xa_T][xa_ldkv], head h at columns
    // 64 h) and writes that to out[0] in Q's place.
    const __bf16* xa_k = nullptr;
    const __bf16* xa_v = nullptr;
    int32_t xa_T = 0, xa_N = 0;
    int64_t xa_ldkv = 0;
    // Set by launch_gemm for a split launch.
    int32_t splitk = 1, n_xcd = 1, tpx = 0, n_tiles = 0;
};
constexpr int GEMM_GN_MAXC = 1280;
constexpr int GEMM_XA_MAXT = 96;  // keys of the cross-attention epilogue

// Bytes of split-K workspace a GEMM of this shape can use (0: it runs
// unsplit); counters come first, at most GEMM_SPLIT_COUNTERS ints.  conv:
// the implicit convolution (128 x 128 tiles), else a plain bf16 GEMM (64 x 64
// tiles; GEGLU and fp32 X never split).
constexpr int GEMM_SPLIT_COUNTERS = 4096;
size_t gemm_split_ws_bytes(int M, int N, int K, bool conv = true);

bool gemm_shape_ok(const GemmParams& p);
hipError_t launch_gemm(const GemmParams& p, hipStream_t s);
// Two independent products (neither reads what the other writes) in one
// launch when both run on the same pipelined kernel, else one after the other.
hipError_t launch_gemm_pair(const GemmParams& a, const GemmParams& b, hipStream_t s);

// GroupNorm with statistics over one image's tokens (per image and group):
// writes bf16 y = (x - mean) * rsqrt(var + eps) * gamma + beta.
struct GroupNormParams {
    const __bf16* x;      // [B, N, C]
    __bf16* y;            // [B, N, C]
    const __bf16* gamma;
    const __bf16* beta;
    float* stats;         // workspace of group_norm_ws_bytes(B, G, N)
    int32_t B, N, C, G, chunks;  // chunks: set by launch_group_norm
    float eps;
    // Synchronized statistics: [n_bands][B][G] x (count, mean, M2) of every
    // band, entry `band` replaced by this band's own; null = this band's only.
    const float* bands;
    int32_t n_bands, band;
    float* own_out;       // [B][G] x (count, mean, M2) of this band, or null
    int32_t silu = 0;     // 1: y = SiLU(normalized value)
    // pad_W > 0: y is the framed band [B][rows + 2][pad_W + 2][C] of a 3x3
    // convolution (rows = N / pad_W): token (row, col) of image b is written
    // at (row + 1, col + 1); framed row 0 takes row 1 of frame_up
    // [B][2][pad_W][C] (zeros if null), framed row rows + 1 row 0 of
    // frame_dn, the side columns zeros; edges_out [B][2][pad_W][C], if not
    // null, receives the band's rows 0 and rows - 1 (all 16-byte aligned).
    int32_t pad_W = 0;
    const __bf16* frame_up = nullptr;
    const __bf16* frame_dn = nullptr;
    __bf16* edges_out = nullptr;
    // n_zero ints at zero and n_zero2 ints at zero2 (if not null) are cleared
    // by the statistics launch: the work counters of the split GEMMs and of
    // the attention launches that follow on the stream.
    int* zero = nullptr;
    int32_t n_zero = 0;
    int* zero2 = nullptr;
    int32_t n_zero2 = 0;
};
size_t group_norm_ws_bytes(int B, int G, int N);
// C % 8 == 0, C <= 2048, 1 <= G <= 256 divides C.
bool norm_shapes_ok(int C, int G);  // GroupNorm and LayerNorm: C <= 2048
bool gn_shapes_ok(int C, int G);    // GroupNorm alone: C <= 2560
hipError_t launch_group_norm(GroupNormParams p, hipStream_t s);
// The statistics launch alone (sets p.chunks): for a GEMM that applies the
// GroupNorm while staging its operand (GemmParams::a_mode).
hipError_t launch_group_norm_stats(GroupNormParams& p, hipStream_t s);

// LayerNorm over the channel axis of fp32 rows, bf16 output.
struct LayerNormParams {
    const float* x;       // [rows, C]
    __bf16* y;            // [rows, C]
    const __bf16* gamma;
    const __bf16* beta;
    int32_t rows, C;
    float eps;
};
hipError_t launch_layer_norm(const LayerNormParams& p, hipStream_t s);

}  // namespace pcpp
