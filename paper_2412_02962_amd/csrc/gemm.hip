// bf16 GEMM on gfx950 MFMA for the transformer block's linear layers:
//   Y[m, n] = sum_k X[m, k] * W[n, k]  (+ bias[n]) (+ residual[m, n])
// with W in nn.Linear layout [out, in].  Optional GEGLU epilogue: the
// workgroup computes the value columns n and the gate columns F + n of the
// same outputs and writes value * GELU(gate) (exact erf GELU).
//
// The product is computed transposed, Y^T = W X^T, with 32x32x16 MFMAs so
// each lane ends up holding four consecutive output features of one token:
// stores are 8-byte (bf16) or 16-byte (fp32) vectors along the row.
// Tiles: BK = 32, LDS rows padded to 40 elements (conflict-free 16-byte
// operand reads), register-staged double buffering of the next K slice.
// X may be bf16 or fp32 (fp32 is rounded to bf16 while staging).

#include <math.h>

#include "common.h"
#include "gemm.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int BK = 32;
constexpr int LSTR = 40;  // LDS row stride in elements

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: erf(x) = 1 - (a1 t + ... + a5 t^5) exp(-x^2), t = 1 / (1 + p x) for
// x >= 0, odd extension; absolute error at most 1.5e-7, far below the bf16
// rounding of the products it feeds.
__device__ __forceinline__ float erf_as(float x) {
    const float a = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, a, 1.0f));
    float y = __builtin_fmaf(1.061405429f, t, -1.453152027f);
    y = __builtin_fmaf(y, t, 1.421413741f);
    y = __builtin_fmaf(y, t, -0.284496736f);
    y = __builtin_fmaf(y, t, 0.254829592f);
    y *= t;
    const float e = __builtin_amdgcn_exp2f(-a * a * 1.4426950408889634f);
    return copysignf(__builtin_fmaf(-y, e, 1.0f), x);
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f)); }

typedef const __attribute__((address_space(1))) u32x4* gchunk;

template <int V>
struct IC {
    static constexpr int value = V;
};

template <int WMB, int WNB, bool AF32>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    constexpr int BM = 2 * 32 * WMB;           // tokens per workgroup
    constexpr int BNW = 2 * 32 * WNB;          // W-tile rows per workgroup
    constexpr int A_CHUNKS = BM * BK / 8;      // 16-byte bf16 chunks of the X tile
    constexpr int W_CHUNKS = BNW * BK / 8;
    constexpr int A_PER = (A_CHUNKS + 255) / 256;
    constexpr int W_PER = (W_CHUNKS + 255) / 256;

    __shared__ __attribute__((aligned(16))) bf16 a_lds[2][BM * LSTR];
    __shared__ __attribute__((aligned(16))) bf16 w_lds[2][BNW * LSTR];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1;
    const int wn = wave >> 1;
    const int col = lane & 31;
    const int half = lane >> 5;
    const int m0 = blockIdx.x * BM;
    // output columns per workgroup: BNW, or BNW/2 with the GEGLU pairing
    const int bn_out = p.geglu ? BNW / 2 : BNW;
    const int n0 = blockIdx.y * bn_out;

    // global W row of W-tile row r
    auto w_row = [&](int r) -> int {
        if (!p.geglu) return n0 + r;
        return r < BNW / 2 ? n0 + r : p.F + n0 + (r - BNW / 2);
    };

    u32x4 a_reg[A_PER * (AF32 ? 2 : 1)];
    u32x4 w_reg[W_PER];

    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int c = tid + 256 * i;
            const int r = c >> 2, kc = (c & 3) * 8;
            const int m = m0 + r;
            const u32x4 z = {0u, 0u, 0u, 0u};
            if (c < A_CHUNKS && m < p.M) {
                if (AF32) {
                    gchunk src = (gchunk)((const float*)p.a + (int64_t)m * p.lda + k0 + kc);
                    a_reg[2 * i] = src[0];
                    a_reg[2 * i + 1] = src[1];
                } else {
                    a_reg[i] = *(gchunk)((const bf16*)p.a + (int64_t)m * p.lda + k0 + kc);
                }
            } else {
                if (AF32) {
                    a_reg[2 * i] = z;
                    a_reg[2 * i + 1] = z;
                } else {
                    a_reg[i] = z;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < W_PER; ++i) {
            const int c = tid + 256 * i;
            const int r = c >> 2, kc = (c & 3) * 8;
            if (c < W_CHUNKS) w_reg[i] = *(gchunk)(p.w + (int64_t)w_row(r) * p.K + k0 + kc);
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int c = tid + 256 * i;
            if (c >= A_CHUNKS) continue;
            const int r = c >> 2, kc = (c & 3) * 8;
            u32x4 v;
            if (AF32) {
                f32x4 lo = __builtin_bit_cast(f32x4, a_reg[2 * i]);
                f32x4 hi = __builtin_bit_cast(f32x4, a_reg[2 * i + 1]);
                bf16x8 b = {f32_to_bf16(lo[0]), f32_to_bf16(lo[1]), f32_to_bf16(lo[2]), f32_to_bf16(lo[3]),
                            f32_to_bf16(hi[0]), f32_to_bf16(hi[1]), f32_to_bf16(hi[2]), f32_to_bf16(hi[3])};
                v = __builtin_bit_cast(u32x4, b);
            } else {
                v = a_reg[i];
            }
            *(u32x4*)(a_lds[buf] + r * LSTR + kc) = v;
        }
#pragma unroll
        for (int i = 0; i < W_PER; ++i) {
            const int c = tid + 256 * i;
            if (c >= W_CHUNKS) continue;
            const int r = c >> 2, kc = (c & 3) * 8;
            *(u32x4*)(w_lds[buf] + r * LSTR + kc) = w_reg[i];
        }
    };

    f32x16 acc[WNB][WMB];
#pragma unroll
    for (int i = 0; i < WNB; ++i)
#pragma unroll
        for (int j = 0; j < WMB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // W-tile row offset of this wave's n-block i
    auto wrow_off = [&](int i) -> int { return p.geglu ? 32 * wn + (BNW / 2) * i : (BNW / 2) * wn + 32 * i; };

    const int nk = p.K / BK;
    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            bf16x8 wop[WNB], aop[WMB];
#pragma unroll
            for (int i = 0; i < WNB; ++i)
                wop[i] = *(const bf16x8*)(w_lds[buf] + (wrow_off(i) + col) * LSTR + 16 * kk + 8 * half);
#pragma unroll
            for (int j = 0; j < WMB; ++j)
                aop[j] = *(const bf16x8*)(a_lds[buf] + (32 * WMB * wm + 32 * j + col) * LSTR + 16 * kk + 8 * half);
#pragma unroll
            for (int i = 0; i < WNB; ++i)
#pragma unroll
                for (int j = 0; j < WMB; ++j) acc[i][j] = mfma32x32x16(wop[i], aop[j], acc[i][j]);
        }
        if (kt + 1 < nk) store(buf ^ 1);
        __syncthreads();
    }

    // Epilogue: lane holds token m = m-block base + col and features
    // n-block base + 8*c + 4*half + (0..3) in registers 4c..4c+3.
    const int n_blocks_out = p.geglu ? 1 : WNB;
#pragma unroll
    for (int i = 0; i < n_blocks_out; ++i) {
#pragma unroll
        for (int j = 0; j < WMB; ++j) {
            const int m = m0 + 32 * WMB * wm + 32 * j + col;
            if (m >= p.M) continue;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int nloc = p.geglu ? 32 * wn + 8 * c + 4 * half : (BNW / 2) * wn + 32 * i + 8 * c + 4 * half;
                const int n = n0 + nloc;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * c + e];
                if (p.bias != nullptr) {
                    bf16x4 bv = *(const bf16x4*)(p.bias + n);
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] += bf16_to_f32(bv[e]);
                }
                if (WNB == 2 && p.geglu) {
                    float g[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) g[e] = acc[WNB - 1][j][4 * c + e];
                    if (p.bias != nullptr) {
                        bf16x4 bg = *(const bf16x4*)(p.bias + p.F + n);
#pragma unroll
                        for (int e = 0; e < 4; ++e) g[e] += bf16_to_f32(bg[e]);
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] *= gelu_erf(g[e]);
                }
                if (p.resid != nullptr) {
                    if (p.resid_f32) {
                        f32x4 rv = *(const f32x4*)((const float*)p.resid + (int64_t)m * p.ldr + n);
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] += rv[e];
                    } else {
                        bf16x4 rv = *(const bf16x4*)((const bf16*)p.resid + (int64_t)m * p.ldr + n);
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] += bf16_to_f32(rv[e]);
                    }
                }
                const int seg = n / p.seg;
                const int ns = n - seg * p.seg;
                void* dst = p.out[seg];
                if (p.out_f32) {
                    f32x4 o = {v[0], v[1], v[2], v[3]};
                    *(f32x4*)((float*)dst + (int64_t)m * p.ldo + ns) = o;
                } else {
                    bf16x4 o = {f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
                    *(bf16x4*)((bf16*)dst + (int64_t)m * p.ldo + ns) = o;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Pipelined variant for bf16 X and K % 64 == 0: X and W tiles (BK = 64) go
// straight from global memory into LDS (direct global->LDS loads, NS stages
// in flight), MFMA operands are read with explicit LDS waits one k-step
// ahead.  LDS rows are 128 bytes with the 16-byte chunk c of row r stored at
// slot c ^ ((r >> 1) & 7), so 32 consecutive rows read at one chunk are
// conflict-free.  Workgroup: 4 wavefronts in a 2 x 2 layout, each
// computing (BM/2) tokens x (BN/2) W rows.
// ---------------------------------------------------------------------------

constexpr int DBK = 64;

typedef const __attribute__((address_space(1))) void* gvoid;
typedef __attribute__((address_space(3))) void* lvoid;

template <int OFF>
__device__ __forceinline__ u32x4 lds_b128(uint32_t a) {
    u32x4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(a), "n"(OFF));
    return r;
}

// s_waitcnt immediate for vmcnt(v) alone (gfx9 layout: low four bits at
// [3:0], high two at [15:14]; expcnt and lgkmcnt left at their maxima).
constexpr int vmcnt_imm(int v) { return 0xF70 | (v & 15) | ((v >> 4) << 14); }

// Waits until at most later * PT vector loads of this thread are in flight:
// the k-tile `later` tiles before the newest issued one has landed.
template <int PT, int L>
__device__ __forceinline__ void wait_tiles_after(int later) {
    if constexpr (L == 0) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    } else {
        if (later >= L)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(L * PT));
        else
            wait_tiles_after<PT, L - 1>(later);
    }
}

// LDS floats of the GroupNorm table of a_mode 1: scale and shift per
// channel (the merge's 256 x 3 scratch shares their space), then the group
// means and reciprocal deviations.
constexpr int GN_TAB_FLOATS = 2 * GEMM_GN_MAXC + 2 * 256;
// LDS floats of the cross-attention epilogue's K rows and transposed V.
constexpr int XA_TAB_FLOATS = (GEMM_XA_MAXT * 128 + 64 * 200) / 4;
static_assert(2 * GEMM_GN_MAXC >= 3 * 256, "the merge scratch fits the scale and shift tables");

// One workgroup's tile of the product; (bx, by) is its place in the
// product's own grid (blockIdx of a single launch); lds holds NS stages,
// gn_tab GN_TAB_FLOATS floats when AMODE is 1.
//
// AMODE 1 applies GroupNorm to X in its LDS stage: after the products of
// k-tile kt every lane rewrites the pieces of k-tile kt + 1 its own direct
// loads brought, published by the next barrier.
template <int BM, int BN, int NS, bool GEGLU, bool CONV, int AMODE>
__device__ __forceinline__ void gemm_dma_body(const GemmParams& p, const int bx, const int by, char* lds,
                                              float* gn_tab) {
    constexpr bool AGN = AMODE == 1;
    constexpr bool XATT = AMODE == 2;
    static_assert(!(AGN || XATT) || (BM == 64 && BN == 64 && !GEGLU && !CONV), "plain 64 x 64 tiles only");
    constexpr int WMB = BM / 64;                      // 32-token blocks per wavefront
    constexpr int WNB = BN / 64;                      // 32-row W blocks per wavefront
    constexpr int XP = BM / 32;                       // 1 KB X pieces per wavefront per k-tile
    constexpr int WP = BN / 32;
    constexpr int PT = XP + WP;                       // loads per thread per k-tile
    constexpr int STAGE = (BM + BN) * DBK * 2;        // bytes per stage
    constexpr int NOPS = WNB + WMB;                   // operand reads per k-step
    static_assert((NS - 2) * PT <= 63, "vmcnt holds at most 63 loads");
    static_assert(!GEGLU || WNB == 2, "GEGLU pairs a value block with a gate block");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1;
    const int wn = wave >> 1;
    const int col = lane & 31;
    const int half = lane >> 5;
    const int bn_out = GEGLU ? BN / 2 : BN;
    // XCD-contiguous tiles (tpx > 0; always with split K): workgroup w runs
    // on XCD w % n_xcd; the tiles of an XCD are a contiguous range of tpx
    // tiles in n-major order (all token tiles of one W tile together), and
    // the splitk pieces of a tile follow each other within it, so all pieces
    // of a tile share one L2.
    int m_tile = bx, n_tile = by, piece = 0, tile = 0, xcd = 0, tl = 0;
    if (p.tpx > 0) {
        xcd = bx % p.n_xcd;
        const int j = bx / p.n_xcd;
        tl = j / p.splitk;
        piece = j - tl * p.splitk;
        tile = xcd * p.tpx + tl;
        if (tl >= p.tpx || tile >= p.n_tiles) return;  // idle slot of the last XCD (uniform)
        const int mt = (p.M + BM - 1) / BM;
        n_tile = tile / mt;
        m_tile = tile - n_tile * mt;
    }
    const int m0 = m_tile * BM;
    const int n0 = n_tile * bn_out;
    const int nk_all = p.K / DBK;
    const int kt0 = (int)((int64_t)nk_all * piece / p.splitk);
    const int kt1 = (int)((int64_t)nk_all * (piece + 1) / p.splitk);

    // Per-lane global source of each staged piece (row 8q + (lane >> 3),
    // chunk (lane & 7) ^ swizzle), k offset added per k-tile.
    const char* xsrc[XP];
    const char* wsrc[WP];
    const int cin = CONV ? p.K / 9 : 0;
#pragma unroll
    for (int i = 0; i < XP; ++i) {
        const int r = 8 * (wave + 4 * i) + (lane >> 3);
        const int m = min(m0 + r, p.M - 1);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        int64_t row = (int64_t)m * p.lda;
        if constexpr (CONV) {  // the tap (0, 0) of output token (b, y, x) sits at framed (s y, s x)
            const int st = p.conv_stride;
            const int wo = p.conv_W / st;
            const int per = (p.conv_rows / st) * wo;
            const int b = m / per, rem = m - b * per;
            const int y = rem / wo, x = rem - y * wo;
            row = ((int64_t)(b * (p.conv_rows + 2) + st * y) * (p.conv_W + 2) + st * x) * cin;
        }
        xsrc[i] = (const char*)p.a + (row + 8 * c) * 2;
    }
    // Convolution: the k-tiles are issued in order, so the X offset of the
    // next one advances by 64 channels, then to the next tap (one token
    // right, or to the next framed row's first tap column).
    int iss_cb = 0, iss_kx = 0;
    int64_t iss_xoff = 0;
    if (CONV && kt0 > 0) {
        const int cbn = cin / DBK;
        const int t = kt0 / cbn, ky = t / 3;
        iss_cb = kt0 - t * cbn;
        iss_kx = t - 3 * ky;
        iss_xoff = ((int64_t)(ky * (p.conv_W + 2) + iss_kx) * cin + iss_cb * DBK) * 2;
    }
    // W of this tile: one of several matrices when w_seg_rows > 0 (a tile's
    // BN rows never straddle two of them).
    const __bf16* wmat = p.w;
    int wrow0 = n0;
    if (!GEGLU && p.w_seg_rows > 0) {
        const int j = n0 / p.w_seg_rows;
        wmat = p.w_seg[j];
        wrow0 = n0 - j * p.w_seg_rows;
    }
#pragma unroll
    for (int i = 0; i < WP; ++i) {
        const int r = 8 * (wave + 4 * i) + (lane >> 3);
        const int wr = GEGLU ? (r < BN / 2 ? n0 + r : p.F + n0 + (r - BN / 2)) : wrow0 + r;
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        wsrc[i] = (const char*)wmat + ((int64_t)wr * p.K + 8 * c) * 2;
    }
    auto issue = [&](int kt, int stage) {
        char* st = lds + stage * STAGE;
        const int koff = kt * DBK * 2;
        const int64_t xoff = CONV ? iss_xoff : koff;
        if constexpr (CONV) {
            if (++iss_cb * DBK == cin) {
                iss_cb = 0;
                if (++iss_kx == 3) {
                    iss_kx = 0;
                    iss_xoff += ((int64_t)(p.conv_W + 2) * cin - 2 * cin - (cin - DBK)) * 2;
                } else {
                    iss_xoff += DBK * 2;
                }
            } else {
                iss_xoff += DBK * 2;
            }
        }
#pragma unroll
        for (int i = 0; i < XP; ++i)
            __builtin_amdgcn_global_load_lds((gvoid)(xsrc[i] + xoff), (lvoid)(st + (wave + 4 * i) * 1024), 16, 0, 0);
#pragma unroll
        for (int i = 0; i < WP; ++i)
            __builtin_amdgcn_global_load_lds((gvoid)(wsrc[i] + koff), (lvoid)(st + BM * 128 + (wave + 4 * i) * 1024),
                                             16, 0, 0);
    };

    // Operand read addresses: row col of each 32-row block, chunk 2kk + half.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
    const int cmask = (col >> 1) & 7;
    uint32_t chunk_off[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) chunk_off[kk] = ((2 * kk + half) ^ cmask) << 4;
    // W rows of block i: value/gate pairing for GEGLU, else contiguous per wavefront.
    const uint32_t w_row0 = BM * 128 + (GEGLU ? 32 * wn : (BN / 2) * wn) * 128 + col * 128;
    const uint32_t x_row0 = ((BM / 2) * wm + col) * 128;
    constexpr int W_BLOCK_STRIDE = GEGLU ? (BN / 2) * 128 : 32 * 128;

    struct Ops {
        u32x4 w[WNB];
        u32x4 x[WMB];
    };
    auto read_ops = [&](uint32_t sbase, int kk, Ops& o) {
        const uint32_t wa = sbase + w_row0 + chunk_off[kk];
        const uint32_t xa = sbase + x_row0 + chunk_off[kk];
        o.w[0] = lds_b128<0>(wa);
        if constexpr (WNB > 1) o.w[1] = lds_b128<W_BLOCK_STRIDE>(wa);
        o.x[0] = lds_b128<0>(xa);
        if constexpr (WMB > 1) o.x[1] = lds_b128<32 * 128>(xa);
    };
    auto wait_ops = [&](Ops& o, auto n_tag) {
        constexpr int N = decltype(n_tag)::value;
        if constexpr (WNB == 2 && WMB == 2)
            asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(o.w[0]), "+v"(o.w[1]), "+v"(o.x[0]), "+v"(o.x[1]) : "n"(N));
        else if constexpr (WNB == 2)
            asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(o.w[0]), "+v"(o.w[1]), "+v"(o.x[0]) : "n"(N));
        else if constexpr (WMB == 2)
            asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(o.w[0]), "+v"(o.x[0]), "+v"(o.x[1]) : "n"(N));
        else
            asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(o.w[0]), "+v"(o.x[0]) : "n"(N));
    };

    f32x16 acc[WNB][WMB];
#pragma unroll
    for (int i = 0; i < WNB; ++i)
#pragma unroll
        for (int j = 0; j < WMB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // The MFMAs of the k-tile in the stage at LDS address sbase.
    auto mfma_tile = [&](uint32_t sbase) {
        Ops o[2];
        read_ops(sbase, 0, o[0]);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            Ops& cur = o[kk & 1];
            if (kk < 3) {
                read_ops(sbase, kk + 1, o[(kk + 1) & 1]);
                wait_ops(cur, IC<NOPS>{});
            } else {
                wait_ops(cur, IC<0>{});
            }
#pragma unroll
            for (int i = 0; i < WNB; ++i)
#pragma unroll
                for (int j = 0; j < WMB; ++j)
                    acc[i][j] = mfma32x32x16(__builtin_bit_cast(bf16x8, cur.w[i]), __builtin_bit_cast(bf16x8, cur.x[j]),
                                             acc[i][j]);
        }
    };

    // Cross-attention (AMODE 2).  gn_tab holds K_h as rows of 128 bytes (the
    // operand swizzle; keys past xa_T zero) and V_h transposed, a row of
    // 200 bytes per head dimension (keys along the row; 200 keeps the eight-
    // byte reads of 32 dimensions on distinct banks).
    constexpr int XA_VT_STRIDE = 200;
    char* xa = (char*)gn_tab;
    char* xa_vt = xa + GEMM_XA_MAXT * 128;
    auto xatt_stage = [&]() {
        const int img = m0 / p.xa_N;
        const int64_t kvo = (int64_t)img * p.xa_T * p.xa_ldkv + n0;
#pragma unroll
        for (int it = 0; it < GEMM_XA_MAXT * 8 / 256; ++it) {
            const int i = tid + 256 * it;
            const int key = i >> 3, c = i & 7;
            u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
            if (key < p.xa_T) {
                kv = *(const u32x4*)(p.xa_k + kvo + (int64_t)key * p.xa_ldkv + 8 * c);
                vv = *(const u32x4*)(p.xa_v + kvo + (int64_t)key * p.xa_ldkv + 8 * c);
            }
            *(u32x4*)(xa + key * 128 + ((c ^ ((key >> 1) & 7)) << 4)) = kv;
            const bf16x8 v8 = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
            for (int e = 0; e < 8; ++e) *(bf16*)(xa_vt + (8 * c + e) * XA_VT_STRIDE + key * 2) = v8[e];
        }
    };
    // After the product: Q (bf16, rows of 128 bytes) into the first stage,
    // then wavefront (qb, dh) = (w % 2, w / 2) computes S^T = K Q^T for
    // queries 32 qb .. + 31 over all keys (a lane holds one query), the
    // softmax in registers (the key halves meet across lanes l and l ^ 32),
    // and O^T = V^T P^T for head dimensions 32 dh .. + 31.  P^T feeds the
    // matrix product straight from the S^T registers: its k-slot e of lane
    // half h is key 16 u + 8 (e / 4) + 4 h + e % 4 of the step, and V^T is
    // read with the same key order.
    auto xatt_epilogue = [&]() {
        __syncthreads();  // every operand read of the last stage is done
        {
            const int t = 32 * wm + col;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int chunk = 4 * wn + c;  // head dimensions 32 wn + 8 c + 4 half + 0..3
                const bf16x4 q4 = {f32_to_bf16(acc[0][0][4 * c]), f32_to_bf16(acc[0][0][4 * c + 1]),
                                   f32_to_bf16(acc[0][0][4 * c + 2]), f32_to_bf16(acc[0][0][4 * c + 3])};
                *(bf16x4*)(lds + t * 128 + ((chunk ^ ((t >> 1) & 7)) << 4) + 8 * half) = q4;
            }
        }
        __syncthreads();
        const int qb = wave & 1, dh = wave >> 1;
        f32x16 sc[3];
#pragma unroll
        for (int kb = 0; kb < 3; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) sc[kb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int ch = 2 * ks + half;
            const int qr = 32 * qb + col;
            const u32x4 qv = *(const u32x4*)(lds + qr * 128 + ((ch ^ ((qr >> 1) & 7)) << 4));
#pragma unroll
            for (int kb = 0; kb < 3; ++kb) {
                const int kr = 32 * kb + col;
                const u32x4 kv = *(const u32x4*)(xa + kr * 128 + ((ch ^ ((kr >> 1) & 7)) << 4));
                sc[kb] = mfma32x32x16(__builtin_bit_cast(bf16x8, kv), __builtin_bit_cast(bf16x8, qv), sc[kb]);
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 3; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
                if (key >= p.xa_T) sc[kb][r] = -INFINITY;
                mx = fmaxf(mx, sc[kb][r]);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float cl = 1.4426950408889634f * 0.125f;  // log2(e) / sqrt(64)
        const float mcl = mx * cl;
        float l = 0.f;
        bf16x8 pb[3][2];
#pragma unroll
        for (int kb = 0; kb < 3; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const bf16 pr = f32_to_bf16(fast_exp2(__builtin_fmaf(sc[kb][r], cl, -mcl)));
                pb[kb][r >> 3][r & 7] = pr;
                l += bf16_to_f32(pr);  // the weights the products use
            }
        l += __shfl_xor(l, 32);
        f32x16 o;
#pragma unroll
        for (int r = 0; r < 16; ++r) o[r] = 0.f;
        const int d = 32 * dh + col;
#pragma unroll
        for (int kb = 0; kb < 3; ++kb)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int k0 = 32 * kb + 16 * u + 4 * half;
                const u32x2 a0 = *(const u32x2*)(xa_vt + d * XA_VT_STRIDE + k0 * 2);
                const u32x2 a1 = *(const u32x2*)(xa_vt + d * XA_VT_STRIDE + (k0 + 8) * 2);
                const u32x4 av = {a0[0], a0[1], a1[0], a1[1]};
                o = mfma32x32x16(__builtin_bit_cast(bf16x8, av), pb[kb][u], o);
            }
        const int m = m0 + 32 * qb + col;
        if (m >= p.M) return;
        const float inv = 1.f / l;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const bf16x4 ov = {f32_to_bf16(o[4 * q] * inv), f32_to_bf16(o[4 * q + 1] * inv),
                               f32_to_bf16(o[4 * q + 2] * inv), f32_to_bf16(o[4 * q + 3] * inv)};
            *(bf16x4*)((bf16*)p.out[0] + (int64_t)m * p.ldo + n0 + 32 * dh + 8 * q + 4 * half) = ov;
        }
    };

    if constexpr (AGN) {
        // X arrives with the direct loads like W; each lane then rewrites in
        // place the 16-byte pieces its own loads brought (so its own wait
        // suffices), with the GroupNorm applied, before the barrier that
        // publishes the stage.  Piece i of the lane: row 8 (wave + 4 i) +
        // lane / 8, source chunk (lane % 8) ^ ((row / 2) % 8).
        float* sc = gn_tab;
        float* sh = gn_tab + GEMM_GN_MAXC;
        auto gn_rewrite = [&](int kt, int stage) {
#pragma unroll
            for (int i = 0; i < XP; ++i) {
                const int r = 8 * (wave + 4 * i) + (lane >> 3);
                const int c0 = kt * DBK + 8 * ((lane & 7) ^ ((r >> 1) & 7));
                bf16x8* at = (bf16x8*)(lds + stage * STAGE + (wave + 4 * i) * 1024 + lane * 16);
                const bf16x8 v = *at;
                float a[8], b[8];
                *(f32x4*)&a[0] = *(const f32x4*)(sc + c0);
                *(f32x4*)&a[4] = *(const f32x4*)(sc + c0 + 4);
                *(f32x4*)&b[0] = *(const f32x4*)(sh + c0);
                *(f32x4*)&b[4] = *(const f32x4*)(sh + c0 + 4);
                bf16x8 y;
#pragma unroll
                for (int e = 0; e < 8; ++e) y[e] = f32_to_bf16(__builtin_fmaf((float)v[e], a[e], b[e]));
                *at = y;
            }
        };
        // The first two k-tiles in flight while the statistics are merged.
        const int nkt = kt1 - kt0;
        issue(kt0, 0);
        if (nkt > 1) issue(kt0 + 1, 1);
        {
            const int img = m0 / p.gn_N;
            float* g_mean = gn_tab + 2 * GEMM_GN_MAXC;
            float* g_rstd = g_mean + 256;
            gn_group_stats(p.gn, img, m0 == img * p.gn_N && n0 == 0 && piece == 0, gn_tab, g_mean, g_rstd);
            const int cg = p.K / p.gn.G;
            for (int c = tid; c < p.K; c += 256) {
                const int g = c / cg;
                const float a = g_rstd[g] * bf16_to_f32(p.gn_gamma[c]);
                sc[c] = a;
                sh[c] = bf16_to_f32(p.gn_beta[c]) - g_mean[g] * a;
            }
            __syncthreads();
        }
        // X(kt0) landed: after it W(kt0) and, if issued, k-tile kt0 + 1.
        if (nkt > 1)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(WP + PT));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(WP));
        gn_rewrite(kt0, 0);
        for (int kt = kt0; kt < kt1; ++kt) {
            const int i = kt - kt0;
            wait_tiles_after<PT, NS - 2>(min(kt1 - 1 - kt, NS - 2));
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this lane's rewrite of X(kt)
            __builtin_amdgcn_s_barrier();
            if (kt + NS - 1 < kt1) issue(kt + NS - 1, (i + NS - 1) % NS);
            mfma_tile(lds0 + (i % NS) * STAGE);
            if (kt + 1 < kt1) {
                // X(kt + 1) landed: after it W(kt + 1) and, if issued, k-tile kt + 2.
                if (kt + 2 < kt1)
                    __builtin_amdgcn_s_waitcnt(vmcnt_imm(WP + PT));
                else
                    __builtin_amdgcn_s_waitcnt(vmcnt_imm(WP));
                gn_rewrite(kt + 1, (i + 1) % NS);
            }
        }
    } else {
#pragma unroll
        for (int s = 0; s < NS - 1; ++s)
            if (kt0 + s < kt1) issue(kt0 + s, s);
        if constexpr (XATT) xatt_stage();  // its loads wait behind the first k-tiles'
        for (int kt = kt0; kt < kt1; ++kt) {
            // k-tiles issued after kt so far: min(kt1 - 1 - kt, NS - 2), PT loads each
            wait_tiles_after<PT, NS - 2>(min(kt1 - 1 - kt, NS - 2));
            __builtin_amdgcn_s_barrier();  // everyone's pieces of tile kt landed; the stage of tile kt-1 is free
            if (kt + NS - 1 < kt1) issue(kt + NS - 1, (kt - kt0 + NS - 1) % NS);
            mfma_tile(lds0 + ((kt - kt0) % NS) * STAGE);
        }
    }

    if constexpr (XATT) {
        xatt_epilogue();
        return;
    }

    // Split K: every piece stores its partial tile (fp32, 1 KB per wavefront
    // store); the last piece of a tile to arrive adds all of them in piece
    // order (its own from registers: the same values) and runs the epilogue.
    if (p.splitk > 1) {
        __shared__ int last_flag;
        constexpr int NQ = WNB * WMB * 4;  // f32x4 chunks per lane
        auto part_of = [&](int wg) { return (float*)p.split_ws + GEMM_SPLIT_COUNTERS + (int64_t)wg * BM * BN; };
        {
            float* dst = part_of(bx) + (wave * 64 + lane) * 4;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const f32x16& a = acc[q / (4 * WMB)][(q / 4) % WMB];
                const f32x4 v = {a[4 * (q & 3)], a[4 * (q & 3) + 1], a[4 * (q & 3) + 2], a[4 * (q & 3) + 3]};
                *(f32x4*)(dst + q * 1024) = v;
            }
        }
        __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): this thread's stores reached the L2
        __syncthreads();
        if (tid == 0) {
            int* counter = (int*)p.split_ws + tile;
            const int prev = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            const int last = prev == p.splitk - 1;
            if (last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            last_flag = last;
        }
        __syncthreads();
        if (!last_flag) return;
        f32x16 own[WNB][WMB];
#pragma unroll
        for (int i = 0; i < WNB; ++i)
#pragma unroll
            for (int j = 0; j < WMB; ++j) {
                own[i][j] = acc[i][j];
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
            }
        for (int pc = 0; pc < p.splitk; ++pc) {
            if (pc == piece) {
#pragma unroll
                for (int i = 0; i < WNB; ++i)
#pragma unroll
                    for (int j = 0; j < WMB; ++j)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[i][j][r] += own[i][j][r];
                continue;
            }
            const float* src = part_of((tl * p.splitk + pc) * p.n_xcd + xcd) + (wave * 64 + lane) * 4;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const f32x4 v = *(const f32x4*)(src + q * 1024);
                f32x16& a = acc[q / (4 * WMB)][(q / 4) % WMB];
#pragma unroll
                for (int e = 0; e < 4; ++e) a[4 * (q & 3) + e] += v[e];
            }
        }
    }

    // Epilogue: lane holds token (m-block base + col) and W rows
    // (n-block base + 8c + 4*half + 0..3) in registers 4c..4c+3.  All bias
    // and residual loads are issued before the first store: the output may
    // be the residual buffer itself (an in-place update, each element read
    // and written by the same lane), so the compiler could not move a load
    // above an earlier store.
    constexpr int NBO = GEGLU ? 1 : WNB;
    auto n_of = [&](int i, int c) {
        return n0 + (GEGLU ? 32 * wn + 8 * c + 4 * half : (BN / 2) * wn + 32 * i + 8 * c + 4 * half);
    };
    auto m_of = [&](int j) { return m0 + (BM / 2) * wm + 32 * j + col; };
    float bias_v[NBO][4][4], bias_g[4][4];
    f32x4 res_v[NBO][WMB][4];
#pragma unroll
    for (int i = 0; i < NBO; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int n = n_of(i, c);
            bf16x4 bv = {}, bg = {};
            if (p.bias != nullptr) {
                bv = *(const bf16x4*)(p.bias + n);
                if constexpr (GEGLU) bg = *(const bf16x4*)(p.bias + p.F + n);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bias_v[i][c][e] = bf16_to_f32(bv[e]);
                if constexpr (GEGLU) bias_g[c][e] = bf16_to_f32(bg[e]);
            }
#pragma unroll
            for (int j = 0; j < WMB; ++j) {
                const int m = min(m_of(j), p.M - 1);
                f32x4 rv = {0.f, 0.f, 0.f, 0.f};
                if (p.resid != nullptr) {
                    if (p.resid_f32) {
                        rv = *(const f32x4*)((const float*)p.resid + (int64_t)m * p.ldr + n);
                    } else {
                        const bf16x4 rb = *(const bf16x4*)((const bf16*)p.resid + (int64_t)m * p.ldr + n);
#pragma unroll
                        for (int e = 0; e < 4; ++e) rv[e] = bf16_to_f32(rb[e]);
                    }
                }
                if (p.bias2 != nullptr) {
                    const f32x4 b2 = *(const f32x4*)(p.bias2 + (int64_t)(m / p.bias2_rows) * p.N + n);
#pragma unroll
                    for (int e = 0; e < 4; ++e) rv[e] += b2[e];
                }
                res_v[i][j][c] = rv;
            }
        }
#pragma unroll
    for (int i = 0; i < NBO; ++i) {
#pragma unroll
        for (int j = 0; j < WMB; ++j) {
            const int m = m_of(j);
            if (m >= p.M) continue;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int n = n_of(i, c);
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * c + e] + bias_v[i][c][e];
                if constexpr (GEGLU) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] *= gelu_erf(acc[1][j][4 * c + e] + bias_g[c][e]);
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] += res_v[i][j][c][e];
                const int seg = n / p.seg;
                const int ns = n - seg * p.seg;
                void* dst = p.seg_stride > 0
                                ? (void*)((char*)p.out[0] + (int64_t)seg * p.seg_stride * (p.out_f32 ? 4 : 2))
                                : p.out[seg];
                if (p.out_f32) {
                    f32x4 o = {v[0], v[1], v[2], v[3]};
                    *(f32x4*)((float*)dst + (int64_t)m * p.ldo + ns) = o;
                } else {
                    bf16x4 o = {f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
                    *(bf16x4*)((bf16*)dst + (int64_t)m * p.ldo + ns) = o;
                }
                if (p.out_bf16 != nullptr) {
                    bf16x4 o = {f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
                    *(bf16x4*)((bf16*)p.out_bf16 + (int64_t)m * p.ldo + n) = o;
                }
            }
        }
    }
}

template <int BM, int BN, int NS, bool GEGLU, bool CONV, int AMODE>
__global__ __launch_bounds__(256) void gemm_dma_kernel(GemmParams p) {
    __shared__ __attribute__((aligned(16))) char lds[NS * (BM + BN) * DBK * 2];
    __shared__ __attribute__((aligned(16))) float gn_tab[AMODE == 1 ? GN_TAB_FLOATS : AMODE == 2 ? XA_TAB_FLOATS : 4];
    gemm_dma_body<BM, BN, NS, GEGLU, CONV, AMODE>(p, blockIdx.x, blockIdx.y, lds, gn_tab);
}

// Two independent plain products in one launch (so that neither pays a
// launch's fixed cost alone): workgroups [0, n_a) run `a`, [b0, b0 + n_b)
// run `b`, each product's grid linearised x-fastest; b0 is a multiple of the
// XCD count, so a product on XCD-ordered tiles keeps its workgroup-to-XCD
// map; the workgroups in between exit at once.
struct GemmPair {
    GemmParams a, b;
    int32_t gx_a, n_a, gx_b, b0;
};

template <int BM, int BN, int NS, int AMODE_A>
__global__ __launch_bounds__(256) void gemm_dma_pair_kernel(GemmPair pp) {
    __shared__ __attribute__((aligned(16))) char lds[NS * (BM + BN) * DBK * 2];
    __shared__ __attribute__((aligned(16))) float gn_tab[AMODE_A == 1 ? GN_TAB_FLOATS : 4];
    const int id = blockIdx.x;
    if (id < pp.n_a)
        gemm_dma_body<BM, BN, NS, false, false, AMODE_A>(pp.a, id % pp.gx_a, id / pp.gx_a, lds, gn_tab);
    else if (id >= pp.b0)
        gemm_dma_body<BM, BN, NS, false, false, 0>(pp.b, (id - pp.b0) % pp.gx_b, (id - pp.b0) / pp.gx_b, lds, gn_tab);
}

// ---------------------------------------------------------------------------
// Balanced tiles for products whose 64 x 64 tiles do not divide evenly over
// the compute units: 64 tokens x 80 W rows per workgroup, so that a
// 2048 x 640 product is 256 tiles, one per compute unit (64 x 64 tiles give
// 320: a quarter of the compute units would run two, and the launch lasts
// as long as they do).  Y^T = W X^T with 16x16x32 MFMAs (a lane ends up with
// four consecutive outputs of one token).  Eight wavefronts: wavefront w
// takes tokens 16 (w % 4) .. + 15 and k-step w / 4 of the two 32-long steps
// of every 64-long k-tile, for all 80 rows (five 16-row blocks); the two
// k-steps' sums meet through LDS at the end.  X and W go straight into LDS
// in the row layout and swizzle of the kernel above: 18 pieces of 1 KB per
// k-tile (8 of X, 10 of W), piece j loaded by wavefront j % 8; NS stages
// (4 with one tile per compute unit, 2 when several share one).
// ---------------------------------------------------------------------------
constexpr int G80_BM = 64, G80_BN = 80;
constexpr int G80_STAGE = (G80_BM + G80_BN) * DBK * 2;  // 18 KB

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int NS>
__global__ __launch_bounds__(512) void gemm80_kernel(GemmParams p) {
    __shared__ __attribute__((aligned(16))) char lds[NS * G80_STAGE];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tb = wave & 3, kg = wave >> 2;
    const int m0 = blockIdx.x * G80_BM, n0 = blockIdx.y * G80_BN;
    const int nk = p.K / DBK;

    // Pieces j = wave + 8 q of this wavefront: LDS rows 8 j .. 8 j + 7 of the
    // stage (X rows 0..63, then W rows 64..143); lane: row 8 j + lane / 8,
    // chunk (lane % 8) ^ ((row / 2) % 8).
    const char* src[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
        const int j = wave + 8 * q;
        const int row = 8 * j + (lane >> 3);
        const int c = (lane & 7) ^ ((row >> 1) & 7);
        if (row < G80_BM) {
            const int m = min(m0 + row, p.M - 1);
            src[q] = (const char*)p.a + ((int64_t)m * p.lda + 8 * c) * 2;
        } else {
            src[q] = (const char*)p.w + ((int64_t)(n0 + min(row, G80_BM + G80_BN - 1) - G80_BM) * p.K + 8 * c) * 2;
        }
    }
    const bool three = wave < 2;  // 18 pieces: wavefronts 0 and 1 load a third
    auto issue = [&](int kt, int stage) {
        char* st = lds + stage * G80_STAGE;
        const int koff = kt * DBK * 2;
#pragma unroll
        for (int q = 0; q < 2; ++q)
            __builtin_amdgcn_global_load_lds((gvoid)(src[q] + koff), (lvoid)(st + (wave + 8 * q) * 1024), 16, 0, 0);
        if (three)
            __builtin_amdgcn_global_load_lds((gvoid)(src[2] + koff), (lvoid)(st + (wave + 16) * 1024), 16, 0, 0);
    };

    // Operands of k-step kg: X rows 16 tb + lane % 16 (B, tokens), W rows
    // 64 + 16 fb + lane % 16 (A, W rows), k-octet lane / 16 of the step.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
    const int chunk = 4 * kg + (lane >> 4);
    const int xr = 16 * tb + (lane & 15);
    const uint32_t xoff = xr * 128 + ((chunk ^ ((xr >> 1) & 7)) << 4);
    uint32_t woff[5];
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) {
        const int r = G80_BM + 16 * fb + (lane & 15);
        woff[fb] = r * 128 + ((chunk ^ ((r >> 1) & 7)) << 4);
    }
    f32x4 acc[5];
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) acc[fb] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int st = 0; st < NS - 1; ++st)
        if (st < nk) issue(st, st);
    for (int kt = 0; kt < nk; ++kt) {
        const int later = min(nk - 1 - kt, NS - 2);
        if (three)
            wait_tiles_after<3, NS - 2>(later);
        else
            wait_tiles_after<2, NS - 2>(later);
        __builtin_amdgcn_s_barrier();  // everyone's pieces of tile kt landed; the stage of tile kt-1 is free
        if (kt + NS - 1 < nk) issue(kt + NS - 1, (kt + NS - 1) % NS);
        const uint32_t sb = lds0 + (kt % NS) * G80_STAGE;
        u32x4 x = lds_b128<0>(sb + xoff);
        u32x4 w0 = lds_b128<0>(sb + woff[0]);
        u32x4 w1 = lds_b128<0>(sb + woff[1]);
        u32x4 w2 = lds_b128<0>(sb + woff[2]);
        u32x4 w3 = lds_b128<0>(sb + woff[3]);
        u32x4 w4 = lds_b128<0>(sb + woff[4]);
        asm volatile("s_waitcnt lgkmcnt(4)" : "+v"(x), "+v"(w0));
        acc[0] = mfma16x16x32(__builtin_bit_cast(bf16x8, w0), __builtin_bit_cast(bf16x8, x), acc[0]);
        asm volatile("s_waitcnt lgkmcnt(3)" : "+v"(w1));
        acc[1] = mfma16x16x32(__builtin_bit_cast(bf16x8, w1), __builtin_bit_cast(bf16x8, x), acc[1]);
        asm volatile("s_waitcnt lgkmcnt(2)" : "+v"(w2));
        acc[2] = mfma16x16x32(__builtin_bit_cast(bf16x8, w2), __builtin_bit_cast(bf16x8, x), acc[2]);
        asm volatile("s_waitcnt lgkmcnt(1)" : "+v"(w3));
        acc[3] = mfma16x16x32(__builtin_bit_cast(bf16x8, w3), __builtin_bit_cast(bf16x8, x), acc[3]);
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(w4));
        acc[4] = mfma16x16x32(__builtin_bit_cast(bf16x8, w4), __builtin_bit_cast(bf16x8, x), acc[4]);
    }

    // The two k-steps' sums: wavefront (tb, 0) finishes blocks 0-2, (tb, 1)
    // blocks 3-4; each hands the other its sums of the other's blocks.
    __syncthreads();  // every wavefront is past its last LDS operand read
    float* red = (float*)lds;  // [tb][block][lane] x 4 floats (20 KB)
    auto owned = [&](int fb) { return kg == 0 ? fb < 3 : fb >= 3; };
#pragma unroll
    for (int fb = 0; fb < 5; ++fb)
        if (!owned(fb)) *(f32x4*)(red + ((tb * 5 + fb) * 64 + lane) * 4) = acc[fb];
    __syncthreads();
#pragma unroll
    for (int fb = 0; fb < 5; ++fb)
        if (owned(fb)) acc[fb] += *(const f32x4*)(red + ((tb * 5 + fb) * 64 + lane) * 4);

    // Epilogue: token m0 + 16 tb + lane % 16, W rows n0 + 16 fb + 4 (lane / 16)
    // + 0..3; all bias and residual loads before the first store (the output
    // may be the residual buffer itself).
    const int m = m0 + 16 * tb + (lane & 15);
    const int mc = min(m, p.M - 1);
    // The epilogue keeps the order of the 64 x 64 kernel: (acc + bias) + residual.
    f32x4 bias_v[5], res_v[5];
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) {
        bias_v[fb] = f32x4{0.f, 0.f, 0.f, 0.f};
        res_v[fb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (!owned(fb)) continue;
        const int n = n0 + 16 * fb + 4 * (lane >> 4);
        if (p.bias != nullptr) {
            const bf16x4 bv = *(const bf16x4*)(p.bias + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) bias_v[fb][e] = bf16_to_f32(bv[e]);
        }
        if (p.resid != nullptr) {
            if (p.resid_f32) {
                res_v[fb] = *(const f32x4*)((const float*)p.resid + (int64_t)mc * p.ldr + n);
            } else {
                const bf16x4 rb = *(const bf16x4*)((const bf16*)p.resid + (int64_t)mc * p.ldr + n);
#pragma unroll
                for (int e = 0; e < 4; ++e) res_v[fb][e] = bf16_to_f32(rb[e]);
            }
        }
    }
    if (m >= p.M) return;
    const int sg = n0 / p.seg;  // output segment of the whole tile (80 divides the segment width)
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) {
        if (!owned(fb)) continue;
        const int n = n0 + 16 * fb + 4 * (lane >> 4);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (acc[fb][e] + bias_v[fb][e]) + res_v[fb][e];
        const int ns = n - sg * p.seg;
        if (p.out_f32) {
            *(f32x4*)((float*)p.out[sg] + (int64_t)m * p.ldo + ns) = f32x4{v[0], v[1], v[2], v[3]};
        } else {
            const bf16x4 o = {f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
            *(bf16x4*)((bf16*)p.out[sg] + (int64_t)m * p.ldo + ns) = o;
        }
        if (p.out_bf16 != nullptr) {
            const bf16x4 o = {f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
            *(bf16x4*)((bf16*)p.out_bf16 + (int64_t)m * p.ldo + n) = o;
        }
    }
}

// ---------------------------------------------------------------------------
// GEGLU on balanced tiles: BM tokens x 160 outputs (their 160 value rows and
// 160 gate rows of W) per workgroup, so that the block's 2048 x 2560 product
// (BM = 128) and the level-2 512 x 5120 product (BM = 64) are 256 tiles, one
// per compute unit.  16x16x32 MFMAs, Y^T = W X^T; eight wavefronts, each
// holding the value and the gate of the same outputs, so the GELU product is
// formed in registers.  BM = 128: wavefront w takes tokens 32 (w % 4) .. + 31
// and outputs 80 (w / 4) .. + 79.  BM = 64: wavefront w takes tokens
// 32 (w % 2) .. + 31, outputs 80 ((w / 2) % 2) .. + 79 and k-step w / 4 of
// the two 32-long steps of each k-tile; the two k-steps' sums meet through
// LDS at the end.  LDS stage: X rows, then value rows, then gate rows, 128
// bytes each (the swizzle above): 448 rows (56 KB, two stages) or 384 rows
// (48 KB, three stages); 1 KB direct-load pieces, the same number per
// wavefront.  With tpx > 0 the tiles run in XCD-contiguous n-major order (W
// at least four times X: a W tile is then fetched into one XCD's L2).
// ---------------------------------------------------------------------------
constexpr int GG_BN = 160;

template <int GBM>
struct GegluShape {
    static constexpr int ROWS = GBM + 2 * GG_BN;
    static constexpr int STAGE = ROWS * DBK * 2;
    static constexpr int NS = GBM == 128 ? 2 : 3;
    static constexpr int PT = ROWS / 8 / 8;  // pieces per wavefront per k-tile
    static constexpr bool KSPLIT = GBM == 64;
};

template <int GBM>
__global__ __launch_bounds__(512) void geglu160_kernel(GemmParams p) {
    using SH = GegluShape<GBM>;
    __shared__ __attribute__((aligned(16))) char lds[SH::NS * SH::STAGE];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tb = SH::KSPLIT ? (wave & 1) : (wave & 3);
    const int vg = SH::KSPLIT ? ((wave >> 1) & 1) : (wave >> 2);
    const int kg = SH::KSPLIT ? (wave >> 2) : 0;
    int m_tile = blockIdx.x, n_tile = blockIdx.y;
    if (p.tpx > 0) {  // XCD-contiguous: workgroup w on XCD w % n_xcd, n-major within an XCD
        const int xcd = blockIdx.x % p.n_xcd;
        const int tl = blockIdx.x / p.n_xcd;
        const int tile = xcd * p.tpx + tl;
        if (tl >= p.tpx || tile >= p.n_tiles) return;  // idle slot of the last XCD (uniform)
        const int mt = (p.M + GBM - 1) / GBM;
        n_tile = tile / mt;
        m_tile = tile - n_tile * mt;
    }
    const int m0 = m_tile * GBM, n0 = n_tile * GG_BN;
    const int nk = p.K / DBK;

    const char* src[SH::PT];
#pragma unroll
    for (int q = 0; q < SH::PT; ++q) {
        const int row = 8 * (wave + 8 * q) + (lane >> 3);
        const int c = (lane & 7) ^ ((row >> 1) & 7);
        int64_t grow;
        const __bf16* base;
        if (row < GBM) {
            base = (const __bf16*)p.a;
            grow = (int64_t)min(m0 + row, p.M - 1) * p.lda;
        } else {
            base = p.w;
            const int r = row - GBM;
            grow = (int64_t)(r < GG_BN ? n0 + r : p.F + n0 + (r - GG_BN)) * p.K;
        }
        src[q] = (const char*)(base + grow + 8 * c);
    }
    auto issue = [&](int kt, int stage) {
        char* st = lds + stage * SH::STAGE;
        const int koff = kt * DBK * 2;
#pragma unroll
        for (int q = 0; q < SH::PT; ++q)
            __builtin_amdgcn_global_load_lds((gvoid)(src[q] + koff), (lvoid)(st + (wave + 8 * q) * 1024), 16, 0, 0);
    };

    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
    // Row offsets (chunk added per k-step): X blocks j, value and gate blocks fb.
    uint32_t xrow[2], vrow[5], grow_[5];
    int xsw[2], vsw[5], gsw[5];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int r = 32 * tb + 16 * j + (lane & 15);
        xrow[j] = r * 128;
        xsw[j] = (r >> 1) & 7;
    }
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) {
        const int rv = GBM + 80 * vg + 16 * fb + (lane & 15);
        const int rg = rv + GG_BN;
        vrow[fb] = rv * 128;
        vsw[fb] = (rv >> 1) & 7;
        grow_[fb] = rg * 128;
        gsw[fb] = (rg >> 1) & 7;
    }
    f32x4 accv[2][5], accg[2][5];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int fb = 0; fb < 5; ++fb) accv[j][fb] = accg[j][fb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // The MFMAs of k-step ks of the stage at sb.
    auto kstep = [&](uint32_t sb, int ks) {
        const int chunk = 4 * ks + (lane >> 4);
        u32x4 x[2], v[5], g[5];
#pragma unroll
        for (int j = 0; j < 2; ++j) x[j] = lds_b128<0>(sb + xrow[j] + ((chunk ^ xsw[j]) << 4));
#pragma unroll
        for (int fb = 0; fb < 5; ++fb) {
            v[fb] = lds_b128<0>(sb + vrow[fb] + ((chunk ^ vsw[fb]) << 4));
            g[fb] = lds_b128<0>(sb + grow_[fb] + ((chunk ^ gsw[fb]) << 4));
        }
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(x[0]), "+v"(x[1]), "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]),
                       "+v"(g[0]), "+v"(g[1]), "+v"(g[2]), "+v"(g[3]), "+v"(g[4]));
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int fb = 0; fb < 5; ++fb) {
                accv[j][fb] = mfma16x16x32(__builtin_bit_cast(bf16x8, v[fb]), __builtin_bit_cast(bf16x8, x[j]),
                                           accv[j][fb]);
                accg[j][fb] = mfma16x16x32(__builtin_bit_cast(bf16x8, g[fb]), __builtin_bit_cast(bf16x8, x[j]),
                                           accg[j][fb]);
            }
    };

#pragma unroll
    for (int st = 0; st < SH::NS - 1; ++st)
        if (st < nk) issue(st, st);
    for (int kt = 0; kt < nk; ++kt) {
        wait_tiles_after<SH::PT, SH::NS - 2>(min(nk - 1 - kt, SH::NS - 2));
        __builtin_amdgcn_s_barrier();  // everyone's pieces of tile kt landed; the stage of tile kt-1 is free
        if (kt + SH::NS - 1 < nk) issue(kt + SH::NS - 1, (kt + SH::NS - 1) % SH::NS);
        const uint32_t sb = lds0 + (kt % SH::NS) * SH::STAGE;
        if constexpr (SH::KSPLIT) {
            kstep(sb, kg);
        } else {
            kstep(sb, 0);
            kstep(sb, 1);
        }
    }

    // BM = 64: wavefront (tb, vg, 1) hands its sums to (tb, vg, 0), which
    // finishes the outputs.
    if constexpr (SH::KSPLIT) {
        __syncthreads();  // every wavefront is past its last LDS operand read
        float* red = (float*)lds + ((tb * 2 + vg) * 20) * 64 * 4;  // 20 f32x4 per lane
        if (kg == 1) {
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int fb = 0; fb < 5; ++fb) {
                    *(f32x4*)(red + ((j * 5 + fb) * 64 + lane) * 4) = accv[j][fb];
                    *(f32x4*)(red + ((10 + j * 5 + fb) * 64 + lane) * 4) = accg[j][fb];
                }
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int fb = 0; fb < 5; ++fb) {
                accv[j][fb] += *(const f32x4*)(red + ((j * 5 + fb) * 64 + lane) * 4);
                accg[j][fb] += *(const f32x4*)(red + ((10 + j * 5 + fb) * 64 + lane) * 4);
            }
    }

    // Epilogue: token m0 + 32 tb + 16 j + lane % 16, outputs n0 + 80 vg + 16 fb
    // + 4 (lane / 16) + 0..3: (value + bias) * GELU(gate + gate bias).
#pragma unroll
    for (int fb = 0; fb < 5; ++fb) {
        const int n = n0 + 80 * vg + 16 * fb + 4 * (lane >> 4);
        float bv[4] = {0.f, 0.f, 0.f, 0.f}, bg[4] = {0.f, 0.f, 0.f, 0.f};
        if (p.bias != nullptr) {
            const bf16x4 b1 = *(const bf16x4*)(p.bias + n);
            const bf16x4 b2 = *(const bf16x4*)(p.bias + p.F + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bv[e] = bf16_to_f32(b1[e]);
                bg[e] = bf16_to_f32(b2[e]);
            }
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int m = m0 + 32 * tb + 16 * j + (lane & 15);
            if (m >= p.M) continue;
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = (accv[j][fb][e] + bv[e]) * gelu_erf(accg[j][fb][e] + bg[e]);
            if (p.out_f32) {
                *(f32x4*)((float*)p.out[0] + (int64_t)m * p.ldo + n) = f32x4{o[0], o[1], o[2], o[3]};
            } else {
                const bf16x4 ob = {f32_to_bf16(o[0]), f32_to_bf16(o[1]), f32_to_bf16(o[2]), f32_to_bf16(o[3])};
                *(bf16x4*)((bf16*)p.out[0] + (int64_t)m * p.ldo + n) = ob;
            }
        }
    }
}

template <int BM, int BN, int NS, bool GEGLU>
hipError_t launch_dma(const GemmParams& p, hipStream_t s) {
    const int bn_out = GEGLU ? BN / 2 : BN;
    dim3 grid((p.M + BM - 1) / BM, p.N / bn_out);
    if (p.tpx > 0) grid = dim3((unsigned)(p.n_xcd * p.tpx * p.splitk), 1);
    if constexpr (!GEGLU && BM == 64 && BN == 64) {
        if (p.a_mode == 1) {
            gemm_dma_kernel<BM, BN, NS, false, false, 1><<<grid, 256, 0, s>>>(p);
            return hipGetLastError();
        }
        if (p.a_mode == 2) {
            gemm_dma_kernel<BM, BN, NS, false, false, 2><<<grid, 256, 0, s>>>(p);
            return hipGetLastError();
        }
    }
    if (!GEGLU && p.conv_W > 0)
        gemm_dma_kernel<BM, BN, NS, GEGLU, true, 0><<<grid, 256, 0, s>>>(p);
    else
        gemm_dma_kernel<BM, BN, NS, GEGLU, false, 0><<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

template <int WMB, int WNB>
hipError_t launch_shape(const GemmParams& p, hipStream_t s) {
    constexpr int BM = 64 * WMB;
    const int bn_out = p.geglu ? 32 * WNB : 64 * WNB;
    dim3 grid((p.M + BM - 1) / BM, p.N / bn_out);
    if (p.a_f32)
        gemm_kernel<WMB, WNB, true><<<grid, 256, 0, s>>>(p);
    else
        gemm_kernel<WMB, WNB, false><<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace

bool gemm_shape_ok(const GemmParams& p) {
    if (p.K % BK != 0 || p.M < 1 || p.N < 1) return false;
    if (p.bias2 != nullptr && (p.bias2_rows < 1 || p.N % 4 != 0)) return false;
    if (p.conv_W > 0) {
        const int st = p.conv_stride;
        if ((st != 1 && st != 2) || (st == 2 && (p.conv_rows % 2 != 0 || p.conv_W % 2 != 0))) return false;
        return !p.a_f32 && !p.geglu && p.conv_rows > 0 && p.K % (9 * DBK) == 0 && p.N % 64 == 0 &&
               p.seg % 4 == 0 && p.M % ((p.conv_rows / st) * (p.conv_W / st)) == 0;
    }
    if (p.geglu) return p.N % 64 == 0;  // two n-blocks of 32 per workgroup pair
    return p.N % 64 == 0 && p.seg % 4 == 0;
}

namespace {

// Split of a convolution GEMM over 128 x 128 tiles: as many pieces per tile
// as still fit one workgroup per compute unit, each at least 16 k-tiles
// long, used only when the split launch fills at least 90% of the compute
// units (else the unsplit 64 x 64 tiles, two workgroups per compute unit,
// are faster).
struct SplitPlan {
    int splitk, n_xcd, tpx, n_tiles;
    size_t bytes;
};

SplitPlan split_plan(int M, int N, int K, const DeviceLayout& d) {
    SplitPlan sp{1, 1, 0, 0, 0};
    const int cus = d.cus;
    if (!d.xcd_merge || N % 128 != 0 || K % DBK != 0) return sp;
    const int64_t tiles = (int64_t)((M + 127) / 128) * (N / 128);
    if (tiles < 1 || tiles > GEMM_SPLIT_COUNTERS) return sp;
    const int n_xcd = d.n_xcd;
    const int64_t tpx = (tiles + n_xcd - 1) / n_xcd;
    int64_t k = cus / (n_xcd * tpx);
    const int64_t k_max = (K / DBK) / 16;
    if (k > k_max) k = k_max;
    if (k > 8) k = 8;
    if (k < 2 || 10 * n_xcd * tpx * k < 9 * (int64_t)cus) return sp;
    sp.splitk = (int)k;
    sp.n_xcd = n_xcd;
    sp.tpx = (int)tpx;
    sp.n_tiles = (int)tiles;
    sp.bytes = (size_t)GEMM_SPLIT_COUNTERS * 4 + (size_t)n_xcd * tpx * k * 128 * 128 * 4;
    return sp;
}

// Split of a plain GEMM over 64 x 64 tiles when they are fewer than the
// compute units (one workgroup per compute unit and the rest idle): about
// kSplitTarget workgroups per compute unit, each piece at least
// kSplitMinTiles k-tiles long.  Measured at 512 x 1280 (2048 px level 2):
// K = 5120 in 3 pieces 21.4 us against 25.8 unsplit (4 or 5 pieces, from a
// target of 3 or 4 workgroups per compute unit: the level-2 block 4-8 us
// slower); K = 1280 in 2 pieces of 10 k-tiles 10.6 against 9.4, hence the
// minimum length.  A deeper LDS
// ring (4, 6 or 8 stages) for the unsplit small launches gained nothing.
constexpr int kSplitTarget = 2;
constexpr int kSplitMinTiles = 16;

SplitPlan split_plan_plain(int M, int N, int K, const DeviceLayout& d) {
    SplitPlan sp{1, 1, 0, 0, 0};
    const int cus = d.cus;
    if (!d.xcd_merge || N % 64 != 0 || K % DBK != 0) return sp;
    const int64_t tiles = (int64_t)((M + 63) / 64) * (N / 64);
    if (tiles < 1 || tiles >= cus || tiles > GEMM_SPLIT_COUNTERS) return sp;
    const int n_xcd = d.n_xcd;
    const int64_t tpx = (tiles + n_xcd - 1) / n_xcd;
    int64_t k = (int64_t)kSplitTarget * cus / (n_xcd * tpx);
    const int64_t k_max = (K / DBK) / kSplitMinTiles;
    if (k > k_max) k = k_max;
    if (k > 8) k = 8;
    if (k < 2) return sp;
    sp.splitk = (int)k;
    sp.n_xcd = n_xcd;
    sp.tpx = (int)tpx;
    sp.n_tiles = (int)tiles;
    sp.bytes = (size_t)GEMM_SPLIT_COUNTERS * 4 + (size_t)n_xcd * tpx * k * 64 * 64 * 4;
    return sp;
}

}  // namespace

// Sized for a launch that may use every compute unit (a CU-masked stream
// only ever needs less).
size_t gemm_split_ws_bytes(int M, int N, int K, bool conv) {
    const DeviceLayout d = device_layout_unmasked();
    return conv ? split_plan(M, N, K, d).bytes : split_plan_plain(M, N, K, d).bytes;
}

namespace {

// The kernel a product runs on.
enum GemmKind { GK_DMA_128, GK_DMA_64, GK_G80, GK_DMA_GEGLU, GK_GEGLU160, GK_GEGLU160_64, GK_REG_22, GK_REG_12, GK_REG_11 };

// Validates p, picks its kernel, and sets the fields of a split or
// XCD-ordered launch.
hipError_t plan_gemm(GemmParams& p, hipStream_t s, GemmKind& kind) {
    if (p.conv_W > 0 && !gemm_shape_ok(p)) return hipErrorInvalidValue;
    if (p.a_mode == 2) {  // cross-attention epilogue: the 64 x 64 pipelined kernel, unsplit
        if (p.a_f32 || p.geglu || p.conv_W > 0 || p.K % DBK != 0 || p.N % 64 != 0 || p.seg < p.N || p.out_f32 ||
            p.resid != nullptr || p.out_bf16 != nullptr || p.bias != nullptr || p.bias2 != nullptr ||
            p.w_seg_rows != 0 || p.seg_stride != 0 || p.xa_k == nullptr || p.xa_v == nullptr || p.xa_T < 1 ||
            p.xa_T > GEMM_XA_MAXT || p.xa_N <= 0 || p.xa_N % 64 != 0 || p.M % p.xa_N != 0 || p.xa_ldkv < p.N ||
            p.xa_ldkv % 8 != 0)
            return hipErrorInvalidValue;
    } else if (p.a_mode != 0) {  // GroupNorm staging: the 64 x 64 pipelined kernel only
        if (p.a_mode != 1 || p.a_f32 || p.geglu || p.conv_W > 0 || p.K % DBK != 0 || p.K > GEMM_GN_MAXC ||
            p.N % 64 != 0 || p.seg % 4 != 0 || p.gn_N <= 0 || p.gn_N % 64 != 0 || p.M % p.gn_N != 0 || p.gn.G < 1 ||
            p.gn.G > 256 || p.K % p.gn.G != 0 || p.gn.stats == nullptr || p.gn_gamma == nullptr ||
            p.gn_beta == nullptr)
            return hipErrorInvalidValue;
    }
    if (p.w_seg_rows != 0 || p.seg_stride != 0) {  // the pipelined kernel's plain form only
        if (p.a_f32 || p.geglu || p.conv_W > 0 || p.K % DBK != 0 || p.seg % 4 != 0 || p.N % 64 != 0 ||
            p.seg_stride < 0 || p.w_seg_rows < 0)
            return hipErrorInvalidValue;
        if (p.w_seg_rows > 0 &&
            (p.w_seg_rows % 128 != 0 || p.N % p.w_seg_rows != 0 || p.N / p.w_seg_rows > GEMM_MAX_WSEG))
            return hipErrorInvalidValue;
    }
    p.splitk = 1;
    p.tpx = 0;
    const DeviceLayout dl = device_layout(s);
    if (p.conv_W > 0 && p.split_ws != nullptr) {
        const SplitPlan sp = split_plan(p.M, p.N, p.K, dl);
        if (sp.splitk > 1 && p.split_ws_bytes >= sp.bytes && ((uintptr_t)p.split_ws & 15u) == 0) {
            p.splitk = sp.splitk;
            p.n_xcd = sp.n_xcd;
            p.tpx = sp.tpx;
            p.n_tiles = sp.n_tiles;
            kind = GK_DMA_128;
            return hipSuccess;
        }
    }
    // Unsplit launches: when W (rows x K) is at least four times X (M x K),
    // each XCD takes a contiguous n-major range of tiles, so a W tile is
    // fetched into one XCD's L2 (the hardware deals workgroups round-robin
    // over the XCDs, which with few token tiles sends every W tile to all of
    // them).  At 512 tokens (2048 px level 2): GEGLU (10240 W rows) 37.4 ->
    // 25.5 us, Q/K/V (3840) 16.4 -> 13.6 us; at ratios of 1 to 2.5 it
    // changed nothing measurable.
    auto map_xcd = [&](int bm, int bn_out) {
        const int64_t w_rows = p.geglu ? 2 * (int64_t)p.N : p.N;
        if (!dl.xcd_merge || w_rows < 4 * (int64_t)p.M) return;
        const int64_t tiles = (int64_t)((p.M + bm - 1) / bm) * (p.N / bn_out);
        const int n_xcd = dl.n_xcd;
        if (tiles < n_xcd || tiles > INT32_MAX / 2) return;
        p.n_xcd = n_xcd;
        p.tpx = (int)((tiles + n_xcd - 1) / n_xcd);
        p.n_tiles = (int)tiles;
    };
    // bf16 X with K % 64 == 0: the pipelined kernel, with the largest tile
    // that still gives about a workgroup per compute unit.
    if (!p.a_f32 && p.K % DBK == 0 && p.seg % 4 == 0) {
        if (!p.geglu && p.conv_W == 0 && p.split_ws != nullptr && p.N % 64 == 0 && p.a_mode != 2) {
            const SplitPlan sp = split_plan_plain(p.M, p.N, p.K, dl);
            if (sp.splitk > 1 && p.split_ws_bytes >= sp.bytes && ((uintptr_t)p.split_ws & 15u) == 0) {
                p.splitk = sp.splitk;
                p.n_xcd = sp.n_xcd;
                p.tpx = sp.tpx;
                p.n_tiles = sp.n_tiles;
                kind = GK_DMA_64;
                return hipSuccess;
            }
        }
        if (p.geglu) {
            // 128 (else 64) tokens x 160 outputs when those tiles fit one per
            // compute unit and fill at least three quarters of them (the
            // block's 2048 x 2560 product, the level-2 512 x 5120 one: 256
            // tiles); the 64-token tiles run XCD-contiguous when W has four
            // times X's rows.
            const bool gg_form = p.N % 160 == 0 && p.resid == nullptr && p.out_bf16 == nullptr &&
                                 p.bias2 == nullptr && p.seg >= p.N && p.w_seg_rows == 0 && p.seg_stride == 0;
            const int64_t t128 = gg_form ? (int64_t)((p.M + 127) / 128) * (p.N / 160) : 0;
            const int64_t t64 = gg_form ? (int64_t)((p.M + 63) / 64) * (p.N / 160) : 0;
            const bool wide_w = 2 * (int64_t)p.N >= 4 * (int64_t)p.M;
            auto fits = [&](int64_t t) { return t > 0 && t <= dl.cus && 4 * t >= 3 * (int64_t)dl.cus; };
            const int64_t tg = fits(t128) ? t128 : (fits(t64) ? t64 : 0);
            if (tg > 0) {
                if (wide_w && dl.xcd_merge && tg >= dl.n_xcd) {
                    p.n_xcd = dl.n_xcd;
                    p.tpx = (int)((tg + dl.n_xcd - 1) / dl.n_xcd);
                    p.n_tiles = (int)tg;
                }
                kind = tg == t128 ? GK_GEGLU160 : GK_GEGLU160_64;
                return hipSuccess;
            }
            // value/gate pairs on 64-token tiles at two stages (48 KB of LDS: three
            // workgroups per compute unit): 25.3 us against 28.7 for 128-token
            // tiles and 35.2 for three stages at the 2048 x 2 x 2560 x 640 shape
            if (p.N % 64 == 0) {
                map_xcd(64, 64);
                kind = GK_DMA_GEGLU;
                return hipSuccess;
            }
        } else {
            // 128x128 tiles only with at least two per compute unit; else 64x64
            // tiles at three stages (48 KB of LDS: three workgroups per compute
            // unit), measured faster at M = 2048 for every N from 640 to 1920.
            // Balanced 64 x 80 tiles when the 64 x 64 ones would divide
            // unevenly over the compute units while the 80-row tiles come to
            // at most three per compute unit and fill at least three quarters
            // of them: a 2048 x 640 product is 256 tiles instead of 320, the
            // 2048 x 1920 Q/K/V product 768 instead of 960.  Not when W has
            // four times X's rows: those keep the XCD-contiguous 64 x 64 tiles.
            const int64_t mt64 = (p.M + 63) / 64;
            const int64_t t80 = p.N % 80 == 0 ? mt64 * (p.N / 80) : 0;
            const bool g80_form = p.a_mode == 0 && p.conv_W == 0 && p.w_seg_rows == 0 && p.seg_stride == 0 &&
                                  p.bias2 == nullptr && (p.seg >= p.N || (p.seg % 80 == 0 && p.N / p.seg <= 3));
            if (g80_form && p.N < 4 * (int64_t)p.M && t80 > 0 && t80 <= 3 * dl.cus && 4 * t80 >= 3 * (int64_t)dl.cus &&
                mt64 * (p.N / 64) > dl.cus) {
                kind = GK_G80;
                return hipSuccess;
            }
            const int64_t mt128 = (p.M + 127) / 128;
            if (p.a_mode == 0 && p.N % 128 == 0 && mt128 * (p.N / 128) >= 2 * (int64_t)dl.cus) {
                map_xcd(128, 128);
                kind = GK_DMA_128;
                return hipSuccess;
            }
            if (p.N % 64 == 0) {
                map_xcd(64, 64);
                kind = GK_DMA_64;
                return hipSuccess;
            }
        }
    }
    // only the pipelined kernel writes a bf16 copy, adds bias2 or convolves
    if (p.out_bf16 != nullptr || p.bias2 != nullptr || p.conv_W > 0) return hipErrorInvalidValue;
    // 128x128 tiles when they still give about a workgroup per compute unit,
    // else 64x128 / 64x64.
    kind = GK_REG_11;
    if (p.geglu) kind = GK_REG_22;
    const int64_t t128 = (int64_t)((p.M + 127) / 128) * (p.N / 128);
    if (!p.geglu && p.N % 128 == 0 && t128 >= 200)
        kind = GK_REG_22;
    else if (!p.geglu && p.N % 128 == 0 && (int64_t)((p.M + 63) / 64) * (p.N / 128) >= 160)
        kind = GK_REG_12;
    return hipSuccess;
}

hipError_t launch_planned(const GemmParams& p, GemmKind kind, hipStream_t s) {
    switch (kind) {
        case GK_DMA_128: return launch_dma<128, 128, 3, false>(p, s);
        case GK_DMA_64: return launch_dma<64, 64, 3, false>(p, s);
        case GK_G80: {
            // two stages (36 KB of LDS) when the tiles need several per compute unit
            const dim3 grid((unsigned)((p.M + G80_BM - 1) / G80_BM), (unsigned)(p.N / G80_BN));
            if ((int64_t)grid.x * grid.y > device_layout(s).cus)
                gemm80_kernel<2><<<grid, 512, 0, s>>>(p);
            else
                gemm80_kernel<4><<<grid, 512, 0, s>>>(p);
            return hipGetLastError();
        }
        case GK_DMA_GEGLU: return launch_dma<64, 128, 2, true>(p, s);
        case GK_GEGLU160:
        case GK_GEGLU160_64: {
            const int bm = kind == GK_GEGLU160 ? 128 : 64;
            const dim3 grid = p.tpx > 0 ? dim3((unsigned)(p.n_xcd * p.tpx), 1)
                                        : dim3((unsigned)((p.M + bm - 1) / bm), (unsigned)(p.N / GG_BN));
            if (kind == GK_GEGLU160)
                geglu160_kernel<128><<<grid, 512, 0, s>>>(p);
            else
                geglu160_kernel<64><<<grid, 512, 0, s>>>(p);
            return hipGetLastError();
        }
        case GK_REG_22: return launch_shape<2, 2>(p, s);
        case GK_REG_12: return launch_shape<1, 2>(p, s);
        default: return launch_shape<1, 1>(p, s);
    }
}

// Workgroups along x and y of a 64 x 64 pipelined launch (launch_dma).
void dma64_grid(const GemmParams& p, int& gx, int& gy) {
    if (p.tpx > 0) {
        gx = p.n_xcd * p.tpx * p.splitk;
        gy = 1;
    } else {
        gx = (p.M + 63) / 64;
        gy = p.N / 64;
    }
}

}  // namespace

hipError_t launch_gemm(const GemmParams& p_in, hipStream_t s) {
    GemmParams p = p_in;
    GemmKind kind;
    const hipError_t e = plan_gemm(p, s, kind);
    return e != hipSuccess ? e : launch_planned(p, kind, s);
}

hipError_t launch_gemm_pair(const GemmParams& a_in, const GemmParams& b_in, hipStream_t s) {
    GemmParams a = a_in, b = b_in;
    GemmKind ka, kb;
    hipError_t e = plan_gemm(a, s, ka);
    if (e != hipSuccess) return e;
    e = plan_gemm(b, s, kb);
    if (e != hipSuccess) return e;
    // One launch when both run on the 64 x 64 pipelined kernel and at most
    // one of them splits K (the split region holds one product's partials);
    // only the first may stage its X with GroupNorm, and neither carries the
    // cross-attention epilogue.
    if (ka == GK_DMA_64 && kb == GK_DMA_64 && a.conv_W == 0 && b.conv_W == 0 && !(a.splitk > 1 && b.splitk > 1) &&
        a.a_mode <= 1 && b.a_mode == 0) {
        GemmPair pp;
        pp.a = a;
        pp.b = b;
        int gy_a, gy_b;
        dma64_grid(a, pp.gx_a, gy_a);
        dma64_grid(b, pp.gx_b, gy_b);
        pp.n_a = pp.gx_a * gy_a;
        const DeviceLayout dl = device_layout(s);
        const int n_xcd = dl.n_xcd > 0 ? dl.n_xcd : 1;
        pp.b0 = (pp.n_a + n_xcd - 1) / n_xcd * n_xcd;
        const int64_t total = (int64_t)pp.b0 + (int64_t)pp.gx_b * gy_b;
        if (total > INT32_MAX) return hipErrorInvalidValue;
        if (a.a_mode == 1)
            gemm_dma_pair_kernel<64, 64, 3, 1><<<dim3((unsigned)total), 256, 0, s>>>(pp);
        else
            gemm_dma_pair_kernel<64, 64, 3, 0><<<dim3((unsigned)total), 256, 0, s>>>(pp);
        return hipGetLastError();
    }
    e = launch_planned(a, ka, s);
    return e != hipSuccess ? e : launch_planned(b, kb, s);
}

}  // namespace pcpp
