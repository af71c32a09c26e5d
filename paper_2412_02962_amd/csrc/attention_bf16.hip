// Partially conditioned self-attention, bf16 storage, on gfx950 MFMA.
//
// Computes, per image and head, softmax(Q K_ctx^T / sqrt(64)) V_ctx where
// the key/value context is the band's fresh tokens plus the stale boundary
// rows of its neighbours (Sec. 3.3 and Eq. 1 of arXiv 2412.02962).  The three
// key/value sources are read in place (no assembled copy): every key row of a
// 64-key tile picks its source from its token index.
//
// Work decomposition: a workgroup of 4 wavefronts owns 4*QW queries of one
// head (QW = 32*NCB per wavefront) and one range of 64-key tiles; with more
// than one range per query block ("splits") the normalised partial outputs
// and row statistics go to the workspace and a merge kernel combines them.
//
// Per 64-key tile, per wavefront and per 32-query column block:
//   S^T = K Q^T      8 MFMA 32x32x16; K from LDS (row-major), Q^T held in
//                    registers for the whole kernel.  The transposed product
//                    leaves each lane with one query (lane % 32) and 32 of
//                    the tile's keys, so the row max needs one exchange with
//                    the partner lane (lane ^ 32) and the row sum none.
//   online softmax   in log2 units, p = exp2(s*log2(e)/8 - m); the running
//                    max m is only raised (and O, l rescaled) when a tile's
//                    max exceeds it by more than 8, so p <= 256 and most
//                    tiles skip the rescale.
//   O^T += V^T P^T   8 MFMA 32x32x16; P^T is the B operand taken straight
//                    from the S^T accumulators (inside each 16-key step the
//                    key order is permuted the same way on both operands);
//                    V^T is read from a row-major LDS tile with the gfx950
//                    transposing LDS read (ds_read_b64_tr_b16).
// Row sums accumulate the bf16 probabilities with v_dot2 against (1, 1), so
// numerator and denominator see the same rounded weights.  K/V tiles are
// double-buffered in LDS; the next tile's global loads are in flight while
// the current tile is computed.

#include <math.h>
#include <stdlib.h>

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int D = 64;
constexpr int BKV = 64;
constexpr int NWAVES = 4;
constexpr int NTHREADS = 64 * NWAVES;
constexpr int KSTR = 72;   // LDS row stride (elements) of the K and V tiles [64 keys][64 dims]
constexpr float RESCALE_SLACK = 8.0f;  // log2 units

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Element address of key row j: the segment base is chosen with selects on
// wave-uniform bases that are pre-offset by -begin*C, so row j of any
// segment is base + j*C.
struct RowBases {
    int64_t k0, k1, k2;   // byte addresses, pre-offset so that row j is base + j*C*2
    int64_t v0, v1, v2;
    int32_t end0, end1;
};

__device__ __forceinline__ int64_t pick(int j, int end0, int end1, int64_t a0, int64_t a1, int64_t a2) {
    const int64_t a12 = j < end1 ? a1 : a2;
    return j < end0 ? a0 : a12;
}

// Global-memory (address space 1) view of a 16-byte chunk: keeps the loads
// on the vector-memory counter only (a flat load would also hold up every
// LDS wait until it lands).
typedef const __attribute__((address_space(1))) u32x4* gchunk;

struct TileRegs {
    u32x4 k0, k1;
    u32x4 v0, v1;
};

__device__ __forceinline__ void load_tile(TileRegs& r, const RowBases& rb, int C, int tile_base, int kv_end,
                                          int tid) {
    const int row = tid >> 2;
    const int col = (tid & 3) * 16;
    const int j = tile_base + row;
    if (j < kv_end) {
        const int64_t roff = (int64_t)j * C * 2 + col * 2;
        gchunk kp = (gchunk)(uintptr_t)(pick(j, rb.end0, rb.end1, rb.k0, rb.k1, rb.k2) + roff);
        gchunk vp = (gchunk)(uintptr_t)(pick(j, rb.end0, rb.end1, rb.v0, rb.v1, rb.v2) + roff);
        r.k0 = kp[0];
        r.k1 = kp[1];
        r.v0 = vp[0];
        r.v1 = vp[1];
    } else {
        const u32x4 z = {0u, 0u, 0u, 0u};
        r.k0 = r.k1 = r.v0 = r.v1 = z;
    }
}

__device__ __forceinline__ void store_tile(const TileRegs& r, bf16* ks, bf16* vs, int tid) {
    const int row = tid >> 2;
    const int col = (tid & 3) * 16;
    u32x4* kp = (u32x4*)(ks + row * KSTR + col);
    u32x4* vp = (u32x4*)(vs + row * KSTR + col);
    kp[0] = r.k0;
    kp[1] = r.k1;
    vp[0] = r.v0;
    vp[1] = r.v1;
}

__device__ __forceinline__ bf16x4 lds_read_tr(const bf16* p) {
    i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
    return __builtin_bit_cast(bf16x4, v);
}

template <int NCB>
__global__ __launch_bounds__(NTHREADS) void attn_bf16_kernel(AttnParams p) {
    __shared__ __attribute__((aligned(16))) bf16 ks_buf[2][BKV * KSTR];
    __shared__ __attribute__((aligned(16))) bf16 vs_buf[2][BKV * KSTR];

    constexpr int QW = 32 * NCB;
    constexpr int BQ = QW * NWAVES;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int col = lane & 31;
    const int half = lane >> 5;
    const int head = blockIdx.y;
    const int b = blockIdx.z / p.splits;
    const int split = blockIdx.z % p.splits;
    const int head_off = head * D;
    const int C = p.C;

    const int n_tiles = (p.kv.n_kv + BKV - 1) / BKV;
    const int t_begin = split * p.tiles_per_split;
    const int t_end = min(t_begin + p.tiles_per_split, n_tiles);
    const int kv_end = p.kv.n_kv;

    RowBases rb;
    {
        const int64_t o0 = (int64_t)b * p.kv.bstride[0] + head_off;
        const int64_t o1 = (int64_t)b * p.kv.bstride[1] - (int64_t)p.kv.end0 * C + head_off;
        const int64_t o2 = (int64_t)b * p.kv.bstride[2] - (int64_t)p.kv.end1 * C + head_off;
        rb.k0 = (int64_t)(uintptr_t)p.kv.k[0] + o0 * 2;
        rb.k1 = (int64_t)(uintptr_t)p.kv.k[1] + o1 * 2;
        rb.k2 = (int64_t)(uintptr_t)p.kv.k[2] + o2 * 2;
        rb.v0 = (int64_t)(uintptr_t)p.kv.v[0] + o0 * 2;
        rb.v1 = (int64_t)(uintptr_t)p.kv.v[1] + o1 * 2;
        rb.v2 = (int64_t)(uintptr_t)p.kv.v[2] + o2 * 2;
        rb.end0 = p.kv.end0;
        rb.end1 = p.kv.end1;
    }

    // Q^T operands: lane holds query q0 + 32*cb + col, dims [16*kk + 8*half, +8).
    const int q0 = blockIdx.x * BQ + wave * QW;
    bf16x8 qop[NCB][4];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const int qrow = min(q0 + 32 * cb + col, p.nq - 1);
        const bf16* qp = (const bf16*)p.q + (int64_t)b * p.q_bstride + (int64_t)qrow * C + head_off + 8 * half;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qop[cb][kk] = *(const bf16x8*)(qp + 16 * kk);
    }
    // Q lands before the loop: otherwise the wait inserted for the first use
    // of Q inside the loop would also drain the next tile's prefetch.
    __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0)

    f32x16 o[NCB][2];
    float m_run[NCB], l_run[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[cb][mb][r] = 0.f;
        m_run[cb] = -INFINITY;
        l_run[cb] = 0.f;
    }
    const float sl2 = p.scale_log2;
    const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};

    // transposing-read addresses (element offsets inside a V tile)
    const int tr_jj = lane & 15;
    const int tr_row = 4 * half + (tr_jj >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (tr_jj & 3);

    TileRegs regs;
    if (t_begin < t_end) {
        load_tile(regs, rb, C, t_begin * BKV, kv_end, tid);
        store_tile(regs, ks_buf[0], vs_buf[0], tid);
    }
    __syncthreads();

    for (int t = t_begin; t < t_end; ++t) {
        const int buf = (t - t_begin) & 1;
        const bool has_next = t + 1 < t_end;
        if (has_next) load_tile(regs, rb, C, (t + 1) * BKV, kv_end, tid);

        const bf16* ks = ks_buf[buf];
        const bf16* vs = vs_buf[buf];

        f32x16 s[NCB][2];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int jb = 0; jb < 2; ++jb)
#pragma unroll
                for (int r = 0; r < 16; ++r) s[cb][jb][r] = 0.f;
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                bf16x8 kop = *(const bf16x8*)(ks + (32 * jb + col) * KSTR + 16 * kk + 8 * half);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) s[cb][jb] = mfma32x32x16(kop, qop[cb][kk], s[cb][jb]);
            }
        }

        const int tile_base = t * BKV;
        if (tile_base + BKV > kv_end) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int jb = 0; jb < 2; ++jb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        int j = tile_base + 32 * jb + 8 * (r >> 2) + 4 * half + (r & 3);
                        if (j >= kv_end) s[cb][jb][r] = -INFINITY;
                    }
        }

        bf16x8 pb[NCB][4];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            float mx = s[cb][0][0];
#pragma unroll
            for (int jb = 0; jb < 2; ++jb)
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[cb][jb][r]);
            mx = fmaxf(mx, __shfl_xor(mx, 32)) * sl2;
            if (__any(mx > m_run[cb] + RESCALE_SLACK)) {
                const float m_new = fmaxf(m_run[cb], mx);
                const float alpha = fast_exp2(m_run[cb] - m_new);
                m_run[cb] = m_new;
                l_run[cb] *= alpha;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) o[cb][mb][r] *= alpha;
            }
            const float mneg = -m_run[cb];
#pragma unroll
            for (int jb = 0; jb < 2; ++jb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    pb[cb][2 * jb + (r >> 3)][r & 7] = f32_to_bf16(fast_exp2(fmaf(s[cb][jb][r], sl2, mneg)));
            float lsum = l_run[cb];
#pragma unroll
            for (int st = 0; st < 4; ++st)
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    bf16x2 pr = {pb[cb][st][2 * w], pb[cb][st][2 * w + 1]};
                    lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, lsum, false);
                }
            l_run[cb] = lsum;
        }

        // O^T (64 dims x 32 queries) += V^T P^T over four 16-key steps.
#pragma unroll
        for (int st = 0; st < 4; ++st) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                const bf16* vp = vs + (16 * st + tr_row) * KSTR + 32 * mb + tr_col;
                bf16x4 lo = lds_read_tr(vp);
                bf16x4 hi = lds_read_tr(vp + 8 * KSTR);
                bf16x8 vop = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) o[cb][mb] = mfma32x32x16(vop, pb[cb][st], o[cb][mb]);
            }
        }

        if (has_next) store_tile(regs, ks_buf[buf ^ 1], vs_buf[buf ^ 1], tid);
        __syncthreads();
    }

#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const float l_tot = l_run[cb] + __shfl_xor(l_run[cb], 32);
        const int q = q0 + 32 * cb + col;
        if (q >= p.nq) continue;
        const float inv = t_begin < t_end ? 1.0f / l_tot : 0.f;
        if (p.splits == 1) {
            bf16* op = (bf16*)p.out + (int64_t)b * p.q_bstride + (int64_t)q * C + head_off;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    bf16x4 v = {f32_to_bf16(o[cb][mb][4 * c] * inv), f32_to_bf16(o[cb][mb][4 * c + 1] * inv),
                                f32_to_bf16(o[cb][mb][4 * c + 2] * inv), f32_to_bf16(o[cb][mb][4 * c + 3] * inv)};
                    *(bf16x4*)(op + 32 * mb + 8 * c + 4 * half) = v;
                }
        } else {
            float* op = p.ws_o + (((int64_t)split * p.batch + b) * p.nq + q) * C + head_off;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    f32x4 v = {o[cb][mb][4 * c] * inv, o[cb][mb][4 * c + 1] * inv, o[cb][mb][4 * c + 2] * inv,
                               o[cb][mb][4 * c + 3] * inv};
                    *(f32x4*)(op + 32 * mb + 8 * c + 4 * half) = v;
                }
            if (half == 0) {
                float* ml = p.ws_ml + ((((int64_t)split * p.batch + b) * p.heads + head) * p.nq + q) * 2;
                ml[0] = t_begin < t_end ? m_run[cb] : -INFINITY;
                ml[1] = t_begin < t_end ? l_tot : 0.f;
            }
        }
    }
}

// Combines the per-split partial outputs: weights l_s * 2^(m_s - max m).
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
    const int64_t groups = (int64_t)p.batch * p.nq * (p.C / 4);
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (gid >= groups) return;
    const int c4 = (int)(gid % (p.C / 4));
    const int64_t bq = gid / (p.C / 4);
    const int q = (int)(bq % p.nq);
    const int b = (int)(bq / p.nq);
    const int head = (c4 * 4) / D;

    float mmax = -INFINITY;
    for (int s = 0; s < p.splits; ++s) {
        const float* ml = p.ws_ml + ((((int64_t)s * p.batch + b) * p.heads + head) * p.nq + q) * 2;
        mmax = fmaxf(mmax, ml[0]);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int s = 0; s < p.splits; ++s) {
        const float* ml = p.ws_ml + ((((int64_t)s * p.batch + b) * p.heads + head) * p.nq + q) * 2;
        float w = ml[1] > 0.f ? ml[1] * fast_exp2(ml[0] - mmax) : 0.f;
        wsum += w;
        f32x4 v = *(const f32x4*)(p.ws_o + (((int64_t)s * p.batch + b) * p.nq + q) * p.C + c4 * 4);
        acc += w * v;
    }
    const float inv = 1.0f / wsum;
    bf16x4 o = {f32_to_bf16(acc[0] * inv), f32_to_bf16(acc[1] * inv), f32_to_bf16(acc[2] * inv),
                f32_to_bf16(acc[3] * inv)};
    *(bf16x4*)((bf16*)p.out + (int64_t)b * p.q_bstride + (int64_t)q * p.C + c4 * 4) = o;
}

int env_int(const char* name, int dflt) {
    const char* e = getenv(name);
    return (e != nullptr && atoi(e) > 0) ? atoi(e) : dflt;
}

// Query column blocks (of 32) per wavefront: 1 unless overridden.
int cols_per_wave() {
    int v = env_int("PCPP_ATTN_NCB", 1);
    return v == 2 ? 2 : 1;
}

}  // namespace

AttnPlan plan_attention_bf16(int32_t nq, int32_t n_kv, int32_t heads, int32_t batch, int32_t C) {
    AttnPlan pl;
    const int64_t bq = 32 * cols_per_wave() * NWAVES;
    const int64_t q_tiles = (nq + bq - 1) / bq;
    const int64_t base = q_tiles * heads * batch;
    const int64_t kv_tiles = (n_kv + BKV - 1) / BKV;
    int64_t splits = env_int("PCPP_ATTN_SPLITS", 0);
    if (splits == 0) {
        const int64_t target = 384;  // about 1.5 workgroups per compute unit
        splits = base < target ? (target + base - 1) / base : 1;
        const int64_t max_splits = kv_tiles / 8;  // keep at least eight tiles per split
        if (splits > max_splits) splits = max_splits;
    }
    if (splits < 1) splits = 1;
    if (splits > kv_tiles) splits = kv_tiles > 0 ? kv_tiles : 1;
    if (splits * batch > 65535) splits = 1;
    int64_t tps = (kv_tiles + splits - 1) / splits;
    if (tps < 1) tps = 1;
    splits = (kv_tiles + tps - 1) / tps;
    if (splits < 1) splits = 1;
    pl.splits = (int32_t)splits;
    pl.tiles_per_split = (int32_t)tps;
    pl.ws_bytes = splits > 1 ? (size_t)splits * batch * nq * C * sizeof(float) +
                                   (size_t)splits * batch * heads * nq * 2 * sizeof(float)
                             : 0;
    return pl;
}

hipError_t launch_attention_bf16(const AttnParams& p, hipStream_t stream) {
    const int ncb = cols_per_wave();
    const int bq = 32 * ncb * NWAVES;
    dim3 grid((p.nq + bq - 1) / bq, p.heads, p.batch * p.splits);
    if (ncb == 1)
        attn_bf16_kernel<1><<<grid, NTHREADS, 0, stream>>>(p);
    else
        attn_bf16_kernel<2><<<grid, NTHREADS, 0, stream>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t groups = (int64_t)p.batch * p.nq * (p.C / 4);
    attn_merge_kernel<<<(unsigned)((groups + 255) / 256), 256, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace pcpp
