// Partially conditioned self-attention, bf16 storage, on gfx950 MFMA.
//
// Computes, per image and head, softmax(Q K_ctx^T / sqrt(64)) V_ctx where
// the key/value context is the band's fresh tokens plus the stale boundary
// rows of its neighbours (Sec. 3.3 and Eq. 1 of arXiv 2412.02962).  The three
// key/value sources are read in place (no assembled copy): every 64-key tile
// row picks its source from the token index.
//
// Work decomposition: a workgroup of 4 wavefronts owns 128 queries of one
// head (32 per wavefront) and one range of 64-key tiles; with more than one
// range per query block ("splits") the normalised partial outputs and row
// statistics go to the workspace and a merge kernel combines them.
//
// Per 64-key tile and wavefront (32 queries):
//   S^T = K Q^T      8 MFMA 32x32x16; K from LDS (row-major), Q^T held in
//                    registers for the whole kernel.  The transposed product
//                    leaves each lane with one query (lane % 32) and 32 of
//                    the tile's keys, so the row max needs one exchange with
//                    the partner lane (lane ^ 32) and the row sum none.
//   online softmax   in log2 units: p = exp2(s * log2(e)/8 - m)
//   O^T += V^T P^T   8 MFMA 32x32x16; P^T is the B operand straight from the
//                    S^T accumulators (the key order inside a 16-key step is
//                    permuted identically on both operands), V^T comes from
//                    an LDS tile written transposed while staging.
// K/V tiles are double-buffered in LDS; the next tile's global loads are in
// flight while the current tile is computed.

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int D = 64;
constexpr int BQ = 128;
constexpr int BKV = 64;
constexpr int NTHREADS = 256;
constexpr int KSTR = 72;   // LDS row stride of the K tile [64 keys][64 dims]
constexpr int VSTR = 72;   // LDS row stride of the V^T tile [64 dims][64 keys]

__device__ __forceinline__ const bf16* kv_ptr(const KvSource& s, bool v, int b, int j, int C,
                                              int head_off) {
    int seg = j < s.end0 ? 0 : (j < s.end1 ? 1 : 2);
    int begin = seg == 0 ? 0 : (seg == 1 ? s.end0 : s.end1);
    const bf16* base = (const bf16*)(v ? s.v[seg] : s.k[seg]);
    return base + (int64_t)b * s.bstride[seg] + (int64_t)(j - begin) * C + head_off;
}

struct TileRegs {
    u32x4 k0, k1;   // 16 key elements of one key row
    u32x4 v0, v1;   // 8 value elements of two consecutive key rows
};

__device__ __forceinline__ void load_tile(TileRegs& r, const KvSource& s, int b, int C, int head_off,
                                          int tile_base, int kv_end, int tid) {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    {
        int row = tid >> 2;
        int col = (tid & 3) * 16;
        int j = tile_base + row;
        if (j < kv_end) {
            const u32x4* p = (const u32x4*)(kv_ptr(s, false, b, j, C, head_off) + col);
            r.k0 = p[0];
            r.k1 = p[1];
        } else {
            r.k0 = zero;
            r.k1 = zero;
        }
    }
    {
        int pair = tid >> 3;
        int col = (tid & 7) * 8;
        int j0 = tile_base + 2 * pair;
        r.v0 = j0 < kv_end ? *(const u32x4*)(kv_ptr(s, true, b, j0, C, head_off) + col) : zero;
        r.v1 = j0 + 1 < kv_end ? *(const u32x4*)(kv_ptr(s, true, b, j0 + 1, C, head_off) + col) : zero;
    }
}

__device__ __forceinline__ void store_tile(const TileRegs& r, bf16* ks, bf16* vt, int tid) {
    {
        int row = tid >> 2;
        int col = (tid & 3) * 16;
        u32x4* p = (u32x4*)(ks + row * KSTR + col);
        p[0] = r.k0;
        p[1] = r.k1;
    }
    {
        int pair = tid >> 3;
        int col = (tid & 7) * 8;
        uint32_t* base = (uint32_t*)(vt + col * VSTR + 2 * pair);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t a = r.v0[w];
            uint32_t c = r.v1[w];
            // dims col+2w and col+2w+1; each word packs (key 2*pair, key 2*pair+1)
            base[(2 * w) * (VSTR / 2)] = (a & 0xFFFFu) | (c << 16);
            base[(2 * w + 1) * (VSTR / 2)] = (a >> 16) | (c & 0xFFFF0000u);
        }
    }
}

__global__ __launch_bounds__(NTHREADS) void attn_bf16_kernel(AttnParams p) {
    __shared__ __attribute__((aligned(16))) bf16 ks_buf[2][BKV * KSTR];
    __shared__ __attribute__((aligned(16))) bf16 vt_buf[2][D * VSTR];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int col = lane & 31;   // query column of this lane in the 32x32 blocks
    const int half = lane >> 5;  // which half of the contraction this lane feeds
    const int head = blockIdx.y;
    const int b = blockIdx.z / p.splits;
    const int split = blockIdx.z % p.splits;
    const int head_off = head * D;
    const int C = p.C;

    const int n_tiles = (p.kv.n_kv + BKV - 1) / BKV;
    const int t_begin = split * p.tiles_per_split;
    int t_end = t_begin + p.tiles_per_split;
    if (t_end > n_tiles) t_end = n_tiles;
    const int kv_end = p.kv.n_kv;

    // Q^T operand: lane holds query q0+col, dims [16*ks + 8*half, +8).
    const int q0 = blockIdx.x * BQ + wave * 32;
    const int qrow = min(q0 + col, p.nq - 1);
    const bf16* qp = (const bf16*)p.q + (int64_t)b * p.q_bstride + (int64_t)qrow * C + head_off + 8 * half;
    bf16x8 qop[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qop[ks] = *(const bf16x8*)(qp + 16 * ks);

    f32x16 o[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[mb][r] = 0.f;
    float m_run = -INFINITY;
    float l_run = 0.f;
    const float sl2 = p.scale_log2;

    TileRegs regs;
    if (t_begin < t_end) {
        load_tile(regs, p.kv, b, C, head_off, t_begin * BKV, kv_end, tid);
        store_tile(regs, ks_buf[0], vt_buf[0], tid);
    }
    __syncthreads();

    for (int t = t_begin; t < t_end; ++t) {
        const int buf = (t - t_begin) & 1;
        const bool has_next = t + 1 < t_end;
        if (has_next) load_tile(regs, p.kv, b, C, head_off, (t + 1) * BKV, kv_end, tid);

        const bf16* ks = ks_buf[buf];
        const bf16* vt = vt_buf[buf];

        // S^T (64 keys x 32 queries) as two 32x32 blocks.
        f32x16 s[2];
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) {
#pragma unroll
            for (int r = 0; r < 16; ++r) s[jb][r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                bf16x8 kop = *(const bf16x8*)(ks + (32 * jb + col) * KSTR + 16 * kk + 8 * half);
                s[jb] = mfma32x32x16(kop, qop[kk], s[jb]);
            }
        }

        const int tile_base = t * BKV;
        if (tile_base + BKV > kv_end) {
#pragma unroll
            for (int jb = 0; jb < 2; ++jb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    int j = tile_base + 32 * jb + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (j >= kv_end) s[jb][r] = -INFINITY;
                }
        }

        float mx = s[0][0];
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[jb][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * sl2);
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[mb][r] *= alpha;

        bf16x8 pb[4];
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float e = fast_exp2(fmaf(s[jb][r], sl2, -m_new));
                l_run += e;
                pb[2 * jb + (r >> 3)][r & 7] = f32_to_bf16(e);
            }

        // O^T (64 dims x 32 queries) += V^T P^T over four 16-key steps.
#pragma unroll
        for (int st = 0; st < 4; ++st) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                const bf16* vrow = vt + (32 * mb + col) * VSTR + 16 * st + 4 * half;
                bf16x4 lo = *(const bf16x4*)(vrow);
                bf16x4 hi = *(const bf16x4*)(vrow + 8);
                bf16x8 vop = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                o[mb] = mfma32x32x16(vop, pb[st], o[mb]);
            }
        }

        if (has_next) store_tile(regs, ks_buf[buf ^ 1], vt_buf[buf ^ 1], tid);
        __syncthreads();
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const int q = q0 + col;
    if (q >= p.nq) return;
    const float inv = t_begin < t_end ? 1.0f / l_tot : 0.f;

    if (p.splits == 1) {
        bf16* op = (bf16*)p.out + (int64_t)b * p.q_bstride + (int64_t)q * C + head_off;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                bf16x4 v = {f32_to_bf16(o[mb][4 * c] * inv), f32_to_bf16(o[mb][4 * c + 1] * inv),
                            f32_to_bf16(o[mb][4 * c + 2] * inv), f32_to_bf16(o[mb][4 * c + 3] * inv)};
                *(bf16x4*)(op + 32 * mb + 8 * c + 4 * half) = v;
            }
    } else {
        float* op = p.ws_o + (((int64_t)split * p.batch + b) * p.nq + q) * C + head_off;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                f32x4 v = {o[mb][4 * c] * inv, o[mb][4 * c + 1] * inv, o[mb][4 * c + 2] * inv,
                           o[mb][4 * c + 3] * inv};
                *(f32x4*)(op + 32 * mb + 8 * c + 4 * half) = v;
            }
        if (half == 0) {
            float* ml = p.ws_ml + ((((int64_t)split * p.batch + b) * p.heads + head) * p.nq + q) * 2;
            ml[0] = t_begin < t_end ? m_run : -INFINITY;
            ml[1] = t_begin < t_end ? l_tot : 0.f;
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

}  // namespace

AttnPlan plan_attention_bf16(int32_t nq, int32_t n_kv, int32_t heads, int32_t batch, int32_t C) {
    AttnPlan pl;
    const int64_t q_tiles = (nq + BQ - 1) / BQ;
    const int64_t base = q_tiles * heads * batch;
    const int64_t kv_tiles = (n_kv + BKV - 1) / BKV;
    int64_t splits = 1;
    const char* env = getenv("PCPP_ATTN_SPLITS");
    if (env != nullptr && atoi(env) > 0) {
        splits = atoi(env);
    } else {
        const int64_t target = 512;  // two workgroups per compute unit
        if (base < target) splits = (target + base - 1) / base;
        int64_t max_splits = kv_tiles / 4;  // keep at least four tiles per split
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
    dim3 grid((p.nq + BQ - 1) / BQ, p.heads, p.batch * p.splits);
    attn_bf16_kernel<<<grid, NTHREADS, 0, stream>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t groups = (int64_t)p.batch * p.nq * (p.C / 4);
    attn_merge_kernel<<<(unsigned)((groups + 255) / 256), 256, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace pcpp
