// Partially conditioned self-attention, float32 storage and arithmetic.
//
// Same mathematics as the bf16 path (Sec. 3.3 and Eq. 1 of arXiv
// 2412.02962): per image and head, softmax(Q K_ctx^T / sqrt(64)) V_ctx over
// the fresh band plus the stale boundary rows of the neighbours, read in
// place from the three sources.  One thread owns one query and keeps its
// 64-dim query and output in registers; 16-key tiles of K and V are staged
// in LDS and read by every thread of the block (LDS broadcast).  Scores of a
// tile are computed first, then one online-softmax update per tile.  Logits,
// softmax weights, their sum and the weighted sum of values accumulate in
// float64 (the float32 inputs widen exactly), so the only float32 rounding is
// the final store.  Meant for small problems and float32 accuracy, not speed.

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int D = 64;
constexpr int BQ = 128;
constexpr int BKV = 16;

__device__ __forceinline__ const float* kv_ptr_f32(const KvSource& s, bool v, int b, int j, int C,
                                                   int head_off) {
    int seg = j < s.end0 ? 0 : (j < s.end1 ? 1 : 2);
    int begin = seg == 0 ? 0 : (seg == 1 ? s.end0 : s.end1);
    const float* base = (const float*)(v ? s.v[seg] : s.k[seg]);
    return base + (int64_t)b * s.bstride[seg] + (int64_t)(j - begin) * C + head_off;
}

__global__ __launch_bounds__(BQ) void attn_f32_kernel(AttnParams p) {
    __shared__ float ks[BKV][D];
    __shared__ float vs[BKV][D];
    const int tid = threadIdx.x;
    const int head = blockIdx.y;
    const int b = blockIdx.z;
    const int head_off = head * D;
    const int q = blockIdx.x * BQ + tid;
    const int qrow = min(q, p.nq - 1);

    float qv[D];
    const float* qp = (const float*)p.q + (int64_t)b * p.q_bstride + (int64_t)qrow * p.C + head_off;
#pragma unroll
    for (int e = 0; e < D; ++e) qv[e] = qp[e];
    const double scale = (double)p.scale;

    double o[D];
#pragma unroll
    for (int e = 0; e < D; ++e) o[e] = 0.0;
    double m_run = -INFINITY;
    double l_run = 0.0;

    const int n_kv = p.kv.n_kv;
    for (int base = 0; base < n_kv; base += BKV) {
        __syncthreads();
        for (int x = tid; x < BKV * D; x += BQ) {
            int r = x / D, e = x % D;
            int j = base + r;
            ks[r][e] = j < n_kv ? kv_ptr_f32(p.kv, false, b, j, p.C, head_off)[e] : 0.f;
            vs[r][e] = j < n_kv ? kv_ptr_f32(p.kv, true, b, j, p.C, head_off)[e] : 0.f;
        }
        __syncthreads();
        const int cnt = min(BKV, n_kv - base);
        double s[BKV];
        double mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < BKV; ++r) {
            double acc = 0.0;
#pragma unroll
            for (int e = 0; e < D; ++e) acc = fma((double)qv[e], (double)ks[r][e], acc);
            s[r] = r < cnt ? acc * scale : -INFINITY;
            mx = fmax(mx, s[r]);
        }
        const double m_new = fmax(m_run, mx);
        const double alpha = exp(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int e = 0; e < D; ++e) o[e] *= alpha;
#pragma unroll
        for (int r = 0; r < BKV; ++r) {
            double w = exp(s[r] - m_new);
            l_run += w;
#pragma unroll
            for (int e = 0; e < D; ++e) o[e] = fma(w, (double)vs[r][e], o[e]);
        }
        m_run = m_new;
    }
    if (q >= p.nq) return;
    const double inv = 1.0 / l_run;
    float* op = (float*)p.out + (int64_t)b * p.q_bstride + (int64_t)q * p.C + head_off;
#pragma unroll
    for (int e = 0; e < D; ++e) op[e] = (float)(o[e] * inv);
}

}  // namespace

hipError_t launch_attention_f32(const AttnParams& p, hipStream_t stream) {
    dim3 grid((p.nq + BQ - 1) / BQ, p.heads, p.batch);
    attn_f32_kernel<<<grid, BQ, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace pcpp
