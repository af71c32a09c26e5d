// GroupNorm statistics of one image from the chunk records of the
// statistics launch: Chan et al.'s pairwise update of (count, mean, M2) in a
// fixed order, then, for the synchronized form (Sec. 3.3 of arXiv
// 2412.02962, kept from DistriFusion), every band's statistics in band order
// with this band's own in its place.  Shared by the GroupNorm apply kernel
// and by the GEMM that applies GroupNorm while it stages its operand, so the
// two produce the same bits.
#pragma once

#include "common.h"

namespace pcpp {

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

struct GnStatsSrc {
    const float* stats;  // [B][chunks][G] x (count, mean, M2)
    int32_t chunks, G, B;
    float eps;
    const float* bands;  // [n_bands][B][G] x (count, mean, M2), or null
    int32_t n_bands, band;
    float* own_out;      // [B][G] x (count, mean, M2) of this band, or null
};

// Statistics of image b for the calling workgroup of exactly 256 threads:
// thread (g, j) of S = 256 / G per group merges chunks j, j + S, ... (the
// records of one chunk are consecutive in g: coalesced), then thread g
// merges the S partial results in order j = 0, 1, ...  mrg: 256 x 3 floats of
// LDS; writes g_mean[G] and g_rstd[G] (LDS) and the band's own statistics if
// write_own; ends with a workgroup barrier.
__device__ __forceinline__ void gn_group_stats(const GnStatsSrc& a, int b, bool write_own, float* mrg, float* g_mean,
                                               float* g_rstd) {
    const int tid = threadIdx.x;
    const int G = a.G;
    const int S = 256 / G;
    const int g = tid % G, j = tid / G;
    float n = 0.f, mean = 0.f, m2 = 0.f;
    if (j < S) {
        const float* st = a.stats + ((int64_t)b * a.chunks * G + g) * 3;
        for (int k0 = j; k0 < a.chunks; k0 += 8 * S) {
            // Records past the last chunk read the last one (every load in
            // bounds, none behind a branch: all in flight together) and count
            // zero, which the update skips.
            float cn[8], cm[8], cq[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int k = k0 + u * S;
                const float* r = st + (int64_t)(k < a.chunks ? k : a.chunks - 1) * G * 3;
                cn[u] = r[0];
                cm[u] = r[1];
                cq[u] = r[2];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (k0 + u * S >= a.chunks) cn[u] = 0.f;
#pragma unroll
            for (int u = 0; u < 8; ++u) chan_merge(n, mean, m2, cn[u], cm[u], cq[u]);
        }
    }
    mrg[3 * tid] = n;
    mrg[3 * tid + 1] = mean;
    mrg[3 * tid + 2] = m2;
    __syncthreads();
    if (tid < G) {
        for (int k = 1; k < S; ++k)
            chan_merge(n, mean, m2, mrg[3 * (tid + k * G)], mrg[3 * (tid + k * G) + 1], mrg[3 * (tid + k * G) + 2]);
        if (a.own_out != nullptr && write_own) {
            float* o = a.own_out + ((int64_t)b * G + tid) * 3;
            o[0] = n;
            o[1] = mean;
            o[2] = m2;
        }
        if (a.bands != nullptr) {
            float tn = 0.f, tm = 0.f, tq = 0.f;
            for (int jb = 0; jb < a.n_bands; ++jb) {
                if (jb == a.band) {
                    chan_merge(tn, tm, tq, n, mean, m2);
                } else {
                    const float* o = a.bands + (((int64_t)jb * a.B + b) * G + tid) * 3;
                    chan_merge(tn, tm, tq, o[0], o[1], o[2]);
                }
            }
            n = tn;
            mean = tm;
            m2 = tq;
        }
        g_mean[tid] = mean;
        g_rstd[tid] = n > 0.f ? rsqrtf(m2 / n + a.eps) : 0.f;
    }
    __syncthreads();
}

}  // namespace pcpp
