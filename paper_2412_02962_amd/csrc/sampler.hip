// pcpp_guided_step: the update of a band's latent at the end of a step
// (Sec. 3.1 of arXiv 2412.02962): classifier-free guidance, Eq. 2,
//   e = eps_u + s (eps_c - eps_u),
// then the reverse step, either Eq. 3 and Eq. 4,
//   x_{t-1} = (x_t - beta_t / sqrt(1 - abar_t) e) / sqrt(alpha_t) + sigma_t z,
// with beta_t = 1 - alpha_t, or the deterministic DDIM update the paper's
// experiments use (Sec. 4),
//   x_{t-1} = sqrt(abar_prev) (x_t - sqrt(1 - abar_t) e) / sqrt(abar_t)
//           + sqrt(1 - abar_prev) e.
// Both are x_{t-1} = a x_t + b e (+ sigma_t z), with a and b computed once
// on the host in double precision.  Elementwise, HBM-bound; each element is
// read and written by one thread, so x_prev may alias x_t.

#include <math.h>
#include <stdint.h>

#include "../../include/pcpp.h"
#include "common.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

constexpr int kThreads = 256;

struct StepCoef {
    float a, b, s, sigma;
};

template <int V>
__global__ __launch_bounds__(kThreads) void guided_step(StepCoef k, int64_t n, const float* x, const float* eu,
                                                        const float* ec, const float* z, float* out) {
    typedef float vec __attribute__((ext_vector_type(V)));
    const int64_t nv = n / V;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < nv; i += (int64_t)gridDim.x * kThreads) {
        const vec xv = ((const vec*)x)[i];
        const vec uv = ((const vec*)eu)[i];
        const vec cv = ((const vec*)ec)[i];
        vec zv = {};
        if (z != nullptr) zv = ((const vec*)z)[i];
        vec o;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float g = __builtin_fmaf(k.s, cv[e] - uv[e], uv[e]);
            o[e] = __builtin_fmaf(k.b, g, k.a * xv[e]);
            if (z != nullptr) o[e] = __builtin_fmaf(k.sigma, zv[e], o[e]);
        }
        ((vec*)out)[i] = o;
    }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT int pcpp_guided_step(const pcpp_step_params_t* sp, int64_t n, const float* x_t, const float* eps_uncond,
                                 const float* eps_cond, const float* z, float* x_prev, void* stream) {
    if (sp == nullptr || sp->reserved != 0 || n < 0) return PCPP_EINVAL;
    if (!isfinite(sp->guidance)) return PCPP_EINVAL;
    StepCoef k;
    k.s = sp->guidance;
    k.sigma = 0.f;
    if (sp->mode == PCPP_STEP_DDPM) {
        const double a = sp->alpha_t, ab = sp->alphabar_t;
        if (!(a > 0.0 && a <= 1.0) || !(ab > 0.0 && ab < 1.0) || !isfinite(sp->sigma_t)) return PCPP_EINVAL;
        k.a = (float)(1.0 / sqrt(a));
        k.b = (float)(-(1.0 - a) / (sqrt(1.0 - ab) * sqrt(a)));
        k.sigma = sp->sigma_t;
    } else if (sp->mode == PCPP_STEP_DDIM) {
        const double ab = sp->alphabar_t, ap = sp->alphabar_prev;
        if (!(ab > 0.0 && ab <= 1.0) || !(ap > 0.0 && ap <= 1.0)) return PCPP_EINVAL;
        k.a = (float)sqrt(ap / ab);
        k.b = (float)(sqrt(1.0 - ap) - sqrt(ap) * sqrt(1.0 - ab) / sqrt(ab));
        if (z != nullptr) return PCPP_EINVAL;  // deterministic: no noise term
    } else {
        return PCPP_EINVAL;
    }
    if (n == 0) return PCPP_OK;
    if (!x_t || !eps_uncond || !eps_cond || !x_prev) return PCPP_EINVAL;
    const bool v4 = n % 4 == 0 && aligned16(x_t) && aligned16(eps_uncond) && aligned16(eps_cond) &&
                    aligned16(x_prev) && (z == nullptr || aligned16(z));
    const int64_t units = v4 ? n / 4 : n;
    int64_t blocks = (units + kThreads - 1) / kThreads;
    if (blocks > 8192) blocks = 8192;
    hipStream_t s = (hipStream_t)stream;
    if (v4)
        guided_step<4><<<(unsigned)blocks, kThreads, 0, s>>>(k, n, x_t, eps_uncond, eps_cond, z, x_prev);
    else
        guided_step<1><<<(unsigned)blocks, kThreads, 0, s>>>(k, n, x_t, eps_uncond, eps_cond, z, x_prev);
    return hipGetLastError() == hipSuccess ? PCPP_OK : PCPP_EHIP;
}
