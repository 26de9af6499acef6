// Optimiser step of the training loop: Alg. 1 updates the weights with ADAM
// after each backward pass (Kingma and Ba, ICLR 2015, Algorithm 1).  One
// streaming pass over a flat parameter buffer: reads p, g, m, v and writes p,
// m, v (28 bytes per parameter), so the bound is HBM bandwidth.
#include <cmath>

#include "common.h"
#include "gcn_optim.h"

namespace gcn {
namespace {

constexpr int kTB = 256;

struct AdamArgs {
    float b1, b2, c1, c2;       // beta1, beta2, 1 - beta1, 1 - beta2
    float step_size;            // lr / (1 - beta1^t)
    float inv_sqrt_bc2;         // 1 / sqrt(1 - beta2^t)
    float eps;
};

__device__ __forceinline__ void adam_one(float &p, float g, float &m, float &v, const AdamArgs &a) {
    m = a.b1 * m + a.c1 * g;
    v = a.b2 * v + a.c2 * (g * g);
    const float denom = sqrtf(v) * a.inv_sqrt_bc2 + a.eps;
    p -= a.step_size * (m / denom);
}

template <bool VEC>
__global__ __launch_bounds__(kTB) void adam_kernel(float *__restrict__ p, const float *__restrict__ g,
                                                   float *__restrict__ m, float *__restrict__ v, int64_t count,
                                                   AdamArgs a) {
    const int64_t stride = (int64_t)gridDim.x * kTB;
    if (VEC) {
        const int64_t n4 = count / 4;
        for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < n4; i += stride) {
            float4 pp = ((float4 *)p)[i], mm = ((float4 *)m)[i], vv = ((float4 *)v)[i];
            const float4 gg = ((const float4 *)g)[i];
            adam_one(pp.x, gg.x, mm.x, vv.x, a);
            adam_one(pp.y, gg.y, mm.y, vv.y, a);
            adam_one(pp.z, gg.z, mm.z, vv.z, a);
            adam_one(pp.w, gg.w, mm.w, vv.w, a);
            ((float4 *)p)[i] = pp;
            ((float4 *)m)[i] = mm;
            ((float4 *)v)[i] = vv;
        }
    } else {
        for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < count; i += stride) {
            float pp = p[i], mm = m[i], vv = v[i];
            adam_one(pp, g[i], mm, vv, a);
            p[i] = pp;
            m[i] = mm;
            v[i] = vv;
        }
    }
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" int gcn_adam_update(float *params, const float *grads, float *m, float *v, int64_t count, double lr,
                               double beta1, double beta2, double eps, int32_t step, void *stream) {
    if (count < 0 || (count > 0 && (!params || !grads || !m || !v))) {
        set_error("gcn_adam_update: null pointer or negative count");
        return GCN_EINVAL;
    }
    if (step < 1 || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps > 0.0) ||
        !std::isfinite(lr)) {
        set_error("gcn_adam_update: need step >= 1, 0 <= beta1, beta2 < 1, eps > 0 and a finite lr");
        return GCN_EINVAL;
    }
    if (count == 0) return GCN_OK;
    AdamArgs a;
    // every coefficient is formed in double from the double hyperparameters
    // and rounded once (1 - beta in float32 arithmetic would differ by
    // the rounding of beta itself)
    a.b1 = (float)beta1;
    a.b2 = (float)beta2;
    a.c1 = (float)(1.0 - beta1);
    a.c2 = (float)(1.0 - beta2);
    const double bc1 = 1.0 - std::pow(beta1, (double)step);
    const double bc2 = 1.0 - std::pow(beta2, (double)step);
    a.step_size = (float)(lr / bc1);
    a.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
    a.eps = (float)eps;
    hipStream_t s = (hipStream_t)stream;
    ProfScope prof(K_ADAM, s, 0.0, 28.0 * (double)count);
    const bool vec = count % 4 == 0 && (((uintptr_t)params | (uintptr_t)grads | (uintptr_t)m | (uintptr_t)v) & 15u) == 0;
    const int64_t work = vec ? count / 4 : count;
    const int blocks = (int)std::min<int64_t>((work + kTB - 1) / kTB, 8192);
    if (vec)
        adam_kernel<true><<<blocks, kTB, 0, s>>>(params, grads, m, v, count, a);
    else
        adam_kernel<false><<<blocks, kTB, 0, s>>>(params, grads, m, v, count, a);
    GCN_LAUNCH_CHECK("adam_kernel");
    return GCN_OK;
}
