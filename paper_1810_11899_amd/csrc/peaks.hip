// Machine-rate probes: the streaming read bandwidth and the matrix-core rate
// this GPU actually sustains.  They give the kernels of the layer a measured
// ceiling next to the datasheet one (HBM 8 TB/s; 157.3 TFLOP/s fp32 matrix,
// 2.5 PFLOP/s dense bf16 matrix).  Neither touches the method's data.
#include "common.h"
#include "gcn_peaks.h"

namespace gcn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kPeakThreads = 256;

// Grid-stride 16-byte loads, four in flight per thread, summed so that no load
// is dead.  Each thread writes one float of the sink.
__global__ __launch_bounds__(kPeakThreads) void stream_read_kernel(const f4 *__restrict__ x, int64_t n4,
                                                                    float *__restrict__ sink) {
    const int64_t tid = (int64_t)blockIdx.x * kPeakThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kPeakThreads;
    f4 s0 = {0, 0, 0, 0}, s1 = s0, s2 = s0, s3 = s0;
    int64_t i = tid;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        s0 += __builtin_nontemporal_load(x + i);
        s1 += __builtin_nontemporal_load(x + i + stride);
        s2 += __builtin_nontemporal_load(x + i + 2 * stride);
        s3 += __builtin_nontemporal_load(x + i + 3 * stride);
    }
    for (; i < n4; i += stride) s0 += x[i];
    const f4 t = (s0 + s1) + (s2 + s3);
    sink[tid] = (t.x + t.y) + (t.z + t.w);
}

// Four independent accumulator chains per wavefront keep the matrix pipe busy
// while each product's latency drains.  Operands are register values that
// depend on the lane, so nothing folds away; the accumulators are summed into
// the sink at the end.
__global__ __launch_bounds__(kPeakThreads) void mfma_f32_kernel(int32_t iters, float *__restrict__ sink) {
    const float a = 1.0f + (threadIdx.x & 7) * 1e-3f;
    const float b = 1.0f - (threadIdx.x & 3) * 1e-3f;
    floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int32_t it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(b, a, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, a, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(b, b, c3, 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    sink[(int64_t)blockIdx.x * kPeakThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kPeakThreads) void mfma_bf16_kernel(int32_t iters, float *__restrict__ sink) {
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(1.0f + ((threadIdx.x + e) & 7) * 0.0625f);
        b[e] = (__bf16)(1.0f - ((threadIdx.x + e) & 3) * 0.0625f);
    }
    floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int32_t it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, b, c3, 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    sink[(int64_t)blockIdx.x * kPeakThreads + threadIdx.x] = s;
}

// Dependent loads: each chain follows next[] for `steps` hops (one lane does
// the walk, the wavefront waits on it as the sampler's wavefront waits on its
// global loads).
__global__ __launch_bounds__(64) void chase_kernel(const int32_t *__restrict__ next, int64_t n, int32_t steps,
                                                   int32_t *__restrict__ sink) {
    int64_t i = ((int64_t)blockIdx.x * 2654435761ll) % n;
    if (threadIdx.x == 0) {
        for (int32_t k = 0; k < steps; ++k) i = next[i];
        sink[blockIdx.x] = (int32_t)i;
    }
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" {

int gcn_peak_stream_read(const float *x, int64_t count, float *sink, int32_t blocks, void *stream) {
    if (!x || !sink || count < 0 || blocks <= 0) {
        set_error("gcn_peak_stream_read: null pointer or bad size");
        return GCN_EINVAL;
    }
    if (count % 4 != 0 || ((uintptr_t)x & 15u) != 0) {
        set_error("gcn_peak_stream_read: count must be a multiple of 4 and x 16-byte aligned");
        return GCN_ESHAPE;
    }
    hipStream_t s = (hipStream_t)stream;
    stream_read_kernel<<<blocks, kPeakThreads, 0, s>>>((const f4 *)x, count / 4, sink);
    GCN_LAUNCH_CHECK("stream_read_kernel");
    return GCN_OK;
}

int gcn_peak_mfma(gcn_prec prec, int32_t blocks, int32_t iters, float *sink, double *flops, void *stream) {
    if (!sink || blocks <= 0 || iters <= 0 || (prec != GCN_F32 && prec != GCN_BF16)) {
        set_error("gcn_peak_mfma: null pointer, bad size or bad precision");
        return GCN_EINVAL;
    }
    hipStream_t s = (hipStream_t)stream;
    const double per_mfma = prec == GCN_F32 ? 2.0 * 32 * 32 * 2 : 2.0 * 32 * 32 * 16;
    if (prec == GCN_F32)
        mfma_f32_kernel<<<blocks, kPeakThreads, 0, s>>>(iters, sink);
    else
        mfma_bf16_kernel<<<blocks, kPeakThreads, 0, s>>>(iters, sink);
    GCN_LAUNCH_CHECK("mfma_kernel");
    if (flops) *flops = per_mfma * 4.0 * iters * (blocks * (kPeakThreads / kWave));
    return GCN_OK;
}

int gcn_peak_chase(const int32_t *next, int64_t n, int32_t steps, int32_t chains, int32_t *sink, void *stream) {
    if (!next || !sink || n <= 0 || steps < 0 || chains <= 0) {
        set_error("gcn_peak_chase: null pointer or bad size");
        return GCN_EINVAL;
    }
    hipStream_t s = (hipStream_t)stream;
    chase_kernel<<<chains, 64, 0, s>>>(next, n, steps, sink);
    GCN_LAUNCH_CHECK("chase_kernel");
    return GCN_OK;
}

}  // extern "C"
