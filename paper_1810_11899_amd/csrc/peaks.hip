// Machine-rate probes: the streaming read bandwidth, the row-gather rate,
// the matrix-core rate and the dependent-load latency this GPU actually
// sustains.  They give the kernels of the layer a measured
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

// Row gathers, the access pattern of the feature propagation.  A wavefront
// takes 64 consecutive indices with one coalesced load and hands them out by
// lane shuffles; a group of G lanes reads one row of `chunks` x G x 16 bytes,
// kGatherU rows in flight per group.  Out-of-range indices are clamped (the
// probe never reads outside X).
constexpr int kGatherU = 8;
template <int CH>
__global__ __launch_bounds__(kPeakThreads) void gather_kernel(const f4 *__restrict__ x, int64_t n_rows,
                                                               int64_t ld4, const int32_t *__restrict__ idx,
                                                               int64_t count, int G, float *__restrict__ sink) {
    const int lane = threadIdx.x & 63;
    const int gpw = 64 / G;                                   // groups per wavefront
    const int g = lane / G, l = lane % G;
    const int64_t wave = ((int64_t)blockIdx.x * kPeakThreads + threadIdx.x) >> 6;
    const int64_t waves = (int64_t)gridDim.x * kPeakThreads >> 6;
    f4 acc = {0, 0, 0, 0};
    for (int64_t base = wave * 64; base < count; base += waves * 64) {
        const int64_t q = base + lane;
        int32_t mine = q < count ? idx[q] : -1;
        mine = mine < 0 ? -1 : (mine >= n_rows ? (int32_t)(n_rows - 1) : mine);
        // rows g, g + gpw, g + 2 gpw, ... of the batch belong to group g
        for (int r0 = 0; r0 < 64; r0 += gpw * kGatherU) {
            int32_t row[kGatherU];
#pragma unroll
            for (int u = 0; u < kGatherU; ++u) {
                const int src = r0 + u * gpw + g;
                row[u] = src < 64 ? __shfl(mine, src) : -1;
            }
            f4 v[kGatherU][CH];
#pragma unroll
            for (int u = 0; u < kGatherU; ++u)
#pragma unroll
                for (int c = 0; c < CH; ++c)
                    v[u][c] = row[u] >= 0 ? x[(int64_t)row[u] * ld4 + c * G + l] : f4{0, 0, 0, 0};
#pragma unroll
            for (int u = 0; u < kGatherU; ++u)
#pragma unroll
                for (int c = 0; c < CH; ++c) acc += v[u][c];
        }
    }
    sink[(int64_t)blockIdx.x * kPeakThreads + threadIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
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

int gcn_peak_gather(const void *X, int64_t n_rows, int32_t row_bytes, int64_t ld_bytes, const int32_t *idx,
                    int64_t count, float *sink, int32_t blocks, void *stream) {
    if (!X || !idx || !sink || n_rows <= 0 || count < 0 || blocks <= 0) {
        set_error("gcn_peak_gather: null pointer or bad size");
        return GCN_EINVAL;
    }
    if (row_bytes < 16 || row_bytes > 4096 || row_bytes % 16 || ld_bytes < row_bytes || ld_bytes % 16 ||
        ((uintptr_t)X & 15u)) {
        set_error("gcn_peak_gather: row_bytes %d must be a multiple of 16 in [16, 4096], ld_bytes %lld a "
                  "multiple of 16 >= row_bytes, X 16-byte aligned", row_bytes, (long long)ld_bytes);
        return GCN_ESHAPE;
    }
    const int r16 = row_bytes / 16;
    int G = 1;
    while (G < 64 && G < r16) G *= 2;
    if (r16 % G || !(r16 / G == 1 || r16 / G == 2 || r16 / G == 4)) {
        set_error("gcn_peak_gather: row_bytes %d is not 16 times a power of two up to 64, 2 KB or 4 KB",
                  row_bytes);
        return GCN_ESHAPE;
    }
    hipStream_t s = (hipStream_t)stream;
    const int chunks = r16 / G;
    const f4 *x4 = (const f4 *)X;
    const int64_t ld4 = ld_bytes / 16;
    if (chunks == 1) gather_kernel<1><<<blocks, kPeakThreads, 0, s>>>(x4, n_rows, ld4, idx, count, G, sink);
    else if (chunks == 2) gather_kernel<2><<<blocks, kPeakThreads, 0, s>>>(x4, n_rows, ld4, idx, count, G, sink);
    else gather_kernel<4><<<blocks, kPeakThreads, 0, s>>>(x4, n_rows, ld4, idx, count, G, sink);
    GCN_LAUNCH_CHECK("gather_kernel");
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
