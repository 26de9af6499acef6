/*
 * gcn_peaks.h -- machine-rate probes of libgcnlayer.
 *
 * These calls do none of the method's arithmetic.  They measure what this
 * GPU sustains for the resources the layer's kernels are bound by: streaming
 * reads from device memory, row gathers from device memory and the caches
 * (the aggregation of Sec. V-A/V-B is bound by them), the matrix cores (the
 * weight application of Sec. V-A is a dense product) and dependent-load
 * latency (the sampler).  Kernel rates are reported against both the
 * datasheet peak and these measured ceilings.
 *
 * Each call only enqueues one kernel on `stream` (a hipStream_t as void*,
 * NULL = default stream); the caller times it with events on that stream.
 * Errors follow gcn_layer.h: a negative gcn_status with a message for
 * gcn_last_error(), nothing launched.
 */
#ifndef GCN_PEAKS_H_
#define GCN_PEAKS_H_

#include <stdint.h>

#include "gcn_layer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Reads every element of the device array x [count] once with 16-byte loads
 * (count % 4 == 0, x 16-byte aligned) and writes one float per thread to the
 * device array sink [blocks * 256].  Bytes moved: 4 * count read. */
int gcn_peak_stream_read(const float *x, int64_t count, float *sink, int32_t blocks, void *stream);

/* Runs `iters` x 4 independent matrix-core products per wavefront, 4
 * wavefronts per block, on `blocks` blocks: v_mfma_f32_32x32x2f32 for GCN_F32,
 * v_mfma_f32_32x32x16_bf16 for GCN_BF16.  Writes one float per thread to
 * sink [blocks * 256] and the number of floating-point operations issued to
 * *flops (host pointer, may be NULL). */
int gcn_peak_mfma(gcn_prec prec, int32_t blocks, int32_t iters, float *sink, double *flops, void *stream);

/* Row gathers, the access pattern of the feature propagation (Sec. V-B,
 * Alg. 6: every stored edge reads one source row of the features): reads the
 * first row_bytes of rows idx[0 .. count) of X (n_rows rows, ld_bytes apart),
 * each row by a group of min(64, row_bytes / 16) lanes with 16-byte loads,
 * eight rows in flight per group; each wavefront takes 64 consecutive
 * indices at a time, wavefronts walking idx in a grid-stride order over
 * `blocks` blocks of 256 threads; writes one float per thread to sink
 * [blocks * 256].  row_bytes: 16 times a power of two up to 64, 2 KB or
 * 4 KB; ld_bytes a multiple of 16 >= row_bytes; X 16-byte aligned.  Indices outside [0, n_rows) are clamped into it.  Bytes
 * gathered: count * row_bytes (plus 4 * count of indices).  With random
 * indices over an array that fits a CU's L1, an XCD's L2, the 256 MB
 * Infinity Cache or none of them, this is the rate a gather of that row size
 * reaches from that level; with a CSR's column indices it is the gather of
 * one propagation pass without its arithmetic. */
int gcn_peak_gather(const void *X, int64_t n_rows, int32_t row_bytes, int64_t ld_bytes, const int32_t *idx,
                    int64_t count, float *sink, int32_t blocks, void *stream);

/* Latency of dependent global loads: `chains` wavefronts each follow
 * i <- next[i] for `steps` hops from their own start, one load in flight per
 * wavefront; sink [chains] receives the last index.  next [n] must hold
 * values in [0, n) (a random cycle measures the latency of the cache level
 * that an array of n int32 lands in).  Time / steps is the latency per load
 * at that concurrency: the bound of the frontier sampler, whose steps are
 * chains of dependent loads (gcn_sampler.h). */
int gcn_peak_chase(const int32_t *next, int64_t n, int32_t steps, int32_t chains, int32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GCN_PEAKS_H_ */
