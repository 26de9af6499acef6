// Feature propagation within the sampled subgraph: out = A X for CSR A.
//
// This is the first of the two training kernels of Sec. V-A.  The paper's
// 40-core Xeon schedule (Alg. 6) slices the feature dimension so that each
// slice of X stays in a core's cache; on gfx950 the same idea becomes the
// column slice of one wavefront, while the graph dimension is balanced with a
// merge path over (rows + edges):
//
//   * the merge sequence lists, row by row, the row's edges followed by one
//     "row end" item; a wavefront owns `ipw` consecutive items, so a vertex of
//     degree 14,000 is spread over many wavefronts and empty rows cost one item;
//   * for every edge the wavefront reads the source row of X, k contiguous
//     values, with each lane loading VEC consecutive columns (one coalesced
//     row read per wavefront per edge); the edge index and weight are
//     wave-uniform scalar loads;
//   * a row completed inside one wavefront is written once, with the
//     epilogue (store / +bias and ReLU / accumulate) fused;
//   * a row cut by wavefront boundaries leaves float32 partial sums in the
//     workspace, and a fix-up pass owned by the wavefront that completes the
//     row adds them in wavefront order.  No atomics: the result is bitwise
//     reproducible.
//
// Accumulation is float32 in increasing edge order within each piece.
#include <type_traits>

#include "common.h"

namespace gcn {
namespace {

constexpr int kWavesPerBlock = 4;
#ifndef GCN_SPMM_MAIN_U
#define GCN_SPMM_MAIN_U 4
#endif
constexpr int kUnroll = GCN_SPMM_MAIN_U;   // edges in flight per wavefront (spmm_main)
constexpr int kMaxIpw = 256;   // merge items per wavefront, at most
#ifndef GCN_SPMM_U
#define GCN_SPMM_U 4
#endif
// wavefronts per SIMD the register allocation must allow: the gathers are
// latency-bound, so the bytes in flight per CU (wavefronts x loads each) set
// the rate; the sliced kernel fits 8 without spilling (64 VGPRs)
#ifndef GCN_SPMM_MAIN_WPE
#define GCN_SPMM_MAIN_WPE 1
#endif
#ifndef GCN_SPMM_SLICED_WPE
#define GCN_SPMM_SLICED_WPE 8
#endif
// float32 sliced kernel: lanes per row piece, 16 or 32 (64- or 128-column
// slices; at 512 columns 32 lanes: 1.120 against 1.147 ms per step of three
// aggregations)
#ifndef GCN_SPMM_LP
#define GCN_SPMM_LP 32
#endif
// bfloat16 rows on the XCD-sliced schedule: switch, edges in flight per lane
// group, lanes per row piece and the occupancy target (measured at 512
// columns: 32 lanes (256-column slices) 0.64 ms per step of three
// aggregations, 16 lanes 0.72, 8 lanes 1.00, whole 1 KB rows unsliced 0.79;
// 2, 6 or 8 edges in flight and 6 wavefronts per SIMD were slower)
#ifndef GCN_SPMM_BF16_SLICED
#define GCN_SPMM_BF16_SLICED 1
#endif
#ifndef GCN_SPMM_BF16_U
#define GCN_SPMM_BF16_U 4
#endif
#ifndef GCN_SPMM_BF16_LP
#define GCN_SPMM_BF16_LP 32   // lanes per row piece: 8, 16 or 32 (64, 128 or 256 columns)
#endif
#ifndef GCN_SPMM_BF16_WPE
#define GCN_SPMM_BF16_WPE 8
#endif


// Smallest r in [0, n_rows] whose row-end item sits at merge position >= d,
// i.e. indptr[r+1] + r >= d (n_rows when none does).  64-ary search: every
// lane probes one point of the current interval per round.
__device__ __forceinline__ int merge_search(const int32_t *__restrict__ indptr, int32_t n_rows,
                                            int64_t d, int lane) {
    int64_t lo = 0, hi = n_rows;
    while (lo < hi) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t q = lo + (int64_t)lane * step;
        bool pred = false;
        if (q < hi) pred = (int64_t)indptr[q + 1] + q >= d;
        const unsigned long long mask = __ballot(pred);
        if (mask) {
            const int l = __ffsll(mask) - 1;
            const int64_t qs = lo + (int64_t)l * step;
            lo = (l == 0) ? lo : qs - step + 1;
            hi = qs;
        } else {
            const int64_t last = (hi - 1 - lo) / step;
            lo = lo + last * step + 1;
        }
    }
    return (int)lo;
}

// The merge range of one wavefront: rows r0..r1 (r1 may be cut or n_rows)
// and edge positions [p0, p1).  Its edges (at most kMaxIpw) and row pointers
// are copied into LDS with coalesced loads, so that the gather loop waits on
// one global load per edge, the feature row, instead of three dependent ones
// (row pointer, edge index, feature row).
struct EdgeStage {
    int32_t idx[kWavesPerBlock][kMaxIpw];
    float val[kWavesPerBlock][kMaxIpw];
    int32_t ptr[kWavesPerBlock][kMaxIpw + 2];
};
struct WaveRange {
    int r0, r1;
    int64_t p0, p1;
};
// Every thread of the block calls it (it ends with a block barrier); `live`
// is false for wavefronts past the last merge range.  bnd[w] is the first row
// of merge range w (spmm_bounds_kernel).
__device__ __forceinline__ WaveRange stage_wave(EdgeStage &st, int wv, int lane, bool live, int64_t wave,
                                                int ipw, int64_t items, int32_t n_rows,
                                                const int32_t *__restrict__ bnd,
                                                const int32_t *__restrict__ indptr,
                                                IdxRef indices,
                                                const float *__restrict__ vals) {
    WaveRange w{0, 0, 0, 0};
    if (live) {
        const int64_t d0 = wave * ipw;
        const int64_t d1 = d0 + ipw < items ? d0 + ipw : items;
        w.r0 = bnd[wave];
        w.r1 = bnd[wave + 1];
        w.p0 = d0 - w.r0;
        w.p1 = d1 - w.r1;
        for (int i = lane; i < (int)(w.p1 - w.p0); i += 64) {
            st.idx[wv][i] = indices[w.p0 + i];
            st.val[wv][i] = vals[w.p0 + i];
        }
        const int nr = min(w.r1, n_rows - 1) - w.r0 + 2;   // pointers r0 .. min(r1, n_rows - 1) + 1
        for (int i = lane; i < nr; i += 64) st.ptr[wv][i] = indptr[w.r0 + i];
    }
    __syncthreads();
    return w;
}

// bnd[w] = the row holding merge position min(w * ipw, items), w = 0 ..
// waves (n_rows for the end): the row ranges of all wavefronts, searched once
// per product rather than by every wavefront of every column slice.
__global__ __launch_bounds__(256) void spmm_bounds_kernel(int32_t n_rows, const int32_t *__restrict__ indptr,
                                                          int64_t items, int ipw, int64_t waves,
                                                          int32_t *__restrict__ bnd) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (w > waves) return;
    const int64_t d = w * ipw < items ? w * ipw : items;
    const int r = merge_search(indptr, n_rows, d, lane);
    if (lane == 0) bnd[w] = r;
}

// One lane's VEC consecutive elements of a gathered row.  bfloat16 rows keep
// the loaded words and widen an element when it is used, so a gather in
// flight holds VEC/2 registers rather than VEC.
template <int VEC, bool BF16> struct Row;
template <int VEC> struct Row<VEC, false> {
    float v[VEC];
    __device__ void load(const float *p) {
        if constexpr (VEC == 4) {
            const float4 t = *(const float4 *)p;
            v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        } else if constexpr (VEC == 2) {
            const float2 t = *(const float2 *)p;
            v[0] = t.x; v[1] = t.y;
        } else {
            v[0] = *p;
        }
    }
    __device__ float get(int i) const { return v[i]; }
};
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
template <int VEC> struct Row<VEC, true> {
    static constexpr int W = VEC >= 2 ? VEC / 2 : 1;
    uint32_t w[W];
    __device__ void load(const uint16_t *p) {
        if constexpr (VEC == 8) {
            const uint4 t = *(const uint4 *)p;
            w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
        } else if constexpr (VEC == 4) {
            const uint2 t = *(const uint2 *)p;
            w[0] = t.x; w[1] = t.y;
        } else if constexpr (VEC == 2) {
            w[0] = *(const uint32_t *)p;
        } else {
            w[0] = (uint32_t)(*p);
        }
    }
    __device__ float get(int i) const {
        if constexpr (VEC == 1) return __uint_as_float(w[0] << 16);
        return (i & 1) ? bf16_hi(w[i >> 1]) : bf16_lo(w[i >> 1]);
    }
};

// float32 -> bfloat16 as to_bf16, written with the NaN case as a branch: in
// the gather kernels this form keeps the bfloat16 variant within its 72-VGPR
// budget (the select form and the paired hardware rounding spill there)
__device__ __forceinline__ uint16_t bf16_round(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x0040u);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Final value of out[r, c .. c+VEC) under the epilogue; `out` is float, or
// bfloat16 bits for EPI_STORE_BF16 (ldo counts elements of either type), and
// may be null when only the bfloat16 copy is wanted.  out16 (when set): the
// same final values as bfloat16 rows (leading dim ld16), for the float32
// epilogues other than accumulate.
// ovec: the VEC elements are one aligned vector (ldo a multiple of VEC and
// `out` aligned to min(16, VEC * element size) bytes, and the same for
// out16 when it is set), moved with 16-, 8- or 4-byte accesses instead of
// one access per element.  bias (EPI_BIAS_RELU): the bias of column c, so
// that bias[v] belongs to column c + v; the gather kernels pass their block's
// copy in LDS, whose reads do not wait behind the row gathers in flight.
// HWR: pairs rounded by the gfx950 pair instruction (pack_bf16x2, the same
// bits), where the kernel's register budget allows it
template <int VEC, bool HWR = false>
__device__ __forceinline__ void store16(uint16_t *__restrict__ o, const float (&x)[VEC], bool ovec) {
    if (VEC >= 2 && ovec) {
        uint32_t w[VEC / 2 > 0 ? VEC / 2 : 1];
#pragma unroll
        for (int i = 0; i < VEC / 2; ++i)
            w[i] = HWR ? pack_bf16x2(x[2 * i], x[2 * i + 1])
                       : (uint32_t)bf16_round(x[2 * i]) | ((uint32_t)bf16_round(x[2 * i + 1]) << 16);
        if constexpr (VEC == 8) *(uint4 *)o = make_uint4(w[0], w[1], w[2], w[3]);
        else if constexpr (VEC == 4) *(uint2 *)o = make_uint2(w[0], w[1]);
        else *(uint32_t *)o = w[0];
        return;
    }
#pragma unroll
    for (int v = 0; v < VEC; ++v) o[v] = bf16_round(x[v]);
}

template <int VEC, int OM = 0, bool HWR = false>
__device__ __forceinline__ void emit(void *__restrict__ out, int64_t ldo, int64_t r, int c,
                                     const float (&acc)[VEC], int epi, const float *__restrict__ bias,
                                     bool ovec, uint16_t *__restrict__ out16 = nullptr, int64_t ld16 = 0) {
    if (epi == EPI_STORE_BF16) {
        store16<VEC, HWR>((uint16_t *)out + r * ldo + c, acc, ovec);
        return;
    }
    if constexpr (OM == 0) {   // one float32 output
        float *o = (float *)out + r * ldo + c;
        if (VEC >= 4 && ovec) {
#pragma unroll
            for (int q = 0; q < VEC / 4; ++q) {
                float x[4] = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
                if (epi == EPI_BIAS_RELU) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) x[e] = fmaxf(x[e] + bias[4 * q + e], 0.0f);
                } else if (epi == EPI_ACCUMULATE) {
                    const float4 p = *(const float4 *)(o + 4 * q);
                    x[0] = p.x + x[0]; x[1] = p.y + x[1]; x[2] = p.z + x[2]; x[3] = p.w + x[3];
                }
                *(float4 *)(o + 4 * q) = make_float4(x[0], x[1], x[2], x[3]);
            }
            return;
        }
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            float x = acc[v];
            if (epi == EPI_BIAS_RELU) x = fmaxf(x + bias[v], 0.0f);
            else if (epi == EPI_ACCUMULATE) x = o[v] + x;
            o[v] = x;
        }
        return;
    }
    if constexpr (OM == 1) {   // the bfloat16 copy only: pack as the values are finished
        uint16_t *o16 = out16 + r * ld16 + c;
        auto fin = [&](int v) {
            return epi == EPI_BIAS_RELU ? fmaxf(acc[v] + bias[v], 0.0f) : acc[v];
        };
        if (VEC >= 2 && ovec) {
            uint32_t w[VEC / 2 > 0 ? VEC / 2 : 1];
#pragma unroll
            for (int i = 0; i < VEC / 2; ++i)
                w[i] = HWR ? pack_bf16x2(fin(2 * i), fin(2 * i + 1))
                           : (uint32_t)bf16_round(fin(2 * i)) | ((uint32_t)bf16_round(fin(2 * i + 1)) << 16);
            if constexpr (VEC == 8) *(uint4 *)o16 = make_uint4(w[0], w[1], w[2], w[3]);
            else if constexpr (VEC == 4) *(uint2 *)o16 = make_uint2(w[0], w[1]);
            else *(uint32_t *)o16 = w[0];
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) o16[v] = bf16_round(fin(v));
        }
        return;
    }
    float *o = out ? (float *)out + r * ldo + c : nullptr;
    float x[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) x[v] = acc[v];
    if (epi == EPI_BIAS_RELU) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) x[v] = fmaxf(x[v] + bias[v], 0.0f);
    } else if (epi == EPI_ACCUMULATE) {
        if (VEC >= 4 && ovec) {
#pragma unroll
            for (int q = 0; q < VEC / 4; ++q) {
                const float4 p = *(const float4 *)(o + 4 * q);
                x[4 * q] = p.x + x[4 * q]; x[4 * q + 1] = p.y + x[4 * q + 1];
                x[4 * q + 2] = p.z + x[4 * q + 2]; x[4 * q + 3] = p.w + x[4 * q + 3];
            }
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) x[v] = o[v] + x[v];
        }
    }
    if (o) {
        if (VEC >= 4 && ovec) {
#pragma unroll
            for (int q = 0; q < VEC / 4; ++q)
                *(float4 *)(o + 4 * q) = make_float4(x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]);
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) o[v] = x[v];
        }
    }
    if (out16) store16<VEC, HWR>(out16 + r * ld16 + c, x, ovec);
}

template <int VEC>
__device__ __forceinline__ void store_raw(float *__restrict__ out, const float (&acc)[VEC]) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) out[v] = acc[v];
}

// One wavefront = `ipw` merge items x one column slice of width 64*VEC*CT.
// OM: the epilogue's outputs, 0 `out` only, 1 the bfloat16 copy out16 only,
// 2 both; separate instantiations, so that the common kernels carry no
// registers for the copy.
template <int VEC, int CT, bool BF16, int OM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(OM == 1 && CT == 1 ? 7 : GCN_SPMM_MAIN_WPE)))
void spmm_main(
    int32_t n_rows, const int32_t *__restrict__ indptr, IdxRef indices,
    const float *__restrict__ vals, const void *__restrict__ Xv, int32_t k, int64_t ldx,
    void *__restrict__ out, int64_t ldo, int epi, const float *__restrict__ bias, int ovec,
    int64_t items, int ipw, int64_t waves, const int32_t *__restrict__ bnd, float *__restrict__ carry,
    int32_t *__restrict__ head_row, int32_t *__restrict__ tail_row, uint16_t *__restrict__ out16, int64_t ld16) {
    using Elem = typename std::conditional<BF16, uint16_t, float>::type;
    const Elem *__restrict__ X = (const Elem *)Xv;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    constexpr int SW = 64 * VEC * CT;
    __shared__ EdgeStage st;
    // the bias of the block's column slice (published by stage_wave's barrier)
    __shared__ float bias_s[SW];
    if (epi == EPI_BIAS_RELU)
        for (int i = threadIdx.x; i < SW; i += 256) {
            const int c = blockIdx.y * SW + i;
            bias_s[i] = c < k ? bias[c] : 0.0f;
        }
    const bool live = wave < waves;
    const WaveRange wr = stage_wave(st, wv, lane, live, wave, ipw, items, n_rows, bnd, indptr, indices, vals);
    if (!live) return;
    const int r0 = wr.r0, r1 = wr.r1;
    const int64_t p0 = wr.p0, p1 = wr.p1;
    const int32_t *const e_idx = st.idx[wv];
    const float *const e_val = st.val[wv];
    const int32_t *const r_ptr = st.ptr[wv];

    const int cbase = blockIdx.y * SW + lane * VEC;
    bool cok[CT];
#pragma unroll
    for (int t = 0; t < CT; ++t) cok[t] = cbase + t * 64 * VEC < k;

    // edge positions relative to p0 (32-bit: nnz < 2^31), as staged in LDS
    const int q0 = (int)p0;
    int32_t hrow = -1, trow = -1;
    for (int r = r0; r <= r1 && r < n_rows; ++r) {
        const int rb = r_ptr[r - r0], re = r_ptr[r - r0 + 1];
        const bool complete = r < r1;
        const int pb = (q0 > rb ? q0 : rb) - q0;
        const int pe = (complete ? re : (int)p1) - q0;
        float acc[CT][VEC];
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[t][v] = 0.0f;

        int p = pb;
        for (; p + kUnroll <= pe; p += kUnroll) {
            int32_t j[kUnroll];
            float w[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) { j[u] = e_idx[p + u]; w[u] = e_val[p + u]; }
            Row<VEC, BF16> x[kUnroll][CT];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int t = 0; t < CT; ++t)
                    if (cok[t]) x[u][t].load(X + (int64_t)j[u] * ldx + cbase + t * 64 * VEC);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int t = 0; t < CT; ++t)
                    if (cok[t])
#pragma unroll
                        for (int v = 0; v < VEC; ++v) acc[t][v] = fmaf(w[u], x[u][t].get(v), acc[t][v]);
        }
        for (; p < pe; ++p) {
            const int32_t j = e_idx[p];
            const float w = e_val[p];
#pragma unroll
            for (int t = 0; t < CT; ++t)
                if (cok[t]) {
                    Row<VEC, BF16> x;
                    x.load(X + (int64_t)j * ldx + cbase + t * 64 * VEC);
#pragma unroll
                    for (int v = 0; v < VEC; ++v) acc[t][v] = fmaf(w, x.get(v), acc[t][v]);
                }
        }

        const bool started = (r > r0) || (q0 == rb);
        if (complete && started) {
#pragma unroll
            for (int t = 0; t < CT; ++t)
                if (cok[t]) {
                    const int c = cbase + t * 64 * VEC;
                    emit<VEC, OM>(out, ldo, r, c, acc[t], epi, bias_s + lane * VEC + t * 64 * VEC, ovec != 0, out16, ld16);
                }
        } else if (complete || pe > pb) {
            // a piece of a row cut by wavefront boundaries: head (the piece
            // that completes the row) or tail (a piece that does not)
            const int slot = complete ? 0 : 1;
            float *dst = carry + (2 * wave + slot) * (int64_t)k;
#pragma unroll
            for (int t = 0; t < CT; ++t)
                if (cok[t]) store_raw<VEC>(dst + cbase + t * 64 * VEC, acc[t]);
            if (complete) hrow = r; else trow = r;
        }
    }
    if (blockIdx.y == 0 && lane == 0) {
        head_row[wave] = hrow;
        tail_row[wave] = trow;
    }
}

// XCD-sliced variant (float32, k % 4 == 0).  The feature dimension is cut
// into slices of 4 * LP columns (128 by default) and workgroups are numbered
// so that, under the round-robin workgroup-to-XCD dispatch, each XCD keeps
// gathering the same slice: its 4 MB L2 then holds the hot rows of one slice
// (512 B per row at 128 columns) instead of whole rows, which raises the hit
// rate on skewed graphs.  This is the feature-only partitioning of Sec. V-B /
// Alg. 6, with the XCD L2 in the role of the per-core cache.  Inside a
// wavefront, lane group g = lane / LP gathers edges g, g + 64/LP, ... of the
// row (LP lanes x float4), and the groups' partial sums are combined with a
// fixed xor-shuffle tree.
struct SliceMap {
    int32_t slices;      // ceil(k / slice width)
    int32_t chunks;      // block chunks of kWavesPerBlock wavefronts
    int32_t mode;        // 0: slice-major multiple of 8, 1: slice divides 8, 2: plain
    int32_t per_xcd;     // slices per XCD (mode 0) or XCDs per slice (mode 1)
};

__device__ __forceinline__ bool slice_of_block(const SliceMap &m, int64_t w, int &slice, int64_t &chunk) {
    if (m.mode == 0) {
        const int64_t x = w & 7, r = w >> 3;
        slice = (int)(x + 8 * (r % m.per_xcd));
        chunk = r / m.per_xcd;
    } else if (m.mode == 1) {
        const int64_t x = w & 7, r = w >> 3;
        slice = (int)(x % m.slices);
        chunk = r * m.per_xcd + x / m.slices;
    } else {
        slice = (int)(w % m.slices);
        chunk = w / m.slices;
    }
    return chunk < m.chunks;
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(GCN_SPMM_SLICED_WPE)))
void spmm_sliced(
    int32_t n_rows, const int32_t *__restrict__ indptr, IdxRef indices,
    const float *__restrict__ vals, const float *__restrict__ X, int32_t k, int64_t ldx,
    void *__restrict__ out, int64_t ldo, int epi, const float *__restrict__ bias,
    int64_t items, int ipw, int64_t waves, SliceMap map, const int32_t *__restrict__ bnd,
    float *__restrict__ carry, int32_t *__restrict__ head_row, int32_t *__restrict__ tail_row,
    uint16_t *__restrict__ out16, int64_t ld16) {
    constexpr int LP = GCN_SPMM_LP;   // lanes per row piece
    constexpr int NG = 64 / LP;       // lane groups
    constexpr int SWD = 4 * LP;       // slice width
    static_assert(LP == 16 || LP == 32, "lane groups of 16 or 32");
    int slice;
    int64_t chunk;
    if (!slice_of_block(map, blockIdx.x, slice, chunk)) return;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t wave = chunk * kWavesPerBlock + wv;
    __shared__ EdgeStage st;
    // the bias of the block's slice (published by stage_wave's barrier)
    __shared__ float bias_s[SWD];
    if (epi == EPI_BIAS_RELU && threadIdx.x < SWD)
        bias_s[threadIdx.x] = slice * SWD + (int)threadIdx.x < k ? bias[slice * SWD + threadIdx.x] : 0.0f;
    const bool live = wave < waves;
    const WaveRange wr = stage_wave(st, wv, lane, live, wave, ipw, items, n_rows, bnd, indptr, indices, vals);
    if (!live) return;
    const int r0 = wr.r0, r1 = wr.r1;
    const int64_t p0 = wr.p0, p1 = wr.p1;
    const int32_t *const e_idx = st.idx[wv];
    const float *const e_val = st.val[wv];
    const int32_t *const r_ptr = st.ptr[wv];
    const int g = lane / LP;
    const int col = slice * SWD + (lane % LP) * 4;
    const bool cok = col < k;
    constexpr int U = GCN_SPMM_U;  // edges per lane group in flight

    // edge positions relative to p0 (32-bit: nnz < 2^31), as staged in LDS
    const int q0 = (int)p0;
    int32_t hrow = -1, trow = -1;
    for (int r = r0; r <= r1 && r < n_rows; ++r) {
        const int rb = r_ptr[r - r0], re = r_ptr[r - r0 + 1];
        const bool complete = r < r1;
        const int pb = (q0 > rb ? q0 : rb) - q0;
        const int pe = (complete ? re : (int)p1) - q0;
        float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, a3 = 0.0f;
        int p = pb + g;
        for (; p + NG * (U - 1) < pe; p += NG * U) {
            int32_t j[U];
            float w[U];
#pragma unroll
            for (int u = 0; u < U; ++u) { j[u] = e_idx[p + NG * u]; w[u] = e_val[p + NG * u]; }
            float4 x[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                x[u] = cok ? *(const float4 *)(X + (int64_t)j[u] * ldx + col) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                a0 = fmaf(w[u], x[u].x, a0);
                a1 = fmaf(w[u], x[u].y, a1);
                a2 = fmaf(w[u], x[u].z, a2);
                a3 = fmaf(w[u], x[u].w, a3);
            }
        }
        for (; p < pe; p += NG) {
            const int32_t j = e_idx[p];
            const float w = e_val[p];
            const float4 x = cok ? *(const float4 *)(X + (int64_t)j * ldx + col) : make_float4(0.f, 0.f, 0.f, 0.f);
            a0 = fmaf(w, x.x, a0);
            a1 = fmaf(w, x.y, a1);
            a2 = fmaf(w, x.z, a2);
            a3 = fmaf(w, x.w, a3);
        }
        // neighbouring groups, then the pairs (a fixed tree)
#pragma unroll
        for (int o = LP; o < 64; o *= 2) {
            a0 += __shfl_xor(a0, o); a1 += __shfl_xor(a1, o); a2 += __shfl_xor(a2, o); a3 += __shfl_xor(a3, o);
        }
        const float acc[4] = {a0, a1, a2, a3};
        const bool started = (r > r0) || (q0 == rb);
        if (g == 0 && cok) {
            if (complete && started) {
                emit<4, 2>(out, ldo, r, col, acc, epi, bias_s + (lane % LP) * 4, true, out16, ld16);   // aligned (host checks)
            } else if (complete || pe > pb) {
                const int slot = complete ? 0 : 1;
                store_raw<4>(carry + (2 * wave + slot) * (int64_t)k + col, acc);
            }
        }
        if (!(complete && started) && (complete || pe > pb)) {
            if (complete) hrow = r; else trow = r;
        }
    }
    if (slice == 0 && lane == 0) {
        head_row[wave] = hrow;
        tail_row[wave] = trow;
    }
}

// The same schedule for bfloat16 rows.  A lane group of LP lanes gathers an
// 8 * LP-column piece of a row (8 bfloat16 columns per lane, kept as loaded
// words and widened on use), 64 / LP edges per gather instruction, and the
// groups' sums are combined by a fixed xor-shuffle tree.  With 32 lanes at 512
// columns there are two slices, each on four XCDs, whose L2s then hold
// 512-byte pieces of twice as many hot rows as whole 1 KB rows would allow.
// OM selects the epilogue's outputs as in spmm_main.
template <int OM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(GCN_SPMM_BF16_WPE)))
void spmm_sliced_bf16(
    int32_t n_rows, const int32_t *__restrict__ indptr, IdxRef indices,
    const float *__restrict__ vals, const uint16_t *__restrict__ X, int32_t k, int64_t ldx,
    void *__restrict__ out, int64_t ldo, int epi, const float *__restrict__ bias,
    int64_t items, int ipw, int64_t waves, SliceMap map, const int32_t *__restrict__ bnd,
    float *__restrict__ carry, int32_t *__restrict__ head_row, int32_t *__restrict__ tail_row,
    uint16_t *__restrict__ out16, int64_t ld16) {
    constexpr int LP = GCN_SPMM_BF16_LP;   // lanes per row piece
    constexpr int NG = 64 / LP;            // lane groups (edges per gather instruction)
    constexpr int SWD = 8 * LP;
    static_assert(LP == 8 || LP == 16 || LP == 32, "lane groups of 8, 16 or 32");
    int slice;
    int64_t chunk;
    if (!slice_of_block(map, blockIdx.x, slice, chunk)) return;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t wave = chunk * kWavesPerBlock + wv;
    __shared__ EdgeStage st;
    // the bias of the block's slice (published by stage_wave's barrier)
    __shared__ float bias_s[SWD];
    if (epi == EPI_BIAS_RELU && threadIdx.x < SWD)
        bias_s[threadIdx.x] = slice * SWD + (int)threadIdx.x < k ? bias[slice * SWD + threadIdx.x] : 0.0f;
    const bool live = wave < waves;
    const WaveRange wr = stage_wave(st, wv, lane, live, wave, ipw, items, n_rows, bnd, indptr, indices, vals);
    if (!live) return;
    const int r0 = wr.r0, r1 = wr.r1;
    const int64_t p0 = wr.p0, p1 = wr.p1;
    const int32_t *const e_idx = st.idx[wv];
    const float *const e_val = st.val[wv];
    const int32_t *const r_ptr = st.ptr[wv];
    const int g = lane / LP;
    const int col = slice * SWD + (lane % LP) * 8;
    const bool cok = col < k;
    constexpr int U = GCN_SPMM_BF16_U;

    const int q0 = (int)p0;
    int32_t hrow = -1, trow = -1;
    for (int r = r0; r <= r1 && r < n_rows; ++r) {
        const int rb = r_ptr[r - r0], re = r_ptr[r - r0 + 1];
        const bool complete = r < r1;
        const int pb = (q0 > rb ? q0 : rb) - q0;
        const int pe = (complete ? re : (int)p1) - q0;
        float a[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) a[v] = 0.0f;
        int p = pb + g;
        for (; p + NG * (U - 1) < pe; p += NG * U) {
            int32_t j[U];
            float w[U];
#pragma unroll
            for (int u = 0; u < U; ++u) { j[u] = e_idx[p + NG * u]; w[u] = e_val[p + NG * u]; }
            Row<8, true> x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (cok) {
                    x[u].load(X + (int64_t)j[u] * ldx + col);
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q) x[u].w[q] = 0u;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int v = 0; v < 8; ++v) a[v] = fmaf(w[u], x[u].get(v), a[v]);
        }
        for (; p < pe; p += NG) {
            const int32_t j = e_idx[p];
            const float w = e_val[p];
            Row<8, true> x;
            if (cok) {
                x.load(X + (int64_t)j * ldx + col);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) x.w[q] = 0u;
            }
#pragma unroll
            for (int v = 0; v < 8; ++v) a[v] = fmaf(w, x.get(v), a[v]);
        }
        // neighbouring groups, then pairs of pairs, ... (a fixed tree)
#pragma unroll
        for (int o = LP; o < 64; o *= 2)
#pragma unroll
            for (int v = 0; v < 8; ++v) a[v] += __shfl_xor(a[v], o);
        const bool started = (r > r0) || (q0 == rb);
        if (g == 0 && cok) {
            if (complete && started) {
                emit<8, OM, OM != 2>(out, ldo, r, col, a, epi, bias_s + (lane % LP) * 8, true, out16, ld16);   // aligned (host checks; the pair rounding where it fits the registers)
            } else if (complete || pe > pb) {
                const int slot = complete ? 0 : 1;
                store_raw<8>(carry + (2 * wave + slot) * (int64_t)k + col, a);
            }
        }
        if (!(complete && started) && (complete || pe > pb)) {
            if (complete) hrow = r; else trow = r;
        }
    }
    if (slice == 0 && lane == 0) {
        head_row[wave] = hrow;
        tail_row[wave] = trow;
    }
}

SliceMap make_slice_map(int32_t k, int64_t waves, int32_t width = 64) {
    SliceMap m;
    m.slices = (k + width - 1) / width;
    const int64_t chunks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    m.chunks = (int32_t)chunks;
    if (m.slices % 8 == 0) {
        m.mode = 0;
        m.per_xcd = m.slices / 8;
    } else if (8 % m.slices == 0) {
        m.mode = 1;
        m.per_xcd = 8 / m.slices;
    } else {
        m.mode = 2;
        m.per_xcd = 1;
    }
    return m;
}

int64_t slice_map_blocks(const SliceMap &m) {
    if (m.mode == 0) return 8 * (int64_t)m.per_xcd * m.chunks;
    if (m.mode == 1) return 8 * (((int64_t)m.chunks + m.per_xcd - 1) / m.per_xcd);
    return (int64_t)m.slices * m.chunks;
}

// Completes every row cut by wavefront boundaries: the wavefront w holding the
// row's head piece sums the tail pieces of the preceding wavefronts in order,
// then its own head piece, and applies the epilogue.
__global__ __launch_bounds__(256) void spmm_fixup(int32_t k, void *__restrict__ out, int64_t ldo,
                                                  int epi, const float *__restrict__ bias,
                                                  int64_t waves, const float *__restrict__ carry,
                                                  const int32_t *__restrict__ head_row,
                                                  const int32_t *__restrict__ tail_row,
                                                  uint16_t *__restrict__ out16, int64_t ld16) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (w >= waves) return;
    // One round of independent loads: the head row of w, the tail rows of
    // its 64 predecessors, w's own head piece and the tail piece of w - 1
    // (the whole run in the common case of a row cut once; both slots are in
    // bounds whether or not they were written), instead of four dependent
    // rounds.
    const int c0 = blockIdx.y * 256 + lane;
    const int64_t q1 = w - 1 - lane;
    const int32_t t1 = q1 >= 0 ? tail_row[q1] : -1;
    const int32_t r = head_row[w];
    float hv[4], tv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int c = c0 + 64 * j;
        hv[j] = c < k ? carry[(2 * w) * (int64_t)k + c] : 0.0f;
        tv[j] = c < k && w > 0 ? carry[(2 * w - 1) * (int64_t)k + c] : 0.0f;
    }
    if (r < 0) return;
    // first wavefront of the run of wavefronts whose tail pieces belong to
    // row r, 64 predecessors per step (a long row spans many wavefronts)
    uint64_t brk = __ballot(t1 != r);
    int64_t ws = w;
    while (brk == 0) {
        ws -= 64;
        const int64_t q = ws - 1 - lane;
        brk = __ballot(!(q >= 0 && tail_row[q] == r));
    }
    ws -= __ffsll((unsigned long long)brk) - 1;
    // four columns per lane; the pieces are added in wavefront order, four
    // loads in flight per column
    float acc[4];
    bool any = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = 0.0f;
    // the pieces of wavefronts ws .. w-2, then that of w-1 (loaded above)
    int64_t q = ws;
    for (; q + 4 <= w - 1; q += 4) {
        float v[4][4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int c = c0 + 64 * j;
                v[u][j] = c < k ? carry[(2 * (q + u) + 1) * (int64_t)k + c] : 0.0f;
            }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[j] = (any || u > 0) ? acc[j] + v[u][j] : v[u][j];
        any = true;
    }
    for (; q < w - 1; ++q) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = c0 + 64 * j;
            const float v = c < k ? carry[(2 * q + 1) * (int64_t)k + c] : 0.0f;
            acc[j] = any ? acc[j] + v : v;
        }
        any = true;
    }
    if (ws < w) {
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = any ? acc[j] + tv[j] : tv[j];
        any = true;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int c = c0 + 64 * j;
        if (c >= k) continue;
        const float a[1] = {any ? acc[j] + hv[j] : hv[j]};
        emit<1, 2>(out, ldo, r, c, a, epi, epi == EPI_BIAS_RELU ? bias + c : bias, false, out16, ld16);
    }
}

template <int VEC, int CT, bool BF16>
void launch_main(dim3 grid, hipStream_t s, int32_t n_rows, const int32_t *indptr,
                 IdxRef indices, const float *vals, const void *X, int32_t k, int64_t ldx,
                 void *out, int64_t ldo, int epi, const float *bias, const SpmmPlan &pl,
                 const int32_t *bnd, float *carry, int32_t *hr, int32_t *tr, uint16_t *out16, int64_t ld16) {
    // the epilogue's per-lane VEC outputs as one vector store when aligned
    const size_t chunk = std::min<size_t>(16, (size_t)VEC * (epi == EPI_STORE_BF16 ? 2 : 4));
    const size_t chunk16 = std::min<size_t>(16, (size_t)VEC * 2);
    const int ovec = ldo % VEC == 0 && (uintptr_t)out % chunk == 0 &&
                     (!out16 || (ld16 % VEC == 0 && (uintptr_t)out16 % chunk16 == 0));
    if (out16 && out)
        hipLaunchKernelGGL((spmm_main<VEC, CT, BF16, 2>), grid, dim3(256), 0, s, n_rows, indptr, indices,
                           vals, X, k, ldx, out, ldo, epi, bias, ovec, pl.items, pl.ipw, pl.waves, bnd, carry, hr,
                           tr, out16, ld16);
    else if (out16)
        hipLaunchKernelGGL((spmm_main<VEC, CT, BF16, 1>), grid, dim3(256), 0, s, n_rows, indptr, indices,
                           vals, X, k, ldx, nullptr, ldo, epi, bias, ovec, pl.items, pl.ipw, pl.waves, bnd, carry,
                           hr, tr, out16, ld16);
    else
        hipLaunchKernelGGL((spmm_main<VEC, CT, BF16, 0>), grid, dim3(256), 0, s, n_rows, indptr, indices,
                           vals, X, k, ldx, out, ldo, epi, bias, ovec, pl.items, pl.ipw, pl.waves, bnd, carry, hr,
                           tr, nullptr, 0);
}

bool aligned(const void *p, int bytes) { return ((uintptr_t)p % (uintptr_t)bytes) == 0; }

int spmm_any(bool bf16, int32_t n_rows, int32_t nnz, const int32_t *indptr, IdxRef indices,
             const float *vals, const void *X, int32_t k, int64_t ldx, void *out, int64_t ldo,
             int epi, const float *bias, void *ws, size_t ws_bytes, hipStream_t s, const int32_t *bounds,
             uint16_t *out16, int64_t ld16) {
    if (n_rows <= 0 || k <= 0) return GCN_OK;
    const SpmmPlan pl = spmm_plan(n_rows, nnz);
    Arena ar(ws, ws_bytes);
    float *carry = ar.take<float>((size_t)2 * pl.waves * k);
    int32_t *hr = ar.take<int32_t>(pl.waves);
    int32_t *tr = ar.take<int32_t>(pl.waves);
    int32_t *bnd_ws = ar.take<int32_t>(pl.waves + 1);
    if (!carry || !hr || !tr || !bnd_ws) {
        set_error("spmm: workspace too small (%zu < %zu bytes)", ws_bytes,
                  spmm_workspace_bytes(n_rows, nnz, k));
        return GCN_EWORKSPACE;
    }
    const int esz = bf16 ? 2 : 4;
    // widest per-lane vector that divides k, the leading dimensions and the
    // base pointers
    int vec = bf16 ? 8 : 4;
    while (vec > 1 && !(k % vec == 0 && ldx % vec == 0 && aligned(X, vec * esz))) vec /= 2;
    // narrow rows: keep lanes busy by lowering the vector width
    while (vec > 1 && 64 * (vec / 2) >= k) vec /= 2;
    int ct = (k + 64 * vec - 1) / (64 * vec);
    if (ct > 2) ct = 2;
    const int sw = 64 * vec * ct;
    dim3 grid((unsigned)((pl.waves + kWavesPerBlock - 1) / kWavesPerBlock), (unsigned)((k + sw - 1) / sw));
    if ((out16 && (epi == EPI_ACCUMULATE || epi == EPI_STORE_BF16)) || (!out && !out16)) {
        set_error("spmm: a bfloat16 copy goes with the store or bias+ReLU epilogue, and some output is needed");
        return GCN_EINVAL;
    }
    if (epi == EPI_BIAS_RELU && !bias) {
        set_error("spmm: the bias+ReLU epilogue needs a bias");
        return GCN_EINVAL;
    }
    const bool sliced = !bf16 && k % 4 == 0 && ldx % 4 == 0 && aligned(X, 16) && ldo % 4 == 0 &&
                        aligned(out, 16) && k >= 128 && (!out16 || (ld16 % 4 == 0 && aligned(out16, 8)));
    // bfloat16 rows on the sliced schedule: whole 8-column lane vectors and
    // 16-byte aligned rows in and out
    const bool sliced16 = GCN_SPMM_BF16_SLICED && bf16 && k >= 256 && k % 8 == 0 && ldx % 8 == 0 &&
                          aligned(X, 16) && (!out || (ldo % 8 == 0 && aligned(out, 16))) &&
                          (!out16 || (ld16 % 8 == 0 && aligned(out16, 16)));
    const double out_bytes = epi == EPI_STORE_BF16 ? 2.0 : (epi == EPI_ACCUMULATE ? 8.0 : 4.0);
    const double bytes = (double)nnz * k * esz + (double)nnz * (indices.i16 ? 6.0 : 8.0) + (double)(n_rows + 1) * 4.0 +
                         (double)n_rows * k * out_bytes;
    {
        ProfScope ps(bf16 ? K_SPMM_BF16 : K_SPMM, s, 2.0 * nnz * k, bytes);
        const int32_t *bnd = bounds;
        if (!bnd) {
            hipLaunchKernelGGL(spmm_bounds_kernel, dim3((unsigned)((pl.waves + kWavesPerBlock) / kWavesPerBlock)),
                               dim3(256), 0, s, n_rows, indptr, pl.items, pl.ipw, pl.waves, bnd_ws);
            GCN_LAUNCH_CHECK("spmm_bounds_kernel");
            bnd = bnd_ws;
        }
        if (sliced) {
            const SliceMap m = make_slice_map(k, pl.waves, 4 * GCN_SPMM_LP);
            hipLaunchKernelGGL(spmm_sliced, dim3((unsigned)slice_map_blocks(m)), dim3(256), 0, s, n_rows, indptr,
                               indices, vals, (const float *)X, k, ldx, out, ldo, epi, bias, pl.items, pl.ipw,
                               pl.waves, m, bnd, carry, hr, tr, out16, ld16);
            GCN_LAUNCH_CHECK("spmm_sliced");
        } else if (sliced16) {
            const SliceMap m = make_slice_map(k, pl.waves, 8 * GCN_SPMM_BF16_LP);
            const dim3 g16((unsigned)slice_map_blocks(m));
            const uint16_t *X16 = (const uint16_t *)X;
            if (out16 && out)
                hipLaunchKernelGGL(spmm_sliced_bf16<2>, g16, dim3(256), 0, s, n_rows, indptr, indices, vals, X16, k,
                                   ldx, out, ldo, epi, bias, pl.items, pl.ipw, pl.waves, m, bnd, carry, hr, tr, out16,
                                   ld16);
            else if (out16)
                hipLaunchKernelGGL(spmm_sliced_bf16<1>, g16, dim3(256), 0, s, n_rows, indptr, indices, vals, X16, k,
                                   ldx, nullptr, ldo, epi, bias, pl.items, pl.ipw, pl.waves, m, bnd, carry, hr, tr,
                                   out16, ld16);
            else
                hipLaunchKernelGGL(spmm_sliced_bf16<0>, g16, dim3(256), 0, s, n_rows, indptr, indices, vals, X16, k,
                                   ldx, out, ldo, epi, bias, pl.items, pl.ipw, pl.waves, m, bnd, carry, hr, tr,
                                   nullptr, 0);
            GCN_LAUNCH_CHECK("spmm_sliced_bf16");
        } else
#define GCN_SPMM_CASE(V, C, B)                                                                   \
    if (vec == V && ct == C && bf16 == B) {                                                      \
        launch_main<V, C, B>(grid, s, n_rows, indptr, indices, vals, X, k, ldx, out, ldo, epi,   \
                             bias, pl, bnd, carry, hr, tr, out16, ld16);                         \
    } else
        GCN_SPMM_CASE(4, 1, false)
        GCN_SPMM_CASE(4, 2, false)
        GCN_SPMM_CASE(2, 1, false)
        GCN_SPMM_CASE(2, 2, false)
        GCN_SPMM_CASE(1, 1, false)
        GCN_SPMM_CASE(1, 2, false)
        GCN_SPMM_CASE(8, 1, true)
        GCN_SPMM_CASE(8, 2, true)
        GCN_SPMM_CASE(4, 1, true)
        GCN_SPMM_CASE(4, 2, true)
        GCN_SPMM_CASE(2, 1, true)
        GCN_SPMM_CASE(2, 2, true)
        GCN_SPMM_CASE(1, 1, true)
        GCN_SPMM_CASE(1, 2, true) {
            set_error("spmm: no kernel for vec=%d ct=%d", vec, ct);
            return GCN_EUNSUPPORTED;
        }
#undef GCN_SPMM_CASE
        GCN_LAUNCH_CHECK("spmm_main");
    }
    {
        ProfScope ps(K_SPMM_FIXUP, s, 0.0, 0.0);
        dim3 g2((unsigned)((pl.waves + kWavesPerBlock - 1) / kWavesPerBlock), (unsigned)((k + 255) / 256));
        hipLaunchKernelGGL(spmm_fixup, g2, dim3(256), 0, s, k, out, ldo, epi, bias, pl.waves, carry,
                           hr, tr, out16, ld16);
        GCN_LAUNCH_CHECK("spmm_fixup");
    }
    return GCN_OK;
}

}  // namespace

SpmmPlan spmm_plan(int32_t n_rows, int32_t nnz) {
    SpmmPlan p;
    p.items = (int64_t)n_rows + (int64_t)nnz;
    // aim for >= 8192 wavefronts (32 per CU) before growing the per-wave share
    int64_t ipw = (p.items + 8191) / 8192;
    ipw = (ipw + 31) / 32 * 32;
    if (ipw < 32) ipw = 32;
    if (ipw > kMaxIpw) ipw = kMaxIpw;
    p.ipw = (int)ipw;
    p.waves = (p.items + ipw - 1) / ipw;
    if (p.waves == 0) p.waves = 1;
    return p;
}

size_t spmm_workspace_bytes(int32_t n_rows, int32_t nnz, int32_t k) {
    if (n_rows <= 0 || k <= 0) return 0;
    const SpmmPlan pl = spmm_plan(n_rows, nnz);
    return align256((size_t)2 * pl.waves * k * sizeof(float)) + 2 * align256(pl.waves * sizeof(int32_t)) +
           align256((pl.waves + 1) * sizeof(int32_t)) + 256;
}

size_t spmm_bounds_bytes(int32_t n_rows, int32_t nnz) {
    if (n_rows <= 0) return 0;
    return align256((spmm_plan(n_rows, nnz).waves + 1) * sizeof(int32_t));
}

int spmm_bounds(int32_t n_rows, int32_t nnz, const int32_t *indptr, int32_t *bounds, hipStream_t s) {
    if (n_rows <= 0) return GCN_OK;
    const SpmmPlan pl = spmm_plan(n_rows, nnz);
    ProfScope ps(K_SPMM_FIXUP, s, 0.0, (double)(pl.waves + 1) * 4.0);
    hipLaunchKernelGGL(spmm_bounds_kernel, dim3((unsigned)((pl.waves + kWavesPerBlock) / kWavesPerBlock)),
                       dim3(256), 0, s, n_rows, indptr, pl.items, pl.ipw, pl.waves, bounds);
    GCN_LAUNCH_CHECK("spmm_bounds_kernel");
    return GCN_OK;
}

int spmm_f32(int32_t n_rows, int32_t nnz, const int32_t *indptr, IdxRef indices,
             const float *vals, const float *X, int32_t k, int64_t ldx, void *out, int64_t ldo,
             int epilogue, const float *bias, void *ws, size_t ws_bytes, hipStream_t s, const int32_t *bounds,
             uint16_t *out16, int64_t ld16) {
    return spmm_any(false, n_rows, nnz, indptr, indices, vals, X, k, ldx, out, ldo, epilogue, bias,
                    ws, ws_bytes, s, bounds, out16, ld16);
}

int spmm_bf16(int32_t n_rows, int32_t nnz, const int32_t *indptr, IdxRef indices,
              const float *vals, const uint16_t *X, int32_t k, int64_t ldx, void *out, int64_t ldo,
              int epilogue, const float *bias, void *ws, size_t ws_bytes, hipStream_t s, const int32_t *bounds,
              uint16_t *out16, int64_t ld16) {
    return spmm_any(true, n_rows, nnz, indptr, indices, vals, X, k, ldx, out, ldo, epilogue, bias,
                    ws, ws_bytes, s, bounds, out16, ld16);
}

}  // namespace gcn
