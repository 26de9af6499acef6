// CSR of A^T for the backward propagation.
//
// Row j of A^T lists the rows i of A that hold column j, in ascending i, with
// equal entries in their CSR order.  The CSR entries are already in row-major
// order, so A^T is exactly a *stable* sort of the entries by column.  This is
// done as an LSD radix sort of (key = column, value = entry position p) with
// 8-bit digits:
//   1. per-tile digit histograms (integer LDS atomics: counts do not depend on
//      the order of the increments);
//   2. one exclusive scan over (digit, tile) in digit-major order;
//   3. a stable scatter: each tile walks its keys in order, 256 at a time, and
//      ranks equal digits with wavefront ballots (lane order) and per-wavefront
//      counts (wavefront order), so every key lands at a position that only
//      depends on the input.
// Then t_indptr[j] = lower_bound(sorted keys, j), and each output entry looks
// up its source row (upper_bound of p in indptr, minus one) and copies vals[p]
// bit for bit.  The integer output is unique, hence bit-exact.
#include "common.h"

namespace gcn {
namespace {

constexpr int kTB = 256;            // threads per tile block
constexpr int kItems = 8;           // keys per thread per tile
constexpr int kTile = kTB * kItems; // keys per tile
constexpr int kRadix = 256;

__global__ __launch_bounds__(kTB) void iota_kernel(int32_t nnz, IdxRef indices,
                                                   uint32_t *__restrict__ keys, int32_t *__restrict__ vals) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < nnz; p += stride) {
        keys[p] = (uint32_t)indices[p];
        vals[p] = (int32_t)p;
    }
}

__global__ __launch_bounds__(kTB) void hist_kernel(int32_t nnz, const uint32_t *__restrict__ keys, int shift,
                                                   int32_t ntiles, int32_t *__restrict__ hist) {
    __shared__ int32_t cnt[kRadix];
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kTile;
    for (int it = 0; it < kItems; ++it) {
        const int64_t p = base + it * kTB + threadIdx.x;
        if (p < nnz) atomicAdd(&cnt[(keys[p] >> shift) & 0xFF], 1);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = cnt[threadIdx.x];
}

// Exclusive scan of `len` ints in three phases: per-segment sums, a scan of
// the segment sums (one block), and a per-segment scan plus its offset.
// Integer sums, so the result does not depend on the schedule.
constexpr int kScanPer = 16;                   // ints per thread
constexpr int kScanSeg = kTB * kScanPer;       // ints per block segment

__global__ __launch_bounds__(kTB) void scan_reduce_kernel(int64_t len, const int32_t *__restrict__ in,
                                                          int32_t *__restrict__ seg_sums) {
    __shared__ int32_t sh[kTB];
    const int64_t base = (int64_t)blockIdx.x * kScanSeg;
    int32_t s = 0;
    for (int i = 0; i < kScanPer; ++i) {
        const int64_t e = base + (int64_t)i * kTB + threadIdx.x;
        if (e < len) s += in[e];
    }
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int o = kTB / 2; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) seg_sums[blockIdx.x] = sh[0];
}

// exclusive scan of a short array by one block of 1024 threads
__global__ __launch_bounds__(1024) void scan_small_kernel(int64_t len, const int32_t *__restrict__ in,
                                                          int32_t *__restrict__ out) {
    __shared__ int32_t sh[1024];
    const int t = threadIdx.x;
    const int64_t per = (len + 1023) / 1024;
    const int64_t b = t * per;
    const int64_t e = b + per < len ? b + per : len;
    int32_t s = 0;
    for (int64_t i = b; i < e; ++i) s += in[i];
    sh[t] = s;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
        const int32_t v = t >= o ? sh[t - o] : 0;
        __syncthreads();
        sh[t] += v;
        __syncthreads();
    }
    int32_t run = sh[t] - s;
    for (int64_t i = b; i < e; ++i) {
        const int32_t v = in[i];
        out[i] = run;
        run += v;
    }
}

__global__ __launch_bounds__(kTB) void scan_down_kernel(int64_t len, const int32_t *__restrict__ in,
                                                        const int32_t *__restrict__ seg_offs,
                                                        int32_t *__restrict__ out) {
    __shared__ int32_t sh[kTB];
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kScanSeg + (int64_t)t * kScanPer;
    int32_t v[kScanPer];
    int32_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        v[i] = base + i < len ? in[base + i] : 0;
        s += v[i];
    }
    sh[t] = s;
    __syncthreads();
    for (int o = 1; o < kTB; o <<= 1) {
        const int32_t x = t >= o ? sh[t - o] : 0;
        __syncthreads();
        sh[t] += x;
        __syncthreads();
    }
    int32_t run = seg_offs[blockIdx.x] + sh[t] - s;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        if (base + i < len) out[base + i] = run;
        run += v[i];
    }
}

__global__ __launch_bounds__(kTB) void scatter_kernel(int32_t nnz, const uint32_t *__restrict__ keys_in,
                                                      const int32_t *__restrict__ vals_in, int shift,
                                                      int32_t ntiles, const int32_t *__restrict__ offs,
                                                      uint32_t *__restrict__ keys_out,
                                                      int32_t *__restrict__ vals_out) {
    __shared__ int32_t run[kRadix];          // keys of each digit placed so far by this tile
    __shared__ int32_t wcnt[kTB / 64][kRadix];
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    run[t] = offs[(int64_t)t * ntiles + blockIdx.x];
    const int64_t base = (int64_t)blockIdx.x * kTile;
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int it = 0; it < kItems; ++it) {
        for (int w = 0; w < kTB / 64; ++w) wcnt[w][t] = 0;
        __syncthreads();
        const int64_t p = base + it * kTB + t;
        const bool valid = p < nnz;
        uint32_t key = 0;
        int32_t val = 0;
        int digit = 0;
        if (valid) {
            key = keys_in[p];
            val = vals_in[p];
            digit = (key >> shift) & 0xFF;
        }
        // lanes of this wavefront holding the same digit
        unsigned long long match = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const unsigned long long bb = __ballot((digit >> bit) & 1);
            match &= ((digit >> bit) & 1) ? bb : ~bb;
        }
        const int wrank = __popcll(match & below);
        if (valid && wrank == 0) wcnt[wave][digit] = __popcll(match);
        __syncthreads();
        if (valid) {
            int pos = run[digit] + wrank;
            for (int w = 0; w < wave; ++w) pos += wcnt[w][digit];
            keys_out[pos] = key;
            vals_out[pos] = val;
        }
        __syncthreads();
        int32_t add = 0;
        for (int w = 0; w < kTB / 64; ++w) add += wcnt[w][t];
        run[t] += add;
        __syncthreads();
    }
}

// t_indptr[j] = number of sorted keys < j, for j in [0, n_cols]
__global__ __launch_bounds__(kTB) void bounds_kernel(int32_t n_cols, int32_t nnz,
                                                     const uint32_t *__restrict__ keys,
                                                     int32_t *__restrict__ t_indptr) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > n_cols) return;
    int64_t lo = 0, hi = nnz;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if ((int64_t)keys[mid] < j) lo = mid + 1; else hi = mid;
    }
    t_indptr[j] = (int32_t)lo;
}

// rowid[p] = the row of A that holds entry p (one wavefront per row)
__global__ __launch_bounds__(kTB) void rowid_kernel(int32_t n_rows, const int32_t *__restrict__ indptr,
                                                    int32_t *__restrict__ rowid) {
    const int64_t r = (int64_t)blockIdx.x * (kTB / 64) + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    const int32_t b = indptr[r], e = indptr[r + 1];
    for (int32_t p = b + (int32_t)(threadIdx.x & 63); p < e; p += 64) rowid[p] = (int32_t)r;
}

// t_indices[q] = row of entry perm[q] in A;  t_vals[q] = vals[perm[q]]
__global__ __launch_bounds__(kTB) void finalize_kernel(int32_t nnz, const int32_t *__restrict__ rowid,
                                                       const float *__restrict__ vals,
                                                       const int32_t *__restrict__ perm,
                                                       int32_t *__restrict__ t_indices,
                                                       float *__restrict__ t_vals) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nnz; q += stride) {
        const int32_t p = perm[q];
        t_indices[q] = rowid[p];
        t_vals[q] = vals[p];
    }
}

// Symmetric pattern: A^T has A's row pointers and indices; the value at
// (row j, column i) is A's value at (i, j).
// Pass 1: whether row i's values are all the same bits (true of every row
// of a mean aggregation matrix, Sec. II), in which case that value is
// A(i, j) for every j.  A wavefront takes four rows, 16 lanes each: a row of
// at most 64 entries is checked by its lane group with four loads per lane
// in flight; the longer rows of the wavefront are then checked one at a time
// by all 64 lanes with eight loads each in flight (a hub row of 14,000
// entries is one wavefront's walk).  Four rows per wavefront, not one: the
// pass is bound by the latency of its two dependent loads, and a quarter of
// the wavefronts cover it in fewer rounds.
__global__ __launch_bounds__(kTB) void sym_rows_kernel(int32_t n, const int32_t *__restrict__ indptr,
                                                       const float *__restrict__ vals,
                                                       uint32_t *__restrict__ rowval, int32_t *__restrict__ rowconst) {
    const int lane = threadIdx.x & 63;
    const int g = lane >> 4, gl = lane & 15;
    const int64_t i = ((int64_t)blockIdx.x * (kTB / 64) + (threadIdx.x >> 6)) * 4 + g;
    const bool live = i < n;
    int32_t b = 0, e = 0;
    if (live) {
        b = indptr[i];
        e = indptr[i + 1];
    }
    const bool shortrow = e - b <= 64;
    const uint32_t first = live && e > b ? __float_as_uint(vals[b]) : 0u;
    bool same = true;
    if (live && shortrow) {
        uint32_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int32_t p = b + gl + 16 * u;
            v[u] = p < e ? __float_as_uint(vals[p]) : first;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) same = same && (v[u] == first);
    }
    const uint64_t bad = __ballot(!same);
    bool row_same = ((bad >> (16 * g)) & 0xFFFFull) == 0;
    // the long rows, one at a time (the loop is uniform over the wavefront)
    uint64_t longs = __ballot(live && !shortrow && gl == 0);
    while (longs) {
        const int lg = (__ffsll((unsigned long long)longs) - 1) >> 4;
        longs &= longs - 1;
        const int32_t lb = __shfl(b, 16 * lg), le = __shfl(e, 16 * lg);
        const uint32_t lf = __shfl(first, 16 * lg);
        bool s2 = true;
        constexpr int U = 8;
        int32_t p = lb + lane;
        for (; p + 64 * (U - 1) < le; p += 64 * U) {
            uint32_t v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = __float_as_uint(vals[p + 64 * u]);
#pragma unroll
            for (int u = 0; u < U; ++u) s2 = s2 && (v[u] == lf);
        }
        for (; p < le; p += 64) s2 = s2 && (__float_as_uint(vals[p]) == lf);
        const bool all_same = __all(s2);
        if (g == lg) row_same = all_same;
    }
    if (live && gl == 0) {
        rowval[i] = first;
        rowconst[i] = row_same ? 1 : 0;
    }
}

// Pass 2, one thread per entry p (row j, column i): the constant value of row
// i, or else j (the row holding p, by a search of indptr) and a binary search
// for j in row i.  An index outside [0, n), or a missing (i, j) found by the
// search, gives NaN.
__global__ __launch_bounds__(kTB) void sym_vals_kernel(int32_t n, int32_t nnz, const int32_t *__restrict__ indptr,
                                                       IdxRef indices,
                                                       const float *__restrict__ vals,
                                                       const uint32_t *__restrict__ rowval,
                                                       const int32_t *__restrict__ rowconst,
                                                       float *__restrict__ t_vals) {
    const int64_t stride = (int64_t)gridDim.x * kTB;
    for (int64_t p = (int64_t)blockIdx.x * kTB + threadIdx.x; p < nnz; p += stride) {
        const int32_t i = indices[p];
        float t = __int_as_float(0x7FC00000);
        if ((uint32_t)i < (uint32_t)n) {
            if (rowconst[i]) {
                t = __uint_as_float(rowval[i]);
            } else {
                int32_t a = 0, b = n;   // the last row r with indptr[r] <= p
                while (a < b) {
                    const int32_t mid = a + ((b - a + 1) >> 1);
                    if (indptr[mid] <= p) a = mid; else b = mid - 1;
                }
                const int32_t j = a;
                int32_t lo = indptr[i], hi = indptr[i + 1];   // first index >= j in row i
                while (lo < hi) {
                    const int32_t mid = lo + ((hi - lo) >> 1);
                    if (indices[mid] < j) lo = mid + 1; else hi = mid;
                }
                if (lo < indptr[i + 1] && indices[lo] == j) t = vals[lo];
            }
        }
        t_vals[p] = t;
    }
}

__global__ void fill_zero_kernel(int32_t *__restrict__ x, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) x[i] = 0;
}

int key_bits(int32_t n_cols) {
    int b = 0;
    while (b < 31 && ((int64_t)1 << b) < (int64_t)n_cols) ++b;
    return b;  // keys are < n_cols <= 2^b
}

}  // namespace

size_t transpose_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz) {
    (void)n_rows;
    (void)n_cols;
    const int64_t ntiles = ((int64_t)nnz + kTile - 1) / kTile;
    size_t b = 0;
    b += 2 * align256((size_t)nnz * 4);          // keys ping-pong
    b += 2 * align256((size_t)nnz * 4);          // values ping-pong
    b += 2 * align256((size_t)ntiles * kRadix * 4);  // hist, offsets
    const int64_t segs = (ntiles * kRadix + kScanSeg - 1) / kScanSeg;
    b += 2 * align256((size_t)(segs + 1) * 4);        // segment sums, segment offsets
    return b + 256;
}

int csr_transpose(int32_t n_rows, int32_t n_cols, int32_t nnz, const int32_t *indptr, IdxRef indices,
                  const float *vals, int32_t *t_indptr, int32_t *t_indices, float *t_vals, void *ws,
                  size_t ws_bytes, hipStream_t s) {
    if (nnz == 0) {
        ProfScope ps(K_T_FINAL, s, 0.0, (double)(n_cols + 1) * 4.0);
        hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n_cols + 1 + 255) / 256)), dim3(256), 0, s,
                           t_indptr, (int64_t)n_cols + 1);
        GCN_LAUNCH_CHECK("fill_zero_kernel");
        return GCN_OK;
    }
    const int32_t ntiles = (int32_t)(((int64_t)nnz + kTile - 1) / kTile);
    Arena ar(ws, ws_bytes);
    uint32_t *ka = ar.take<uint32_t>(nnz), *kb = ar.take<uint32_t>(nnz);
    int32_t *va = ar.take<int32_t>(nnz), *vb = ar.take<int32_t>(nnz);
    int32_t *hist = ar.take<int32_t>((size_t)ntiles * kRadix);
    int32_t *offs = ar.take<int32_t>((size_t)ntiles * kRadix);
    const int64_t scan_len = (int64_t)ntiles * kRadix;
    const int64_t segs = (scan_len + kScanSeg - 1) / kScanSeg;
    int32_t *seg_sums = ar.take<int32_t>((size_t)segs + 1);
    int32_t *seg_offs = ar.take<int32_t>((size_t)segs + 1);
    if (!ka || !kb || !va || !vb || !hist || !offs || !seg_sums || !seg_offs) {
        set_error("csr_transpose: workspace too small (%zu < %zu bytes)", ws_bytes,
                  transpose_workspace_bytes(n_rows, n_cols, nnz));
        return GCN_EWORKSPACE;
    }
    unsigned g = (unsigned)((nnz + kTB - 1) / kTB);
    if (g > 16384) g = 16384;
    {
        ProfScope ps(K_T_COUNT, s, 0.0, (double)nnz * 12.0);
        hipLaunchKernelGGL(iota_kernel, dim3(g), dim3(kTB), 0, s, nnz, indices, ka, va);
        GCN_LAUNCH_CHECK("iota_kernel");
    }
    const int bits = key_bits(n_cols);
    for (int shift = 0; shift < bits || shift == 0; shift += 8) {
        {
            ProfScope ps(K_T_COUNT, s, 0.0, (double)nnz * 4.0);
            hipLaunchKernelGGL(hist_kernel, dim3(ntiles), dim3(kTB), 0, s, nnz, ka, shift, ntiles, hist);
            GCN_LAUNCH_CHECK("hist_kernel");
        }
        {
            ProfScope ps(K_T_SCAN, s, 0.0, (double)scan_len * 8.0);
            hipLaunchKernelGGL(scan_reduce_kernel, dim3((unsigned)segs), dim3(kTB), 0, s, scan_len, hist,
                               seg_sums);
            hipLaunchKernelGGL(scan_small_kernel, dim3(1), dim3(1024), 0, s, segs, seg_sums, seg_offs);
            hipLaunchKernelGGL(scan_down_kernel, dim3((unsigned)segs), dim3(kTB), 0, s, scan_len, hist, seg_offs,
                               offs);
            GCN_LAUNCH_CHECK("scan kernels");
        }
        {
            ProfScope ps(K_T_FILL, s, 0.0, (double)nnz * 16.0);
            hipLaunchKernelGGL(scatter_kernel, dim3(ntiles), dim3(kTB), 0, s, nnz, ka, va, shift, ntiles, offs,
                               kb, vb);
            GCN_LAUNCH_CHECK("scatter_kernel");
        }
        std::swap(ka, kb);
        std::swap(va, vb);
    }
    {
        ProfScope ps(K_T_FINAL, s, 0.0, (double)(n_cols + 1) * 4.0);
        hipLaunchKernelGGL(bounds_kernel, dim3((unsigned)((n_cols + 1 + kTB - 1) / kTB)), dim3(kTB), 0, s,
                           n_cols, nnz, ka, t_indptr);
        GCN_LAUNCH_CHECK("bounds_kernel");
    }
    {
        // the spare key buffer holds the row of every entry
        int32_t *rowid = (int32_t *)kb;
        ProfScope ps(K_T_FINAL, s, 0.0, (double)nnz * 20.0);
        hipLaunchKernelGGL(rowid_kernel, dim3((unsigned)((n_rows + kTB / 64 - 1) / (kTB / 64))), dim3(kTB), 0, s,
                           n_rows, indptr, rowid);
        hipLaunchKernelGGL(finalize_kernel, dim3(g), dim3(kTB), 0, s, nnz, rowid, vals, va, t_indices, t_vals);
        GCN_LAUNCH_CHECK("finalize_kernel");
    }
    return GCN_OK;
}

size_t transpose_symmetric_workspace_bytes(int32_t n, int32_t nnz) {
    (void)nnz;
    return 2 * align256((size_t)n * 4) + 256;
}

int csr_transpose_symmetric(int32_t n, int32_t nnz, const int32_t *indptr, IdxRef indices,
                            const float *vals, float *t_vals, void *ws, size_t ws_bytes, hipStream_t s) {
    if (n == 0 || nnz == 0) return GCN_OK;
    Arena ar(ws, ws_bytes);
    uint32_t *rowval = ar.take<uint32_t>(n);
    int32_t *rowconst = ar.take<int32_t>(n);
    if (!rowval || !rowconst) {
        set_error("csr_transpose_symmetric: workspace too small (%zu < %zu bytes)", ws_bytes,
                  transpose_symmetric_workspace_bytes(n, nnz));
        return GCN_EWORKSPACE;
    }
    ProfScope ps(K_T_SYM, s, 0.0, (double)nnz * 12.0 + (double)n * 16.0);
    hipLaunchKernelGGL(sym_rows_kernel, dim3((unsigned)((n + kTB / 16 - 1) / (kTB / 16))), dim3(kTB), 0, s, n,
                       indptr, vals, rowval, rowconst);
    unsigned g = (unsigned)std::min<int64_t>(((int64_t)nnz + kTB - 1) / kTB, 16384);
    hipLaunchKernelGGL(sym_vals_kernel, dim3(g), dim3(kTB), 0, s, n, nnz, indptr, indices, vals, rowval,
                       rowconst, t_vals);
    GCN_LAUNCH_CHECK("transpose_symmetric kernels");
    return GCN_OK;
}

// ------------------------------------------------------- content check
// The first violation in row order, as a 64-bit key for an integer atomicMin
// (the minimum is unique, so the result does not depend on timing):
//   endpoints:        key = which (0: indptr[0] != 0, 1: indptr[n_rows] != nnz)
//   row r decreasing: key = (r + 1) << 32
//   row r, entry q (q-th of the row) out of range / not ascending:
//                     key = (r + 1) << 32 | (1 + 2q + (not ascending))
namespace {
constexpr int64_t kValidKey = 0x7fffffffffffffffLL;

__global__ void validate_init_kernel(int64_t *key) { *key = kValidKey; }

__global__ __launch_bounds__(256) void validate_rows_kernel(int32_t n_rows, int32_t n_cols, int32_t nnz,
                                                            const int32_t *__restrict__ indptr,
                                                            IdxRef indices, int sorted,
                                                            int64_t *__restrict__ key) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r == 0 && lane == 0) {
        if (indptr[0] != 0) atomicMin((long long *)key, 0LL);
        if (indptr[n_rows] != nnz) atomicMin((long long *)key, 1LL);
    }
    if (r >= n_rows) return;
    const int32_t b = indptr[r], e = indptr[r + 1];
    const int64_t base = (r + 1) << 32;
    if (e < b) {
        if (lane == 0) atomicMin((long long *)key, (long long)base);
        return;
    }
    if (b < 0 || e > nnz) return;   // then an endpoint or a decrease is reported elsewhere
    // the row's first bad entry: lanes take entries b + lane, b + lane + 64, ...
    int64_t mine = kValidKey;
    for (int32_t p = b + lane; p < e; p += 64) {
        const int32_t j = indices[p];
        int bad = -1;
        if (j < 0 || j >= n_cols) bad = 0;
        else if (sorted && p > b && indices[p - 1] >= j) bad = 1;
        if (bad >= 0) {
            mine = base | (int64_t)(1 + 2 * (int64_t)(p - b) + bad);
            break;
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const int64_t other = __shfl_xor(mine, o);
        mine = other < mine ? other : mine;
    }
    if (lane == 0 && mine != kValidKey) atomicMin((long long *)key, (long long)mine);
}

// status[0] = code (0 valid, 1 endpoints, 2 indptr decreases, 3 index out of
// range, 4 not ascending), status[1] = row (0 or n_rows for endpoints)
__global__ void validate_final_kernel(int32_t n_rows, int64_t *key_status) {
    const int64_t key = *key_status;
    int32_t code = 0, row = 0;
    if (key != kValidKey) {
        const int64_t r = (key >> 32) - 1;
        const int64_t sub = key & 0xffffffffLL;
        if (r < 0) {
            code = 1;
            row = sub == 0 ? 0 : n_rows;
        } else {
            row = (int32_t)r;
            code = sub == 0 ? 2 : (((sub - 1) & 1) ? 4 : 3);
        }
    }
    int32_t *st = (int32_t *)key_status;
    st[0] = code;
    st[1] = row;
}
}  // namespace

int csr_validate_device(int32_t n_rows, int32_t n_cols, int32_t nnz, const int32_t *indptr,
                        IdxRef indices, int sorted, int32_t *status, hipStream_t s) {
    int64_t *key = (int64_t *)status;
    hipLaunchKernelGGL(validate_init_kernel, dim3(1), dim3(1), 0, s, key);
    GCN_LAUNCH_CHECK("validate_init_kernel");
    const int64_t blocks = ((int64_t)n_rows + 3) / 4;
    hipLaunchKernelGGL(validate_rows_kernel, dim3((unsigned)(blocks > 0 ? blocks : 1)), dim3(256), 0, s, n_rows,
                       n_cols, nnz, indptr, indices, sorted, key);
    GCN_LAUNCH_CHECK("validate_rows_kernel");
    hipLaunchKernelGGL(validate_final_kernel, dim3(1), dim3(1), 0, s, n_rows, key);
    GCN_LAUNCH_CHECK("validate_final_kernel");
    return GCN_OK;
}

}  // namespace gcn
