// Streaming kernels around the two training kernels: the ReLU derivative with
// the bias gradient, column sums, the PREDICT/LOSS rows of Alg. 1, and the
// float32 -> bfloat16 rounding.  All are HBM-bound; reductions run in a fixed
// order (per-chunk partial sums, then one pass over the chunks), so results
// are bitwise reproducible.
#include "common.h"

namespace gcn {
namespace {

// Column sums run in two fixed-order stages.  A block of kRowWaves
// wavefronts covers a chunk of rows: its lanes span 64 x VEC adjacent columns
// (coalesced rows), each wavefront adds every kRowWaves-th row of the chunk,
// and the wavefronts' sums are added in order into one partial row per chunk;
// a second pass adds the chunks' partial rows in order.
constexpr int kRowWaves = 4;

// Rows per chunk: enough chunks for about 2048 blocks, at least 16 rows, a
// multiple of kRowWaves.  `width` is the row width in floats.
__host__ __device__ inline int32_t chunk_rows(int32_t n, int32_t width) {
    const int64_t xblocks = ((int64_t)width + 255) / 256;
    int64_t r = ((int64_t)n * xblocks + 2047) / 2048;
    if (r < 16) r = 16;
    r = (r + kRowWaves - 1) / kRowWaves * kRowWaves;
    return (int32_t)(r > 0x40000000 ? 0x40000000 : r);
}

inline int32_t chunk_count(int32_t n, int32_t width) {
    const int32_t r = chunk_rows(n, width);
    return (int32_t)(((int64_t)n + r - 1) / r);
}


// Adds the block's kRowWaves per-wavefront sums in wavefront order and writes
// the chunk's partial row.  Every thread of the block must call it.
template <int VEC>
__device__ __forceinline__ void block_col_partial(const float (&sum)[VEC], int lane, int wv, int c, int width,
                                                  bool active, float *__restrict__ part_row) {
    __shared__ float red[kRowWaves - 1][64 * VEC];
    if (wv > 0) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) red[wv - 1][lane * VEC + v] = sum[v];
    }
    __syncthreads();
    if (wv == 0 && active) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            float t = sum[v];
#pragma unroll
            for (int k = 0; k < kRowWaves - 1; ++k) t += red[k][lane * VEC + v];
            if (c + v < width) part_row[c + v] = t;
        }
    }
}

// dZ = dY * [Y > thr] for a chunk of rows, VEC columns per lane.  Writes the two
// halves to their destinations and the chunk's column sums (the bias gradient).
template <int VEC>
__global__ __launch_bounds__(256) void relu_bwd_kernel(int32_t n, int32_t h, int32_t rpc,
                                                       const float *__restrict__ dY, int64_t lddy,
                                                       const float *__restrict__ Y, int64_t ldy,
                                                       float *__restrict__ outS, int64_t ldS,
                                                       float *__restrict__ outN, int64_t ldN,
                                                       uint16_t *__restrict__ outS16,
                                                       uint16_t *__restrict__ outN16,
                                                       float *__restrict__ part, float thr) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = (blockIdx.x * 64 + lane) * VEC;
    const int w = 2 * h;
    const bool active = c < w;
    const int chunk = blockIdx.y;
    const int r0 = chunk * rpc;
    const int r1 = min(r0 + rpc, n);
    const bool self = c < h;  // VEC divides h, so a vector never straddles
    float *dst = self ? outS : outN;
    uint16_t *dst16 = self ? outS16 : outN16;
    const int64_t ldd = self ? ldS : ldN;
    const int cc = self ? c : c - h;
    float sum[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) sum[v] = 0.0f;
    if (active) {
#pragma unroll 2
        for (int r = r0 + wv; r < r1; r += kRowWaves) {
            float g[VEC], y[VEC];
            if (VEC == 4) {
                const float4 a = *(const float4 *)(dY + (int64_t)r * lddy + c);
                const float4 b = *(const float4 *)(Y + (int64_t)r * ldy + c);
                g[0] = a.x; g[1] = a.y; g[2] = a.z; g[3] = a.w;
                y[0] = b.x; y[1] = b.y; y[2] = b.z; y[3] = b.w;
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    g[v] = dY[(int64_t)r * lddy + c + v];
                    y[v] = Y[(int64_t)r * ldy + c + v];
                }
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                g[v] = y[v] > thr ? g[v] : 0.0f;
                sum[v] += g[v];
            }
            if (dst) {
                float *o = dst + (int64_t)r * ldd + cc;
                if (VEC == 4) {
                    *(float4 *)o = make_float4(g[0], g[1], g[2], g[3]);
                } else {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) o[v] = g[v];
                }
            }
            if (dst16) {
                uint16_t *o16 = dst16 + (int64_t)r * ldd + cc;
                if (VEC == 4) {
                    const uint32_t lo = pack_bf16x2(g[0], g[1]);
                    const uint32_t hi = pack_bf16x2(g[2], g[3]);
                    *(uint2 *)o16 = make_uint2(lo, hi);
                } else {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) o16[v] = to_bf16(g[v]);
                }
            }
        }
    }
    block_col_partial<VEC>(sum, lane, wv, c, w, active, part + (int64_t)chunk * w);
}

// Column sums of a chunk of rows (generic matrix).
__global__ __launch_bounds__(256) void colsum_part_kernel(int32_t n, int32_t C, int32_t rpc,
                                                          const float *__restrict__ G, int64_t ldg,
                                                          float *__restrict__ part) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    const bool active = c < C;
    const int chunk = blockIdx.y;
    const int r0 = chunk * rpc;
    const int r1 = min(r0 + rpc, n);
    float sum[1] = {0.0f};
    if (active) {
#pragma unroll 4
        for (int r = r0 + wv; r < r1; r += kRowWaves) sum[0] += G[(int64_t)r * ldg + c];
    }
    block_col_partial<1>(sum, lane, wv, c, C, active, part + (int64_t)chunk * C);
}

// out[c] = sum over chunks of part[chunk][c]: one wavefront per column; lane
// l adds chunks l, l+64, ... in order, then a fixed xor-shuffle tree.
__global__ __launch_bounds__(256) void colsum_reduce_kernel(int32_t chunks, int32_t C,
                                                            const float *__restrict__ part,
                                                            float *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (c >= C) return;
    // a lane's chunks in order, eight loads in flight (the same sum as one
    // load at a time)
    float s = 0.0f;
    int k = lane;
    for (; k + 64 * 7 < chunks; k += 64 * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(k + 64 * u) * C + c];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; k < chunks; k += 64) s += part[(int64_t)k * C + c];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) out[c] = s;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// One wavefront per row of logits.  In place: X[i, :] <- dLoss/dX[i, :].
__global__ __launch_bounds__(256) void loss_rows_kernel(int kind, int32_t n, int32_t C, float *__restrict__ X,
                                                        const int32_t *__restrict__ labels,
                                                        const float *__restrict__ targets,
                                                        float *__restrict__ rowloss) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n) return;
    float *x = X + i * C;
    if (kind == GCN_SOFTMAX_CE) {
        float m = -INFINITY;
        for (int c = lane; c < C; c += 64) m = fmaxf(m, x[c]);
        m = wave_max(m);
        float s = 0.0f;
        for (int c = lane; c < C; c += 64) s += expf(x[c] - m);
        s = wave_sum(s);
        const float lse = m + logf(s);
        const int y = labels[i];
        const float inv_n = 1.0f / (float)n;
        float xy = 0.0f;
        for (int c = lane; c < C; c += 64) {
            const float v = x[c];
            if (c == y) xy = v;
            const float p = expf(v - lse);
            x[c] = (p - (c == y ? 1.0f : 0.0f)) * inv_n;
        }
        xy = wave_sum(xy);
        if (lane == 0) rowloss[i] = lse - xy;
    } else {
        const float *t = targets + i * C;
        const float inv = 1.0f / ((float)n * (float)C);
        float s = 0.0f;
        for (int c = lane; c < C; c += 64) {
            const float v = x[c];
            const float tv = t[c];
            const float e = expf(-fabsf(v));
            s += fmaxf(v, 0.0f) - v * tv + log1pf(e);
            const float sg = v >= 0.0f ? 1.0f / (1.0f + e) : e / (1.0f + e);
            x[c] = (sg - tv) * inv;
        }
        s = wave_sum(s);
        if (lane == 0) rowloss[i] = s;
    }
}

// The same for rows of at most R * V classes: R lanes per row, 256 / R rows
// per block, each lane holding the V logits of columns g, g + R, ... in
// registers (one read of the row), reductions over the R lanes by xor
// shuffles.  Beside G in place it writes, per block, the sum of its rows'
// losses (double, rows in order) and the column sums of its G rows (lpart,
// cpart: the head's loss and bias gradient finish in head_reduce_kernel).
// G16 (optional): the gradient rows also as bfloat16, Cp wide, columns
// C .. Cp-1 zero (the class-padded operand of the head's products).
template <int R, int V>
__global__ __launch_bounds__(256) void loss_group_kernel(int kind, int32_t n, int32_t C, float *__restrict__ X,
                                                         const int32_t *__restrict__ labels,
                                                         const float *__restrict__ targets,
                                                         double *__restrict__ lpart, float *__restrict__ cpart,
                                                         uint16_t *__restrict__ G16, int32_t Cp) {
    static_assert(R == 16 && V * R <= 128, "four row groups per wavefront, 128 columns at most");
    constexpr int RPB = 256 / R;   // rows per block
    __shared__ float sh_loss[RPB];
    __shared__ float sh_col[4][R * V];
    const int g = threadIdx.x % R;
    const int rg = threadIdx.x / R;           // row group of the block
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * RPB + rg;
    const bool live = i < n;                  // rows past n take part in the block sums as zeros
    float *x = X + i * C;
    auto gmax = [](float v) {
#pragma unroll
        for (int o = R / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, R));
        return v;
    };
    auto gsum = [](float v) {
#pragma unroll
        for (int o = R / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, R);
        return v;
    };
    float v[V], gr[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int c = g + R * k;
        v[k] = live && c < C ? x[c] : 0.0f;
    }
    float rl = 0.0f;
    if (kind == GCN_SOFTMAX_CE) {
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < V; ++k)
            if (g + R * k < C) m = fmaxf(m, v[k]);
        m = gmax(m);
        float sum = 0.0f;
#pragma unroll
        for (int k = 0; k < V; ++k)
            if (g + R * k < C) sum += expf(v[k] - m);
        sum = gsum(sum);
        const float lse = m + logf(sum);
        const int y = live ? labels[i] : -1;
        const float inv_n = 1.0f / (float)n;
        float xy = 0.0f;
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const int c = g + R * k;
            if (c == y) xy = v[k];
            gr[k] = live && c < C ? (expf(v[k] - lse) - (c == y ? 1.0f : 0.0f)) * inv_n : 0.0f;
        }
        xy = gsum(xy);
        rl = live ? lse - xy : 0.0f;
    } else {
        const float *t = targets + i * C;
        const float inv = 1.0f / ((float)n * (float)C);
        float sum = 0.0f;
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const int c = g + R * k;
            const bool ok = live && c < C;
            const float tv = ok ? t[c] : 0.0f;
            const float e = expf(-fabsf(v[k]));
            if (ok) sum += fmaxf(v[k], 0.0f) - v[k] * tv + log1pf(e);
            const float sg = v[k] >= 0.0f ? 1.0f / (1.0f + e) : e / (1.0f + e);
            gr[k] = ok ? (sg - tv) * inv : 0.0f;
        }
        rl = gsum(sum);
    }
    // G in place of the logits, or only its bfloat16 rows when those are
    // asked for (the bfloat16 head reads nothing else)
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int c = g + R * k;
        if (live && !G16 && c < C) x[c] = gr[k];
        if (live && G16 && c < Cp) G16[i * Cp + c] = c < C ? to_bf16(gr[k]) : (uint16_t)0;
    }
    // block sums: the four row groups of a wavefront share columns (lanes
    // g, g+16, g+32, g+48), then the four wavefronts in order
#pragma unroll
    for (int k = 0; k < V; ++k) {
        float c = gr[k] + __shfl_xor(gr[k], 16);
        c += __shfl_xor(c, 32);
        gr[k] = c;
    }
    if (lane < R)
#pragma unroll
        for (int k = 0; k < V; ++k) sh_col[wv][g + R * k] = gr[k];
    if (g == 0) sh_loss[rg] = rl;
    __syncthreads();
    if ((int)threadIdx.x < C)   // column-major: column c's block sums are contiguous
        cpart[(int64_t)threadIdx.x * gridDim.x + blockIdx.x] =
            ((sh_col[0][threadIdx.x] + sh_col[1][threadIdx.x]) + sh_col[2][threadIdx.x]) + sh_col[3][threadIdx.x];
    if (threadIdx.x == 0) {
        double t = 0.0;
#pragma unroll
        for (int r = 0; r < RPB; ++r) t += (double)sh_loss[r];
        lpart[blockIdx.x] = t;
    }
}

// The head's sums from the loss kernel's block partials, in fixed order:
// blocks 0 .. ceil(C/4)-1 one wavefront per column (db_pred[c] = sum over
// blocks b of cpart[c][b], read contiguously, four per lane per step), the
// last block the loss (scale x the sum of the blocks' double loss sums).
__global__ __launch_bounds__(256) void head_reduce_kernel(int32_t nb, int32_t C, const float *__restrict__ cpart,
                                                          const double *__restrict__ lpart, double scale,
                                                          float *__restrict__ loss, float *__restrict__ db) {
    const int cblocks = (C + 3) / 4;
    if ((int)blockIdx.x < cblocks) {
        const int lane = threadIdx.x & 63;
        const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
        if (c >= C) return;
        const float *col = cpart + (int64_t)c * nb;
        float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
        int b = lane;
        for (; b + 192 < nb; b += 256) {
            s0 += col[b];
            s1 += col[b + 64];
            s2 += col[b + 128];
            s3 += col[b + 192];
        }
        for (; b < nb; b += 64) s0 += col[b];
        float s = (s0 + s1) + (s2 + s3);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
        if (lane == 0) db[c] = s;
        return;
    }
    __shared__ double sh[256];
    double t = 0.0;
    for (int b = threadIdx.x; b < nb; b += 256) t += lpart[b];
    sh[threadIdx.x] = t;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = (float)(sh[0] * scale);
}

// loss = scale * sum_i rowloss[i] in fixed order.  Up to kLossOne rows: one
// block of 1024 threads writes the loss directly.  Beyond: blocks of kLossSeg
// rows reduce to one double each, then one block adds those.
constexpr int kLossSeg = 2048;
constexpr int kLossOne = 16384;

template <int T>
__global__ __launch_bounds__(T) void loss_partial_kernel(int32_t n, int64_t seg, const float *__restrict__ rowloss,
                                                         double *__restrict__ part, double scale,
                                                         float *__restrict__ loss) {
    __shared__ double sh[T];
    const int64_t base = (int64_t)blockIdx.x * seg;
    const int64_t end = min((int64_t)n, base + seg);
    double s = 0.0;
    for (int64_t i = base + threadIdx.x; i < end; i += T) s += (double)rowloss[i];
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int o = T / 2; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (loss) *loss = (float)(sh[0] * scale);
        else part[blockIdx.x] = sh[0];
    }
}

__global__ __launch_bounds__(256) void loss_reduce_kernel(int32_t nparts, const double *__restrict__ part,
                                                          double scale, float *__restrict__ loss) {
    __shared__ double sh[256];
    double s = 0.0;
    for (int i = threadIdx.x; i < nparts; i += 256) s += part[i];
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = (float)(sh[0] * scale);
}

// rows on gridDim.y (strided), columns four per thread
__global__ __launch_bounds__(256) void cvt_bf16_kernel(int64_t rows, int64_t cols, int64_t ycols,
                                                       const float *__restrict__ x, int64_t ldx,
                                                       uint16_t *__restrict__ y, int64_t ldy, int vec4) {
    const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (c >= ycols) return;
    for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
        const float *xr = x + r * ldx;
        uint16_t *yr = y + r * ldy;
        if (vec4 && c + 4 <= cols) {
            const float4 v = *(const float4 *)(xr + c);
            const uint32_t lo = pack_bf16x2(v.x, v.y);
            const uint32_t hi = pack_bf16x2(v.z, v.w);
            *(uint2 *)(yr + c) = make_uint2(lo, hi);
        } else {
            for (int64_t e = c; e < c + 4 && e < ycols; ++e) yr[e] = e < cols ? to_bf16(xr[e]) : 0;
        }
    }
}

// The 16-byte path: a row's 4-column groups over tpr lanes (a power of two
// covering the groups, up to 256) and 256 / tpr rows per block, rows strided
// over the grid, kCvtRows rows' loads in flight per thread.  Columns from
// `cols` to `ycols` are written as zeros.
constexpr int kCvtRows = 4;
__global__ __launch_bounds__(256) void cvt_bf16_vec_kernel(int64_t rows, int64_t cols, int64_t ycols, int tpr,
                                                           const float *__restrict__ x, int64_t ldx,
                                                           uint16_t *__restrict__ y, int64_t ldy) {
    const int64_t c = ((int64_t)blockIdx.x * tpr + (threadIdx.x % tpr)) * 4;
    if (c >= ycols) return;
    const int64_t rstep = (int64_t)gridDim.y * (256 / tpr);
    const bool full = c + 4 <= cols;
    for (int64_t r0 = (int64_t)blockIdx.y * (256 / tpr) + threadIdx.x / tpr; r0 < rows; r0 += rstep * kCvtRows) {
        float4 v[kCvtRows];
#pragma unroll
        for (int u = 0; u < kCvtRows; ++u) {
            const int64_t r = r0 + u * rstep;
            v[u] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (r < rows) {
                const float *xr = x + r * ldx + c;
                if (full) {
                    v[u] = *(const float4 *)xr;
                } else {
                    if (c < cols) v[u].x = xr[0];
                    if (c + 1 < cols) v[u].y = xr[1];
                    if (c + 2 < cols) v[u].z = xr[2];
                    if (c + 3 < cols) v[u].w = xr[3];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kCvtRows; ++u) {
            const int64_t r = r0 + u * rstep;
            if (r < rows) {
                uint16_t *yr = y + r * ldy + c;
                const uint32_t lo = pack_bf16x2(v[u].x, v[u].y), hi = pack_bf16x2(v[u].z, v[u].w);
                if (c + 4 <= ycols) {
                    *(uint2 *)yr = make_uint2(lo, hi);
                } else {
                    const uint16_t h[4] = {(uint16_t)lo, (uint16_t)(lo >> 16), (uint16_t)hi, (uint16_t)(hi >> 16)};
                    for (int e = 0; e < 4 && c + e < ycols; ++e) yr[e] = h[e];
                }
            }
        }
    }
}

// dst[c][r] = bf16(src[r][c]) through a 64 x 64 LDS tile.  Reads: each thread
// takes 4 consecutive source columns of a row; writes: each thread emits 4
// consecutive destination columns (8 bytes), so both sides stay coalesced.
template <typename TIn>
__global__ __launch_bounds__(256) void transpose_bf16_kernel(int64_t rows, int64_t cols, const TIn *__restrict__ src,
                                                             int64_t lds_, uint16_t *__restrict__ dst, int64_t ldd,
                                                             uint16_t *__restrict__ copy, int64_t ldc, int vec) {
    __shared__ uint16_t tile[64][64 + 4];
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const int tq = threadIdx.x & 15, tr = threadIdx.x >> 4;  // 16 quads x 16 rows
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = tr + 16 * i;
        const int64_t r = r0 + rr, c = c0 + tq * 4;
        uint16_t v[4] = {0, 0, 0, 0};
        if (r < rows) {
            if (vec && c + 4 <= cols) {
                if constexpr (sizeof(TIn) == 4) {
                    const float4 f = *(const float4 *)(src + r * lds_ + c);
                    v[0] = to_bf16(f.x); v[1] = to_bf16(f.y);
                    v[2] = to_bf16(f.z); v[3] = to_bf16(f.w);
                } else {
                    const uint2 u = *(const uint2 *)(src + r * lds_ + c);
                    v[0] = (uint16_t)(u.x & 0xFFFF); v[1] = (uint16_t)(u.x >> 16);
                    v[2] = (uint16_t)(u.y & 0xFFFF); v[3] = (uint16_t)(u.y >> 16);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (c + e < cols) {
                        if constexpr (sizeof(TIn) == 4) v[e] = to_bf16(src[r * lds_ + c + e]);
                        else v[e] = (uint16_t)src[r * lds_ + c + e];
                    }
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) tile[rr][tq * 4 + e] = v[e];
        if (copy && r < rows) {   // the untransposed bfloat16 copy, from the same registers
            uint16_t *o = copy + r * ldc + c;
            if (vec && c + 4 <= cols) {
                *(uint2 *)o = make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (c + e < cols) o[e] = v[e];
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int cc = tr + 16 * i;            // destination row = source column
        const int64_t c = c0 + cc, r = r0 + tq * 4;
        if (c >= cols) continue;
        uint16_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = tile[tq * 4 + e][cc];
        uint16_t *o = dst + c * ldd + r;
        if (vec && r + 4 <= rows) {
            *(uint2 *)o = make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (r + e < rows) o[e] = v[e];
        }
    }
}

__global__ __launch_bounds__(256) void fill_zero_f32_kernel(float *__restrict__ x, int64_t count) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) x[i] = 0.0f;
}

}  // namespace

int fill_zero(float *x, int64_t count, hipStream_t s) {
    if (count <= 0) return GCN_OK;
    int64_t g = (count + 255) / 256;
    if (g > 4096) g = 4096;
    hipLaunchKernelGGL(fill_zero_f32_kernel, dim3((unsigned)g), dim3(256), 0, s, x, count);
    GCN_LAUNCH_CHECK("fill_zero_f32_kernel");
    return GCN_OK;
}

size_t relu_bwd_workspace_bytes(int32_t n, int32_t h) {
    return align256((size_t)chunk_count(n, 2 * h) * 2 * h * sizeof(float)) + 256;
}

int relu_bwd(int32_t n, int32_t h, const float *dY, int64_t lddy, const float *Y, int64_t ldy,
             float *outS, int64_t ldS, float *outN, int64_t ldN, uint16_t *outS16, uint16_t *outN16,
             float *dbias, void *ws, size_t ws_bytes, hipStream_t s, float thr) {
    if (h <= 0) return GCN_OK;
    const int w = 2 * h;
    const int32_t rpc = chunk_rows(n, w);
    const int32_t chunks = chunk_count(n, w);
    Arena ar(ws, ws_bytes);
    float *part = ar.take<float>((size_t)chunks * w + 1);
    if (!part) {
        set_error("relu_bwd: workspace too small");
        return GCN_EWORKSPACE;
    }
    if (n > 0) {
        auto al = [](const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; };
        const bool v4 = h % 4 == 0 && lddy % 4 == 0 && ldy % 4 == 0 && ldS % 4 == 0 && ldN % 4 == 0 &&
                        al(dY, 16) && al(Y, 16) && al(outS, 16) && al(outN, 16) && al(outS16, 8) &&
                        al(outN16, 8);
        const double bytes = (double)n * w * 8.0 + (outS ? (double)n * w * 4.0 : 0.0) +
                             (outS16 ? (double)n * w * 2.0 : 0.0);
        ProfScope ps(K_RELU_MASK, s, 0.0, bytes);
        if (v4) {
            dim3 g((unsigned)((w / 4 + 63) / 64), (unsigned)chunks);
            hipLaunchKernelGGL(relu_bwd_kernel<4>, g, dim3(256), 0, s, n, h, rpc, dY, lddy, Y, ldy, outS, ldS,
                               outN, ldN, outS16, outN16, part, thr);
        } else {
            dim3 g((unsigned)((w + 63) / 64), (unsigned)chunks);
            hipLaunchKernelGGL(relu_bwd_kernel<1>, g, dim3(256), 0, s, n, h, rpc, dY, lddy, Y, ldy, outS, ldS,
                               outN, ldN, outS16, outN16, part, thr);
        }
        GCN_LAUNCH_CHECK("relu_bwd_kernel");
    }
    {
        ProfScope ps(K_COLSUM_REDUCE, s, 0.0, (double)chunks * w * 4.0);
        hipLaunchKernelGGL(colsum_reduce_kernel, dim3((unsigned)((w + 3) / 4)), dim3(256), 0, s, chunks, w,
                           part, dbias);
        GCN_LAUNCH_CHECK("colsum_reduce_kernel");
    }
    return GCN_OK;
}

size_t colsum_workspace_bytes(int32_t n, int32_t C) {
    return align256((size_t)chunk_count(n, C) * C * sizeof(float)) + 256;
}

int colsum(int32_t n, int32_t C, const float *G, int64_t ldg, float *out, void *ws, size_t ws_bytes,
           hipStream_t s) {
    if (C <= 0) return GCN_OK;
    const int32_t rpc = chunk_rows(n, C);
    const int32_t chunks = chunk_count(n, C);
    Arena ar(ws, ws_bytes);
    float *part = ar.take<float>((size_t)chunks * C + 1);
    if (!part) {
        set_error("colsum: workspace too small");
        return GCN_EWORKSPACE;
    }
    if (n > 0) {
        ProfScope ps(K_COLSUM_REDUCE, s, 0.0, (double)n * C * 4.0);
        hipLaunchKernelGGL(colsum_part_kernel, dim3((unsigned)((C + 63) / 64), (unsigned)chunks), dim3(256), 0,
                           s, n, C, rpc, G, ldg, part);
        GCN_LAUNCH_CHECK("colsum_part_kernel");
    }
    {
        ProfScope ps(K_COLSUM_REDUCE, s, 0.0, (double)chunks * C * 4.0);
        hipLaunchKernelGGL(colsum_reduce_kernel, dim3((unsigned)((C + 3) / 4)), dim3(256), 0, s, chunks, C,
                           part, out);
        GCN_LAUNCH_CHECK("colsum_reduce_kernel");
    }
    return GCN_OK;
}

int colsum_reduce_rows(int32_t rows, int32_t C, const float *part, float *out, hipStream_t s) {
    if (C <= 0) return GCN_OK;
    ProfScope ps(K_COLSUM_REDUCE, s, 0.0, (double)rows * C * 4.0);
    hipLaunchKernelGGL(colsum_reduce_kernel, dim3((unsigned)((C + 3) / 4)), dim3(256), 0, s, rows, C, part, out);
    GCN_LAUNCH_CHECK("colsum_reduce_kernel");
    return GCN_OK;
}

int loss_rows(int kind, int32_t n, int32_t C, float *X, const int32_t *labels, const float *targets,
              float *rowloss, hipStream_t s) {
    if (n <= 0) return GCN_OK;
    ProfScope ps(K_LOSS_ROWS, s, 0.0, (double)n * C * 4.0 * (kind == GCN_SIGMOID_BCE ? 3.0 : 2.0));
    hipLaunchKernelGGL(loss_rows_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s, kind, n, C, X, labels,
                       targets, rowloss);
    GCN_LAUNCH_CHECK("loss_rows_kernel");
    return GCN_OK;
}

namespace {
constexpr int kLossR = 16, kLossV = 8;
int32_t loss_blocks(int32_t n) { return (int32_t)(((int64_t)n * kLossR + 255) / 256); }
}  // namespace

// (the bfloat16 head pads the classes to a multiple of 32, which stays within 128)
bool loss_fused_ok(int32_t C) { return C >= 1 && C <= kLossR * kLossV; }

size_t loss_fused_workspace_bytes(int32_t n, int32_t C) {
    const size_t nb = (size_t)loss_blocks(n);
    return align256(nb * sizeof(double)) + align256(nb * (size_t)C * sizeof(float)) + 512;
}

int loss_fused(int kind, int32_t n, int32_t C, float *X, const int32_t *labels, const float *targets,
               double scale, float *loss, float *db, uint16_t *G16, int32_t Cp, void *ws, size_t ws_bytes,
               hipStream_t s) {
    if (n <= 0) return GCN_OK;
    const int32_t nb = loss_blocks(n);
    Arena ar(ws, ws_bytes);
    double *lpart = ar.take<double>(nb);
    float *cpart = ar.take<float>((size_t)nb * C);
    if (!lpart || !cpart || !loss_fused_ok(C)) {
        set_error("loss: workspace too small or classes > %d", kLossR * kLossV);
        return GCN_EWORKSPACE;
    }
    {
        ProfScope ps(K_LOSS_ROWS, s, 0.0,
                     (double)n * C * 4.0 * (kind == GCN_SIGMOID_BCE ? 3.0 : 2.0) + (G16 ? (double)n * Cp * 2.0 : 0.0));
        hipLaunchKernelGGL((loss_group_kernel<kLossR, kLossV>), dim3((unsigned)nb), dim3(256), 0, s, kind, n, C, X,
                           labels, targets, lpart, cpart, G16, Cp);
        GCN_LAUNCH_CHECK("loss_group_kernel");
    }
    ProfScope ps(K_LOSS_REDUCE, s, 0.0, (double)nb * (C * 4.0 + 8.0));
    hipLaunchKernelGGL(head_reduce_kernel, dim3((unsigned)((C + 3) / 4 + 1)), dim3(256), 0, s, nb, C, cpart, lpart,
                       scale, loss, db);
    GCN_LAUNCH_CHECK("head_reduce_kernel");
    return GCN_OK;
}

size_t loss_reduce_workspace_bytes(int32_t n) {
    return align256((size_t)((n + kLossSeg - 1) / kLossSeg + 1) * sizeof(double)) + 256;
}

int loss_reduce(int32_t n, const float *rowloss, double scale, float *loss, void *ws, size_t ws_bytes,
                hipStream_t s) {
    const int32_t nparts = (n + kLossSeg - 1) / kLossSeg;
    Arena ar(ws, ws_bytes);
    double *part = ar.take<double>((size_t)nparts + 1);
    if (!part) {
        set_error("loss_reduce: workspace too small");
        return GCN_EWORKSPACE;
    }
    ProfScope ps(K_LOSS_REDUCE, s, 0.0, (double)n * 4.0);
    if (n <= kLossOne) {
        hipLaunchKernelGGL(loss_partial_kernel<1024>, dim3(1), dim3(1024), 0, s, n, (int64_t)kLossOne, rowloss,
                           part, scale, loss);
    } else {
        hipLaunchKernelGGL(loss_partial_kernel<256>, dim3((unsigned)nparts), dim3(256), 0, s, n, (int64_t)kLossSeg,
                           rowloss, part, 0.0, (float *)nullptr);
        hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(256), 0, s, nparts, part, scale, loss);
    }
    GCN_LAUNCH_CHECK("loss_reduce_kernel");
    return GCN_OK;
}

int transpose_bf16_copy(int64_t rows, int64_t cols, const void *src, int src_is_bf16, int64_t lds_, uint16_t *dst,
                        int64_t ldd, uint16_t *copy, int64_t ldc, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return GCN_OK;
    ProfScope ps(K_TRANSPOSE_BF16, s, 0.0,
                 (double)rows * cols * ((src_is_bf16 ? 4.0 : 6.0) + (copy ? 2.0 : 0.0)));
    dim3 g((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64));
    const int esz = src_is_bf16 ? 2 : 4;
    const int vec = (lds_ % 4 == 0 && ldd % 4 == 0 && ((uintptr_t)src % (4 * esz)) == 0 && ((uintptr_t)dst % 8) == 0 &&
                     (!copy || (ldc % 4 == 0 && ((uintptr_t)copy % 8) == 0)))
                        ? 1 : 0;
    if (src_is_bf16)
        hipLaunchKernelGGL(transpose_bf16_kernel<uint16_t>, g, dim3(256), 0, s, rows, cols, (const uint16_t *)src,
                           lds_, dst, ldd, copy, ldc, vec);
    else
        hipLaunchKernelGGL(transpose_bf16_kernel<float>, g, dim3(256), 0, s, rows, cols, (const float *)src, lds_,
                           dst, ldd, copy, ldc, vec);
    GCN_LAUNCH_CHECK("transpose_bf16_kernel");
    return GCN_OK;
}

int transpose_bf16(int64_t rows, int64_t cols, const void *src, int src_is_bf16, int64_t lds_, uint16_t *dst,
                   int64_t ldd, hipStream_t s) {
    return transpose_bf16_copy(rows, cols, src, src_is_bf16, lds_, dst, ldd, nullptr, 0, s);
}

int cvt_bf16_pad(int64_t rows, int64_t cols, const float *x, int64_t ldx, uint16_t *y, int64_t ldy,
                 int64_t ycols, hipStream_t s) {
    if (rows <= 0 || ycols <= 0) return GCN_OK;
    const int vec4 = (ldx % 4 == 0 && ldy % 4 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)y & 7) == 0) ? 1 : 0;
    const int64_t gx = (ycols + 1023) / 1024;
    int64_t gy = rows < 65535 ? rows : 65535;
    if (gx * gy > 16384) gy = (16384 + gx - 1) / gx;
    ProfScope ps(K_CVT_BF16, s, 0.0, (double)rows * cols * 4.0 + (double)rows * ycols * 2.0);
    if (vec4) {
        const int64_t groups = (ycols + 3) / 4;
        int tpr = 1;
        while (tpr < groups && tpr < 256) tpr *= 2;
        const int64_t bx = (groups + tpr - 1) / tpr;
        const int64_t rpb = 256 / tpr;
        int64_t by = (rows + rpb * kCvtRows - 1) / (rpb * kCvtRows);
        if (by > 65535) by = 65535;
        if (bx * by > 8192) by = std::max<int64_t>(1, 8192 / bx);
        hipLaunchKernelGGL(cvt_bf16_vec_kernel, dim3((unsigned)bx, (unsigned)by), dim3(256), 0, s, rows, cols, ycols,
                           tpr, x, ldx, y, ldy);
        GCN_LAUNCH_CHECK("cvt_bf16_vec_kernel");
        return GCN_OK;
    }
    hipLaunchKernelGGL(cvt_bf16_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, s, rows, cols, ycols, x,
                       ldx, y, ldy, vec4);
    GCN_LAUNCH_CHECK("cvt_bf16_kernel");
    return GCN_OK;
}

// Several small float32 matrices (a step's weights) to bfloat16 in one
// launch: each job is a plain copy (columns cols .. dcols-1 of a row zero)
// or a transposed one (dst, cols x rows, = bf16(src)^T), in 32 x 32 tiles,
// the transposed ones through LDS so that reads and writes stay coalesced.
// Each block finds its job among the batch's block ranges.
namespace {
__global__ __launch_bounds__(256) void prep_bf16_kernel(Bf16PrepBatch b) {
    int j = 0;
    while (j + 1 < b.njobs && (int64_t)blockIdx.x >= b.job[j + 1].first_block) ++j;
    const Bf16PrepJob &J = b.job[j];
    const int64_t t = (int64_t)blockIdx.x - J.first_block;
    const int tr = (int)(t / J.tiles_c), tc = (int)(t % J.tiles_c);
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    if (J.transpose) {
        __shared__ float tile[32][33];
#pragma unroll
        for (int k = 0; k < 32; k += 8) {
            const int r = tr * 32 + ty + k, c = tc * 32 + tx;
            tile[ty + k][tx] = (r < J.rows && c < J.cols) ? J.src[(int64_t)r * J.lds + c] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 32; k += 8) {
            const int c = tc * 32 + ty + k, r = tr * 32 + tx;
            if (c < J.cols && r < J.rows) J.dst[(int64_t)c * J.ldd + r] = to_bf16(tile[tx][ty + k]);
        }
    } else {
#pragma unroll
        for (int k = 0; k < 32; k += 8) {
            const int r = tr * 32 + ty + k, c = tc * 32 + tx;
            if (r < J.rows && c < J.dcols)
                J.dst[(int64_t)r * J.ldd + c] = c < J.cols ? to_bf16(J.src[(int64_t)r * J.lds + c]) : (uint16_t)0;
        }
    }
}
}  // namespace

int prep_bf16(Bf16PrepBatch &b, hipStream_t s) {
    int64_t blocks = 0;
    double bytes = 0.0;
    for (int j = 0; j < b.njobs; ++j) {
        Bf16PrepJob &J = b.job[j];
        const int wc = J.transpose ? J.cols : J.dcols;
        J.tiles_c = (wc + 31) / 32;
        J.first_block = blocks;
        blocks += (int64_t)((J.rows + 31) / 32) * J.tiles_c;
        bytes += (double)J.rows * J.cols * 4.0 + (double)J.rows * wc * 2.0;
    }
    if (blocks == 0) return GCN_OK;
    ProfScope ps(K_CVT_BF16, s, 0.0, bytes);
    hipLaunchKernelGGL(prep_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, b);
    GCN_LAUNCH_CHECK("prep_bf16_kernel");
    return GCN_OK;
}

int cvt_bf16(int64_t rows, int64_t cols, const float *x, int64_t ldx, uint16_t *y, int64_t ldy,
             hipStream_t s) {
    return cvt_bf16_pad(rows, cols, x, ldx, y, ldy, cols, s);
}

}  // namespace gcn
