// Graph sampling and GCN construction on the sample (Sec. IV; Alg. 1-5):
//
//   frontier_kernel  frontier sampling with the Dashboard (Sec. IV-A/IV-B,
//                    Alg. 2-4); one wavefront per sampler instance, the 64
//                    lanes are the p processors of the probing step and of
//                    the Dashboard updates (intra-subgraph parallelism), one
//                    workgroup per sampler (inter-subgraph parallelism,
//                    Sec. IV-C)
//   induce kernels   the subgraph of G induced by each sampled vertex list, as
//                    a mean-normalised CSR with local ids, for a batch of
//                    samples at once (the last step of Alg. 2 / Alg. 3)
//   gather kernel    feature (or label) rows of the sampled vertices
//
// Dashboard layout (LDS, per sampler): db[entries] holds, for every entry, the
// Index-Array slot it belongs to (16 bits); slot k holds its vertex, the start
// of its neighbour list in G and its degree, with the live flag in bit 31.
// Popping a vertex clears one flag, which invalidates all of its entries at
// once (the paper's Alg. 4 writes INV into each of them), and reads no global
// memory; a step then costs two dependent global loads (the chosen neighbour,
// then its row bounds).  Random numbers: Philox4x64-10 (Salmon et al.,
// SC 2011) keyed by (seed, sampler id); each block gives four draws.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "common.h"
#include "gcn_sampler.h"

namespace gcn {
namespace {

constexpr size_t kSamplerMaxLds = 160 * 1024;  // LDS of one gfx950 CU

constexpr int kSampThreads = 64;          // one wavefront per sampler
constexpr uint32_t kLive = 0x80000000u;
constexpr uint64_t kKindRoot = 1, kKindProbe = 2, kKindNeigh = 3;
constexpr int64_t kProbeRoundLimit = 1 << 20;

// ---------------------------------------------------------------- Philox
// One Philox4x64-10 block: counter (c0, kind, c2, 0), key (seed, sampler id).
struct Words {
    uint64_t w0, w1, w2, w3;
    __device__ __forceinline__ uint64_t get(uint32_t i) const {
        return i == 0 ? w0 : (i == 1 ? w1 : (i == 2 ? w2 : w3));
    }
};
__device__ __forceinline__ Words philox(uint64_t c0, uint64_t kind, uint64_t c2, uint64_t seed, uint64_t sid) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = c0, x1 = kind, x2 = c2, x3 = 0, k0 = seed, k1 = sid;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t lo0 = M0 * x0, hi0 = __umul64hi(M0, x0);
        const uint64_t lo1 = M1 * x2, hi1 = __umul64hi(M1, x2);
        x0 = hi1 ^ x1 ^ k0;
        x1 = lo1;
        x2 = hi0 ^ x3 ^ k1;
        x3 = lo0;
        k0 += W0;
        k1 += W1;
    }
    return Words{x0, x1, x2, x3};
}
// integer uniform on [0, n): high word of r * n
__device__ __forceinline__ int64_t below(uint64_t r, int64_t n) { return (int64_t)__umul64hi(r, (uint64_t)n); }

__device__ __forceinline__ int32_t weight_of_deg(uint32_t d, int32_t cap) {
    return (cap > 0 && (int32_t)d > cap) ? cap : (int32_t)d;
}

// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int64_t wave_incl_scan(int64_t x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}

// ------------------------------------------------------- frontier sampling
struct SampArgs {
    int32_t nV;
    const int32_t *indptr;
    const int32_t *indices;
    int32_t m, n, db_cap, ia_cap, cap;
    uint64_t seed;
    int64_t first_sampler;
    int32_t *vertices;   // [S][n]
    int32_t *counts;     // [S]
    int32_t *status;     // [S]
};

// Index-Array slots in LDS: vertex, start of its neighbour list in G, and
// degree with the live flag (the slot keeps what a pop needs, so popping
// reads no global memory).
struct Slots {
    int32_t *v;
    int32_t *beg;
    uint32_t *deg;   // degree | kLive
};

// Cleanup (Alg. 4): keep the live slots in slot order, renumber them, and
// rebuild the Dashboard from their weights.  Whole wavefront.
__device__ void dashboard_cleanup(uint16_t *db, Slots sl, int32_t cap, int32_t &s, int64_t &used) {
    const int lane = threadIdx.x;
    int32_t ns = 0;
    for (int32_t base = 0; base < s; base += 64) {
        const int32_t k = base + lane;
        const bool in = k < s;
        const int32_t v = in ? sl.v[k] : 0;
        const int32_t b = in ? sl.beg[k] : 0;
        const uint32_t d = in ? sl.deg[k] : 0u;
        const bool live = in && (d & kLive);
        const uint64_t mask = __ballot(live);
        const int rank = __popcll(mask & ((1ull << lane) - 1ull));
        __syncthreads();            // every lane has read its slot before any moves
        if (live) {
            sl.v[ns + rank] = v;
            sl.beg[ns + rank] = b;
            sl.deg[ns + rank] = d;
        }
        ns += __popcll(mask);
        __syncthreads();
    }
    s = ns;
    int64_t off = 0;
    for (int32_t base = 0; base < ns; base += 64) {
        const int32_t k = base + lane;
        const int32_t w = k < ns ? weight_of_deg(sl.deg[k] & ~kLive, cap) : 0;
        const int64_t incl = wave_incl_scan(w);
        const int64_t start = off + incl - w;
        for (int32_t e = 0; e < w; ++e) db[start + e] = (uint16_t)k;
        off += __shfl(incl, 63, 64);
    }
    used = off;
    __syncthreads();
}

__global__ __launch_bounds__(kSampThreads) void frontier_kernel(SampArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    Slots sl;
    sl.v = (int32_t *)lds;                              // [ia_cap]
    sl.beg = sl.v + a.ia_cap;                           // [ia_cap]
    sl.deg = (uint32_t *)(sl.beg + a.ia_cap);           // [ia_cap]
    uint16_t *db = (uint16_t *)(sl.deg + a.ia_cap);     // Dashboard [db_cap]
    const int lane = threadIdx.x;
    const uint64_t sid = (uint64_t)(a.first_sampler + blockIdx.x);
    int32_t *out = a.vertices + (int64_t)blockIdx.x * a.n;
    int status = GCN_SAMPLE_OK;
    int32_t count = 0;

    // ---- roots: m distinct vertices; candidate t is kept unless it repeats an
    // earlier root (the lanes of a round take candidates t = 64 r + lane in order)
    {
        const uint64_t limit = 64ull * (uint64_t)a.m + 65536ull;
        int32_t got = 0;
        for (uint64_t base = 0; got < a.m; base += 64) {
            if (base >= limit) { status = GCN_SAMPLE_ROOT_LIMIT; break; }
            const uint64_t t = base + lane;
            const int32_t c = (int32_t)below(philox(t, kKindRoot, 0, a.seed, sid).w0, a.nV);
            bool dup = t >= limit;
            for (int32_t k = 0; k < got && !dup; ++k) dup = (sl.v[k] == c);
            for (int j = 0; j < 64; ++j) {
                const int32_t cj = __shfl(c, j, 64);
                if (j < lane && cj == c) dup = true;
            }
            const uint64_t mask = __ballot(!dup);
            const int rank = __popcll(mask & ((1ull << lane) - 1ull));
            if (!dup && got + rank < a.m) {
                sl.v[got + rank] = c;
                out[got + rank] = c;
            }
            got += min(__popcll(mask), a.m - got);
            __syncthreads();
        }
        count = got;
    }

    int64_t used = 0, live_weight = 0;
    int32_t s = 0;
    if (status == GCN_SAMPLE_OK) {
        // ---- Dashboard from the roots (Alg. 3, initialisation)
        for (int32_t base = 0; base < a.m; base += 64) {
            const int32_t k = base + lane;
            int32_t b = 0;
            uint32_t d = 0;
            if (k < a.m) {
                const int32_t v = sl.v[k];
                b = a.indptr[v];
                d = (uint32_t)(a.indptr[v + 1] - b);
            }
            const int32_t w = weight_of_deg(d, a.cap);
            const int64_t incl = wave_incl_scan(w);
            const int64_t total = __shfl(incl, 63, 64);
            if (used + total > a.db_cap) { status = GCN_SAMPLE_OVERFLOW; break; }
            const int64_t start = used + incl - w;
            if (k < a.m) {
                sl.beg[k] = b;
                sl.deg[k] = d | kLive;
                for (int32_t e = 0; e < w; ++e) db[start + e] = (uint16_t)k;
            }
            used += total;
        }
        live_weight = used;
        s = a.m;
        __syncthreads();
    }

    // ---- main loop: pop a frontier vertex, step to a neighbour, add it.
    // Random blocks are drawn ahead, while the step's global loads are in
    // flight: probe block r/4 of this lane, neighbour block t/4.
    uint64_t round = 0;
    int64_t pblk = -1, nblk = -1;
    Words pw{0, 0, 0, 0}, nw{0, 0, 0, 0};
    for (int32_t i = a.m; status == GCN_SAMPLE_OK && i < a.n; ++i) {
        if (live_weight == 0) { status = GCN_SAMPLE_EXHAUSTED; break; }
        const uint64_t t = (uint64_t)(i - a.m);
        if ((int64_t)(t >> 2) != nblk) {
            nw = philox(t >> 2, kKindNeigh, 0, a.seed, sid);
            nblk = (int64_t)(t >> 2);
        }
        const uint64_t rn = nw.get((uint32_t)(t & 3));
        int32_t k = -1;
        for (int64_t rr = 0;; ++rr) {
            if (rr >= kProbeRoundLimit) { status = GCN_SAMPLE_PROBE_LIMIT; break; }
            if ((int64_t)(round >> 2) != pblk) {
                pw = philox(round >> 2, kKindProbe, (uint64_t)lane, a.seed, sid);
                pblk = (int64_t)(round >> 2);
            }
            const int64_t idx = below(pw.get((uint32_t)(round & 3)), used);
            const int32_t slot = db[idx];
            const uint64_t mask = __ballot((sl.deg[slot] & kLive) != 0u);
            ++round;
            if (mask) {
                k = __shfl(slot, __ffsll((unsigned long long)mask) - 1, 64);
                break;
            }
        }
        if (status != GCN_SAMPLE_OK) break;
        const int32_t beg = sl.beg[k];
        const uint32_t deg = sl.deg[k] & ~kLive;    // >= 1: its weight was > 0
        __syncthreads();
        if (lane == 0) sl.deg[k] = deg;             // no longer in the frontier
        live_weight -= weight_of_deg(deg, a.cap);

        const int32_t v_new = a.indices[beg + below(rn, (int64_t)deg)];
        // draw ahead while the load is in flight
        if ((int64_t)((t + 1) >> 2) != nblk) {
            nw = philox((t + 1) >> 2, kKindNeigh, 0, a.seed, sid);
            nblk = (int64_t)((t + 1) >> 2);
        }
        if ((int64_t)(round >> 2) != pblk) {
            pw = philox(round >> 2, kKindProbe, (uint64_t)lane, a.seed, sid);
            pblk = (int64_t)(round >> 2);
        }
        if ((uint32_t)v_new >= (uint32_t)a.nV) { status = GCN_SAMPLE_BAD_GRAPH; break; }
        const int32_t b2 = a.indptr[v_new];
        const uint32_t d2 = (uint32_t)(a.indptr[v_new + 1] - b2);
        const int32_t w = weight_of_deg(d2, a.cap);

        __syncthreads();
        if (used + w > a.db_cap || s == a.ia_cap) dashboard_cleanup(db, sl, a.cap, s, used);
        if (used + w > a.db_cap) { status = GCN_SAMPLE_OVERFLOW; break; }
        for (int32_t e = lane; e < w; e += 64) db[used + e] = (uint16_t)s;
        if (lane == 0) {
            sl.v[s] = v_new;
            sl.beg[s] = b2;
            sl.deg[s] = d2 | kLive;
            out[i] = v_new;
        }
        used += w;
        live_weight += w;
        ++s;
        count = i + 1;
        __syncthreads();
    }
    if (lane == 0) {
        a.counts[blockIdx.x] = count;
        a.status[blockIdx.x] = status;
    }
}

// ------------------------------------------------------- induced subgraphs
constexpr int kTB = 256;
constexpr int kItems = 8;
constexpr int kTile = kTB * kItems;   // elements per scan tile

// exclusive scan of one value per thread over the block; returns the total
__device__ __forceinline__ int64_t block_excl_scan(int64_t x, int64_t &total) {
    __shared__ int64_t wsum[kTB / 64];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int64_t incl = wave_incl_scan(x);
    if (lane == 63) wsum[wid] = incl;
    __syncthreads();
    int64_t before = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kTB / 64; ++w) {
        if (w < wid) before += wsum[w];
        total += wsum[w];
    }
    __syncthreads();
    return before + incl - x;
}

__global__ __launch_bounds__(kTB) void fill_i32_kernel(int32_t *__restrict__ x, int64_t n, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < n; i += (int64_t)gridDim.x * kTB) x[i] = v;
}

// The sample sets are membership bitmaps, one bit per vertex of G per list:
// bits[s][v / 32] bit v % 32.  With wpre[s][k], the number of sampled
// vertices in words 0 .. k-1, the local id of a sampled vertex v (its rank
// among the list's distinct vertices in ascending order) is
// wpre[s][v / 32] + popcount of the bits of word v / 32 below v.  A list's
// bitmap and prefix take 8 bytes per 32 vertices of G, so the row kernels
// hold them in LDS and look each neighbour up there (the neighbour lists of
// G stream from memory coalesced; nothing else is read per neighbour).

// bits[s][v / 32] |= bit v % 32 for every sampled v of list s (duplicates collapse)
__global__ __launch_bounds__(kTB) void mark_kernel(int32_t nV, int32_t n, int32_t W,
                                                   const int32_t *__restrict__ vertices,
                                                   const int32_t *__restrict__ counts, uint32_t *__restrict__ bits) {
    const int s = blockIdx.y;
    const int32_t cnt = min(counts[s], n);
    for (int32_t i = blockIdx.x * kTB + threadIdx.x; i < cnt; i += gridDim.x * kTB) {
        const int32_t v = vertices[(int64_t)s * n + i];
        if ((uint32_t)v < (uint32_t)nV) atomicOr(&bits[(int64_t)s * W + (v >> 5)], 1u << (v & 31));
    }
}

// per (list, tile of kTile words): the number of set bits in the tile
__global__ __launch_bounds__(kTB) void popc_tile_sum_kernel(const uint32_t *__restrict__ bits, int32_t W,
                                                            int64_t *__restrict__ tsum, int32_t tiles) {
    const int s = blockIdx.y;
    const int64_t t0 = (int64_t)blockIdx.x * kTile;
    const uint32_t *bs = bits + (int64_t)s * W;
    int64_t acc = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t i = t0 + (int64_t)threadIdx.x * kItems + j;
        if (i < W) acc += __popc(bs[i]);
    }
    int64_t total;
    block_excl_scan(acc, total);
    if (threadIdx.x == 0) tsum[(int64_t)s * tiles + blockIdx.x] = total;
}

// per segment: exclusive scan of its tile sums (in place), segment total
__global__ __launch_bounds__(kTB) void seg_tile_scan_kernel(int64_t *__restrict__ tsum, int32_t tiles,
                                                            int64_t *__restrict__ seg_total) {
    const int s = blockIdx.x;
    int64_t *t = tsum + (int64_t)s * tiles;
    int64_t carry = 0;
    for (int32_t base = 0; base < tiles; base += kTB) {
        const int32_t i = base + threadIdx.x;
        const int64_t v = i < tiles ? t[i] : 0;
        int64_t total;
        const int64_t ex = block_excl_scan(v, total);
        if (i < tiles) t[i] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) seg_total[s] = carry;
}

// wpre[s][k] = sampled vertices in words 0 .. k-1;  vsub[s][local id] = v
__global__ __launch_bounds__(kTB) void rank_kernel(int32_t n, int32_t W, const uint32_t *__restrict__ bits,
                                                   const int64_t *__restrict__ toff, int32_t tiles,
                                                   int32_t *__restrict__ wpre, int32_t *__restrict__ vsub) {
    const int s = blockIdx.y;
    const int64_t t0 = (int64_t)blockIdx.x * kTile;
    const uint32_t *bs = bits + (int64_t)s * W;
    uint32_t words[kItems];
    int64_t acc = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t i = t0 + (int64_t)threadIdx.x * kItems + j;
        words[j] = i < W ? bs[i] : 0u;
        acc += __popc(words[j]);
    }
    int64_t total;
    int64_t r = toff[(int64_t)s * tiles + blockIdx.x] + block_excl_scan(acc, total);
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t i = t0 + (int64_t)threadIdx.x * kItems + j;
        if (i < W) wpre[(int64_t)s * W + i] = (int32_t)r;
        for (uint32_t b = words[j]; b; b &= b - 1u) {
            if (r < n) vsub[(int64_t)s * n + r] = (int32_t)(32 * i + __builtin_ctz(b));
            ++r;
        }
    }
}

// Row kernels: one block of kRowThreads takes rows [b R, (b+1) R) of list s
// (R = kRowsPerBlock), clipped to the list's distinct vertices; its
// wavefronts take the next row from an LDS counter (hub rows of G are
// hundreds of times longer than the median one).  TABLE_LDS: the list's
// bitmap (and prefix) copied into LDS first; otherwise read where they are.
constexpr int kRowThreads = 1024;
constexpr int kRowsPerBlock = 256;
constexpr size_t kInduceMaxLds = 128 * 1024;

__device__ __forceinline__ int32_t next_row(int32_t *ctr, int lane) {
    int32_t r = 0;
    if (lane == 0) r = atomicAdd(ctr, 1);
    return __shfl(r, 0);
}

// row length of every local row: neighbours of vsub[s][i] that are in the list
template <bool TABLE_LDS>
__global__ __launch_bounds__(kRowThreads) void row_count_kernel(int32_t nV, int32_t n, int32_t W,
                                                                const int32_t *__restrict__ indptr,
                                                                const int32_t *__restrict__ indices,
                                                                const uint32_t *__restrict__ bits,
                                                                const int64_t *__restrict__ n_sub,
                                                                const int32_t *__restrict__ vsub,
                                                                int32_t *__restrict__ rowlen) {
    extern __shared__ uint32_t tab[];
    __shared__ int32_t ctr;
    const int s = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int32_t r0 = blockIdx.x * kRowsPerBlock;
    const int32_t r1 = (int32_t)min<int64_t>((int64_t)r0 + kRowsPerBlock, min<int64_t>(n_sub[s], n));
    if (r0 >= r1) return;
    const uint32_t *bs = bits + (int64_t)s * W;
    if (TABLE_LDS) {
        for (int32_t k = threadIdx.x; k < W; k += kRowThreads) tab[k] = bs[k];
        bs = tab;
    }
    if (threadIdx.x == 0) ctr = r0;
    __syncthreads();
    for (int32_t i = next_row(&ctr, lane); i < r1; i = next_row(&ctr, lane)) {
        const int32_t u = vsub[(int64_t)s * n + i];
        const int32_t p1 = indptr[u + 1];
        int32_t cnt = 0;
        for (int32_t p = indptr[u] + lane; p < p1; p += 64) {
            const int32_t w = indices[p];
            cnt += ((uint32_t)w < (uint32_t)nV) ? (int32_t)((bs[w >> 5] >> (w & 31)) & 1u) : 0;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
        if (lane == 0) rowlen[(int64_t)s * n + i] = cnt;
    }
}

// per subgraph: indptr = exclusive scan of the row lengths (one block each);
// rows past the list's distinct vertices are empty
__global__ __launch_bounds__(kTB) void row_scan_kernel(int32_t n, const int32_t *__restrict__ rowlen,
                                                       const int64_t *__restrict__ n_sub,
                                                       int32_t *__restrict__ indptr_sub,
                                                       int64_t *__restrict__ nnz_sub) {
    const int s = blockIdx.x;
    const int32_t *rl = rowlen + (int64_t)s * n;
    int32_t *ip = indptr_sub + (int64_t)s * (n + 1);
    const int64_t ns = n_sub[s];
    int64_t carry = 0;
    for (int32_t base = 0; base < n; base += kTB) {
        const int32_t i = base + threadIdx.x;
        const int64_t v = i < ns ? rl[i] : 0;
        int64_t total;
        const int64_t ex = block_excl_scan(v, total);
        if (i < n) ip[i] = (int32_t)(carry + ex);
        carry += total;
    }
    if (threadIdx.x == 0) {
        ip[n] = (int32_t)carry;
        nnz_sub[s] = carry;
    }
}

// edge offsets of the subgraphs in the packed edge arrays; overflow flag
__global__ __launch_bounds__(kTB) void edge_offsets_kernel(int32_t S, const int64_t *__restrict__ nnz_sub,
                                                           int64_t *__restrict__ off, int64_t e_cap,
                                                           int32_t *__restrict__ status) {
    int64_t carry = 0;
    for (int32_t base = 0; base < S; base += kTB) {
        const int32_t i = base + threadIdx.x;
        const int64_t v = i < S ? nnz_sub[i] : 0;
        int64_t total;
        const int64_t ex = block_excl_scan(v, total);
        if (i < S) off[i] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) {
        off[S] = carry;
        *status = carry > e_cap ? 1 : 0;
    }
}

// local column ids and mean weights of every row, in neighbour order
template <bool TABLE_LDS>
__global__ __launch_bounds__(kRowThreads) void fill_rows_kernel(int32_t nV, int32_t n, int32_t W,
                                                                const int32_t *__restrict__ indptr,
                                                                const int32_t *__restrict__ indices,
                                                                const uint32_t *__restrict__ bits,
                                                                const int32_t *__restrict__ wpre,
                                                                const int64_t *__restrict__ n_sub,
                                                                const int32_t *__restrict__ vsub,
                                                                const int32_t *__restrict__ indptr_sub,
                                                                const int64_t *__restrict__ off,
                                                                const int32_t *__restrict__ status,
                                                                int32_t *__restrict__ sub_indices,
                                                                float *__restrict__ sub_vals,
                                                                float *__restrict__ sub_vals_t) {
    extern __shared__ uint32_t tab[];
    __shared__ int32_t ctr;
    const int s = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int32_t r0 = blockIdx.x * kRowsPerBlock;
    const int32_t r1 = (int32_t)min<int64_t>((int64_t)r0 + kRowsPerBlock, min<int64_t>(n_sub[s], n));
    if (*status != 0 || r0 >= r1) return;
    const uint32_t *bs = bits + (int64_t)s * W;
    const int32_t *ps = wpre + (int64_t)s * W;
    if (TABLE_LDS) {
        for (int32_t k = threadIdx.x; k < W; k += kRowThreads) {
            tab[k] = bs[k];
            tab[W + k] = (uint32_t)ps[k];
        }
        bs = tab;
        ps = (const int32_t *)(tab + W);
    }
    if (threadIdx.x == 0) ctr = r0;
    __syncthreads();
    const int32_t *ip = indptr_sub + (int64_t)s * (n + 1);
    for (int32_t i = next_row(&ctr, lane); i < r1; i = next_row(&ctr, lane)) {
        const int32_t u = vsub[(int64_t)s * n + i];
        const int32_t len = ip[i + 1] - ip[i];
        const float val = 1.0f / (float)len;
        int64_t pos = off[s] + ip[i];
        const int32_t p1 = indptr[u + 1];
        for (int32_t p0 = indptr[u]; p0 < p1; p0 += 64) {
            const int32_t p = p0 + lane;
            int32_t loc = -1;
            if (p < p1) {
                const int32_t w = indices[p];
                if ((uint32_t)w < (uint32_t)nV) {
                    const uint32_t word = bs[w >> 5], below = word & ((1u << (w & 31)) - 1u);
                    if ((word >> (w & 31)) & 1u) loc = ps[w >> 5] + __popc(below);
                }
            }
            const uint64_t mask = __ballot(loc >= 0);
            if (loc >= 0) {
                const int64_t q = pos + __popcll(mask & ((1ull << lane) - 1ull));
                sub_indices[q] = loc;
                sub_vals[q] = val;
                if (sub_vals_t) sub_vals_t[q] = 1.0f / (float)(ip[loc + 1] - ip[loc]);
            }
            pos += __popcll(mask);
        }
    }
}

__global__ __launch_bounds__(kTB) void copy_n_sub_kernel(int32_t S, const int64_t *__restrict__ a,
                                                         int32_t *__restrict__ b) {
    const int32_t i = blockIdx.x * kTB + threadIdx.x;
    if (i < S) b[i] = (int32_t)a[i];
}

// ------------------------------------------------------------------ gather
// out[i, :] = X[rows[i], :] for 4-byte elements; a row index outside
// [0, n_rows_X) gives a row of zeros.  VEC: 16-byte moves.
template <bool VEC>
__global__ __launch_bounds__(kTB) void gather_kernel(const uint32_t *__restrict__ X, int32_t n_rows_X,
                                                     int32_t width, int64_t ldx, const int32_t *__restrict__ rows,
                                                     int32_t count, uint32_t *__restrict__ out, int64_t ldo) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * (kTB / 64) + (threadIdx.x >> 6);
    if (i >= count) return;
    const int32_t r = rows[i];
    const bool ok = (uint32_t)r < (uint32_t)n_rows_X;
    const uint32_t *src = X + (int64_t)(ok ? r : 0) * ldx;
    uint32_t *dst = out + i * ldo;
    if (VEC) {
        for (int32_t c = lane * 4; c < width; c += 256) {
            uint4 v = ok ? *(const uint4 *)(src + c) : uint4{0, 0, 0, 0};
            *(uint4 *)(dst + c) = v;
        }
    } else {
        for (int32_t c = lane; c < width; c += 64) dst[c] = ok ? src[c] : 0u;
    }
}

int blocks_for(int64_t n, int per) { return (int)std::min<int64_t>((n + per - 1) / per, 65535); }

}  // namespace

size_t sampler_lds_bytes(int32_t db_cap, int32_t ia_cap) {
    return align256((size_t)ia_cap * 12 + (size_t)db_cap * 2);
}

int frontier_sample(const SampArgs &a, int32_t S, size_t lds, hipStream_t s) {
    static bool attr_set = false;
    if (!attr_set) {
        hipFuncSetAttribute((const void *)frontier_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            kSamplerMaxLds);
        attr_set = true;
    }
    frontier_kernel<<<S, kSampThreads, lds, s>>>(a);
    GCN_LAUNCH_CHECK("frontier_kernel");
    return GCN_OK;
}

}  // namespace gcn

using namespace gcn;

namespace {
struct InduceWs {
    uint32_t *bits;     // [S][W]: membership bitmap of each list (W = words of nV bits)
    int32_t *wpre;      // [S][W]: sampled vertices in the words before each word
    int64_t *tsum;      // [S][tiles]: tile sums, then their exclusive scan
    int64_t *n_sub64;   // [S]
    int64_t *nnz_sub;   // [S]
    int32_t *rowlen;    // [S][n]
};
InduceWs carve_induce(Arena &ar, int32_t nV, int32_t n, int32_t S) {
    InduceWs w;
    const int32_t W = (nV + 31) / 32;
    const int32_t tiles = (int32_t)((W + kTile - 1) / kTile);
    w.bits = ar.take<uint32_t>((size_t)S * W);
    w.wpre = ar.take<int32_t>((size_t)S * W);
    w.tsum = ar.take<int64_t>((size_t)S * tiles);
    w.n_sub64 = ar.take<int64_t>(S);
    w.nnz_sub = ar.take<int64_t>(S);
    w.rowlen = ar.take<int32_t>((size_t)S * n);
    return w;
}
}  // namespace

extern "C" {

int gcn_sampler_plan(int32_t n_vertices, const int32_t *indptr_host, int32_t m, int32_t n, double eta,
                     int32_t cap, uint64_t seed, gcn_sampler_params *out) {
    if (!indptr_host || !out || n_vertices <= 0 || m <= 0 || m > n_vertices || n < m || !(eta > 1.0) ||
        cap < 0) {
        set_error("gcn_sampler_plan: need indptr_host, out, 0 < m <= n_vertices, n >= m, eta > 1, cap >= 0");
        return GCN_EINVAL;
    }
    double sum_w = 0.0;
    int64_t wmax = 0;
    for (int32_t v = 0; v < n_vertices; ++v) {
        int64_t d = (int64_t)indptr_host[v + 1] - indptr_host[v];
        if (cap > 0 && d > cap) d = cap;
        sum_w += (double)d;
        wmax = std::max(wmax, d);
    }
    // Dashboard of eta * m * (mean entries per vertex) entries (Sec. IV-B), and
    // at least a frontier of m vertices of the largest weight (no overflow is
    // then possible); Index Array m + 512 slots.  Clamped to one CU's LDS;
    // at <= 80 KB two samplers share a CU.
    const int64_t ia = std::min<int64_t>((int64_t)m + 512, 65535);
    if (ia <= m || (size_t)ia * 12 + 2 > kSamplerMaxLds) {
        set_error("gcn_sampler_plan: a frontier of m = %d does not fit the %zu bytes of LDS", m,
                  (size_t)kSamplerMaxLds);
        return GCN_EUNSUPPORTED;
    }
    int64_t db = (int64_t)std::ceil(eta * (double)m * (sum_w / n_vertices));
    db = std::max<int64_t>(db, (int64_t)m * wmax);
    db = std::max<int64_t>(db, 1);
    db = std::min<int64_t>(db, ((int64_t)kSamplerMaxLds - ia * 12) / 2);
    out->m = m;
    out->n = n;
    out->db_entries = (int32_t)db;
    out->ia_slots = (int32_t)ia;
    out->cap = cap;
    out->seed = seed;
    return GCN_OK;
}

int gcn_frontier_sample(const gcn_csr *G, const gcn_sampler_params *p, int64_t first_sampler, int32_t S,
                        int32_t *vertices, int32_t *counts, int32_t *status, void *stream) {
    if (!G || !p || !vertices || !counts || !status || S < 0 || first_sampler < 0) {
        set_error("gcn_frontier_sample: null argument or negative count");
        return GCN_EINVAL;
    }
    if (G->n_rows != G->n_cols || G->n_rows <= 0 || !G->indptr || (G->nnz > 0 && !G->indices) || G->indices16) {
        set_error("gcn_frontier_sample: G must be a square CSR with at least one vertex and int32 indices");
        return GCN_ESHAPE;
    }
    if (p->m <= 0 || p->m > G->n_rows || p->n < p->m || p->ia_slots <= p->m || p->ia_slots > 65535 ||
        p->db_entries <= 0 || p->cap < 0) {
        set_error("gcn_frontier_sample: need 0 < m <= n_vertices, n >= m, m < ia_slots <= 65535, db_entries > 0");
        return GCN_EINVAL;
    }
    const size_t lds = sampler_lds_bytes(p->db_entries, p->ia_slots);
    int dev = 0, max_lds = 0;
    GCN_HIP_CHECK(hipGetDevice(&dev));
    GCN_HIP_CHECK(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
    const size_t limit = std::min<size_t>((size_t)max_lds, kSamplerMaxLds);
    if (lds > limit) {
        set_error("gcn_frontier_sample: Dashboard of %d entries and %d slots needs %zu bytes of LDS (limit %zu)",
                  p->db_entries, p->ia_slots, lds, limit);
        return GCN_EUNSUPPORTED;
    }
    if (S == 0) return GCN_OK;
    SampArgs a;
    a.nV = G->n_rows;
    a.indptr = G->indptr;
    a.indices = G->indices;
    a.m = p->m;
    a.n = p->n;
    a.db_cap = p->db_entries;
    a.ia_cap = p->ia_slots;
    a.cap = p->cap;
    a.seed = p->seed;
    a.first_sampler = first_sampler;
    a.vertices = vertices;
    a.counts = counts;
    a.status = status;
    hipStream_t s = (hipStream_t)stream;
    ProfScope prof(K_SAMPLE, s, 0.0, 0.0);
    return frontier_sample(a, S, lds, s);
}

size_t gcn_induce_workspace_bytes(int32_t n_vertices, int32_t n, int32_t S) {
    if (n_vertices <= 0 || n < 0 || S <= 0) return 256;
    Arena ar(nullptr, 0);
    carve_induce(ar, n_vertices, n, S);
    return ar.used;
}

int gcn_induce_subgraphs(const gcn_csr *G, int32_t S, int32_t n, const int32_t *vertices, const int32_t *counts,
                         int32_t *n_sub, int32_t *vsub, int32_t *indptr_sub, int64_t *edge_offsets,
                         int32_t *sub_indices, float *sub_vals, float *sub_vals_t, int64_t edge_capacity,
                         int32_t *status, void *ws, size_t ws_bytes, void *stream) {
    if (!G || !vertices || !counts || !n_sub || !vsub || !indptr_sub || !edge_offsets || !status || S < 0 ||
        n < 0 || edge_capacity < 0 || (edge_capacity > 0 && (!sub_indices || !sub_vals))) {
        set_error("gcn_induce_subgraphs: null argument or negative size");
        return GCN_EINVAL;
    }
    if (G->n_rows != G->n_cols || G->n_rows <= 0 || !G->indptr || (G->nnz > 0 && !G->indices) || G->indices16) {
        set_error("gcn_induce_subgraphs: G must be a square CSR with at least one vertex and int32 indices");
        return GCN_ESHAPE;
    }
    if (S == 0) return GCN_OK;
    const int32_t nV = G->n_rows;
    Arena ar(ws, ws_bytes);
    InduceWs w = carve_induce(ar, nV, n, S);
    if (!w.bits || !w.rowlen || ((uintptr_t)ws & 255u)) {
        set_error("gcn_induce_subgraphs: workspace of %zu bytes is too small or misaligned (need %zu)", ws_bytes,
                  gcn_induce_workspace_bytes(nV, n, S));
        return GCN_EWORKSPACE;
    }
    if (S > 65535) {
        set_error("gcn_induce_subgraphs: at most 65535 subgraphs per call");
        return GCN_EINVAL;
    }
    hipStream_t s = (hipStream_t)stream;
    ProfScope prof(K_INDUCE, s, 0.0, 0.0);
    const int32_t W = (nV + 31) / 32;
    const int32_t tiles = (W + kTile - 1) / kTile;
    const int64_t words = (int64_t)S * W;
    fill_i32_kernel<<<blocks_for(words, kTB * 8), kTB, 0, s>>>((int32_t *)w.bits, words, 0);
    if (n > 0) {
        mark_kernel<<<dim3(blocks_for(n, kTB), S), kTB, 0, s>>>(nV, n, W, vertices, counts, w.bits);
    }
    popc_tile_sum_kernel<<<dim3(tiles, S), kTB, 0, s>>>(w.bits, W, w.tsum, tiles);
    seg_tile_scan_kernel<<<S, kTB, 0, s>>>(w.tsum, tiles, w.n_sub64);
    rank_kernel<<<dim3(tiles, S), kTB, 0, s>>>(n, W, w.bits, w.tsum, tiles, w.wpre, vsub);
    copy_n_sub_kernel<<<blocks_for(S, kTB), kTB, 0, s>>>(S, w.n_sub64, n_sub);
    // the row kernels hold a list's bitmap (and prefix) in LDS when they fit
    const size_t count_lds = (size_t)W * 4, fill_lds = (size_t)W * 8;
    const bool lds = fill_lds <= kInduceMaxLds;
    static std::once_flag lds_attr;
    std::call_once(lds_attr, [] {
        hipFuncSetAttribute((const void *)row_count_kernel<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            kInduceMaxLds);
        hipFuncSetAttribute((const void *)fill_rows_kernel<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            kInduceMaxLds);
    });
    const dim3 rgrid((n + kRowsPerBlock - 1) / kRowsPerBlock, S);
    if (n > 0) {
        if (lds)
            row_count_kernel<true><<<rgrid, kRowThreads, count_lds, s>>>(nV, n, W, G->indptr, G->indices, w.bits,
                                                                        w.n_sub64, vsub, w.rowlen);
        else
            row_count_kernel<false><<<rgrid, kRowThreads, 0, s>>>(nV, n, W, G->indptr, G->indices, w.bits,
                                                                 w.n_sub64, vsub, w.rowlen);
    }
    row_scan_kernel<<<S, kTB, 0, s>>>(n, w.rowlen, w.n_sub64, indptr_sub, w.nnz_sub);
    edge_offsets_kernel<<<1, kTB, 0, s>>>(S, w.nnz_sub, edge_offsets, edge_capacity, status);
    if (n > 0) {
        if (lds)
            fill_rows_kernel<true><<<rgrid, kRowThreads, fill_lds, s>>>(
                nV, n, W, G->indptr, G->indices, w.bits, w.wpre, w.n_sub64, vsub, indptr_sub, edge_offsets, status,
                sub_indices, sub_vals, sub_vals_t);
        else
            fill_rows_kernel<false><<<rgrid, kRowThreads, 0, s>>>(
                nV, n, W, G->indptr, G->indices, w.bits, w.wpre, w.n_sub64, vsub, indptr_sub, edge_offsets, status,
                sub_indices, sub_vals, sub_vals_t);
    }
    GCN_LAUNCH_CHECK("induce kernels");
    return GCN_OK;
}

int gcn_gather_rows(const void *X, int32_t n_rows_X, int32_t width, int64_t ldx, const int32_t *rows,
                    int32_t count, void *out, int64_t ldo, void *stream) {
    if (count < 0 || width < 0 || n_rows_X < 0 || (count > 0 && (!X || !rows || !out))) {
        set_error("gcn_gather_rows: null argument or negative size");
        return GCN_EINVAL;
    }
    if (ldx < width || ldo < width) {
        set_error("gcn_gather_rows: leading dimensions must be >= width");
        return GCN_ESHAPE;
    }
    if (count == 0 || width == 0) return GCN_OK;
    hipStream_t s = (hipStream_t)stream;
    ProfScope prof(K_GATHER, s, 0.0, 2.0 * 4.0 * (double)count * width);
    const bool vec = width % 4 == 0 && ldx % 4 == 0 && ldo % 4 == 0 && ((uintptr_t)X & 15u) == 0 &&
                     ((uintptr_t)out & 15u) == 0;
    const int blocks = (int)(((int64_t)count + kTB / 64 - 1) / (kTB / 64));
    if (vec)
        gather_kernel<true><<<blocks, kTB, 0, s>>>((const uint32_t *)X, n_rows_X, width, ldx, rows, count,
                                                   (uint32_t *)out, ldo);
    else
        gather_kernel<false><<<blocks, kTB, 0, s>>>((const uint32_t *)X, n_rows_X, width, ldx, rows, count,
                                                    (uint32_t *)out, ldo);
    GCN_LAUNCH_CHECK("gather_kernel");
    return GCN_OK;
}

}  // extern "C"

extern "C" int gcn_csr_pattern_symmetric_host(int32_t n, const int32_t *indptr, const int32_t *indices) {
    if (n < 0 || !indptr || (indptr[n] > 0 && !indices)) {
        set_error("gcn_csr_pattern_symmetric_host: null pointer or negative size");
        return GCN_EINVAL;
    }
    for (int32_t i = 0; i < n; ++i) {
        for (int32_t p = indptr[i]; p < indptr[i + 1]; ++p) {
            const int32_t j = indices[p];
            if (j < 0 || j >= n || (p > indptr[i] && indices[p - 1] >= j)) {
                set_error("gcn_csr_pattern_symmetric_host: row %d is not strictly ascending within [0, n)", i);
                return GCN_EINVAL;
            }
        }
    }
    for (int32_t i = 0; i < n; ++i) {
        for (int32_t p = indptr[i]; p < indptr[i + 1]; ++p) {
            const int32_t j = indices[p];
            if (!std::binary_search(indices + indptr[j], indices + indptr[j + 1], i)) return 0;
        }
    }
    return 1;
}
