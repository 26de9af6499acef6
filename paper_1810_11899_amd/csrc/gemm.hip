// Weight application: dense products on the matrix cores (the second training
// kernel of Sec. V-A, which the paper runs with a BLAS dgemm).
//
// One kernel family covers every dense product of the layer:
//   NN  C = A B        forward:   H W_self, AGG W_neigh, H [W_self W_neigh], HL W_pred
//   TN  C = A^T B      weights:   H^T dZ_s, AGG^T dZ_n, HL^T G     (K = n, split-K)
//   NT  C = A B^T      inputs:    dZ_s W_self^T + G W_neigh^T, G W_pred^T
// Each problem may sum two K-segments with their own operands (the concat of
// the layer turns into a K-concat in the backward pass), and two problems of
// one layout share a launch.
//
// Tiles: 256 threads = 4 wavefronts in a 2 x 2 grid; block tile 128 x 128,
// wavefront tile 64 x 64 = 2 x 2 blocks of v_mfma_f32_32x32x2f32 (float32
// operands, float32 accumulate) or v_mfma_f32_32x32x16_bf16 (bfloat16
// operands).  K advances by BK per step through a double-buffered LDS tile
// stored k-major, so that the matrix-core operand reads (32 consecutive m or n
// per half-wavefront) hit 32 distinct banks.  Split-K partial tiles go to the
// workspace and a second kernel adds them in split order (no atomics).
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace gcn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int PAD = 4;
#ifndef GCN_GEMM_XK
#define GCN_GEMM_XK 1
#endif
#ifndef GCN_GEMM_XK_NN
#define GCN_GEMM_XK_NN 0
#endif
constexpr int PAD_XK = 4;   // [x][k] tiles: rows of BK + 4 floats (conflict-free 16-byte reads and stores)
constexpr int kThreads = 256;

struct Segs {
    const void *A[2];
    int64_t lda[2];
    const void *B[2];
    int64_t ldb[2];
    int32_t K[2];
    int32_t kt[2];  // k-tiles per segment
};

struct DevProblem {
    int32_t M, N;
    int32_t tiles_m, tiles_n;
    int32_t split;      // number of K splits
    int32_t kt_per_split;
    int32_t kt_total;
    int64_t block_begin;  // first flat block of this problem
    Segs s;
    float *C;
    int64_t ldc;
    const float *bias;
    int relu;
    float *partial;     // split x M x N when split > 1
    uint16_t *C16;      // bfloat16 rows of the output (ldc16), besides or instead of C
    int64_t ldc16;
    uint16_t *C16T;     // bfloat16 transposed output, columns < n16t (ldc16t),
    int64_t ldc16t;     // written by a pass after the product
    int32_t n16t;
    const float *mask;  // float32 kernel, no split: keep C where mask > 0 (leading dim ldm)
    const uint16_t *mask16;  // bfloat16 kernels: the same rule on bfloat16 bits
    int64_t ldm;
    float *colpart;     // float32, no split: per-row-tile column sums of C
};

struct DevArgs {
    DevProblem p[2];
    int nprob;
    int64_t total;     // logical blocks: splits x tiles_m x nprob x tiles_n
    int64_t per_xcd;   // ceil(total / 8)
};

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup b runs on
// XCD b % 8).  Logical blocks are numbered XCD-major, so that the column tiles
// of one row block, and the two problems of a grouped launch (which share
// their row operand in the forward pass), run on the same XCD and its L2
// serves the shared operand panel.  Order within an XCD: split, row tile,
// problem, column tile.  Grouped problems have equal M, N and K.
struct BlockCoord {
    int pi, split, tm, tn;
};
__device__ __forceinline__ bool decode_block(const DevArgs &a, BlockCoord &c) {
    const int64_t b = blockIdx.x;
    const int64_t L = (b & 7) * a.per_xcd + (b >> 3);
    if (L >= a.total) return false;
    const DevProblem &P = a.p[0];
    const int64_t row = (int64_t)a.nprob * P.tiles_n;   // logical blocks per row tile
    const int64_t per_split = (int64_t)P.tiles_m * row;
    c.split = (int)(L / per_split);
    int64_t r = L % per_split;
    c.tm = (int)(r / row);
    r %= row;
    c.pi = (int)(r / P.tiles_n);
    c.tn = (int)(r % P.tiles_n);
    return true;
}

// ------------------------------------------------------------------ loading
// Element type: float (fp32 path) or uint16_t (bf16 bits).
template <typename T> __device__ __forceinline__ T zero_elem() { return T(0); }

#ifndef GCN_GEMM_SWZ
#define GCN_GEMM_SWZ 1
#endif
// Column swizzle of the float32 operand tiles: row k of lds[k][x] holds
// element x at x ^ kswz(k).  The transposing store of an operand contiguous
// along k (four consecutive k of one x per thread, eight consecutive x per
// half-wavefront) then puts the half-wavefront's 32 values in 32 distinct
// banks: with rows 132 floats apart, k-groups 0/8 and 4/12 would otherwise
// share banks.  Reads of 32 consecutive x in one row stay conflict-free.
__device__ __forceinline__ int kswz(int k) { return GCN_GEMM_SWZ ? ((k >> 3) & 1) << 3 : 0; }

// Tile of one operand, BK x XT elements, kept k-major in LDS: lds[k][x].
//   KMAJOR: element (x, k) sits at ptr[k*ld + x]   (contiguous along x)
//   else  : element (x, k) sits at ptr[x*ld + k]   (contiguous along k)
template <typename T, int BK, bool KMAJOR, bool VEC, int XT = 128>
struct TileLoader {
    // 16-byte vectors of T
    static constexpr int E = 16 / sizeof(T);
    static constexpr int kElems = BK * XT;
    static constexpr int kVecs = kElems / E;
    static constexpr int kPer = kVecs / kThreads;  // vectors per thread
    static_assert(kPer >= 1, "tile too small");
    typedef typename std::conditional<sizeof(T) == 4, float4, uint4>::type V;
    V reg[kPer];

    __device__ __forceinline__ void coords(int i, int &x, int &k) const {
        const int v = threadIdx.x + i * kThreads;
        if (KMAJOR) {            // vectors along x
            constexpr int per_row = XT / E;
            k = v / per_row;
            x = (v % per_row) * E;
        } else {                 // vectors along k
            constexpr int per_row = BK / E;
            x = v / per_row;
            k = (v % per_row) * E;
        }
    }

    __device__ __forceinline__ void load(const T *__restrict__ ptr, int64_t ld, int x0, int xlim,
                                         int k0, int klim) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            const int gx = x0 + x, gk = k0 + k;
            if (VEC) {
                // xlim / klim are multiples of E on the vector path
                if (gx < xlim && gk < klim) {
                    const T *p = KMAJOR ? ptr + (int64_t)gk * ld + gx : ptr + (int64_t)gx * ld + gk;
                    reg[i] = *(const V *)p;
                } else {
                    reg[i] = V{};
                }
            } else {
                T tmp[E];
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const int ex = KMAJOR ? gx + e : gx;
                    const int ek = KMAJOR ? gk : gk + e;
                    tmp[e] = (ex < xlim && ek < klim)
                                 ? (KMAJOR ? ptr[(int64_t)ek * ld + ex] : ptr[(int64_t)ex * ld + ek])
                                 : zero_elem<T>();
                }
                reg[i] = *(V *)tmp;
            }
        }
    }

    // Fast path of the vector loader, for k-tiles wholly inside a K-segment:
    // per-thread element offsets of the vectors (at k = 0), computed once per
    // segment, with rows / column chunks past the extent clamped to the last
    // valid ones (their products land in outputs the epilogue drops).  A
    // k-tile is then one add and one load per vector, with no bounds branches.
    int64_t off[kPer];
    __device__ __forceinline__ void prepare(int64_t ld, int x0, int xlim) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            if (KMAJOR) off[i] = (int64_t)k * ld + min(x0 + x, xlim - E);
            else off[i] = (int64_t)min(x0 + x, xlim - 1) * ld + k;
        }
    }
    // kofs: k0 (operand contiguous along k) or k0 * ld (contiguous along x)
    __device__ __forceinline__ void load_fast(const T *__restrict__ ptr, int64_t kofs) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) reg[i] = *(const V *)(ptr + off[i] + kofs);
    }

    // [x][k] layout (k contiguous, rows of BK + PAD_XK): an operand contiguous
    // along k goes in as its loaded 16-byte vectors
    template <int RS>
    __device__ __forceinline__ void store_xk(T (*lds)[RS]) const {
        static_assert(!KMAJOR, "the [x][k] layout takes operands contiguous along k");
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            *(V *)&lds[x][k] = reg[i];
        }
    }

    __device__ __forceinline__ void store(T (*lds)[XT + PAD]) const {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            const T *t = (const T *)&reg[i];
            if (KMAJOR) {
                *(V *)&lds[k][sizeof(T) == 4 ? x ^ kswz(k) : x] = reg[i];
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) lds[k + e][sizeof(T) == 4 ? x ^ kswz(k + e) : x] = t[e];
            }
        }
    }
};

// -------------------------------------------------------------- main kernel
#ifndef GCN_GEMM_BK
#define GCN_GEMM_BK 16
#endif
constexpr int kBK = GCN_GEMM_BK;  // K depth of one LDS stage
#ifndef GCN_GEMM_TBM
#define GCN_GEMM_TBM 128
#endif
#ifndef GCN_GEMM_TBN
#define GCN_GEMM_TBN 128
#endif
constexpr int kTBM = GCN_GEMM_TBM;  // float32 block tile (M x N), 2 x 2 wavefronts
constexpr int kTBN = GCN_GEMM_TBN;

#ifndef GCN_GEMM_WAVES_PER_EU
#define GCN_GEMM_WAVES_PER_EU 4
#endif
// A wavefront issuing matrix-core products runs at raised priority, so that
// the SIMD's arbiter feeds the matrix pipe before the other wavefronts' loads.
#ifndef GCN_GEMM_SETPRIO
#define GCN_GEMM_SETPRIO 1
#endif
#if GCN_GEMM_SETPRIO
#define GCN_PRIO_UP() __builtin_amdgcn_s_setprio(1)
#define GCN_PRIO_DOWN() __builtin_amdgcn_s_setprio(0)
#else
#define GCN_PRIO_UP() ((void)0)
#define GCN_PRIO_DOWN() ((void)0)
#endif
template <int LAYOUT, bool VEC, int TBM, int TBN>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(GCN_GEMM_WAVES_PER_EU)))
void gemm_kernel(DevArgs args) {
    using T = float;
    constexpr int BK = kBK;
    constexpr bool A_KMAJOR = (LAYOUT == L_TN);
    constexpr bool B_KMAJOR = (LAYOUT != L_NT);
    constexpr int WTM = TBM / 2, WTN = TBN / 2;     // wavefront tile (2 x 2 wavefronts)
    constexpr int FM = WTM / 32, FN = WTN / 32;     // 32x32 accumulator blocks per wavefront
    // An operand contiguous along k (A in NN and NT, B in NT) is kept [x][k]
    // in LDS and read 4 consecutive k per lane: one ds_read_b128 feeds four
    // products.  A k-major operand keeps the [k][x] layout (one 4-byte read
    // per product), read in the same k order.
    constexpr bool XKA = GCN_GEMM_XK && !A_KMAJOR && (LAYOUT == L_NT || GCN_GEMM_XK_NN);
    constexpr bool XKB = GCN_GEMM_XK && !B_KMAJOR;
    constexpr bool XK = XKA || XKB;
    constexpr int RS = BK + PAD_XK;                 // [x][k] row stride
    constexpr int kSmemA = XKA ? 2 * TBM * RS : 2 * BK * (TBM + PAD);
    constexpr int kSmemB = XKB ? 2 * TBN * RS : 2 * BK * (TBN + PAD);
    // one LDS block: the two operand double buffers, reused by the epilogue
    __shared__ __attribute__((aligned(16))) T smem[kSmemA + kSmemB];
    T(*As)[BK][TBM + PAD] = (T(*)[BK][TBM + PAD])smem;
    T(*Bs)[BK][TBN + PAD] = (T(*)[BK][TBN + PAD])(smem + kSmemA);
    T(*Ax)[TBM][RS] = (T(*)[TBM][RS])smem;
    T(*Bx)[TBN][RS] = (T(*)[TBN][RS])(smem + kSmemA);

    // ---- which problem / split / tile
    BlockCoord bc;
    if (!decode_block(args, bc)) return;
    const DevProblem &P = args.p[bc.pi];
    const int split = bc.split;
    const int m0 = bc.tm * TBM, n0 = bc.tn * TBN;
    const int kt_begin = split * P.kt_per_split;
    int kt_end = kt_begin + P.kt_per_split;
    if (kt_end > P.kt_total) kt_end = P.kt_total;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    TileLoader<T, BK, A_KMAJOR, VEC, TBM> la;
    TileLoader<T, BK, B_KMAJOR, VEC, TBN> lb;

    // the two K-segments' descriptors, read once
    const T *const A0 = (const T *)P.s.A[0], *const A1 = (const T *)P.s.A[1];
    const T *const B0 = (const T *)P.s.B[0], *const B1 = (const T *)P.s.B[1];
    const int64_t lda0 = P.s.lda[0], lda1 = P.s.lda[1], ldb0 = P.s.ldb[0], ldb1 = P.s.ldb[1];
    const int K0 = P.s.K[0], K1 = P.s.K[1], kt0 = P.s.kt[0];
    const int Mp = P.M, Np = P.N;
    // the clamped fast loads need M (TN) and N (NN, TN) of at least one vector
    const bool fast = VEC && (!A_KMAJOR || Mp >= 4) && (!B_KMAJOR || Np >= 4);
    int ready = -1;   // the K-segment whose offsets are prepared
    auto load = [&](int kt) {
        const int sg = kt < kt0 ? 0 : 1;
        const int kk = (sg ? kt - kt0 : kt) * BK;
        const T *A = sg ? A1 : A0;
        const T *Bm = sg ? B1 : B0;
        const int64_t lda = sg ? lda1 : lda0, ldb = sg ? ldb1 : ldb0;
        const int K = sg ? K1 : K0;
        if (fast && kk + BK <= K) {
            if (ready != sg) {
                la.prepare(lda, m0, Mp);
                lb.prepare(ldb, n0, Np);
                ready = sg;
            }
            la.load_fast(A, A_KMAJOR ? (int64_t)kk * lda : (int64_t)kk);
            lb.load_fast(Bm, B_KMAJOR ? (int64_t)kk * ldb : (int64_t)kk);
        } else {
            la.load(A, lda, m0, Mp, kk, K);
            lb.load(Bm, ldb, n0, Np, kk, K);
        }
    };

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    if (kt_begin < kt_end) load(kt_begin);
    int buf = 0;
    const int kh = lane >> 5;
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      if constexpr (XK) {
        if constexpr (XKA) la.template store_xk<RS>(Ax[buf]);
        else la.store(As[buf]);
        if constexpr (XKB) lb.template store_xk<RS>(Bx[buf]);
        else lb.store(Bs[buf]);
        if (kt + 1 < kt_end) load(kt + 1);
        __syncthreads();
        // k order shared by both operands: in group g of 8 k, lanes 0-31 take
        // k = 8g + u and lanes 32-63 k = 8g + 4 + u for the u-th product
        float4 a4[FM], b4[FN];
        auto rd4 = [&](float4 *a, float4 *b, int g) {
            const int kc = 8 * g + 4 * (lane >> 5);
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int x = wm * WTM + i * 32 + (lane & 31);
                if constexpr (XKA) a[i] = *(const float4 *)&Ax[buf][x][kc];
                else
#pragma unroll
                    for (int u = 0; u < 4; ++u) a[i][u] = As[buf][kc + u][x ^ kswz(kc + u)];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int x = wn * WTN + j * 32 + (lane & 31);
                if constexpr (XKB) b[j] = *(const float4 *)&Bx[buf][x][kc];
                else
#pragma unroll
                    for (int u = 0; u < 4; ++u) b[j][u] = Bs[buf][kc + u][x ^ kswz(kc + u)];
            }
        };
        auto mma4 = [&](const float4 *a, const float4 *b) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][u], b[j][u], acc[i][j], 0, 0, 0);
        };
        static_assert(BK % 8 == 0, "whole groups of 8 k");
        // one group's fragments in flight (the other wavefronts on the SIMD
        // cover the read latency): 16 registers instead of 32
#pragma unroll
        for (int g = 0; g < BK / 8; ++g) {
            rd4(a4, b4, g);
            GCN_PRIO_UP();
            mma4(a4, b4);
            GCN_PRIO_DOWN();
        }
        buf ^= 1;
        continue;
      }
        la.store(As[buf]);
        lb.store(Bs[buf]);
        // the staging registers are free once stored: the next tile's loads
        // go out before the barrier, not after it (+3% over loading after it)
        if (kt + 1 < kt_end) load(kt + 1);
        __syncthreads();
        // two register sets of operands: the LDS reads of k-step s + 1 are
        // issued before the matrix-core products of k-step s
        float a0[FM], b0[FN], a1[FM], b1[FN];
        auto rd = [&](float *a, float *b, int kr) {
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = As[buf][kr][(wm * WTM + i * 32 + (lane & 31)) ^ kswz(kr)];
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = Bs[buf][kr][(wn * WTN + j * 32 + (lane & 31)) ^ kswz(kr)];
        };
        auto mma = [&](const float *a, const float *b) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
        };
        // (scheduling barriers keep each group of reads ahead of the products
        // that do not need it; without them the compiler sinks the reads
        // below the products and waits on them at once)
        rd(a0, b0, kh);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            rd(a1, b1, kk + 2 + kh);
            __builtin_amdgcn_sched_barrier(0);
            GCN_PRIO_UP();
            mma(a0, b0);
            GCN_PRIO_DOWN();
            __builtin_amdgcn_sched_barrier(0);
            if (kk + 4 < BK) rd(a0, b0, kk + 4 + kh);
            __builtin_amdgcn_sched_barrier(0);
            GCN_PRIO_UP();
            mma(a1, b1);
            GCN_PRIO_DOWN();
            __builtin_amdgcn_sched_barrier(0);
        }
        buf ^= 1;
    }

    const bool to_partial = P.split > 1;
    float *dst = to_partial ? P.partial + (int64_t)split * P.M * P.N : P.C;
    const int64_t ldd = to_partial ? P.N : P.ldc;
    // ---- epilogue through LDS, 32 rows per pass: the two wavefronts holding
    // those rows deposit their accumulator blocks row-major (row stride 136
    // floats: the two half-wavefronts' rows, four apart, land 32 banks apart),
    // then all four wavefronts write whole 128-column rows, 16 bytes per lane.
    static_assert(FM == 2 && FN == 2 && TBN == 128, "epilogue written for 2 x 2 blocks of a 128-wide tile");
    constexpr int SLD = 136;
    static_assert(32 * SLD <= kSmemA + kSmemB, "staging fits the operand buffers");
    float *stg = smem;
    const int ecol = n0 + 4 * (lane & 31);
    float ebv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (!to_partial && P.bias)
#pragma unroll
        for (int e = 0; e < 4; ++e) ebv[e] = ecol + e < P.N ? P.bias[ecol + e] : 0.0f;
    const bool erelu = !to_partial && P.relu;
    const bool evec = ldd % 4 == 0 && ((uintptr_t)dst & 15) == 0;
    // optional mask operand (a [mask > 0] factor on every stored value), read
    // for a pass's four rows before that pass's barrier; optional column sums
    // of the stored values over this thread's 16 rows of the tile
    const float *const emask = to_partial ? nullptr : P.mask;
    const bool mvec = emask && P.ldm % 4 == 0 && ((uintptr_t)emask & 15) == 0 && ecol + 3 < P.N;
    const bool ecs = !to_partial && P.colpart;
    float4 mk[4];
    float cs[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    auto put = [&](const floatx16 &v, int jb) {
        const int lc = wn * WTN + jb * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) stg[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * SLD + lc] = v[r];
    };
    __syncthreads();   // the last tile's operand reads are done
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        if (emask) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int row = m0 + 32 * h + wave * 8 + q * 2 + (lane >> 5);
                mk[q] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                if (row < P.M && ecol < P.N) {
                    const float *mp = emask + (int64_t)row * P.ldm + ecol;
                    if (mvec) {
                        mk[q] = *(const float4 *)mp;
                    } else {
                        mk[q].x = mp[0];
                        if (ecol + 1 < P.N) mk[q].y = mp[1];
                        if (ecol + 2 < P.N) mk[q].z = mp[2];
                        if (ecol + 3 < P.N) mk[q].w = mp[3];
                    }
                }
            }
        }
        if (wm == (h >> 1)) {
            put(acc[h & 1][0], 0);
            put(acc[h & 1][1], 1);
        }
        __syncthreads();
        // rows 32h .. 32h+31 of the tile; a wavefront writes two rows per store
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int lr = wave * 8 + q * 2 + (lane >> 5);
            const int row = m0 + 32 * h + lr;
            if (row < P.M && ecol < P.N) {
                const float4 x = *(const float4 *)&stg[lr * SLD + 4 * (lane & 31)];
                float o[4] = {x.x + ebv[0], x.y + ebv[1], x.z + ebv[2], x.w + ebv[3]};
                if (erelu)
#pragma unroll
                    for (int e = 0; e < 4; ++e) o[e] = fmaxf(o[e], 0.0f);
                if (emask) {
                    o[0] = mk[q].x > 0.0f ? o[0] : 0.0f;
                    o[1] = mk[q].y > 0.0f ? o[1] : 0.0f;
                    o[2] = mk[q].z > 0.0f ? o[2] : 0.0f;
                    o[3] = mk[q].w > 0.0f ? o[3] : 0.0f;
                }
                if (ecs)
#pragma unroll
                    for (int e = 0; e < 4; ++e) cs[e] += o[e];
                float *d = dst + (int64_t)row * ldd + ecol;
                if (evec && ecol + 3 < P.N) {
                    *(float4 *)d = make_float4(o[0], o[1], o[2], o[3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (ecol + e < P.N) d[e] = o[e];
                }
            }
        }
        __syncthreads();
    }
    if (ecs) {
        // the 8 row groups (wavefront, half) of each column, added in order
        const int grp = wave * 2 + (lane >> 5);
#pragma unroll
        for (int e = 0; e < 4; ++e) stg[grp * 128 + 4 * (lane & 31) + e] = cs[e];
        __syncthreads();
        if (threadIdx.x < 128) {
            float t = 0.0f;
#pragma unroll
            for (int g = 0; g < 8; ++g) t += stg[g * 128 + threadIdx.x];
            const int col = n0 + (int)threadIdx.x;
            if (col < P.N) P.colpart[(int64_t)bc.tm * P.N + col] = t;
        }
    }
}

// ------------------------------------------------------------ bf16 kernel
// bfloat16 operands, float32 accumulation on v_mfma_f32_32x32x16_bf16.  Both
// operand tiles sit in LDS as [row][k] with k contiguous (64-byte rows whose
// 16-byte chunks are XOR-swizzled by row), so a lane's eight consecutive k
// values are one ds_read_b128 and both the fragment reads and the tile stores
// are free of bank conflicts.  Operands that are contiguous along k in memory are copied as
// 16-byte vectors; operands contiguous along the row index are transposed on
// the way into LDS.
#ifndef GCN_BF16_BK
#define GCN_BF16_BK 32
#endif
#ifndef GCN_BF16_BIG
#define GCN_BF16_BIG 1
#endif
#ifndef GCN_BF16_TBM
#define GCN_BF16_TBM 128
#endif
#ifndef GCN_BF16_TBN
#define GCN_BF16_TBN 128
#endif
#ifndef GCN_BF16_WAVES_PER_EU
#define GCN_BF16_WAVES_PER_EU 4
#endif
constexpr int BK16 = GCN_BF16_BK;
constexpr int LDK16 = BK16;                 // no padding: chunks are XOR-swizzled
constexpr int kChunks16 = BK16 / 8;         // 16-byte chunks per row
constexpr int kRowsPerSpan16 = 256 / (BK16 * 2);  // rows that share the 64 banks once
static_assert(kRowsPerSpan16 >= 1 && (kChunks16 & (kChunks16 - 1)) == 0, "BK16 must be 32 or 64");
// Chunk c of row r is stored at chunk c ^ swz16(r): the 16 lanes that one LDS
// cycle serves (16 consecutive rows of a fragment read, or 4 rows x 4 chunks
// of a tile store) then fall in 16 distinct 4-bank groups.
__device__ __forceinline__ int swz16(int r) { return (r / kRowsPerSpan16) & (kChunks16 - 1); }
constexpr int kTBM16 = GCN_BF16_TBM;
constexpr int kTBN16 = GCN_BF16_TBN;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <bool KMAJOR, bool VEC, int XT>
struct TileLoader16 {
    static constexpr int kPer = (BK16 * XT / 8) / kThreads;  // 16-byte vectors per thread
    static_assert(kPer >= 1, "tile too small");
    uint4 reg[kPer];

    __device__ __forceinline__ void coords(int i, int &x, int &k) const {
        const int v = threadIdx.x + i * kThreads;
        if (KMAJOR) {   // vectors along x
            k = v / (XT / 8);
            x = (v % (XT / 8)) * 8;
        } else {        // vectors along k
            x = v / (BK16 / 8);
            k = (v % (BK16 / 8)) * 8;
        }
    }
    __device__ __forceinline__ void load(const uint16_t *__restrict__ ptr, int64_t ld, int x0, int xlim, int k0,
                                         int klim) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            const int gx = x0 + x, gk = k0 + k;
            if (VEC) {
                if (gx < xlim && gk < klim) {
                    const uint16_t *p = KMAJOR ? ptr + (int64_t)gk * ld + gx : ptr + (int64_t)gx * ld + gk;
                    reg[i] = *(const uint4 *)p;
                } else {
                    reg[i] = uint4{0u, 0u, 0u, 0u};
                }
            } else {
                uint16_t t[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int ex = KMAJOR ? gx + e : gx;
                    const int ek = KMAJOR ? gk : gk + e;
                    t[e] = (ex < xlim && ek < klim)
                               ? (KMAJOR ? ptr[(int64_t)ek * ld + ex] : ptr[(int64_t)ex * ld + ek])
                               : (uint16_t)0;
                }
                reg[i] = *(uint4 *)t;
            }
        }
    }
    __device__ __forceinline__ void store(uint16_t (*lds)[LDK16]) const {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            int x, k;
            coords(i, x, k);
            if (KMAJOR) {
                const uint16_t *t = (const uint16_t *)&reg[i];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    lds[x + e][((k >> 3) ^ swz16(x + e)) * 8 + (k & 7)] = t[e];
            } else {
                *(uint4 *)&lds[x][((k >> 3) ^ swz16(x)) * 8] = reg[i];
            }
        }
    }
};

// a bfloat16 value (raw bits) compares > 0 exactly when its float32 widening does
__device__ __forceinline__ bool bf16_bits_positive(uint32_t b) { return __uint_as_float(b << 16) > 0.0f; }

template <int LAYOUT, bool VEC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(GCN_BF16_WAVES_PER_EU)))
void gemm_bf16_kernel(DevArgs args) {
    constexpr bool A_KMAJOR = (LAYOUT == L_TN);
    constexpr bool B_KMAJOR = (LAYOUT != L_NT);
    constexpr int WTM = kTBM16 / 2, WTN = kTBN16 / 2;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    __shared__ __attribute__((aligned(16))) uint16_t As[2][kTBM16][LDK16];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kTBN16][LDK16];

    BlockCoord bc;
    if (!decode_block(args, bc)) return;
    const DevProblem &P = args.p[bc.pi];
    const int split = bc.split;
    const int m0 = bc.tm * kTBM16, n0 = bc.tn * kTBN16;
    const int kt_begin = split * P.kt_per_split;
    int kt_end = kt_begin + P.kt_per_split;
    if (kt_end > P.kt_total) kt_end = P.kt_total;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    TileLoader16<A_KMAJOR, VEC, kTBM16> la;
    TileLoader16<B_KMAJOR, VEC, kTBN16> lb;
    auto load = [&](int kt) {
        const int sg = kt < P.s.kt[0] ? 0 : 1;
        const int kk = (sg == 0 ? kt : kt - P.s.kt[0]) * BK16;
        la.load((const uint16_t *)P.s.A[sg], P.s.lda[sg], m0, P.M, kk, P.s.K[sg]);
        lb.load((const uint16_t *)P.s.B[sg], P.s.ldb[sg], n0, P.N, kk, P.s.K[sg]);
    };

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    if (kt_begin < kt_end) load(kt_begin);
    int buf = 0;
    const int koff = (lane >> 5) * 8;
    for (int kt = kt_begin; kt < kt_end; ++kt) {
        la.store(As[buf]);
        lb.store(Bs[buf]);
        if (kt + 1 < kt_end) load(kt + 1);   // staging registers free: load before the barrier
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK16; kk += 16) {
            bf16x8 a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = wm * WTM + i * 32 + (lane & 31);
                a[i] = *(const bf16x8 *)&As[buf][r][(((kk + koff) >> 3) ^ swz16(r)) * 8];
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = wn * WTN + j * 32 + (lane & 31);
                b[j] = *(const bf16x8 *)&Bs[buf][r][(((kk + koff) >> 3) ^ swz16(r)) * 8];
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        buf ^= 1;
    }

    const bool to_partial = P.split > 1;
    float *dst = to_partial ? P.partial + (int64_t)split * P.M * P.N : P.C;
    const int64_t ldd = to_partial ? P.N : P.ldc;
    // optional [mask > 0] factor (bfloat16 mask) and per-row-tile column
    // sums, as in the float32 kernel
    const uint16_t *const emask = to_partial ? nullptr : P.mask16;
    const bool ecs = !to_partial && P.colpart;
    float cs[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) cs[j] = 0.0f;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn * WTN + j * 32 + (lane & 31);
            if (col >= P.N) continue;
            const float bv = (!to_partial && P.bias) ? P.bias[col] : 0.0f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row < P.M) {
                    float v = acc[i][j][r];
                    if (!to_partial) {
                        v += bv;
                        if (P.relu) v = fmaxf(v, 0.0f);
                        if (emask) v = bf16_bits_positive(emask[(int64_t)row * P.ldm + col]) ? v : 0.0f;
                        if (ecs) cs[j] += v;
                        if (P.C16) P.C16[(int64_t)row * P.ldc16 + col] = to_bf16(v);
                        if (!P.C) continue;
                    }
                    dst[(int64_t)row * ldd + col] = v;
                }
            }
        }
    if (ecs) {
        // the 4 row groups (wavefront row, half) of each column, in order
        static_assert(kTBM16 == 128, "column-sum rows are 128-row tiles");
        float *red = (float *)&As[0][0][0];
        static_assert(4 * kTBN16 * sizeof(float) <= sizeof(As), "column sums fit the operand buffer");
        __syncthreads();   // operand reads done
        const int grp = wm * 2 + (lane >> 5);
#pragma unroll
        for (int j = 0; j < FN; ++j) red[grp * kTBN16 + wn * WTN + j * 32 + (lane & 31)] = cs[j];
        __syncthreads();
        if (threadIdx.x < kTBN16) {
            float t = 0.0f;
#pragma unroll
            for (int g = 0; g < 4; ++g) t += red[g * kTBN16 + threadIdx.x];
            const int col = n0 + (int)threadIdx.x;
            if (col < P.N) P.colpart[(int64_t)bc.tm * P.N + col] = t;
        }
    }
}

// C = sum over splits of the partial tiles, then the epilogue.  A block
// covers 256 / G output elements (float4 groups when VEC: N, ldc and the
// output 16-byte aligned) with G threads each: thread group g adds splits g,
// g + G, g + 2G, ... in increasing order, and the G group sums are added in
// group order.  The order is fixed, so results are bitwise reproducible; G > 1
// gives small outputs with many splits (weight gradients) enough threads.
template <bool VEC>
__global__ __launch_bounds__(256) void splitk_reduce(DevArgs args, int G) {
    using V = typename std::conditional<VEC, float4, float>::type;
    __shared__ V sh[256];
    const int pi = blockIdx.y;
    const DevProblem &P = args.p[pi];
    const int64_t total = (int64_t)P.M * P.N;
    const int W = VEC ? 4 : 1;
    const int nw = P.N / W;                     // vectors per row
    const int64_t count = (int64_t)P.M * nw;    // vectors in the output
    const int epb = 256 / G;
    const int el = threadIdx.x % epb, g = threadIdx.x / epb;
    const V *part = (const V *)P.partial;
    const int64_t pstride = total / W;          // one split's partials, in vectors
    for (int64_t base = (int64_t)blockIdx.x * epb; base < count; base += (int64_t)gridDim.x * epb) {
        const int64_t e = base + el;
        V acc{};
        if (e < count && g < P.split) {
            acc = part[(int64_t)g * pstride + e];
            for (int s = g + G; s < P.split; s += G) {
                const V v = part[(int64_t)s * pstride + e];
                if constexpr (VEC) {
                    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
                } else {
                    acc += v;
                }
            }
        }
        sh[threadIdx.x] = acc;
        __syncthreads();
        if (g == 0 && e < count) {
            for (int q = 1; q < G && q < P.split; ++q) {
                const V v = sh[q * epb + el];
                if constexpr (VEC) {
                    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
                } else {
                    acc += v;
                }
            }
            const int row = (int)(e / nw), col = (int)(e - (int64_t)row * nw) * W;
            float o[W];
            if constexpr (VEC) {
                o[0] = acc.x; o[1] = acc.y; o[2] = acc.z; o[3] = acc.w;
            } else {
                o[0] = acc;
            }
#pragma unroll
            for (int j = 0; j < W; ++j) {
                if (P.bias) o[j] += P.bias[col + j];
                if (P.relu) o[j] = fmaxf(o[j], 0.0f);
            }
            if (P.C16) {
                uint16_t *d = P.C16 + (int64_t)row * P.ldc16 + col;
#pragma unroll
                for (int j = 0; j < W; ++j) d[j] = to_bf16(o[j]);
            }
            if (!P.C) {
            } else if constexpr (VEC) {
                *(float4 *)(P.C + (int64_t)row * P.ldc + col) = float4{o[0], o[1], o[2], o[3]};
            } else {
                P.C[(int64_t)row * P.ldc + col] = o[0];
            }
        }
        __syncthreads();
    }
}

bool al(const void *p, int b) { return ((uintptr_t)p % (uintptr_t)b) == 0; }

// Vector loads need every contiguous extent, leading dimension and base
// pointer to be a multiple of the 16-byte vector.
// ---------------------------------------------------- bf16, large tiles
// The bf16 product of the layer (NT form, both operands contiguous along k):
// 256 x 256 block tiles, eight wavefronts each owning a 128 x 64 tile
// (4 x 2 v_mfma_f32_32x32x16_bf16 blocks), two wavefronts per SIMD, one block
// per CU.  Operand tiles of 256 rows x 32 k are copied from global
// memory straight into LDS (16-byte global_load_lds, no staging registers)
// through a ring of kBigStages stages, so the copies of the next two or three
// tiles are in flight while one is multiplied: a 128 x 128 x 32 tile of the
// smaller kernel is too short to cover the load latency with a single
// prefetch.  Rows are 64 bytes with their 16-byte
// chunks XOR-swizzled by row (conflict-free fragment reads); a lane's
// global address is chosen so that the chunk it deposits lands in its
// swizzled place.  Requires every K-segment to be a multiple of 32 and
// 16-byte aligned rows; rows past M or N are clamped to the last row and
// their results dropped.
#ifndef GCN_BIG_TN
#define GCN_BIG_TN 256
#endif
constexpr int kBigT = 256;       // block tile along M
constexpr int kBigTN = GCN_BIG_TN;   // block tile along N: 256, or 128 with 4 wavefronts (two blocks per CU)
constexpr int kBigBK = 32;       // k per stage
#ifndef GCN_BIG_STAGES
#define GCN_BIG_STAGES 4
#endif
constexpr int kBigStages = GCN_BIG_STAGES;   // 3..5 (5 x 32 KB is all of the CU's LDS)
#ifndef GCN_BIG_MASKED
#define GCN_BIG_MASKED 1
#endif
#ifndef GCN_BIG_MASK_PREFETCH
#define GCN_BIG_MASK_PREFETCH 8
#endif
#ifndef GCN_BIG_WAVES
#define GCN_BIG_WAVES 8
#endif
#ifndef GCN_BIG_NARROW_TILES
#define GCN_BIG_NARROW_TILES 256
#endif
#ifndef GCN_BIG_COPY_SPREAD
#define GCN_BIG_COPY_SPREAD 1
#endif
#ifndef GCN_BIG_READS_PER_MFMA
#define GCN_BIG_READS_PER_MFMA 3
#endif
constexpr int kBigWaves = GCN_BIG_WAVES;
                 // 4 (2 x 2) or 8 (2 x 4)
constexpr int kBigThreads = 64 * kBigWaves;
constexpr int kBigWN = kBigWaves / 2;                     // wavefronts along N
constexpr int kBigWTM = 128, kBigWTN = kBigTN / kBigWN;   // wavefront tile
constexpr int kBigFM = kBigWTM / 32, kBigFN = kBigWTN / 32;
// 1 KB (16 bytes per lane) loads per wavefront per stage, for A and for B
constexpr int kBigQA = kBigT * kBigBK / 8 / (64 * kBigWaves);
constexpr int kBigQB = kBigTN * kBigBK / 8 / (64 * kBigWaves);
static_assert(kBigQA * 64 * kBigWaves * 8 == kBigT * kBigBK && kBigQB * 64 * kBigWaves * 8 == kBigTN * kBigBK,
              "whole 16-byte chunks per lane");
constexpr int kBigStageA = kBigT * kBigBK, kBigStageB = kBigTN * kBigBK;   // elements per stage
__device__ __forceinline__ int bigswz(int r) { return (r >> 2) & 3; }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// scheduling groups: one matrix instruction, then PER LDS reads (the last
// group takes the remainder of TOT), for groups Q .. NG-1
template <int Q, int NG, int PER, int TOT>
__device__ __forceinline__ void sched_reads() {
    if constexpr (Q < NG) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, Q + 1 < NG ? PER : TOT - Q * PER, 0);
        sched_reads<Q + 1, NG, PER, TOT>();
    }
}
// the same, then one global-to-LDS copy behind each of the next NC matrix
// instructions (groups Q .. NM-1, one matrix instruction each)
template <int Q, int NM, int NG, int PER, int TOT, int NC>
__device__ __forceinline__ void sched_reads_copies() {
    if constexpr (Q < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (Q < NG) __builtin_amdgcn_sched_group_barrier(0x100, Q + 1 < NG ? PER : TOT - Q * PER, 0);
        else if constexpr (Q < NG + NC) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        sched_reads_copies<Q + 1, NM, NG, PER, TOT, NC>();
    }
}

// k-major operand tiles (an operand stored K x rows, contiguous along its
// rows: the K = n operands of the weight gradients, H and dZ, as the layer
// keeps them).  A stage holds 32 k-rows of 256 elements as 32 chunks of 16
// bytes; chunk position p of k-row kk holds the tile's chunk p ^ kmswz(kk).
// The matrix-core fragments (8 consecutive k of one row index per lane) are
// read with the gfx950 transposing LDS read: in each group of 16 lanes, lane
// j addresses 4 elements of k-row kbase + j/4 at row index x0 + 4 (j%4), and
// lane i receives element i%4 of the pieces of lanes i/4, i/4+4, i/4+8,
// i/4+12, i.e. x0 + i at k-rows kbase .. kbase+3.  With the swizzle the 16
// pieces of the 32 lanes of one LDS cycle fall in 16 distinct 4-bank groups.
__device__ __forceinline__ int kmswz(int kk) { return 4 * (kk & 3); }
typedef short v4i16 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8 tr_frag(const uint16_t *tile, int off0, int off1) {
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(tile + off0));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(tile + off1));
    bf16x8 r;
    __builtin_memcpy(&r, &lo, 8);
    __builtin_memcpy((char *)&r + 8, &hi, 8);
    return r;
}

// Output sets of the large-tile kernel, one instantiation each so that the
// hot ones carry no code (and no registers) for outputs they never write.
enum BigOut {
    BIG_F32 = 0,   // float32 C (or split partials) only
    BIG_B16 = 1,   // bfloat16 rows C16 only
    BIG_ALL = 2    // float32 C and bfloat16 rows C16
};
// LAYOUT: L_NT (both operands contiguous along k), L_TN (both k-major) or
// L_NN (A contiguous along k, B k-major).
template <int OUT, int LAYOUT>
__global__ __launch_bounds__(kBigThreads) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_bf16_big_kernel(DevArgs args) {
    constexpr bool KMA = LAYOUT == L_TN, KMB = LAYOUT != L_NT;
    __shared__ __attribute__((aligned(16))) uint16_t lds[kBigStages][kBigStageA + kBigStageB];

    BlockCoord bc;
    if (!decode_block(args, bc)) return;
    const DevProblem &P = args.p[bc.pi];
    const int m0 = bc.tm * kBigT, n0 = bc.tn * kBigTN;
    const int kt_begin = bc.split * P.kt_per_split;
    const int kt_end = min(kt_begin + P.kt_per_split, P.kt_total);
    const int ntiles = kt_end - kt_begin;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / kBigWN, wn = wave % kBigWN;

    const uint16_t *const A0 = (const uint16_t *)P.s.A[0], *const A1 = (const uint16_t *)P.s.A[1];
    const uint16_t *const B0 = (const uint16_t *)P.s.B[0], *const B1 = (const uint16_t *)P.s.B[1];
    const int64_t lda0 = P.s.lda[0], lda1 = P.s.lda[1], ldb0 = P.s.ldb[0], ldb1 = P.s.ldb[1];
    const int kt0 = P.s.kt[0];
    const int Mlast = P.M - 1, Nlast = P.N - 1;

    // Lane `lane` of load q deposits chunk position (wave*Q + q)*64 + lane of
    // the stage's operand tile: row pos/4, stored chunk pos%4, which holds
    // global chunk (pos%4) ^ swizzle(row).
    // A k-major operand: k-row pos/32, stored chunk pos%32, which holds the
    // tile's chunk (pos%32) ^ kmswz(k-row), at row index x0 + 8 * chunk
    // (clamped to the last whole chunk, rows are a multiple of 8).
    // (B's k-rows hold kBigTN / 8 chunks)
    int rowA[kBigQA], rowB[kBigQB], chkA[kBigQA], chkB[kBigQB], kmA[kBigQA], kmB[kBigQB];
#pragma unroll
    for (int q = 0; q < kBigQA; ++q) {
        const int pos = (wave * kBigQA + q) * 64 + lane;
        const int r = pos >> 2;
        chkA[q] = ((pos & 3) ^ bigswz(r)) * 8;
        const int kk = pos >> 5, xc = 8 * ((pos & 31) ^ kmswz(kk));
        kmA[q] = kk;
        // a k-major side reads whole 8-element chunks up to its size rounded
        // up to 8 (the host checks the rows hold that many)
        rowA[q] = KMA ? min(m0 + xc, ((P.M + 7) & ~7) - 8) : min(m0 + r, Mlast);
    }
#pragma unroll
    for (int q = 0; q < kBigQB; ++q) {
        constexpr int CPR = kBigTN / 8;   // chunks per k-row of a k-major B
        const int pos = (wave * kBigQB + q) * 64 + lane;
        const int r = pos >> 2;
        chkB[q] = ((pos & 3) ^ bigswz(r)) * 8;
        const int kk = pos / CPR, xc = 8 * ((pos % CPR) ^ kmswz(kk));
        kmB[q] = kk;
        rowB[q] = KMB ? min(n0 + xc, ((P.N + 7) & ~7) - 8) : min(n0 + r, Nlast);
    }
    auto issue = [&](int kt, int stage) {
        const bool s1 = kt >= kt0;
        const uint16_t *A = s1 ? A1 : A0;
        const uint16_t *Bm = s1 ? B1 : B0;
        const int64_t lda = s1 ? lda1 : lda0, ldb = s1 ? ldb1 : ldb0;
        const int k0 = (s1 ? kt - kt0 : kt) * kBigBK;
#pragma unroll
        for (int q = 0; q < kBigQA; ++q) {
            const uint16_t *g = KMA ? A + (int64_t)(k0 + kmA[q]) * lda + rowA[q] : A + (int64_t)rowA[q] * lda + k0 + chkA[q];
            __builtin_amdgcn_global_load_lds((const void *)g,
                                             (void __attribute__((address_space(3))) *)&lds[stage][(wave * kBigQA + q) * 512],
                                             16, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < kBigQB; ++q) {
            const uint16_t *g = KMB ? Bm + (int64_t)(k0 + kmB[q]) * ldb + rowB[q] : Bm + (int64_t)rowB[q] * ldb + k0 + chkB[q];
            __builtin_amdgcn_global_load_lds((const void *)g,
                                             (void __attribute__((address_space(3))) *)&lds[stage][kBigStageA + (wave * kBigQB + q) * 512],
                                             16, 0, 0);
        }
    };

    floatx16 acc[kBigFM][kBigFN];
#pragma unroll
    for (int i = 0; i < kBigFM; ++i)
#pragma unroll
        for (int j = 0; j < kBigFN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // tile t goes to stage t % kBigStages
    auto issue_tile = [&](int t) { issue(kt_begin + t, t % kBigStages); };
#pragma unroll
    for (int st = 0; st < kBigStages - 1; ++st)
        if (st < ntiles) issue_tile(st);

    constexpr int G = kBigQA + kBigQB;   // loads per tile per wavefront
    // Software pipeline over the two 16-k steps of a stage.  The operand
    // fragments of one k-step are read from LDS while the products of the
    // other run (the reads are interleaved with the matrix instructions), so
    // the LDS reads and the tile copies overlap the matrix-core time instead
    // of adding to it.  The barrier that publishes tile t+1 sits between
    // tile t's two k-steps:
    //   f0 = k-step 0 of tile t (in registers)
    //   products(f0) while f1 <- k-step 1 of tile t
    //   wait for tile t+1, barrier, copy tile t+3
    //   products(f1) while f0 <- k-step 0 of tile t+1
    // A stage is refilled only after every wavefront has consumed (not just
    // issued) its last read of that stage: stage (t+3) % 4 held tile t-1,
    // whose reads fed tile t-1's products.
    constexpr int KS = kBigBK / 16;
    static_assert(KS == 2, "the pipeline alternates two k-steps per stage");
    static_assert(kBigStages >= 3, "tile t+1 must be in flight behind tile t");
    bf16x8 fa[2][kBigFM], fb[2][kBigFN];
    // a k-major fragment: the two transposing reads of k-rows kb .. kb+3 and
    // kb+4 .. kb+7 (kb = 16 ks + 8 (lane / 32)) for the 32 row indices x0 ..
    auto km_frag = [&](const uint16_t *T, int RS, int ks, int x0) {   // RS: elements per k-row
        const int kk = 16 * ks + 8 * (lane >> 5) + ((lane & 15) >> 2);
        const int x = x0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
        const int off0 = kk * RS + ((x >> 3) ^ kmswz(kk)) * 8 + (x & 7);
        const int off1 = (kk + 4) * RS + ((x >> 3) ^ kmswz(kk + 4)) * 8 + (x & 7);
        return tr_frag(T, off0, off1);
    };
    auto read_frags = [&](int stage, int ks, bf16x8 (&a)[kBigFM], bf16x8 (&b)[kBigFN]) {
        const uint16_t *As = lds[stage];
        const uint16_t *Bs = lds[stage] + kBigStageA;
        const int c = 2 * ks + (lane >> 5);
#pragma unroll
        for (int i = 0; i < kBigFM; ++i) {
            if constexpr (KMA) {
                a[i] = km_frag(As, kBigT, ks, wm * kBigWTM + i * 32);
            } else {
                const int r = wm * kBigWTM + i * 32 + (lane & 31);
                a[i] = *(const bf16x8 *)&As[(r * 4 + (c ^ bigswz(r))) * 8];
            }
        }
#pragma unroll
        for (int j = 0; j < kBigFN; ++j) {
            if constexpr (KMB) {
                b[j] = km_frag(Bs, kBigTN, ks, wn * kBigWTN + j * 32);
            } else {
                const int r = wn * kBigWTN + j * 32 + (lane & 31);
                b[j] = *(const bf16x8 *)&Bs[(r * 4 + (c ^ bigswz(r))) * 8];
            }
        }
    };
    auto products = [&](const bf16x8 (&a)[kBigFM], const bf16x8 (&b)[kBigFN]) {
#pragma unroll
        for (int i = 0; i < kBigFM; ++i)
#pragma unroll
            for (int j = 0; j < kBigFN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };
    // the next k-step's LDS reads go out behind the first few products, so
    // they have the rest of the k-step to land
    constexpr int kReads = (KMA ? 2 : 1) * kBigFM + (KMB ? 2 : 1) * kBigFN;   // a k-major fragment is 2 reads
    constexpr int kReadsPer = GCN_BIG_READS_PER_MFMA;
    constexpr int kReadGroups = (kReads + kReadsPer - 1) / kReadsPer;
    static_assert(kReadGroups <= kBigFM * kBigFN, "a product ahead of every read group");
    auto interleave = [&]() {
        sched_reads<0, kReadGroups, kReadsPer, kReads>();
        __builtin_amdgcn_sched_group_barrier(0x008, kBigFM * kBigFN - kReadGroups, 0);
    };
    // the loads of a tile are done when at most `later` tiles' loads issued
    // after it are still outstanding; then a bare s_barrier: the fence of
    // __syncthreads would also wait for those later loads, which is the
    // latency the ring hides.  The empty asm statements keep the compiler
    // from moving LDS accesses across it.
    auto barrier_after_vmcnt = [&]() {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // wait until at most `later` tiles' copies (issued after the awaited
    // tile) are outstanding
    auto wait_tile = [&](int later) {
        if (later >= 3) wait_vmcnt<3 * G>();
        else if (later == 2) wait_vmcnt<2 * G>();
        else if (later == 1) wait_vmcnt<G>();
        else wait_vmcnt<0>();
    };
    auto half0 = [&](int t) {   // products of k-step 0 of tile t, reads of its k-step 1
        read_frags(t % kBigStages, 1, fa[1], fb[1]);
        products(fa[0], fb[0]);
        interleave();
    };
    auto half1 = [&](int t) {   // products of k-step 1 of tile t, reads of k-step 0 of tile t+1
        // (on the last tile the read is of a stale stage, in bounds and unused)
        read_frags((t + 1) % kBigStages, 0, fa[0], fb[0]);
        products(fa[1], fb[1]);
        interleave();
    };
    // the same, with tile t+stages-1's copies issued among the products
    // rather than in one burst after the barrier (every wavefront of the CU
    // issuing its copies at once stalls them all on the vector-memory queue)
    // (the copies follow the reads in program order: the compiler keeps LDS
    // reads and copies into LDS in order, not knowing their stages differ)
    auto half1_copy = [&](int t) {
        read_frags((t + 1) % kBigStages, 0, fa[0], fb[0]);
        issue_tile(t + kBigStages - 1);
        products(fa[1], fb[1]);
        sched_reads_copies<0, kBigFM * kBigFN, kReadGroups, kReadsPer, kReads, G>();
    };
    if (ntiles > 0) {
        wait_tile(min(ntiles - 1, kBigStages - 2));   // tile 0
        barrier_after_vmcnt();
        read_frags(0, 0, fa[0], fb[0]);
    }
    // Steady state: tile t+1 is awaited with tiles t+2 .. t+stages-2 still in
    // flight, then tile t+stages-1 is copied.  No branches in this loop.
    int t = 0;
    for (; t < ntiles - kBigStages + 1; ++t) {
        half0(t);
        wait_vmcnt<(kBigStages - 3) * G>();
        barrier_after_vmcnt();
        if constexpr (GCN_BIG_COPY_SPREAD) {
            half1_copy(t);
        } else {
            issue_tile(t + kBigStages - 1);
            half1(t);
        }
    }
    // The last tiles: nothing left to copy, fewer copies in flight.
    for (; t < ntiles; ++t) {
        half0(t);
        if (t + 1 < ntiles) {
            wait_tile(min(ntiles - 2 - t, kBigStages - 3));
            barrier_after_vmcnt();
        }
        half1(t);
    }

    const bool to_partial = P.split > 1;
    float *dst = to_partial ? P.partial + (int64_t)bc.split * P.M * P.N : P.C;
    const int64_t ldd = to_partial ? P.N : P.ldc;
    // ---- epilogue through LDS, in two passes of 128 rows: the wavefronts
    // holding those rows deposit their accumulators row-major in the (now
    // idle) operand ring, then every wavefront writes whole 256-column rows,
    // 16 bytes per lane.  Accumulator blocks are moved by calls with constant
    // indices, so that they stay in registers.
    static_assert(128 * kBigTN * sizeof(float) <= sizeof(lds), "the epilogue stages 128 rows of floats in the ring");
    static_assert(kBigFM == 4 && (kBigFN == 4 || kBigFN == 2), "epilogue unrolled for 4 x 4 or 4 x 2 blocks");
    float *stg = (float *)&lds[0][0];
    auto put = [&](const floatx16 &v, int i, int j) {
        const int lc = wn * kBigWTN + j * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int lr = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            stg[lr * kBigTN + lc] = v[r];
        }
    };
    // a row of the tile is kColLanes lanes x 4 columns; a wavefront writes
    // kRowsPerInstr rows per instruction
    constexpr int kColLanes = kBigTN / 4, kRowsPerInstr = 64 / kColLanes;
    const int sub = lane / kColLanes;
    const bool c16 = OUT != BIG_F32 && !to_partial && P.C16 != nullptr;
    const bool c32 = OUT != BIG_B16 && (to_partial || P.C != nullptr);
    const bool vec16 = c16 && P.ldc16 % 4 == 0 && ((uintptr_t)P.C16 & 7) == 0;
    const bool vec32 = c32 && ldd % 4 == 0 && ((uintptr_t)dst & 15) == 0;
    const int col = n0 + 4 * (lane % kColLanes);
    float bv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (!to_partial && P.bias)
#pragma unroll
        for (int e = 0; e < 4; ++e) bv[e] = col + e < P.N ? P.bias[col + e] : 0.0f;
    const bool relu = !to_partial && P.relu;
    // optional [mask > 0] factor (bfloat16 mask) and column sums per 128-row
    // half of the tile
    const uint16_t *const emask = to_partial ? nullptr : P.mask16;
    const bool mvec = emask && P.ldm % 4 == 0 && ((uintptr_t)emask & 7) == 0 && col + 3 <= Nlast;
    const bool ecs = !to_partial && P.colpart;
    float cs[2][4] = {{0.0f, 0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f, 0.0f}};
    // the mask of a pass's rows is loaded in batches of kMaskBatch rows: the
    // first batch before that pass's deposit and barrier (its latency
    // overlaps them), each later one as the previous batch is used up
    constexpr int kRowsPerWave = 128 / (kBigWaves * kRowsPerInstr);   // instructions per 128-row pass
    constexpr int kMaskBatch = GCN_BIG_MASK_PREFETCH;
    static_assert(kRowsPerWave % kMaskBatch == 0, "whole mask batches");
    uint2 mk[kMaskBatch];   // 4 bfloat16 mask values per row
    auto load_mask = [&](int h, int k0) {
#pragma unroll
        for (int k = 0; k < kMaskBatch; ++k) {
            const int row = m0 + h * 128 + ((k0 + k) * kBigWaves + wave) * kRowsPerInstr + sub;
            mk[k] = make_uint2(0u, 0u);
            if (row <= Mlast && col <= Nlast) {
                const uint16_t *mp = emask + (int64_t)row * P.ldm + col;
                if (mvec) {
                    mk[k] = *(const uint2 *)mp;
                } else {
                    mk[k].x = mp[0];
                    if (col + 1 <= Nlast) mk[k].x |= (uint32_t)mp[1] << 16;
                    if (col + 2 <= Nlast) mk[k].y = mp[2];
                    if (col + 3 <= Nlast) mk[k].y |= (uint32_t)mp[3] << 16;
                }
            }
        }
    };
    __syncthreads();   // every wavefront is done reading the ring
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if (emask) load_mask(h, 0);
        if (wm == h) {
            put(acc[0][0], 0, 0); put(acc[0][1], 0, 1);
            put(acc[1][0], 1, 0); put(acc[1][1], 1, 1);
            put(acc[2][0], 2, 0); put(acc[2][1], 2, 1);
            put(acc[3][0], 3, 0); put(acc[3][1], 3, 1);
            if constexpr (kBigFN == 4) {
                put(acc[0][2], 0, 2); put(acc[0][3], 0, 3);
                put(acc[1][2], 1, 2); put(acc[1][3], 1, 3);
                put(acc[2][2], 2, 2); put(acc[2][3], 2, 3);
                put(acc[3][2], 3, 2); put(acc[3][3], 3, 3);
            }
        }
        __syncthreads();
        // rows rr = (k * kBigWaves + wave) * kRowsPerInstr + sub of the pass;
        // their LDS reads go out kRB at a time, ahead of the stores, and the
        // output offsets advance by a fixed row step
        constexpr int kRowStep = kBigWaves * kRowsPerInstr;
        constexpr int kRB = 4;
        static_assert(kRowsPerWave % kRB == 0 && kMaskBatch % kRB == 0, "whole row batches");
        const int rr0 = wave * kRowsPerInstr + sub;
        const int row0 = m0 + h * 128 + rr0;
        const float *const srow = stg + rr0 * kBigTN + 4 * (lane % kColLanes);
        const bool colok = col <= Nlast;
        // whole 4-column groups on the vector paths (uniform over the launch)
        const bool v16 = vec16 && P.N % 4 == 0, v32 = vec32 && P.N % 4 == 0;
        // output row addresses, advanced by one row step per row
        uint16_t *p16 = c16 ? P.C16 + (int64_t)row0 * P.ldc16 + col : nullptr;
        float *p32 = c32 ? dst + (int64_t)row0 * ldd + col : nullptr;
        const int64_t s16 = (int64_t)kRowStep * P.ldc16, s32 = (int64_t)kRowStep * ldd;
#pragma unroll
        for (int k0 = 0; k0 < kRowsPerWave; k0 += kRB) {
            if (emask && k0 > 0 && k0 % kMaskBatch == 0) load_mask(h, k0);
            float4 qb[kRB];
#pragma unroll
            for (int u = 0; u < kRB; ++u) qb[u] = *(const float4 *)(srow + (k0 + u) * kRowStep * kBigTN);
#pragma unroll
            for (int u = 0; u < kRB; ++u) {
                const int k = k0 + u;
                const bool ok = colok && row0 + k * kRowStep <= Mlast;
                const float4 q = qb[u];
                float o[4] = {q.x + bv[0], q.y + bv[1], q.z + bv[2], q.w + bv[3]};
                if (relu)
#pragma unroll
                    for (int e = 0; e < 4; ++e) o[e] = fmaxf(o[e], 0.0f);
                if (emask) {
                    const uint2 m = mk[k % kMaskBatch];
                    o[0] = bf16_bits_positive(m.x & 0xFFFFu) ? o[0] : 0.0f;
                    o[1] = bf16_bits_positive(m.x >> 16) ? o[1] : 0.0f;
                    o[2] = bf16_bits_positive(m.y & 0xFFFFu) ? o[2] : 0.0f;
                    o[3] = bf16_bits_positive(m.y >> 16) ? o[3] : 0.0f;
                }
                if (ok) {
                    if (ecs)
#pragma unroll
                        for (int e = 0; e < 4; ++e) cs[h][e] += o[e];
                    if (c16) {
                        uint16_t *d = p16;
                        if (v16) {
                            *(uint2 *)d = make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (col + e <= Nlast) d[e] = to_bf16(o[e]);
                        }
                    }
                    if (c32) {
                        float *d = p32;
                        if (v32) {
                            *(float4 *)d = make_float4(o[0], o[1], o[2], o[3]);
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (col + e <= Nlast) d[e] = o[e];
                        }
                    }
                }
                if (c16) p16 += s16;
                if (c32) p32 += s32;
            }
        }
        __syncthreads();
    }
    if (ecs) {
        // per half: the 8 wavefronts' sums of each column, in order; the
        // half's rows are column-sum row 2 * tm + h (128-row tiles)
        static_assert(2 * kBigWaves * kBigTN * sizeof(float) <= sizeof(lds), "column sums fit the ring");
        static_assert((2 * kBigTN) % kBigThreads == 0, "whole (half, column) sweeps");
        // the rows a wavefront's two lane halves summed (when a row is half a
        // wavefront wide), added in a fixed way
        if constexpr (kRowsPerInstr == 2) {
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int e = 0; e < 4; ++e) cs[h][e] += __shfl_xor(cs[h][e], 32);
        }
        static_assert(kRowsPerInstr == 1 || kRowsPerInstr == 2, "one or two rows per instruction");
        if (sub == 0)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int e = 0; e < 4; ++e) stg[(h * kBigWaves + wave) * kBigTN + 4 * lane + e] = cs[h][e];
        __syncthreads();
#pragma unroll
        for (int idx = (int)threadIdx.x; idx < 2 * kBigTN; idx += kBigThreads) {
            const int h = idx / kBigTN, c = idx % kBigTN;
            float t = 0.0f;
#pragma unroll
            for (int w = 0; w < kBigWaves; ++w) t += stg[(h * kBigWaves + w) * kBigTN + c];
            if (m0 + h * 128 <= Mlast && n0 + c <= Nlast) P.colpart[(int64_t)(2 * bc.tm + h) * P.N + n0 + c] = t;
        }
    }
}

bool vec_ok(int layout, const GemmProblem &g, int esz) {
    const int E = 16 / esz;
    const bool a_km = layout == L_TN, b_km = layout != L_NT;
    for (int s = 0; s < 2; ++s) {
        const GemmSeg &sg = g.seg[s];
        if (sg.K == 0) continue;
        if (sg.lda % E || sg.ldb % E || !al(sg.A, 16) || !al(sg.B, 16)) return false;
        if (a_km ? (g.M % E) : (sg.K % E)) return false;
        if (b_km ? (g.N % E) : (sg.K % E)) return false;
    }
    return true;
}

// mode 0: float32 kernel; 1: bf16 kernel; 2: bf16 large-tile kernel
int bk_of(int mode) { return mode == 2 ? kBigBK : (mode ? BK16 : kBK); }
int tile_m_of(int mode) { return mode == 2 ? kBigT : (mode ? kTBM16 : kTBM); }
int tile_n_of(int mode) { return mode == 2 ? kBigTN : (mode ? kTBN16 : kTBN); }

// The large-tile bf16 kernel takes NT, TN and NN products whose K-segments
// are multiples of its k-stage, with 16-byte aligned operand rows; a k-major
// operand (A of TN, B of TN and NN) is read in chunks of 8 along M (or N),
// so its rows must hold M (N) rounded up to 8 (the extra columns only feed
// outputs that are dropped).
#ifndef GCN_BIG_NARROW_K
#define GCN_BIG_NARROW_K 16384
#endif
bool big_ok(int layout, int nprob, const GemmProblem *probs) {
    if (GCN_BF16_BIG == 0) return false;
    const bool kma = layout == L_TN, kmb = layout != L_NT;
    for (int i = 0; i < nprob; ++i) {
        if (!GCN_BIG_MASKED && probs[i].mask16) return false;
        // A side of 128 or less leaves most of a 256-wide tile idle.  Still
        // worth it for a side of 64+ when the other one alone gives every CU
        // a tile (the logits of a large subgraph): the product is then bound
        // by its operand and output traffic, not by the idle matrix work.
        // Also for a long-K product (a weight gradient over the subgraph's
        // vertices), whose split-K blocks fill the GPU whatever the tiles.
        const int lo = min(probs[i].M, probs[i].N);
        const int64_t tiles = (int64_t)((probs[i].M + kBigT - 1) / kBigT) * ((probs[i].N + kBigTN - 1) / kBigTN);
        const int64_t K = (int64_t)probs[i].seg[0].K + probs[i].seg[1].K;
        if (lo <= 128 && !(lo >= 64 && (tiles >= GCN_BIG_NARROW_TILES || K >= GCN_BIG_NARROW_K))) return false;
        for (int s = 0; s < 2; ++s) {
            const GemmSeg &sg = probs[i].seg[s];
            if (sg.K == 0) continue;
            if (sg.K % kBigBK || sg.lda % 8 || sg.ldb % 8 || !al(sg.A, 16) || !al(sg.B, 16)) return false;
        }
        const int64_t M8 = (probs[i].M + 7) & ~7, N8 = (probs[i].N + 7) & ~7;
        for (int s = 0; s < 2; ++s) {
            const GemmSeg &sg = probs[i].seg[s];
            if (sg.K == 0) continue;
            if ((kma && sg.lda < M8) || (kmb && sg.ldb < N8)) return false;
        }
    }
    return true;
}

void fill_dev(int layout, int nprob, const GemmProblem *probs, int bf16, int split_k, float *partial,
              DevArgs &a, int64_t &blocks) {
    const int BK = bk_of(bf16);  // bf16 here is the kernel mode (0, 1, 2)
    blocks = 0;
    a.nprob = nprob;
    size_t poff = 0;
    for (int i = 0; i < nprob; ++i) {
        const GemmProblem &g = probs[i];
        DevProblem &d = a.p[i];
        d.M = g.M;
        d.N = g.N;
        d.tiles_m = (g.M + tile_m_of(bf16) - 1) / tile_m_of(bf16);
        d.tiles_n = (g.N + tile_n_of(bf16) - 1) / tile_n_of(bf16);
        d.kt_total = 0;
        for (int s = 0; s < 2; ++s) {
            d.s.A[s] = g.seg[s].A;
            d.s.B[s] = g.seg[s].B;
            d.s.lda[s] = g.seg[s].lda;
            d.s.ldb[s] = g.seg[s].ldb;
            d.s.K[s] = g.seg[s].K;
            d.s.kt[s] = (g.seg[s].K + BK - 1) / BK;
            d.kt_total += d.s.kt[s];
        }
        int sp = split_k < 1 ? 1 : split_k;
        if (sp > d.kt_total) sp = d.kt_total > 0 ? d.kt_total : 1;
        d.kt_per_split = d.kt_total > 0 ? (d.kt_total + sp - 1) / sp : 0;
        // recompute so that no split is empty
        d.split = d.kt_per_split > 0 ? (d.kt_total + d.kt_per_split - 1) / d.kt_per_split : 1;
        d.block_begin = blocks;
        blocks += (int64_t)d.tiles_m * d.tiles_n * d.split;
        d.C = g.C;
        d.ldc = g.ldc;
        d.bias = g.bias;
        d.relu = g.relu;
        d.partial = nullptr;
        d.C16 = g.C16;
        d.ldc16 = g.ldc16 ? g.ldc16 : g.ldc;
        d.C16T = g.C16T;
        d.ldc16t = g.ldc16t;
        d.n16t = g.C16T ? min(g.n16t, g.N) : 0;
        d.mask = g.mask;
        d.mask16 = g.mask16;
        d.ldm = g.ldm;
        d.colpart = g.colpart;
        if (d.split > 1) {
            d.partial = partial ? (float *)((char *)partial + poff) : nullptr;
            poff += align256((size_t)d.split * g.M * g.N * sizeof(float));
        }
    }
    if (nprob < 2) a.p[1] = a.p[0];
    a.total = (int64_t)a.p[0].split * a.p[0].tiles_m * nprob * a.p[0].tiles_n;
    a.per_xcd = (a.total + 7) / 8;
    blocks = a.total > 0 ? 8 * a.per_xcd : 0;
}

template <int LAYOUT>
void launch(bool vec, bool bf16, dim3 grid, hipStream_t s, const DevArgs &a) {
    if (bf16) {
        if (vec)
            hipLaunchKernelGGL((gemm_bf16_kernel<LAYOUT, true>), grid, dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL((gemm_bf16_kernel<LAYOUT, false>), grid, dim3(kThreads), 0, s, a);
    } else if (vec) {
        hipLaunchKernelGGL((gemm_kernel<LAYOUT, true, kTBM, kTBN>), grid, dim3(kThreads), 0, s, a);
    } else {
        hipLaunchKernelGGL((gemm_kernel<LAYOUT, false, kTBM, kTBN>), grid, dim3(kThreads), 0, s, a);
    }
}

}  // namespace

bool gemm_bf16_big_ok(int layout, int nprob, const GemmProblem *probs) { return big_ok(layout, nprob, probs); }

#ifndef GCN_SPLIT_MIN_TILES
#define GCN_SPLIT_MIN_TILES 256
#endif
#ifndef GCN_SPLIT_TARGET
#define GCN_SPLIT_TARGET 512
#endif
#ifndef GCN_SPLIT_CAP
#define GCN_SPLIT_CAP 64
#endif
int gemm_pick_split(int nprob, const GemmProblem *probs, bool k_is_rows) {
    int64_t tiles = 0, kt = 0;
    for (int i = 0; i < nprob; ++i) {
        tiles += (int64_t)((probs[i].M + kTBM - 1) / kTBM) * ((probs[i].N + kTBN - 1) / kTBN);
        int64_t k = 0;
        for (int s = 0; s < 2; ++s) k += (probs[i].seg[s].K + kBK - 1) / kBK;
        if (k > kt) kt = k;
    }
    if (tiles <= 0) return 1;
    // Weight gradients (K = the subgraph's vertices, few output tiles): split
    // to about four blocks per CU.  Other products: split only when the tiles
    // do not give every CU a block, since the reduce pass costs a read of
    // every partial.
    int64_t sp;
    if (k_is_rows) sp = 1024 / tiles;
    else sp = tiles >= GCN_SPLIT_MIN_TILES ? 1 : GCN_SPLIT_TARGET / tiles;
    const int64_t max_sp = kt / 8;      // keep >= 8 k-tiles per split
    if (sp > max_sp) sp = max_sp;
    if (sp > GCN_SPLIT_CAP) sp = GCN_SPLIT_CAP;   // partials are written and read once each
    if (sp < 1) sp = 1;
    return (int)sp;
}

int32_t gemm_colpart_rows(int32_t M) { return M > 0 ? (M + kTBM - 1) / kTBM : 0; }

size_t gemm_workspace_bytes(int nprob, const GemmProblem *probs, int split_k) {
    if (split_k <= 1) return 0;
    size_t b = 0;
    for (int i = 0; i < nprob; ++i)
        b += align256((size_t)split_k * probs[i].M * probs[i].N * sizeof(float));
    return b + 256;
}

int gemm(int layout, int nprob, const GemmProblem *probs, int bf16, int split_k, void *ws,
         size_t ws_bytes, hipStream_t s) {
    if (nprob < 1 || nprob > 2) {
        set_error("gemm: nprob %d", nprob);
        return GCN_EINVAL;
    }
    if (nprob == 2 && (probs[0].M != probs[1].M || probs[0].N != probs[1].N ||
                       probs[0].seg[0].K + probs[0].seg[1].K != probs[1].seg[0].K + probs[1].seg[1].K)) {
        set_error("gemm: grouped problems must have equal M, N and K");
        return GCN_EINVAL;
    }
    bool vec = true;
    double flops = 0.0, bytes = 0.0;
    for (int i = 0; i < nprob; ++i) {
        const GemmProblem &g = probs[i];
        vec = vec && vec_ok(layout, g, bf16 ? 2 : 4);
        const double K = (double)g.seg[0].K + g.seg[1].K;
        flops += 2.0 * g.M * g.N * (K - g.k_pad);
        // algorithmic bytes: each operand read once, the output written once
        // (float32 or bfloat16), the mask read once, the bias read once
        const double esz = bf16 ? 2.0 : 4.0;
        bytes += esz * K * ((double)g.M + g.N) + (double)g.M * g.N * ((g.C16 ? 2.0 : 0.0) + (g.C ? 4.0 : 0.0)) +
                 (g.C16T ? 2.0 * g.M * std::min(g.n16t, g.N) : 0.0) +
                 (g.mask ? 4.0 * g.M * g.N : 0.0) + (g.mask16 ? 2.0 * g.M * g.N : 0.0) + (g.bias ? 4.0 * g.N : 0.0);
    }
    float *partial = nullptr;
    if (split_k > 1) {
        if (!ws || ws_bytes < gemm_workspace_bytes(nprob, probs, split_k)) {
            set_error("gemm: split-K workspace too small");
            return GCN_EWORKSPACE;
        }
        partial = (float *)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    }
    const bool big = bf16 && big_ok(layout, nprob, probs);
    DevArgs a;
    int64_t blocks = 0;
    fill_dev(layout, nprob, probs, big ? 2 : (bf16 ? 1 : 0), split_k, partial, a, blocks);
    if (blocks == 0) return GCN_OK;
    if (nprob == 2 && (a.p[0].kt_total != a.p[1].kt_total || a.p[0].split != a.p[1].split)) {
        set_error("gemm: grouped problems must have the same K-tiling");
        return GCN_EINVAL;
    }
    bool any_split = false;
    for (int i = 0; i < nprob; ++i) {
        any_split = any_split || a.p[i].split > 1;
        const bool masked = probs[i].mask || probs[i].mask16;
        if (!probs[i].C && !probs[i].C16) {
            set_error("gemm: no output");
            return GCN_EINVAL;
        }
        if (probs[i].C16T && !bf16 && !probs[i].C) {
            set_error("gemm: a transposed bfloat16 output needs a row output to come from");
            return GCN_EINVAL;
        }
        if ((masked || probs[i].colpart) && a.p[i].split > 1) {
            set_error("gemm: the mask and column-sum epilogue needs an unsplit product");
            return GCN_EINVAL;
        }
        if (bf16 ? probs[i].mask != nullptr : probs[i].mask16 != nullptr) {
            set_error("gemm: bfloat16 products take a bfloat16 mask (mask16), float32 products a float32 one");
            return GCN_EINVAL;
        }
        if (masked && probs[i].ldm < probs[i].N) {
            set_error("gemm: mask leading dimension %lld < N=%d", (long long)probs[i].ldm, probs[i].N);
            return GCN_ESHAPE;
        }
    }
    int cls = layout == L_NN ? K_GEMM_NN : (layout == L_TN ? K_GEMM_TN : K_GEMM_NT);
    if (bf16) cls += K_GEMM_NN_BF16 - K_GEMM_NN;
    if (big) {
        bool masked = false;
        for (int i = 0; i < nprob; ++i) masked = masked || probs[i].mask16;
        cls = masked ? K_GEMM_NT_BF16_BIG_MASKED : (layout == L_NT ? K_GEMM_NT_BF16_BIG : K_GEMM_TN_BF16_BIG);
    }
    {
        ProfScope ps(cls, s, flops, bytes);
        dim3 grid((unsigned)blocks);
        if (big) {
            // the output set every problem of the launch fits in
            bool any32 = false, any16 = false;
            for (int i = 0; i < nprob; ++i) {
                any32 = any32 || a.p[i].split > 1 || probs[i].C;
                any16 = any16 || (a.p[i].split == 1 && probs[i].C16);
            }
            const int out = !any16 ? BIG_F32 : (!any32 ? BIG_B16 : BIG_ALL);
#define GCN_BIG_LAUNCH(O, LY)                                                                           \
    if (out == O && layout == LY) hipLaunchKernelGGL((gemm_bf16_big_kernel<O, LY>), grid, dim3(kBigThreads), 0, s, a);
            GCN_BIG_LAUNCH(BIG_F32, L_NT) GCN_BIG_LAUNCH(BIG_B16, L_NT) GCN_BIG_LAUNCH(BIG_ALL, L_NT)
            GCN_BIG_LAUNCH(BIG_F32, L_TN) GCN_BIG_LAUNCH(BIG_B16, L_TN) GCN_BIG_LAUNCH(BIG_ALL, L_TN)
            GCN_BIG_LAUNCH(BIG_F32, L_NN) GCN_BIG_LAUNCH(BIG_B16, L_NN) GCN_BIG_LAUNCH(BIG_ALL, L_NN)
#undef GCN_BIG_LAUNCH
        }
        else if (layout == L_NN) launch<L_NN>(vec, bf16 != 0, grid, s, a);
        else if (layout == L_TN) launch<L_TN>(vec, bf16 != 0, grid, s, a);
        else launch<L_NT>(vec, bf16 != 0, grid, s, a);
        GCN_LAUNCH_CHECK("gemm_kernel");
    }
    if (any_split) {
        double rbytes = 0.0;
        for (int i = 0; i < nprob; ++i)
            rbytes += (double)a.p[i].M * a.p[i].N * 4.0 * (a.p[i].split + 1);
        ProfScope ps(K_SPLITK_REDUCE, s, 0.0, rbytes);
        int64_t maxe = 0;
        int maxsplit = 1;
        for (int i = 0; i < nprob; ++i) {
            maxe = std::max<int64_t>(maxe, (int64_t)a.p[i].M * a.p[i].N);
            maxsplit = std::max(maxsplit, a.p[i].split);
        }
        // a problem without splits is written by the main kernel already; the
        // reduce skips it by running over zero elements
        DevArgs r = a;
        bool v4 = true;
        for (int i = 0; i < nprob; ++i) {
            if (r.p[i].split <= 1) { r.p[i].M = 0; }
            const DevProblem &q = r.p[i];
            v4 = v4 && q.N % 4 == 0 && (!q.C || (q.ldc % 4 == 0 && al(q.C, 16)));
        }
        const int64_t vecs = v4 ? maxe / 4 : maxe;
        // threads per output element: up to 8, for about 2^20 elements-threads
        // per pair of problems.  It depends on a problem's own size and split
        // only (not on how many problems share the launch, nor on the vector
        // width), so a product reduces to the same bits alone or grouped.
        int G = 1;
        while (G < 8 && 2 * G <= maxsplit && maxe * 2 * G < (1 << 20)) G *= 2;
        int64_t g = (vecs + 256 / G - 1) / (256 / G);
        if (g > 4096) g = 4096;
        if (g < 1) g = 1;
        if (v4) hipLaunchKernelGGL(splitk_reduce<true>, dim3((unsigned)g, (unsigned)nprob), dim3(256), 0, s, r, G);
        else hipLaunchKernelGGL(splitk_reduce<false>, dim3((unsigned)g, (unsigned)nprob), dim3(256), 0, s, r, G);
        GCN_LAUNCH_CHECK("splitk_reduce");
    }
    // transposed bfloat16 outputs: one pass over the bfloat16 rows (or the
    // float32 ones) after the product.  (Written from the large-tile epilogue
    // instead, a tile's 256 transposed rows all land at one offset inside
    // rows n elements apart, which puts the tile's writes in one memory
    // channel; the separate pass spreads its blocks over the offsets.)
    for (int i = 0; i < nprob; ++i) {
        const GemmProblem &g = probs[i];
        if (!g.C16T) continue;
        const int32_t cols = std::min(g.n16t, g.N);
        if (cols <= 0) continue;
        const int rc = g.C16 ? transpose_bf16(g.M, cols, g.C16, 1, g.ldc16 ? g.ldc16 : g.ldc, g.C16T, g.ldc16t, s)
                             : transpose_bf16(g.M, cols, g.C, 0, g.ldc, g.C16T, g.ldc16t, s);
        if (rc) return rc;
    }
    return GCN_OK;
}

}  // namespace gcn
