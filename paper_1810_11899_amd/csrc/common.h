// Internal declarations shared by the HIP sources of libgcnlayer (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "gcn_layer.h"

namespace gcn {

constexpr int kWave = 64;  // CDNA wavefront width

// ------------------------------------------------------- bfloat16 rounding
// float32 -> bfloat16, round to nearest even; a NaN stays NaN (quiet bit set)
__device__ __forceinline__ uint16_t to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return (uint16_t)((u & 0x7FFFFFFFu) > 0x7F800000u ? ((u >> 16) | 0x0040u) : r);
}
#ifndef GCN_HW_BF16
#define GCN_HW_BF16 1
#endif
typedef float gcn_float2 __attribute__((ext_vector_type(2)));
typedef __bf16 gcn_bf16x2 __attribute__((ext_vector_type(2)));
// Two values rounded as to_bf16 does, packed (a in the low half).  gfx950
// rounds a pair in one instruction (v_cvt_pk_bf16_f32, round to nearest even),
// with to_bf16's bits on every float32 input, NaN payloads included.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
#if GCN_HW_BF16
    const gcn_float2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, gcn_bf16x2));
#else
    return (uint32_t)to_bf16(a) | ((uint32_t)to_bf16(b) << 16);
#endif
}

// ------------------------------------------------------------------ errors
void set_error(const char *fmt, ...);
int hip_fail(hipError_t e, const char *what);
#define GCN_HIP_CHECK(expr)                                   \
    do {                                                      \
        hipError_t e_ = (expr);                               \
        if (e_ != hipSuccess) return ::gcn::hip_fail(e_, #expr); \
    } while (0)
#define GCN_LAUNCH_CHECK(what)                                \
    do {                                                      \
        hipError_t e_ = hipGetLastError();                    \
        if (e_ != hipSuccess) return ::gcn::hip_fail(e_, what); \
    } while (0)

// ---------------------------------------------------------------- profiling
enum KernelClass {
    K_SPMM = 0,
    K_SPMM_FIXUP,
    K_GEMM_NN,
    K_GEMM_TN,
    K_GEMM_NT,
    K_SPLITK_REDUCE,
    K_RELU_MASK,
    K_COLSUM_REDUCE,
    K_LOSS_ROWS,
    K_LOSS_REDUCE,
    K_T_COUNT,
    K_T_SCAN,
    K_T_FILL,
    K_T_SORT,
    K_T_FINAL,
    K_CVT_BF16,
    K_GEMM_NN_BF16,
    K_GEMM_TN_BF16,
    K_GEMM_NT_BF16,
    K_SPMM_BF16,
    K_TRANSPOSE_BF16,
    K_SAMPLE,
    K_INDUCE,
    K_GATHER,
    K_ADAM,
    K_T_SYM,
    K_GEMM_NT_BF16_BIG,         // the bfloat16 large-tile kernel
    K_GEMM_NT_BF16_BIG_MASKED,  // the same with the ReLU-derivative epilogue
    K_GEMM_TN_BF16_BIG,         // the large-tile kernel on k-major operands (weight gradients)
    K_CLASS_COUNT
};
const char *class_name(int cls);
// While one of these lives on a thread, that thread's launches are not
// timed even with profiling on (timing creates events, and the entry point
// that promises to allocate nothing must not create any).
struct ProfSuppress {
    ProfSuppress();
    ~ProfSuppress();
};
// Recorded around one launch when profiling is on; no-ops otherwise.
struct ProfScope {
    ProfScope(int cls, hipStream_t s, double flops, double bytes);
    ~ProfScope();
    int cls_;
    hipStream_t s_;
    int slot_;
};

// ------------------------------------------------------------- CSR indices
// The column indices of a CSR: int32, or uint16 when the columns number at
// most 65,536 (half the index bytes; the INT16 indices of Sec. V-B).
struct IdxRef {
    const int32_t *i32;
    const uint16_t *i16;
    __host__ __device__ __forceinline__ int32_t operator[](int64_t p) const {
        return i16 ? (int32_t)i16[p] : i32[p];
    }
};
inline IdxRef idx_of(const gcn_csr *A) { return IdxRef{A->indices, A->indices16}; }

// --------------------------------------------------------------- workspace
// Bump allocator over the caller's workspace; every carve is 256-byte aligned.
struct Arena {
    char *base;
    size_t cap;
    size_t used;
    Arena(void *b, size_t c) : base((char *)b), cap(c), used(0) {}
    template <class T> T *take(size_t count) {
        size_t off = (used + 255) & ~(size_t)255;
        used = off + ((count * sizeof(T) + 255) & ~(size_t)255);
        return (base && used <= cap) ? (T *)(base + off) : nullptr;
    }
};
inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// --------------------------------------------------------------- launchers
// SpMM (feature propagation) -------------------------------------------------
// out is float for the first three, bfloat16 bits for EPI_STORE_BF16
enum SpmmEpilogue { EPI_STORE = 0, EPI_BIAS_RELU = 1, EPI_ACCUMULATE = 2, EPI_STORE_BF16 = 3 };
struct SpmmPlan {
    int64_t items;      // n_rows + nnz (merge-path length)
    int ipw;            // merge items per wavefront
    int64_t waves;      // wavefronts in the main kernel
};
SpmmPlan spmm_plan(int32_t n_rows, int32_t nnz);
size_t spmm_workspace_bytes(int32_t n_rows, int32_t nnz, int32_t k);
// the merge-path row ranges of a CSR (first row of every wavefront's range,
// spmm_plan(n_rows, nnz).waves + 1 entries), which depend only on indptr
size_t spmm_bounds_bytes(int32_t n_rows, int32_t nnz);
int spmm_bounds(int32_t n_rows, int32_t nnz, const int32_t *indptr, int32_t *bounds, hipStream_t s);
// out[i, c] (epilogue) sum_p vals[p] * X[indices[p], c].  `bounds`: the row
// ranges from spmm_bounds for this indptr, or NULL to compute them here.
// out16 (EPI_STORE / EPI_BIAS_RELU): the same values also as bfloat16 rows
// (leading dim ld16); `out` may then be NULL.
int spmm_f32(int32_t n_rows, int32_t nnz, const int32_t *indptr, IdxRef indices,
             const float *vals, const float *X, int32_t k, int64_t ldx, void *out, int64_t ldo,
             int epilogue, const float *bias, void *ws, size_t ws_bytes, hipStream_t s,
             const int32_t *bounds = nullptr, uint16_t *out16 = nullptr, int64_t ld16 = 0);
// same with bfloat16 rows of X (uint16 bits), float32 accumulation
int spmm_bf16(int32_t n_rows, int32_t nnz, const int32_t *indptr, IdxRef indices,
              const float *vals, const uint16_t *X, int32_t k, int64_t ldx, void *out, int64_t ldo,
              int epilogue, const float *bias, void *ws, size_t ws_bytes, hipStream_t s,
              const int32_t *bounds = nullptr, uint16_t *out16 = nullptr, int64_t ld16 = 0);

// GEMM on the matrix cores -----------------------------------------------------
// C[M x N] = sum over up to two K-segments of op(A_s) op(B_s), then epilogue.
//   layout NN: A_s is M x K_s (lda), B_s is K_s x N (ldb)
//   layout TN: A_s is stored K_s x M (A^T is used), B_s is K_s x N
//   layout NT: A_s is M x K_s, B_s is stored N x K_s (B^T is used)
enum GemmLayout { L_NN = 0, L_TN = 1, L_NT = 2 };
struct GemmSeg {
    const void *A;
    int64_t lda;
    const void *B;
    int64_t ldb;
    int32_t K;
};
struct GemmProblem {
    int32_t M, N;
    GemmSeg seg[2];   // seg[1].K == 0 when unused
    float *C;
    int64_t ldc;
    const float *bias;  // [N] or null
    int relu;
    // Outputs, each written when set (at least one of C, C16): C float32
    // (leading dim ldc); C16 the same values as bfloat16 (RNE) rows (leading
    // dim ldc16, ldc when 0); C16T bfloat16 transposed, element (i, j) at
    // C16T[j * ldc16t + i], for the columns j < n16t only.
    uint16_t *C16;
    int64_t ldc16;
    uint16_t *C16T;
    int64_t ldc16t;
    int32_t n16t;
    int32_t k_pad;      // trailing K columns that are zero padding (left out of the flop count)
    // float32 kernel, unsplit only: C[i][j] is kept where mask[i][j] > 0 and
    // set to 0 elsewhere (leading dim ldm), after bias and ReLU
    const float *mask;
    // bfloat16 kernels: the mask as bfloat16 bits, same rule and leading dim
    // (a bfloat16 product takes only this one, a float32 product only mask)
    const uint16_t *mask16;
    int64_t ldm;
    // unsplit only: colpart[t][j] = sum of the stored C[i][j]
    // over the rows i of row tile t (gemm_colpart_rows(M) x N, leading dim N)
    float *colpart;
};
// Up to two problems of equal layout and equal M, N, K in one launch
// (grouped).  `bf16` selects bfloat16 operands (uint16 bits) instead of
// float32.  split_k > 1 needs workspace (gemm_workspace_bytes).
int gemm(int layout, int nprob, const GemmProblem *probs, int bf16, int split_k,
         void *ws, size_t ws_bytes, hipStream_t s);
size_t gemm_workspace_bytes(int nprob, const GemmProblem *probs, int split_k);
// whether bfloat16 products of this layout and shape run on the large-tile
// kernel (which reads k-major operands, TN and NN, with transposing LDS reads)
bool gemm_bf16_big_ok(int layout, int nprob, const GemmProblem *probs);
// split-K count; k_is_rows: a weight gradient (K = vertices, few output tiles)
int gemm_pick_split(int nprob, const GemmProblem *probs, bool k_is_rows);
// row tiles of a float32 product with M rows (the rows of colpart)
int32_t gemm_colpart_rows(int32_t M);

// elementwise / reductions ----------------------------------------------------
// dZ = dY * [Y > thr] (thr = 0, or kBf16ReluThreshold on the bfloat16 path);
// columns [0,h) -> outS (ldS), [h,2h) -> outN (ldN);
// optional bf16 copies of the same values (outS16/outN16, same leading dims).
// dbias[c] = sum_i dZ[i, c] in a fixed order.
size_t relu_bwd_workspace_bytes(int32_t n, int32_t h);
// The bfloat16 path takes the ReLU derivative on the bfloat16-rounded layer
// output (the operand the next layer reads): bf16_rne(y) > 0 exactly when
// y > 2^-134, half the smallest bfloat16 subnormal (the tie rounds to 0).
constexpr float kBf16ReluThreshold = 0x1p-134f;
int relu_bwd(int32_t n, int32_t h, const float *dY, int64_t lddy, const float *Y, int64_t ldy,
             float *outS, int64_t ldS, float *outN, int64_t ldN,
             uint16_t *outS16, uint16_t *outN16, float *dbias,
             void *ws, size_t ws_bytes, hipStream_t s, float thr = 0.0f);
// out[c] = sum over r < rows of part[r * C + c], in a fixed order
int colsum_reduce_rows(int32_t rows, int32_t C, const float *part, float *out, hipStream_t s);
// column sums of an n x C matrix, fixed order
size_t colsum_workspace_bytes(int32_t n, int32_t C);
int colsum(int32_t n, int32_t C, const float *G, int64_t ldg, float *out, void *ws, size_t ws_bytes,
           hipStream_t s);
// Row-wise loss on logits X (n x C, ldx == C), in place: X <- G.  rowloss[n].
int loss_rows(int kind, int32_t n, int32_t C, float *X, const int32_t *labels, const float *targets,
              float *rowloss, hipStream_t s);
// The head for up to 128 classes in two launches: G in place of X, or, when
// G16 is given, only G's class-padded bfloat16 rows G16 (X is then left as
// the logits); the loss and db = sum_i G[i, :]
bool loss_fused_ok(int32_t C);
size_t loss_fused_workspace_bytes(int32_t n, int32_t C);
int loss_fused(int kind, int32_t n, int32_t C, float *X, const int32_t *labels, const float *targets,
               double scale, float *loss, float *db, uint16_t *G16, int32_t Cp, void *ws, size_t ws_bytes,
               hipStream_t s);
size_t loss_reduce_workspace_bytes(int32_t n);
int loss_reduce(int32_t n, const float *rowloss, double scale, float *loss, void *ws, size_t ws_bytes,
                hipStream_t s);
// x[0..count) = 0 with a kernel (no memset nodes, so callers may capture it)
int fill_zero(float *x, int64_t count, hipStream_t s);
// dst (cols x rows, ldd) = bf16 of src (rows x cols, lds) transposed; src is
// float32 or (src_is_bf16) bfloat16 bits
int transpose_bf16(int64_t rows, int64_t cols, const void *src, int src_is_bf16, int64_t lds, uint16_t *dst,
                   int64_t ldd, hipStream_t s);
// the same, and (copy non-null) the untransposed bfloat16 rows into copy (ldc)
int transpose_bf16_copy(int64_t rows, int64_t cols, const void *src, int src_is_bf16, int64_t lds, uint16_t *dst,
                        int64_t ldd, uint16_t *copy, int64_t ldc, hipStream_t s);
// float32 -> bfloat16 bits (RNE), 2-D with leading dimensions
// A batch of small float32 -> bfloat16 conversions (plain, zero-padded to
// dcols columns, or transposed) in one launch
struct Bf16PrepJob {
    const float *src;
    int64_t lds;
    uint16_t *dst;
    int64_t ldd;
    int32_t rows, cols;    // of src
    int32_t dcols;         // plain: columns written per row (cols .. dcols-1 zero)
    int32_t transpose;     // 1: dst (cols x rows) = bf16(src)^T
    int32_t tiles_c;       // set by prep_bf16
    int64_t first_block;   // set by prep_bf16
};
constexpr int kPrepMaxJobs = 16;
struct Bf16PrepBatch {
    Bf16PrepJob job[kPrepMaxJobs];
    int32_t njobs = 0;
    void add(const float *src, int64_t lds, int32_t rows, int32_t cols, uint16_t *dst, int64_t ldd, int32_t dcols,
             bool transpose) {
        Bf16PrepJob &J = job[njobs++];
        J.src = src;
        J.lds = lds;
        J.dst = dst;
        J.ldd = ldd;
        J.rows = rows;
        J.cols = cols;
        J.dcols = dcols;
        J.transpose = transpose ? 1 : 0;
        J.tiles_c = 0;
        J.first_block = 0;
    }
};
int prep_bf16(Bf16PrepBatch &b, hipStream_t s);
int cvt_bf16(int64_t rows, int64_t cols, const float *x, int64_t ldx, uint16_t *y, int64_t ldy,
             hipStream_t s);
// the same, and columns cols .. ycols-1 of y set to zero (K padding)
int cvt_bf16_pad(int64_t rows, int64_t cols, const float *x, int64_t ldx, uint16_t *y, int64_t ldy,
                 int64_t ycols, hipStream_t s);

// CSR transpose --------------------------------------------------------------
// values of A^T for a symmetric pattern (A^T shares A's indptr / indices)
size_t transpose_symmetric_workspace_bytes(int32_t n, int32_t nnz);
// device-side CSR content check; status: 8-byte aligned int32[2]
int csr_validate_device(int32_t n_rows, int32_t n_cols, int32_t nnz, const int32_t *indptr,
                        IdxRef indices, int sorted, int32_t *status, hipStream_t s);
int csr_transpose_symmetric(int32_t n, int32_t nnz, const int32_t *indptr, IdxRef indices,
                            const float *vals, float *t_vals, void *ws, size_t ws_bytes, hipStream_t s);
size_t transpose_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz);
int csr_transpose(int32_t n_rows, int32_t n_cols, int32_t nnz, const int32_t *indptr,
                  IdxRef indices, const float *vals, int32_t *t_indptr, int32_t *t_indices,
                  float *t_vals, void *ws, size_t ws_bytes, hipStream_t s);

}  // namespace gcn
