/*
 * gcn_layer.h -- C ABI of the MI355X (gfx950) library for the feature
 * propagation hot path of graph-sampling GCN training (Zeng et al.,
 * "Accurate, Efficient and Scalable Graph Embedding", arXiv 1810.11899).
 *
 * The layer (Sec. II; Alg. 1, forward loop; concat self-first, bias, ReLU):
 *
 *     AGG = A H                       mean of the in-neighbour features
 *     Z   = [ H W_self || AGG W_neigh ] + b
 *     Y   = max(Z, 0)
 *
 * and its backward pass (Sec. III-B: the same two kernels, transposed), plus
 * the linear PREDICT head and LOSS of Alg. 1 that drive it.
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer owned by the caller, unless the
 *     name says _host.  Dense matrices are row-major with an explicit leading
 *     dimension (in elements, >= the row width).  Floating point at the
 *     boundary is IEEE float32 for both precisions.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Calls only enqueue work on it; outputs are valid once it is synchronised.
 *   - The library allocates no device memory on any of these paths: scratch
 *     comes from the caller's workspace `ws` of `ws_bytes` bytes (or, for
 *     gcn_aggregate_noalloc, a static array), sized by the
 *     matching *_workspace_bytes query (any 256-byte aligned region at least
 *     that large).  Workspace contents need not be initialised and are
 *     clobbered.
 *   - Argument, shape and workspace checks run on the host before any launch.
 *     A failing call returns a negative gcn_status, launches nothing, and
 *     leaves a message for gcn_last_error() (thread-local).  HIP launch or
 *     runtime failures return GCN_EHIP.
 *   - Results are deterministic: the same inputs on the same device give
 *     bitwise identical outputs (no floating-point atomics; every reduction
 *     runs in a fixed order).
 *   - The library is reentrant: it keeps no device state between calls
 *     (the one exception, gcn_aggregate_noalloc, keeps its scratch in a
 *     static device array and says so).  Calls that share a workspace must
 *     be ordered on one stream.
 */
#ifndef GCN_LAYER_H_
#define GCN_LAYER_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GCN_OK = 0,
    GCN_EINVAL = -1,        /* null pointer, bad enum, malformed CSR (validators) */
    GCN_ESHAPE = -2,        /* inconsistent sizes or leading dimensions           */
    GCN_EWORKSPACE = -3,    /* workspace or saved buffer too small / misaligned   */
    GCN_EHIP = -4,          /* a HIP runtime call or kernel launch failed         */
    GCN_EUNSUPPORTED = -5   /* valid request that the library does not implement */
} gcn_status;

/* Arithmetic of the dense transforms and the gather.
 * GCN_F32 : float32 operands, float32 accumulation.
 * GCN_BF16: operands rounded to bfloat16 (round-to-nearest-even), float32
 *           accumulation; inputs and outputs at the boundary stay float32.
 *           The ReLU derivative is taken on the bfloat16-rounded layer
 *           output, the operand the next layer reads: dZ = dY * [bf16(Y) > 0],
 *           which is dY * [Y > 2^-134] (it drops only outputs below half the
 *           smallest bfloat16 subnormal).  */
typedef enum { GCN_F32 = 0, GCN_BF16 = 1 } gcn_prec;

/* Grouping of the neighbour branch, (A H) W_neigh vs A (H W_neigh).  Equal in
 * exact arithmetic (Alg. 1 writes the first); the second aggregates at width
 * h instead of f_in.  The same order must be passed to fwd and bwd. */
typedef enum { GCN_AGGREGATE_FIRST = 0, GCN_TRANSFORM_FIRST = 1 } gcn_order;

typedef enum { GCN_SOFTMAX_CE = 0, GCN_SIGMOID_BCE = 1 } gcn_loss_kind;

/* Sparse aggregation matrix A in CSR (Sec. V-B streams neighbour lists in this
 * format).  Row i = destination vertex i; its entries are the source vertices
 * j with weight vals[p] (for the mean of Sec. II, vals[p] = 1/deg(i)).
 *   indptr   [n_rows+1], indptr[0] = 0, non-decreasing, indptr[n_rows] = nnz
 *   indices  [nnz] int32 in [0, n_cols), or
 *   indices16[nnz] uint16 in [0, n_cols) for n_cols <= 65,536: the column
 *            indices in half the bytes (the paper's subgraphs use 16-bit
 *            indices, Sec. V-B); exactly one of the two is set when nnz > 0
 *            (the other NULL), and every entry point that takes the CSR reads
 *            either, with the same results bit for bit
 *   vals     [nnz]
 * 0 <= nnz < 2^31.  Duplicated (i, j) entries add up.  Content is NOT checked
 * on the hot path; see gcn_csr_validate_host.  A struct initialised with the
 * first six fields only has indices16 = NULL (int32 indices). */
typedef struct {
    int32_t n_rows;
    int32_t n_cols;
    int32_t nnz;
    const int32_t *indptr;
    const int32_t *indices;
    const float *vals;
    const uint16_t *indices16;
} gcn_csr;

/* Message for the last non-OK return on this thread ("" if none). */
const char *gcn_last_error(void);

/* Library ABI version (major*10000 + minor*100 + patch). */
int gcn_version(void);

/* Host-side structural check of a CSR held in HOST memory: indptr starts at 0,
 * is non-decreasing and ends at nnz; every index is in [0, n_cols); indices
 * are strictly ascending within each row when `require_sorted` is non-zero.
 * Returns GCN_OK or GCN_EINVAL (message names the first offending row). */
int gcn_csr_validate_host(int32_t n_rows, int32_t n_cols, int32_t nnz,
                          const int32_t *indptr_host, const int32_t *indices_host,
                          int require_sorted);

/* The same checks on a CSR held in DEVICE memory, enqueued on `stream`; for
 * callers whose graphs never visit the host (the sampled subgraphs of
 * gcn_induce_subgraphs).  Writes status[0] = 0 if the CSR is valid, else the
 * kind of the first violation in row order (1 indptr[0] != 0 or
 * indptr[n_rows] != nnz, checked before the rows; 2 indptr decreases at row
 * status[1]; 3 an index outside [0, n_cols) in row status[1]; 4 row status[1]
 * not strictly ascending, with require_sorted), and status[1] = that row (0 or
 * n_rows for the endpoints).  status: device int32[2], 8-byte aligned, valid
 * after the stream is synchronized.  Rows whose indptr bounds leave [0, nnz]
 * are not read (a decrease or an endpoint violation is then reported).
 * Returns GCN_EINVAL for null or misaligned arguments, before any launch. */
int gcn_csr_validate(const gcn_csr *A, int require_sorted, int32_t *status, void *stream);

/* ---------------------------------------------------------------- a0 ----
 * CSR of A^T, the transposed aggregation used by the backward propagation
 * (Alg. 1 propagates with the transpose of the bi-adjacency matrix; the
 * backward pass of Sec. III-B applies the other orientation).
 * Output: t_indptr[n_cols+1], t_indices[nnz] (int32 for either index width of
 * A), t_vals[nnz]; row j of A^T holds
 * the rows i of A that contain column j, in ascending i (equal entries keep
 * their CSR order), with the values copied bit for bit.  The integer output is
 * unique, so it is bit-exact against any correct transpose. */
size_t gcn_csr_transpose_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz);
int gcn_csr_transpose(const gcn_csr *A, int32_t *t_indptr, int32_t *t_indices, float *t_vals,
                      void *ws, size_t ws_bytes, void *stream);

/* The same transpose for a square A whose pattern is symmetric, with strictly
 * ascending rows (gcn_csr_pattern_symmetric_host, gcn_sampler.h, checks it
 * on the host): A^T then has A's indptr and indices, and only its values
 * differ.  Writes t_vals[nnz]: for entry p of row j (column i), the value A
 * holds at (i, j) -- the row's value when all of row i's values are equal (as
 * in the mean aggregation of Sec. II), else found by binary search in row i.
 * Outside this contract, an index outside [0, n) or a missing (i, j) in a row
 * with unequal values gives NaN.  On such input A^T = (A.indptr, A.indices,
 * t_vals) equals the output of gcn_csr_transpose bit for bit.  Undirected
 * graphs (every workload here, and the subgraphs a symmetric training graph
 * induces) have this form. */
size_t gcn_csr_transpose_symmetric_workspace_bytes(int32_t n, int32_t nnz);
int gcn_csr_transpose_symmetric(const gcn_csr *A, float *t_vals, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- a1 ----
 * Feature propagation (the first kernel of Sec. V-A; Sec. V-B, Alg. 6):
 *     out[i, c] = sum_p vals[p] * X[indices[p], c],   c in [0, k)
 * X is n_cols x k (ldx), out is n_rows x k (ldo); out must not overlap X.
 * An empty row gives 0.  In GCN_BF16 the gathered X values are rounded to
 * bfloat16 first (accumulation stays float32). */
size_t gcn_aggregate_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz, int32_t k, gcn_prec prec);
int gcn_aggregate(const gcn_csr *A, const float *X, int32_t k, int32_t ldx,
                  float *out, int32_t ldo, gcn_prec prec,
                  void *ws, size_t ws_bytes, void *stream);

/* --------------------------------------------- a1, no allocation ----
 * For callers that cannot allocate device memory or hand over a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  gcn_aggregate_noalloc computes exactly what gcn_aggregate
 * computes (same arguments without ws / ws_bytes, same kernels, bitwise equal
 * results), with its scratch in one file-scope device array of
 * GCN_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until the
 * process ends.  It allocates nothing: no hipMalloc / hipFree, no allocating
 * library call, and no timing events (gcn_profile_* does not see its
 * launches).  When gcn_aggregate_workspace_bytes(n_rows, n_cols, nnz, k, prec)
 * exceeds the array it returns GCN_EUNSUPPORTED before any launch (float32
 * fits 65,536 rows with 3.3 M edges at k = 512; the bfloat16 copy of X
 * counts too).  Nothing in the array has to start at zero.  Every call on one
 * GPU uses that GPU's array, which keeps the last call's contents: calls that
 * can overlap on one GPU (other streams, other threads) race, and the caller
 * must order them.  The stream's device (the current device for NULL) runs
 * the work. */
#define GCN_NOALLOC_SCRATCH_BYTES (64u << 20)
int gcn_aggregate_noalloc(const gcn_csr *A, const float *X, int32_t k, int32_t ldx,
                          float *out, int32_t ldo, gcn_prec prec, void *stream);

/* ------------------------------------------------------------ a1 - a3 ----
 * Forward of one layer on an n-vertex subgraph (A is n x n):
 *   H [n x f_in] (ldh); W_self, W_neigh [f_in x h] (row-major, leading dim h);
 *   bias [2h]; Y [n x 2h] (ldy): columns [0,h) self branch, [h,2h) neighbour.
 * `saved` (gcn_layer_saved_bytes) receives what bwd needs besides H and Y
 * (AGG for GCN_AGGREGATE_FIRST; bf16 operand copies for GCN_BF16) and must be
 * passed unchanged to gcn_layer_bwd.  Y must not overlap H. */
int gcn_layer_pick_order(int32_t f_in, int32_t h, int need_dH);
size_t gcn_layer_saved_bytes(int32_t n, int32_t f_in, int32_t h, gcn_order order, gcn_prec prec);
size_t gcn_layer_workspace_bytes(int32_t n, int32_t nnz, int32_t f_in, int32_t h,
                                 gcn_order order, gcn_prec prec);
int gcn_layer_fwd(const gcn_csr *A, const float *H, int32_t f_in, int32_t ldh,
                  const float *W_self, const float *W_neigh, const float *bias, int32_t h,
                  float *Y, int32_t ldy, void *saved, size_t saved_bytes,
                  gcn_order order, gcn_prec prec, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------ a6 - a8 ----
 * Backward of the same layer.  AT is gcn_csr_transpose(A).  dY [n x 2h] (lddy)
 * is the gradient of the loss with respect to Y.  Outputs are overwritten:
 *   dZ       = dY * [Y > 0]            (the ReLU derivative is taken as 0 at 0)
 *   dbias    [2h]      = sum_i dZ[i, :]
 *   dW_self  [f_in x h] = H^T dZ[:, :h]
 *   dW_neigh [f_in x h] = (A H)^T dZ[:, h:]
 *   dH       [n x f_in] (lddh) = dZ[:, :h] W_self^T + A^T (dZ[:, h:] W_neigh^T)
 * dH == NULL skips the input gradient (a first layer never needs it).
 * dH must not overlap dY, Y or H. */
int gcn_layer_bwd(const gcn_csr *A, const gcn_csr *AT, const float *H, int32_t f_in, int32_t ldh,
                  const float *W_self, const float *W_neigh, int32_t h,
                  const float *Y, int32_t ldy, const void *saved, size_t saved_bytes,
                  const float *dY, int32_t lddy, float *dH, int32_t lddh,
                  float *dW_self, float *dW_neigh, float *dbias,
                  gcn_order order, gcn_prec prec, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------ a4 - a5 ----
 * PREDICT + LOSS of Alg. 1 and their gradient, for the last layer's output
 * HL [n x f] (ldhl):
 *   X = HL W_pred + b_pred            W_pred [f x C] (leading dim C), b_pred [C]
 *   GCN_SOFTMAX_CE : loss = (1/n) sum_i (logsumexp(X_i) - X[i, labels[i]]),
 *                    labels [n] int32 in [0, C) (out-of-range labels are a
 *                    caller error: their rows contribute garbage)
 *                    G = (softmax(X) - onehot(labels)) / n
 *   GCN_SIGMOID_BCE: loss = (1/(nC)) sum_{i,c} (max(x,0) - x t + log(1 + e^-|x|)),
 *                    targets [n x C] float32 (leading dim C)
 *                    G = (sigmoid(X) - targets) / (nC)
 *   loss [1] (device scalar), dHL = G W_pred^T [n x f] (lddhl),
 *   dW_pred = HL^T G [f x C], db_pred = sum_i G [C].
 * The pointer not used by `kind` may be NULL.  With n = 0 the loss, dW_pred
 * and db_pred are written as 0 (sums over no rows), and HL, dHL, labels and
 * targets may be NULL. */
size_t gcn_loss_workspace_bytes(int32_t n, int32_t f, int32_t C, gcn_prec prec);
int gcn_loss_grad(const float *HL, int32_t n, int32_t f, int32_t ldhl,
                  const float *W_pred, const float *b_pred, int32_t C,
                  gcn_loss_kind kind, const int32_t *labels, const float *targets,
                  float *loss, float *dHL, int32_t lddhl, float *dW_pred, float *db_pred,
                  gcn_prec prec, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------ whole step ----
 * One fwd+bwd step of an L-layer model on one subgraph (Alg. 1: the forward
 * loop, PREDICT, LOSS and the backward pass whose gradients ADAM consumes),
 * as the sequence gcn_layer_fwd (l = 0..L-1), gcn_loss_grad, gcn_layer_bwd
 * (l = L-1..0) with the same meaning for every buffer, in one call: the
 * per-layer buffers are described once (gcn_layer_args) and reused for every
 * subgraph.  Layer l's input is H0 for l = 0 and layer l-1's Y otherwise
 * (f_in of layer l must be 2h of layer l-1); layer l's dH (NULL allowed for
 * l = 0 only) is the output gradient of layer l-1.  With head == NULL the
 * output gradient dY [n x 2h_L] (lddy) is given instead of PREDICT/LOSS.
 * The workspace (gcn_model_workspace_bytes) holds the merge-path row ranges
 * of A and A^T, computed once for all of the step's aggregations, with
 * GCN_BF16 the step's weight matrices as bfloat16 (each in the forms its
 * products read, converted in one launch at the start of the step), and the
 * scratch shared by the calls, which run in order on `stream`.  Errors are
 * those of the calls it makes.
 * Buffers between the calls: head->dHL and the dH of layers 1..L-1 carry the
 * gradient from one call to the next, and their contents on return are
 * unspecified.  The step multiplies such a gradient by the ReLU derivative
 * of the layer that consumes it as the gradient is written (the head's dHL,
 * and a layer's dH when its input-gradient product runs unsplit; with
 * GCN_BF16 the buffer then holds that layer's bfloat16 operand rows), and
 * that layer's bias gradient is summed in the same pass; every other output
 * equals the separate calls' bit for bit, and those bias gradients equal
 * theirs up to the order of the sum.  Layer 0's dH, when given, is the
 * gradient with respect to H0 as in gcn_layer_bwd. */
/* With GCN_BF16 a layer's Y may be NULL when its output gradient arrives
 * masked in bfloat16 form: the last layer under a head, and layer l < L-1
 * when layer l+1's input-gradient product runs unsplit (the products of a
 * subgraph of tens of thousands of vertices do; GCN_EINVAL when not).  The
 * step's product epilogues write every layer's output as bfloat16 rows (and
 * transposed rows) for the next layer and the head anyway; a NULL Y skips the
 * float32 copy, and the output of layer l < L-1 is then readable as the first
 * n x 2h bfloat16 values (leading dim 2h) of layer l+1's saved buffer. */
typedef struct {
    int32_t f_in, h;
    gcn_order order;
    const float *W_self, *W_neigh, *bias;   /* f_in x h (leading dim h), f_in x h, [2h] */
    float *Y;                               /* n x 2h (ldy); NULL allowed, see above */
    int32_t ldy;
    void *saved;                            /* gcn_layer_saved_bytes */
    size_t saved_bytes;
    float *dH;                              /* n x f_in (lddh), NULL for layer 0 */
    int32_t lddh;
    float *dW_self, *dW_neigh, *dbias;      /* f_in x h, f_in x h, [2h] */
} gcn_layer_args;

typedef struct {
    const float *W_pred, *b_pred;           /* 2h_L x C (leading dim C), [C] */
    int32_t C;
    gcn_loss_kind kind;
    const int32_t *labels;                  /* CE: [n] */
    const float *targets;                   /* BCE: n x C */
    float *loss;                            /* [1] */
    float *dHL;                             /* n x 2h_L (lddhl) */
    int32_t lddhl;
    float *dW_pred, *db_pred;               /* 2h_L x C, [C] */
} gcn_head_args;

size_t gcn_model_workspace_bytes(int32_t n, int32_t nnz, int32_t L, const gcn_layer_args *layers,
                                 const gcn_head_args *head, gcn_prec prec);
int gcn_model_step(const gcn_csr *A, const gcn_csr *AT, const float *H0, int32_t ldh0, int32_t L,
                   const gcn_layer_args *layers, const gcn_head_args *head, const float *dY, int32_t lddy,
                   gcn_prec prec, void *ws, size_t ws_bytes, void *stream);

/* float32 -> bfloat16 bits, round to nearest even (NaN stays NaN): the
 * rounding every GCN_BF16 operand goes through.  x and y are device arrays of
 * `count` elements. */
int gcn_f32_to_bf16(const float *x, uint16_t *y, int64_t count, void *stream);

/* ------------------------------------------------------------ timing ----
 * Optional per-kernel timing.  While enabled, every kernel the library
 * launches is bracketed by two hipEvents recorded on the launch stream; the
 * events are read (after the caller has synchronised) by gcn_profile_read,
 * which accumulates per kernel class.  Classes are numbered 0..count-1 with
 * stable names.  Disabled by default; costs two event records per launch.
 * The switch and the accumulated times are process-wide host state (guarded
 * by a lock): while profiling is on, the launches of every thread are
 * counted together, so profile one workload at a time.  This is the one
 * exception to the reentrancy above on the host side. */
int gcn_profile_enable(int on);
int gcn_profile_reset(void);
int gcn_profile_class_count(void);
const char *gcn_profile_class_name(int cls);
/* Totals since the last reset: milliseconds, launches, and the algorithmic
 * work the launches were given (flops for GEMMs, bytes for streaming kernels,
 * both under the per-class model documented with the kernel). */
int gcn_profile_read(int cls, double *ms, int64_t *launches, double *flops, double *bytes);

#ifdef __cplusplus
}
#endif

#endif /* GCN_LAYER_H_ */
