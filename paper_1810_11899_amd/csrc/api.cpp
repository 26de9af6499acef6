// Host side of libgcnlayer: the C ABI of gcn_layer.h.  Validates arguments,
// carves the caller's workspace, picks the kernels and enqueues them on the
// caller's stream.  No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace gcn {

// ------------------------------------------------------------------ errors
static thread_local std::string g_last_error;

void set_error(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

int hip_fail(hipError_t e, const char *what) {
    set_error("HIP error in %s: %s", what, hipGetErrorString(e));
    return GCN_EHIP;
}

// --------------------------------------------------------------- profiling
static const char *kClassNames[K_CLASS_COUNT] = {
    "spmm", "spmm_fixup", "gemm_nn", "gemm_tn", "gemm_nt", "splitk_reduce", "relu_bwd",
    "colsum", "loss_rows", "loss_reduce", "transpose_count", "transpose_scan", "transpose_scatter",
    "transpose_sort", "transpose_final", "cvt_bf16", "gemm_nn_bf16", "gemm_tn_bf16", "gemm_nt_bf16",
    "spmm_bf16", "transpose_bf16", "frontier_sample", "induce_subgraphs", "gather_rows", "adam", "transpose_symmetric",
    "gemm_nt_bf16_big", "gemm_nt_bf16_big_masked", "gemm_tn_bf16_big"};

const char *class_name(int cls) {
    return (cls >= 0 && cls < K_CLASS_COUNT) ? kClassNames[cls] : "";
}

namespace {
struct Record {
    int cls;
    hipEvent_t a, b;
    double flops, bytes;
};
struct Totals {
    double ms = 0.0, flops = 0.0, bytes = 0.0;
    int64_t launches = 0;
};
struct Profiler {
    std::mutex mu;
    bool on = false;
    std::vector<hipEvent_t> pool;
    std::vector<Record> pending;
    Totals tot[K_CLASS_COUNT];

    hipEvent_t get() {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
    int drain() {
        int rc = GCN_OK;
        for (Record &r : pending) {
            float ms = 0.0f;
            hipError_t e = hipEventSynchronize(r.b);
            if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
            if (e != hipSuccess) rc = hip_fail(e, "profiler event");
            Totals &t = tot[r.cls];
            t.ms += ms;
            t.flops += r.flops;
            t.bytes += r.bytes;
            t.launches += 1;
            pool.push_back(r.a);
            pool.push_back(r.b);
        }
        pending.clear();
        return rc;
    }
};
Profiler &prof() {
    static Profiler *p = new Profiler();  // never destroyed: events may outlive static teardown
    return *p;
}
}  // namespace

static thread_local int g_prof_suppress = 0;
ProfSuppress::ProfSuppress() { ++g_prof_suppress; }
ProfSuppress::~ProfSuppress() { --g_prof_suppress; }

ProfScope::ProfScope(int cls, hipStream_t s, double flops, double bytes) : cls_(cls), s_(s), slot_(-1) {
    if (g_prof_suppress) return;
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (!p.on) return;
    Record r{cls, p.get(), p.get(), flops, bytes};
    if (!r.a || !r.b) return;
    if (hipEventRecord(r.a, s) != hipSuccess) return;
    p.pending.push_back(r);
    slot_ = (int)p.pending.size() - 1;
}

ProfScope::~ProfScope() {
    if (slot_ < 0) return;
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (slot_ < (int)p.pending.size()) hipEventRecord(p.pending[slot_].b, s_);
}

}  // namespace gcn

using namespace gcn;

// =================================================================== helpers
namespace {

hipStream_t as_stream(void *s) { return (hipStream_t)s; }

#define REQUIRE(cond, code, ...)       \
    do {                               \
        if (!(cond)) {                 \
            set_error(__VA_ARGS__);    \
            return (code);             \
        }                              \
    } while (0)

int check_csr(const gcn_csr *A, const char *name) {
    REQUIRE(A, GCN_EINVAL, "%s: null CSR", name);
    REQUIRE(A->n_rows >= 0 && A->n_cols >= 0 && A->nnz >= 0, GCN_ESHAPE, "%s: negative size", name);
    REQUIRE(A->n_rows == 0 || A->indptr, GCN_EINVAL, "%s: null indptr", name);
    REQUIRE(!(A->indices && A->indices16), GCN_EINVAL, "%s: both indices and indices16 are set", name);
    REQUIRE(A->nnz == 0 || ((A->indices || A->indices16) && A->vals), GCN_EINVAL, "%s: null indices/vals", name);
    REQUIRE(!A->indices16 || A->n_cols <= 65536, GCN_ESHAPE, "%s: uint16 indices need n_cols <= 65536 (%d)", name,
            A->n_cols);
    return GCN_OK;
}

// ----------------------------------------------------------- layer planning
struct LayerPlan {
    bool need_G;        // backward forms G = A^T dZ_n
    bool bf16;
    size_t fwd_T, fwd_W16, fwd_spmm, fwd_gemm;
    size_t bwd_P, bwd_PT, bwd_D, bwd_DT, bwd_T2, bwd_W16, bwd_relu, bwd_spmm, bwd_gemm, bwd_cp;
    size_t fwd_total, bwd_total, total;
};

// bfloat16 weight gradients straight from the row-major operands the layer
// keeps (H, AGG, dZ, G: n rows): a TN product on the large-tile kernel, whose
// k-major operand tiles are read transposed from LDS.  Then no transposed
// copy of those operands is made.  Otherwise (shapes the large-tile kernel
// does not take) the products run NT on transposed copies.
bool bf16_dw_rowmajor(int32_t n, int32_t f_in, int32_t h) {
    if (n <= 0) return false;
    const void *p = (const void *)(uintptr_t)256;   // stands for 256-byte aligned buffers
    GemmProblem g[2] = {};
    for (int i = 0; i < 2; ++i) {
        g[i].M = f_in;
        g[i].N = h;
        g[i].seg[0] = GemmSeg{p, f_in, p, 2 * (int64_t)h, n};
    }
    return gemm_bf16_big_ok(L_TN, 2, g) && h % 8 == 0;
}

int32_t pad_classes(int32_t C);

// The head's bfloat16 weight gradient dW_pred = HL^T G as a TN product on the
// row-major HL and G (the class-padded bfloat16 rows the head keeps) on the
// large-tile kernel; otherwise NT on transposed copies.
bool head_dw_rowmajor(int32_t n, int32_t f, int32_t C) {
    if (n <= 0) return false;
    const void *p = (const void *)(uintptr_t)256;
    GemmProblem g = {};
    g.M = f;
    g.N = C;
    g.seg[0] = GemmSeg{p, f, p, pad_classes(C), n};
    return gemm_bf16_big_ok(L_TN, 1, &g);
}

bool bwd_uses_G(int order, bool dH, int32_t f_in, int32_t h) {
    return order == GCN_TRANSFORM_FIRST || (dH && h <= f_in);
}

// The input-gradient product of a layer whose backward forms G:
// dH = [dZ_s || G] [W_self || W_neigh]^T, one product with K = 2h.  When it
// runs unsplit, a model step has its epilogue multiply dH by the ReLU
// derivative of the layer below, [H > 0] (H = that layer's output Y), and sum
// the columns of the result: the layer below then receives its dZ and bias
// gradient ready (Sec. III-A's backward pass, with the mask of the layer
// below applied where its input gradient is written).  With bfloat16
// operands the epilogue stores dZ as the bfloat16 rows the layer below
// multiplies with (n x f_in, leading dimension f_in, in the dH buffer).
bool dH_mask_fusable(int32_t n, int32_t f_in, int32_t h, int order, int prec) {
    (void)prec;
    if (n <= 0 || !bwd_uses_G(order, true, f_in, h)) return false;
    GemmProblem d{};
    d.M = n;
    d.N = f_in;
    d.seg[0].K = h;
    d.seg[1].K = h;
    return gemm_pick_split(1, &d, false) == 1;
}

size_t colpart_bytes(int32_t n, int32_t N) { return align256((size_t)gemm_colpart_rows(n) * N * sizeof(float)); }

GemmProblem dw_problem(int32_t f_in, int32_t h, int32_t n) {
    GemmProblem g{};
    g.M = f_in;
    g.N = h;
    g.seg[0].K = n;
    g.seg[0].lda = f_in;
    g.seg[0].ldb = h;
    return g;
}

LayerPlan plan_layer(int32_t n, int32_t nnz, int32_t f_in, int32_t h, int order, bool dH, int prec) {
    LayerPlan p{};
    p.need_G = bwd_uses_G(order, dH, f_in, h);
    p.bf16 = prec == GCN_BF16;
    const size_t E = p.bf16 ? 2 : 4;  // bytes per stored intermediate element
    const size_t W16 = p.bf16 ? 2 * align256((size_t)f_in * h * 2) : 0;
    // bfloat16 products run with both operands contiguous along K: the
    // backward also keeps P^T (and dZ_n^T for aggregate-first with G)
    p.bwd_PT = p.bf16 ? align256((size_t)n * 2 * h * 2) : 0;
    p.bwd_DT = (p.bf16 && p.need_G && order == GCN_AGGREGATE_FIRST) ? align256((size_t)n * h * 2) : 0;
    if (order == GCN_TRANSFORM_FIRST) {
        p.fwd_T = align256((size_t)n * h * E);
        p.fwd_spmm = spmm_workspace_bytes(n, nnz, h);
    } else {
        p.fwd_spmm = spmm_workspace_bytes(n, nnz, f_in);
    }
    p.fwd_W16 = W16;
    // split-K partials of the forward products, when there are too few row
    // tiles to fill the GPU (a few thousand vertices)
    {
        GemmProblem f[2] = {};
        f[0].M = f[1].M = n;
        f[0].N = f[1].N = h;
        f[0].seg[0].K = f[1].seg[0].K = f_in;
        p.fwd_gemm = gemm_workspace_bytes(2, f, gemm_pick_split(2, f, false));
    }
    p.fwd_total = p.fwd_T + p.fwd_W16 + p.fwd_spmm + p.fwd_gemm + 1024;

    p.bwd_P = align256((size_t)n * 2 * h * E);
    if (p.need_G) {
        p.bwd_D = align256((size_t)n * h * E);
        p.bwd_spmm = spmm_workspace_bytes(n, nnz, h);
    }
    if (dH && !p.need_G) {
        p.bwd_T2 = align256((size_t)n * f_in * E);
        p.bwd_spmm = std::max(p.bwd_spmm, spmm_workspace_bytes(n, nnz, f_in));
    }
    p.bwd_W16 = dH ? W16 : 0;
    p.bwd_relu = relu_bwd_workspace_bytes(n, h);
    GemmProblem pr[2] = {dw_problem(f_in, h, n), dw_problem(f_in, h, n)};
    p.bwd_gemm = gemm_workspace_bytes(2, pr, gemm_pick_split(2, pr, true));
    if (p.bf16) {  // weight gradients as NT products
        pr[0].seg[0].lda = n;
        pr[0].seg[0].ldb = n;
        pr[1] = pr[0];
        p.bwd_gemm = gemm_workspace_bytes(2, pr, gemm_pick_split(2, pr, true));
    }
    if (dH) {  // the input-gradient product reuses the weight-gradient partials' region
        // the same problems gcn_layer_bwd forms: with G one product of two
        // K = h segments ([dZ_s || G] [W_self || W_neigh]^T), else two of K = h
        // (the split count depends on the segments' k-tiles)
        GemmProblem d[2] = {};
        d[0].M = d[1].M = n;
        d[0].N = d[1].N = f_in;
        d[0].seg[0].K = d[1].seg[0].K = h;
        if (p.need_G) d[0].seg[1].K = h;
        const int nd = p.need_G ? 1 : 2;
        p.bwd_gemm = std::max(p.bwd_gemm, gemm_workspace_bytes(nd, d, gemm_pick_split(nd, d, false)));
    }
    p.bwd_cp = (dH && dH_mask_fusable(n, f_in, h, order, prec)) ? colpart_bytes(n, f_in) : 0;
    p.bwd_total = p.bwd_P + p.bwd_PT + p.bwd_D + p.bwd_DT + p.bwd_T2 + p.bwd_W16 + p.bwd_relu + p.bwd_spmm +
                  p.bwd_gemm + p.bwd_cp + 3072;
    p.total = std::max(p.fwd_total, p.bwd_total);
    return p;
}

// float32: AGG (aggregate-first only).  bfloat16: H16, H16^T, then AGG16 and
// AGG16^T (aggregate-first), each n x f_in.
size_t saved_bytes(int32_t n, int32_t f_in, int32_t h, int order, int prec) {
    (void)h;
    if (prec == GCN_BF16) {
        const size_t one = align256((size_t)n * f_in * 2);
        return order == GCN_AGGREGATE_FIRST ? 4 * one : 2 * one;
    }
    if (order == GCN_AGGREGATE_FIRST) return align256((size_t)n * f_in * sizeof(float));
    return 0;
}

int check_layer_common(const gcn_csr *A, const float *H, int32_t f_in, int32_t ldh, const float *W_self,
                       const float *W_neigh, int32_t h, int order, int prec, const char *who, bool need_H = true) {
    int rc = check_csr(A, who);
    if (rc) return rc;
    REQUIRE(A->n_rows == A->n_cols, GCN_ESHAPE, "%s: aggregation matrix must be square (%d x %d)", who,
            A->n_rows, A->n_cols);
    REQUIRE(f_in > 0 && h > 0, GCN_ESHAPE, "%s: f_in=%d h=%d must be positive", who, f_in, h);
    REQUIRE(ldh >= f_in, GCN_ESHAPE, "%s: ldh=%d < f_in=%d", who, ldh, f_in);
    REQUIRE(order == GCN_AGGREGATE_FIRST || order == GCN_TRANSFORM_FIRST, GCN_EINVAL, "%s: bad order %d",
            who, order);
    REQUIRE(prec == GCN_F32 || prec == GCN_BF16, GCN_EINVAL, "%s: bad precision %d", who, prec);
    REQUIRE(A->n_rows == 0 || ((H || !need_H) && W_self && W_neigh), GCN_EINVAL, "%s: null H or weights", who);
    return GCN_OK;
}

}  // namespace

// ==================================================================== ABI
extern "C" {

const char *gcn_last_error(void) { return g_last_error.c_str(); }

int gcn_version(void) { return 100; }

int gcn_csr_validate_host(int32_t n_rows, int32_t n_cols, int32_t nnz, const int32_t *indptr,
                          const int32_t *indices, int require_sorted) {
    REQUIRE(n_rows >= 0 && n_cols >= 0 && nnz >= 0, GCN_EINVAL, "csr: negative size");
    REQUIRE(indptr, GCN_EINVAL, "csr: null indptr");
    REQUIRE(nnz == 0 || indices, GCN_EINVAL, "csr: null indices");
    REQUIRE(indptr[0] == 0, GCN_EINVAL, "csr: indptr[0] = %d, expected 0", indptr[0]);
    REQUIRE(indptr[n_rows] == nnz, GCN_EINVAL, "csr: indptr[n_rows] = %d, expected nnz = %d",
            indptr[n_rows], nnz);
    for (int32_t i = 0; i < n_rows; ++i) {
        const int32_t b = indptr[i], e = indptr[i + 1];
        REQUIRE(b <= e, GCN_EINVAL, "csr: indptr decreases at row %d", i);
        for (int32_t p = b; p < e; ++p) {
            REQUIRE(indices[p] >= 0 && indices[p] < n_cols, GCN_EINVAL,
                    "csr: row %d holds column %d outside [0, %d)", i, indices[p], n_cols);
            if (require_sorted && p > b)
                REQUIRE(indices[p] > indices[p - 1], GCN_EINVAL,
                        "csr: row %d is not strictly ascending at entry %d", i, p);
        }
    }
    return GCN_OK;
}

int gcn_csr_validate(const gcn_csr *A, int require_sorted, int32_t *status, void *stream) {
    REQUIRE(A && status, GCN_EINVAL, "gcn_csr_validate: null argument");
    REQUIRE(A->n_rows >= 0 && A->n_cols >= 0 && A->nnz >= 0, GCN_EINVAL, "gcn_csr_validate: negative size");
    REQUIRE(A->indptr && (A->nnz == 0 || A->indices || A->indices16), GCN_EINVAL,
            "gcn_csr_validate: null indptr or indices");
    REQUIRE(!(A->indices && A->indices16), GCN_EINVAL, "gcn_csr_validate: both indices and indices16 are set");
    REQUIRE(((uintptr_t)status & 7u) == 0, GCN_EINVAL, "gcn_csr_validate: status must be 8-byte aligned");
    return csr_validate_device(A->n_rows, A->n_cols, A->nnz, A->indptr, idx_of(A), require_sorted != 0, status,
                               as_stream(stream));
}

// -------------------------------------------------------------- transpose
size_t gcn_csr_transpose_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz) {
    return transpose_workspace_bytes(n_rows, n_cols, nnz);
}

int gcn_csr_transpose(const gcn_csr *A, int32_t *t_indptr, int32_t *t_indices, float *t_vals, void *ws,
                      size_t ws_bytes, void *stream) {
    int rc = check_csr(A, "gcn_csr_transpose");
    if (rc) return rc;
    REQUIRE(t_indptr, GCN_EINVAL, "gcn_csr_transpose: null t_indptr");
    REQUIRE(A->nnz == 0 || (t_indices && t_vals), GCN_EINVAL, "gcn_csr_transpose: null outputs");
    const size_t need = transpose_workspace_bytes(A->n_rows, A->n_cols, A->nnz);
    REQUIRE(A->nnz == 0 || (ws && ws_bytes >= need), GCN_EWORKSPACE,
            "gcn_csr_transpose: workspace %zu < %zu bytes", ws_bytes, need);
    return csr_transpose(A->n_rows, A->n_cols, A->nnz, A->indptr, idx_of(A), A->vals, t_indptr, t_indices,
                         t_vals, ws, ws_bytes, as_stream(stream));
}

// ------------------------------------------------------------- aggregate
size_t gcn_csr_transpose_symmetric_workspace_bytes(int32_t n, int32_t nnz) {
    return (n < 0 || nnz < 0) ? 0 : transpose_symmetric_workspace_bytes(n, nnz);
}

int gcn_csr_transpose_symmetric(const gcn_csr *A, float *t_vals, void *ws, size_t ws_bytes, void *stream) {
    int rc = check_csr(A, "gcn_csr_transpose_symmetric");
    if (rc) return rc;
    REQUIRE(A->n_rows == A->n_cols, GCN_ESHAPE, "gcn_csr_transpose_symmetric: A must be square (%d x %d)",
            A->n_rows, A->n_cols);
    REQUIRE(A->nnz == 0 || t_vals, GCN_EINVAL, "gcn_csr_transpose_symmetric: null t_vals");
    const size_t need = transpose_symmetric_workspace_bytes(A->n_rows, A->nnz);
    REQUIRE(A->nnz == 0 || A->n_rows == 0 || (ws && ws_bytes >= need && ((uintptr_t)ws & 255u) == 0),
            GCN_EWORKSPACE, "gcn_csr_transpose_symmetric: workspace %zu < %zu bytes or misaligned", ws_bytes,
            need);
    return csr_transpose_symmetric(A->n_rows, A->nnz, A->indptr, idx_of(A), A->vals, t_vals, ws, ws_bytes,
                                   (hipStream_t)stream);
}

size_t gcn_aggregate_workspace_bytes(int32_t n_rows, int32_t n_cols, int32_t nnz, int32_t k, gcn_prec prec) {
    return spmm_workspace_bytes(n_rows, nnz, k) +
           (prec == GCN_BF16 ? align256((size_t)n_cols * k * 2) + 256 : 0);
}

int gcn_aggregate(const gcn_csr *A, const float *X, int32_t k, int32_t ldx, float *out, int32_t ldo,
                  gcn_prec prec, void *ws, size_t ws_bytes, void *stream) {
    int rc = check_csr(A, "gcn_aggregate");
    if (rc) return rc;
    REQUIRE(k >= 0 && ldx >= k && ldo >= k, GCN_ESHAPE, "gcn_aggregate: k=%d ldx=%d ldo=%d", k, ldx, ldo);
    REQUIRE(prec == GCN_F32 || prec == GCN_BF16, GCN_EINVAL, "gcn_aggregate: bad precision");
    if (A->n_rows == 0 || k == 0) return GCN_OK;
    REQUIRE(out && (A->nnz == 0 || X), GCN_EINVAL, "gcn_aggregate: null X or out");
    const size_t need = gcn_aggregate_workspace_bytes(A->n_rows, A->n_cols, A->nnz, k, prec);
    REQUIRE(ws && ws_bytes >= need, GCN_EWORKSPACE, "gcn_aggregate: workspace %zu < %zu bytes", ws_bytes,
            need);
    hipStream_t s = as_stream(stream);
    if (prec == GCN_BF16) {
        // the source rows of X are the gathered operand: round them (all n_cols rows)
        Arena ar(ws, ws_bytes);
        uint16_t *X16 = ar.take<uint16_t>((size_t)A->n_cols * k);
        const size_t sw = spmm_workspace_bytes(A->n_rows, A->nnz, k);
        void *w = ar.take<char>(sw);
        int rc = cvt_bf16(A->n_cols, k, X, ldx, X16, k, s);
        if (rc) return rc;
        return spmm_bf16(A->n_rows, A->nnz, A->indptr, idx_of(A), A->vals, X16, k, k, out, ldo, EPI_STORE,
                         nullptr, w, sw, s);
    }
    return spmm_f32(A->n_rows, A->nnz, A->indptr, idx_of(A), A->vals, X, k, ldx, out, ldo, EPI_STORE,
                    nullptr, ws, ws_bytes, s);
}

// ----------------------------------------------------------------- layer
int gcn_layer_pick_order(int32_t f_in, int32_t h, int need_dH) {
    // cheaper total aggregation width: forward at f_in (aggregate-first) or h
    // (transform-first); the backward pass adds min(f_in, h) for the input
    // gradient under aggregate-first, h under transform-first
    if (need_dH) return f_in < h ? GCN_AGGREGATE_FIRST : GCN_TRANSFORM_FIRST;
    return f_in <= 2 * h ? GCN_AGGREGATE_FIRST : GCN_TRANSFORM_FIRST;
}

size_t gcn_layer_saved_bytes(int32_t n, int32_t f_in, int32_t h, gcn_order order, gcn_prec prec) {
    return saved_bytes(n, f_in, h, order, prec);
}

size_t gcn_layer_workspace_bytes(int32_t n, int32_t nnz, int32_t f_in, int32_t h, gcn_order order,
                                 gcn_prec prec) {
    return plan_layer(n, nnz, f_in, h, order, true, prec).total;
}

// Links between the bfloat16 calls of a model step: a layer's product
// epilogues also write its output as the bfloat16 rows and transposed rows
// the next consumer multiplies with (the next layer's input copies in its
// saved buffer, or the head's), and that consumer skips its conversion.
struct Bf16Link {
    bool in_ready = false;        // saved already holds this layer's H16 and H16^T
    uint16_t *out16 = nullptr;    // bf16(Y) rows, n x 2h (leading dim 2h)
    uint16_t *out16T = nullptr;   // bf16(Y)^T, 2h x n (leading dim n)
    const uint16_t *WsT = nullptr, *WnT = nullptr;   // bf16(W_self)^T, bf16(W_neigh)^T, already made
};

// launch == false: the argument checks only, nothing enqueued
static int layer_fwd(bool launch, const gcn_csr *A, const float *H, int32_t f_in, int32_t ldh,
                     const float *W_self, const float *W_neigh, const float *bias, int32_t h, float *Y, int32_t ldy,
                     void *saved, size_t saved_bytes_, gcn_order order, gcn_prec prec, void *ws, size_t ws_bytes,
                     void *stream, const int32_t *bA = nullptr, const Bf16Link &lk = Bf16Link{}) {
    // bA: A's merge-path row ranges (spmm_bounds), or NULL
    // a bfloat16 layer whose input copies are ready does not read H
    int rc = check_layer_common(A, H, f_in, ldh, W_self, W_neigh, h, order, prec, "gcn_layer_fwd",
                                !(prec == GCN_BF16 && lk.in_ready));
    if (rc) return rc;
    const int32_t n = A->n_rows;
    REQUIRE(ldy >= 2 * h, GCN_ESHAPE, "gcn_layer_fwd: ldy=%d < 2h=%d", ldy, 2 * h);
    if (n == 0) return GCN_OK;
    REQUIRE(bias && (Y || (prec == GCN_BF16 && lk.out16)), GCN_EINVAL, "gcn_layer_fwd: null Y or bias");
    REQUIRE(!lk.out16T || lk.out16, GCN_EINVAL, "gcn_layer_fwd: a transposed bfloat16 output needs the rows too");
    const size_t sneed = saved_bytes(n, f_in, h, order, prec);
    REQUIRE(saved_bytes_ >= sneed && (sneed == 0 || saved), GCN_EWORKSPACE,
            "gcn_layer_fwd: saved buffer %zu < %zu bytes", saved_bytes_, sneed);
    const LayerPlan pl = plan_layer(n, A->nnz, f_in, h, order, true, prec);
    REQUIRE(ws && ws_bytes >= pl.fwd_total, GCN_EWORKSPACE, "gcn_layer_fwd: workspace %zu < %zu bytes",
            ws_bytes, pl.fwd_total);
    if (!launch) return GCN_OK;
    hipStream_t s = as_stream(stream);
    Arena ar(ws, ws_bytes);
    const bool bf = prec == GCN_BF16;
    const bool af = order == GCN_AGGREGATE_FIRST;

    if (bf) {
        // bfloat16 operands, every product in NT form (both operands contiguous
        // along K); saved = H16 | H16^T | AGG16 | AGG16^T
        const size_t one = align256((size_t)n * f_in * 2);
        uint16_t *H16 = (uint16_t *)saved;
        uint16_t *H16T = (uint16_t *)((char *)saved + one);
        uint16_t *AGG16 = af ? (uint16_t *)((char *)saved + 2 * one) : nullptr;
        uint16_t *AGG16T = af ? (uint16_t *)((char *)saved + 3 * one) : nullptr;
        uint16_t *WsT = ar.take<uint16_t>((size_t)f_in * h);
        uint16_t *WnT = ar.take<uint16_t>((size_t)f_in * h);
        // H16 (and H16T for the transposed weight-gradient products) in one
        // pass over H, unless the layer below wrote them
        const bool tnw = bf16_dw_rowmajor(n, f_in, h);
        if (!lk.in_ready) {
            rc = tnw ? cvt_bf16(n, f_in, H, ldh, H16, f_in, s) : transpose_bf16_copy(n, f_in, H, 0, ldh, H16T, n, H16, f_in, s);
            if (rc) return rc;
        }
        if (lk.WsT) {
            WsT = const_cast<uint16_t *>(lk.WsT);
            WnT = const_cast<uint16_t *>(lk.WnT);
        } else {
            if ((rc = transpose_bf16(f_in, h, W_self, 0, h, WsT, f_in, s))) return rc;
            if ((rc = transpose_bf16(f_in, h, W_neigh, 0, h, WnT, f_in, s))) return rc;
        }
        GemmProblem g[2] = {};
        g[0].M = g[1].M = n;
        g[0].N = g[1].N = h;
        g[0].seg[0] = GemmSeg{H16, f_in, WsT, f_in, f_in};
        g[0].C = Y;
        g[0].ldc = ldy;
        g[0].bias = bias;
        g[0].relu = 1;
        // the output's bfloat16 rows, per half, from the product epilogue;
        // their transposed copy in one pass over both halves at the end
        auto link_out = [&](GemmProblem &q, int half) {
            if (lk.out16) {
                q.C16 = lk.out16 + (size_t)half * h;
                q.ldc16 = 2 * h;
            }
        };
        auto link_out_t = [&]() {
            return lk.out16T ? transpose_bf16(n, 2 * h, lk.out16, 1, 2 * h, lk.out16T, n, s) : GCN_OK;
        };
        link_out(g[0], 0);
        if (af) {
            void *sw = ar.take<char>(pl.fwd_spmm);
            rc = spmm_bf16(n, A->nnz, A->indptr, idx_of(A), A->vals, H16, f_in, f_in, AGG16, f_in,
                           EPI_STORE_BF16, nullptr, sw, pl.fwd_spmm, s, bA);
            if (rc) return rc;
            if (!tnw && (rc = transpose_bf16(n, f_in, AGG16, 1, f_in, AGG16T, n, s))) return rc;
            g[1].seg[0] = GemmSeg{AGG16, f_in, WnT, f_in, f_in};
            g[1].C = Y ? Y + h : nullptr;   // no float32 copy when Y is NULL
            g[1].ldc = ldy;
            g[1].bias = bias + h;
            g[1].relu = 1;
            link_out(g[1], 1);
            void *gw = pl.fwd_gemm ? ar.take<char>(pl.fwd_gemm) : nullptr;
            rc = gemm(L_NT, 2, g, 1, gemm_pick_split(2, g, false), gw, pl.fwd_gemm, s);
            return rc ? rc : link_out_t();
        }
        uint16_t *T16 = (uint16_t *)ar.take<char>(pl.fwd_T);
        void *sw = ar.take<char>(pl.fwd_spmm);
        g[1].seg[0] = GemmSeg{H16, f_in, WnT, f_in, f_in};
        g[1].C16 = T16;
        g[1].ldc = h;
        void *gw = pl.fwd_gemm ? ar.take<char>(pl.fwd_gemm) : nullptr;
        if ((rc = gemm(L_NT, 2, g, 1, gemm_pick_split(2, g, false), gw, pl.fwd_gemm, s))) return rc;
        // the neighbour half: ReLU(A T + b), and its bfloat16 rows from the
        // same epilogue
        rc = spmm_bf16(n, A->nnz, A->indptr, idx_of(A), A->vals, T16, h, h, Y ? Y + h : nullptr, ldy, EPI_BIAS_RELU,
                       bias + h, sw, pl.fwd_spmm, s, bA, lk.out16 ? lk.out16 + h : nullptr, 2 * h);
        return rc ? rc : link_out_t();
    }

    GemmProblem g[2] = {};
    g[0].M = g[1].M = n;
    g[0].N = g[1].N = h;
    g[0].seg[0] = GemmSeg{H, ldh, W_self, h, f_in};
    g[0].C = Y;
    g[0].ldc = ldy;
    g[0].bias = bias;
    g[0].relu = 1;
    if (af) {
        void *sw = ar.take<char>(pl.fwd_spmm);
        float *AGG = (float *)saved;
        rc = spmm_f32(n, A->nnz, A->indptr, idx_of(A), A->vals, H, f_in, ldh, AGG, f_in, EPI_STORE, nullptr, sw,
                      pl.fwd_spmm, s, bA);
        if (rc) return rc;
        g[1].seg[0] = GemmSeg{AGG, f_in, W_neigh, h, f_in};
        g[1].C = Y + h;
        g[1].ldc = ldy;
        g[1].bias = bias + h;
        g[1].relu = 1;
        void *gw = pl.fwd_gemm ? ar.take<char>(pl.fwd_gemm) : nullptr;
        return gemm(L_NN, 2, g, 0, gemm_pick_split(2, g, false), gw, pl.fwd_gemm, s);
    }
    // transform-first: T = H W_neigh, then the neighbour half of Y = ReLU(A T + b)
    float *T = (float *)ar.take<char>(pl.fwd_T);
    void *sw = ar.take<char>(pl.fwd_spmm);
    g[1].seg[0] = GemmSeg{H, ldh, W_neigh, h, f_in};
    g[1].C = T;
    g[1].ldc = h;
    void *gw = pl.fwd_gemm ? ar.take<char>(pl.fwd_gemm) : nullptr;
    if ((rc = gemm(L_NN, 2, g, 0, gemm_pick_split(2, g, false), gw, pl.fwd_gemm, s))) return rc;
    return spmm_f32(n, A->nnz, A->indptr, idx_of(A), A->vals, T, h, h, Y + h, ldy, EPI_BIAS_RELU, bias + h, sw,
                    pl.fwd_spmm, s, bA);
}

static int layer_bwd(bool launch, const gcn_csr *A, const gcn_csr *AT, const float *H, int32_t f_in,
                     int32_t ldh, const float *W_self, const float *W_neigh, int32_t h, const float *Y, int32_t ldy,
                     const void *saved, size_t saved_bytes_, const float *dY, int32_t lddy, float *dH,
                     int32_t lddh, float *dW_self, float *dW_neigh, float *dbias, gcn_order order, gcn_prec prec,
                     void *ws, size_t ws_bytes, void *stream, bool dz_ready = false,
                     float *below_dbias = nullptr, const int32_t *bAT = nullptr, bool dzT_ready = false,
                     int32_t below_tcols = 0, const uint16_t *Ws16_ready = nullptr,
                     const uint16_t *Wn16_ready = nullptr) {
    // bAT: A^T's merge-path row ranges (spmm_bounds), or NULL
    // dzT_ready (bfloat16, with dz_ready): the producer of dY also wrote
    // dZ^T (2h x n, leading dim n) behind the packed dZ rows in the same
    // buffer, at least its first h rows (all 2h for aggregate-first).
    // below_tcols (bfloat16, with below_dbias): also write the first
    // below_tcols columns of the layer below's dZ transposed, behind its rows
    // in the dH buffer.
    // dz_ready: dY already holds dZ = dY * [Y > 0] (float32 with leading
    // dimension lddy, or bfloat16 n x 2h with leading dimension 2h) and dbias
    // is already written (by the producer of dY).  below_dbias: write dH
    // multiplied by [H > 0] (bfloat16 n x f_in rows with bfloat16 operands)
    // and its column sums to below_dbias (dH_mask_fusable only).
    // the bfloat16 backward reads H only through its saved bfloat16 copies
    int rc = check_layer_common(A, H, f_in, ldh, W_self, W_neigh, h, order, prec, "gcn_layer_bwd",
                                prec == GCN_F32);
    if (rc) return rc;
    rc = check_csr(AT, "gcn_layer_bwd (transpose)");
    if (rc) return rc;
    const int32_t n = A->n_rows;
    REQUIRE(AT->n_rows == n && AT->n_cols == n && AT->nnz == A->nnz, GCN_ESHAPE,
            "gcn_layer_bwd: transpose is %d x %d with %d entries, expected %d x %d with %d", AT->n_rows,
            AT->n_cols, AT->nnz, n, n, A->nnz);
    REQUIRE(ldy >= 2 * h && lddy >= 2 * h, GCN_ESHAPE, "gcn_layer_bwd: ldy=%d lddy=%d < 2h=%d", ldy, lddy,
            2 * h);
    REQUIRE(!dH || lddh >= f_in, GCN_ESHAPE, "gcn_layer_bwd: lddh=%d < f_in=%d", lddh, f_in);
    REQUIRE(dW_self && dW_neigh && dbias, GCN_EINVAL, "gcn_layer_bwd: null weight/bias gradient");
    REQUIRE(n == 0 || ((Y || dz_ready) && dY), GCN_EINVAL,
            "gcn_layer_bwd: null Y or dY (Y may be NULL only when the output gradient arrives masked)");
    const size_t sneed = saved_bytes(n, f_in, h, order, prec);
    REQUIRE(saved_bytes_ >= sneed && (sneed == 0 || saved), GCN_EWORKSPACE,
            "gcn_layer_bwd: saved buffer %zu < %zu bytes", saved_bytes_, sneed);
    const bool want_dH = dH != nullptr;
    REQUIRE(!dz_ready || n > 0, GCN_EINVAL, "gcn_layer_bwd: masked dY needs n > 0");
    REQUIRE(!below_dbias || (want_dH && dH_mask_fusable(n, f_in, h, order, prec)), GCN_EINVAL,
            "gcn_layer_bwd: the masked input gradient needs an unsplit product");
    const LayerPlan pl = plan_layer(n, A->nnz, f_in, h, order, want_dH, prec);
    REQUIRE(ws && ws_bytes >= pl.bwd_total, GCN_EWORKSPACE, "gcn_layer_bwd: workspace %zu < %zu bytes",
            ws_bytes, pl.bwd_total);
    if (!launch) return GCN_OK;
    hipStream_t s = as_stream(stream);
    Arena ar(ws, ws_bytes);
    const bool bf = prec == GCN_BF16;
    const bool af = order == GCN_AGGREGATE_FIRST;
    const size_t E = bf ? 2 : 4;
    char *P = ar.take<char>(pl.bwd_P);                      // [dZ_s || G or dZ_n], n x 2h
    char *D = pl.need_G ? ar.take<char>(pl.bwd_D) : nullptr;  // dZ_n, n x h
    char *T2 = (want_dH && !pl.need_G) ? ar.take<char>(pl.bwd_T2) : nullptr;
    uint16_t *Ws16 = pl.bwd_W16 ? ar.take<uint16_t>((size_t)f_in * h) : nullptr;
    uint16_t *Wn16 = pl.bwd_W16 ? ar.take<uint16_t>((size_t)f_in * h) : nullptr;
    void *rw = ar.take<char>(pl.bwd_relu);
    void *sw = pl.bwd_spmm ? ar.take<char>(pl.bwd_spmm) : nullptr;
    void *gw = pl.bwd_gemm ? ar.take<char>(pl.bwd_gemm) : nullptr;
    float *cp = pl.bwd_cp ? ar.take<float>(pl.bwd_cp / sizeof(float)) : nullptr;
    const int64_t ldP = 2 * (int64_t)h;
    char *Pn = P + (size_t)h * E;                              // second half of P
    // where dZ_s, dZ_n and G = A^T dZ_n live: in the workspace, or, with dZ
    // given, dZ in dY and G at the start of P
    const char *Zs = dz_ready ? (const char *)dY : P;
    const int64_t ldZs = dz_ready ? (bf ? ldP : lddy) : ldP;
    char *ZnW = pl.need_G ? D : Pn;
    const char *Zn = dz_ready ? Zs + (size_t)h * E : ZnW;
    const int64_t ldZn = dz_ready ? ldZs : (pl.need_G ? h : ldP);
    char *Gp = dz_ready ? P : Pn;
    const int64_t ldG = dz_ready ? h : ldP;

    // a6: dZ = dY * [Y > 0] and dbias
    if (!dz_ready) {
        if (bf)
            rc = relu_bwd(n, h, dY, lddy, Y, ldy, nullptr, ldP, nullptr, ldZn, (uint16_t *)P, (uint16_t *)ZnW,
                          dbias, rw, pl.bwd_relu, s, kBf16ReluThreshold);
        else
            rc = relu_bwd(n, h, dY, lddy, Y, ldy, (float *)P, ldP, (float *)ZnW, ldZn, nullptr, nullptr, dbias, rw,
                          pl.bwd_relu, s);
        if (rc) return rc;
    }
    if (n == 0) {
        rc = fill_zero(dW_self, (int64_t)f_in * h, s);
        return rc ? rc : fill_zero(dW_neigh, (int64_t)f_in * h, s);
    }
    // G = A^T dZ_n into the second half of P
    if (pl.need_G) {
        rc = bf ? spmm_bf16(AT->n_rows, AT->nnz, AT->indptr, idx_of(AT), AT->vals, (const uint16_t *)Zn, h, ldZn,
                            Gp, ldG, EPI_STORE_BF16, nullptr, sw, pl.bwd_spmm, s, bAT)
                : spmm_f32(AT->n_rows, AT->nnz, AT->indptr, idx_of(AT), AT->vals, (const float *)Zn, h, ldZn, Gp,
                           ldG, EPI_STORE, nullptr, sw, pl.bwd_spmm, s, bAT);
        if (rc) return rc;
    }
    // a7: weight gradients, K = n, split-K
    GemmProblem g[2] = {dw_problem(f_in, h, n), dw_problem(f_in, h, n)};
    int layout = L_TN;
    if (bf && bf16_dw_rowmajor(n, f_in, h)) {
        // TN form on the row-major operands: dW_self = H^T dZ_s, dW_neigh =
        // AGG^T dZ_n (aggregate-first) or H^T G (transform-first)
        const size_t one = align256((size_t)n * f_in * 2);
        const uint16_t *H16 = (const uint16_t *)saved;
        layout = L_TN;
        g[0].seg[0] = GemmSeg{H16, f_in, Zs, ldZs, n};
        if (!af) g[1].seg[0] = GemmSeg{H16, f_in, Gp, ldG, n};
        else g[1].seg[0] = GemmSeg{(const char *)saved + 2 * one, f_in, Zn, ldZn, n};
    } else if (bf) {
        // NT form: dW = (H^T) (P^T)^T with H^T (f_in x n) and P^T (2h x n) contiguous along n
        const size_t one = align256((size_t)n * f_in * 2);
        const uint16_t *H16T = (const uint16_t *)((const char *)saved + one);
        const uint16_t *AGG16T = af ? (const uint16_t *)((const char *)saved + 3 * one) : nullptr;
        uint16_t *PT = (uint16_t *)ar.take<char>(pl.bwd_PT);
        uint16_t *DT = pl.bwd_DT ? (uint16_t *)ar.take<char>(pl.bwd_DT) : nullptr;
        if (dz_ready && dzT_ready) PT = (uint16_t *)const_cast<float *>(dY) + (size_t)n * 2 * h;
        if (!dz_ready) {
            if ((rc = transpose_bf16(n, 2 * h, P, 1, ldP, PT, n, s))) return rc;
            if (DT && (rc = transpose_bf16(n, h, D, 1, h, DT, n, s))) return rc;
        } else if (af) {   // PT = [dZ_s || dZ_n]^T
            if (!dzT_ready && (rc = transpose_bf16(n, 2 * h, Zs, 1, ldZs, PT, n, s))) return rc;
            DT = nullptr;
        } else {           // PT = [dZ_s || G]^T
            if (!dzT_ready && (rc = transpose_bf16(n, h, Zs, 1, ldZs, PT, n, s))) return rc;
            if ((rc = transpose_bf16(n, h, Gp, 1, ldG, PT + (size_t)h * n, n, s))) return rc;
        }
        layout = L_NT;
        g[0].seg[0] = GemmSeg{H16T, n, PT, n, n};
        if (!af) g[1].seg[0] = GemmSeg{H16T, n, PT + (size_t)h * n, n, n};
        else g[1].seg[0] = GemmSeg{AGG16T, n, DT ? DT : PT + (size_t)h * n, n, n};
    } else {
        g[0].seg[0] = GemmSeg{H, ldh, Zs, ldZs, n};
        if (!af)
            g[1].seg[0] = GemmSeg{H, ldh, Gp, ldG, n};                 // H^T (A^T dZ_n)
        else
            g[1].seg[0] = GemmSeg{saved, f_in, Zn, ldZn, n};           // AGG^T dZ_n
    }
    g[0].C = dW_self;
    g[0].ldc = h;
    g[1].C = dW_neigh;
    g[1].ldc = h;
    const int split = gemm_pick_split(2, g, true);
    if ((rc = gemm(layout, 2, g, bf, split, gw, pl.bwd_gemm, s))) return rc;
    if (!want_dH) return GCN_OK;
    // a8: input gradient
    const void *Wsop = W_self, *Wnop = W_neigh;
    if (bf) {
        if (Ws16_ready) {   // the model step converted the weights up front
            Wsop = Ws16_ready;
            Wnop = Wn16_ready;
        } else {
            if ((rc = cvt_bf16(f_in, h, W_self, h, Ws16, h, s))) return rc;
            if ((rc = cvt_bf16(f_in, h, W_neigh, h, Wn16, h, s))) return rc;
            Wsop = Ws16;
            Wnop = Wn16;
        }
    }
    if (pl.need_G) {
        GemmProblem d{};
        d.M = n;
        d.N = f_in;
        d.seg[0] = GemmSeg{Zs, ldZs, Wsop, h, h};
        d.seg[1] = GemmSeg{Gp, ldG, Wnop, h, h};
        d.C = dH;
        d.ldc = lddh;
        if (below_dbias) {  // dZ of the layer below, and its bias gradient
            d.colpart = cp;
            if (bf) {
                // the layer's bfloat16 input rows (saved by the forward pass)
                // are the mask: [bf16(H) > 0] is the relu_bwd rule of the
                // bfloat16 path, [H > 2^-134]
                d.mask16 = (const uint16_t *)saved;
                d.ldm = f_in;
                d.C = nullptr;
                d.C16 = (uint16_t *)dH;
                d.ldc = f_in;
                if (below_tcols > 0) {   // and its transposed rows behind them
                    d.C16T = (uint16_t *)dH + (size_t)n * f_in;
                    d.ldc16t = n;
                    d.n16t = below_tcols;
                }
            } else {
                d.mask = H;
                d.ldm = ldh;
            }
        }
        if ((rc = gemm(L_NT, 1, &d, bf, gemm_pick_split(1, &d, false), gw, pl.bwd_gemm, s))) return rc;
        return below_dbias ? colsum_reduce_rows(gemm_colpart_rows(n), f_in, cp, below_dbias, s) : GCN_OK;
    }
    GemmProblem d[2] = {};
    d[0].M = d[1].M = n;
    d[0].N = d[1].N = f_in;
    d[0].seg[0] = GemmSeg{Zs, ldZs, Wsop, h, h};
    d[0].C = dH;
    d[0].ldc = lddh;
    d[1].seg[0] = GemmSeg{Zn, ldZn, Wnop, h, h};
    d[1].ldc = f_in;
    if (bf) d[1].C16 = (uint16_t *)T2;
    else d[1].C = (float *)T2;
    if ((rc = gemm(L_NT, 2, d, bf, gemm_pick_split(2, d, false), gw, pl.bwd_gemm, s))) return rc;
    return bf ? spmm_bf16(AT->n_rows, AT->nnz, AT->indptr, idx_of(AT), AT->vals, (const uint16_t *)T2, f_in,
                          f_in, dH, lddh, EPI_ACCUMULATE, nullptr, sw, pl.bwd_spmm, s, bAT)
              : spmm_f32(AT->n_rows, AT->nnz, AT->indptr, idx_of(AT), AT->vals, (const float *)T2, f_in, f_in,
                         dH, lddh, EPI_ACCUMULATE, nullptr, sw, pl.bwd_spmm, s, bAT);
}

// ------------------------------------------------------------------ loss
namespace {
struct LossPlan {
    size_t X, rows, HL16, HL16T, Wp16, Wp16T, G16, G16T, gemm, colsum, red, cp, total;
    int split;
};
// bfloat16 class dimension padded with zero columns to a multiple of 32, so
// that dHL = G W_pred^T (K = classes) runs on the large-tile product
int32_t pad_classes(int32_t C) { return (C + 31) / 32 * 32; }

LossPlan plan_loss(int32_t n, int32_t f, int32_t C, int prec) {
    LossPlan p{};
    p.X = align256((size_t)n * C * sizeof(float));
    p.rows = align256((size_t)n * sizeof(float) + 4);
    if (prec == GCN_BF16) {
        const size_t Cp = pad_classes(C);
        p.HL16 = p.HL16T = align256((size_t)n * f * 2);
        p.Wp16 = align256((size_t)f * Cp * 2);
        p.Wp16T = align256((size_t)f * C * 2);
        p.G16 = align256((size_t)n * Cp * 2);
        p.G16T = align256((size_t)n * C * 2);
    }
    GemmProblem g = dw_problem(f, C, n);
    p.split = gemm_pick_split(1, &g, true);
    p.gemm = gemm_workspace_bytes(1, &g, p.split);
    if (loss_fused_ok(C)) {   // the loss and db_pred from the loss kernel's block partials
        p.colsum = 256;
        p.red = loss_fused_workspace_bytes(n, C);
    } else {
        p.colsum = colsum_workspace_bytes(n, C);
        p.red = loss_reduce_workspace_bytes(n);
    }
    p.cp = colpart_bytes(n, f);
    p.total = p.X + p.rows + p.HL16 + p.HL16T + p.Wp16 + p.Wp16T + p.G16 + p.G16T + p.gemm + p.colsum + p.red +
              p.cp + 3584;
    return p;
}
}  // namespace

size_t gcn_loss_workspace_bytes(int32_t n, int32_t f, int32_t C, gcn_prec prec) {
    return plan_loss(n, f, C, prec).total;
}

static int loss_grad(bool launch, const float *HL, int32_t n, int32_t f, int32_t ldhl, const float *W_pred,
                     const float *b_pred, int32_t C, gcn_loss_kind kind, const int32_t *labels,
                     const float *targets, float *loss, float *dHL, int32_t lddhl, float *dW_pred, float *db_pred,
                     gcn_prec prec, void *ws, size_t ws_bytes, void *stream, float *below_dbias = nullptr,
                     const uint16_t *HL16_ready = nullptr, const uint16_t *HL16T_ready = nullptr,
                     int32_t below_tcols = 0, const uint16_t *Wp16_ready = nullptr,
                     const uint16_t *Wp16T_ready = nullptr) {
    // HL16_ready / HL16T_ready (bfloat16): HL's bfloat16 rows and transposed
    // rows, already written by the last layer's epilogues.  below_tcols (with
    // below_dbias): also write the first below_tcols columns of the last
    // layer's dZ transposed, behind its rows in the dHL buffer.
    // below_dbias: write dHL multiplied by [HL > 0] (HL is the last layer's
    // ReLU output), i.e. that layer's dZ (bfloat16 n x f rows, leading
    // dimension f, with bfloat16 operands), and its column sums to below_dbias
    REQUIRE(n >= 0 && f > 0 && C > 0, GCN_ESHAPE, "gcn_loss_grad: n=%d f=%d C=%d", n, f, C);
    REQUIRE(!below_dbias || n > 0, GCN_EINVAL, "gcn_loss_grad: the masked gradient needs n > 0");
    REQUIRE(ldhl >= f && lddhl >= f, GCN_ESHAPE, "gcn_loss_grad: ldhl=%d lddhl=%d < f=%d", ldhl, lddhl, f);
    REQUIRE(kind == GCN_SOFTMAX_CE || kind == GCN_SIGMOID_BCE, GCN_EINVAL, "gcn_loss_grad: bad kind %d",
            kind);
    REQUIRE(prec == GCN_F32 || prec == GCN_BF16, GCN_EINVAL, "gcn_loss_grad: bad precision");
    REQUIRE(W_pred && b_pred && loss && dW_pred && db_pred, GCN_EINVAL, "gcn_loss_grad: null pointer");
    REQUIRE(n == 0 || ((HL || HL16_ready) && dHL), GCN_EINVAL, "gcn_loss_grad: null HL or dHL");
    REQUIRE(n == 0 || (kind == GCN_SOFTMAX_CE ? labels != nullptr : targets != nullptr), GCN_EINVAL,
            "gcn_loss_grad: null labels/targets");
    const LossPlan pl = plan_loss(n, f, C, prec);
    REQUIRE(ws && ws_bytes >= pl.total, GCN_EWORKSPACE, "gcn_loss_grad: workspace %zu < %zu bytes", ws_bytes,
            pl.total);
    if (!launch) return GCN_OK;
    hipStream_t s = as_stream(stream);
    Arena ar(ws, ws_bytes);
    const bool bf = prec == GCN_BF16;
    float *X = ar.take<float>((size_t)n * C);
    float *rows = ar.take<float>((size_t)n + 1);
    const uint16_t *HL16 = bf ? ar.take<uint16_t>((size_t)n * f) : nullptr;
    const uint16_t *HL16T = bf ? ar.take<uint16_t>((size_t)n * f) : nullptr;
    if (bf && HL16_ready) {
        HL16 = HL16_ready;
        HL16T = HL16T_ready;
    }
    const bool tn_dw = bf && head_dw_rowmajor(n, f, C);   // dW_pred from the rows: no transposed copies
    REQUIRE(!bf || !HL16_ready || tn_dw || HL16T, GCN_EINVAL, "gcn_loss_grad: transposed HL rows missing");
    const int32_t Cp = pad_classes(C);
    uint16_t *Wp16 = bf ? ar.take<uint16_t>((size_t)f * Cp) : nullptr;
    uint16_t *Wp16T = bf ? ar.take<uint16_t>((size_t)f * C) : nullptr;
    uint16_t *G16 = bf ? ar.take<uint16_t>((size_t)n * Cp) : nullptr;
    uint16_t *G16T = bf ? ar.take<uint16_t>((size_t)n * C) : nullptr;
    void *gw = pl.gemm ? ar.take<char>(pl.gemm) : nullptr;
    void *cw = ar.take<char>(pl.colsum);
    void *lw = ar.take<char>(pl.red);
    float *cp = pl.cp ? ar.take<float>(pl.cp / sizeof(float)) : nullptr;
    int rc;
    if (n == 0) {
        rc = fill_zero(dW_pred, (int64_t)f * C, s);
        if (!rc) rc = fill_zero(db_pred, C, s);
        return rc ? rc : fill_zero(loss, 1, s);
    }
    // a4: logits X = HL W_pred + b_pred
    GemmProblem g{};
    g.M = n;
    g.N = C;
    g.C = X;
    g.ldc = C;
    g.bias = b_pred;
    if (bf) {
        // NT form: B = W_pred^T (C x f)
        if (!HL16_ready &&
            (rc = tn_dw ? cvt_bf16(n, f, HL, ldhl, const_cast<uint16_t *>(HL16), f, s)
                        : transpose_bf16_copy(n, f, HL, 0, ldhl, const_cast<uint16_t *>(HL16T), n,
                                              const_cast<uint16_t *>(HL16), f, s)))
            return rc;
        if (Wp16_ready) {   // the model step converted W_pred up front
            Wp16 = const_cast<uint16_t *>(Wp16_ready);
            Wp16T = const_cast<uint16_t *>(Wp16T_ready);
        } else {
            if ((rc = cvt_bf16_pad(f, C, W_pred, C, Wp16, Cp, Cp, s))) return rc;
            if ((rc = transpose_bf16(f, C, Wp16, 1, Cp, Wp16T, f, s))) return rc;
        }
        g.seg[0] = GemmSeg{HL16, f, Wp16T, f, f};
        rc = gemm(L_NT, 1, &g, 1, 1, nullptr, 0, s);
    } else {
        g.seg[0] = GemmSeg{HL, ldhl, W_pred, C, f};
        rc = gemm(L_NN, 1, &g, 0, 1, nullptr, 0, s);
    }
    if (rc) return rc;
    // row losses, X <- G in place (bfloat16: G's class-padded bfloat16 rows
    // G16 alongside); up to 128 classes the same pass leaves block partials
    // from which one more launch forms the loss and db_pred
    const double scale = kind == GCN_SOFTMAX_CE ? 1.0 / (double)n : 1.0 / ((double)n * (double)C);
    const bool fused = loss_fused_ok(C);
    if (fused) {
        if ((rc = loss_fused(kind, n, C, X, labels, targets, scale, loss, db_pred, G16, Cp, lw, pl.red, s)))
            return rc;
    } else {
        if ((rc = loss_rows(kind, n, C, X, labels, targets, rows, s))) return rc;
        if ((rc = loss_reduce(n, rows, scale, loss, lw, pl.red, s))) return rc;
        if (bf && (rc = cvt_bf16_pad(n, C, X, C, G16, Cp, Cp, s))) return rc;
    }
    // a5: dW_pred = HL^T G, db_pred = sum_i G, dHL = G W_pred^T
    GemmProblem w = dw_problem(f, C, n);
    w.C = dW_pred;
    w.ldc = C;
    GemmProblem d{};
    d.M = n;
    d.N = f;
    d.C = dHL;
    d.ldc = lddhl;
    if (bf) {
        if (tn_dw) {
            w.seg[0] = GemmSeg{HL16, f, G16, Cp, n};
            if ((rc = gemm(L_TN, 1, &w, 1, pl.split, gw, pl.gemm, s))) return rc;
        } else {
            if ((rc = transpose_bf16(n, C, G16, 1, Cp, G16T, n, s))) return rc;
            w.seg[0] = GemmSeg{HL16T, n, G16T, n, n};
            if ((rc = gemm(L_NT, 1, &w, 1, pl.split, gw, pl.gemm, s))) return rc;
        }
        d.seg[0] = GemmSeg{G16, Cp, Wp16, Cp, Cp};   // the zero columns add nothing
        d.k_pad = Cp - C;
    } else {
        w.seg[0] = GemmSeg{HL, ldhl, X, C, n};
        if ((rc = gemm(L_TN, 1, &w, 0, pl.split, gw, pl.gemm, s))) return rc;
        d.seg[0] = GemmSeg{X, C, W_pred, C, C};
    }
    if (!fused && (rc = colsum(n, C, X, C, db_pred, cw, pl.colsum, s))) return rc;
    if (below_dbias) {
        d.colpart = cp;
        if (bf) {
            d.mask16 = HL16;   // [bf16(HL) > 0], as in relu_bwd's bfloat16 rule
            d.ldm = f;
            d.C = nullptr;
            d.C16 = (uint16_t *)dHL;
            d.ldc = f;
            if (below_tcols > 0) {
                d.C16T = (uint16_t *)dHL + (size_t)n * f;
                d.ldc16t = n;
                d.n16t = below_tcols;
            }
        } else {
            d.mask = HL;
            d.ldm = ldhl;
        }
    }
    if ((rc = gemm(L_NT, 1, &d, bf, 1, nullptr, 0, s))) return rc;
    return below_dbias ? colsum_reduce_rows(gemm_colpart_rows(n), f, cp, below_dbias, s) : GCN_OK;
}

// ------------------------------------------------------------------ bf16
int gcn_f32_to_bf16(const float *x, uint16_t *y, int64_t count, void *stream) {
    REQUIRE(count >= 0, GCN_ESHAPE, "gcn_f32_to_bf16: negative count");
    if (count == 0) return GCN_OK;
    REQUIRE(x && y, GCN_EINVAL, "gcn_f32_to_bf16: null pointer");
    return cvt_bf16(1, count, x, count, y, count, as_stream(stream));
}

// ------------------------------------------------------------- profiling
int gcn_profile_enable(int on) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    p.on = on != 0;
    return GCN_OK;
}

int gcn_profile_reset(void) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    int rc = p.drain();
    for (auto &t : p.tot) t = Totals{};
    return rc;
}

int gcn_profile_class_count(void) { return K_CLASS_COUNT; }

const char *gcn_profile_class_name(int cls) { return class_name(cls); }

int gcn_profile_read(int cls, double *ms, int64_t *launches, double *flops, double *bytes) {
    REQUIRE(cls >= 0 && cls < K_CLASS_COUNT, GCN_EINVAL, "gcn_profile_read: class %d", cls);
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    int rc = p.drain();
    const Totals &t = p.tot[cls];
    if (ms) *ms = t.ms;
    if (launches) *launches = t.launches;
    if (flops) *flops = t.flops;
    if (bytes) *bytes = t.bytes;
    return rc;
}

// ------------------------------------------------------------ entry points
int gcn_layer_fwd(const gcn_csr *A, const float *H, int32_t f_in, int32_t ldh, const float *W_self,
                  const float *W_neigh, const float *bias, int32_t h, float *Y, int32_t ldy, void *saved,
                  size_t saved_bytes_, gcn_order order, gcn_prec prec, void *ws, size_t ws_bytes, void *stream) {
    return layer_fwd(true, A, H, f_in, ldh, W_self, W_neigh, bias, h, Y, ldy, saved, saved_bytes_, order, prec,
                     ws, ws_bytes, stream);
}

int gcn_layer_bwd(const gcn_csr *A, const gcn_csr *AT, const float *H, int32_t f_in, int32_t ldh,
                  const float *W_self, const float *W_neigh, int32_t h, const float *Y, int32_t ldy,
                  const void *saved, size_t saved_bytes_, const float *dY, int32_t lddy, float *dH, int32_t lddh,
                  float *dW_self, float *dW_neigh, float *dbias, gcn_order order, gcn_prec prec, void *ws,
                  size_t ws_bytes, void *stream) {
    return layer_bwd(true, A, AT, H, f_in, ldh, W_self, W_neigh, h, Y, ldy, saved, saved_bytes_, dY, lddy, dH,
                     lddh, dW_self, dW_neigh, dbias, order, prec, ws, ws_bytes, stream);
}

int gcn_loss_grad(const float *HL, int32_t n, int32_t f, int32_t ldhl, const float *W_pred, const float *b_pred,
                  int32_t C, gcn_loss_kind kind, const int32_t *labels, const float *targets, float *loss,
                  float *dHL, int32_t lddhl, float *dW_pred, float *db_pred, gcn_prec prec, void *ws,
                  size_t ws_bytes, void *stream) {
    return loss_grad(true, HL, n, f, ldhl, W_pred, b_pred, C, kind, labels, targets, loss, dHL, lddhl, dW_pred,
                     db_pred, prec, ws, ws_bytes, stream);
}

// ------------------------------------------------------------ model step
static size_t model_hl16_bytes(int32_t n, int32_t L, const gcn_layer_args *layers, const gcn_head_args *head,
                               gcn_prec prec) {
    if (prec != GCN_BF16 || !head || n <= 0) return 0;
    return 2 * align256((size_t)n * 2 * layers[L - 1].h * 2);
}

// bfloat16: every weight matrix of the step in the forms its products read
// (W^T for the forward NT products, W for the input-gradient products,
// W_pred zero-padded to the padded classes and transposed), converted in one
// launch at the start of the step
struct ModelW16 {
    const uint16_t *WsT[8] = {}, *WnT[8] = {}, *Ws16[8] = {}, *Wn16[8] = {};
    const uint16_t *Wp16 = nullptr, *Wp16T = nullptr;
};
static size_t model_w16_bytes(int32_t n, int32_t L, const gcn_layer_args *layers, const gcn_head_args *head,
                              gcn_prec prec, Bf16PrepBatch *batch = nullptr, ModelW16 *out = nullptr,
                              char *base = nullptr) {
    if (prec != GCN_BF16 || n <= 0 || L > 8 || 4 * L + 2 > kPrepMaxJobs) return 0;
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        uint16_t *p = base ? (uint16_t *)(base + off) : nullptr;
        off += align256(bytes);
        return p;
    };
    for (int32_t l = 0; l < L; ++l) {
        const gcn_layer_args &a = layers[l];
        const size_t one = (size_t)a.f_in * a.h * 2;
        uint16_t *st = carve(one), *nt = carve(one);
        if (batch) {
            batch->add(a.W_self, a.h, a.f_in, a.h, st, a.f_in, 0, true);
            batch->add(a.W_neigh, a.h, a.f_in, a.h, nt, a.f_in, 0, true);
            out->WsT[l] = st;
            out->WnT[l] = nt;
        }
        if (a.dH) {
            uint16_t *sr = carve(one), *nr = carve(one);
            if (batch) {
                batch->add(a.W_self, a.h, a.f_in, a.h, sr, a.h, a.h, false);
                batch->add(a.W_neigh, a.h, a.f_in, a.h, nr, a.h, a.h, false);
                out->Ws16[l] = sr;
                out->Wn16[l] = nr;
            }
        }
    }
    if (head) {
        const int32_t f = 2 * layers[L - 1].h, C = head->C, Cp = pad_classes(C);
        uint16_t *wp = carve((size_t)f * Cp * 2), *wpt = carve((size_t)f * C * 2);
        if (batch) {
            batch->add(head->W_pred, C, f, C, wp, Cp, Cp, false);
            batch->add(head->W_pred, C, f, C, wpt, f, 0, true);
            out->Wp16 = wp;
            out->Wp16T = wpt;
        }
    }
    return off;
}

size_t gcn_model_workspace_bytes(int32_t n, int32_t nnz, int32_t L, const gcn_layer_args *layers,
                                 const gcn_head_args *head, gcn_prec prec) {
    if (n < 0 || nnz < 0 || L < 1 || !layers) return 0;
    size_t b = 0;
    for (int32_t l = 0; l < L; ++l)
        b = std::max(b, plan_layer(n, nnz, layers[l].f_in, layers[l].h, layers[l].order, true, prec).total);
    if (head) b = std::max(b, plan_loss(n, 2 * layers[L - 1].h, head->C, prec).total);
    // the row ranges of A and A^T, shared by the calls, and with bfloat16
    // operands the last layer's output as the head's bfloat16 rows and
    // transposed rows
    return b + 2 * spmm_bounds_bytes(n, nnz) + model_hl16_bytes(n, L, layers, head, prec) +
           model_w16_bytes(n, L, layers, head, prec);
}

namespace {
// The step's calls in order; with launch == false only their argument checks
// run, so that a bad descriptor is reported before anything is enqueued.
int model_step(bool launch, const gcn_csr *A, const gcn_csr *AT, const float *H0, int32_t ldh0, int32_t L,
               const gcn_layer_args *layers, const gcn_head_args *head, const float *dY, int32_t lddy,
               gcn_prec prec, void *ws, size_t ws_bytes, void *stream) {
    const int32_t n = A->n_rows;
    int rc;
    // the merge-path row ranges of A and A^T, computed once for every SpMM of
    // the step (they depend only on the row pointers; A^T shares A's when it
    // shares A's row pointers), ahead of the calls' workspace
    const size_t rb = spmm_bounds_bytes(n, A->nnz);
    const int32_t *bA = nullptr, *bAT = nullptr;
    if (rb) {
        REQUIRE(ws && ws_bytes >= 2 * rb, GCN_EWORKSPACE, "gcn_model_step: workspace %zu bytes too small",
                ws_bytes);
        int32_t *ra = (int32_t *)ws;
        int32_t *rt = AT->indptr == A->indptr ? ra : (int32_t *)((char *)ws + rb);
        ws = (char *)ws + 2 * rb;
        ws_bytes -= 2 * rb;
        if (launch) {
            hipStream_t s = as_stream(stream);
            if ((rc = spmm_bounds(n, A->nnz, A->indptr, ra, s))) return rc;
            if (rt != ra && (rc = spmm_bounds(n, AT->nnz, AT->indptr, rt, s))) return rc;
        }
        bA = ra;
        bAT = rt;
    }
    // bfloat16: each layer's product epilogues write its output straight into
    // the bfloat16 copies (rows and transposed rows) the next consumer reads:
    // the next layer's saved buffer, or the head's region below
    const bool bf = prec == GCN_BF16;
    uint16_t *HL16 = nullptr, *HL16T = nullptr;
    if (const size_t hb = model_hl16_bytes(n, L, layers, head, prec)) {
        REQUIRE(ws && ws_bytes >= hb, GCN_EWORKSPACE, "gcn_model_step: workspace %zu bytes too small", ws_bytes);
        HL16 = (uint16_t *)ws;
        HL16T = (uint16_t *)((char *)ws + hb / 2);
        ws = (char *)ws + hb;
        ws_bytes -= hb;
    }
    ModelW16 w16;
    if (const size_t wb = model_w16_bytes(n, L, layers, head, prec)) {
        REQUIRE(ws && ws_bytes >= wb, GCN_EWORKSPACE, "gcn_model_step: workspace %zu bytes too small", ws_bytes);
        Bf16PrepBatch batch;
        model_w16_bytes(n, L, layers, head, prec, &batch, &w16, (char *)ws);
        ws = (char *)ws + wb;
        ws_bytes -= wb;
        if (launch && (rc = prep_bf16(batch, as_stream(stream)))) return rc;
    }
    const float *H = H0;  // forward: layer l reads layer l-1's output
    int32_t ldh = ldh0;
    for (int32_t l = 0; l < L; ++l) {
        const gcn_layer_args &a = layers[l];
        Bf16Link lk;
        if (bf && n > 0) {
            lk.in_ready = l > 0;
            if (l + 1 < L) {
                const gcn_layer_args &nx = layers[l + 1];
                lk.out16 = (uint16_t *)nx.saved;
                if (!bf16_dw_rowmajor(n, nx.f_in, nx.h))   // only the transposed products read H16T
                    lk.out16T = (uint16_t *)((char *)nx.saved + align256((size_t)n * nx.f_in * 2));
            } else if (head) {
                lk.out16 = HL16;
                if (!head_dw_rowmajor(n, 2 * a.h, head->C)) lk.out16T = HL16T;   // read by an NT dW_pred only
            }
            lk.WsT = w16.WsT[l];
            lk.WnT = w16.WnT[l];
        }
        if ((rc = layer_fwd(launch, A, H, a.f_in, ldh, a.W_self, a.W_neigh, a.bias, a.h, a.Y, a.ldy, a.saved,
                            a.saved_bytes, a.order, prec, ws, ws_bytes, stream, bA, lk)))
            return rc;
        H = a.Y;
        ldh = a.ldy;
    }
    // columns of a layer's dZ that its backward reads transposed: all 2h for
    // aggregate-first (dW_self and dW_neigh), the self half for
    // transform-first (dW_neigh takes A^T dZ_n, transposed after the SpMM)
    auto tcols = [&](int32_t l) {
        if (!bf || bf16_dw_rowmajor(n, layers[l].f_in, layers[l].h)) return 0;
        return layers[l].order == GCN_AGGREGATE_FIRST ? 2 * layers[l].h : layers[l].h;
    };
    const float *g = dY;  // PREDICT + LOSS, or the given output gradient
    int32_t ldg = lddy;
    // the head, and a layer whose input-gradient product runs unsplit, write
    // the next layer down its dZ and bias gradient directly
    bool ready = false;
    if (head) {
        const gcn_layer_args &last = layers[L - 1];
        const bool fuse = n > 0;
        if ((rc = loss_grad(launch, last.Y, n, 2 * last.h, last.ldy, head->W_pred, head->b_pred, head->C,
                            head->kind, head->labels, head->targets, head->loss, head->dHL, head->lddhl,
                            head->dW_pred, head->db_pred, prec, ws, ws_bytes, stream,
                            fuse ? last.dbias : nullptr, HL16, HL16T, fuse ? tcols(L - 1) : 0, w16.Wp16,
                            w16.Wp16T)))
            return rc;
        g = head->dHL;
        ldg = head->lddhl;
        ready = fuse;
    }
    for (int32_t l = L - 1; l >= 0; --l) {  // backward: layer l's dH is layer l-1's output gradient
        const gcn_layer_args &a = layers[l];
        const float *Hin = l == 0 ? H0 : layers[l - 1].Y;
        const int32_t ldin = l == 0 ? ldh0 : layers[l - 1].ldy;
        const bool fuse = l > 0 && dH_mask_fusable(n, a.f_in, a.h, a.order, prec);
        if ((rc = layer_bwd(launch, A, AT, Hin, a.f_in, ldin, a.W_self, a.W_neigh, a.h, a.Y, a.ldy, a.saved,
                            a.saved_bytes, g, ldg, a.dH, a.lddh, a.dW_self, a.dW_neigh, a.dbias, a.order, prec, ws,
                            ws_bytes, stream, ready, fuse ? layers[l - 1].dbias : nullptr, bAT,
                            ready && tcols(l) > 0, fuse ? tcols(l - 1) : 0, w16.Ws16[l], w16.Wn16[l])))
            return rc;
        g = a.dH;
        ldg = a.lddh;
        ready = fuse;
    }
    return GCN_OK;
}
}  // namespace

int gcn_model_step(const gcn_csr *A, const gcn_csr *AT, const float *H0, int32_t ldh0, int32_t L,
                   const gcn_layer_args *layers, const gcn_head_args *head, const float *dY, int32_t lddy,
                   gcn_prec prec, void *ws, size_t ws_bytes, void *stream) {
    REQUIRE(A && AT && layers && L >= 1, GCN_EINVAL, "gcn_model_step: null argument or L < 1");
    REQUIRE(head || dY, GCN_EINVAL, "gcn_model_step: neither a head nor an output gradient dY");
    for (int32_t l = 1; l < L; ++l) {
        REQUIRE(layers[l].f_in == 2 * layers[l - 1].h, GCN_ESHAPE,
                "gcn_model_step: layer %d takes %d features, layer %d gives %d", l, layers[l].f_in, l - 1,
                2 * layers[l - 1].h);
        REQUIRE(layers[l].dH, GCN_EINVAL, "gcn_model_step: layer %d needs dH (the gradient of layer %d)", l,
                l - 1);
    }
    int rc = model_step(false, A, AT, H0, ldh0, L, layers, head, dY, lddy, prec, ws, ws_bytes, stream);
    return rc ? rc : model_step(true, A, AT, H0, ldh0, L, layers, head, dY, lddy, prec, ws, ws_bytes, stream);
}

}  // extern "C"
