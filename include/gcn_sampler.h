/*
 * gcn_sampler.h -- graph sampling and GCN construction on the sample: the
 * stage of graph-sampling GCN training that feeds the layer of gcn_layer.h
 * (Zeng et al., arXiv 1810.11899, Sec. IV and Alg. 2-5).
 *
 * Pipeline for a batch of S subgraphs of a training graph G:
 *   gcn_frontier_sample   S frontier-sampling runs (Sec. IV-A, Alg. 2) with the
 *                         Dashboard (Sec. IV-B/IV-C, Alg. 3 and Alg. 4), one
 *                         wavefront per run, the Dashboard in LDS;
 *   gcn_induce_subgraphs  the subgraph of G induced by each run's vertices, as
 *                         the mean-normalised CSR the layer takes (Sec. II);
 *   gcn_gather_rows       the input features H^(0) (and labels) of the sampled
 *                         vertices (GCN construction on the subgraph, Alg. 5).
 *
 * Conventions are those of gcn_layer.h: device pointers owned by the caller,
 * `stream` a hipStream_t as void*, host-side argument checks before any
 * launch, negative gcn_status on failure with a message for gcn_last_error(),
 * caller workspace for scratch, deterministic results.  G is not checked on
 * the device: every index of G must be in [0, n_vertices) (see
 * gcn_csr_validate_host); an index outside it ends that run with
 * GCN_SAMPLE_BAD_GRAPH instead of a fault.
 *
 * Method details fixed here (the paper leaves them open):
 *   - a run's vertex list is its m roots (distinct, uniform) followed by the
 *     vertex added to the frontier at each of the n - m steps; it may repeat a
 *     vertex, and the induced subgraph uses the distinct ones;
 *   - a vertex takes w(v) = deg(v) Dashboard entries, or min(deg(v), cap)
 *     with cap > 0 (the per-vertex limit of Sec. VI-C-2 for skewed graphs);
 *   - the 64 lanes of a wavefront are the p = 64 processors of the probing
 *     step (Alg. 4); probes are uniform over the used Dashboard entries and the
 *     lowest lane that hits a valid entry wins;
 *   - a cleanup (Alg. 4) runs before an append that would overflow the
 *     Dashboard or the Index Array;
 *   - random numbers: Philox4x64-10 keyed by (seed, first_sampler + run
 *     index); word w of the block with counter (c0, kind, c2, 0) gives an
 *     integer uniform on [0, N) as the high 64 bits of the word times N.
 *     Root candidate t: counter (t, 1, 0, 0), word 0.  Probe of lane j in
 *     probing round r: counter (r / 4, 2, j, 0), word r % 4.  Neighbour
 *     choice of step t (t = 0 for the first step after the roots): counter
 *     (t / 4, 3, 0, 0), word t % 4.  The same (seed, run id) gives the same
 *     subgraph on every device.
 */
#ifndef GCN_SAMPLER_H_
#define GCN_SAMPLER_H_

#include <stdint.h>

#include "gcn_layer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Per-run outcome written to the status array of gcn_frontier_sample. */
typedef enum {
    GCN_SAMPLE_OK = 0,           /* n vertices                                    */
    GCN_SAMPLE_EXHAUSTED = 1,    /* every frontier vertex had weight 0: stopped   */
    GCN_SAMPLE_OVERFLOW = 2,     /* the frontier's entries outgrew the Dashboard  */
    GCN_SAMPLE_PROBE_LIMIT = 3,  /* a pop needed more than 2^20 probing rounds    */
    GCN_SAMPLE_ROOT_LIMIT = 4,   /* more than 64 m + 65536 root candidates        */
    GCN_SAMPLE_BAD_GRAPH = 5     /* an index of G outside [0, n_vertices)         */
} gcn_sample_status;

typedef struct {
    int32_t m;           /* frontier size (the paper uses 1000)               */
    int32_t n;           /* vertex-list length: m roots + (n - m) steps        */
    int32_t db_entries;  /* Dashboard capacity, entries                        */
    int32_t ia_slots;    /* Index-Array capacity, slots; m < ia_slots <= 65535 */
    int32_t cap;         /* Dashboard entries per vertex at most; 0 = deg(v)   */
    uint64_t seed;
} gcn_sampler_params;

/* Sizes the Dashboard for enlargement factor eta > 1 (Sec. IV-B: eta * m *
 * the mean number of entries per vertex of G, and at least a frontier of m
 * vertices of the largest weight, so that no run can overflow) with an Index
 * Array of m + 512 slots, clamped to one CU's LDS (160 KB).  indptr_host is
 * G's row pointer in HOST memory [n_vertices + 1].  GCN_EUNSUPPORTED when
 * the Index Array alone cannot fit. */
int gcn_sampler_plan(int32_t n_vertices, const int32_t *indptr_host, int32_t m, int32_t n, double eta,
                     int32_t cap, uint64_t seed, gcn_sampler_params *out);

/* S runs with ids first_sampler .. first_sampler + S - 1 on G (square CSR;
 * vals unused).  Outputs, device arrays:
 *   vertices [S x n]  run r's list in row r (entries past counts[r] untouched)
 *   counts   [S]      list length (n unless the status says otherwise)
 *   status   [S]      gcn_sample_status
 * Each run uses 12 ia_slots + 2 db_entries bytes of LDS (one CU's at most);
 * runs of at most 80 KB share a CU two at a time. */
int gcn_frontier_sample(const gcn_csr *G, const gcn_sampler_params *p, int64_t first_sampler, int32_t S,
                        int32_t *vertices, int32_t *counts, int32_t *status, void *stream);

/* Induced subgraphs of S vertex lists (rows of `vertices`, leading dim n,
 * lengths counts[S], e.g. from gcn_frontier_sample).  For list s:
 *   n_sub[s]                      number of distinct vertices
 *   vsub[s*n .. s*n + n_sub[s])   those vertices ascending; local id = position
 *   indptr_sub[s*(n+1) ..]        n+1 row offsets, local to the subgraph (rows
 *                                 past n_sub[s] are empty)
 *   sub_indices / sub_vals        from edge_offsets[s] to edge_offsets[s+1]:
 *                                 row i lists the local ids of the neighbours
 *                                 of vsub[i] in the set, ascending, with value
 *                                 1/(row length) (float32 quotient)
 *   sub_vals_t (may be NULL)      entry p of row i, column j = sub_indices[p],
 *                                 gets 1/(row length of j): when G's pattern
 *                                 is symmetric (gcn_csr_pattern_symmetric_host)
 *                                 so is each induced subgraph's, and
 *                                 (indptr_sub, sub_indices, sub_vals_t) is then
 *                                 the CSR of the transposed aggregation
 *                                 matrix, equal bit for bit to what
 *                                 gcn_csr_transpose returns
 *   edge_offsets [S+1]            int64 prefix of the subgraphs' edge counts
 *   status [1]                    0, or 1 when edge_offsets[S] > edge_capacity
 *                                 (then no edge is written; size the arrays
 *                                 from edge_offsets[S] and call again)
 * Vertex ids outside [0, n_vertices) in `vertices` are skipped.  The
 * workspace holds, per list, a membership bitmap of n_vertices bits and an
 * int32 prefix count per 32 vertices (8 bytes per 32 vertices of G). */
size_t gcn_induce_workspace_bytes(int32_t n_vertices, int32_t n, int32_t S);
int gcn_induce_subgraphs(const gcn_csr *G, int32_t S, int32_t n, const int32_t *vertices, const int32_t *counts,
                         int32_t *n_sub, int32_t *vsub, int32_t *indptr_sub, int64_t *edge_offsets,
                         int32_t *sub_indices, float *sub_vals, float *sub_vals_t, int64_t edge_capacity,
                         int32_t *status, void *ws, size_t ws_bytes, void *stream);

/* 1 when every stored (i, j) of the CSR in HOST memory has a stored (j, i),
 * 0 when not; rows must hold ascending column indices (GCN_EINVAL if not, or
 * if an index is out of range).  O(nnz log(max degree)). */
int gcn_csr_pattern_symmetric_host(int32_t n, const int32_t *indptr_host, const int32_t *indices_host);

/* out[i, 0:width] = X[rows[i], 0:width] for i < count, 4-byte elements (float
 * features or int32 labels), leading dimensions in elements.  A row index
 * outside [0, n_rows_X) gives a row of zeros. */
int gcn_gather_rows(const void *X, int32_t n_rows_X, int32_t width, int64_t ldx, const int32_t *rows,
                    int32_t count, void *out, int64_t ldo, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GCN_SAMPLER_H_ */
