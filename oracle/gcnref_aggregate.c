/*
 * CPU oracle for the graph-sampling GCN layer (arXiv 1810.11899).
 * TEST INFRASTRUCTURE ONLY: used by the tests, by the smoke check and by the
 * CPU-baseline leg of the benchmark.  Shares no code with the HIP library.
 *
 * Feature aggregation, Sec. II (step 1 of the forward propagation) and the
 * feature-propagation kernel of Sec. V-A: every destination vertex i takes the
 * weighted sum of the feature rows of its in-neighbours,
 *
 *     out[i, :] = sum_{p = indptr[i]}^{indptr[i+1]-1} vals[p] * X[indices[p], :]
 *
 * With vals[p] = 1/deg(i) this is the mean of Sec. II.  The terms are added in
 * increasing p, in double precision; an empty row gives zeros.  Rows are
 * independent, so OpenMP threads take whole rows (the order inside a row never
 * changes).  The paper's feature-sliced schedule (Alg. 6) only reorders these
 * same sums; it is not reproduced here.
 */
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

void gcnref_aggregate(int64_t n_rows, int64_t k,
                      const int32_t *indptr, const int32_t *indices,
                      const double *vals,
                      const double *X, int64_t ldx,
                      double *out, int64_t ldo)
{
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < n_rows; ++i) {
        double *o = out + i * ldo;
        for (int64_t c = 0; c < k; ++c)
            o[c] = 0.0;
        for (int64_t p = indptr[i]; p < indptr[i + 1]; ++p) {
            const double w = vals[p];
            const double *x = X + (int64_t)indices[p] * ldx;
            for (int64_t c = 0; c < k; ++c)
                o[c] += w * x[c];
        }
    }
}

/* Threads for the following aggregations (timing of a serial run); n < 1
 * leaves the setting alone.  Not part of the arithmetic. */
void gcnref_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int gcnref_num_threads(void)
{
    int t = 1;
    #pragma omp parallel
    {
        #pragma omp single
        {
#ifdef _OPENMP
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
