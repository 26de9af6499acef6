/*
 * CPU oracle of the graph sampler (test infrastructure only; the HIP library
 * never links this file and it includes nothing of the library).
 *
 * Frontier sampling (Sec. IV-A, Alg. 2) with the Dashboard of Sec. IV-B, as
 * parallelised in Sec. IV-C (Alg. 3 and Alg. 4): one sampler instance, run
 * sequentially, the p processors of the probing step emulated one after the
 * other.  Random numbers come from
 * Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011), written here from that definition.
 *
 * Readings taken where the paper is silent or inconsistent:
 *   - the subgraph's vertex list is the m roots followed by the n - m vertices
 *     added to the frontier (Alg. 3 adds v_new to V_sub); duplicates are kept
 *     in the list and removed by the induced-subgraph step;
 *   - a vertex holds w(v) = deg(v) Dashboard entries, or min(deg(v), cap) when
 *     a cap is given (the cap of Sec. VI-C-2 for skewed graphs);
 *   - a Dashboard entry holds the index of its Index-Array slot; a slot holds
 *     (vertex, weight, live).  Popping clears the slot's live flag, which
 *     invalidates all of the vertex's entries at once (Alg. 4 marks each of
 *     them INV: same set of valid entries);
 *   - probes are uniform over the used part of the Dashboard; one probing
 *     round draws p indices, and the lowest-numbered processor whose probe
 *     hits a valid entry wins (Alg. 4 leaves the winner open);
 *   - cleanup (Alg. 4) runs before an append that would overflow the
 *     Dashboard or the Index Array; it keeps the live slots in slot order;
 *   - the m roots are distinct: candidates are drawn one by one and a repeat
 *     is skipped.
 * Random draws: word w of the Philox4x64-10 block with counter (c0, kind, c2,
 * 0) and key (seed, sampler id); an integer uniform on [0, N) is the high 64
 * bits of the word times N.  Root candidate t: kind 1, counter (t, 1, 0, 0),
 * word 0.  Probe of processor j in probing round r: kind 2, counter
 * (r / 4, 2, j, 0), word r % 4.  Neighbour choice of step t = i - m: kind 3,
 * counter (t / 4, 3, 0, 0), word t % 4.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GCNREF_SAMPLE_OK 0
#define GCNREF_SAMPLE_EXHAUSTED 1   /* every frontier vertex has weight 0 */
#define GCNREF_SAMPLE_OVERFLOW 2    /* the frontier's entries exceed the Dashboard */
#define GCNREF_SAMPLE_PROBE_LIMIT 3 /* a pop needed more probing rounds than the limit */
#define GCNREF_SAMPLE_ROOT_LIMIT 4  /* too many repeated root candidates */
#define GCNREF_SAMPLE_EINVAL (-1)

#define KIND_ROOT 1u
#define KIND_PROBE 2u
#define KIND_NEIGH 3u
#define PROBE_ROUND_LIMIT (1 << 20)

/* ----------------------------------------------------------- Philox4x64-10 */
static void mulhilo64(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo) {
    unsigned __int128 p = (unsigned __int128)a * b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void gcnref_philox4x64(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
    const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
    uint64_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; ++r) {
        uint64_t hi0, lo0, hi1, lo1;
        mulhilo64(M0, c0, &hi0, &lo0);
        mulhilo64(M1, c2, &hi1, &lo1);
        const uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += W0;
        k1 += W1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static uint64_t draw(uint64_t seed, uint64_t sid, uint64_t kind, uint64_t c0, uint64_t c2, int word) {
    const uint64_t ctr[4] = {c0, kind, c2, 0}, key[2] = {seed, sid};
    uint64_t out[4];
    gcnref_philox4x64(ctr, key, out);
    return out[word];
}

static int64_t below(uint64_t r, int64_t n) {
    return (int64_t)(((unsigned __int128)r * (uint64_t)n) >> 64);
}

/* ------------------------------------------------------------- the sampler */
typedef struct {
    int32_t vertex;
    int32_t weight;
    int32_t live;
} Slot;

static int32_t weight_of(const int32_t *indptr, int32_t v, int32_t cap) {
    const int32_t d = indptr[v + 1] - indptr[v];
    return (cap > 0 && d > cap) ? cap : d;
}

/* Cleanup of Alg. 4: a fresh Dashboard holding the live slots' entries, slots
 * renumbered in their old order. */
static void cleanup(int32_t *db, Slot *ia, int32_t *s, int64_t *used) {
    int32_t ns = 0;
    int64_t nu = 0;
    for (int32_t k = 0; k < *s; ++k) {
        if (!ia[k].live) continue;
        ia[ns] = ia[k];
        for (int32_t e = 0; e < ia[ns].weight; ++e) db[nu + e] = ns;
        nu += ia[ns].weight;
        ++ns;
    }
    *s = ns;
    *used = nu;
}

int gcnref_frontier_sample(int64_t nV, const int32_t *indptr, const int32_t *indices, int32_t m, int32_t n,
                           int64_t db_cap, int32_t ia_cap, int32_t cap, int32_t p, uint64_t seed,
                           uint64_t sampler_id, int32_t *out, int32_t *count) {
    *count = 0;
    if (nV <= 0 || m <= 0 || m > nV || n < m || ia_cap <= m || db_cap <= 0 || p <= 0)
        return GCNREF_SAMPLE_EINVAL;
    int32_t *db = (int32_t *)malloc(sizeof(int32_t) * (size_t)db_cap);
    Slot *ia = (Slot *)malloc(sizeof(Slot) * (size_t)ia_cap);
    unsigned char *is_root = (unsigned char *)calloc((size_t)nV, 1);
    int status = GCNREF_SAMPLE_OK;

    /* roots: m distinct vertices, uniform */
    int32_t got = 0;
    const uint64_t root_limit = 64ull * (uint64_t)m + 65536ull;
    for (uint64_t t = 0; got < m; ++t) {
        if (t >= root_limit) { status = GCNREF_SAMPLE_ROOT_LIMIT; break; }
        const int32_t v = (int32_t)below(draw(seed, sampler_id, KIND_ROOT, t, 0, 0), nV);
        if (is_root[v]) continue;
        is_root[v] = 1;
        out[got++] = v;
    }
    *count = got;
    if (status != GCNREF_SAMPLE_OK) goto done;

    /* Dashboard and Index Array from the roots (Alg. 3, initialisation) */
    int64_t used = 0, live_weight = 0;
    int32_t s = 0;
    for (int32_t i = 0; i < m; ++i) {
        const int32_t w = weight_of(indptr, out[i], cap);
        if (used + w > db_cap) { status = GCNREF_SAMPLE_OVERFLOW; goto done; }
        ia[s].vertex = out[i];
        ia[s].weight = w;
        ia[s].live = 1;
        for (int32_t e = 0; e < w; ++e) db[used + e] = s;
        used += w;
        live_weight += w;
        ++s;
    }

    /* main loop: pop, step to a neighbour, add */
    uint64_t round = 0;
    for (int32_t i = m; i < n; ++i) {
        if (live_weight == 0) { status = GCNREF_SAMPLE_EXHAUSTED; break; }
        int32_t k = -1;
        for (int64_t rr = 0; k < 0; ++rr, ++round) {
            if (rr >= PROBE_ROUND_LIMIT) { status = GCNREF_SAMPLE_PROBE_LIMIT; goto done; }
            for (int32_t j = 0; j < p; ++j) {
                const int64_t idx = below(draw(seed, sampler_id, KIND_PROBE, round >> 2, (uint64_t)j, (int)(round & 3)),
                                          used);
                if (ia[db[idx]].live) { k = db[idx]; break; }
            }
        }
        const int32_t v_pop = ia[k].vertex;
        ia[k].live = 0;
        live_weight -= ia[k].weight;

        const int32_t deg = indptr[v_pop + 1] - indptr[v_pop];  /* >= 1: its weight was > 0 */
        const uint64_t t = (uint64_t)(i - m);
        const int64_t pick = below(draw(seed, sampler_id, KIND_NEIGH, t >> 2, 0, (int)(t & 3)), deg);
        const int32_t v_new = indices[indptr[v_pop] + pick];
        const int32_t w = weight_of(indptr, v_new, cap);

        if (used + w > db_cap || s == ia_cap) cleanup(db, ia, &s, &used);
        if (used + w > db_cap) { status = GCNREF_SAMPLE_OVERFLOW; break; }
        ia[s].vertex = v_new;
        ia[s].weight = w;
        ia[s].live = 1;
        for (int32_t e = 0; e < w; ++e) db[used + e] = s;
        used += w;
        live_weight += w;
        ++s;
        out[i] = v_new;
        *count = i + 1;
    }
done:
    free(db);
    free(ia);
    free(is_root);
    return status;
}
