/*
 * CPU oracle for BOA's batched filtered beam search with online beamwidth
 * adaptation. TEST INFRASTRUCTURE ONLY: it is linked by the tests, by the
 * smoke check and by the benchmark's CPU-baseline leg, never by the
 * product library, and it shares no code with the GPU implementation.
 *
 * It is deliberately plain: one query at a time, a sorted array for the
 * worklist, a stamp array for the set of scored nodes, a full merge per
 * iteration. Independent queries may run on several threads; every
 * query's result depends only on its own inputs.
 *
 * Paper: "BOA: Beamwidth Online Adaptation for Filtered-ANNS on a GPU".
 * Each function cites the passage it follows. Readings of points the
 * paper leaves open are marked READING.
 *
 * Build: gcc -O2 -mfma -ffp-contract=off (no fast-math): the distance
 * below relies on explicit fused multiply-adds and no other contraction.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_PAD 0xFFFFFFFFu
#define ORC_VEC_F32 0
#define ORC_VEC_U8 1
#define ORC_ATTR_I32 0
#define ORC_ATTR_F32 1

typedef struct {
    int64_t n;
    int32_t d;
    int32_t vec_dtype;
    const void *vectors;        /* n x d, float32 or uint8 */
    int32_t m;
    const int32_t *attrs;       /* n x m 4-byte cells */
    const int32_t *attr_dtypes; /* m */
    int32_t R;
    const uint32_t *adj;        /* n x R, ORC_PAD padded */
    int64_t entry;              /* entry point s */
    /* product quantisation (pq_m = 0: none): pq_m subspaces of d / pq_m
     * dimensions, 16 centroids each (pq_cb: pq_m x 16 x ds float32), codes
     * n x pq_m / 2 bytes, subspace 2b in the low nibble of byte b */
    int32_t pq_m;
    const float *pq_cb;
    const uint8_t *pq_codes;
} orc_index;

/* One worklist entry: the search orders by the filter distance phi first,
 * then vector distance, then id (Sec. III-A "How Filtered Search Works":
 * with the penalty lambda well above the distance scale, every valid
 * candidate ranks ahead of every invalid one and distance orders each
 * group). READING: lambda is taken to infinity, i.e. the lexicographic
 * order (phi, d, id); id breaks exact distance ties deterministically. */
typedef struct {
    int32_t phi;
    float d;
    uint32_t id;
    int32_t expanded;
} orc_entry;

static int entry_before(const orc_entry *a, const orc_entry *b)
{
    if (a->phi != b->phi) return a->phi < b->phi;
    if (a->d != b->d) return a->d < b->d;
    return a->id < b->id;
}

/* ------------------------------------------------------------------------
 * Squared Euclidean distance (Def. 1 uses the Euclidean norm throughout;
 * squared distance orders identically).
 *
 * float32 vectors: the distance decides orderings, so it is computed in
 * the kernel's precision (float32) in one fixed order. 16 partial sums;
 * chunk c = dims 4c..4c+3 goes to partial c mod 16, chunks in increasing
 * order, dims in order within a chunk, each term added with one fused
 * multiply-add of the float32 difference; the 16 partials are then summed
 * pairwise (p += p+8, p += p+4, p += p+2, p += p+1). d must be a multiple
 * of 4.
 * uint8 vectors: exact int32 sum of squared differences (at most
 * d * 255^2, exact in float32 for d <= 258). */
float orc_dist_f32(const float *x, const float *q, int32_t d)
{
    float acc[16];
    for (int p = 0; p < 16; ++p) acc[p] = 0.0f;
    for (int c = 0; c < d / 4; ++c) {
        int p = c % 16;
        for (int t = 0; t < 4; ++t) {
            float diff = x[4 * c + t] - q[4 * c + t];
            acc[p] = fmaf(diff, diff, acc[p]);
        }
    }
    for (int s = 8; s >= 1; s /= 2)
        for (int p = 0; p < s; ++p) acc[p] = acc[p] + acc[p + s];
    return acc[0];
}

float orc_dist_u8(const uint8_t *x, const uint8_t *q, int32_t d)
{
    int32_t sum = 0;
    for (int i = 0; i < d; ++i) {
        int32_t diff = (int32_t)x[i] - (int32_t)q[i];
        sum += diff * diff;
    }
    return (float)sum;
}

static float point_dist(const orc_index *ix, uint32_t v, const void *q)
{
    if (ix->vec_dtype == ORC_VEC_U8)
        return orc_dist_u8((const uint8_t *)ix->vectors + (int64_t)v * ix->d,
                           (const uint8_t *)q, ix->d);
    return orc_dist_f32((const float *)ix->vectors + (int64_t)v * ix->d,
                        (const float *)q, ix->d);
}

/* ------------------------------------------------------------------------
 * Product-quantised asymmetric distance (Alg. 2 "PQDist"; Sec. III-B: the
 * GPU builds each query's distance table, then scores a candidate as the
 * sum of table entries indexed by its codes).
 *   table:    T[m][c] = squared distance of the query's subvector m to
 *             centroid c of subspace m, float32, one fused multiply-add per
 *             dimension in dimension order from +0;
 *   distance: 16 partial sums, subspace m added (float32) to partial
 *             m mod 16 in increasing m, then the partials summed pairwise
 *             (p += p+8, +4, +2, +1), the order of the exact distance. */
void orc_pq_table(const orc_index *ix, const void *q, float *table)
{
    const int32_t M = ix->pq_m, ds = ix->d / M;
    for (int m = 0; m < M; ++m)
        for (int c = 0; c < 16; ++c) {
            float acc = 0.0f;
            for (int j = 0; j < ds; ++j) {
                float qv = ix->vec_dtype == ORC_VEC_U8 ? (float)((const uint8_t *)q)[m * ds + j]
                                                       : ((const float *)q)[m * ds + j];
                float diff = qv - ix->pq_cb[((int64_t)m * 16 + c) * ds + j];
                acc = fmaf(diff, diff, acc);
            }
            table[m * 16 + c] = acc;
        }
}

float orc_pq_dist(const float *table, const uint8_t *code, int32_t M)
{
    float acc[16];
    for (int p = 0; p < 16; ++p) acc[p] = 0.0f;
    for (int m = 0; m < M; ++m) {
        int c = (code[m / 2] >> (4 * (m % 2))) & 15;
        acc[m % 16] = acc[m % 16] + table[m * 16 + c];
    }
    for (int s = 8; s >= 1; s /= 2)
        for (int p = 0; p < s; ++p) acc[p] = acc[p] + acc[p + s];
    return acc[0];
}

/* ------------------------------------------------------------------------
 * Filter distance phi: the number of the query's range predicates the
 * point violates (Sec. II, JAG paragraph; Alg. 2). A predicate on
 * attribute j holds when lo_j <= a^j <= hi_j, bounds inclusive (Def. 2,
 * Eq. 2); phi = 0 exactly when the matching function g is 1. Each column
 * compares in its own type: int32 as integers, float32 as floats. */
int32_t orc_phi(const int32_t *attr_row, const int32_t *range_row,
                const int32_t *attr_dtypes, int32_t m)
{
    int32_t phi = 0;
    for (int j = 0; j < m; ++j) {
        int ok;
        if (attr_dtypes[j] == ORC_ATTR_F32) {
            float a, lo, hi;
            memcpy(&a, &attr_row[j], 4);
            memcpy(&lo, &range_row[2 * j], 4);
            memcpy(&hi, &range_row[2 * j + 1], 4);
            ok = (lo <= a) && (a <= hi);
        } else {
            int32_t a = attr_row[j], lo = range_row[2 * j], hi = range_row[2 * j + 1];
            ok = (lo <= a) && (a <= hi);
        }
        if (!ok) phi += 1;
    }
    return phi;
}

/* ------------------------------------------------------------------------
 * Per-thread scratch: a stamp per point marks membership in the set of
 * scored nodes of the current search (a fresh stamp = an empty set). */
typedef struct {
    uint32_t *stamp;
    uint32_t cur;
    orc_entry *beam, *cand, *tmp;
    int64_t cap_beam;
    float *table;       /* the current query's PQ distance table (PQ only) */
} orc_ws;

static int ws_init(orc_ws *w, const orc_index *ix, int32_t Lmax)
{
    w->stamp = (uint32_t *)calloc((size_t)ix->n, sizeof(uint32_t));
    w->cur = 0;
    w->cap_beam = Lmax;
    w->beam = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(Lmax + ix->R + 1));
    w->cand = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(ix->R + 1));
    w->tmp = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(Lmax + ix->R + 1));
    w->table = ix->pq_m > 0 ? (float *)malloc(sizeof(float) * 16 * (size_t)ix->pq_m) : NULL;
    return w->stamp && w->beam && w->cand && w->tmp && (ix->pq_m == 0 || w->table);
}

static void ws_free(orc_ws *w)
{
    free(w->stamp); free(w->beam); free(w->cand); free(w->tmp); free(w->table);
}

static void ws_new_search(orc_ws *w, int64_t n)
{
    w->cur += 1;
    if (w->cur == 0) { /* wrapped: clear all stamps */
        memset(w->stamp, 0, sizeof(uint32_t) * (size_t)n);
        w->cur = 1;
    }
}

/* A candidate's key. With product quantisation the traversal orders by the
 * asymmetric distance through the query's table (Alg. 2 "PQDist"). */
static orc_entry score(const orc_index *ix, uint32_t v, const void *q, const int32_t *rr, const float *table)
{
    orc_entry e;
    e.phi = orc_phi(ix->attrs + (int64_t)v * ix->m, rr, ix->attr_dtypes, ix->m);
    e.d = table ? orc_pq_dist(table, ix->pq_codes + (int64_t)v * (ix->pq_m / 2), ix->pq_m)
                : point_dist(ix, v, q);
    e.id = v;
    e.expanded = 0;
    return e;
}

/* The result of a search (the first L entries of its sorted list): the
 * filter-valid entries, in order. With product quantisation they are
 * re-ranked by exact distance (Sec. III-B step 8: on convergence the
 * accumulated candidates are ranked by exact distance under a hard
 * predicate), ordered by (exact distance, id). Returns n_valid; out holds
 * the valid entries with their reported distances. */
static int valid_results(const orc_index *ix, const orc_entry *beam, int lim, const void *q, orc_entry *out)
{
    int n_valid = 0;
    while (n_valid < lim && beam[n_valid].phi == 0) {
        out[n_valid] = beam[n_valid];
        ++n_valid;
    }
    if (ix->pq_m > 0) {
        for (int a = 0; a < n_valid; ++a) out[a].d = point_dist(ix, out[a].id, q);
        for (int a = 1; a < n_valid; ++a) {   /* insertion sort by (d, id) */
            orc_entry x = out[a];
            int b = a - 1;
            while (b >= 0 && entry_before(&x, &out[b])) { out[b + 1] = out[b]; --b; }
            out[b + 1] = x;
        }
    }
    return n_valid;
}

/* ------------------------------------------------------------------------
 * Filter-aware beam search of one query at beamwidth L (Alg. 2, with the
 * generic beam search of Sec. II "Beam search").
 *   - The worklist starts as {s}; s is scored and entered in the set of
 *     scored nodes before the first expansion (READING: Alg. 2 starts
 *     the list at s without saying how s is marked).
 *   - Each iteration expands exactly one node: the nearest not-yet-expanded
 *     entry of the worklist.
 *   - Its out-neighbours are read in row order; a neighbour already scored
 *     in this search is dropped (READING: the paper's Bloom filter is
 *     replaced by an exact set, so results never depend on its size);
 *     every other neighbour is scored, marked, and merged into the sorted
 *     worklist, which is then cut to its L best entries.
 *   - The search ends when every entry of the worklist has been expanded
 *     (READING: every entry is expanded before the loop ends, as in the
 *     generic beam search).
 * Returns the final worklist (sorted) and adds to *E (expansions) and *S
 * (scored nodes, s included). */
static int search_one(const orc_index *ix, orc_ws *w, const void *q, const int32_t *rr,
                      int32_t L, int *out_len, int64_t *E, int64_t *S)
{
    orc_entry *beam = w->beam, *cand = w->cand, *tmp = w->tmp;
    ws_new_search(w, ix->n);
    if (w->table) orc_pq_table(ix, q, w->table);
    int len = 1;
    beam[0] = score(ix, (uint32_t)ix->entry, q, rr, w->table);
    w->stamp[ix->entry] = w->cur;
    *S += 1;

    for (;;) {
        int j = 0;
        while (j < len && beam[j].expanded) ++j;
        if (j == len) break; /* converged */
        beam[j].expanded = 1;
        uint32_t u = beam[j].id;
        *E += 1;

        int c = 0;
        for (int r = 0; r < ix->R; ++r) {
            uint32_t v = ix->adj[(int64_t)u * ix->R + r];
            if (v == ORC_PAD) continue;
            if (w->stamp[v] == w->cur) continue;
            w->stamp[v] = w->cur;
            cand[c++] = score(ix, v, q, rr, w->table);
        }
        *S += c;

        /* sort the new candidates (insertion sort), merge, keep the L best */
        for (int a = 1; a < c; ++a) {
            orc_entry x = cand[a];
            int b = a - 1;
            while (b >= 0 && entry_before(&x, &cand[b])) { cand[b + 1] = cand[b]; --b; }
            cand[b + 1] = x;
        }
        int ia = 0, ib = 0, o = 0;
        while ((ia < len || ib < c) && o < L) {
            if (ib >= c || (ia < len && entry_before(&beam[ia], &cand[ib])))
                tmp[o++] = beam[ia++];
            else
                tmp[o++] = cand[ib++];
        }
        memcpy(beam, tmp, sizeof(orc_entry) * (size_t)o);
        len = o;
    }
    *out_len = len;
    return 0;
}

/* ------------------------------------------------------------------------
 * Confidence test (Eq. 3). Over the filter-valid entries of the final
 * sorted worklist, gamma = (D_max - D_k) / D_max with D the Euclidean
 * distance (square root of the stored squared distance), computed in
 * double; confident when gamma <= eps.
 * READING: the test presumes the list holds more valid entries than the k
 * returned; with n_valid <= k the query is not confident and escalates.
 * READING: D_max = 0 (all valid entries at distance zero) gives gamma = 0. */
int orc_confident(const float *valid_sq_dists, int32_t n_valid, int32_t k, double eps)
{
    if (n_valid <= k) return 0;
    double dk = sqrt((double)valid_sq_dists[k - 1]);
    double dmax = sqrt((double)valid_sq_dists[n_valid - 1]);
    double gamma = (dmax == 0.0) ? 0.0 : (dmax - dk) / dmax;
    return gamma <= eps;
}

/* Beam schedule (Alg. 1: the width grows by alpha each phase).
 * READING: L_{p+1} = min(ceil(alpha * L_p), Lmax), computed in double, and
 * the phase that runs at Lmax is the last. Returns the number of phases. */
int32_t orc_schedule(int32_t L0, double alpha, int32_t Lmax, int32_t *out, int32_t cap)
{
    int32_t n = 0;
    int64_t L = L0;
    for (;;) {
        if (n >= cap) return -1;
        out[n++] = (int32_t)L;
        if (L >= Lmax) break;
        int64_t nx = (int64_t)ceil(alpha * (double)L);
        if (nx <= L) nx = L + 1;
        L = nx < Lmax ? nx : Lmax;
    }
    return n;
}

/* ------------------------------------------------------------------------
 * The multi-phase driver (Alg. 1, Sec. III-A "How adaptation works").
 *   - All queries start active; a phase runs while more than tau * nq
 *     queries are active.
 *   - Every active query is searched afresh at the phase's width (each
 *     phase calls the beam search anew: it restarts from s).
 *   - Its result (the first min(k, n_valid) valid entries; padded with
 *     id 0xFFFFFFFF and distance +inf) is stored at the query's original
 *     index, whichever phase produced it; final_L records that phase's L.
 *   - Confident queries leave; the rest go on at the next width.
 *     Queries still active after the last width keep their last result.
 * Per-phase statistics (phase_stats[p*5 + ...]): L, |A|, confident, sum E,
 * sum S. Returns the number of phases run. */
typedef struct {
    const orc_index *ix;
    const void *queries;
    const int32_t *ranges;
    const int64_t *active;
    int64_t n_active;
    int32_t k, L;
    double eps;
    uint32_t *ids;
    float *dists;
    int32_t *final_L;
    int64_t *q_E, *q_S;
    uint8_t *conf;
    int64_t next;             /* work counter */
    pthread_mutex_t mu;
    int32_t Lmax;
    int failed;
} phase_job;

static void run_query(phase_job *J, orc_ws *w, int64_t t)
{
    const orc_index *ix = J->ix;
    int64_t i = J->active[t];
    size_t qbytes = (size_t)ix->d * (ix->vec_dtype == ORC_VEC_U8 ? 1 : 4);
    const void *q = (const char *)J->queries + (size_t)i * qbytes;
    const int32_t *rr = J->ranges + (int64_t)i * ix->m * 2;
    int len = 0;
    int64_t E = 0, S = 0;
    search_one(ix, w, q, rr, J->L, &len, &E, &S);

    orc_entry *res = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(len > 0 ? len : 1));
    int n_valid = valid_results(ix, w->beam, len, q, res);
    float *vd = (float *)malloc(sizeof(float) * (size_t)(n_valid > 0 ? n_valid : 1));
    for (int a = 0; a < n_valid; ++a) vd[a] = res[a].d;
    for (int a = 0; a < J->k; ++a) {
        if (a < n_valid) {
            J->ids[i * J->k + a] = res[a].id;
            J->dists[i * J->k + a] = res[a].d;
        } else {
            J->ids[i * J->k + a] = ORC_PAD;
            J->dists[i * J->k + a] = INFINITY;
        }
    }
    J->final_L[i] = J->L;
    J->conf[t] = (uint8_t)orc_confident(vd, n_valid, J->k, J->eps);
    free(vd);
    free(res);
    if (J->q_E) J->q_E[i] += E;
    if (J->q_S) J->q_S[i] += S;
}

static void *phase_worker(void *arg)
{
    phase_job *J = (phase_job *)arg;
    orc_ws w;
    if (!ws_init(&w, J->ix, J->Lmax)) {
        pthread_mutex_lock(&J->mu); J->failed = 1; pthread_mutex_unlock(&J->mu);
        return NULL;
    }
    for (;;) {
        pthread_mutex_lock(&J->mu);
        int64_t t = J->next++;
        pthread_mutex_unlock(&J->mu);
        if (t >= J->n_active) break;
        run_query(J, &w, t);
    }
    ws_free(&w);
    return NULL;
}

int32_t orc_boa(const orc_index *ix, const void *queries, const int32_t *ranges, int64_t nq,
                int32_t k, const int32_t *schedule, int32_t n_phases, double eps, double tau,
                uint32_t *ids, float *dists, int32_t *final_L, int64_t *q_E, int64_t *q_S,
                int64_t *phase_stats, int32_t nthreads)
{
    if (nq <= 0 || n_phases <= 0) return 0;
    int32_t Lmax = 0;
    for (int p = 0; p < n_phases; ++p) if (schedule[p] > Lmax) Lmax = schedule[p];
    int64_t *A = (int64_t *)malloc(sizeof(int64_t) * (size_t)nq);
    uint8_t *conf = (uint8_t *)malloc((size_t)nq);
    if (!A || !conf) { free(A); free(conf); return -2; }
    int64_t nA = nq;
    for (int64_t i = 0; i < nq; ++i) A[i] = i;
    if (q_E) memset(q_E, 0, sizeof(int64_t) * (size_t)nq);
    if (q_S) memset(q_S, 0, sizeof(int64_t) * (size_t)nq);
    if (nthreads < 1) nthreads = 1;

    int32_t ran = 0;
    for (int p = 0; p < n_phases; ++p) {
        if (!((double)nA > tau * (double)nq)) break;
        phase_job J;
        memset(&J, 0, sizeof(J));
        J.ix = ix; J.queries = queries; J.ranges = ranges; J.active = A; J.n_active = nA;
        J.k = k; J.L = schedule[p]; J.eps = eps; J.ids = ids; J.dists = dists;
        J.final_L = final_L; J.q_E = q_E; J.q_S = q_S; J.conf = conf; J.next = 0;
        J.Lmax = Lmax;
        pthread_mutex_init(&J.mu, NULL);
        int64_t E0 = 0, S0 = 0;
        if (phase_stats) {
            for (int64_t t = 0; t < nA; ++t) {
                if (q_E) E0 += q_E[A[t]];
                if (q_S) S0 += q_S[A[t]];
            }
        }
        int nt = nthreads;
        if (nt > nA) nt = (int)nA;
        if (nt <= 1) {
            phase_worker(&J);
        } else {
            pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
            for (int t = 0; t < nt; ++t) pthread_create(&th[t], NULL, phase_worker, &J);
            for (int t = 0; t < nt; ++t) pthread_join(th[t], NULL);
            free(th);
        }
        pthread_mutex_destroy(&J.mu);
        if (J.failed) { free(A); free(conf); return -2; }

        int64_t n_conf = 0, nA2 = 0, E1 = 0, S1 = 0;
        for (int64_t t = 0; t < nA; ++t) {
            if (q_E) E1 += q_E[A[t]];
            if (q_S) S1 += q_S[A[t]];
            if (conf[t]) ++n_conf; else A[nA2++] = A[t];
        }
        if (phase_stats) {
            phase_stats[p * 5 + 0] = schedule[p];
            phase_stats[p * 5 + 1] = nA;
            phase_stats[p * 5 + 2] = n_conf;
            phase_stats[p * 5 + 3] = E1 - E0;
            phase_stats[p * 5 + 4] = S1 - S0;
        }
        nA = nA2;
        ran = p + 1;
    }
    free(A);
    free(conf);
    return ran;
}

/* Beam search of every query at one width, returning the whole final
 * worklist (ids, phi, squared distance; padded to L) and E, S per query. */
int32_t orc_search_lists(const orc_index *ix, const void *queries, const int32_t *ranges,
                         int64_t nq, int32_t L, uint32_t *out_ids, int32_t *out_phi,
                         float *out_d, int32_t *out_len, int64_t *q_E, int64_t *q_S)
{
    orc_ws w;
    if (!ws_init(&w, ix, L)) return -2;
    size_t qbytes = (size_t)ix->d * (ix->vec_dtype == ORC_VEC_U8 ? 1 : 4);
    for (int64_t i = 0; i < nq; ++i) {
        int len = 0;
        int64_t E = 0, S = 0;
        search_one(ix, &w, (const char *)queries + (size_t)i * qbytes,
                   ranges + i * ix->m * 2, L, &len, &E, &S);
        for (int a = 0; a < L; ++a) {
            out_ids[i * L + a] = a < len ? w.beam[a].id : ORC_PAD;
            out_phi[i * L + a] = a < len ? w.beam[a].phi : -1;
            out_d[i * L + a] = a < len ? w.beam[a].d : INFINITY;
        }
        out_len[i] = len;
        q_E[i] = E;
        q_S[i] = S;
    }
    ws_free(&w);
    return 0;
}

/* ------------------------------------------------------------------------
 * Exact filtered k-NN (Def. 1 with the matching function of Eq. 2): the k
 * valid points nearest the query by the distance above, ties by id; fewer
 * than k valid points give all of them (padded). n_valid[i] = |D_f|. */
int32_t orc_bruteforce(const orc_index *ix, const void *queries, const int32_t *ranges,
                       int64_t nq, int32_t k, uint32_t *ids, float *dists, int64_t *n_valid)
{
    orc_entry *best = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)(k + 1));
    if (!best) return -2;
    size_t qbytes = (size_t)ix->d * (ix->vec_dtype == ORC_VEC_U8 ? 1 : 4);
    for (int64_t i = 0; i < nq; ++i) {
        const void *q = (const char *)queries + (size_t)i * qbytes;
        const int32_t *rr = ranges + i * ix->m * 2;
        int nb = 0;
        int64_t nv = 0;
        for (int64_t v = 0; v < ix->n; ++v) {
            if (orc_phi(ix->attrs + v * ix->m, rr, ix->attr_dtypes, ix->m) != 0) continue;
            ++nv;
            orc_entry e;
            e.phi = 0; e.d = point_dist(ix, (uint32_t)v, q); e.id = (uint32_t)v; e.expanded = 0;
            if (nb == k && !entry_before(&e, &best[k - 1])) continue;
            int b = nb < k ? nb : k - 1;
            while (b > 0 && entry_before(&e, &best[b - 1])) { best[b] = best[b - 1]; --b; }
            best[b] = e;
            if (nb < k) ++nb;
        }
        for (int a = 0; a < k; ++a) {
            ids[i * k + a] = a < nb ? best[a].id : ORC_PAD;
            dists[i * k + a] = a < nb ? best[a].d : INFINITY;
        }
        if (n_valid) n_valid[i] = nv;
    }
    free(best);
    return 0;
}

/* ------------------------------------------------------------------------
 * Warm-start escalation (Sec. III-A "Redundancy Avoidance": a query that
 * runs at width L and then at alpha L should not redo the width-L work;
 * the width-L phase keeps its best L results and the next phase adds the
 * next alpha L - L). That paragraph is garbled; READING:
 *   - during phase p (width L_p) the query's sorted candidate list holds up
 *     to L_{p+1} entries (its own width at the last phase): new candidates
 *     are merged into it and it is cut to that capacity, but only entries
 *     among its first L_p are expanded (still one per iteration, the first
 *     unexpanded one), and the phase ends when those are all expanded;
 *   - the first L_p entries are the phase's worklist: the result and the
 *     confidence test (Eq. 3) read them; they equal the worklist of a fresh
 *     width-L_p search (the best L_p of a longer list of everything scored
 *     are the best L_p of everything scored), so phase 0 is unchanged;
 *   - a query that escalates keeps its list, expanded flags and set of
 *     scored nodes: phase p+1 continues from them instead of restarting at
 *     s. E and S count each phase's own new work.
 * Queries are independent, so each runs its phases back to back here (the
 * residual fraction tau is 0 in this mode). */
static void search_continue(const orc_index *ix, orc_ws *w, const void *q, const int32_t *rr, int32_t L_sel,
                            int32_t L_cap, int *len_io, int64_t *E, int64_t *S)
{
    orc_entry *beam = w->beam, *cand = w->cand, *tmp = w->tmp;
    int len = *len_io;
    for (;;) {
        int lim = len < L_sel ? len : L_sel;
        int j = 0;
        while (j < lim && beam[j].expanded) ++j;
        if (j == lim) break; /* the phase's worklist is fully expanded */
        beam[j].expanded = 1;
        uint32_t u = beam[j].id;
        *E += 1;

        int c = 0;
        for (int r = 0; r < ix->R; ++r) {
            uint32_t v = ix->adj[(int64_t)u * ix->R + r];
            if (v == ORC_PAD) continue;
            if (w->stamp[v] == w->cur) continue;
            w->stamp[v] = w->cur;
            cand[c++] = score(ix, v, q, rr, w->table);
        }
        *S += c;

        for (int a = 1; a < c; ++a) {
            orc_entry x = cand[a];
            int b = a - 1;
            while (b >= 0 && entry_before(&x, &cand[b])) { cand[b + 1] = cand[b]; --b; }
            cand[b + 1] = x;
        }
        int ia = 0, ib = 0, o = 0;
        while ((ia < len || ib < c) && o < L_cap) {
            if (ib >= c || (ia < len && entry_before(&beam[ia], &cand[ib])))
                tmp[o++] = beam[ia++];
            else
                tmp[o++] = cand[ib++];
        }
        memcpy(beam, tmp, sizeof(orc_entry) * (size_t)o);
        len = o;
    }
    *len_io = len;
}

int32_t orc_boa_warm(const orc_index *ix, const void *queries, const int32_t *ranges, int64_t nq, int32_t k,
                     const int32_t *schedule, int32_t n_phases, double eps, uint32_t *ids, float *dists,
                     int32_t *final_L, int64_t *q_E, int64_t *q_S, int64_t *phase_stats)
{
    if (nq <= 0 || n_phases <= 0) return 0;
    int32_t Lmax = 0;
    for (int p = 0; p < n_phases; ++p) if (schedule[p] > Lmax) Lmax = schedule[p];
    orc_ws w;
    if (!ws_init(&w, ix, Lmax)) return -2;
    float *vd = (float *)malloc(sizeof(float) * (size_t)Lmax);
    orc_entry *res = (orc_entry *)malloc(sizeof(orc_entry) * (size_t)Lmax);
    if (!vd || !res) { free(vd); free(res); ws_free(&w); return -2; }
    size_t qbytes = (size_t)ix->d * (ix->vec_dtype == ORC_VEC_U8 ? 1 : 4);
    if (phase_stats) memset(phase_stats, 0, sizeof(int64_t) * 5 * (size_t)n_phases);
    int32_t ran = 0;
    for (int64_t i = 0; i < nq; ++i) {
        const void *q = (const char *)queries + (size_t)i * qbytes;
        const int32_t *rr = ranges + i * ix->m * 2;
        int64_t Et = 0, St = 0;
        /* the entry point, scored and marked before the first expansion */
        ws_new_search(&w, ix->n);
        if (w.table) orc_pq_table(ix, q, w.table);
        int len = 1;
        w.beam[0] = score(ix, (uint32_t)ix->entry, q, rr, w.table);
        w.stamp[ix->entry] = w.cur;
        int64_t S0 = 1;
        for (int p = 0; p < n_phases; ++p) {
            int32_t L = schedule[p];
            int32_t cap = p + 1 < n_phases ? schedule[p + 1] : L;
            int64_t E = 0, S = S0;
            S0 = 0;
            search_continue(ix, &w, q, rr, L, cap, &len, &E, &S);
            int lim = len < L ? len : L;
            int n_valid = valid_results(ix, w.beam, lim, q, res);
            for (int a = 0; a < n_valid; ++a) vd[a] = res[a].d;
            for (int a = 0; a < k; ++a) {
                ids[i * k + a] = a < n_valid ? res[a].id : ORC_PAD;
                dists[i * k + a] = a < n_valid ? res[a].d : INFINITY;
            }
            final_L[i] = L;
            Et += E;
            St += S;
            int conf = orc_confident(vd, n_valid, k, eps);
            if (phase_stats) {
                phase_stats[p * 5 + 0] = L;
                phase_stats[p * 5 + 1] += 1;
                phase_stats[p * 5 + 2] += conf;
                phase_stats[p * 5 + 3] += E;
                phase_stats[p * 5 + 4] += S;
            }
            if (p + 1 > ran) ran = p + 1;
            if (conf) break;
        }
        if (q_E) q_E[i] = Et;
        if (q_S) q_S[i] = St;
    }
    free(vd);
    free(res);
    ws_free(&w);
    return ran;
}
