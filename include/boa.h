/*
 * boa.h — C ABI of the MI355X (gfx950) filtered beam search with online
 * beamwidth adaptation ("BOA: Beamwidth Online Adaptation for
 * Filtered-ANNS on a GPU").
 *
 * Problem (Sec. II, Def. 1 and Def. 2): each base point carries a vector
 * and m numeric attributes; a query carries a vector and one inclusive
 * range [lo, hi] per attribute (Eq. 2). The answer is the k points nearest
 * to the query vector (Euclidean) among those satisfying every range.
 *
 * Method: every query is searched first at a narrow beamwidth L0; queries
 * whose result fails the confidence test (Eq. 3) are compacted on the
 * device and searched again, from scratch, at the next wider width
 * (Alg. 1); each search is the filter-aware beam search of Alg. 2 with
 * exact squared-L2 distances. BOA+ (Sec. III-A "Pipelining Multiple
 * Batches") issues the first phase as sub-batches on one stream while the
 * pooled survivors are escalated on a second stream.
 *
 * Conventions for every entry point:
 *   - Return value: BOA_OK (0) or a negative BOA_E* code; no C++ exception
 *     crosses this boundary and the library never aborts. On a non-zero
 *     return, boa_last_error() describes the failure (thread-local string).
 *   - Validation happens before any device work: on BOA_EINVAL the output
 *     buffers are untouched.
 *   - Attribute and range cells are 4 bytes: int32 for BOA_ATTR_I32
 *     columns, the IEEE bit pattern of a float32 for BOA_ATTR_F32 columns.
 *   - Distances are squared Euclidean distances in float32 (exact integers
 *     for uint8 data). float32 distances use one fixed summation order:
 *     16 partial sums, chunk c = dims 4c..4c+3 accumulated into partial
 *     c mod 16 by fused multiply-add of the float32 difference, chunks in
 *     increasing order, then the partials summed pairwise (p += p+8, +4,
 *     +2, +1).
 *   - Search ordering is lexicographic on (number of violated predicates,
 *     distance, id): the filter penalty of Alg. 2 taken larger than any
 *     distance, ties broken by id.
 *   - Not thread-safe per index: one boa_search at a time per boa_index.
 */
#ifndef BOA_H
#define BOA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct boa_index boa_index; /* opaque; owns all of its device memory */

enum {
    BOA_OK = 0,
    BOA_EINVAL = -1,       /* invalid argument */
    BOA_ENOMEM = -2,       /* host or device allocation failed */
    BOA_EHIP = -3,         /* HIP runtime error */
    BOA_EUNSUPPORTED = -4, /* valid but not supported by this build */
    BOA_EOVERFLOW = -5     /* a per-query visited table overflowed (results invalid) */
};

enum { BOA_VEC_F32 = 0, BOA_VEC_U8 = 1 };
enum { BOA_ATTR_I32 = 0, BOA_ATTR_F32 = 1 };

#define BOA_MAX_M 8          /* attributes per point */
#define BOA_MAX_R 64         /* graph out-degree */
#define BOA_MAX_L 2048       /* beamwidth */
#define BOA_MAX_PHASES 32
#define BOA_MAX_N ((int64_t)1 << 24) /* ids are packed into 24 bits */
#define BOA_MAX_BUILD_N ((int64_t)2 << 20) /* graph construction inside the library */

/*
 * Build an index from host arrays (copied into device memory; the caller
 * may free its arrays on return).
 *   vectors     host, row-major n x d; float32 (BOA_VEC_F32) or uint8 (BOA_VEC_U8).
 *               d % 4 == 0 (float32) or d % 16 == 0 (uint8); d <= 1024.
 *   attrs       host, row-major n x m 4-byte cells; 1 <= m <= BOA_MAX_M.
 *   attr_dtypes host, m entries of BOA_ATTR_I32 / BOA_ATTR_F32.
 *   adjacency   host, row-major n x R uint32 neighbour ids, padded with
 *               0xFFFFFFFF; 1 <= R <= BOA_MAX_R. A row may not hold its own
 *               id, nor any id twice.
 *               NULL: the library builds the graph (Sec. II "Graph
 *               construction"; boa_build_params): DiskANN alpha-pruning of
 *               each point's min(2R, 128) exact nearest neighbours, then of
 *               its forward and reverse neighbours; attribute-aware edges
 *               from JAG-style threshold passes (R >= 8); every row leaves
 *               one slot free, and every point is made reachable from the
 *               entry point through an in-edge from its nearest reachable
 *               candidate. Needs n <= BOA_MAX_BUILD_N (the candidates come
 *               from brute-force scans), else BOA_EUNSUPPORTED.
 *   R           the row width, 1 <= R <= BOA_MAX_R: one neighbour per lane of
 *               a 64-wide wavefront.
 *   entry       the entry point s of every search (Alg. 2), 0 <= entry < n;
 *               -1: the medoid, the point nearest (float64) to the float64
 *               centroid of the vectors, ties to the lowest id.
 *   n           1 <= n < BOA_MAX_N.
 *   out         receives the index; free it with boa_free_index.
 * Errors: BOA_EINVAL (bad sizes, null pointers, out-of-range ids in the
 * adjacency), BOA_EUNSUPPORTED, BOA_ENOMEM, BOA_EHIP.
 */
int boa_build_index_from_arrays(const void *vectors, int64_t n, int32_t d, int32_t vec_dtype,
                                const int32_t *attrs, int32_t m, const int32_t *attr_dtypes,
                                const uint32_t *adjacency, int32_t R, int64_t entry,
                                boa_index **out);

/* Graph construction parameters (used when adjacency is NULL). */
typedef struct {
    double alpha;        /* pruning slack of DiskANN's dominance rule: v is dropped
                            when a kept w has alpha * d(w, v) <= d(u, v) (Euclidean);
                            1 <= alpha <= 4; default 1.2 */
    int32_t attr_levels; /* attribute-aware passes (JAG threshold pruning, Sec. II
                            "Graph construction"), 0..4; default 4. Level l keeps, for
                            each point, R/8 alpha-pruned nearest vectors among the
                            points whose attribute distance (the largest gap of
                            per-column quantile ranks) is within the point's
                            0.1% / 1% / 5% / 20% quantile of that distance to an evenly
                            spaced sample of 4096 points. The vector-distance pass
                            keeps the rest of the row but one slot. Needs R >= 8. */
} boa_build_params;

void boa_default_build_params(boa_build_params *bp);

/* boa_build_index_from_arrays with explicit graph construction parameters
 * (bp must not be NULL). */
int boa_build_index_ex(const void *vectors, int64_t n, int32_t d, int32_t vec_dtype, const int32_t *attrs,
                       int32_t m, const int32_t *attr_dtypes, const uint32_t *adjacency, int32_t R,
                       int64_t entry, const boa_build_params *bp, boa_index **out);

/* Search parameters (Alg. 1 inputs). boa_default_params fills the defaults. */
typedef struct {
    int32_t k;              /* neighbours returned; 1 <= k <= L of the first phase */
    int32_t L0;             /* first-phase beamwidth (L_min of Alg. 1) */
    int32_t Lmax;           /* widest beamwidth; the phase at Lmax is the last */
    double alpha;           /* growth factor > 1: L <- min(ceil(alpha * L), Lmax); default 2 */
    double eps;             /* confidence threshold of Eq. 3; default 0.05 */
    double tau;             /* residual fraction: a phase runs while more than tau*nq
                               queries are active; 0 <= tau < 1; default 0 */
    int32_t fixed_L;        /* > 0: a single non-adaptive phase at this width (the
                               fixed-beamwidth baseline); overrides L0/Lmax/schedule */
    int32_t boa_plus;       /* 1: BOA+ sub-batched first phase overlapped with escalation */
    int32_t sub_batches;    /* BOA+ first-phase sub-batches; default 10 */
    int32_t lds_hash_slots; /* 0: automatic; else a power of two in [64, 16384] that forces
                               the 16-bit slots of the per-wave LDS visited table (tests
                               force spills to the HBM bitmap); at least 8 * 2^(B-15)
                               for ids of B bits */
    const int32_t *schedule; /* optional host array of explicit phase widths
                                (strictly increasing); overrides L0/Lmax/alpha */
    int32_t n_schedule;
    int32_t fused;          /* 1: run every phase in one persistent launch, each wave
                               carrying its query from width to width without waiting
                               for the other queries (identical results, since every
                               phase restarts the search; needs tau == 0). 2: split:
                               the first phase in one launch, then (after compaction
                               and a 4-byte read of the survivor count) every later
                               phase in one persistent launch over the survivors, whose
                               waves get the largest visited table that still lets all
                               survivors run at once (identical results; needs
                               tau == 0). 0: one launch per phase with device-side
                               compaction between them. */
    int32_t warm_start;     /* 1: warm-start escalation (Sec. III-A "Redundancy
                               Avoidance"): during a phase of width L the sorted list
                               keeps up to the next phase's width, only its first L
                               entries are expanded and read by the result and Eq. 3,
                               and an escalated query continues from that list and its
                               visited set instead of restarting at the entry point.
                               The first phase is unchanged; later phases differ from a
                               restart. Runs in the fused mode only (fused = 1, so
                               tau == 0), else BOA_EUNSUPPORTED. 0: every phase restarts. */
    int32_t pq;             /* 1: traverse with product-quantised distances (Alg. 2 "PQDist",
                               the index needs boa_set_pq), then at each phase's end
                               re-rank the phase's valid worklist entries by exact
                               distance (Sec. III-B step 8); the result and Eq. 3 read
                               the re-ranked entries. k <= 128. 0: exact distances. */
    int32_t escalation_waves; /* split mode (fused = 2), when the escalation launch keeps
                               its visited set as an LDS bitmap over all ids and the
                               distances are exact: 0 (default) two waves per query, one
                               merging the worklist while the other runs the visited test,
                               gathers and scoring of the node it expects next (the
                               selected node when the guess misses; identical results);
                               1: one wave per query. Ignored elsewhere. */
} boa_params;

void boa_default_params(boa_params *p);

/*
 * Batched adaptive filtered search.
 *   queries   DEVICE, nq x d, same element type as the index vectors.
 *   ranges    DEVICE, nq x m x 2 cells [lo, hi] (inclusive), per-column type;
 *             an unconstrained attribute is [INT32_MIN, INT32_MAX] or [-inf, +inf].
 *   nq        >= 0 (0 is a no-op).
 *   ids       DEVICE, nq x k uint32: ids of the valid points found, nearest first;
 *             0xFFFFFFFF where fewer than k valid points were found.
 *   dists     DEVICE, nq x k float32 squared distances (+inf in padded slots).
 *   final_L   DEVICE, nq int32: beamwidth of the phase that produced the result.
 *   expansions, scored  DEVICE nq uint32 each, or NULL: per query, nodes expanded
 *             and nodes scored, summed over the phases the query ran in.
 *   stream    hipStream_t of the caller (NULL = default stream). Device buffers
 *             must be valid on it. The call returns after the results are
 *             complete (it synchronises the stream once at the end).
 * Errors: BOA_EINVAL, BOA_EUNSUPPORTED, BOA_ENOMEM, BOA_EHIP, BOA_EOVERFLOW.
 */
int boa_search(boa_index *idx, const void *queries, const int32_t *ranges, int64_t nq,
               const boa_params *p, uint32_t *ids, float *dists, int32_t *final_L,
               uint32_t *expansions, uint32_t *scored, void *stream);

/*
 * Allocation-free variant of boa_search, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and error codes
 * as boa_search; it calls no hipMalloc, hipFree or other allocating routine.
 *   - Its work memory (active lists, counters, confidence flags, the visited
 *     spill bitmaps) lives in one file-scope device array of
 *     BOA_NOALLOC_SCRATCH_MB MiB per GPU, held by the library until the
 *     process ends. Every call on a GPU shares that GPU's array: calls that
 *     overlap on one GPU (other streams, other threads) race and must be
 *     serialised by the caller. What must start at zero is cleared by a fill
 *     kernel at the start of each call.
 *   - nq <= BOA_NOALLOC_MAX_NQ, else BOA_EINVAL before any device work.
 *   - BOA+ (boa_plus = 1) returns BOA_EUNSUPPORTED (it needs a second
 *     stream). The other modes run; where the spill bitmaps of the planned
 *     grid (n/8 bytes per resident wave) do not fit the array, the
 *     persistent grid is made smaller (same results, less parallelism), and
 *     an index whose single block does not fit returns BOA_EUNSUPPORTED.
 *   - It keeps no statistics: boa_get_stats afterwards reports no search.
 * It synchronises `stream` before returning, like boa_search.
 */
#define BOA_NOALLOC_SCRATCH_MB 64
#define BOA_NOALLOC_MAX_NQ (1 << 18)
int boa_search_noalloc(boa_index *idx, const void *queries, const int32_t *ranges, int64_t nq,
                       const boa_params *p, uint32_t *ids, float *dists, int32_t *final_L,
                       uint32_t *expansions, uint32_t *scored, void *stream);

/* Statistics of the last boa_search on this index, one row per phase. */
typedef struct {
    int32_t L;              /* phase beamwidth */
    int32_t active;         /* queries searched in the phase */
    int32_t confident;      /* of which resolved by the confidence test */
    int32_t launches;       /* kernel launches of the phase (BOA+: sub-batches) */
    int64_t expansions;     /* nodes expanded, summed over the phase's queries */
    int64_t scored;         /* nodes scored (distance + predicates) */
    double gathered_bytes;  /* algorithmic bytes the phase had to read */
    float kernel_ms;        /* device time of the phase's search launches */
} boa_phase_stats;

typedef struct {
    int32_t n_phases;
    int32_t waves_per_block, blocks; /* launch shape of the first phase */
    int32_t lds_hash_slots;          /* of the first phase */
    int64_t spilled_queries;         /* query-phases whose visited set left LDS */
    float total_ms;                  /* device time of the whole search */
    /* accumulated since boa_reset_counters: searches, search-kernel launches,
       and their summed device time (HIP events around every launch) */
    int64_t cum_searches, cum_launches;
    double cum_kernel_ms;
    boa_phase_stats phase[BOA_MAX_PHASES];
    /* accumulated like cum_*, split by the phase a launch starts at (a fused
       launch counts under phase 0, a split search's second launch under 1) */
    int64_t cum_phase_launches[BOA_MAX_PHASES];
    double cum_phase_kernel_ms[BOA_MAX_PHASES];
} boa_stats;

/* Statistics of the last search (per phase) plus the accumulated counters.
 * Copies per-query counters back from the device: call it outside timed code. */
int boa_get_stats(const boa_index *idx, boa_stats *out);

/* Zero the accumulated counters of boa_stats. */
int boa_reset_counters(boa_index *idx);

/*
 * Product-quantisation data of an index (Alg. 2 "PQDist"; Sec. III-B), copied
 * to the device (the caller may free its arrays on return).
 *   codebook  HOST, M x 16 x (d / M) float32: 16 centroids per subspace of
 *             d / M consecutive dimensions.
 *   codes     HOST, n x M / 2 bytes: byte b holds the centroid of subspace 2b
 *             in its low nibble and of subspace 2b + 1 in its high nibble.
 *   M         even, <= 256, dividing d.
 * The per-query distance table entry (m, c) is the float32 fused
 * multiply-add chain over the subspace's dimensions of (q - centroid)^2; the
 * asymmetric distance adds a point's table entries in 16 partial sums
 * (subspace m into partial m mod 16, increasing m) summed pairwise.
 * Errors: BOA_EINVAL, BOA_ENOMEM, BOA_EHIP. */
int boa_set_pq(boa_index *idx, const float *codebook, const uint8_t *codes, int32_t M);

/* The graph and entry point an index searches (e.g. the ones the library
 * built). adjacency: HOST n x R uint32, or NULL; entry: the entry point s,
 * or NULL; repaired: in-edges the library's construction added to reach
 * every point (-1 when the caller passed the adjacency), or NULL. */
int boa_get_graph(const boa_index *idx, uint32_t *adjacency, int64_t *entry, int64_t *repaired);

void boa_free_index(boa_index *idx);

const char *boa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BOA_H */
