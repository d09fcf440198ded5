// Internal types shared by the host driver and the kernels of libboa.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "boa.h"

#define BOA_PAD 0xFFFFFFFFu
#define BOA_STATUS_OVERFLOW 1u
#define BOA_PROF_SLOTS 16
// Spill-bitmap log: a wave slot's bitmap is followed by a 4-word header
// (word 0: the number of logged ids, or BOA_LOG_DIRTY) and the ids whose
// bits were set since the bitmap was last clear.
#define BOA_LOG_HDR 4u
#define BOA_LOG_DIRTY 0xFFFFFFFFu

namespace boa {

// Worklist slots of a wave: a power of two at least L (entries past the
// list's length hold the largest key, so a search for an insertion point
// runs over a power-of-two span without bounds checks).
__host__ __device__ inline int32_t beam_slots(int32_t L)
{
    int32_t p = 2;
    while (p < L) p <<= 1;
    return p;
}

// A float32 attribute cell as an order-preserving int32: for floats a, b
// that are not NaN, a <= b exactly when f32_ord(a) <= f32_ord(b) (both zeros
// map to 0, so -0 and +0 compare equal as floats do). NaN maps to INT32_MIN,
// below the image of every other value (-inf maps to -2^31 + 2^23 - 1).
__host__ __device__ inline int32_t f32_ord(uint32_t x)
{
    const uint32_t mag = x & 0x7FFFFFFFu;
    if (mag == 0u) return 0;
    if (mag > 0x7F800000u) return (int32_t)0x80000000u;
    return (int32_t)(x ^ ((uint32_t)((int32_t)x >> 31) & 0x7FFFFFFFu));
}

// Device-resident index. Attribute rows are padded to m_pad in {1, 2, 4, 8}
// cells so one aligned vector load fetches a whole record.
struct IndexView {
    const void *vectors;      // n x d (float32 or uint8)
    const int32_t *attrs;     // n x m_pad cells; float32 columns as f32_ord
    const uint32_t *adj;      // n x R
    int64_t n;
    int32_t d, m, m_pad, R;
    uint32_t entry;
    uint32_t f32_mask;        // bit j set: attribute j is float32
};

struct PhaseArgs {
    IndexView ix;
    const void *queries;      // nq x d
    const int32_t *ranges;    // nq x m x 2
    const uint32_t *active;   // active list of this phase (query indices)
    const uint32_t *n_active; // its length (device)
    uint32_t t_begin, t_end;  // slice of the active list served by this launch
    uint32_t *queue;          // work counter of this launch
    uint8_t *conf;            // per active slot: confident flag
    uint32_t *ids;
    float *dists;
    int32_t *final_L;
    uint8_t *qstat;           // [phase][query]: 0 not run, 1 ran, 2 ran+confident, +4 spilled
    uint32_t *qE, *qS;        // [phase][query]: expansions, scored
    int64_t nq;               // stride of the per-phase arrays
    uint32_t *user_E, *user_S;// optional per-query totals over phases
    uint32_t *bits;           // per wave slot (slot_words u32): spill bitmap, then its log
    uint32_t bits_words;      // bitmap words (a multiple of 4)
    uint32_t slot_words;      // bits_words + BOA_LOG_HDR + log_cap
    uint32_t log_cap;         // ids the log holds (0: no log, every clear is whole)
    uint32_t *status;
    double eps;
    uint32_t tau_count;       // the phase runs only if n_active > tau_count
    int32_t k;
    int32_t sched[BOA_MAX_PHASES]; // phase widths
    int32_t p_begin, p_end;   // phases run by this launch (one, or all when fused)
    int32_t write_conf;       // record each query's confidence for a compaction/append
    int32_t warm;             // warm-start escalation: phases continue from the previous one's state
    int32_t pq;               // traverse with product-quantised distances, re-rank exactly
    int32_t pq_m;             // subspaces (16 centroids each)
    const float *pq_cb;       // pq_m x 16 x d/pq_m
    const uint8_t *pq_codes;  // n x pq_m/2, subspace 2b in the low nibble of byte b
    int32_t vec_u8;           // the vectors are uint8 (the exact re-rank's arithmetic)
    int32_t L_alloc;          // widest of them: sizes the per-wave LDS
    int32_t h_log2;           // log2 of the LDS visited-table slots (16-bit entries)
    int32_t vis_bitmap;       // 1: the visited set is instead an LDS bitmap over all n ids
    uint32_t vis_words;       // its size in 32-bit words (a multiple of 4)
    uint32_t id_bits;         // bits of the largest id (ceil(log2 n))
    int32_t lds_per_wave, waves_per_block;
    uint32_t slot_base;
    unsigned long long *prof; // per wave slot: BOA_PROF_SLOTS stage counters (profiling builds)
};

struct CompactArgs {
    const uint32_t *in;
    const uint32_t *n_in;
    const uint8_t *conf;
    uint32_t *out;
    uint32_t *n_out;
    uint32_t tau_count;
};

struct AppendArgs {
    const uint32_t *in;       // slice of the active list
    const uint8_t *conf;      // its confidence flags
    uint32_t n;               // slice length
    uint32_t *pool;           // destination pool
    uint32_t *pool_count;     // its length (device; read, then advanced)
};

struct InitArgs {
    uint32_t *active0;
    uint32_t *n_active;
    uint32_t *counters;
    uint8_t *qstat;
    uint32_t *user_E, *user_S;
    uint32_t *status;
    int64_t nq;
    int32_t n_phases;
    int32_t n_counters;
    // spill-log headers of the first reset_slots wave slots set to
    // BOA_LOG_DIRTY (their bitmaps' contents unknown)
    uint32_t *bits;
    uint32_t slot_words, bits_words;
    uint64_t reset_slots;
};

// Index construction (boa_build.hip): the medoid entry point, and the graph
// when the caller passes no adjacency.
struct BuildStats {
    int32_t K;                 // exact nearest candidates per point
    int64_t edges;             // edges of the final graph
    int64_t repaired;          // in-edges added to reach every point from s
    int64_t repair_fallback;   // of which not from the point's own candidates
    int64_t attr_edges;        // edges from the attribute-threshold passes
};
hipError_t compute_medoid(const void *d_vectors, int64_t n, int32_t d, int vec_dtype, uint32_t *entry);
// h_attrs: HOST n x m cells (float32 columns flagged in f32_mask), or null
// for a graph from vector distances only
hipError_t build_graph(const void *d_vectors, int64_t n, int32_t d, int vec_dtype, int32_t R, uint32_t entry,
                       const int32_t *h_attrs, int32_t m, uint32_t f32_mask, float alpha, int32_t attr_levels,
                       uint32_t *d_adj, BuildStats *stats);

// wide: the scorer variant with twice the rows in flight (for launches that
// hold few waves per CU)
hipError_t launch_phase(const PhaseArgs &a, int vec_dtype, int blocks, hipStream_t st, bool wide = false);
// pq_m > 0: the product-quantised scorer with that many subspaces
int phase_occupancy(int vec_dtype, int d, int wpb, size_t lds, bool wide = false, int pq_m = 0);
// per-wave LDS bytes the distance scorer keeps (its copy of the query, or
// the product-quantisation distance table)
int scorer_lds_bytes(int vec_dtype, int d, bool wide = false, int pq_m = 0);
// The escalation launch of a split search with two waves per query (LDS
// bitmap visited set, exact distances): its LDS per block, resident blocks
// per CU, and the launch (lds_per_wave carries the block's LDS bytes).
size_t pair_lds_bytes(int32_t L, uint32_t vis_words, int scorer_lds);
int pair_occupancy(int vec_dtype, int d, size_t lds);
hipError_t launch_pair(const PhaseArgs &a, int vec_dtype, int blocks, hipStream_t st);
hipError_t launch_compact(const CompactArgs &a, hipStream_t st);
hipError_t launch_append(const AppendArgs &a, hipStream_t st);
hipError_t launch_init(const InitArgs &a, hipStream_t st);

}  // namespace boa
