// Host side of libboa: index upload, validation, the multi-phase driver of
// Alg. 1 (device-side compaction, no host round trip between phases), the
// BOA+ two-stream schedule, and statistics.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "boa_internal.h"

using namespace boa;

namespace {

// last error message: a fixed per-thread buffer, so that reporting an error
// allocates nothing
thread_local char g_err[512];

int fail(int code, const char *msg)
{
    std::snprintf(g_err, sizeof(g_err), "%s", msg);
    return code;
}

int fail(int code, const std::string &msg) { return fail(code, msg.c_str()); }

#define HIP_TRY(expr)                                                                  \
    do {                                                                               \
        hipError_t e_ = (expr);                                                        \
        if (e_ != hipSuccess)                                                          \
            return fail(BOA_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_));  \
    } while (0)

template <class T>
int dalloc(T **p, size_t count)
{
    *p = nullptr;
    if (count == 0) count = 1;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(p), count * sizeof(T));
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        return fail(BOA_ENOMEM, "hipMalloc of " + std::to_string(count * sizeof(T)) + " bytes failed");
    }
    return BOA_OK;
}

template <class T>
void dfree(T *&p)
{
    if (p) (void)hipFree(p);
    p = nullptr;
}

uint32_t next_pow2(uint64_t x)
{
    uint32_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

int ilog2(uint32_t x)
{
    int r = 0;
    while ((1u << r) < x) ++r;
    return r;
}

struct PhasePlan {
    int32_t L;
    int32_t h_slots, wpb, blocks, lds_per_wave;
    int32_t vis_bitmap;  // visited set as an LDS bitmap over all ids (0: hashed table)
    int32_t launches;
    int64_t capacity;   // waves resident at once on the whole GPU
    bool wide;          // scorer variant with twice the rows in flight
};

}  // namespace

// Scratch of the allocation-free search (boa_search_noalloc): one array per
// GPU the library runs on, held until the process ends. Host code never
// names it directly (in host code the name is a stand-in, not a device
// address); it uses the address hipGetSymbolAddress returns for the current
// device.
static __device__ __align__(256) unsigned char scratch[(size_t)BOA_NOALLOC_SCRATCH_MB << 20];

struct boa_index {
    int device = 0;
    int num_cu = 0;
    size_t lds_per_block_max = 65536;
    size_t lds_per_block_hw = 65536;   // the device's own limit (bitmap escalations only)
    int vec_dtype = 0;
    IndexView view{};
    void *d_vectors = nullptr;
    int32_t *d_attrs = nullptr;
    uint32_t *d_adj = nullptr;

    float *d_pq_cb = nullptr;        // product quantisation (boa_set_pq)
    uint8_t *d_pq_codes = nullptr;
    int32_t pq_m = 0;
    bool built_graph = false;        // the graph was constructed by the library
    BuildStats build_stats{};

    // workspace, grown on demand
    int64_t nq_cap = 0;
    int32_t ph_cap = 0;
    uint32_t *active[2] = {nullptr, nullptr};
    uint32_t *n_active = nullptr;    // BOA_MAX_PHASES + 1
    uint32_t *counters = nullptr;    // work counters, n_counters
    int32_t n_counters = 0;
    uint8_t *conf = nullptr;         // nq
    uint8_t *qstat = nullptr;        // ph_cap x nq
    uint32_t *qE = nullptr, *qS = nullptr;  // ph_cap x nq
    uint32_t *status = nullptr;
    uint32_t *bits = nullptr;        // visited spill bitmaps and their logs, slot_words per wave slot
    uint32_t bits_words = 0;
    uint32_t slot_words = 0, log_cap = 0;
    bool logs_fresh = false;         // the logs' headers are not yet set (next search sets them)
    uint64_t slots_cap = 0;
    uint32_t *pool = nullptr;        // BOA+ survivor pools (ph_cap x nq)
    hipStream_t aux = nullptr;       // BOA+ second stream
    std::vector<hipEvent_t> ev_start, ev_end;  // per launch

    // last search
    int64_t last_nq = 0;
    int32_t last_k = 0;
    int32_t last_pq_m = 0;
    std::vector<PhasePlan> plans;
    std::vector<std::pair<int, int>> launch_phase;  // (phase, event index)
    hipEvent_t ev_all0 = nullptr, ev_all1 = nullptr;
    hipEvent_t ev_pool = nullptr, ev_join = nullptr;   // BOA+ cross-stream ordering
    bool have_stats = false;
    int64_t cum_searches = 0, cum_launches = 0;
    double cum_kernel_ms = 0.0;
    int64_t cum_phase_launches[BOA_MAX_PHASES] = {};
    double cum_phase_kernel_ms[BOA_MAX_PHASES] = {};
};

extern "C" {

const char *boa_last_error(void) { return g_err; }

void boa_default_params(boa_params *p)
{
    if (!p) return;
    std::memset(p, 0, sizeof(*p));
    p->k = 10;
    p->L0 = 16;
    p->Lmax = 512;
    p->alpha = 2.0;
    p->eps = 0.05;
    p->tau = 0.0;
    p->fixed_L = 0;
    p->boa_plus = 0;
    p->sub_batches = 10;
    p->lds_hash_slots = 0;
    p->schedule = nullptr;
    p->n_schedule = 0;
    p->fused = 0;
}

void boa_free_index(boa_index *ix)
{
    if (!ix) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(ix->device);
    dfree(ix->d_vectors);
    dfree(ix->d_attrs);
    dfree(ix->d_adj);
    dfree(ix->d_pq_cb);
    dfree(ix->d_pq_codes);
    dfree(ix->active[0]);
    dfree(ix->active[1]);
    dfree(ix->n_active);
    dfree(ix->counters);
    dfree(ix->conf);
    dfree(ix->qstat);
    dfree(ix->qE);
    dfree(ix->qS);
    dfree(ix->status);
    dfree(ix->bits);
    dfree(ix->pool);
    for (auto e : ix->ev_start) (void)hipEventDestroy(e);
    for (auto e : ix->ev_end) (void)hipEventDestroy(e);
    if (ix->ev_all0) (void)hipEventDestroy(ix->ev_all0);
    if (ix->ev_all1) (void)hipEventDestroy(ix->ev_all1);
    if (ix->ev_pool) (void)hipEventDestroy(ix->ev_pool);
    if (ix->ev_join) (void)hipEventDestroy(ix->ev_join);
    if (ix->aux) (void)hipStreamDestroy(ix->aux);
    (void)hipSetDevice(cur);
    delete ix;
}

void boa_default_build_params(boa_build_params *bp)
{
    if (!bp) return;
    std::memset(bp, 0, sizeof(*bp));
    bp->alpha = 1.2;
    bp->attr_levels = 4;
}

int boa_build_index_from_arrays(const void *vectors, int64_t n, int32_t d, int32_t vec_dtype,
                                const int32_t *attrs, int32_t m, const int32_t *attr_dtypes,
                                const uint32_t *adjacency, int32_t R, int64_t entry, boa_index **out)
{
    boa_build_params bp;
    boa_default_build_params(&bp);
    return boa_build_index_ex(vectors, n, d, vec_dtype, attrs, m, attr_dtypes, adjacency, R, entry, &bp, out);
}

int boa_build_index_ex(const void *vectors, int64_t n, int32_t d, int32_t vec_dtype, const int32_t *attrs,
                       int32_t m, const int32_t *attr_dtypes, const uint32_t *adjacency, int32_t R, int64_t entry,
                       const boa_build_params *bp, boa_index **out)
{
    if (!out) return fail(BOA_EINVAL, "out is NULL");
    if (!bp) return fail(BOA_EINVAL, "NULL build parameters");
    if (!(bp->alpha >= 1.0 && bp->alpha <= 4.0)) return fail(BOA_EINVAL, "alpha must be in [1, 4]");
    if (bp->attr_levels < 0 || bp->attr_levels > 4) return fail(BOA_EINVAL, "attr_levels must be in [0, 4]");
    *out = nullptr;
    if (!vectors || !attrs || !attr_dtypes) return fail(BOA_EINVAL, "NULL input array");
    if (n < 1 || n >= BOA_MAX_N) return fail(BOA_EINVAL, "n out of range [1, 2^24)");
    if (!adjacency && n > BOA_MAX_BUILD_N)
        return fail(BOA_EUNSUPPORTED, "graph construction by exact nearest neighbours is limited to "
                                      "BOA_MAX_BUILD_N points; pass an adjacency");
    if (vec_dtype != BOA_VEC_F32 && vec_dtype != BOA_VEC_U8) return fail(BOA_EINVAL, "bad vec_dtype");
    if (d < 4 || d > 1024) return fail(BOA_EINVAL, "d out of range [4, 1024]");
    if (vec_dtype == BOA_VEC_F32 && d % 4) return fail(BOA_EINVAL, "float32 vectors need d % 4 == 0");
    if (vec_dtype == BOA_VEC_U8 && d % 16) return fail(BOA_EINVAL, "uint8 vectors need d % 16 == 0");
    if (m < 1 || m > BOA_MAX_M) return fail(BOA_EINVAL, "m out of range [1, 8]");
    if (R < 1 || R > BOA_MAX_R) return fail(BOA_EINVAL, "R out of range [1, 64]");
    if (entry < -1 || entry >= n) return fail(BOA_EINVAL, "entry out of range (-1: the medoid)");
    uint32_t f32_mask = 0;
    for (int j = 0; j < m; ++j) {
        if (attr_dtypes[j] == BOA_ATTR_F32) f32_mask |= 1u << j;
        else if (attr_dtypes[j] != BOA_ATTR_I32) return fail(BOA_EINVAL, "bad attribute dtype");
    }
    if (adjacency) {
        std::vector<uint32_t> row((size_t)R);
        for (int64_t u = 0; u < n; ++u) {
            int cnt = 0;
            for (int r = 0; r < R; ++r) {
                uint32_t v = adjacency[u * R + r];
                if (v == BOA_PAD) continue;
                if ((int64_t)v >= n) return fail(BOA_EINVAL, "adjacency id out of range");
                if ((int64_t)v == u) return fail(BOA_EINVAL, "adjacency row holds its own id");
                row[cnt++] = v;
            }
            std::sort(row.begin(), row.begin() + cnt);
            if (std::adjacent_find(row.begin(), row.begin() + cnt) != row.begin() + cnt)
                return fail(BOA_EINVAL, "adjacency row holds an id twice");
        }
    }

    boa_index *ix = new (std::nothrow) boa_index();
    if (!ix) return fail(BOA_ENOMEM, "host allocation failed");
    if (hipGetDevice(&ix->device) != hipSuccess) {
        delete ix;
        return fail(BOA_EHIP, "hipGetDevice failed (no GPU?)");
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, ix->device) != hipSuccess) {
        delete ix;
        return fail(BOA_EHIP, "hipGetDeviceProperties failed");
    }
    ix->num_cu = prop.multiProcessorCount;
    ix->lds_per_block_max = std::min<size_t>(prop.sharedMemPerBlock, 65536);
    ix->lds_per_block_hw = prop.sharedMemPerBlock;
    ix->vec_dtype = vec_dtype;

    const int m_pad = m <= 1 ? 1 : (m <= 2 ? 2 : (m <= 4 ? 4 : 8));
    const size_t esz = vec_dtype == BOA_VEC_U8 ? 1 : 4;
    int rc;
    if ((rc = dalloc(reinterpret_cast<uint8_t **>(&ix->d_vectors), (size_t)n * d * esz)) ||
        (rc = dalloc(&ix->d_attrs, (size_t)n * m_pad)) || (rc = dalloc(&ix->d_adj, (size_t)n * R))) {
        boa_free_index(ix);
        return rc;
    }
    // the search's copy of the attributes: rows padded to m_pad cells, float32
    // columns as order-preserving integers, so that every range test is an
    // integer compare (the caller's array is not modified)
    std::vector<int32_t> padded;
    const int32_t *attr_src = attrs;
    if (m_pad != m || f32_mask != 0) {
        try {
            padded.assign((size_t)n * m_pad, 0);
        } catch (...) {
            boa_free_index(ix);
            return fail(BOA_ENOMEM, "host allocation failed");
        }
        for (int64_t i = 0; i < n; ++i) {
            int32_t *dst = &padded[(size_t)i * m_pad];
            const int32_t *src = attrs + (size_t)i * m;
            for (int j = 0; j < m; ++j)
                dst[j] = ((f32_mask >> j) & 1u) ? f32_ord((uint32_t)src[j]) : src[j];
        }
        attr_src = padded.data();
    }
    if (hipMemcpy(ix->d_vectors, vectors, (size_t)n * d * esz, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(ix->d_attrs, attr_src, (size_t)n * m_pad * 4, hipMemcpyHostToDevice) != hipSuccess ||
        (adjacency && hipMemcpy(ix->d_adj, adjacency, (size_t)n * R * 4, hipMemcpyHostToDevice) != hipSuccess)) {
        boa_free_index(ix);
        return fail(BOA_EHIP, "index upload failed");
    }
    // the entry point s of Alg. 2: the medoid unless the caller names one
    if (entry < 0) {
        uint32_t s = 0;
        hipError_t e = compute_medoid(ix->d_vectors, n, d, vec_dtype, &s);
        if (e != hipSuccess) {
            boa_free_index(ix);
            return fail(BOA_EHIP, std::string("medoid computation failed: ") + hipGetErrorString(e));
        }
        entry = s;
    }
    if (!adjacency) {
        BuildStats bs{};
        hipError_t e = build_graph(ix->d_vectors, n, d, vec_dtype, R, (uint32_t)entry, attrs, m, f32_mask,
                                   (float)bp->alpha, bp->attr_levels, ix->d_adj, &bs);
        if (e != hipSuccess) {
            boa_free_index(ix);
            return fail(e == hipErrorOutOfMemory ? BOA_ENOMEM : BOA_EHIP,
                        std::string("graph construction failed: ") + hipGetErrorString(e));
        }
        ix->built_graph = true;
        ix->build_stats = bs;
    }
    ix->view.vectors = ix->d_vectors;
    ix->view.attrs = ix->d_attrs;
    ix->view.adj = ix->d_adj;
    ix->view.n = n;
    ix->view.d = d;
    ix->view.m = m;
    ix->view.m_pad = m_pad;
    ix->view.R = R;
    ix->view.entry = (uint32_t)entry;
    ix->view.f32_mask = f32_mask;
    if (hipEventCreate(&ix->ev_all0) != hipSuccess || hipEventCreate(&ix->ev_all1) != hipSuccess) {
        boa_free_index(ix);
        return fail(BOA_EHIP, "hipEventCreate failed");
    }
    *out = ix;
    return BOA_OK;
}

}  // extern "C"

namespace {

int ensure_events(boa_index *ix, size_t count)
{
    while (ix->ev_start.size() < count) {
        hipEvent_t a, b;
        HIP_TRY(hipEventCreate(&a));
        HIP_TRY(hipEventCreate(&b));
        ix->ev_start.push_back(a);
        ix->ev_end.push_back(b);
    }
    return BOA_OK;
}

// A wave slot's spill bitmap: one bit per point, whole 16-byte units.
uint32_t bitmap_words(const boa_index *ix)
{
    return (uint32_t)(((ix->view.n + 127) / 128) * 4);
}

// Ids the spill log holds: clearing by the log writes about one 64-byte
// line per logged id, so it pays while the log is under 1/16 of the
// bitmap's words; at most 16380 (a 64 KB log); none for small bitmaps.
uint32_t spill_log_cap(uint32_t bits_words)
{
    uint32_t c = std::min<uint32_t>(bits_words / 16u, 16380u) & ~3u;
    return c < 64u ? 0u : c;
}

int ensure_workspace(boa_index *ix, int64_t nq, int32_t n_phases, uint64_t slots, int32_t n_counters, bool plus)
{
    int rc;
    if (nq > ix->nq_cap || n_phases > ix->ph_cap) {
        int64_t cap = std::max<int64_t>(nq, ix->nq_cap);
        int32_t pc = std::max<int32_t>(n_phases, ix->ph_cap);
        dfree(ix->active[0]);
        dfree(ix->active[1]);
        dfree(ix->conf);
        dfree(ix->qstat);
        dfree(ix->qE);
        dfree(ix->qS);
        dfree(ix->pool);
        if ((rc = dalloc(&ix->active[0], cap)) || (rc = dalloc(&ix->active[1], cap)) ||
            (rc = dalloc(&ix->conf, cap)) || (rc = dalloc(&ix->qstat, (size_t)cap * pc)) ||
            (rc = dalloc(&ix->qE, (size_t)cap * pc)) || (rc = dalloc(&ix->qS, (size_t)cap * pc)) ||
            (rc = dalloc(&ix->pool, (size_t)cap * 2))) {
            ix->nq_cap = 0;
            ix->ph_cap = 0;
            return rc;
        }
        ix->nq_cap = cap;
        ix->ph_cap = pc;
    }
    // each under its own check: a failed allocation of one is retried by the
    // next search instead of leaving the other null
    if (!ix->n_active && (rc = dalloc(&ix->n_active, 2 * (BOA_MAX_PHASES + 1)))) return rc;
    if (!ix->status && (rc = dalloc(&ix->status, 16))) return rc;
    if (n_counters > ix->n_counters) {
        dfree(ix->counters);
        if ((rc = dalloc(&ix->counters, n_counters))) return rc;
        ix->n_counters = n_counters;
    }
    if (slots > ix->slots_cap) {
        // one bit per point per wave slot, in whole 16-byte units, and the
        // log of the bits set; a query clears its slot's bitmap when it first
        // spills (by the log, or whole when the log's header says so), so no
        // clearing here: the next search marks every header unknown first
        uint64_t sc = std::max<uint64_t>(slots, ix->slots_cap);
        const uint32_t words = bitmap_words(ix);
        const uint32_t cap = spill_log_cap(words);
        dfree(ix->bits);
        if ((rc = dalloc(&ix->bits, (size_t)sc * (words + BOA_LOG_HDR + cap)))) {
            ix->slots_cap = 0;
            return rc;
        }
        ix->slots_cap = sc;
        ix->bits_words = words;
        ix->log_cap = cap;
        ix->slot_words = words + BOA_LOG_HDR + cap;
        ix->logs_fresh = true;
    }
    if (plus && !ix->aux) {
        HIP_TRY(hipStreamCreateWithFlags(&ix->aux, hipStreamNonBlocking));
        HIP_TRY(hipEventCreateWithFlags(&ix->ev_pool, hipEventDisableTiming));
        HIP_TRY(hipEventCreateWithFlags(&ix->ev_join, hipEventDisableTiming));
    }
    return BOA_OK;
}

// Beam schedule: L_{p+1} = min(ceil(alpha * L_p), Lmax); the phase at Lmax is the last.
// (fixed-size output: the search path allocates no host memory either)
int make_schedule(const boa_params *p, int32_t *s, int32_t *n)
{
    *n = 0;
    if (p->fixed_L > 0) {
        s[(*n)++] = p->fixed_L;
        return BOA_OK;
    }
    if (p->schedule && p->n_schedule > 0) {
        if (p->n_schedule > BOA_MAX_PHASES) return fail(BOA_EINVAL, "too many phases");
        for (int i = 0; i < p->n_schedule; ++i) {
            if (p->schedule[i] < 1 || (i && p->schedule[i] <= p->schedule[i - 1]))
                return fail(BOA_EINVAL, "schedule must be positive and strictly increasing");
            s[(*n)++] = p->schedule[i];
        }
        return BOA_OK;
    }
    if (!(p->alpha > 1.0) || !std::isfinite(p->alpha)) return fail(BOA_EINVAL, "alpha must be > 1");
    if (p->L0 < 1 || p->Lmax < p->L0) return fail(BOA_EINVAL, "need 1 <= L0 <= Lmax");
    int64_t L = p->L0;
    for (;;) {
        if (*n >= BOA_MAX_PHASES) return fail(BOA_EINVAL, "schedule exceeds BOA_MAX_PHASES");
        s[(*n)++] = (int32_t)L;
        if (L >= p->Lmax) break;
        int64_t nx = (int64_t)std::ceil(p->alpha * (double)L);
        if (nx <= L) nx = L + 1;
        L = nx < p->Lmax ? nx : p->Lmax;
    }
    return BOA_OK;
}

uint32_t id_bits(const boa_index *ix)
{
    uint32_t b = 1;
    while (b < 32 && ((int64_t)1 << b) < ix->view.n) ++b;
    return b;
}

// 8 slots per bucket, at most 15 stored bits per id
uint32_t min_table_slots(const boa_index *ix)
{
    const uint32_t B = id_bits(ix);
    return std::max<uint32_t>(64u, B > 15 ? (8u << (B - 15)) : 64u);
}

PhasePlan plan_phase(const boa_index *ix, int32_t L, int32_t forced_h, int64_t max_active, bool wide = false,
                     int pq_m = 0)
{
    PhasePlan pl{};
    pl.L = L;
    pl.wide = wide;
    // visited table: 16-bit slots, 16 per expected scored node of a width-L
    // search, between 1024 and 4096 (2-8 KB); ids that find both of their
    // buckets full go to the HBM bitmap. The table must leave at most 15
    // stored bits per id.
    uint32_t h = forced_h > 0 ? (uint32_t)forced_h
                              : std::min<uint32_t>(4096u, std::max<uint32_t>(1024u, next_pow2(16ull * L)));
    h = std::max<uint32_t>(h, min_table_slots(ix));
    pl.h_slots = (int32_t)h;
    const int32_t Lb = beam_slots(L), pw = ((L >> 6) + 3) & ~1;
    // (a product-quantised search also keeps its re-rank keys, Lb of them)
    pl.lds_per_wave = 8 * Lb + 8 * 64 + 8 * pw + 4 * 64 + 4 * 64 +
                      scorer_lds_bytes(ix->vec_dtype, ix->view.d, wide, pq_m) + (pq_m ? 8 * Lb : 0) + 2 * (int32_t)h;
    pl.lds_per_wave = (pl.lds_per_wave + 15) & ~15;
    // waves per block: the choice with the most resident waves per CU
    int best_w = 0, best_wpb = 1, best_occ = 1;
    for (int wpb = 4; wpb >= 1; wpb >>= 1) {
        if ((size_t)wpb * pl.lds_per_wave > ix->lds_per_block_max) continue;
        int occ = phase_occupancy(ix->vec_dtype, ix->view.d, wpb, (size_t)wpb * pl.lds_per_wave, wide, pq_m);
        if (occ * wpb > best_w) {
            best_w = occ * wpb;
            best_wpb = wpb;
            best_occ = occ;
        }
    }
    pl.wpb = best_wpb;
    int64_t blocks = (int64_t)std::max(best_occ, 1) * ix->num_cu;
    pl.capacity = best_w > 0 ? blocks * best_wpb : 0;
    int64_t need = (max_active + best_wpb - 1) / best_wpb;
    if (need < 1) need = 1;
    pl.blocks = (int32_t)std::min<int64_t>(blocks, need);
    pl.launches = 0;
    return pl;
}

#ifdef BOA_STAGE_PROFILE
// Per-stage cycle counters of one launch (a diagnostic build only).
int stage_profile_begin(unsigned long long **prof, size_t pn, hipStream_t st)
{
    HIP_TRY(hipMalloc(reinterpret_cast<void **>(prof), pn * 8));
    HIP_TRY(hipMemsetAsync(*prof, 0, pn * 8, st));
    return BOA_OK;
}

int stage_profile_end(unsigned long long *prof, size_t pn, int L, int waves, hipStream_t st)
{
    std::vector<unsigned long long> h(pn);
    HIP_TRY(hipMemcpyAsync(h.data(), prof, pn * 8, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    double tot[BOA_PROF_SLOTS] = {0};
    for (size_t i = 0; i < pn; ++i) tot[i % BOA_PROF_SLOTS] += (double)h[i];
    const double ne = tot[10] > 0 ? tot[10] : 1;
    std::fprintf(stderr,
                 "[stage-profile] L=%d waves=%d expansions=%.0f cycles/expansion: select %.0f "
                 "visit %.0f score %.0f sort %.0f rank %.0f rebuild %.0f | spilled %.2f chunks %.2f "
                 "row-prefetch hit %.2f reissued %.2f | visit: row %.0f table %.0f; no new candidate %.2f\n",
                 L, waves, tot[10], tot[0] / ne, tot[1] / ne, tot[2] / ne, tot[3] / ne, tot[4] / ne,
                 tot[5] / ne, tot[6] / ne, tot[7] / ne, tot[8] / ne, tot[9] / ne, tot[12] / ne, tot[13] / ne,
                 tot[14] / ne);
    (void)hipFree(prof);
    return BOA_OK;
}

// the same for the two-wave escalation launch (one row per block)
int stage_profile_pair_end(unsigned long long *prof, size_t pn, int L, int blocks, hipStream_t st)
{
    std::vector<unsigned long long> h(pn);
    HIP_TRY(hipMemcpyAsync(h.data(), prof, pn * 8, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    double tot[BOA_PROF_SLOTS] = {0};
    for (size_t i = 0; i < pn; ++i) tot[i % BOA_PROF_SLOTS] += (double)h[i];
    const double ne = tot[10] > 0 ? tot[10] : 1;
    std::fprintf(stderr,
                 "[stage-profile] two-wave escalation L=%d blocks=%d expansions=%.0f cycles/expansion: "
                 "iteration %.0f | worklist wave: merge and select %.0f, wait %.0f | gather wave: guessed "
                 "expansion %.0f, wait %.0f, hand-over %.0f | guesses: hit %.3f miss %.3f none %.3f, of a new "
                 "key %.3f; no entry after the selected one %.3f\n",
                 L, blocks, tot[10], tot[5] / ne, tot[0] / ne, tot[3] / ne, tot[1] / ne, tot[4] / ne, tot[2] / ne,
                 tot[8] / ne, tot[9] / ne, tot[14] / ne, tot[13] / ne, tot[12] / ne);
    (void)hipFree(prof);
    return BOA_OK;
}
#endif

// A phase's launch: the automatic table of plan_phase, then doubled (up to
// 16384 slots) while that keeps as many waves resident (registers, not LDS,
// often bound narrow phases, so a wider table and fewer spills come free).
PhasePlan plan_phase_widest(const boa_index *ix, int32_t L, int32_t forced_h, int64_t max_active, bool wide = false,
                            int pq_m = 0)
{
    PhasePlan best = plan_phase(ix, L, forced_h, max_active, wide, pq_m);
    if (forced_h > 0) return best;
    for (uint32_t h = 2u * (uint32_t)best.h_slots; h <= 16384u; h <<= 1) {
        PhasePlan pl = plan_phase(ix, L, (int32_t)h, max_active, wide, pq_m);
        if ((size_t)pl.lds_per_wave > ix->lds_per_block_max || pl.capacity < best.capacity) break;
        best = pl;
    }
    return best;
}

// The escalation launch of a split search: S survivors, all phases after the
// first. Widest visited table (fewest spills to the HBM bitmap) whose LDS
// footprint still lets all S waves be resident at once; the default table
// when even that is not possible.
// The same launch with the visited set as an LDS bitmap over all n ids (one
// wave per block): an exact set tested by a single LDS atomic, for indexes
// small enough (n/8 bytes plus the worklist within the device's per-block
// LDS) and survivor counts that it still lets be resident at once.
PhasePlan plan_bitmap(const boa_index *ix, int32_t L, int64_t S, int pq_m = 0)
{
    PhasePlan pl{};
    pl.L = L;
    pl.wide = true;
    pl.vis_bitmap = 1;
    pl.h_slots = 0;
    const int64_t words = ((ix->view.n + 31) / 32 + 3) & ~(int64_t)3;
    const int32_t Lb = beam_slots(L), pw = ((L >> 6) + 3) & ~1;
    const int64_t lds = 8 * Lb + 8 * 64 + 8 * pw + 4 * 64 + 4 * 64 + scorer_lds_bytes(ix->vec_dtype, ix->view.d, true, pq_m) +
                        (pq_m ? 8 * Lb : 0) + 4 * words;
    pl.lds_per_wave = (int32_t)((lds + 15) & ~(int64_t)15);
    pl.wpb = 1;
    if ((size_t)pl.lds_per_wave > ix->lds_per_block_hw) return pl;   // capacity 0: not possible
    const int occ = phase_occupancy(ix->vec_dtype, ix->view.d, 1, (size_t)pl.lds_per_wave, true, pq_m);
    const int64_t blocks = (int64_t)std::max(occ, 0) * ix->num_cu;
    pl.capacity = blocks;
    pl.blocks = (int32_t)std::min<int64_t>(blocks, std::max<int64_t>(S, 1));
    return pl;
}

PhasePlan plan_escalation(const boa_index *ix, int32_t L, int64_t S, int32_t forced_h, int pq_m = 0)
{
    if (forced_h > 0) return plan_phase(ix, L, forced_h, S, true, pq_m);
    {
        PhasePlan bm = plan_bitmap(ix, L, S, pq_m);
        if (bm.capacity >= S) return bm;
    }
    PhasePlan dflt = plan_phase(ix, L, 0, S, true, pq_m);
    for (uint32_t h = 16384; h > (uint32_t)dflt.h_slots; h >>= 1) {
        PhasePlan pl = plan_phase(ix, L, (int32_t)h, S, true, pq_m);
        if (pl.capacity >= S && (size_t)pl.lds_per_wave <= ix->lds_per_block_max) return pl;
    }
    return dflt;
}

// Device memory one search works in: the index's grown-on-demand workspace
// (boa_search) or a carve-out of the file-scope scratch array
// (boa_search_noalloc).
struct Workspace {
    uint32_t *active[2];
    uint32_t *n_active;       // 2 (BOA_MAX_PHASES + 1): per-phase active counts, BOA+ pool counts
    uint32_t *counters;       // per-launch work counters
    uint8_t *conf;            // nq
    uint8_t *qstat;           // per phase x nq, with qE and qS (null: no per-phase statistics)
    uint32_t *qE, *qS;
    uint32_t *status;
    uint32_t *bits;           // visited spill bitmaps and logs, slot_words u32 per wave slot
    uint32_t bits_words, slot_words, log_cap;
    bool reset_logs;          // the logs' headers must be marked unknown before the search
    bool *logs_fresh;         // cleared once that reset is enqueued (null: reset every search)
    uint64_t slots;           // wave slots that have a spill bitmap
    uint32_t *pool;           // BOA+ survivor pools, 2 nq (null: no BOA+)
    bool timing;              // HIP events around launches; statistics of the search kept
};

// A validated search request (everything decided before device work).
struct Request {
    int32_t sched[BOA_MAX_PHASES];
    int32_t n_phases;
    bool plus, split, fused, warm;
    bool pair;                // split escalation with two waves per query where it applies
    int32_t pq_m;             // > 0: product-quantised traversal with that many subspaces
    int32_t sub;              // BOA+ sub-batches (1 otherwise)
    int32_t n_counters;
    uint32_t tau_count;
};

int validate(const boa_index *ix, const void *queries, const int32_t *ranges, int64_t nq, const boa_params *p,
             uint32_t *ids, float *dists, int32_t *final_L, Request &rq)
{
    if (!ix || !p) return fail(BOA_EINVAL, "NULL index or params");
    if (nq < 0 || nq >= (int64_t)1 << 31) return fail(BOA_EINVAL, "nq out of range");
    if (nq > 0 && (!queries || !ranges || !ids || !dists || !final_L))
        return fail(BOA_EINVAL, "NULL device buffer");
    int rc = make_schedule(p, rq.sched, &rq.n_phases);
    if (rc) return rc;
    for (int i = 0; i < rq.n_phases; ++i)
        if (rq.sched[i] < 1 || rq.sched[i] > BOA_MAX_L) return fail(BOA_EINVAL, "beamwidth out of range [1, 2048]");
    if (p->k < 1 || p->k > rq.sched[0]) return fail(BOA_EINVAL, "need 1 <= k <= first-phase beamwidth");
    if (!(p->eps >= 0.0) || !std::isfinite(p->eps)) return fail(BOA_EINVAL, "eps must be >= 0");
    if (!(p->tau >= 0.0 && p->tau < 1.0)) return fail(BOA_EINVAL, "tau must be in [0, 1)");
    if (p->lds_hash_slots && (p->lds_hash_slots < 64 || (p->lds_hash_slots & (p->lds_hash_slots - 1)) ||
                              p->lds_hash_slots > 16384))
        return fail(BOA_EINVAL, "lds_hash_slots must be 0 or a power of two in [64, 16384]");
    if (p->lds_hash_slots && (uint32_t)p->lds_hash_slots < min_table_slots(ix))
        return fail(BOA_EINVAL, "lds_hash_slots too small for this index's id width");
    rq.plus = p->boa_plus != 0 && p->fixed_L <= 0;
    if (p->fused < 0 || p->fused > 2) return fail(BOA_EINVAL, "fused must be 0, 1 or 2");
    rq.split = p->fused == 2;
    rq.fused = p->fused == 1;
    if (p->fused != 0 && p->tau != 0.0)
        return fail(BOA_EINVAL, "fused phases need tau == 0 (the residual test counts all queries of a phase)");
    if (p->fused != 0 && rq.plus) return fail(BOA_EINVAL, "fused and boa_plus are exclusive");
    if (rq.plus && p->tau != 0.0)
        return fail(BOA_EINVAL, "BOA+ needs tau == 0 (the residual test counts all queries of a phase)");
    if (rq.plus && (p->sub_batches < 1 || p->sub_batches > 1024)) return fail(BOA_EINVAL, "sub_batches out of range");
    if (p->warm_start != 0 && p->warm_start != 1) return fail(BOA_EINVAL, "warm_start must be 0 or 1");
    if (p->warm_start && !rq.fused)
        return fail(BOA_EUNSUPPORTED, "warm-start escalation runs in the fused mode (fused = 1)");
    rq.warm = p->warm_start == 1;
    if (p->pq != 0 && p->pq != 1) return fail(BOA_EINVAL, "pq must be 0 or 1");
    if (p->pq && ix->pq_m == 0) return fail(BOA_EINVAL, "pq = 1 needs product-quantisation codes (boa_set_pq)");
    if (p->pq && p->k > 128) return fail(BOA_EUNSUPPORTED, "a product-quantised search returns at most k = 128");
    rq.pq_m = p->pq ? ix->pq_m : 0;
    if (p->escalation_waves != 0 && p->escalation_waves != 1)
        return fail(BOA_EINVAL, "escalation_waves must be 0 or 1");
    rq.pair = p->escalation_waves == 0 && rq.pq_m == 0;
    rq.sub = rq.plus ? std::min<int64_t>(p->sub_batches, std::max<int64_t>(nq, 1)) : 1;
    rq.n_counters = rq.n_phases * (rq.sub + 1) + 8;
    rq.tau_count = (uint32_t)std::floor(p->tau * (double)nq);
    return BOA_OK;
}

// Launch plans of every phase, and the number of wave slots (spill bitmaps)
// the search may use at once.
int plan_search(const boa_index *ix, const Request &rq, int64_t nq, int32_t forced_h, PhasePlan *plans,
                uint64_t *slots_out)
{
    uint64_t slots = 0;
    const int32_t Lw = rq.sched[rq.n_phases - 1];
    for (int32_t ph = 0; ph < rq.n_phases; ++ph) {
        // a fused launch, and a BOA+ escalation launch, size LDS for the widest phase
        const bool widest = rq.fused || (rq.plus && ph > 0);
        PhasePlan pl = plan_phase_widest(ix, widest ? Lw : rq.sched[ph], forced_h, nq, false, rq.pq_m);
        if (rq.fused && Lw > 64) {
            // the wide variant (eight-way worklist search, more rows in
            // flight) wherever it keeps as many waves resident
            const PhasePlan w = plan_phase_widest(ix, Lw, forced_h, nq, true, rq.pq_m);
            if (w.capacity >= pl.capacity && (size_t)w.lds_per_wave <= ix->lds_per_block_max) pl = w;
        }
        pl.L = rq.sched[ph];
        if ((size_t)pl.lds_per_wave > ix->lds_per_block_max)
            return fail(BOA_EUNSUPPORTED, "beamwidth too wide for the LDS budget");
        slots = std::max<uint64_t>(slots, (uint64_t)pl.blocks * pl.wpb);
        plans[ph] = pl;
    }
    if (rq.split && rq.n_phases > 1) {
        // every grid the escalation launch may take (it has at most nq waves)
        const PhasePlan d = plan_phase(ix, Lw, forced_h, nq, true, rq.pq_m);
        slots = std::max<uint64_t>(slots, (uint64_t)d.blocks * d.wpb);
        if (forced_h <= 0)
            for (uint32_t h = 16384; h > (uint32_t)d.h_slots; h >>= 1) {
                const PhasePlan c = plan_phase(ix, Lw, (int32_t)h, nq, true, rq.pq_m);
                slots = std::max<uint64_t>(slots, (uint64_t)c.blocks * c.wpb);
            }
    }
    *slots_out = slots;
    return BOA_OK;
}

// Fewer blocks of a persistent launch (each wave pulls queries from the
// launch's counter, so results do not change) where the workspace has spill
// bitmaps for fewer wave slots than the plan would use.
int cap_to_slots(PhasePlan &pl, uint64_t slots)
{
    const uint64_t b = slots / (uint64_t)pl.wpb;
    if (b < 1) return fail(BOA_EUNSUPPORTED, "the index is too large for the scratch memory of this search");
    if ((uint64_t)pl.blocks > b) pl.blocks = (int32_t)b;
    return BOA_OK;
}

int run_search(boa_index *ix, const void *queries, const int32_t *ranges, int64_t nq, const boa_params *p,
               const Request &rq, PhasePlan *plans, uint32_t *ids, float *dists, int32_t *final_L,
               uint32_t *expansions, uint32_t *scored, const Workspace &ws, hipStream_t st)
{
    const int32_t n_phases = rq.n_phases;
    const int32_t *sched = rq.sched;
    const int32_t Lw = sched[n_phases - 1];
    for (int32_t ph = 0; ph < n_phases; ++ph)
        if (int rc = cap_to_slots(plans[ph], ws.slots)) return rc;

    InitArgs ia{};
    ia.active0 = ws.active[0];
    ia.n_active = ws.n_active;
    ia.counters = ws.counters;
    ia.qstat = ws.qstat;
    ia.user_E = expansions;
    ia.user_S = scored;
    ia.status = ws.status;
    ia.nq = nq;
    ia.n_phases = n_phases;
    ia.n_counters = rq.n_counters;
    ia.bits = ws.bits;
    ia.slot_words = ws.slot_words;
    ia.bits_words = ws.bits_words;
    ia.reset_slots = ws.reset_logs ? ws.slots : 0;

    if (ws.timing) {
        ix->launch_phase.clear();
        HIP_TRY(hipEventRecord(ix->ev_all0, st));
    }
    ix->have_stats = false;
    HIP_TRY(launch_init(ia, st));
    if (ws.reset_logs && ws.logs_fresh) *ws.logs_fresh = false;

    PhaseArgs base{};
    base.ix = ix->view;
    base.queries = queries;
    base.ranges = ranges;
    base.ids = ids;
    base.dists = dists;
    base.final_L = final_L;
    base.user_E = expansions;
    base.user_S = scored;
    base.bits = ws.bits;
    base.bits_words = ws.bits_words;
    base.slot_words = ws.slot_words;
    base.log_cap = ws.log_cap;
    base.id_bits = id_bits(ix);
    base.status = ws.status;
    base.eps = p->eps;
    base.tau_count = rq.tau_count;
    base.k = p->k;
    base.conf = ws.conf;
    base.nq = nq;
    base.qstat = ws.qstat;
    base.qE = ws.qE;
    base.qS = ws.qS;
    base.pq = rq.pq_m > 0 ? 1 : 0;
    base.pq_m = rq.pq_m;
    base.pq_cb = ix->d_pq_cb;
    base.pq_codes = ix->d_pq_codes;
    base.vec_u8 = ix->vec_dtype == BOA_VEC_U8 ? 1 : 0;
    for (int32_t ph = 0; ph < n_phases; ++ph) base.sched[ph] = sched[ph];
    int ev = 0;
    // one search launch, bracketed by HIP events when timing
    auto launch = [&](const PhaseArgs &a, int blocks, hipStream_t s, bool wide, int phase) -> int {
        if (ws.timing) HIP_TRY(hipEventRecord(ix->ev_start[ev], s));
        HIP_TRY(launch_phase(a, ix->vec_dtype, blocks, s, wide));
        if (ws.timing) {
            HIP_TRY(hipEventRecord(ix->ev_end[ev], s));
            ix->launch_phase.push_back({phase, ev});
            ++ev;
        }
        return BOA_OK;
    };

    if (rq.fused) {
        PhasePlan &pl = plans[0];
        PhaseArgs a = base;
        a.active = ws.active[0];
        a.n_active = ws.n_active;
        a.t_begin = 0;
        a.t_end = 0xFFFFFFFFu;
        a.queue = ws.counters;
        a.p_begin = 0;
        a.p_end = n_phases;
        a.warm = rq.warm ? 1 : 0;
        a.L_alloc = Lw;
        a.h_log2 = ilog2((uint32_t)pl.h_slots);
        a.lds_per_wave = pl.lds_per_wave;
        a.waves_per_block = pl.wpb;
        a.slot_base = 0;
#ifdef BOA_STAGE_PROFILE
        unsigned long long *prof = nullptr;
        const size_t pn = (size_t)pl.blocks * pl.wpb * BOA_PROF_SLOTS;
        if (int rc2 = stage_profile_begin(&prof, pn, st)) return rc2;
        a.prof = prof;
#endif
        if (int rc = launch(a, pl.blocks, st, pl.wide, 0)) return rc;
#ifdef BOA_STAGE_PROFILE
        std::fprintf(stderr, "[stage-profile] fused launch%s: table %d slots, %d waves (all phases)\n",
                     rq.warm ? " (warm start)" : "", pl.h_slots, pl.blocks * pl.wpb);
        if (int rc2 = stage_profile_end(prof, pn, Lw, pl.blocks * pl.wpb, st)) return rc2;
#endif
        pl.launches = 1;
    } else if (rq.split) {
        // the first phase over every query at its own width ...
        PhasePlan &p0 = plans[0];
        PhaseArgs a = base;
        a.active = ws.active[0];
        a.n_active = ws.n_active;
        a.t_begin = 0;
        a.t_end = 0xFFFFFFFFu;
        a.queue = ws.counters;
        a.p_begin = 0;
        a.p_end = 1;
        a.write_conf = 1;
        a.L_alloc = sched[0];
        a.h_log2 = ilog2((uint32_t)p0.h_slots);
        a.lds_per_wave = p0.lds_per_wave;
        a.waves_per_block = p0.wpb;
        a.slot_base = 0;
        if (int rc = launch(a, p0.blocks, st, false, 0)) return rc;
        p0.launches = 1;
        if (n_phases > 1) {
            // ... then its survivors, compacted, through every later width
            CompactArgs ca{};
            ca.in = ws.active[0];
            ca.n_in = ws.n_active;
            ca.conf = ws.conf;
            ca.out = ws.active[1];
            ca.n_out = ws.n_active + 1;
            ca.tau_count = rq.tau_count;
            HIP_TRY(launch_compact(ca, st));
            uint32_t S = 0;
            HIP_TRY(hipMemcpyAsync(&S, ws.n_active + 1, sizeof(S), hipMemcpyDeviceToHost, st));
            HIP_TRY(hipStreamSynchronize(st));
            if (S > 0) {
                PhasePlan pe = plan_escalation(ix, Lw, S, p->lds_hash_slots, rq.pq_m);
                if ((size_t)pe.lds_per_wave > (pe.vis_bitmap ? ix->lds_per_block_hw : ix->lds_per_block_max))
                    return fail(BOA_EUNSUPPORTED, "beamwidth too wide for the LDS budget");
                if (int rc = cap_to_slots(pe, ws.slots)) return rc;
                PhaseArgs e = base;
                e.active = ws.active[1];
                e.n_active = ws.n_active + 1;
                e.t_begin = 0;
                e.t_end = 0xFFFFFFFFu;
                e.queue = ws.counters + 1;
                e.p_begin = 1;
                e.p_end = n_phases;
                e.L_alloc = Lw;
                e.h_log2 = pe.vis_bitmap ? 3 : ilog2((uint32_t)pe.h_slots);   // (unused with the bitmap)
                e.vis_bitmap = pe.vis_bitmap;
                e.vis_words = pe.vis_bitmap ? (uint32_t)(((ix->view.n + 31) / 32 + 3) & ~(int64_t)3) : 0u;
                e.lds_per_wave = pe.lds_per_wave;
                e.waves_per_block = pe.wpb;
                e.slot_base = 0;
#ifdef BOA_STAGE_PROFILE
                unsigned long long *prof = nullptr;
                const size_t pn = (size_t)pe.blocks * pe.wpb * BOA_PROF_SLOTS;
                if (int rc2 = stage_profile_begin(&prof, pn, st)) return rc2;
                e.prof = prof;
#endif
                // two waves per query where the bitmap plan applies and every
                // survivor's block is still resident at once
                bool pair = rq.pair && pe.vis_bitmap;
                if (pair) {
                    const size_t lds = pair_lds_bytes(Lw, e.vis_words,
                                                      scorer_lds_bytes(ix->vec_dtype, ix->view.d, true, 0));
                    const int occ = lds <= ix->lds_per_block_hw ? pair_occupancy(ix->vec_dtype, ix->view.d, lds) : 0;
                    const int64_t cap = (int64_t)occ * ix->num_cu;
                    pair = cap >= (int64_t)S;
                    if (pair) {
                        pe.blocks = (int32_t)S;
                        pe.wpb = 2;
                        e.lds_per_wave = (int32_t)lds;
                        e.waves_per_block = 2;
                    }
                }
                if (pair) {
#ifdef BOA_STAGE_PROFILE
                    unsigned long long *pprof = nullptr;
                    const size_t ppn = (size_t)pe.blocks * BOA_PROF_SLOTS;
                    if (int rc2 = stage_profile_begin(&pprof, ppn, st)) return rc2;
                    e.prof = pprof;
#endif
                    if (ws.timing) HIP_TRY(hipEventRecord(ix->ev_start[ev], st));
                    HIP_TRY(launch_pair(e, ix->vec_dtype, pe.blocks, st));
                    if (ws.timing) {
                        HIP_TRY(hipEventRecord(ix->ev_end[ev], st));
                        ix->launch_phase.push_back({1, ev});
                        ++ev;
                    }
#ifdef BOA_STAGE_PROFILE
                    if (int rc2 = stage_profile_pair_end(pprof, ppn, Lw, (int)S, st)) return rc2;
#endif
                } else if (int rc = launch(e, pe.blocks, st, true, 1)) {
                    return rc;
                }
#ifdef BOA_STAGE_PROFILE
                std::fprintf(stderr, "[stage-profile] split escalation: %u survivors, table %d slots, %d waves\n",
                             S, pe.h_slots, pe.blocks * pe.wpb);
                if (int rc2 = stage_profile_end(prof, pn, Lw, pe.blocks * pe.wpb, st)) return rc2;
#endif
                plans[1].launches = 1;
                plans[1].h_slots = pe.h_slots;
                plans[1].wpb = pe.wpb;
                plans[1].blocks = pe.blocks;
            }
        }
    } else if (!rq.plus) {
        for (int32_t ph = 0; ph < n_phases; ++ph) {
            PhasePlan &pl = plans[ph];
            PhaseArgs a = base;
            a.active = ws.active[ph & 1];
            a.n_active = ws.n_active + ph;
            a.t_begin = 0;
            a.t_end = 0xFFFFFFFFu;
            a.queue = ws.counters + ph;
            a.p_begin = ph;
            a.p_end = ph + 1;
            a.write_conf = 1;
            a.L_alloc = pl.L;
            a.h_log2 = ilog2((uint32_t)pl.h_slots);
            a.lds_per_wave = pl.lds_per_wave;
            a.waves_per_block = pl.wpb;
            a.slot_base = 0;
#ifdef BOA_STAGE_PROFILE
            unsigned long long *prof = nullptr;
            const size_t pn = (size_t)pl.blocks * pl.wpb * BOA_PROF_SLOTS;
            if (int rc2 = stage_profile_begin(&prof, pn, st)) return rc2;
            a.prof = prof;
#endif
            if (int rc = launch(a, pl.blocks, st, false, ph)) return rc;
#ifdef BOA_STAGE_PROFILE
            if (int rc2 = stage_profile_end(prof, pn, pl.L, pl.blocks * pl.wpb, st)) return rc2;
#endif
            pl.launches = 1;
            if (ph + 1 < n_phases) {
                CompactArgs ca{};
                ca.in = ws.active[ph & 1];
                ca.n_in = ws.n_active + ph;
                ca.conf = ws.conf;
                ca.out = ws.active[(ph + 1) & 1];
                ca.n_out = ws.n_active + ph + 1;
                ca.tau_count = rq.tau_count;
                HIP_TRY(launch_compact(ca, st));
            }
        }
    } else {
        // BOA+ (Sec. III-A, "Pipelining Multiple Batches"): phase 0 runs as
        // `sub` sub-batches on the caller's stream; the survivors of the
        // first half are pooled and escalated through the remaining widths
        // in one launch on a second stream while the second half of phase 0
        // runs; the second half's pooled survivors follow on the caller's
        // stream. Each escalation launch carries its queries through all
        // remaining widths (results are those of BOA).
        if (!ws.pool || !ix->aux) return fail(BOA_EUNSUPPORTED, "BOA+ needs the index's own workspace");
        const int32_t sub = rq.sub;
        const int64_t B = (nq + sub - 1) / sub;
        const int32_t nsub = (int32_t)((nq + B - 1) / B);
        const int32_t half = (nsub + 1) / 2;
        uint32_t *pool[2] = {ws.pool, ws.pool + nq};
        uint32_t *pool_n[2] = {ws.n_active + BOA_MAX_PHASES + 1, ws.n_active + BOA_MAX_PHASES + 2};
        // the second stream's waves use the spill bitmaps above the first's
        const uint64_t half_slots = ws.slots / 2;
        for (int32_t ph = 0; ph < n_phases; ++ph)
            if (int rc = cap_to_slots(plans[ph], half_slots)) return rc;
        PhasePlan &p0 = plans[0];
        for (int32_t b = 0; b < nsub; ++b) {
            PhaseArgs a = base;
            a.active = ws.active[0];
            a.n_active = ws.n_active;
            a.t_begin = (uint32_t)(b * B);
            a.t_end = (uint32_t)std::min<int64_t>(nq, (b + 1) * B);
            a.queue = ws.counters + b;
            a.p_begin = 0;
            a.p_end = 1;
            a.write_conf = 1;
            a.L_alloc = sched[0];
            a.h_log2 = ilog2((uint32_t)p0.h_slots);
            a.lds_per_wave = p0.lds_per_wave;
            a.waves_per_block = p0.wpb;
            a.slot_base = 0;
            const int64_t span = a.t_end - a.t_begin;
            const int blocks = (int)std::min<int64_t>(p0.blocks, (span + p0.wpb - 1) / p0.wpb);
            if (int rc = launch(a, blocks, st, false, 0)) return rc;
            p0.launches += 1;
            AppendArgs ap{};
            ap.in = ws.active[0] + a.t_begin;
            ap.conf = ws.conf + a.t_begin;
            ap.n = (uint32_t)span;
            const int g = b < half ? 0 : 1;
            ap.pool = pool[g];
            ap.pool_count = pool_n[g];
            HIP_TRY(launch_append(ap, st));
            if (b == half - 1 && n_phases > 1) {
                // first pool complete: escalate it on the second stream
                HIP_TRY(hipEventRecord(ix->ev_pool, st));
                HIP_TRY(hipStreamWaitEvent(ix->aux, ix->ev_pool, 0));
                PhasePlan &pe = plans[1];
                PhaseArgs e = base;
                e.active = pool[0];
                e.n_active = pool_n[0];
                e.t_begin = 0;
                e.t_end = 0xFFFFFFFFu;
                e.queue = ws.counters + nsub;
                e.p_begin = 1;
                e.p_end = n_phases;
                e.L_alloc = Lw;
                e.h_log2 = ilog2((uint32_t)pe.h_slots);
                e.lds_per_wave = pe.lds_per_wave;
                e.waves_per_block = pe.wpb;
                e.slot_base = (uint32_t)half_slots;   // disjoint spill bitmaps from stream 0
                if (int rc = launch(e, pe.blocks, ix->aux, false, 1)) return rc;
                pe.launches += 1;
            }
        }
        if (n_phases > 1 && nsub > half) {
            PhasePlan &pe = plans[1];
            PhaseArgs e = base;
            e.active = pool[1];
            e.n_active = pool_n[1];
            e.t_begin = 0;
            e.t_end = 0xFFFFFFFFu;
            e.queue = ws.counters + nsub + 1;
            e.p_begin = 1;
            e.p_end = n_phases;
            e.L_alloc = Lw;
            e.h_log2 = ilog2((uint32_t)pe.h_slots);
            e.lds_per_wave = pe.lds_per_wave;
            e.waves_per_block = pe.wpb;
            e.slot_base = 0;
            if (int rc = launch(e, pe.blocks, st, false, 1)) return rc;
            pe.launches += 1;
        }
        if (n_phases > 1) {
            HIP_TRY(hipEventRecord(ix->ev_join, ix->aux));
            HIP_TRY(hipStreamWaitEvent(st, ix->ev_join, 0));
        }
    }

    if (ws.timing) HIP_TRY(hipEventRecord(ix->ev_all1, st));
    uint32_t status = 0;
    HIP_TRY(hipMemcpyAsync(&status, ws.status, sizeof(uint32_t), hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    if (ws.timing) {
        ix->plans.assign(plans, plans + n_phases);
        ix->last_nq = nq;
        ix->last_k = p->k;
        ix->last_pq_m = rq.pq_m;
        ix->have_stats = true;
        ix->cum_searches += 1;
        for (auto &lp : ix->launch_phase) {
            float ms = 0.f;
            HIP_TRY(hipEventElapsedTime(&ms, ix->ev_start[lp.second], ix->ev_end[lp.second]));
            ix->cum_kernel_ms += ms;
            ix->cum_launches += 1;
            ix->cum_phase_kernel_ms[lp.first] += ms;
            ix->cum_phase_launches[lp.first] += 1;
        }
    }
    if (status & BOA_STATUS_OVERFLOW)
        return fail(BOA_EOVERFLOW, "a visited table overflowed; results are not valid");
    return BOA_OK;
}

constexpr size_t kScratchBytes = (size_t)BOA_NOALLOC_SCRATCH_MB << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char *g_scratch_ptr[kMaxDevices] = {};

int scratch_for_device(int dev, unsigned char **out)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(BOA_EUNSUPPORTED, "device ordinal beyond the scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return fail(BOA_EHIP, "hipGetSymbolAddress of the scratch array failed");
        }
        g_scratch_ptr[dev] = reinterpret_cast<unsigned char *>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return BOA_OK;
}

}  // namespace

extern "C" int boa_search(boa_index *ix, const void *queries, const int32_t *ranges, int64_t nq,
                          const boa_params *p, uint32_t *ids, float *dists, int32_t *final_L,
                          uint32_t *expansions, uint32_t *scored, void *stream_v)
{
    Request rq;
    if (int rc = validate(ix, queries, ranges, nq, p, ids, dists, final_L, rq)) return rc;
    if (nq == 0) return BOA_OK;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream_v);
    int cur_dev = 0;
    HIP_TRY(hipGetDevice(&cur_dev));
    if (cur_dev != ix->device) return fail(BOA_EINVAL, "index lives on another device than the current one");

    PhasePlan plans[BOA_MAX_PHASES];
    uint64_t slots = 0;
    if (int rc = plan_search(ix, rq, nq, p->lds_hash_slots, plans, &slots)) return rc;
    if (int rc = ensure_workspace(ix, nq, rq.n_phases, rq.plus ? 2 * slots : slots, rq.n_counters, rq.plus))
        return rc;
    if (int rc = ensure_events(ix, (size_t)rq.n_phases * (rq.sub + 1))) return rc;
    Workspace ws{};
    ws.active[0] = ix->active[0];
    ws.active[1] = ix->active[1];
    ws.n_active = ix->n_active;
    ws.counters = ix->counters;
    ws.conf = ix->conf;
    ws.qstat = ix->qstat;
    ws.qE = ix->qE;
    ws.qS = ix->qS;
    ws.status = ix->status;
    ws.bits = ix->bits;
    ws.bits_words = ix->bits_words;
    ws.slot_words = ix->slot_words;
    ws.log_cap = ix->log_cap;
    ws.reset_logs = ix->logs_fresh;
    ws.logs_fresh = &ix->logs_fresh;
    ws.slots = ix->slots_cap;
    ws.pool = ix->pool;
    ws.timing = true;
    return run_search(ix, queries, ranges, nq, p, rq, plans, ids, dists, final_L, expansions, scored, ws, st);
}

extern "C" int boa_search_noalloc(boa_index *ix, const void *queries, const int32_t *ranges, int64_t nq,
                                  const boa_params *p, uint32_t *ids, float *dists, int32_t *final_L,
                                  uint32_t *expansions, uint32_t *scored, void *stream_v)
{
    Request rq;
    if (int rc = validate(ix, queries, ranges, nq, p, ids, dists, final_L, rq)) return rc;
    if (nq > BOA_NOALLOC_MAX_NQ) return fail(BOA_EINVAL, "nq exceeds the allocation-free search's maximum");
    if (rq.plus) return fail(BOA_EUNSUPPORTED, "BOA+ needs a second stream: not available without allocation");
    if (nq == 0) return BOA_OK;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream_v);
    int cur_dev = 0;
    HIP_TRY(hipGetDevice(&cur_dev));
    if (cur_dev != ix->device) return fail(BOA_EINVAL, "index lives on another device than the current one");
    unsigned char *base = nullptr;
    if (int rc = scratch_for_device(cur_dev, &base)) return rc;

    PhasePlan plans[BOA_MAX_PHASES];
    uint64_t slots = 0;
    if (int rc = plan_search(ix, rq, nq, p->lds_hash_slots, plans, &slots)) return rc;

    // carve the scratch: fixed-size pieces first (256-byte aligned), then
    // the spill bitmaps of as many wave slots as the rest holds
    size_t off = 0;
    auto take = [&](size_t bytes) -> unsigned char * {
        unsigned char *q = base + off;
        off += (bytes + 255) & ~(size_t)255;
        return q;
    };
    Workspace ws{};
    ws.n_active = reinterpret_cast<uint32_t *>(take(4 * 2 * (BOA_MAX_PHASES + 1)));
    ws.status = reinterpret_cast<uint32_t *>(take(4 * 16));
    ws.counters = reinterpret_cast<uint32_t *>(take(4 * (size_t)rq.n_counters));
    ws.active[0] = reinterpret_cast<uint32_t *>(take(4 * (size_t)nq));
    ws.active[1] = reinterpret_cast<uint32_t *>(take(4 * (size_t)nq));
    ws.conf = reinterpret_cast<uint8_t *>(take((size_t)nq));
    ws.qstat = nullptr;
    ws.qE = ws.qS = nullptr;
    ws.pool = nullptr;
    ws.timing = false;
    ws.bits_words = bitmap_words(ix);
    ws.log_cap = spill_log_cap(ws.bits_words);
    ws.slot_words = ws.bits_words + BOA_LOG_HDR + ws.log_cap;
    // (the carve-out moves with nq: no log header of an earlier call is trusted)
    ws.reset_logs = true;
    ws.logs_fresh = nullptr;
    ws.bits = reinterpret_cast<uint32_t *>(base + off);
    ws.slots = off < kScratchBytes ? (kScratchBytes - off) / ((size_t)ws.slot_words * 4) : 0;
    if (ws.slots > slots) ws.slots = slots;
    return run_search(ix, queries, ranges, nq, p, rq, plans, ids, dists, final_L, expansions, scored, ws, st);
}

extern "C" int boa_get_stats(const boa_index *ix, boa_stats *out)
{
    if (!ix || !out) return fail(BOA_EINVAL, "NULL argument");
    std::memset(out, 0, sizeof(*out));
    if (!ix->have_stats) return fail(BOA_EINVAL, "no completed search on this index");
    const int64_t nq = ix->last_nq;
    const int32_t np = (int32_t)ix->plans.size();
    out->n_phases = np;
    out->waves_per_block = ix->plans[0].wpb;
    out->blocks = ix->plans[0].blocks;
    out->lds_hash_slots = ix->plans[0].h_slots;
    std::vector<uint8_t> st((size_t)nq * np);
    std::vector<uint32_t> E((size_t)nq * np), S((size_t)nq * np);
    HIP_TRY(hipMemcpy(st.data(), ix->qstat, st.size(), hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(E.data(), ix->qE, E.size() * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(S.data(), ix->qS, S.size() * 4, hipMemcpyDeviceToHost));
    const IndexView &v = ix->view;
    const double e = ix->vec_dtype == BOA_VEC_U8 ? 1.0 : 4.0;
    for (int32_t ph = 0; ph < np; ++ph) {
        boa_phase_stats &ps = out->phase[ph];
        ps.L = ix->plans[ph].L;
        ps.launches = ix->plans[ph].launches;
        for (int64_t i = 0; i < nq; ++i) {
            uint8_t s = st[(size_t)ph * nq + i];
            if (!s) continue;
            ps.active += 1;
            ps.confident += (s & 3u) == 2u;
            out->spilled_queries += (s & 4u) != 0;
            ps.expansions += E[(size_t)ph * nq + i];
            ps.scored += S[(size_t)ph * nq + i];
        }
        // a product-quantised search reads a point's code instead of its
        // vector (the exact re-rank's reads are not counted here)
        const double per_scored = ix->last_pq_m ? 4.0 * v.m + ix->last_pq_m / 2 : 4.0 * v.m + v.d * e;
        ps.gathered_bytes = 4.0 * v.R * (double)ps.expansions + per_scored * (double)ps.scored +
                            (v.d * e + 8.0 * v.m + 8.0 * ix->last_k + 4.0) * (double)ps.active;
    }
    for (auto &lp : ix->launch_phase) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, ix->ev_start[lp.second], ix->ev_end[lp.second]));
        out->phase[lp.first].kernel_ms += ms;
    }
    float tot = 0.f;
    HIP_TRY(hipEventElapsedTime(&tot, ix->ev_all0, ix->ev_all1));
    out->total_ms = tot;
    out->cum_searches = ix->cum_searches;
    out->cum_launches = ix->cum_launches;
    out->cum_kernel_ms = ix->cum_kernel_ms;
    for (int i = 0; i < BOA_MAX_PHASES; ++i) {
        out->cum_phase_launches[i] = ix->cum_phase_launches[i];
        out->cum_phase_kernel_ms[i] = ix->cum_phase_kernel_ms[i];
    }
    return BOA_OK;
}

extern "C" int boa_reset_counters(boa_index *ix)
{
    if (!ix) return fail(BOA_EINVAL, "NULL index");
    ix->cum_searches = 0;
    ix->cum_launches = 0;
    ix->cum_kernel_ms = 0.0;
    for (int i = 0; i < BOA_MAX_PHASES; ++i) {
        ix->cum_phase_launches[i] = 0;
        ix->cum_phase_kernel_ms[i] = 0.0;
    }
    return BOA_OK;
}

extern "C" int boa_get_graph(const boa_index *ix, uint32_t *adjacency, int64_t *entry, int64_t *repaired)
{
    if (!ix) return fail(BOA_EINVAL, "NULL index");
    if (entry) *entry = ix->view.entry;
    if (repaired) *repaired = ix->built_graph ? ix->build_stats.repaired : -1;
    if (adjacency) {
        int cur = 0;
        HIP_TRY(hipGetDevice(&cur));
        if (cur != ix->device) return fail(BOA_EINVAL, "index lives on another device than the current one");
        HIP_TRY(hipMemcpy(adjacency, ix->d_adj, (size_t)ix->view.n * ix->view.R * 4, hipMemcpyDeviceToHost));
    }
    return BOA_OK;
}

extern "C" int boa_set_pq(boa_index *ix, const float *codebook, const uint8_t *codes, int32_t M)
{
    if (!ix || !codebook || !codes) return fail(BOA_EINVAL, "NULL argument");
    const int32_t d = ix->view.d;
    if (M < 2 || M % 2 || M > 256 || d % M) return fail(BOA_EINVAL, "M must be even, <= 256 and divide d");
    const int64_t n = ix->view.n;
    int cur = 0;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != ix->device) return fail(BOA_EINVAL, "index lives on another device than the current one");
    float *cb = nullptr;
    uint8_t *cc = nullptr;
    int rc;
    if ((rc = dalloc(&cb, (size_t)M * 16 * (d / M)))) return rc;
    if ((rc = dalloc(&cc, (size_t)n * (M / 2)))) {
        dfree(cb);
        return rc;
    }
    if (hipMemcpy(cb, codebook, (size_t)M * 16 * (d / M) * 4, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(cc, codes, (size_t)n * (M / 2), hipMemcpyHostToDevice) != hipSuccess) {
        dfree(cb);
        dfree(cc);
        return fail(BOA_EHIP, "upload of the product-quantisation data failed");
    }
    dfree(ix->d_pq_cb);
    dfree(ix->d_pq_codes);
    ix->d_pq_cb = cb;
    ix->d_pq_codes = cc;
    ix->pq_m = M;
    return BOA_OK;
}
