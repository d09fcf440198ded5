// Device side of the BOA filtered beam search for gfx950 (CDNA4).
//
// One 64-lane wavefront runs one query at a time: a persistent grid of
// waves pulls query slots from a per-launch atomic counter. Per expansion
// (Alg. 2, one node per iteration):
//   1. select the first not-yet-expanded worklist entry (ballot scan);
//   2. gather its adjacency row, one neighbour per lane (one coalesced load);
//   3. test-and-insert every neighbour into the query's visited set: a
//      two-choice bucketed table of 16-bit entries in LDS whose overflow
//      goes to a per-wave bitmap over all points in HBM, or (the escalation
//      launch of a split search, when it fits) an LDS bitmap over all ids;
//   4. for the unseen neighbours: gather the attribute cells and count the
//      violated range predicates (phi, Eq. 2), gather the vector and compute
//      the squared L2 distance with a 16-lane (float32) or G-lane (uint8)
//      group per candidate and a butterfly reduction;
//   5. pack (phi, distance, id) into one 64-bit key, drop keys that cannot
//      enter the worklist, sort the rest by counting (each key's rank is the
//      number of survivors below it), and merge them into the sorted
//      worklist held in LDS: each new key's rank by binary search (eight-
//      way in the escalation variant), its
//      output slot marked in a bitmap, and the suffix rebuilt backwards in
//      64-entry chunks where a popcount of the bitmap tells every output
//      slot where its entry comes from.
// The epilogue writes the first k filter-valid entries, the phase width,
// and the Eq. 3 confidence flag.
//
// The escalation launch of a split search can instead give each query two
// waves (pair_kernel, below): one merges and selects while the other runs
// the visited test, gathers and scoring of the node it expects next.
//
// Worklist key (unsigned 64-bit, compared as an integer):
//   bits 63..60 phi (violations, <= 8), bits 59..28 float32 bits of the
//   squared distance (non-negative floats order like their bit patterns),
//   bits 27..4 point id (< 2^24), bit 0 expanded flag. Distinct ids make
//   distinct keys, so the flag bits never decide an order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "boa_internal.h"

namespace boa {

// Optional per-stage cycle accounting (build with -DBOA_STAGE_PROFILE): each
// wave adds the shader-clock cycles of every stage of every expansion to its
// slot's row of PhaseArgs::prof. Off in the product build.
#ifdef BOA_STAGE_PROFILE
#define PROF_T(var) const uint64_t var = __builtin_amdgcn_s_memtime()
#define PROF_ADD(i, v) (prof_acc[(i)] += (v))
#else
#define PROF_T(var)
#define PROF_ADD(i, v)
#endif

static constexpr uint64_t KEY_NONE = ~0ull;
static constexpr uint64_t KEY_PHI1 = 1ull << 60;  // smallest key with phi >= 1

__device__ __forceinline__ uint64_t make_key(uint32_t phi, float d, uint32_t id)
{
    return ((uint64_t)phi << 60) | ((uint64_t)__float_as_uint(d) << 28) | ((uint64_t)id << 4);
}
__device__ __forceinline__ uint32_t key_id(uint64_t k) { return (uint32_t)(k >> 4) & 0xFFFFFFu; }
__device__ __forceinline__ float key_dist(uint64_t k) { return __uint_as_float((uint32_t)(k >> 28)); }

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Compiler-level ordering point for LDS data exchanged between lanes of one
// wave (the wave executes in lockstep; this keeps the compiler from caching
// or reordering the shared accesses across it).
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t bcast0(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// value of lane l (wave-uniform l) in every lane, without an LDS round trip
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// first index i in [0, n) with a[i] >= key (a sorted ascending)
__device__ __forceinline__ uint32_t lower_bound64(const uint64_t *a, uint32_t n, uint64_t key)
{
    uint32_t lo = 0, hi = n;
    while (lo < hi) {
        uint32_t mid = (lo + hi) >> 1;
        if (a[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo;
}
// The same index in a[0, P) for a power of two P whose entries from n on
// hold KEY_NONE (greater than any key), by eight-way steps: seven
// independent LDS reads per step at shifted offsets, the same number of
// steps in every lane (512 entries: three eight-way steps and one compare).
// The answer stays in [b, b + s]; pivot j of a step (stride s / 8) is below
// the key exactly when at least j s / 8 entries from b are.
__device__ __forceinline__ uint32_t lower_bound64_p2(const uint64_t *a, uint32_t P, uint64_t key)
{
    uint32_t b = 0, sh = 31u - (uint32_t)__clz(P);   // s = 2^sh = P
    while (sh >= 3u) {   // uniform
        sh -= 3u;
        uint32_t below = 0;
#pragma unroll
        for (uint32_t j = 1; j <= 7; ++j) below += a[b + (j << sh) - 1u] < key ? 1u : 0u;
        b += below << sh;
    }
    while (sh > 0u) {    // s in {2, 4}: halve
        sh -= 1u;
        if (a[b + (1u << sh) - 1u] < key) b += 1u << sh;
    }
    return b + (a[b] < key ? 1u : 0u);
}

// Cross-lane move inside a 16-lane row by DPP (no LDS round trip):
// row_shr:J gives lane i the value of lane i-J; lanes whose source falls
// outside the row receive 0.
template <int J>
__device__ __forceinline__ uint32_t from_lane_minus(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 + J, 0xF, 0xF, false);
}
template <int J>
__device__ __forceinline__ float from_lane_minus_f(float v)
{
    return __uint_as_float(from_lane_minus<J>(__float_as_uint(v)));
}
// ---------------------------------------------------------------------------
// Distance policies. Each lane group computes one candidate's distance per
// round; rounds are unrolled by RU so that RU rows of loads are in flight.

// W = 2 is the variant for launches that hold few waves per CU (the
// escalation of a split search): twice the rows in flight per round trip,
// paid for in registers that such launches do not need for occupancy.
template <int T, int W = 1>
struct F32Scorer {
    // lane p = lane & 15 accumulates float4 chunks p, p+16, p+32, ...
    static constexpr bool kWide = W == 2;
    static constexpr bool kSpec = false;
    static constexpr int kSpecMaxR = 0;
    struct RowGather {};
    __device__ __forceinline__ void gather_row(const void *, int, uint32_t, int, int, RowGather &) const {}
    __device__ __forceinline__ void score_row(const RowGather &, int, int, float *, int) const {}
    // rows of more than 320 dimensions keep the query in LDS rather than in
    // 4T registers (every 16-lane group reads the same chunks: broadcasts)
    static constexpr bool kQueryLds = T >= 6;
    static constexpr int kLdsBytes = kQueryLds ? 16 * T * 16 : 0;
    static constexpr bool kPQ = false;
    float4 q[kQueryLds ? 1 : T];
    float4 *ql = nullptr;

    __device__ __forceinline__ void bind_lds(void *buf) { ql = reinterpret_cast<float4 *>(buf); }

    __device__ __forceinline__ float4 qchunk(int t, int p) const
    {
        if constexpr (kQueryLds) return ql[p + 16 * t];
        else return q[t];
    }

    __device__ __forceinline__ void load_query(const void *Q, uint32_t qi, int d, int lane)
    {
        const float4 *qq = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(Q) + (size_t)qi * d);
        int p = lane & 15, nch = d >> 2;
        if constexpr (kQueryLds) {
            // chunks 0 .. 16T-1, zero past the row (the caller's wave_sync
            // orders these writes before the reads)
            for (int cc = lane; cc < 16 * T; cc += 64) ql[cc] = cc < nch ? qq[cc] : make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
#pragma unroll
            for (int t = 0; t < T; ++t) {
                int cc = p + 16 * t;
                q[t] = cc < nch ? qq[cc] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }

    // rows in flight per round trip: the narrow variant keeps registers for
    // occupancy; the wide one covers most expansions in one round trip
    static constexpr int RU = W == 1 ? (T <= 2 ? 4 : (T <= 4 ? 2 : 1))
                                     : (T <= 2 ? 16 : (T <= 4 ? 8 : (T <= 6 ? 4 : (T <= 12 ? 2 : 1))));
    struct Ids {
        uint32_t v[RU];
    };

    // candidate ids of the round starting at r0 (independent LDS reads; a
    // lane past the candidates takes candidate 0)
    __device__ __forceinline__ void read_ids(const uint32_t *cid, int c, int r0, int lane, Ids &ids) const
    {
        const int g = lane >> 4;
#pragma unroll
        for (int u = 0; u < RU; ++u) {
            const int cj = r0 + 4 * u + g;
            ids.v[u] = cid[cj < c ? cj : 0];
        }
    }

    // `first` holds the ids of the first round, read by the caller together
    // with its own reads of the candidate list
    __device__ __forceinline__ void score(const void *V, int d, const uint32_t *cid, int c, float *cd, int lane,
                                          const Ids &first)
    {
        const float *vec = reinterpret_cast<const float *>(V);
        const int g = lane >> 4, p = lane & 15, nch = d >> 2;
        for (int r0 = 0; r0 < c; r0 += 4 * RU) {
            // the rows: unconditional loads from valid global addresses (a
            // chunk past the row end re-reads its last chunk), masked afterwards
            Ids ids = first;
            if (r0 > 0) read_ids(cid, c, r0, lane, ids);
            const uint32_t *idv = ids.v;
            float4 x[RU][T];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + 4 * u < c) {   // uniform: a candidate left in this round
                    const float4 *row = reinterpret_cast<const float4 *>(vec + (size_t)idv[u] * d);
#pragma unroll
                    for (int t = 0; t < T; ++t) {
                        const int cc = p + 16 * t;
                        x[u][t] = row[cc < nch ? cc : nch - 1];
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + 4 * u >= c) break;   // uniform: no candidate left in this round
                const float acc = dist(x[u], p, nch);
                const int cj = r0 + 4 * u + g;
                if (p == 15 && cj < c) cd[cj] = acc;
            }
        }
    }

    // squared distance of one row held by a 16-lane group (chunk p + 16 t in
    // x[t]); lane 15 of the group returns it
    __device__ __forceinline__ float dist(float4 (&x)[T], int p, int nch) const
    {
        float acc = 0.0f;
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const float4 qv = qchunk(t, p);
            if (p + 16 * t >= nch) x[t] = qv;   // past the row end: adds zero
            float a0 = x[t].x - qv.x;
            acc = __builtin_fmaf(a0, a0, acc);
            float a1 = x[t].y - qv.y;
            acc = __builtin_fmaf(a1, a1, acc);
            float a2 = x[t].z - qv.z;
            acc = __builtin_fmaf(a2, a2, acc);
            float a3 = x[t].w - qv.w;
            acc = __builtin_fmaf(a3, a3, acc);
        }
        // pairwise tree over the 16 partials (p += p+8, +4, +2, +1), mirrored
        // onto the row's top lanes: lane 15 ends with the same sums in the
        // same order (each add is commutative)
        acc = acc + from_lane_minus_f<8>(acc);
        acc = acc + from_lane_minus_f<4>(acc);
        acc = acc + from_lane_minus_f<2>(acc);
        acc = acc + from_lane_minus_f<1>(acc);
        return acc;
    }
};

template <int G, int W = 1>
struct U8Scorer {
    // lane p = lane % G holds the query's 16-byte chunk p (p < d/16); the
    // exact int32 sum is order-free. Per chunk, |x - q|^2 = x.x - 2 x.q + q.q
    // from unsigned 4-byte dot products: every term is an exact integer
    // (at most 16 * 255^2 per lane), so the result is the exact sum of
    // squared differences.
    static constexpr bool kWide = W == 2;
    // rows of at most 128 bytes gather every neighbour of an expanded node
    // before its visited test (gather_row / score_row below)
    static constexpr bool kSpec = G <= 8;
    static constexpr int kLdsBytes = 0;
    static constexpr bool kPQ = false;
    uint4 q;
    uint32_t qq;   // q.q of this lane's chunk

    __device__ __forceinline__ void bind_lds(void *) {}

    __device__ __forceinline__ void load_query(const void *Q, uint32_t qi, int d, int lane)
    {
        const uint8_t *qb = reinterpret_cast<const uint8_t *>(Q) + (size_t)qi * d;
        int p = lane % G;
        q = p < (d >> 4) ? reinterpret_cast<const uint4 *>(qb)[p] : make_uint4(0, 0, 0, 0);
        qq = dot16(q, q);
    }

    static __device__ __forceinline__ uint32_t dot16(const uint4 &a, const uint4 &b)
    {
        uint32_t s = __builtin_amdgcn_udot4(a.x, b.x, 0u, false);
        s = __builtin_amdgcn_udot4(a.y, b.y, s, false);
        s = __builtin_amdgcn_udot4(a.z, b.z, s, false);
        return __builtin_amdgcn_udot4(a.w, b.w, s, false);
    }

    static constexpr int PER = 64 / G;   // candidates per round
    // rows in flight per round trip of score(); with row gathers it scores
    // only the entry point and rows longer than the gathers cover
    static constexpr int RU = (W == 1 || G <= 8) ? (G <= 8 ? 2 : 4) : (G <= 16 ? G : 16);
    struct Ids {
        uint32_t v[RU];
    };

    __device__ __forceinline__ void read_ids(const uint32_t *cid, int c, int r0, int lane, Ids &ids) const
    {
        const int g = lane / G;
#pragma unroll
        for (int u = 0; u < RU; ++u) {
            const int cj = r0 + PER * u + g;
            ids.v[u] = cid[cj < c ? cj : 0];
        }
    }

    __device__ __forceinline__ void score(const void *V, int d, const uint32_t *cid, int c, float *cd, int lane,
                                          const Ids &first)
    {
        const uint8_t *vec = reinterpret_cast<const uint8_t *>(V);
        const int g = lane / G, p = lane % G, nch = d >> 4;
        for (int r0 = 0; r0 < c; r0 += PER * RU) {
            // unconditional loads from valid addresses, masked afterwards (as
            // in F32Scorer)
            Ids ids = first;
            if (r0 > 0) read_ids(cid, c, r0, lane, ids);
            const uint32_t *idv = ids.v;
            uint4 x[RU];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + PER * u < c)   // uniform
                    x[u] = reinterpret_cast<const uint4 *>(vec + (size_t)idv[u] * d)[p < nch ? p : nch - 1];
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + PER * u >= c) break;   // uniform: no candidate left in this round
                const int32_t acc = dist(x[u], p, nch);
                const int cj = r0 + PER * u + g;
                if (p == G - 1 && cj < c) cd[cj] = (float)acc;
            }
        }
    }

    // Every neighbour of an expanded node, before its visited test: lane j
    // holds row entry j (padding replaced by a valid id), and round u's
    // G-lane group g loads chunk p of entry PER u + g. All rounds' loads are
    // issued together; score_row waits for them.
    static constexpr int RS_ALL = (BOA_MAX_R + PER - 1) / PER;
    static constexpr int RS = !kSpec ? 1 : (RS_ALL < 4 ? RS_ALL : 4);
    static constexpr int kSpecMaxR = kSpec ? PER * RS : 0;   // longer rows take the other path
    struct RowGather {
        uint4 x[RS];
    };

    __device__ __forceinline__ void gather_row(const void *V, int d, uint32_t v, int R, int lane,
                                               RowGather &rg) const
    {
        const uint8_t *vec = reinterpret_cast<const uint8_t *>(V);
        const int g = lane / G, p = lane % G, nch = d >> 4;
        // every round's id first (cross-lane reads in flight together), then
        // the loads
        uint32_t id[RS];
#pragma unroll
        for (int u = 0; u < RS; ++u) id[u] = (uint32_t)__shfl((int)v, (PER * u + g) & 63);
#pragma unroll
        for (int u = 0; u < RS; ++u) {
            if (PER * u < R)   // uniform
                rg.x[u] = reinterpret_cast<const uint4 *>(vec + (size_t)id[u] * d)[p < nch ? p : nch - 1];
        }
    }

    // distances of the gathered entries: cd[j] for j < R
    __device__ __forceinline__ void score_row(const RowGather &rg, int d, int R, float *cd, int lane) const
    {
        const int g = lane / G, p = lane % G, nch = d >> 4;
#pragma unroll
        for (int u = 0; u < RS; ++u) {
            if (PER * u >= R) break;   // uniform
            const int32_t acc = dist(rg.x[u], p, nch);
            const int cj = PER * u + g;
            if (p == G - 1) cd[cj] = (float)acc;   // (cj < 32: slots past R are not read)
        }
    }

    // exact squared distance of one row held by a G-lane group (16-byte
    // chunk p in x); the group's top lane returns it
    __device__ __forceinline__ int32_t dist(uint4 x, int p, int nch) const
    {
        int32_t acc = (int32_t)(dot16(x, x) + qq - 2u * dot16(x, q));
        if (nch < G) {         // (uniform) lanes past the row add zero
            if (p >= nch) acc = 0;
        }
        // exact integer sum over the group; the group's top lane holds it
#pragma unroll
        for (int s = G >> 1; s >= 16; s >>= 1) acc += __shfl_xor(acc, s);
        if (G >= 16) acc += (int32_t)from_lane_minus<8>((uint32_t)acc);
        if (G >= 8) acc += (int32_t)from_lane_minus<4>((uint32_t)acc);
        if (G >= 4) acc += (int32_t)from_lane_minus<2>((uint32_t)acc);
        if (G >= 2) acc += (int32_t)from_lane_minus<1>((uint32_t)acc);
        return acc;
    }
};

// Product-quantised asymmetric distance (Alg. 2 "PQDist"): 4-bit codes, 16
// centroids per subspace. The query's distance table (M x 16 float32) lives
// in LDS; a 16-lane group scores one candidate, lane p adding the entries of
// subspaces p, p+16, ... in increasing order (nibble (p + 16t) of the packed
// code), then the same pairwise tree as the exact float32 distance.
template <int T>
struct PQScorer {
    static constexpr bool kWide = false;
    static constexpr bool kSpec = false;
    static constexpr int kSpecMaxR = 0;
    struct RowGather {};
    __device__ __forceinline__ void gather_row(const void *, int, uint32_t, int, int, RowGather &) const {}
    __device__ __forceinline__ void score_row(const RowGather &, int, int, float *, int) const {}
    static constexpr bool kPQ = true;
    static constexpr int kLdsBytes = 16 * T * 16 * 4;   // the table of up to 16 T subspaces
    float *lut = nullptr;
    const uint8_t *codes = nullptr;
    const float *cb = nullptr;
    int M = 0, half = 0, ds = 0, u8 = 0;

    __device__ __forceinline__ void bind_lds(void *buf) { lut = reinterpret_cast<float *>(buf); }
    __device__ __forceinline__ void bind_pq(const uint8_t *c, int m, const float *codebook, int d, int vec_u8)
    {
        codes = c;
        M = m;
        half = m >> 1;
        cb = codebook;
        ds = d / m;
        u8 = vec_u8;
    }

    // table entry (m, c): fma chain over the subspace's dimensions from +0
    // (the caller's wave_sync orders these writes before the reads)
    __device__ __forceinline__ void load_query(const void *Q, uint32_t qi, int d, int lane)
    {
        for (int e = lane; e < M * 16; e += 64) {
            const int m = e >> 4, c = e & 15;
            float acc = 0.0f;
            for (int j = 0; j < ds; ++j) {
                const size_t qo = (size_t)qi * d + m * ds + j;
                const float qv = u8 ? (float)reinterpret_cast<const uint8_t *>(Q)[qo]
                                    : reinterpret_cast<const float *>(Q)[qo];
                const float diff = qv - cb[((size_t)m * 16 + c) * ds + j];
                acc = __builtin_fmaf(diff, diff, acc);
            }
            lut[e] = acc;
        }
    }

    static constexpr int RU = T <= 4 ? 4 : 2;   // rounds of 4 candidates per round trip
    struct Ids {
        uint32_t v[RU];
    };

    __device__ __forceinline__ void read_ids(const uint32_t *cid, int c, int r0, int lane, Ids &ids) const
    {
        const int g = lane >> 4;
#pragma unroll
        for (int u = 0; u < RU; ++u) {
            const int cj = r0 + 4 * u + g;
            ids.v[u] = cid[cj < c ? cj : 0];
        }
    }

    __device__ __forceinline__ void score(const void *, int, const uint32_t *cid, int c, float *cd, int lane,
                                          const Ids &first)
    {
        const int g = lane >> 4, p = lane & 15;
        for (int r0 = 0; r0 < c; r0 += 4 * RU) {
            Ids ids = first;
            if (r0 > 0) read_ids(cid, c, r0, lane, ids);
            uint32_t b[RU][T];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + 4 * u < c) {   // uniform
                    const uint8_t *row = codes + (size_t)ids.v[u] * half;
#pragma unroll
                    for (int t = 0; t < T; ++t) {
                        const int m = p + 16 * t;
                        b[u][t] = row[(m < M ? m : M - 1) >> 1];   // a valid byte; masked below
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                if (r0 + 4 * u >= c) break;   // uniform
                float acc = 0.0f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const int m = p + 16 * t;
                    if (m < M) acc = acc + lut[m * 16 + ((b[u][t] >> (4 * (m & 1))) & 15u)];
                }
                acc = acc + from_lane_minus_f<8>(acc);
                acc = acc + from_lane_minus_f<4>(acc);
                acc = acc + from_lane_minus_f<2>(acc);
                acc = acc + from_lane_minus_f<1>(acc);
                const int cj = r0 + 4 * u + g;
                if (p == 15 && cj < c) cd[cj] = acc;
            }
        }
    }
};

// Exact squared distance of one point to the query, computed by one lane in
// the fixed order of the float32 path (16 partials over 4-dimension chunks,
// then pairwise), or exactly in int32 for uint8 vectors: the re-rank of a
// product-quantised search.
__device__ __forceinline__ float exact_dist_lane(const void *V, const void *Q, uint32_t qi, uint32_t id, int d,
                                                 bool u8)
{
    if (u8) {
        const uint4 *x = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint8_t *>(V) + (size_t)id * d);
        const uint4 *q = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint8_t *>(Q) + (size_t)qi * d);
        int32_t s = 0;
        for (int c = 0; c < (d >> 4); ++c) {
            const uint4 a = x[c], b = q[c];
            const uint32_t wa[4] = {a.x, a.y, a.z, a.w}, wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int w = 0; w < 4; ++w)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int32_t t = (int32_t)((wa[w] >> (8 * i)) & 0xFF) - (int32_t)((wb[w] >> (8 * i)) & 0xFF);
                    s += t * t;
                }
        }
        return (float)s;
    }
    const float4 *x = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(V) + (size_t)id * d);
    const float4 *q = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(Q) + (size_t)qi * d);
    const int nch = d >> 2;
    float acc[16];
#pragma unroll
    for (int pp = 0; pp < 16; ++pp) acc[pp] = 0.0f;
    for (int c0 = 0; c0 < nch; c0 += 16) {
#pragma unroll
        for (int pp = 0; pp < 16; ++pp) {
            if (c0 + pp < nch) {
                const float4 a = x[c0 + pp], b = q[c0 + pp];
                float t = a.x - b.x;
                acc[pp] = __builtin_fmaf(t, t, acc[pp]);
                t = a.y - b.y;
                acc[pp] = __builtin_fmaf(t, t, acc[pp]);
                t = a.z - b.z;
                acc[pp] = __builtin_fmaf(t, t, acc[pp]);
                t = a.w - b.w;
                acc[pp] = __builtin_fmaf(t, t, acc[pp]);
            }
        }
    }
#pragma unroll
    for (int st = 8; st >= 1; st >>= 1)
#pragma unroll
        for (int pp = 0; pp < st; ++pp) acc[pp] = acc[pp] + acc[pp + st];
    return acc[0];
}

__device__ __forceinline__ uint64_t wave_min64(uint64_t v)
{
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        const uint64_t o = ((uint64_t)(uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), s) << 32) |
                           (uint32_t)__shfl_xor((int)(uint32_t)v, s);
        v = o < v ? o : v;
    }
    return v;
}

// ---------------------------------------------------------------------------
// Attribute filter (Eq. 2). A point's record is m_pad cells, loaded as one
// aligned vector load (int4 halves w0, w1). The index holds float32 cells
// as order-preserving integers (f32_ord), and RangeTest maps each query's
// bounds the same way, so a cell satisfies its range [lo, hi] exactly when
// (uint32)(x - lo) <= hi - lo. A range that nothing satisfies (lo > hi, or a
// NaN bound of a float32 column, which fails every comparison) counts in
// phi0 for every point; its cell, like a padding cell, then passes.

__device__ __forceinline__ void load_attr_record(const IndexView &ix, uint32_t id, int4 &w0, int4 &w1)
{
    const int32_t *ar = ix.attrs + (size_t)id * ix.m_pad;
    if (ix.m_pad >= 4) {
        w0 = reinterpret_cast<const int4 *>(ar)[0];
        if (ix.m_pad == 8) w1 = reinterpret_cast<const int4 *>(ar)[1];
    } else if (ix.m_pad == 2) {
        const int2 t2 = reinterpret_cast<const int2 *>(ar)[0];
        w0.x = t2.x;
        w0.y = t2.y;
    } else {
        w0.x = ar[0];
    }
}

struct RangeTest {
    int32_t flo[BOA_MAX_M];
    uint32_t fspan[BOA_MAX_M];
    uint32_t phi0;

    // query qi's m ranges (row-major nq x m x 2 cells)
    __device__ __forceinline__ void set(const int32_t *ranges, uint32_t qi, int m, uint32_t f32_mask)
    {
        phi0 = 0;
#pragma unroll
        for (int j = 0; j < BOA_MAX_M; ++j) {
            int32_t l = 0;
            uint32_t s = 0xFFFFFFFFu;   // (padding cells pass)
            if (j < m) {
                int32_t lo = ranges[((size_t)qi * m + j) * 2 + 0];
                int32_t hi = ranges[((size_t)qi * m + j) * 2 + 1];
                bool none = false;
                if ((f32_mask >> j) & 1u) {
                    none = ((uint32_t)lo & 0x7FFFFFFFu) > 0x7F800000u || ((uint32_t)hi & 0x7FFFFFFFu) > 0x7F800000u;
                    lo = f32_ord((uint32_t)lo);
                    hi = f32_ord((uint32_t)hi);
                }
                if (none || lo > hi) {
                    phi0 += 1;
                } else {
                    l = lo;
                    s = (uint32_t)hi - (uint32_t)lo;
                }
            }
            // (held in vector registers: kept uniform they would be spilled
            // scalars, reloaded at every use)
            asm volatile("" : "+v"(l), "+v"(s));
            flo[j] = l;
            fspan[j] = s;
        }
    }

    // phi of a record: its m_pad cells (one uniform dispatch, no per-cell tests)
    __device__ __forceinline__ uint32_t phi(const int4 &w0, const int4 &w1, int m_pad) const
    {
        const int32_t av[BOA_MAX_M] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
        auto cells = [&](auto nc_tag) -> uint32_t {
            constexpr int NC = decltype(nc_tag)::value;
            uint32_t p = phi0;
#pragma unroll
            for (int j = 0; j < NC; ++j) p += (uint32_t)(av[j] - flo[j]) > fspan[j] ? 1u : 0u;
            return p;
        };
        switch (m_pad) {
        case 1: return cells(std::integral_constant<int, 1>{});
        case 2: return cells(std::integral_constant<int, 2>{});
        case 4: return cells(std::integral_constant<int, 4>{});
        default: return cells(std::integral_constant<int, 8>{});
        }
    }
};

// ---------------------------------------------------------------------------
// Visited set (exact). LDS part: a two-choice bucketed table of 16-bit
// entries. A bijective mix of the id's B bits gives h; its top bits select
// the home bucket b1, the low r = B - log2(buckets) <= 15 bits are stored.
// The alternate bucket is b2 = b1 ^ alt(r) (alt odd, so b2 != b1). An entry
// is r in b1 or 0x8000 | r in b2, so (bucket, entry) identifies the id
// uniquely; 0xFFFF marks a free slot, so an id whose r is 0x7FFF has no
// alternate bucket. A bucket holds 8 entries (16 bytes, one LDS read).
// Insert goes to the emptier bucket through a 32-bit CAS on the word that
// holds the slot. When both buckets are full the id goes to the wave slot's
// bitmap over all points in HBM (cleared when a query first overflows).
// Buckets only fill up, so an id absent from a bucket pair that still has
// room has never been inserted anywhere: the bitmap is consulted only when
// both buckets are full.
// The bitmap keeps a log of the ids whose bits were set since it was last
// clear, so that the clear rewrites only their words; when the log is full
// (or its state unknown, header BOA_LOG_DIRTY) the whole bitmap is cleared.
// The wave holds the log's length in a register and writes it back to the
// header when it exits.

struct Visited {
    uint32_t *words;     // LDS table, 2 entries per word, 4 words per bucket
    uint32_t bmask;      // buckets - 1
    uint32_t rbits;      // stored bits per id
    uint32_t idbits;     // B
    uint32_t *bits;      // this wave slot's HBM bitmap, words32 words
    uint32_t words32;
    uint32_t *log;       // its log: header word, then (after BOA_LOG_HDR words) log_cap ids
    uint32_t log_cap;
    uint32_t *status;
};

// ids have at most 24 bits (BOA_MAX_N), so 24-bit multiplies (full rate)
// by odd constants are bijections modulo 2^B
__device__ __forceinline__ uint32_t mix_id(uint32_t v, uint32_t B)
{
    const uint32_t mask = (1u << B) - 1u;
    uint32_t h = __umul24(v, 0x3779B1u) & mask;
    h ^= h >> ((B + 1u) >> 1);
    return __umul24(h, 0xEBCA6Bu) & mask;
}

// Bit 15 of each 16-bit half of the result is set when that half of w is
// zero (the masked add sets bit 15 of a half exactly when its low 15 bits
// are not all zero, and no carry crosses into the other half).
__device__ __forceinline__ uint32_t zero_halves(uint32_t w)
{
    const uint32_t t = (w & 0x7FFF7FFFu) + 0x7FFF7FFFu;
    return ~(t | w) & 0x80008000u;
}

__device__ __forceinline__ bool has16(const uint4 &b, uint32_t e)
{
    const uint32_t ee = e * 0x00010001u;
    return (zero_halves(b.x ^ ee) | zero_halves(b.y ^ ee) | zero_halves(b.z ^ ee) | zero_halves(b.w ^ ee)) != 0u;
}

// free slots (0xFFFF halves) of a bucket
__device__ __forceinline__ uint32_t empties16(const uint4 &b)
{
    return (uint32_t)__popc(zero_halves(~b.x) | (zero_halves(~b.y) >> 1) | (zero_halves(~b.z) >> 2) |
                            (zero_halves(~b.w) >> 3));
}

// 1: v was not in the set and now is (in LDS); 0: v was already there;
// -1: both buckets full and v not in them (the caller consults the bitmap).
__device__ __forceinline__ int visit_lds(const Visited &s, uint32_t v)
{
    const uint32_t h = mix_id(v, s.idbits);
    const uint32_t r = h & ((1u << s.rbits) - 1u);
    const uint32_t b1 = h >> s.rbits;
    const uint32_t b2 = (b1 ^ (((__umul24(r, 0xD1E995u) + 0x7F4A7C15u) >> 7) | 1u)) & s.bmask;
    const uint32_t e1 = r, e2 = 0x8000u | r;
    const bool alt_ok = e2 != 0xFFFFu;
    const uint4 *bk = reinterpret_cast<const uint4 *>(s.words);
    for (int attempt = 0; attempt < 256; ++attempt) {
        // both buckets read before either is tested: one LDS round trip
        const uint4 B1 = bk[b1], B2 = bk[b2];
        if (has16(B1, e1) | (alt_ok && has16(B2, e2))) return 0;
        const uint32_t n1 = empties16(B1), n2 = alt_ok ? empties16(B2) : 0u;
        if (n1 == 0u && n2 == 0u) return -1;
        const bool use1 = n1 >= n2;
        const uint4 Bc = use1 ? B1 : B2;
        const uint32_t e = use1 ? e1 : e2;
        const uint32_t bi = use1 ? b1 : b2;
        // first (lowest) free half-word: the lowest word with a free half,
        // its low half when that one is free
        const uint32_t w[4] = {Bc.x, Bc.y, Bc.z, Bc.w};
        uint32_t wi = 0, old = 0, neu = 0;
#pragma unroll
        for (int q = 3; q >= 0; --q) {
            const uint32_t zq = zero_halves(~w[q]);
            if (zq) {
                wi = q;
                old = w[q];
                neu = (zq & 0x8000u) ? ((w[q] & 0xFFFF0000u) | e) : ((w[q] & 0x0000FFFFu) | (e << 16));
            }
        }
        if (atomicCAS(&s.words[bi * 4u + wi], old, neu) == old) return 1;
        // another lane changed that word: look again
    }
    atomicOr(s.status, BOA_STATUS_OVERFLOW);
    return 0;
}

__device__ __forceinline__ bool visit_bits(const Visited &s, uint32_t v)
{
    uint32_t bit = 1u << (v & 31u);
    uint32_t old = atomicOr(&s.bits[v >> 5], bit);
    return (old & bit) == 0u;
}

// Clear the bitmap before a query's first spill: the words of the n_log
// logged ids, or every word when the log does not cover the set bits.
__device__ __forceinline__ void clear_bits(const Visited &s, uint32_t n_log, int lane)
{
    if (n_log <= s.log_cap) {
        const uint32_t *ids = s.log + BOA_LOG_HDR;
        uint32_t i = lane;
        for (; i + 192 < n_log; i += 256) {   // four loads in flight, then their stores
            const uint32_t v0 = ids[i], v1 = ids[i + 64], v2 = ids[i + 128], v3 = ids[i + 192];
            s.bits[v0 >> 5] = 0u;
            s.bits[v1 >> 5] = 0u;
            s.bits[v2 >> 5] = 0u;
            s.bits[v3 >> 5] = 0u;
        }
        for (; i < n_log; i += 64) s.bits[ids[i] >> 5] = 0u;
    } else {
        uint4 z = make_uint4(0, 0, 0, 0);
        uint4 *b4 = reinterpret_cast<uint4 *>(s.bits);
        for (uint32_t i = lane; i < (s.words32 >> 2); i += 64) b4[i] = z;
    }
    // the stores must land before this wave's atomics on the same words
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
}

// ---------------------------------------------------------------------------

template <class Scorer>
__global__ void __launch_bounds__(256) phase_kernel(PhaseArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = lane_id();
    const int wid = threadIdx.x >> 6;
    const uint32_t slot = a.slot_base + blockIdx.x * a.waves_per_block + wid;

    // per-wave LDS: worklist, sorted new keys, output-slot bitmap, candidate
    // ids and distances, visited table; sized for the widest phase of the launch
    unsigned char *mine = smem + (size_t)wid * a.lds_per_wave;
    // (sizes keep every array 16-byte aligned: Lb and the bitmap word count are even)
    const int Lb = beam_slots(a.L_alloc);
    const int pw = ((a.L_alloc >> 6) + 3) & ~1;
    uint64_t *beam = reinterpret_cast<uint64_t *>(mine);         // Lb
    uint64_t *nkey = beam + Lb;                                  // 64
    uint64_t *posbm = nkey + 64;                                 // pw >= L/64 + 2
    uint32_t *cid = reinterpret_cast<uint32_t *>(posbm + pw);   // 64
    float *cd = reinterpret_cast<float *>(cid + 64);             // 64
    unsigned char *qlds = reinterpret_cast<unsigned char *>(cd + 64);   // the scorer's query copy or table
    // the exact re-rank keys of a product-quantised search (Lb entries)
    uint64_t *rrk = reinterpret_cast<uint64_t *>(qlds + Scorer::kLdsBytes);
    uint32_t *htab = reinterpret_cast<uint32_t *>(rrk + (Scorer::kPQ ? Lb : 0));   // H/2 words (H 16-bit slots)

    const IndexView ix = a.ix;
    int R = ix.R;   // (made opaque once per expansion, see there)
    const int d = ix.d, m = ix.m;
    // row gathers ahead of the visited test (scorers that have them, rows they cover)
    const bool spec = Scorer::kSpec && R <= Scorer::kSpecMaxR;

    const uint32_t n_in = bcast0(*a.n_active);
    if (n_in <= a.tau_count) return;   // the loop of Alg. 1 has stopped
    const uint32_t nA = a.t_end < n_in ? a.t_end : n_in;

    Visited vs;
    vs.words = htab;
    vs.bmask = (1u << (a.h_log2 - 3)) - 1u;       // 8 slots per bucket
    vs.idbits = a.id_bits;
    vs.rbits = a.id_bits > (uint32_t)(a.h_log2 - 3) ? a.id_bits - (uint32_t)(a.h_log2 - 3) : 0u;
    vs.words32 = a.bits_words;
    vs.bits = a.bits + (size_t)slot * a.slot_words;
    vs.log = vs.bits + a.bits_words;
    vs.log_cap = a.log_cap;
    vs.status = a.status;
    // ids logged in this slot's bitmap (its header, kept in a register while
    // this wave runs: no other wave uses the slot meanwhile)
    uint32_t n_log = a.vis_bitmap ? 0u : __builtin_amdgcn_readfirstlane(vs.log[0]);
    const uint32_t table_words = a.vis_bitmap ? a.vis_words : (1u << a.h_log2) >> 1;

    Scorer sc;
    sc.bind_lds(qlds);
    if constexpr (Scorer::kPQ) sc.bind_pq(a.pq_codes, a.pq_m, a.pq_cb, d, a.vec_u8);
    // one point's attribute record (m_pad cells) and its violation count (Eq. 2)
    auto load_attrs = [&](uint32_t id, int4 &w0, int4 &w1) { load_attr_record(ix, id, w0, w1); };
    RangeTest rt;
    auto count_phi = [&](const int4 &w0, const int4 &w1) -> uint32_t { return rt.phi(w0, w1, ix.m_pad); };
#ifdef BOA_STAGE_PROFILE
    uint64_t prof_acc[BOA_PROF_SLOTS] = {};
#endif
    for (;;) {
        uint32_t t = 0;
        if (lane == 0) t = atomicAdd(a.queue, 1u);
        t = bcast0(t) + a.t_begin;
        if (t >= nA) break;
        const uint32_t qi = bcast0(a.active[t]);

        sc.load_query(a.queries, qi, d, lane);
        rt.set(a.ranges, qi, m, ix.f32_mask);
        // the phases of this launch: each restarts the search from the entry
        // point at its own width (Alg. 1 calls Alg. 2 afresh)
        // search state; in the warm-start mode it carries over from phase to
        // phase (the worklist, its expanded flags and the visited set)
        bool spill = false;
        uint32_t len = 0;
        for (int p = a.p_begin; p < a.p_end; ++p) {
        const int L = a.sched[p];
        // warm start: the list keeps up to the next phase's width while only
        // its first L entries are expanded (the last phase keeps L)
        const int Lcap = (a.warm && p + 1 < a.p_end) ? a.sched[p + 1] : L;
        const bool fresh = !a.warm || p == a.p_begin;
        if (fresh) {
            // the bitmap starts with no bit set, the table with every slot
            // free, the worklist with every slot past its (zero) length KEY_NONE
            const uint32_t f = a.vis_bitmap ? 0u : 0xFFFFFFFFu;
            const uint4 z = make_uint4(f, f, f, f);
            uint4 *h4 = reinterpret_cast<uint4 *>(htab);
            for (uint32_t i = lane; i < table_words >> 2; i += 64) h4[i] = z;
            for (int i = lane; i < Lb; i += 64) beam[i] = KEY_NONE;
            spill = false;
            len = 0;
        }
        wave_sync();

        // test-and-insert of this lane's neighbour: 1 new, 0 seen (or padding)
        auto visit_test = [&](uint32_t v) -> int {
            if (a.vis_bitmap) {   // one bit per id: a single LDS atomic
                if (v == BOA_PAD) return 0;
                const uint32_t bit = 1u << (v & 31u);
                return (atomicOr(&htab[v >> 5], bit) & bit) ? 0 : 1;
            }
            int vst = 0;
            if (v != BOA_PAD) vst = visit_lds(vs, v);
            if (__ballot(vst < 0) != 0ull) {
                if (!spill) {          // first overflow of this query: reset the bitmap
                    spill = true;
                    clear_bits(vs, n_log, lane);
                    n_log = 0;
                }
                const bool to_bits = vst < 0;
                if (to_bits) vst = visit_bits(vs, v) ? 1 : 0;
                // log the ids whose bits this wave has just set
                const uint64_t lm = __ballot(to_bits && vst > 0);
                if (lm) {
                    const uint32_t cnt = (uint32_t)__popcll(lm);
                    if (n_log <= vs.log_cap && cnt <= vs.log_cap - n_log) {
                        if (to_bits && vst > 0) vs.log[BOA_LOG_HDR + n_log + lanes_below(lm)] = v;
                        n_log += cnt;
                    } else {
                        n_log = BOA_LOG_DIRTY;
                    }
                }
            }
            return vst;
        };
        uint32_t E = 0, S = 0;
        int expanded_j = -1;
        // adjacency row already in flight for the node expected next
        uint32_t pf_id = BOA_PAD;
        uint64_t pf_key = KEY_NONE;
        uint32_t pf_row = BOA_PAD;

        // the entry point is scored and entered before the first expansion
        // (a warm phase continues with nothing new to score)
        uint32_t c = fresh ? 1u : 0u;
        if (fresh && lane == 0) {
            if (a.vis_bitmap) htab[ix.entry >> 5] |= 1u << (ix.entry & 31u);
            else visit_lds(vs, ix.entry);
            cid[0] = ix.entry;
        }
        // row-gather scorers: the keys of the last expansion's new
        // neighbours (one per row position, KEY_NONE elsewhere), scored in
        // that expansion and entered at the top of the next iteration
        uint32_t spec_c = 0;
        uint64_t spec_key = KEY_NONE;

        for (;;) {
            // Row-gather scorers re-read the row length as an opaque (uniform)
            // value at every expansion, so that tests on it (lane < R, the
            // number of gather rounds) are recomputed where they are used
            // instead of being hoisted out of the loop as lane masks, which
            // would not fit the scalar registers and would be reloaded from
            // spill lanes at every use. (The other scorers spill more with it.
            // The same for the lane number moves waits for the prefetched row
            // earlier.)
            if constexpr (Scorer::kSpec) {
                int r = R;
                asm volatile("" : "+v"(r));
                R = __builtin_amdgcn_readfirstlane(r);
            }
            uint32_t scan_from = (uint32_t)(expanded_j + 1);
            // ---- score the c new candidates listed in cid[0, c)
            PROF_T(t_score0);
            if (c > 0 || spec_c > 0) {
                wave_sync();
                uint64_t key = KEY_NONE;
                if (Scorer::kSpec && spec_c > 0) {
                    S += spec_c;
                    key = spec_key;
                    spec_c = 0;
                } else {
                    S += c;
                    // attribute records first, then the vectors, so that both
                    // gathers are in flight together; phi is counted afterwards.
                    // This lane's candidate (for its attribute record) and the
                    // scorer's first round of ids: LDS reads issued together
                    const uint32_t my_id = cid[lane];
                    typename Scorer::Ids ids0;
                    sc.read_ids(cid, (int)c, 0, lane, ids0);
                    int4 w0 = make_int4(0, 0, 0, 0), w1 = make_int4(0, 0, 0, 0);
                    if (lane < (int)c) load_attrs(my_id, w0, w1);
                    sc.score(a.ix.vectors, d, cid, (int)c, cd, lane, ids0);
                    const uint32_t phi = count_phi(w0, w1);
                    wave_sync();
                    if (lane < (int)c) key = make_key(phi, cd[lane], cid[lane]);
                    c = 0;
                }
                PROF_T(t_score1);
                PROF_ADD(2, t_score1 - t_score0);
                if (len == (uint32_t)Lcap && key >= beam[Lcap - 1]) key = KEY_NONE;  // cannot enter
                const uint64_t keep = __ballot(key != KEY_NONE);
                const uint32_t kept = __popcll(keep);
                if (kept > 0) {
                    // sort the survivors: each one's rank is the number of
                    // survivors below it (keys are distinct), read back from
                    // LDS as broadcasts, two keys per read
                    // survivors first, the other lanes' KEY_NONE after them, so
                    // that reads past the survivors compare false
                    nkey[key != KEY_NONE ? lanes_below(keep) : kept + lanes_below(~keep)] = key;
                    wave_sync();
                    uint32_t rank = 0;
                    {
                        // eight keys per step: four independent LDS reads in flight
                        const ulonglong2 *nk2 = reinterpret_cast<const ulonglong2 *>(nkey);
                        for (uint32_t i = 0; i < kept; i += 8) {
                            const ulonglong2 a0 = nk2[(i >> 1) + 0], a1 = nk2[(i >> 1) + 1];
                            const ulonglong2 a2 = nk2[(i >> 1) + 2], a3 = nk2[(i >> 1) + 3];
                            rank += (a0.x < key ? 1u : 0u) + (a0.y < key ? 1u : 0u);
                            rank += (a1.x < key ? 1u : 0u) + (a1.y < key ? 1u : 0u);
                            rank += (a2.x < key ? 1u : 0u) + (a2.y < key ? 1u : 0u);
                            rank += (a3.x < key ? 1u : 0u) + (a3.y < key ? 1u : 0u);
                        }
                    }
                    wave_sync();
                    if (key != KEY_NONE) nkey[rank] = key;
                    wave_sync();
                    key = lane < (int)kept ? nkey[lane] : KEY_NONE;
                    // the next node is the smaller of the best new key and the
                    // entry predicted at selection: start its row load now
                    {
                        const uint64_t k0 = __shfl(key, 0);
                        if (k0 < pf_key) {
                            pf_key = k0;
                            pf_id = key_id(k0);
                            pf_row = ix.adj[(size_t)pf_id * R + (lane < R ? lane : R - 1)];
                            PROF_ADD(9, 1);
                        }
                    }
                    PROF_T(t_sort1);
                    PROF_ADD(3, t_sort1 - t_score1);
                    // rank of each new key in the worklist and its output slot
                    uint32_t f = 0xFFFFFFFFu;
                    uint32_t pos = 0;
                    if (lane < (int)kept) {
                        pos = lower_bound64_p2(beam, (uint32_t)beam_slots((int32_t)len), key);
                        f = pos + lane;
                    }
                    const uint32_t p0 = bcast0(pos);
                    const uint32_t newlen = min((uint32_t)Lcap, len + kept);
                    const uint32_t w_lo = bcast0(p0 >> 6), w_hi = bcast0((newlen - 1u) >> 6);
                    for (uint32_t w = w_lo + lane; w <= w_hi; w += 64) posbm[w] = 0ull;
                    wave_sync();
                    const bool placed = f < (uint32_t)Lcap;
                    if (placed) atomicOr(reinterpret_cast<unsigned long long *>(&posbm[f >> 6]),
                                         1ull << (f & 63u));
                    const uint32_t n_placed = __popcll(__ballot(placed));
                    wave_sync();
                    PROF_T(t_rank1);
                    PROF_ADD(4, t_rank1 - t_sort1);
                    PROF_ADD(7, w_hi - w_lo + 1);
                    // rebuild [p0, newlen) from the last 64-slot chunk down
                    uint64_t word = posbm[w_hi];
                    uint32_t below = n_placed - (uint32_t)__popcll(word);   // new keys before chunk
                    for (int w = (int)w_hi; w >= (int)w_lo; --w) {
                        const uint32_t o = ((uint32_t)w << 6) + lane;
                        const bool act = o >= p0 && o < newlen;
                        const bool isnew = (word >> lane) & 1ull;
                        const uint32_t cnt = below + (uint32_t)__popcll(word & ((1ull << lane) - 1ull));
                        uint64_t val = 0;
                        if (act) val = isnew ? nkey[cnt] : beam[o - cnt];
                        wave_sync();
                        if (act) beam[o] = val;
                        if (w > (int)w_lo) {
                            word = posbm[w - 1];
                            below -= (uint32_t)__popcll(word);
                        }
                        wave_sync();
                    }
                    len = newlen;
                    if (p0 < scan_from) scan_from = p0;
                    PROF_T(t_merge1);
                    PROF_ADD(5, t_merge1 - t_rank1);
                }
            }
            PROF_T(t_sel0);

            // ---- select the nearest unexpanded entry among the first L (and
            // predict the one after it)
            const uint32_t lim = min(len, (uint32_t)L);
            int j = -1, j2 = -1;
            uint64_t ku = 0, kn = KEY_NONE;   // their keys, taken from the lanes that read them
            for (uint32_t b0 = scan_from; b0 < lim; b0 += 64) {
                const uint32_t i = b0 + lane;
                const uint64_t bk = i < lim ? beam[i] : 1ull;
                const uint64_t mk = __ballot(!(bk & 1ull));
                if (mk) {
                    const int l1 = __ffsll((unsigned long long)mk) - 1;
                    j = (int)b0 + l1;
                    ku = readlane64(bk, l1);
                    const uint64_t rest = mk & (mk - 1ull);
                    if (rest) {
                        const int l2 = __ffsll((unsigned long long)rest) - 1;
                        j2 = (int)b0 + l2;
                        kn = readlane64(bk, l2);
                    }
                    break;
                }
            }
            if (j < 0) break;   // converged: every entry expanded
            PROF_T(t_sel1);
            PROF_ADD(0, t_sel1 - t_sel0);
            expanded_j = j;
            wave_sync();
            if (lane == 0) beam[j] = ku | 1ull;
            const uint32_t u = key_id(ku);
            E += 1;

            // ---- adjacency row (prefetched if predicted)
            uint32_t v;
            if (u == pf_id) {
                v = lane < R ? pf_row : BOA_PAD;
                PROF_ADD(8, 1);
            } else {
                v = lane < R ? ix.adj[(size_t)u * R + lane] : BOA_PAD;
            }
            PROF_ADD(10, 1);
#ifdef BOA_STAGE_PROFILE
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // row in hand, for the split below
#endif
            PROF_T(t_row);
            PROF_ADD(12, t_row - t_sel1);

            // row-gather scorers: every neighbour's attribute record and
            // vector requested now, so that the gathers overlap the visited
            // test; only the new neighbours' keys are entered (the same
            // candidates, distances and keys as scoring after the test)
            typename Scorer::RowGather rg;
            int4 aw0 = make_int4(0, 0, 0, 0), aw1 = make_int4(0, 0, 0, 0);
            if (spec) {
                const uint32_t vv = v != BOA_PAD ? v : ix.entry;   // padding: any valid row, unused
                if (lane < R) load_attrs(vv, aw0, aw1);
                sc.gather_row(ix.vectors, d, vv, R, lane, rg);
            }

            // ---- test-and-insert into the visited set
            const int vst = visit_test(v);
            PROF_T(t_vl);
            PROF_ADD(13, t_vl - t_row);
            const bool is_new = vst > 0;
            const uint64_t nm = __ballot(is_new);
            c = __popcll(nm);
            PROF_ADD(14, c == 0 ? 1 : 0);
            if (!spec && is_new) cid[lanes_below(nm)] = v;
            // the row of the entry expected next is requested only now: a
            // load issued before the visited test would be waited for there
            // (loads retire in order), while from here it overlaps the gathers.
            // It is requested on every path (the entry's row when nothing is
            // predicted), so that waiting for the gathers is one fixed count.
            pf_key = kn;
            {
                // (every lane loads, lanes past R from the row's last slot:
                // a load under a branch would leave the count unknown; the
                // row is masked where it is used, since a select here would
                // wait for the load at once)
                const uint32_t pid = j2 >= 0 ? key_id(kn) : ix.entry;
                pf_id = j2 >= 0 ? pid : BOA_PAD;
                pf_row = ix.adj[(size_t)pid * R + (lane < R ? lane : R - 1)];
            }
            PROF_T(t_vis1);
            PROF_ADD(1, t_vis1 - t_sel1);
            PROF_ADD(6, spill ? 1 : 0);
            if (spec) {
                // the gathered neighbours' distances, then the new ones' keys
                const uint32_t phi = count_phi(aw0, aw1);
                sc.score_row(rg, d, R, cd, lane);
                wave_sync();
                spec_key = is_new ? make_key(phi, cd[lane], v) : KEY_NONE;
                spec_c = c;
                c = 0;
                PROF_T(t_spec1);
                PROF_ADD(2, t_spec1 - t_vis1);
            }
        }

        // ---- epilogue: confidence (Eq. 3) over the phase's worklist (its
        // first L entries); the result is written by the last phase the
        // query runs in this launch
        wave_sync();
        const uint32_t n_valid = lower_bound64(beam, min(len, (uint32_t)L), KEY_PHI1);
        const int k = a.k;
        uint32_t conf = 0;
        // the result (the first valid entries) and the two distances of Eq. 3
        uint64_t res_key[2] = {KEY_NONE, KEY_NONE};   // (product-quantised search: lanes' top-k keys)
        float d_k = 0.f, d_max = 0.f;
        if constexpr (Scorer::kPQ) {
            // re-rank the valid entries by exact distance (Sec. III-B step 8):
            // keys (exact distance bits, id); the k smallest in order by k
            // rounds of a wave minimum, the largest by one wave maximum
            for (uint32_t b0 = 0; b0 < n_valid; b0 += 64) {
                const uint32_t e = b0 + lane;
                if (e < n_valid) {
                    const uint32_t id = key_id(beam[e]);
                    const float dx = exact_dist_lane(a.ix.vectors, a.queries, qi, id, d, a.vec_u8 != 0);
                    rrk[e] = ((uint64_t)__float_as_uint(dx) << 32) | id;
                }
            }
            wave_sync();
            uint64_t prev = 0, mx = 0;
            for (uint32_t i = lane; i < n_valid; i += 64) mx = max(mx, rrk[i]);
            mx = ~wave_min64(~mx);
            const int kk = min(k, (int)n_valid);
            for (int q = 0; q < kk; ++q) {
                uint64_t mn = KEY_NONE;
                for (uint32_t i = lane; i < n_valid; i += 64) {
                    const uint64_t x = rrk[i];
                    if ((q == 0 || x > prev) && x < mn) mn = x;
                }
                mn = wave_min64(mn);
                if ((q & 63) == lane) res_key[q >> 6] = mn;
                prev = mn;
            }
            if (kk > 0) d_k = __uint_as_float((uint32_t)(prev >> 32));
            d_max = __uint_as_float((uint32_t)(mx >> 32));
        } else if (n_valid > (uint32_t)k) {
            d_k = key_dist(beam[k - 1]);
            d_max = key_dist(beam[n_valid - 1]);
        }
        if (n_valid > (uint32_t)k) {
            double dk = sqrt((double)d_k);
            double dmax = sqrt((double)d_max);
            double gamma = dmax == 0.0 ? 0.0 : (dmax - dk) / dmax;
            conf = gamma <= a.eps ? 1u : 0u;
        }
        const bool last = conf != 0u || p + 1 == a.p_end;
        if (lane == 0) {
            const size_t ps = (size_t)p * a.nq + qi;
            if (a.qstat) {   // per-phase statistics (absent in the allocation-free search)
                a.qstat[ps] = (uint8_t)(1u + conf + (spill ? 4u : 0u));
                a.qE[ps] = E;
                a.qS[ps] = S;
            }
            if (a.user_E) a.user_E[qi] += E;
            if (a.user_S) a.user_S[qi] += S;
            if (a.write_conf) a.conf[t] = (uint8_t)conf;
            if (last) a.final_L[qi] = L;
        }
        if (last) {
            for (int q = lane; q < k; q += 64) {
                uint32_t id = BOA_PAD;
                float dd = __int_as_float(0x7f800000);
                if ((uint32_t)q < n_valid) {
                    if constexpr (Scorer::kPQ) {
                        const uint64_t kk = res_key[q >> 6];
                        id = (uint32_t)kk;
                        dd = __uint_as_float((uint32_t)(kk >> 32));
                    } else {
                        uint64_t kk = beam[q];
                        id = key_id(kk);
                        dd = key_dist(kk);
                    }
                }
                a.ids[(size_t)qi * k + q] = id;
                a.dists[(size_t)qi * k + q] = dd;
            }
        }
        wave_sync();
        if (last) break;
        }   // phases
    }       // queries
    if (!a.vis_bitmap && lane == 0) vs.log[0] = n_log;
#ifdef BOA_STAGE_PROFILE
    if (lane == 0 && a.prof) {
        for (int i = 0; i < BOA_PROF_SLOTS; ++i) a.prof[(size_t)slot * BOA_PROF_SLOTS + i] += prof_acc[i];
    }
#endif
}

// ---------------------------------------------------------------------------
// The escalation launch of a split search with two waves per query (a
// 128-thread block), when its visited set is the LDS bitmap over all ids.
// One wave owns the worklist: it merges each expansion's keys and selects
// the next node. The other owns the bitmap: it tests a row's neighbours,
// gathers and scores the new ones. The expansions stay one node at a time
// in the order of Alg. 2; what overlaps is the guess of the next node. After
// handing over an expansion's keys, the gather wave takes as the next node
// the smaller of its best new key and the entry that followed the expanded
// one (the selection after the merge is exactly that whenever the entry is
// known), and runs that node's visited test, gathers and scoring while the
// worklist wave merges. If the selection differs, the guessed node's bits are
// cleared again (the gather wave is the only writer of the bitmap, so the set
// returns to its state before the guess) and the selected node is expanded.
// The visited set sees the same inserts in the same order, so results and
// counts are those of the one-wave launch.
//
// Control flow that both waves share (the query loop, the phase loop, the
// end of a phase's search) is decided from values they read from LDS after
// the same block barrier, so both run the same sequence of barriers.
struct PairCtrl {
    uint64_t kn;       // the entry after the selected one (KEY_NONE: not known)
    uint32_t t;        // query slot taken by the block
    uint32_t sel;      // the selected node's id, or PAIR_DONE
    uint32_t S;        // scored nodes of the phase (gather wave)
    uint32_t last;     // the query's result has been written
    uint32_t pad[2];
};
static constexpr uint32_t PAIR_DONE = 0xFFFFFFFFu;

template <class Scorer>
__global__ void __launch_bounds__(128) pair_kernel(PhaseArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = lane_id();
    const bool merger = threadIdx.x < 64;   // wave 0: worklist; wave 1: bitmap and scoring
    const int Lb = beam_slots(a.L_alloc);
    const int pw = ((a.L_alloc >> 6) + 3) & ~1;
    uint64_t *beam = reinterpret_cast<uint64_t *>(smem);        // Lb
    uint64_t *nkey = beam + Lb;                                   // 64
    uint64_t *posbm = nkey + 64;                                  // pw
    uint64_t *kbuf = posbm + pw;                                  // 64: an expansion's keys
    uint32_t *krow = reinterpret_cast<uint32_t *>(kbuf + 64);   // 64: the row of ctl->kn
    PairCtrl *ctl = reinterpret_cast<PairCtrl *>(krow + 64);
    uint32_t *cid = reinterpret_cast<uint32_t *>(ctl + 1);      // 64
    float *cd = reinterpret_cast<float *>(cid + 64);             // 64
    unsigned char *qlds = reinterpret_cast<unsigned char *>(cd + 64);
    uint32_t *bits = reinterpret_cast<uint32_t *>(qlds + Scorer::kLdsBytes);   // vis_words

    const IndexView ix = a.ix;
    const int R = ix.R, d = ix.d, m = ix.m;
    const uint32_t n_in = bcast0(*a.n_active);
    if (n_in <= a.tau_count) return;   // (the same for both waves)
    const uint32_t nA = a.t_end < n_in ? a.t_end : n_in;

    Scorer sc;
    sc.bind_lds(qlds);
    RangeTest rt;   // the gather wave's attribute test
    // keys of the candidates cid[0, c): one per lane, KEY_NONE past c
    auto score_cands = [&](uint32_t c) -> uint64_t {
        if (c == 0) return KEY_NONE;
        wave_sync();
        const uint32_t my_id = cid[lane];
        typename Scorer::Ids ids0;
        sc.read_ids(cid, (int)c, 0, lane, ids0);
        int4 w0 = make_int4(0, 0, 0, 0), w1 = make_int4(0, 0, 0, 0);
        if (lane < (int)c) load_attr_record(ix, my_id, w0, w1);
        sc.score(ix.vectors, d, cid, (int)c, cd, lane, ids0);
        const uint32_t phi = rt.phi(w0, w1, ix.m_pad);
        wave_sync();
        return lane < (int)c ? make_key(phi, cd[lane], cid[lane]) : KEY_NONE;
    };
    // test-and-insert of a row (one neighbour per lane); the new ones go to
    // cid in lane order
    auto visit_row = [&](uint32_t v, uint64_t &nm) -> uint32_t {
        bool is_new = false;
        if (v != BOA_PAD) {
            const uint32_t bit = 1u << (v & 31u);
            is_new = (atomicOr(&bits[v >> 5], bit) & bit) == 0u;
        }
        nm = __ballot(is_new);
        if (is_new) cid[lanes_below(nm)] = v;
        return (uint32_t)__popcll(nm);
    };
    auto undo_row = [&](uint32_t v, uint64_t nm) {
        if ((nm >> lane) & 1ull) atomicAnd(&bits[v >> 5], ~(1u << (v & 31u)));
        wave_sync();
    };
    auto row_of = [&](uint32_t u) -> uint32_t { return lane < R ? ix.adj[(size_t)u * R + lane] : BOA_PAD; };
#ifdef BOA_STAGE_PROFILE
    // worklist wave: 0 merge and select, 3 wait for the guess, 5 whole
    // iteration, 10 expansions; gather wave: 1 guessed expansion, 4 wait for
    // the selection, 2 hand-over (and the expansion after a miss), 8 hits,
    // 9 misses, 14 no guess, 13 guesses of a new key; 12 (worklist wave) no
    // entry known after the selected one
    uint64_t prof_acc[BOA_PROF_SLOTS] = {};
#endif

    for (;;) {
        if (merger && lane == 0) ctl->t = atomicAdd(a.queue, 1u);
        __syncthreads();
        const uint32_t t = bcast0(ctl->t) + a.t_begin;
        if (t >= nA) break;   // (both waves)
        const uint32_t qi = bcast0(a.active[t]);
        if (!merger) {
            sc.load_query(a.queries, qi, d, lane);
            rt.set(a.ranges, qi, m, ix.f32_mask);
        }
        // every phase restarts from the entry point (Alg. 1 calls Alg. 2 afresh)
        for (int p = a.p_begin; p < a.p_end; ++p) {
            const int L = a.sched[p];
            // worklist wave
            uint32_t len = 0, E = 0;
            int expanded_j = -1;
            // gather wave: the keys of the last expansion handed over, the
            // entry known to follow the last selected node, its row in flight,
            // and the guessed expansion (row, new-neighbour mask, keys)
            uint32_t S = 0;
            uint64_t ckey = KEY_NONE, kn_prev = KEY_NONE;
            uint32_t kn_row = BOA_PAD;   // row of kn_prev (read from krow)
            bool guess = false;
            uint32_t g_id = BOA_PAD, g_v = BOA_PAD, g_c = 0;
            uint64_t g_nm = 0, g_key = KEY_NONE;
            if (merger) {
                for (int i = lane; i < Lb; i += 64) beam[i] = KEY_NONE;
            } else {
                const uint4 z = make_uint4(0u, 0u, 0u, 0u);
                uint4 *b4 = reinterpret_cast<uint4 *>(bits);
                for (uint32_t i = lane; i < (a.vis_words >> 2); i += 64) b4[i] = z;
                wave_sync();
                if (lane == 0) {
                    bits[ix.entry >> 5] |= 1u << (ix.entry & 31u);
                    cid[0] = ix.entry;
                }
                ckey = score_cands(1u);   // the entry point, scored before the first expansion
                S = 1;
                kbuf[lane] = ckey;
            }
            for (;;) {
                __syncthreads();   // kbuf holds the last expansion's keys
                PROF_T(t_b1);
                if (merger) {
                    // ---- drop, sort and merge the keys (as in phase_kernel)
                    uint64_t key = kbuf[lane];
                    uint32_t scan_from = (uint32_t)(expanded_j + 1);
                    if (len == (uint32_t)L && key >= beam[L - 1]) key = KEY_NONE;   // cannot enter
                    const uint64_t keep = __ballot(key != KEY_NONE);
                    const uint32_t kept = __popcll(keep);
                    if (kept > 0) {
                        nkey[key != KEY_NONE ? lanes_below(keep) : kept + lanes_below(~keep)] = key;
                        wave_sync();
                        uint32_t rank = 0;
                        {
                            const ulonglong2 *nk2 = reinterpret_cast<const ulonglong2 *>(nkey);
                            for (uint32_t i = 0; i < kept; i += 8) {
                                const ulonglong2 a0 = nk2[(i >> 1) + 0], a1 = nk2[(i >> 1) + 1];
                                const ulonglong2 a2 = nk2[(i >> 1) + 2], a3 = nk2[(i >> 1) + 3];
                                rank += (a0.x < key ? 1u : 0u) + (a0.y < key ? 1u : 0u);
                                rank += (a1.x < key ? 1u : 0u) + (a1.y < key ? 1u : 0u);
                                rank += (a2.x < key ? 1u : 0u) + (a2.y < key ? 1u : 0u);
                                rank += (a3.x < key ? 1u : 0u) + (a3.y < key ? 1u : 0u);
                            }
                        }
                        wave_sync();
                        if (key != KEY_NONE) nkey[rank] = key;
                        wave_sync();
                        key = lane < (int)kept ? nkey[lane] : KEY_NONE;
                        uint32_t f = 0xFFFFFFFFu, pos = 0;
                        if (lane < (int)kept) {
                            pos = lower_bound64_p2(beam, (uint32_t)beam_slots((int32_t)len), key);
                            f = pos + lane;
                        }
                        const uint32_t p0 = bcast0(pos);
                        const uint32_t newlen = min((uint32_t)L, len + kept);
                        const uint32_t w_lo = bcast0(p0 >> 6), w_hi = bcast0((newlen - 1u) >> 6);
                        for (uint32_t w = w_lo + lane; w <= w_hi; w += 64) posbm[w] = 0ull;
                        wave_sync();
                        const bool placed = f < (uint32_t)L;
                        if (placed) atomicOr(reinterpret_cast<unsigned long long *>(&posbm[f >> 6]),
                                             1ull << (f & 63u));
                        const uint32_t n_placed = __popcll(__ballot(placed));
                        wave_sync();
                        uint64_t word = posbm[w_hi];
                        uint32_t below = n_placed - (uint32_t)__popcll(word);
                        for (int w = (int)w_hi; w >= (int)w_lo; --w) {
                            const uint32_t o = ((uint32_t)w << 6) + lane;
                            const bool act = o >= p0 && o < newlen;
                            const bool isnew = (word >> lane) & 1ull;
                            const uint32_t cnt = below + (uint32_t)__popcll(word & ((1ull << lane) - 1ull));
                            uint64_t val = 0;
                            if (act) val = isnew ? nkey[cnt] : beam[o - cnt];
                            wave_sync();
                            if (act) beam[o] = val;
                            if (w > (int)w_lo) {
                                word = posbm[w - 1];
                                below -= (uint32_t)__popcll(word);
                            }
                            wave_sync();
                        }
                        len = newlen;
                        if (p0 < scan_from) scan_from = p0;
                    }
                    // ---- select the first unexpanded entry among the first L,
                    // and the one after it when the same scan sees it
                    const uint32_t lim = min(len, (uint32_t)L);
                    int j = -1, j2 = -1;
                    uint64_t ku = 0, kn = KEY_NONE;
                    for (uint32_t b0 = scan_from; b0 < lim; b0 += 64) {
                        const uint32_t i = b0 + lane;
                        const uint64_t bk = i < lim ? beam[i] : 1ull;
                        const uint64_t mk = __ballot(!(bk & 1ull));
                        if (mk) {
                            const int l1 = __ffsll((unsigned long long)mk) - 1;
                            j = (int)b0 + l1;
                            ku = readlane64(bk, l1);
                            const uint64_t rest = mk & (mk - 1ull);
                            if (rest) {
                                const int l2 = __ffsll((unsigned long long)rest) - 1;
                                j2 = (int)b0 + l2;
                                kn = readlane64(bk, l2);
                            }
                            break;
                        }
                    }
                    wave_sync();
                    if (j >= 0) {
                        expanded_j = j;
                        E += 1;
                        if (lane == 0) beam[j] = ku | 1ull;
                    }
                    if (lane == 0) {
                        ctl->sel = j >= 0 ? key_id(ku) : PAIR_DONE;
                        ctl->kn = j2 >= 0 ? kn : KEY_NONE;
                    }
                    // the row of the entry after the selected node, for the
                    // gather wave's next guess (this wave waits at the barrier
                    // for the guessed expansion anyway)
                    if (j2 >= 0) krow[lane] = lane < R ? ix.adj[(size_t)key_id(kn) * R + lane] : BOA_PAD;
                    PROF_T(t_m1);
                    PROF_ADD(0, t_m1 - t_b1);
                    PROF_ADD(10, j >= 0 ? 1 : 0);
                    PROF_ADD(12, j >= 0 && j2 < 0 ? 1 : 0);
                } else {
                    // ---- the guessed next node: visited test, gathers, keys
                    const uint64_t mk = wave_min64(ckey);
                    const uint64_t gk = mk < kn_prev ? mk : kn_prev;
                    guess = gk != KEY_NONE;
                    if (guess) {
                        g_id = key_id(gk);
                        // the entry after the last selected node: its row came
                        // from the worklist wave; a new key: its row is loaded
                        // now. (A row of the best new key requested ahead was
                        // measured slower: the compiler waits for it before the
                        // gathers of the next expansion, whichever row is used.)
                        if (bcast0(gk == kn_prev ? 1u : 0u)) {   // (uniform: a scalar branch)
                            g_v = kn_row;
                        } else {
                            g_v = row_of(g_id);
                            PROF_ADD(13, 1);
                        }
                        g_c = visit_row(g_v, g_nm);
                        g_key = score_cands(g_c);
                    }
                    PROF_T(t_g1);
                    PROF_ADD(1, t_g1 - t_b1);
                }
                PROF_T(t_pre2);
                __syncthreads();   // the selection is published
                PROF_T(t_b2);
                PROF_ADD(merger ? 3 : 4, t_b2 - t_pre2);
                const uint32_t sel = bcast0(ctl->sel);
                if (sel == PAIR_DONE) {   // converged (both waves)
                    if (!merger && guess) undo_row(g_v, g_nm);
                    break;
                }
                if (!merger) {
                    const uint64_t kn_new = ctl->kn;
                    uint32_t c;
                    PROF_ADD(guess ? (g_id == sel ? 8 : 9) : 14, 1);
                    if (guess && g_id == sel) {
                        ckey = g_key;
                        c = g_c;
                    } else {
                        if (guess) undo_row(g_v, g_nm);
                        uint64_t nm;
                        const uint32_t v = sel == key_id(kn_prev) && kn_prev != KEY_NONE ? kn_row : row_of(sel);
                        c = visit_row(v, nm);
                        ckey = score_cands(c);
                    }
                    S += c;
                    kbuf[lane] = ckey;
                    // the entry after the selected node and its row, which the
                    // worklist wave loaded
                    kn_prev = kn_new;
                    kn_row = krow[lane];
                    PROF_T(t_g2);
                    PROF_ADD(2, t_g2 - t_b2);
                }
                if (merger) {
                    PROF_T(t_m2);
                    PROF_ADD(5, t_m2 - t_b1);
                }
            }
            // ---- epilogue (worklist wave): Eq. 3 over the first L entries
            if (!merger && lane == 0) ctl->S = S;
            __syncthreads();
            if (merger) {
                const uint32_t n_valid = lower_bound64(beam, min(len, (uint32_t)L), KEY_PHI1);
                const int k = a.k;
                uint32_t conf = 0;
                if (n_valid > (uint32_t)k) {
                    const double dk = sqrt((double)key_dist(beam[k - 1]));
                    const double dmax = sqrt((double)key_dist(beam[n_valid - 1]));
                    const double gamma = dmax == 0.0 ? 0.0 : (dmax - dk) / dmax;
                    conf = gamma <= a.eps ? 1u : 0u;
                }
                const bool last = conf != 0u || p + 1 == a.p_end;
                const uint32_t Sp = bcast0(ctl->S);
                if (lane == 0) {
                    const size_t ps = (size_t)p * a.nq + qi;
                    if (a.qstat) {
                        a.qstat[ps] = (uint8_t)(1u + conf);
                        a.qE[ps] = E;
                        a.qS[ps] = Sp;
                    }
                    if (a.user_E) a.user_E[qi] += E;
                    if (a.user_S) a.user_S[qi] += Sp;
                    if (a.write_conf) a.conf[t] = (uint8_t)conf;
                    if (last) a.final_L[qi] = L;
                    ctl->last = last ? 1u : 0u;
                }
                if (last) {
                    for (int q = lane; q < k; q += 64) {
                        uint32_t id = BOA_PAD;
                        float dd = __int_as_float(0x7f800000);
                        if ((uint32_t)q < n_valid) {
                            id = key_id(beam[q]);
                            dd = key_dist(beam[q]);
                        }
                        a.ids[(size_t)qi * k + q] = id;
                        a.dists[(size_t)qi * k + q] = dd;
                    }
                }
            }
            __syncthreads();
            if (bcast0(ctl->last)) break;   // (both waves)
        }   // phases
    }       // queries
#ifdef BOA_STAGE_PROFILE
    if (lane == 0 && a.prof) {
        static constexpr int mine_m[] = {0, 3, 5, 10, 12};
        static constexpr int mine_g[] = {1, 2, 4, 8, 9, 13, 14};
        if (merger)
            for (int i : mine_m) a.prof[(size_t)blockIdx.x * BOA_PROF_SLOTS + i] += prof_acc[i];
        else
            for (int i : mine_g) a.prof[(size_t)blockIdx.x * BOA_PROF_SLOTS + i] += prof_acc[i];
    }
#endif
}

// Stable compaction of the active list (Alg. 1: survivors escalate). One
// block: flags -> ballot prefix within waves -> wave totals in LDS.
__global__ void __launch_bounds__(1024) compact_kernel(CompactArgs a)
{
    __shared__ uint32_t wsum[16];
    __shared__ uint32_t base_s;
    const uint32_t n_in = *a.n_in;
    const bool stopped = n_in <= a.tau_count;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    if (threadIdx.x == 0) base_s = 0;
    __syncthreads();
    for (uint32_t b0 = 0; !stopped && b0 < n_in; b0 += blockDim.x) {
        uint32_t t = b0 + threadIdx.x;
        bool keep = t < n_in && a.conf[t] == 0;
        uint64_t mk = __ballot(keep);
        if (lane == 0) wsum[w] = __popcll(mk);
        __syncthreads();
        uint32_t off = base_s;
        for (int i = 0; i < w; ++i) off += wsum[i];
        if (keep) a.out[off + lanes_below(mk)] = a.in[t];
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t tot = 0;
            for (int i = 0; i < nw; ++i) tot += wsum[i];
            base_s += tot;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) *a.n_out = stopped ? 0u : base_s;
}

// BOA+ survivor pooling: append the non-confident entries of one phase-0
// sub-batch (a slice of the active list) to a pool, stably, after the
// pool's current entries; then publish the new count. One block.
__global__ void __launch_bounds__(1024) append_kernel(AppendArgs a)
{
    __shared__ uint32_t wsum[16];
    __shared__ uint32_t base_s;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    if (threadIdx.x == 0) base_s = *a.pool_count;
    __syncthreads();
    for (uint32_t b0 = 0; b0 < a.n; b0 += blockDim.x) {
        uint32_t t = b0 + threadIdx.x;
        bool keep = t < a.n && a.conf[t] == 0;
        uint64_t mk = __ballot(keep);
        if (lane == 0) wsum[w] = __popcll(mk);
        __syncthreads();
        uint32_t off = base_s;
        for (int i = 0; i < w; ++i) off += wsum[i];
        if (keep) a.pool[off + lanes_below(mk)] = a.in[t];
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t tot = 0;
            for (int i = 0; i < nw; ++i) tot += wsum[i];
            base_s += tot;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) *a.pool_count = base_s;
}

__global__ void init_kernel(InitArgs a)
{
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < (size_t)a.nq) {
        a.active0[i] = (uint32_t)i;
        if (a.user_E) a.user_E[i] = 0;
        if (a.user_S) a.user_S[i] = 0;
    }
    if (a.qstat && i < (size_t)a.nq * a.n_phases) a.qstat[i] = 0;
    if (i < (size_t)a.n_counters) a.counters[i] = 0;
    if (i < a.reset_slots) a.bits[i * a.slot_words + a.bits_words] = BOA_LOG_DIRTY;
    if (i == 0) {
        a.n_active[0] = (uint32_t)a.nq;
        // later phases' counts and the BOA+ pool counts
        for (int p = 1; p < 2 * (BOA_MAX_PHASES + 1); ++p) a.n_active[p] = 0;
        *a.status = 0;
    }
}

// ---------------------------------------------------------------------------
// launch helpers (host)

template <class Scorer>
static hipError_t launch_phase_t(const PhaseArgs &a, int blocks, hipStream_t st)
{
    size_t lds = (size_t)a.lds_per_wave * a.waves_per_block;
    hipLaunchKernelGGL(phase_kernel<Scorer>, dim3(blocks), dim3(64 * a.waves_per_block), lds, st, a);
    return hipGetLastError();
}

template <class Scorer>
static int occupancy_t(int wpb, size_t lds)
{
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, phase_kernel<Scorer>, 64 * wpb, lds) != hipSuccess)
        return 0;
    return nb;
}

#define BOA_DISPATCH_W(VEC, DIM, W, CALL)                                    \
    do {                                                                     \
        if ((VEC) == BOA_VEC_F32) {                                          \
            int T_ = ((DIM) + 63) / 64;                                      \
            if (T_ <= 1) { using S_ = F32Scorer<1, W>; CALL; }               \
            else if (T_ <= 2) { using S_ = F32Scorer<2, W>; CALL; }          \
            else if (T_ <= 3) { using S_ = F32Scorer<3, W>; CALL; }          \
            else if (T_ <= 4) { using S_ = F32Scorer<4, W>; CALL; }          \
            else if (T_ <= 6) { using S_ = F32Scorer<6, W>; CALL; }          \
            else if (T_ <= 8) { using S_ = F32Scorer<8, W>; CALL; }          \
            else if (T_ <= 12) { using S_ = F32Scorer<12, W>; CALL; }        \
            else { using S_ = F32Scorer<16, W>; CALL; }                      \
        } else {                                                             \
            int G_ = (DIM) / 16;                                             \
            if (G_ <= 1) { using S_ = U8Scorer<1, W>; CALL; }                \
            else if (G_ <= 2) { using S_ = U8Scorer<2, W>; CALL; }           \
            else if (G_ <= 4) { using S_ = U8Scorer<4, W>; CALL; }           \
            else if (G_ <= 8) { using S_ = U8Scorer<8, W>; CALL; }           \
            else if (G_ <= 16) { using S_ = U8Scorer<16, W>; CALL; }         \
            else if (G_ <= 32) { using S_ = U8Scorer<32, W>; CALL; }         \
            else { using S_ = U8Scorer<64, W>; CALL; }                       \
        }                                                                    \
    } while (0)

#define BOA_DISPATCH_PQ(PQM, CALL)                                           \
    do {                                                                     \
        int T_ = ((PQM) + 15) / 16;                                          \
        if (T_ <= 1) { using S_ = PQScorer<1>; CALL; }                       \
        else if (T_ <= 2) { using S_ = PQScorer<2>; CALL; }                  \
        else if (T_ <= 4) { using S_ = PQScorer<4>; CALL; }                  \
        else if (T_ <= 8) { using S_ = PQScorer<8>; CALL; }                  \
        else if (T_ <= 12) { using S_ = PQScorer<12>; CALL; }                \
        else { using S_ = PQScorer<16>; CALL; }                              \
    } while (0)

// product-quantised searches (PQM > 0) take the PQ scorer, which has no
// wide variant; the others the exact scorer of the vector type
#define BOA_DISPATCH(VEC, DIM, WIDE, CALL, PQM)                              \
    do {                                                                     \
        if ((PQM) > 0) BOA_DISPATCH_PQ(PQM, CALL);                           \
        else if (WIDE) BOA_DISPATCH_W(VEC, DIM, 2, CALL);                    \
        else BOA_DISPATCH_W(VEC, DIM, 1, CALL);                              \
    } while (0)

template <class Scorer>
static hipError_t launch_pair_t(const PhaseArgs &a, int blocks, hipStream_t st)
{
    hipLaunchKernelGGL(pair_kernel<Scorer>, dim3(blocks), dim3(128), (size_t)a.lds_per_wave, st, a);
    return hipGetLastError();
}

template <class Scorer>
static int pair_occupancy_t(size_t lds)
{
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, pair_kernel<Scorer>, 128, lds) != hipSuccess) return 0;
    return nb;
}

// the two-wave escalation launch (wide scorers; lds_per_wave is the block's LDS)
hipError_t launch_pair(const PhaseArgs &a, int vec_dtype, int blocks, hipStream_t st)
{
    hipError_t e = hipSuccess;
    BOA_DISPATCH_W(vec_dtype, a.ix.d, 2, e = launch_pair_t<S_>(a, blocks, st));
    return e;
}

int pair_occupancy(int vec_dtype, int d, size_t lds)
{
    int r = 0;
    BOA_DISPATCH_W(vec_dtype, d, 2, r = pair_occupancy_t<S_>(lds));
    return r;
}

size_t pair_lds_bytes(int32_t L, uint32_t vis_words, int scorer_lds)
{
    const int32_t Lb = beam_slots(L), pw = ((L >> 6) + 3) & ~1;
    return (size_t)8 * Lb + 8 * 64 + 8 * (size_t)pw + 8 * 64 + 4 * 64 + sizeof(PairCtrl) + 4 * 64 + 4 * 64 +
           (size_t)scorer_lds + 4 * (size_t)vis_words;
}

hipError_t launch_phase(const PhaseArgs &a, int vec_dtype, int blocks, hipStream_t st, bool wide)
{
    hipError_t e = hipSuccess;
    BOA_DISPATCH(vec_dtype, a.ix.d, wide, e = launch_phase_t<S_>(a, blocks, st), a.pq ? a.pq_m : 0);
    return e;
}

template <class Scorer>
static int scorer_lds_t()
{
    return Scorer::kLdsBytes;
}

int scorer_lds_bytes(int vec_dtype, int d, bool wide, int pq_m)
{
    int r = 0;
    BOA_DISPATCH(vec_dtype, d, wide, r = scorer_lds_t<S_>(), pq_m);
    return r;
}

int phase_occupancy(int vec_dtype, int d, int wpb, size_t lds, bool wide, int pq_m)
{
    int r = 0;
    BOA_DISPATCH(vec_dtype, d, wide, r = occupancy_t<S_>(wpb, lds), pq_m);
    return r;
}

hipError_t launch_compact(const CompactArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(append_kernel, dim3(1), dim3(1024), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_init(const InitArgs &a, hipStream_t st)
{
    size_t n = (size_t)a.nq * (a.n_phases > 1 ? a.n_phases : 1);
    if ((size_t)a.n_counters > n) n = a.n_counters;
    if (a.reset_slots > n) n = (size_t)a.reset_slots;
    if (n == 0) n = 1;
    unsigned blocks = (unsigned)((n + 255) / 256);
    hipLaunchKernelGGL(init_kernel, dim3(blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace boa
