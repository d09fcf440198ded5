// Device side of the BOA filtered beam search for gfx950 (CDNA4).
//
// One 64-lane wavefront runs one query at a time: a persistent grid of
// waves pulls query slots from a per-launch atomic counter. Per expansion
// (Alg. 2, one node per iteration):
//   1. select the first not-yet-expanded worklist entry (ballot scan);
//   2. gather its adjacency row, one neighbour per lane (one coalesced load);
//   3. test-and-insert every neighbour into the query's visited set: an
//      open-addressing table in LDS that spills into a per-wave table in
//      HBM once its load passes one half;
//   4. for the unseen neighbours: gather the attribute cells and count the
//      violated range predicates (phi, Eq. 2), gather the vector and compute
//      the squared L2 distance with a 16-lane (float32) or G-lane (uint8)
//      group per candidate and a butterfly reduction;
//   5. pack (phi, distance, id) into one 64-bit key, drop keys that cannot
//      enter the worklist, bitonic-sort the rest across the wave and merge
//      them into the sorted worklist held in LDS (binary-search ranks,
//      suffix shifted backwards in 64-entry chunks).
// The epilogue writes the first k filter-valid entries, the phase width,
// and the Eq. 3 confidence flag.
//
// Worklist key (unsigned 64-bit, compared as an integer):
//   bits 63..60 phi (violations, <= 8), bits 59..28 float32 bits of the
//   squared distance (non-negative floats order like their bit patterns),
//   bits 27..4 point id (< 2^24), bit 0 expanded flag. Distinct ids make
//   distinct keys, so the flag bits never decide an order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "boa_internal.h"

namespace boa {

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

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t hash32(uint32_t v) { return v * 0x9E3779B1u; }

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
// number of entries of a[0, n) that are <= x (a sorted ascending)
__device__ __forceinline__ uint32_t upper_bound32(const uint32_t *a, uint32_t n, uint32_t x)
{
    uint32_t lo = 0, hi = n;
    while (lo < hi) {
        uint32_t mid = (lo + hi) >> 1;
        if (a[mid] <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m)
{
    uint32_t lo = __shfl_xor((uint32_t)v, m);
    uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

// Ascending bitonic sort of one 64-bit key per lane across the wave.
__device__ __forceinline__ uint64_t wave_sort64(uint64_t key, int lane)
{
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            uint64_t o = shfl_xor64(key, j);
            bool up = (lane & k) == 0;
            bool lower = (lane & j) == 0;
            uint64_t mn = key < o ? key : o;
            uint64_t mx = key < o ? o : key;
            key = (lower == up) ? mn : mx;
        }
    }
    return key;
}

// ---------------------------------------------------------------------------
// Distance policies. Each lane group computes one candidate's distance per
// round; rounds are unrolled by RU so that RU rows of loads are in flight.

template <int T>
struct F32Scorer {
    // lane p = lane & 15 accumulates float4 chunks p, p+16, p+32, ...
    static constexpr int kGroup = 16;
    float4 q[T];

    __device__ __forceinline__ void load_query(const void *Q, uint32_t qi, int d, int lane)
    {
        const float4 *qq = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(Q) + (size_t)qi * d);
        int p = lane & 15, nch = d >> 2;
#pragma unroll
        for (int t = 0; t < T; ++t) {
            int cc = p + 16 * t;
            q[t] = cc < nch ? qq[cc] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }

    __device__ __forceinline__ void score(const void *V, int d, const uint32_t *cid, int c, float *cd, int lane)
    {
        constexpr int RU = T <= 2 ? 4 : (T <= 4 ? 2 : 1);
        const float *vec = reinterpret_cast<const float *>(V);
        const int g = lane >> 4, p = lane & 15, nch = d >> 2;
        for (int r0 = 0; r0 < c; r0 += 4 * RU) {
            float4 x[RU][T];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                int cj = r0 + 4 * u + g;
                uint32_t id = cj < c ? cid[cj] : 0u;
                const float4 *row = reinterpret_cast<const float4 *>(vec + (size_t)id * d);
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    int cc = p + 16 * t;
                    float4 val = q[t];
                    if (cj < c && cc < nch) val = row[cc];
                    x[u][t] = val;
                }
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                float acc = 0.0f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    float a0 = x[u][t].x - q[t].x;
                    acc = __builtin_fmaf(a0, a0, acc);
                    float a1 = x[u][t].y - q[t].y;
                    acc = __builtin_fmaf(a1, a1, acc);
                    float a2 = x[u][t].z - q[t].z;
                    acc = __builtin_fmaf(a2, a2, acc);
                    float a3 = x[u][t].w - q[t].w;
                    acc = __builtin_fmaf(a3, a3, acc);
                }
                // pairwise tree over the 16 partials: p += p+8, p+4, p+2, p+1
                acc = acc + __shfl_xor(acc, 8);
                acc = acc + __shfl_xor(acc, 4);
                acc = acc + __shfl_xor(acc, 2);
                acc = acc + __shfl_xor(acc, 1);
                int cj = r0 + 4 * u + g;
                if (p == 0 && cj < c) cd[cj] = acc;
            }
        }
    }
};

template <int G>
struct U8Scorer {
    // lane p = lane % G holds the query's 16-byte chunk p (p < d/16); the
    // exact int32 sum is order-free.
    static constexpr int kGroup = G;
    uint4 q;

    __device__ __forceinline__ void load_query(const void *Q, uint32_t qi, int d, int lane)
    {
        const uint8_t *qq = reinterpret_cast<const uint8_t *>(Q) + (size_t)qi * d;
        int p = lane % G;
        q = p < (d >> 4) ? reinterpret_cast<const uint4 *>(qq)[p] : make_uint4(0, 0, 0, 0);
    }

    static __device__ __forceinline__ int32_t sq4(uint32_t a, uint32_t b)
    {
        int32_t s = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int32_t da = (int32_t)((a >> (8 * i)) & 0xFF) - (int32_t)((b >> (8 * i)) & 0xFF);
            s += da * da;
        }
        return s;
    }

    __device__ __forceinline__ void score(const void *V, int d, const uint32_t *cid, int c, float *cd, int lane)
    {
        constexpr int PER = 64 / G;            // candidates per round
        constexpr int RU = G <= 8 ? 2 : 4;
        const uint8_t *vec = reinterpret_cast<const uint8_t *>(V);
        const int g = lane / G, p = lane % G, nch = d >> 4;
        for (int r0 = 0; r0 < c; r0 += PER * RU) {
            uint4 x[RU];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                int cj = r0 + PER * u + g;
                uint32_t id = cj < c ? cid[cj] : 0u;
                uint4 val = q;
                if (cj < c && p < nch) val = reinterpret_cast<const uint4 *>(vec + (size_t)id * d)[p];
                x[u] = val;
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                int32_t acc = sq4(x[u].x, q.x) + sq4(x[u].y, q.y) + sq4(x[u].z, q.z) + sq4(x[u].w, q.w);
#pragma unroll
                for (int s = G >> 1; s > 0; s >>= 1) acc += __shfl_xor(acc, s);
                int cj = r0 + PER * u + g;
                if (p == 0 && cj < c) cd[cj] = (float)acc;
            }
        }
    }
};

// ---------------------------------------------------------------------------
// Visited set. LDS table: 0 = empty, else id + 1. Global table (per wave
// slot, in HBM): entry = epoch << 24 | id; entries of another epoch are
// free. A wave bumps its epoch for every query that used the table and
// clears the table when the 8-bit epoch wraps.

struct Visited {
    uint32_t *lds;
    uint32_t lmask, lshift;
    uint32_t *gt;
    uint32_t gmask, gshift;
    uint32_t epoch;
    uint32_t *status;
};

// true if v was not in the set (and is now)
__device__ __forceinline__ bool visit_lds(const Visited &s, uint32_t v)
{
    uint32_t key = v + 1u;
    uint32_t h = hash32(v) >> s.lshift;
    for (uint32_t probe = 0; probe <= s.lmask; ++probe) {
        uint32_t cur = s.lds[h];
        if (cur == key) return false;
        if (cur == 0u) {
            uint32_t old = atomicCAS(&s.lds[h], 0u, key);
            if (old == 0u) return true;
            if (old == key) return false;
        }
        h = (h + 1u) & s.lmask;
    }
    atomicOr(s.status, BOA_STATUS_OVERFLOW);
    return false;
}

__device__ __forceinline__ bool in_lds(const Visited &s, uint32_t v)
{
    uint32_t key = v + 1u;
    uint32_t h = hash32(v) >> s.lshift;
    for (uint32_t probe = 0; probe <= s.lmask; ++probe) {
        uint32_t cur = s.lds[h];
        if (cur == key) return true;
        if (cur == 0u) return false;
        h = (h + 1u) & s.lmask;
    }
    return false;
}

__device__ __forceinline__ bool visit_global(const Visited &s, uint32_t v)
{
    uint32_t tag = (s.epoch << 24) | v;
    uint32_t h = (hash32(v) >> s.gshift);
    uint32_t probe = 0;
    uint32_t cur = s.gt[h];
    while (probe <= s.gmask) {
        if (cur == tag) return false;
        if ((cur >> 24) != s.epoch) {
            uint32_t old = atomicCAS(&s.gt[h], cur, tag);
            if (old == cur) return true;
            if (old == tag) return false;
            cur = old;          // slot changed under us: look at it again
            continue;
        }
        h = (h + 1u) & s.gmask;
        ++probe;
        cur = s.gt[h];
    }
    atomicOr(s.status, BOA_STATUS_OVERFLOW);
    return false;
}

// ---------------------------------------------------------------------------

template <class Scorer>
__global__ void __launch_bounds__(256) phase_kernel(PhaseArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = lane_id();
    const int wid = threadIdx.x >> 6;
    const uint32_t slot = a.slot_base + blockIdx.x * a.waves_per_block + wid;

    const int L = a.L;
    unsigned char *mine = smem + (size_t)wid * a.lds_per_wave;
    uint64_t *beam = reinterpret_cast<uint64_t *>(mine);
    uint64_t *nkey = beam + L;                                   // 64
    uint32_t *npos = reinterpret_cast<uint32_t *>(nkey + 64);    // 64
    uint32_t *cid = npos + 64;                                   // 64
    float *cd = reinterpret_cast<float *>(cid + 64);             // 64
    uint32_t *htab = reinterpret_cast<uint32_t *>(cd + 64);      // H

    const IndexView ix = a.ix;
    const int R = ix.R, d = ix.d, m = ix.m;

    uint32_t nA = bcast0(*a.n_active);
    if (a.t_end < nA) nA = a.t_end;
    if (*a.n_active <= a.tau_count) return;   // the loop of Alg. 1 has stopped

    Visited vs;
    vs.lds = htab;
    vs.lmask = (1u << a.h_log2) - 1u;
    vs.lshift = 32u - a.h_log2;
    vs.gt = a.gtab + (size_t)slot * (1ull << a.g_log2);
    vs.gmask = (1u << a.g_log2) - 1u;
    vs.gshift = 32u - a.g_log2;
    vs.epoch = bcast0(a.epochs[slot]);
    if (vs.epoch == 0u || vs.epoch > 255u) vs.epoch = 1u;   // epoch 0 marks a zeroed table
    vs.status = a.status;
    const uint32_t spill_at = (1u << a.h_log2) >> 1;

    Scorer sc;
    for (;;) {
        uint32_t t = 0;
        if (lane == 0) t = atomicAdd(a.queue, 1u);
        t = bcast0(t) + a.t_begin;
        if (t >= nA) break;
        const uint32_t qi = bcast0(a.active[t]);

        sc.load_query(a.queries, qi, d, lane);
        int32_t lo[BOA_MAX_M], hi[BOA_MAX_M];
#pragma unroll
        for (int j = 0; j < BOA_MAX_M; ++j) {
            lo[j] = j < m ? a.ranges[((size_t)qi * m + j) * 2 + 0] : 0;
            hi[j] = j < m ? a.ranges[((size_t)qi * m + j) * 2 + 1] : 0;
        }
        for (uint32_t i = lane; i < (1u << a.h_log2); i += 64) htab[i] = 0u;
        wave_sync();

        bool spill = false, used_global = false;
        uint32_t lds_count = 0;
        uint32_t E = 0, S = 0;
        uint32_t len = 0, scan_from = 0;
        int expanded_j = -1;

        // the entry point is scored and entered before the first expansion
        uint32_t c = 0;
        {
            uint32_t s = ix.entry;
            if (lane == 0) {
                visit_lds(vs, s);
                cid[0] = s;
            }
            lds_count = 1;
            c = 1;
        }

        for (;;) {
            // ---- score the c new candidates listed in cid[0, c)
            if (c > 0) {
                wave_sync();
                S += c;
                uint32_t phi = 0;
                if (lane < (int)c) {
                    const int32_t *ar = ix.attrs + (size_t)cid[lane] * ix.m_pad;
                    int4 w0 = make_int4(0, 0, 0, 0), w1 = make_int4(0, 0, 0, 0);
                    if (ix.m_pad >= 4) {
                        w0 = reinterpret_cast<const int4 *>(ar)[0];
                        if (ix.m_pad == 8) w1 = reinterpret_cast<const int4 *>(ar)[1];
                    } else if (ix.m_pad == 2) {
                        int2 t2 = reinterpret_cast<const int2 *>(ar)[0];
                        w0.x = t2.x;
                        w0.y = t2.y;
                    } else {
                        w0.x = ar[0];
                    }
                    const int32_t av[BOA_MAX_M] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
                    for (int j = 0; j < BOA_MAX_M; ++j) {
                        if (j < m) {
                            bool ok;
                            if ((ix.f32_mask >> j) & 1u) {
                                float x = __int_as_float(av[j]);
                                ok = (__int_as_float(lo[j]) <= x) && (x <= __int_as_float(hi[j]));
                            } else {
                                ok = (lo[j] <= av[j]) && (av[j] <= hi[j]);
                            }
                            phi += ok ? 0u : 1u;
                        }
                    }
                }
                sc.score(a.ix.vectors, d, cid, (int)c, cd, lane);
                wave_sync();

                uint64_t key = KEY_NONE;
                if (lane < (int)c) key = make_key(phi, cd[lane], cid[lane]);
                if (len == (uint32_t)L) {
                    uint64_t kth = beam[L - 1];
                    if (key >= kth) key = KEY_NONE;   // cannot enter the worklist
                }
                uint64_t keep = __ballot(key != KEY_NONE);
                uint32_t kept = __popcll(keep);
                uint32_t next_scan = expanded_j + 1;
                if (kept > 0) {
                    key = wave_sort64(key, lane);
                    uint32_t pos = 0;
                    if (lane < (int)kept) {
                        pos = lower_bound64(beam, len, key);
                        nkey[lane] = key;
                        npos[lane] = pos;
                    }
                    wave_sync();
                    const uint32_t p0 = npos[0];
                    // shift the suffix [p0, len) right; last chunk first
                    if (len > p0) {
                        int b = (int)(((len - 1) >> 6) << 6);
                        int bmin = (int)((p0 >> 6) << 6);
                        for (; b >= bmin; b -= 64) {
                            uint32_t i = (uint32_t)b + lane;
                            uint64_t val = 0;
                            uint32_t dst = 0xFFFFFFFFu;
                            if (i >= p0 && i < len) {
                                val = beam[i];
                                dst = i + upper_bound32(npos, kept, i);
                            }
                            wave_sync();
                            if (dst < (uint32_t)L) beam[dst] = val;
                            wave_sync();
                        }
                    }
                    if (lane < (int)kept) {
                        uint32_t dst = pos + lane;
                        if (dst < (uint32_t)L) beam[dst] = key;
                    }
                    len = min((uint32_t)L, len + kept);
                    if (p0 < next_scan) next_scan = p0;
                    wave_sync();
                }
                scan_from = next_scan;
            } else {
                scan_from = expanded_j + 1;
            }

            // ---- select the nearest unexpanded entry
            int j = -1;
            for (uint32_t b = scan_from; b < len; b += 64) {
                uint32_t i = b + lane;
                bool un = (i < len) && !(beam[i] & 1ull);
                uint64_t mk = __ballot(un);
                if (mk) {
                    j = (int)(b + __ffsll((unsigned long long)mk) - 1);
                    break;
                }
            }
            if (j < 0) break;   // converged: every entry expanded
            expanded_j = j;
            const uint64_t ku = beam[j];
            wave_sync();
            if (lane == 0) beam[j] = ku | 1ull;
            const uint32_t u = key_id(ku);
            E += 1;

            // ---- gather the adjacency row and test-and-insert into the visited set
            uint32_t v = lane < R ? ix.adj[(size_t)u * R + lane] : BOA_PAD;
            if (!spill && lds_count + (uint32_t)R > spill_at) {
                spill = true;
                used_global = true;
            }
            bool is_new = false;
            if (v != BOA_PAD) {
                if (!spill) is_new = visit_lds(vs, v);
                else is_new = !in_lds(vs, v) && visit_global(vs, v);
            }
            uint64_t nm = __ballot(is_new);
            c = __popcll(nm);
            if (!spill) lds_count += c;
            if (is_new) cid[lanes_below(nm)] = v;
        }

        // ---- epilogue: result, phase width, confidence (Eq. 3)
        wave_sync();
        const uint32_t n_valid = lower_bound64(beam, len, KEY_PHI1);
        const int k = a.k;
        for (int q = lane; q < k; q += 64) {
            uint32_t id = BOA_PAD;
            float dd = __int_as_float(0x7f800000);
            if ((uint32_t)q < n_valid) {
                uint64_t kk = beam[q];
                id = key_id(kk);
                dd = key_dist(kk);
            }
            a.ids[(size_t)qi * k + q] = id;
            a.dists[(size_t)qi * k + q] = dd;
        }
        if (lane == 0) {
            a.final_L[qi] = L;
            uint32_t conf = 0;
            if (n_valid > (uint32_t)k) {
                double dk = sqrt((double)key_dist(beam[k - 1]));
                double dmax = sqrt((double)key_dist(beam[n_valid - 1]));
                double gamma = dmax == 0.0 ? 0.0 : (dmax - dk) / dmax;
                conf = gamma <= a.eps ? 1u : 0u;
            }
            a.conf[t] = (uint8_t)conf;
            a.qstat[qi] = (uint8_t)(1u + conf + (used_global ? 4u : 0u));
            a.qE[qi] = E;
            a.qS[qi] = S;
            if (a.user_E) a.user_E[qi] += E;
            if (a.user_S) a.user_S[qi] += S;
        }
        if (used_global) {
            vs.epoch += 1u;
            if (vs.epoch == 256u) {   // wrap: clear this wave's table
                uint4 z = make_uint4(0, 0, 0, 0);
                uint4 *g4 = reinterpret_cast<uint4 *>(vs.gt);
                for (uint32_t i = lane; i < ((vs.gmask + 1u) >> 2); i += 64) g4[i] = z;
                vs.epoch = 1u;
            }
        }
        wave_sync();
    }
    if (lane == 0) a.epochs[slot] = vs.epoch;
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

__global__ void init_kernel(InitArgs a)
{
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < (size_t)a.nq) {
        a.active0[i] = (uint32_t)i;
        if (a.user_E) a.user_E[i] = 0;
        if (a.user_S) a.user_S[i] = 0;
    }
    if (i < (size_t)a.nq * a.n_phases) a.qstat[i] = 0;
    if (i < (size_t)a.n_counters) a.counters[i] = 0;
    if (i == 0) {
        a.n_active[0] = (uint32_t)a.nq;
        for (int p = 1; p <= a.n_phases; ++p) a.n_active[p] = 0;
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

#define BOA_DISPATCH(VEC, DIM, CALL)                                         \
    do {                                                                     \
        if ((VEC) == BOA_VEC_F32) {                                          \
            int T_ = ((DIM) + 63) / 64;                                      \
            if (T_ <= 1) { using S_ = F32Scorer<1>; CALL; }                  \
            else if (T_ <= 2) { using S_ = F32Scorer<2>; CALL; }             \
            else if (T_ <= 3) { using S_ = F32Scorer<3>; CALL; }             \
            else if (T_ <= 4) { using S_ = F32Scorer<4>; CALL; }             \
            else if (T_ <= 6) { using S_ = F32Scorer<6>; CALL; }             \
            else if (T_ <= 8) { using S_ = F32Scorer<8>; CALL; }             \
            else if (T_ <= 12) { using S_ = F32Scorer<12>; CALL; }           \
            else { using S_ = F32Scorer<16>; CALL; }                         \
        } else {                                                             \
            int G_ = (DIM) / 16;                                             \
            if (G_ <= 1) { using S_ = U8Scorer<1>; CALL; }                   \
            else if (G_ <= 2) { using S_ = U8Scorer<2>; CALL; }              \
            else if (G_ <= 4) { using S_ = U8Scorer<4>; CALL; }              \
            else if (G_ <= 8) { using S_ = U8Scorer<8>; CALL; }              \
            else if (G_ <= 16) { using S_ = U8Scorer<16>; CALL; }            \
            else if (G_ <= 32) { using S_ = U8Scorer<32>; CALL; }            \
            else { using S_ = U8Scorer<64>; CALL; }                          \
        }                                                                    \
    } while (0)

hipError_t launch_phase(const PhaseArgs &a, int vec_dtype, int blocks, hipStream_t st)
{
    hipError_t e = hipSuccess;
    BOA_DISPATCH(vec_dtype, a.ix.d, e = launch_phase_t<S_>(a, blocks, st));
    return e;
}

int phase_occupancy(int vec_dtype, int d, int wpb, size_t lds)
{
    int r = 0;
    BOA_DISPATCH(vec_dtype, d, r = occupancy_t<S_>(wpb, lds));
    return r;
}

hipError_t launch_compact(const CompactArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_init(const InitArgs &a, hipStream_t st)
{
    size_t n = (size_t)a.nq * (a.n_phases > 1 ? a.n_phases : 1);
    if ((size_t)a.n_counters > n) n = a.n_counters;
    if (n == 0) n = 1;
    unsigned blocks = (unsigned)((n + 255) / 256);
    hipLaunchKernelGGL(init_kernel, dim3(blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace boa
