// Index construction on the GPU: the entry point s (the medoid) and, when
// the caller passes no adjacency, the proximity graph itself.
//
// The paper builds a Vamana graph with JAG threshold pruning (Sec. II
// "Graph construction") and enters every search at the medoid s (Alg. 2).
// This library's builder follows the same pruning rule on a different
// candidate source: exact nearest neighbours instead of Vamana's
// incremental beam-search insertion.
//   1. medoid: the point nearest (float64) to the float64 centroid, ties to
//      the lowest id; the centroid is reduced in one fixed order;
//   2. candidates: the K = min(2R, 128, n - 1) nearest points of every
//      point by brute force, ordered by (distance, id);
//   3. alpha-pruning (DiskANN's dominance rule, alpha = 1.2 on Euclidean
//      distances): a candidate v of u is dropped when a kept w has
//      alpha^2 d(w, v) <= d(u, v) on squared distances;
//   4. reverse edges: every kept edge u -> v proposes v -> u; each point's
//      forward and reverse neighbours are pruned again by the same rule to
//      R - 1 edges, leaving one free slot per row;
//   5. connectivity repair from s (host): a point that a breadth-first
//      search from s does not reach gets an in-edge from its nearest
//      reached candidate that still has a free slot.
// Distances here are this builder's own: float32 sums of squared float32
// differences in dimension order, exact int32 for uint8 vectors.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <queue>
#include <thread>
#include <vector>

#include "boa_internal.h"

namespace boa {

static constexpr uint64_t BKEY_NONE = ~0ull;
static constexpr int KNN_ROWS_W = 8;      // rows per wave in the kNN scan
static constexpr int KNN_WAVES = 4;       // waves per block
static constexpr int KNN_ROWS_B = KNN_ROWS_W * KNN_WAVES;
static constexpr int KNN_LIST = 128;      // top-K capacity per row
static constexpr int KNN_BUF = 64;        // new-candidate buffer per row
static constexpr int KNN_KC = 64;         // dimensions per staged column chunk

__device__ __forceinline__ uint64_t bkey(float d, uint32_t id)
{
    return ((uint64_t)__float_as_uint(d) << 32) | id;
}

// ---------------------------------------------------------------------------
// pair distances (builder's own arithmetic)

// squared distance of two float32 rows, dimensions in order
__device__ __forceinline__ float pair_dist_f32(const float *x, const float *y, int d)
{
    const float4 *a = reinterpret_cast<const float4 *>(x);
    const float4 *b = reinterpret_cast<const float4 *>(y);
    float acc = 0.f;
    for (int c = 0; c < (d >> 2); ++c) {
        const float4 p = a[c], q = b[c];
        float t = p.x - q.x;
        acc = __builtin_fmaf(t, t, acc);
        t = p.y - q.y;
        acc = __builtin_fmaf(t, t, acc);
        t = p.z - q.z;
        acc = __builtin_fmaf(t, t, acc);
        t = p.w - q.w;
        acc = __builtin_fmaf(t, t, acc);
    }
    return acc;
}

// exact squared distance of two uint8 rows: |x|^2 + |y|^2 - 2 x.y in int32
__device__ __forceinline__ float pair_dist_u8(const uint8_t *x, const uint8_t *y, int d, uint32_t nx, uint32_t ny)
{
    const uint32_t *a = reinterpret_cast<const uint32_t *>(x);
    const uint32_t *b = reinterpret_cast<const uint32_t *>(y);
    uint32_t dot = 0;
    for (int c = 0; c < (d >> 2); ++c) dot = __builtin_amdgcn_udot4(a[c], b[c], dot, false);
    return (float)(int32_t)(nx + ny - 2u * dot);
}

struct BuildView {
    const void *vectors;
    const uint32_t *norms;   // uint8 vectors: |x|^2 per point (else null)
    int64_t n;
    int32_t d;
    int32_t u8;
};

__device__ __forceinline__ float dist_ids(const BuildView &v, uint32_t a, uint32_t b)
{
    if (v.u8) {
        const uint8_t *X = reinterpret_cast<const uint8_t *>(v.vectors);
        return pair_dist_u8(X + (size_t)a * v.d, X + (size_t)b * v.d, v.d, v.norms[a], v.norms[b]);
    }
    const float *X = reinterpret_cast<const float *>(v.vectors);
    return pair_dist_f32(X + (size_t)a * v.d, X + (size_t)b * v.d, v.d);
}

// ---------------------------------------------------------------------------
// in-wave bitonic sort of 256 u64 keys held in LDS (ascending)

__device__ __forceinline__ void wave_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ void bitonic256(uint64_t *a, int lane)
{
    for (int k = 2; k <= 256; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            // 128 compare-exchanges per step, two per lane
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int t = lane + 64 * h;                       // pair index 0..127
                const int i = ((t / j) * 2 * j) + (t % j);         // lower element
                const int p = i + j;
                const bool up = (i & k) == 0;
                const uint64_t x = a[i], y = a[p];
                if ((x > y) == up) {
                    a[i] = y;
                    a[p] = x;
                }
            }
            wave_fence();
        }
    }
}

// ---------------------------------------------------------------------------
// 1. medoid

struct CentroidArgs {
    BuildView v;
    double *partial;     // nblocks x d
    int64_t per_block;
};

// each block sums its contiguous range of points, dimension by dimension,
// in point order (float64)
__global__ void __launch_bounds__(256) centroid_partial_kernel(CentroidArgs a)
{
    const int64_t p0 = (int64_t)blockIdx.x * a.per_block;
    const int64_t p1 = p0 + a.per_block < a.v.n ? p0 + a.per_block : a.v.n;
    for (int j = threadIdx.x; j < a.v.d; j += blockDim.x) {
        double s = 0.0;
        if (a.v.u8) {
            const uint8_t *X = reinterpret_cast<const uint8_t *>(a.v.vectors);
            for (int64_t i = p0; i < p1; ++i) s += (double)X[(size_t)i * a.v.d + j];
        } else {
            const float *X = reinterpret_cast<const float *>(a.v.vectors);
            for (int64_t i = p0; i < p1; ++i) s += (double)X[(size_t)i * a.v.d + j];
        }
        a.partial[(size_t)blockIdx.x * a.v.d + j] = s;
    }
}

struct MedoidArgs {
    BuildView v;
    const double *centroid;  // d
    double *best_d;          // per block
    uint32_t *best_id;       // per block
};

// float64 distance of every point to the centroid; each block reports its
// nearest point (ties: lowest id)
__global__ void __launch_bounds__(256) medoid_partial_kernel(MedoidArgs a)
{
    __shared__ double sd[256];
    __shared__ uint32_t si[256];
    double bd = INFINITY;
    uint32_t bi = 0xFFFFFFFFu;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.v.n;
         i += (int64_t)gridDim.x * blockDim.x) {
        double s = 0.0;
        for (int j = 0; j < a.v.d; ++j) {
            const double x = a.v.u8 ? (double)reinterpret_cast<const uint8_t *>(a.v.vectors)[(size_t)i * a.v.d + j]
                                    : (double)reinterpret_cast<const float *>(a.v.vectors)[(size_t)i * a.v.d + j];
            const double t = x - a.centroid[j];
            s = fma(t, t, s);
        }
        if (s < bd || (s == bd && (uint32_t)i < bi)) {
            bd = s;
            bi = (uint32_t)i;
        }
    }
    sd[threadIdx.x] = bd;
    si[threadIdx.x] = bi;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) {
            const double od = sd[threadIdx.x + w];
            const uint32_t oi = si[threadIdx.x + w];
            if (od < sd[threadIdx.x] || (od == sd[threadIdx.x] && oi < si[threadIdx.x])) {
                sd[threadIdx.x] = od;
                si[threadIdx.x] = oi;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        a.best_d[blockIdx.x] = sd[0];
        a.best_id[blockIdx.x] = si[0];
    }
}

__global__ void norms_kernel(BuildView v, uint32_t *norms)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= v.n) return;
    const uint32_t *x = reinterpret_cast<const uint32_t *>(reinterpret_cast<const uint8_t *>(v.vectors) + (size_t)i * v.d);
    uint32_t s = 0;
    for (int c = 0; c < (v.d >> 2); ++c) s = __builtin_amdgcn_udot4(x[c], x[c], s, false);
    norms[i] = s;
}

// ---------------------------------------------------------------------------
// 2. exact K nearest candidates of every point
//
// A block of 4 waves owns 32 rows (8 per wave) and streams every column
// tile of 64 points through LDS, dimension-major in chunks of 64 dims (lane
// j reads column j, conflict-free). Each lane accumulates its column's
// distance to the wave's 8 rows (row values are wave-uniform). Each row
// keeps its K best (distance, id) keys in LDS plus a buffer of new keys
// below its current K-th; a full buffer is merged by a bitonic sort.

struct KnnArgs {
    BuildView v;
    int32_t K;
    uint32_t *cand;    // n x K ids (0xFFFFFFFF padded)
    float *cand_d;     // n x K squared distances
    // attribute-threshold pass: only points within a row's threshold count
    const int32_t *ranks;   // n x m quantile ranks (null: no filter)
    const int32_t *thr;     // n thresholds in rank units
    int32_t m;
};

// attribute distance of two points: the largest gap between their ranks
// over the columns
__device__ __forceinline__ int32_t rank_gap(const int32_t *ranks, int m, int64_t a, int64_t b)
{
    int32_t g = 0;
    for (int j = 0; j < m; ++j) {
        const int32_t t = ranks[a * m + j] - ranks[b * m + j];
        g = max(g, t < 0 ? -t : t);
    }
    return g;
}

template <bool U8>
__global__ void __launch_bounds__(256) knn_kernel(KnnArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int d = a.v.d, K = a.K;
    const int64_t n = a.v.n;
    // LDS: per wave 8 rows x (list 128 + buffer 64) keys and a 256-key sort
    // scratch; then the staged column chunk (64 columns x 64 dims) and row
    // chunk (32 rows x 64 dims), both in 4-dimension units
    constexpr int PER_WAVE = KNN_ROWS_W * (KNN_LIST + KNN_BUF) + 256;
    uint64_t *lists = reinterpret_cast<uint64_t *>(smem) + (size_t)wid * PER_WAVE;
    uint64_t *scratch = lists + KNN_ROWS_W * (KNN_LIST + KNN_BUF);
    unsigned char *colbase = smem + (size_t)KNN_WAVES * PER_WAVE * 8;
    constexpr int UNIT = U8 ? 4 : 16;   // bytes per 4-dimension unit
    unsigned char *rowbase = colbase + (size_t)(KNN_KC / 4) * 64 * UNIT;

    const int64_t blk_row0 = (int64_t)blockIdx.x * KNN_ROWS_B;
    const int64_t row0 = blk_row0 + wid * KNN_ROWS_W;
    for (int i = lane; i < KNN_ROWS_W * (KNN_LIST + KNN_BUF); i += 64) lists[i] = BKEY_NONE;
    uint64_t thr[KNN_ROWS_W];
    uint32_t bufn[KNN_ROWS_W], listn[KNN_ROWS_W], rnorm[KNN_ROWS_W];
#pragma unroll
    for (int r = 0; r < KNN_ROWS_W; ++r) {
        thr[r] = BKEY_NONE;
        bufn[r] = 0;
        listn[r] = 0;
        const int64_t row = row0 + r;
        rnorm[r] = (U8 && row < n) ? a.v.norms[row] : 0u;
    }
    wave_fence();

    // merge row r's buffer into its list: both copied into the scratch,
    // sorted, the K best written back
    auto merge_row = [&](int r) {
        uint64_t *L = lists + r * (KNN_LIST + KNN_BUF);
        uint64_t *B = L + KNN_LIST;
        for (int i = lane; i < 256; i += 64) {
            uint64_t x = BKEY_NONE;
            if (i < KNN_LIST) x = L[i];
            else if (i < KNN_LIST + KNN_BUF) x = B[i - KNN_LIST];
            scratch[i] = x;
        }
        wave_fence();
        bitonic256(scratch, lane);
        for (int i = lane; i < KNN_LIST + KNN_BUF; i += 64) {
            if (i < KNN_LIST) L[i] = i < K ? scratch[i] : BKEY_NONE;
            else B[i - KNN_LIST] = BKEY_NONE;
        }
        wave_fence();
        const uint32_t tot = min(listn[r] + bufn[r], (uint32_t)K);
        listn[r] = tot;
        bufn[r] = 0;
        thr[r] = tot == (uint32_t)K ? L[K - 1] : BKEY_NONE;
    };

    const int nchunk = (d + KNN_KC - 1) / KNN_KC;
    for (int64_t c0 = 0; c0 < n; c0 += 64) {
        const int64_t col = c0 + lane;
        const bool colv = col < n;
        float accf[KNN_ROWS_W];
        uint32_t acci[KNN_ROWS_W];
#pragma unroll
        for (int r = 0; r < KNN_ROWS_W; ++r) {
            accf[r] = 0.f;
            acci[r] = 0u;
        }
        for (int ch = 0; ch < nchunk; ++ch) {
            const int k0 = ch * KNN_KC;
            const int nu = min(KNN_KC, d - k0) >> 2;   // 4-dimension units in this chunk
            __syncthreads();   // the previous chunk is consumed
            // unit u of column j at colT[u * 64 + j]; of row r at rowT[r * 16 + u]
            for (int e = threadIdx.x; e < nu * 64; e += 256) {
                const int u = e >> 6, j = e & 63;
                const int64_t cj = c0 + j;
                if (U8) {
                    const uint8_t *X = reinterpret_cast<const uint8_t *>(a.v.vectors);
                    reinterpret_cast<uint32_t *>(colbase)[e] =
                        cj < n ? reinterpret_cast<const uint32_t *>(X + (size_t)cj * d + k0)[u] : 0u;
                } else {
                    const float *X = reinterpret_cast<const float *>(a.v.vectors);
                    reinterpret_cast<float4 *>(colbase)[e] =
                        cj < n ? reinterpret_cast<const float4 *>(X + (size_t)cj * d + k0)[u]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
            for (int e = threadIdx.x; e < KNN_ROWS_B * 16; e += 256) {
                const int r = e >> 4, u = e & 15;
                const int64_t rr = blk_row0 + r;
                if (u >= nu) continue;
                if (U8) {
                    const uint8_t *X = reinterpret_cast<const uint8_t *>(a.v.vectors);
                    reinterpret_cast<uint32_t *>(rowbase)[e] =
                        rr < n ? reinterpret_cast<const uint32_t *>(X + (size_t)rr * d + k0)[u] : 0u;
                } else {
                    const float *X = reinterpret_cast<const float *>(a.v.vectors);
                    reinterpret_cast<float4 *>(rowbase)[e] =
                        rr < n ? reinterpret_cast<const float4 *>(X + (size_t)rr * d + k0)[u]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
            __syncthreads();
            if (U8) {
                const uint32_t *colT = reinterpret_cast<const uint32_t *>(colbase);
                const uint32_t *rowT = reinterpret_cast<const uint32_t *>(rowbase) + wid * KNN_ROWS_W * 16;
                for (int u = 0; u < nu; ++u) {
                    const uint32_t cv = colT[u * 64 + lane];
#pragma unroll
                    for (int r = 0; r < KNN_ROWS_W; ++r)
                        acci[r] = __builtin_amdgcn_udot4(cv, rowT[r * 16 + u], acci[r], false);
                }
            } else {
                const float4 *colT = reinterpret_cast<const float4 *>(colbase);
                const float4 *rowT = reinterpret_cast<const float4 *>(rowbase) + wid * KNN_ROWS_W * 16;
                for (int u = 0; u < nu; ++u) {
                    const float4 cv = colT[u * 64 + lane];
#pragma unroll
                    for (int r = 0; r < KNN_ROWS_W; ++r) {
                        const float4 rv = rowT[r * 16 + u];   // the same address in every lane
                        float t = cv.x - rv.x;
                        accf[r] = __builtin_fmaf(t, t, accf[r]);
                        t = cv.y - rv.y;
                        accf[r] = __builtin_fmaf(t, t, accf[r]);
                        t = cv.z - rv.z;
                        accf[r] = __builtin_fmaf(t, t, accf[r]);
                        t = cv.w - rv.w;
                        accf[r] = __builtin_fmaf(t, t, accf[r]);
                    }
                }
            }
        }
        const uint32_t cnorm = (U8 && colv) ? a.v.norms[col] : 0u;
        // candidates below each row's K-th key go to its buffer
#pragma unroll
        for (int r = 0; r < KNN_ROWS_W; ++r) {
            const int64_t row = row0 + r;
            if (row >= n) continue;   // uniform
            const float dd = U8 ? (float)(int32_t)(rnorm[r] + cnorm - 2u * acci[r]) : accf[r];
            bool within = colv && col != row;
            if (a.ranks && within) within = rank_gap(a.ranks, a.m, row, col) <= a.thr[row];
            const uint64_t key = within ? bkey(dd, (uint32_t)col) : BKEY_NONE;
            const uint64_t m = __ballot(key < thr[r]);
            if (m) {
                if (bufn[r] + (uint32_t)__popcll(m) > (uint32_t)KNN_BUF) merge_row(r);
                // re-test against the threshold the merge may have tightened
                const bool pass = key < thr[r];
                const uint64_t m2 = __ballot(pass);
                if (m2) {
                    uint64_t *B = lists + r * (KNN_LIST + KNN_BUF) + KNN_LIST;
                    const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m2 >> 32),
                                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m2, 0u));
                    if (pass) B[bufn[r] + below] = key;
                    bufn[r] += (uint32_t)__popcll(m2);
                    wave_fence();
                }
            }
        }
    }
    // final merges and output
#pragma unroll
    for (int r = 0; r < KNN_ROWS_W; ++r) {
        const int64_t row = row0 + r;
        if (row >= n) continue;
        if (bufn[r] > 0) merge_row(r);
        const uint64_t *L = lists + r * (KNN_LIST + KNN_BUF);
        for (int i = lane; i < K; i += 64) {
            const uint64_t x = L[i];
            a.cand[(size_t)row * K + i] = x == BKEY_NONE ? BOA_PAD : (uint32_t)x;
            a.cand_d[(size_t)row * K + i] =
                x == BKEY_NONE ? __int_as_float(0x7f800000) : __uint_as_float((uint32_t)(x >> 32));
        }
    }
}

// ---------------------------------------------------------------------------
// 3./4. alpha-pruning of a sorted candidate list, one wave per point

struct PruneArgs {
    BuildView v;
    // source lists: forward prune reads the kNN lists (n x K); the re-prune
    // reads, per point, its forward row (n x R) and its reverse neighbours
    // (CSR rev_off / rev)
    const uint32_t *cand;
    int32_t K;
    const uint32_t *fwd;
    const uint32_t *rev_off;
    const uint32_t *rev;
    int32_t R;
    int32_t budget;
    float alpha2;      // the pruning slack alpha, squared (squared distances)
    uint32_t *out;     // n x R (0xFFFFFFFF padded)
};

// Prune the keys sorted in `keys[0, cnt)` (cnt <= 256) for point u into out
// (at most `budget` ids), by the alpha-dominance rule. Lanes test each
// candidate against all kept points at once.
__device__ void alpha_prune(const BuildView &v, uint32_t u, const uint64_t *keys, int cnt, int budget,
                            float alpha2, uint32_t *kept, uint32_t *out_row, int R, int lane)
{
    int nk = 0;
    for (int c = 0; c < cnt && nk < budget; ++c) {
        const uint64_t key = keys[c];
        if (key == BKEY_NONE) break;
        const uint32_t cv = (uint32_t)key;
        const float duv = __uint_as_float((uint32_t)(key >> 32));
        bool dom = false;
        for (int j0 = 0; j0 < nk; j0 += 64) {
            const int j = j0 + lane;
            bool hit = false;
            if (j < nk) hit = alpha2 * dist_ids(v, kept[j], cv) <= duv;
            if (__ballot(hit)) {
                dom = true;
                break;
            }
        }
        if (!dom) {
            if (lane == 0) kept[nk] = cv;
            ++nk;
            wave_fence();
        }
    }
    for (int i = lane; i < R; i += 64) out_row[i] = i < nk ? kept[i] : BOA_PAD;
    (void)u;
}

__global__ void __launch_bounds__(256) prune_fwd_kernel(PruneArgs a)
{
    __shared__ uint64_t keys_s[4][256];
    __shared__ uint32_t kept_s[4][128];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int64_t u = (int64_t)blockIdx.x * 4 + wid;
    if (u >= a.v.n) return;
    uint64_t *keys = keys_s[wid];
    // the candidates in (distance, id) order, with this pass's own distance
    for (int i = lane; i < 256; i += 64) {
        uint64_t k = BKEY_NONE;
        if (i < a.K) {
            const uint32_t c = a.cand[(size_t)u * a.K + i];
            if (c != BOA_PAD) k = bkey(dist_ids(a.v, (uint32_t)u, c), c);
        }
        keys[i] = k;
    }
    wave_fence();
    bitonic256(keys, lane);
    alpha_prune(a.v, (uint32_t)u, keys, min(a.K, 256), a.budget, a.alpha2, kept_s[wid], a.out + (size_t)u * a.R,
                a.R, lane);
}

// Re-prune each point's forward row together with its reverse neighbours
// (the nearest 256 - R of them when there are more) to `budget` edges.
__global__ void __launch_bounds__(256) prune_union_kernel(PruneArgs a)
{
    __shared__ uint64_t keys_s[4][256];
    __shared__ uint64_t buf_s[4][256];
    __shared__ uint32_t kept_s[4][128];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int64_t u = (int64_t)blockIdx.x * 4 + wid;
    if (u >= a.v.n) return;
    uint64_t *keys = keys_s[wid];
    uint64_t *buf = buf_s[wid];
    const uint32_t *frow = a.fwd + (size_t)u * a.R;
    for (int i = lane; i < 256; i += 64) {
        uint64_t k = BKEY_NONE;
        if (i < a.R) {
            const uint32_t c = frow[i];
            if (c != BOA_PAD) k = bkey(dist_ids(a.v, (uint32_t)u, c), c);
        }
        keys[i] = k;
    }
    wave_fence();
    bitonic256(keys, lane);
    // reverse neighbours not already forward ones, merged 128 at a time
    // into the 256 best (a row holds at most R <= 64 forward ids)
    const uint32_t r0 = a.rev_off[u], r1 = a.rev_off[u + 1];
    for (uint32_t b0 = r0; b0 < r1; b0 += 128) {
        for (int h = 0; h < 4; ++h) {
            const int i = lane + 64 * h;
            uint64_t k = BKEY_NONE;
            if (i < 128) {
                const uint32_t t = b0 + (uint32_t)i;
                if (t < r1) {
                    const uint32_t c = a.rev[t];
                    bool dup = false;
                    for (int q = 0; q < a.R; ++q) dup |= frow[q] == c;
                    if (!dup) k = bkey(dist_ids(a.v, (uint32_t)u, c), c);
                }
            } else {
                k = keys[i];   // the current upper half
            }
            buf[i] = k;
        }
        wave_fence();
        // the 256 best of keys[0,256) and the new 128: the first 128 of the
        // sorted keys stay; sort (keys[128..256) + new 128) and keep the best
        // 128 of those as the upper half
        bitonic256(buf, lane);
        for (int i = lane; i < 128; i += 64) keys[128 + i] = buf[i];
        wave_fence();
        bitonic256(keys, lane);
    }
    alpha_prune(a.v, (uint32_t)u, keys, 256, a.budget, a.alpha2, kept_s[wid], a.out + (size_t)u * a.R, a.R, lane);
}

__global__ void count_in_kernel(const uint32_t *adj, int64_t n, int R, uint32_t *indeg)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * R) return;
    const uint32_t v = adj[i];
    if (v != BOA_PAD) atomicAdd(&indeg[v], 1u);
}

__global__ void scatter_rev_kernel(const uint32_t *adj, int64_t n, int R, const uint32_t *off, uint32_t *cursor,
                                   uint32_t *rev)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * R) return;
    const uint32_t v = adj[i];
    if (v == BOA_PAD) return;
    const uint32_t pos = atomicAdd(&cursor[v], 1u);
    rev[off[v] + pos] = (uint32_t)(i / R);
}

// ---------------------------------------------------------------------------
// host side

namespace {

struct DevBuf {
    void *p = nullptr;
    ~DevBuf()
    {
        if (p) (void)hipFree(p);
    }
    hipError_t alloc(size_t bytes) { return hipMalloc(&p, bytes ? bytes : 1); }
    template <class T>
    T *as() const { return reinterpret_cast<T *>(p); }
};

#define BTRY(expr)                                  \
    do {                                            \
        hipError_t e_ = (expr);                     \
        if (e_ != hipSuccess) {                     \
            (void)hipGetLastError();                \
            return e_;                              \
        }                                           \
    } while (0)

}  // namespace

hipError_t compute_medoid(const void *d_vectors, int64_t n, int32_t d, int vec_dtype, uint32_t *entry)
{
    BuildView v{d_vectors, nullptr, n, d, vec_dtype == BOA_VEC_U8 ? 1 : 0};
    const int nb = (int)std::min<int64_t>(512, n);
    const int64_t per = (n + nb - 1) / nb;
    DevBuf part, cen, bd, bi;
    BTRY(part.alloc((size_t)nb * d * 8));
    BTRY(cen.alloc((size_t)d * 8));
    CentroidArgs ca{v, part.as<double>(), per};
    hipLaunchKernelGGL(centroid_partial_kernel, dim3(nb), dim3(256), 0, 0, ca);
    BTRY(hipGetLastError());
    // the partial sums added in block order on the host (float64)
    std::vector<double> hp((size_t)nb * d), c((size_t)d, 0.0);
    BTRY(hipMemcpy(hp.data(), part.p, hp.size() * 8, hipMemcpyDeviceToHost));
    for (int b = 0; b < nb; ++b)
        for (int j = 0; j < d; ++j) c[j] += hp[(size_t)b * d + j];
    for (int j = 0; j < d; ++j) c[j] /= (double)n;
    BTRY(hipMemcpy(cen.p, c.data(), (size_t)d * 8, hipMemcpyHostToDevice));
    const int mb = 1024;
    BTRY(bd.alloc((size_t)mb * 8));
    BTRY(bi.alloc((size_t)mb * 4));
    MedoidArgs ma{v, cen.as<double>(), bd.as<double>(), bi.as<uint32_t>()};
    hipLaunchKernelGGL(medoid_partial_kernel, dim3(mb), dim3(256), 0, 0, ma);
    BTRY(hipGetLastError());
    std::vector<double> hd(mb);
    std::vector<uint32_t> hi(mb);
    BTRY(hipMemcpy(hd.data(), bd.p, (size_t)mb * 8, hipMemcpyDeviceToHost));
    BTRY(hipMemcpy(hi.data(), bi.p, (size_t)mb * 4, hipMemcpyDeviceToHost));
    double best = INFINITY;
    uint32_t id = 0xFFFFFFFFu;
    for (int b = 0; b < mb; ++b)
        if (hd[b] < best || (hd[b] == best && hi[b] < id)) {
            best = hd[b];
            id = hi[b];
        }
    *entry = id;
    return hipSuccess;
}

size_t knn_lds_bytes(int vec_dtype)
{
    const size_t lists = (size_t)KNN_WAVES * (KNN_ROWS_W * (KNN_LIST + KNN_BUF) + 256) * 8;
    const size_t unit = vec_dtype == BOA_VEC_U8 ? 4 : 16;
    return lists + (size_t)(KNN_KC / 4) * 64 * unit + (size_t)KNN_ROWS_B * (KNN_KC / 4) * unit;
}

namespace {

// Quantile rank of every attribute cell within its column: the number of
// strictly smaller values (equal values share a rank); float32 columns
// compare as floats.
std::vector<int32_t> column_ranks(const int32_t *attrs, int64_t n, int m, uint32_t f32_mask)
{
    std::vector<int32_t> rk((size_t)n * m);
    std::vector<int64_t> ord((size_t)n);
    for (int j = 0; j < m; ++j) {
        const bool f = (f32_mask >> j) & 1u;
        auto val = [&](int64_t i) -> double {
            const int32_t c = attrs[(size_t)i * m + j];
            if (!f) return (double)c;
            float x;
            std::memcpy(&x, &c, 4);
            return (double)x;
        };
        for (int64_t i = 0; i < n; ++i) ord[i] = i;
        std::sort(ord.begin(), ord.end(), [&](int64_t a, int64_t b) { return val(a) < val(b); });
        int64_t r = 0;
        for (int64_t t = 0; t < n; ++t) {
            if (t > 0 && val(ord[t]) != val(ord[t - 1])) r = t;
            rk[(size_t)ord[t] * m + j] = (int32_t)r;
        }
    }
    return rk;
}

// Per point and level: the q-quantile of its attribute distance to an
// evenly spaced sample of S points (ids floor(i n / S)).
std::vector<int32_t> level_thresholds(const std::vector<int32_t> &rk, int64_t n, int m, const double *q, int levels)
{
    const int64_t S = std::min<int64_t>(4096, n);
    std::vector<int64_t> smp((size_t)S);
    for (int64_t i = 0; i < S; ++i) smp[i] = (i * n) / S;
    std::vector<int32_t> thr((size_t)levels * n);
    auto work = [&](int64_t u0, int64_t u1) {
        std::vector<int32_t> g((size_t)S);
        for (int64_t u = u0; u < u1; ++u) {
            for (int64_t i = 0; i < S; ++i) {
                int32_t x = 0;
                for (int j = 0; j < m; ++j) {
                    const int32_t t = rk[(size_t)u * m + j] - rk[(size_t)smp[i] * m + j];
                    x = std::max(x, t < 0 ? -t : t);
                }
                g[i] = x;
            }
            for (int l = 0; l < levels; ++l) {
                const int64_t idx = std::max<int64_t>(0, (int64_t)std::ceil(q[l] * (double)S) - 1);
                std::nth_element(g.begin(), g.begin() + idx, g.end());
                thr[(size_t)l * n + u] = g[idx];
            }
        }
    };
    const int nt = (int)std::max<unsigned>(1u, std::min<unsigned>(16u, std::thread::hardware_concurrency()));
    std::vector<std::thread> th;
    for (int t = 0; t < nt; ++t) th.emplace_back(work, n * t / nt, n * (t + 1) / nt);
    for (auto &x : th) x.join();
    return thr;
}

hipError_t knn_launch(const KnnArgs &ka, int vec_dtype, int64_t n)
{
    const size_t lds = knn_lds_bytes(vec_dtype);
    const unsigned blocks = (unsigned)((n + KNN_ROWS_B - 1) / KNN_ROWS_B);
    if (vec_dtype == BOA_VEC_U8) {
        BTRY(hipFuncSetAttribute(reinterpret_cast<const void *>(knn_kernel<true>),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        hipLaunchKernelGGL(knn_kernel<true>, dim3(blocks), dim3(256), lds, 0, ka);
    } else {
        BTRY(hipFuncSetAttribute(reinterpret_cast<const void *>(knn_kernel<false>),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        hipLaunchKernelGGL(knn_kernel<false>, dim3(blocks), dim3(256), lds, 0, ka);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t build_graph(const void *d_vectors, int64_t n, int32_t d, int vec_dtype, int32_t R, uint32_t entry,
                       const int32_t *h_attrs, int32_t m, uint32_t f32_mask, float alpha, int32_t attr_levels,
                       uint32_t *d_adj, BuildStats *stats)
{
    const bool u8 = vec_dtype == BOA_VEC_U8;
    const float alpha2 = alpha * alpha;
    // budgets: each attribute level R/8 edges, the vector pass the rest but
    // one (the free slot the connectivity repair may take)
    static const double kLevelQ[4] = {0.001, 0.01, 0.05, 0.2};
    const int levels = (h_attrs && m > 0 && R >= 8) ? std::min(attr_levels, 4) : 0;
    const int b_lvl = std::max(1, R / 8);
    const int budget = std::max(1, R - 1 - levels * b_lvl);
    const int K = (int)std::min<int64_t>(std::min(2 * R, KNN_LIST), n - 1);
    DevBuf norms;
    BuildView v{d_vectors, nullptr, n, d, u8 ? 1 : 0};
    if (u8) {
        BTRY(norms.alloc((size_t)n * 4));
        hipLaunchKernelGGL(norms_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, 0, v, norms.as<uint32_t>());
        BTRY(hipGetLastError());
        v.norms = norms.as<uint32_t>();
    }
    if (K < 1) {   // a single point: no edges
        BTRY(hipMemset(d_adj, 0xFF, (size_t)n * R * 4));
        return hipSuccess;
    }
    // 2. candidates by vector distance
    DevBuf cand, cand_d;
    BTRY(cand.alloc((size_t)n * K * 4));
    BTRY(cand_d.alloc((size_t)n * K * 4));
    {
        KnnArgs ka{v, K, cand.as<uint32_t>(), cand_d.as<float>(), nullptr, nullptr, 0};
        BTRY(knn_launch(ka, vec_dtype, n));
    }
    // 3. forward prune
    DevBuf fwd;
    BTRY(fwd.alloc((size_t)n * R * 4));
    {
        PruneArgs pa{};
        pa.v = v;
        pa.cand = cand.as<uint32_t>();
        pa.K = K;
        pa.R = R;
        pa.budget = budget;
        pa.alpha2 = alpha2;
        pa.out = fwd.as<uint32_t>();
        hipLaunchKernelGGL(prune_fwd_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, 0, pa);
        BTRY(hipGetLastError());
    }
    // 4. reverse edges (CSR), then the union re-pruned
    DevBuf indeg, off, cursor, rev;
    BTRY(indeg.alloc((size_t)n * 4));
    BTRY(hipMemset(indeg.p, 0, (size_t)n * 4));
    const unsigned eb = (unsigned)((n * R + 255) / 256);
    hipLaunchKernelGGL(count_in_kernel, dim3(eb), dim3(256), 0, 0, fwd.as<uint32_t>(), n, R, indeg.as<uint32_t>());
    BTRY(hipGetLastError());
    std::vector<uint32_t> h_in((size_t)n), h_off((size_t)n + 1);
    BTRY(hipMemcpy(h_in.data(), indeg.p, (size_t)n * 4, hipMemcpyDeviceToHost));
    h_off[0] = 0;
    for (int64_t i = 0; i < n; ++i) h_off[i + 1] = h_off[i] + h_in[i];
    BTRY(off.alloc(((size_t)n + 1) * 4));
    BTRY(cursor.alloc((size_t)n * 4));
    BTRY(rev.alloc((size_t)h_off[n] * 4));
    BTRY(hipMemcpy(off.p, h_off.data(), ((size_t)n + 1) * 4, hipMemcpyHostToDevice));
    BTRY(hipMemset(cursor.p, 0, (size_t)n * 4));
    hipLaunchKernelGGL(scatter_rev_kernel, dim3(eb), dim3(256), 0, 0, fwd.as<uint32_t>(), n, R, off.as<uint32_t>(),
                       cursor.as<uint32_t>(), rev.as<uint32_t>());
    BTRY(hipGetLastError());
    {
        PruneArgs pa{};
        pa.v = v;
        pa.fwd = fwd.as<uint32_t>();
        pa.rev_off = off.as<uint32_t>();
        pa.rev = rev.as<uint32_t>();
        pa.R = R;
        pa.budget = budget;
        pa.alpha2 = alpha2;
        pa.out = d_adj;
        hipLaunchKernelGGL(prune_union_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, 0, pa);
        BTRY(hipGetLastError());
    }
    std::vector<uint32_t> adj((size_t)n * R), hc((size_t)n * K);
    BTRY(hipMemcpy(adj.data(), d_adj, adj.size() * 4, hipMemcpyDeviceToHost));
    BTRY(hipMemcpy(hc.data(), cand.p, hc.size() * 4, hipMemcpyDeviceToHost));
    // 5. attribute-aware edges (JAG threshold pruning, Sec. II "Graph
    // construction"): per level, the alpha-pruned nearest vectors among the
    // points within the point's attribute threshold (where the capped
    // attribute distance is zero), b_lvl edges each, appended to the row
    int64_t attr_edges = 0;
    if (levels > 0) {
        const std::vector<int32_t> rk = column_ranks(h_attrs, n, m, f32_mask);
        const std::vector<int32_t> thr = level_thresholds(rk, n, m, kLevelQ, levels);
        const int Kl = (int)std::min<int64_t>(std::min(4 * b_lvl, KNN_LIST), n - 1);
        DevBuf d_rk, d_thr, lc, lcd, lrow;
        BTRY(d_rk.alloc(rk.size() * 4));
        BTRY(d_thr.alloc((size_t)n * 4));
        BTRY(lc.alloc((size_t)n * Kl * 4));
        BTRY(lcd.alloc((size_t)n * Kl * 4));
        BTRY(lrow.alloc((size_t)n * R * 4));
        BTRY(hipMemcpy(d_rk.p, rk.data(), rk.size() * 4, hipMemcpyHostToDevice));
        std::vector<uint32_t> hl((size_t)n * R);
        for (int l = 0; l < levels; ++l) {
            BTRY(hipMemcpy(d_thr.p, thr.data() + (size_t)l * n, (size_t)n * 4, hipMemcpyHostToDevice));
            KnnArgs ka{v, Kl, lc.as<uint32_t>(), lcd.as<float>(), d_rk.as<int32_t>(), d_thr.as<int32_t>(), m};
            BTRY(knn_launch(ka, vec_dtype, n));
            PruneArgs pa{};
            pa.v = v;
            pa.cand = lc.as<uint32_t>();
            pa.K = Kl;
            pa.R = R;
            pa.budget = b_lvl;
            pa.alpha2 = alpha2;
            pa.out = lrow.as<uint32_t>();
            hipLaunchKernelGGL(prune_fwd_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, 0, pa);
            BTRY(hipGetLastError());
            BTRY(hipMemcpy(hl.data(), lrow.p, hl.size() * 4, hipMemcpyDeviceToHost));
            for (int64_t u = 0; u < n; ++u) {
                uint32_t *row = &adj[(size_t)u * R];
                int cnt = 0;
                while (cnt < R && row[cnt] != BOA_PAD) ++cnt;
                for (int i = 0; i < b_lvl && cnt < R - 1; ++i) {
                    const uint32_t x = hl[(size_t)u * R + i];
                    if (x == BOA_PAD) break;
                    bool dup = false;
                    for (int t = 0; t < cnt; ++t) dup |= row[t] == x;
                    if (!dup) {
                        row[cnt++] = x;
                        ++attr_edges;
                    }
                }
            }
        }
    }
    // 6. connectivity repair from s (host): breadth-first search, then each
    // unreached point (ascending id) gets an in-edge from its nearest
    // reached kNN candidate with a free slot; the search then continues
    // from it
    std::vector<uint8_t> seen((size_t)n, 0);
    std::vector<uint32_t> queue;
    queue.reserve((size_t)n);
    auto bfs_from = [&](uint32_t s) {
        size_t h = queue.size();
        seen[s] = 1;
        queue.push_back(s);
        while (h < queue.size()) {
            const uint32_t x = queue[h++];
            for (int r = 0; r < R; ++r) {
                const uint32_t y = adj[(size_t)x * R + r];
                if (y != BOA_PAD && !seen[y]) {
                    seen[y] = 1;
                    queue.push_back(y);
                }
            }
        }
    };
    bfs_from(entry);
    int64_t repaired = 0, fallback = 0;
    auto free_slot = [&](uint32_t w) -> int {
        for (int r = 0; r < R; ++r)
            if (adj[(size_t)w * R + r] == BOA_PAD) return r;
        return -1;
    };
    for (int64_t u = 0; u < n; ++u) {
        if (seen[u]) continue;
        int64_t w = -1;
        for (int c = 0; c < K; ++c) {   // candidates are nearest first
            const uint32_t x = hc[(size_t)u * K + c];
            if (x != BOA_PAD && seen[x] && free_slot(x) >= 0) {
                w = x;
                break;
            }
        }
        if (w < 0) {
            // no reached candidate with room: the first reached point (in
            // search order) with a free slot (every row keeps one)
            for (size_t q = 0; q < queue.size() && w < 0; ++q)
                if (free_slot(queue[q]) >= 0) w = queue[q];
            ++fallback;
        }
        if (w < 0) return hipErrorUnknown;   // cannot happen: s itself has a free slot
        adj[(size_t)w * R + free_slot((uint32_t)w)] = (uint32_t)u;
        ++repaired;
        bfs_from((uint32_t)u);
    }
    BTRY(hipMemcpy(d_adj, adj.data(), adj.size() * 4, hipMemcpyHostToDevice));
    if (stats) {
        stats->K = K;
        stats->repaired = repaired;
        stats->repair_fallback = fallback;
        stats->attr_edges = attr_edges;
        int64_t edges = 0;
        for (uint32_t x : adj) edges += x != BOA_PAD;
        stats->edges = edges;
    }
    return hipSuccess;
}

}  // namespace boa
