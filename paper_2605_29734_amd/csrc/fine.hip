// Fine stage of hierarchical retrieval on gfx950: candidates restricted to
// the selected clusters' child segments (Eq. local nodes), each scored by an
// inner product with the query (Eq. local policy), with temperature-softmax
// statistics and the top-k kept per (query, selected cluster).
//
// Kernels, in launch order:
//   route_fused (few pairs: one block), or route_zero / route_count /
//   route_plan / route_emit
//       group the (query, slot) pairs by selected cluster, choose the chunk
//       length that splits long segments, and number the work items
//       (cluster, chunk) and their partial results;
//   fine_stream
//       one work item per block iteration: the chunk's key rows are streamed
//       from HBM once and multiplied on MFMA against every query that selected
//       the cluster; scores feed an online (max, sum) and an LDS top-k per
//       query; one partial (m, Z, top-k keys) per (query, chunk) is written;
//   slot_merge
//       merges the chunk partials of each (query, slot) into the per-slot
//       outputs of htam_attend_transitions.
#include "dev.hpp"
#include "internal.hpp"
#include "stream.hpp"

namespace htam {

namespace {

constexpr int kPlanThreads = 1024;
constexpr int64_t kChunkFloor = 64;
constexpr size_t kRouteLdsBytes = 128 * 1024;  // per-cluster tables of the fused routing kernel
// above this many pairs, route with many blocks (one block: zipf_bf16, 2,048
// pairs, 14 us against 25; many: mixture_bf16, 16,384 pairs, 27 us against 30)
constexpr int64_t kFusedRoutePairs = 8192;
constexpr int64_t kChunkCeil = 4096;
constexpr int kMergeWaves = 4;                   // waves per merge block
constexpr int kMergeBatch = 8;                   // 64-entry groups per merge request
constexpr int kMergeDirect = 4;                  // requests a one-level merge may take
constexpr int kMergeDirectSmall = 8;             // the same where it rules out level one

// Chunk partials per level-one merge group for a cluster of nch chunks whose
// partials hold kp key slots each (k rounded up to a power of two): 0 (no
// groups) when they hold at most `direct` keys (a one-level merge: a short
// chain of prefetched requests costs less than a second merge level), else
// about sqrt(nch), so that the two merge levels read about as many keys each
// and a long cluster's merge is not a long chain of requests in one wave.
__host__ __device__ inline int64_t group_span(int64_t nch, int64_t kp, int64_t direct) {
    if (nch * kp <= direct) return 0;
    int64_t r = 2;
    while (r * r < nch) r *= 2;                   // power-of-two bracket, then refine
    int64_t lo = r / 2;
    while (lo + 1 < r) {
        const int64_t mid = (lo + r) / 2;
        if (mid * mid >= nch) r = mid; else lo = mid;
    }
    return r < 2 ? 2 : r;
}
// ceil(a / b) for 0 <= a < 2^31 and 1 <= b < 2^31, in 32-bit arithmetic
// (chunk and group counts: the plan numbers its items in 32 bits)
__host__ __device__ inline int64_t div_up32(int64_t a, int64_t b) {
    return (int64_t)(((uint32_t)a + (uint32_t)b - 1u) / (uint32_t)b);
}
__host__ __device__ inline int64_t group_count(int64_t nch, int64_t kp, int64_t direct) {
    const int64_t r = group_span(nch, kp, direct);
    return r ? div_up32(nch, r) : 0;
}

// ---------------------------------------------------------------------------
// routing
// ---------------------------------------------------------------------------
// A slice of the fp32 queries' bf16 copy (8-element groups [begin, end),
// rounded to nearest even as the LDS staging rounds them). The routing
// kernels wait mostly on memory latency on a few blocks; blocks past their
// routing grid copy a slice each, so the copy's bandwidth hides in that wait.
struct QCopy {
    const float *q;
    __bf16 *q16;
    int64_t begin, end;
};
__device__ __forceinline__ void copy_queries(const QCopy &qc, int64_t blk, int64_t nblk) {
    for (int64_t i = qc.begin + blk * blockDim.x + threadIdx.x; i < qc.end;
         i += nblk * blockDim.x)
        reinterpret_cast<bf16x8_t *>(qc.q16)[i] = load8(qc.q + i * 8);
}

// Clears the per-cluster pair counters and the plan's flags (and copies a
// slice of the queries).
__global__ void route_zero(int32_t G, int32_t *cnt, Plan *plan, QCopy qc) {
    const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = i0; i < G; i += stride) cnt[i] = 0;
    if (i0 == 0) {
        plan->next = 0;
        plan->bad_sel = 0;
        plan->bad_off = 0;
    }
    copy_queries(qc, blockIdx.x, gridDim.x);
}

// Most blocks of the planning kernel (one wave scans their totals) and of
// the counting kernel (one pair per thread up to 131,072 pairs).
constexpr int kRouteBlocks = 64;
constexpr int kCountBlocks = 128;
constexpr int kCountThreads = 1024;
constexpr int kRouteThreads = 256;

// Counts the (query, slot) pairs of each cluster; a pair's place in its
// cluster's list is the count its atomic increment returns. For the choice
// of the chunk length, each block also counts, over its pairs with a
// nonempty segment of len rows, how many have bit b of len - 1 set (b >=
// lmin; the partial results at chunk 2^j then sum exactly from these:
// ceil(len / 2^j) = 1 + sum over b >= j of bit b times 2^(b-j)), and lane 63
// how many such pairs there are: bits[block][64].
__global__ __launch_bounds__(kCountThreads) void route_count(const int32_t *sel, int64_t n, int32_t G,
                                                            const int64_t *off, int lmin,
                                                            int32_t *cnt, int32_t *pos, Plan *plan,
                                                            uint32_t *bits, int32_t n_route, QCopy qc) {
    if ((int32_t)blockIdx.x >= n_route) {
        copy_queries(qc, blockIdx.x - n_route, gridDim.x - n_route);
        return;
    }
    __shared__ uint32_t s_bits[kWave];
    const int t = threadIdx.x, lane = t & 63;
    if (t < kWave) s_bits[t] = 0;
    __syncthreads();
    uint32_t acc = 0;      // lane b: pairs with bit b of len - 1 set; lane 63: pairs with len > 0
    int32_t nbad = 0;
    for (int64_t e0 = (int64_t)blockIdx.x * kCountThreads; e0 < n;
         e0 += (int64_t)n_route * kCountThreads) {
        const int64_t e = e0 + t;
        const int32_t g = e < n ? sel[e] : 0;
        const bool valid = e < n && g >= 0 && g < G;
        uint64_t hi = 0;
        bool has = false;
        if (valid) {
            pos[e] = atomicAdd(&cnt[g], 1);
            const int64_t len = off[g + 1] - off[g];
            has = len > 0;
            hi = has ? (uint64_t)(len - 1) >> lmin : 0;
        }
        const uint64_t bm = __ballot(e < n && !valid);
        if (lane == 0) nbad += __popcll(bm);
        const uint64_t hm = __ballot(has);
        if (lane == kWave - 1) acc += __popcll(hm);
        for (int b = lmin; b < kWave - 1 && __ballot(hi != 0) != 0; ++b, hi >>= 1) {
            const uint64_t m = __ballot((hi & 1) != 0);
            if (lane == b) acc += __popcll(m);
        }
    }
    if (acc) atomicAdd(&s_bits[lane], acc);
    if (nbad) atomicAdd(&plan->bad_sel, nbad);
    __syncthreads();
    if (t < kWave) bits[(int64_t)blockIdx.x * kWave + t] = s_bits[t];
}

// Inputs and outputs of the planning step (device pointers).
struct PlanArgs {
    int32_t G;
    int64_t n_rows;           // N, the bank's rows
    const int64_t *off;
    const int64_t *toff;      // [G+1] the tiled copy's segment starts, or NULL
    int32_t *qoff;            // [G+1]
    int32_t *wstart;          // [G+1] first full-length chunk item of each cluster
    int32_t *wlast;           // [G]   item of the cluster's shorter last chunk (-1: none)
    int32_t *gstart;          // [G+1] first level-one merge group of each cluster
    int32_t *mstart;          // [G+1] first merge-list entry of each cluster
    int64_t *pbase;           // [G]
    int64_t *ubase;           // [G]
    Plan *plan;
    int64_t chunk_min, p_cap;
    int64_t direct;           // most keys a one-level merge of a pair reads
    int32_t kp;               // key slots per partial (k rounded up to a power of two)
};

// One DPP move of a 64-bit value (both halves with the same control); lanes
// outside row_mask, or reading outside their row, get 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int64_t dpp64(int64_t x) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, ROW_MASK, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)((uint64_t)x >> 32), CTRL, ROW_MASK,
                                               0xF, true);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Inclusive prefix sum within each 16-lane row (row_shr 1, 2, 4, 8).
__device__ __forceinline__ int64_t row_scan64(int64_t x) {
    x += dpp64<0x111, 0xF>(x);
    x += dpp64<0x112, 0xF>(x);
    x += dpp64<0x114, 0xF>(x);
    x += dpp64<0x118, 0xF>(x);
    return x;
}

// Inclusive prefix sum over the wave: rows, then row_bcast:15 into rows 1
// and 3 and row_bcast:31 into rows 2 and 3.
__device__ __forceinline__ int64_t wave_scan64(int64_t x) {
    x = row_scan64(x);
    x += dpp64<0x142, 0xA>(x);
    x += dpp64<0x143, 0xC>(x);
    return x;
}

// Exclusive scan and total of N values per thread over the 1024-thread block,
// in two barriers: each wave scans with DPP, then the 16 wave totals of each
// value are scanned by one 16-lane row. s: LDS of at least 17 * N int64. v
// becomes the exclusive prefix.
template <int N>
__device__ void block_scan_n(int64_t (&v)[N], int64_t (&total)[N], int64_t *s) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int waves = kPlanThreads / kWave;
    static_assert(waves == 16, "the wave totals are scanned by one 16-lane row per value");
    // a wave whose values are all zero (threads past the last cluster) skips
    // the DPP scans: 16 waves share one CU here
    bool any = false;
#pragma unroll
    for (int i = 0; i < N; ++i) any |= v[i] != 0;
    const bool live = __ballot(any) != 0;
    int64_t x[N];
    if (live) {
#pragma unroll
        for (int i = 0; i < N; ++i) x[i] = wave_scan64(v[i]);
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i) x[i] = 0;
    }
    if (lane == kWave - 1) {
#pragma unroll
        for (int i = 0; i < N; ++i) s[wave * N + i] = x[i];
    }
    __syncthreads();
    if (threadIdx.x < waves * N) {  // row = one value, lane in row = one wave
        const int vi = threadIdx.x >> 4, w = threadIdx.x & 15;
        const int64_t c = s[w * N + vi];
        const int64_t incl = row_scan64(c);
        s[waves * N + w * N + vi] = incl - c;
        if (w == waves - 1) s[2 * waves * N + vi] = incl;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < N; ++i) {
        v[i] = s[waves * N + wave * N + i] + x[i] - v[i];
        total[i] = s[2 * waves * N + i];
    }
    __syncthreads();
}

// Sum over the wave of a 64-bit value, in every lane (DPP / permlane).
__device__ __forceinline__ int64_t wave_sum64(int64_t x) {
    const int lane = threadIdx.x & 63;
    x += (int64_t)lane_xor64<1>((uint64_t)x, lane);
    x += (int64_t)lane_xor64<2>((uint64_t)x, lane);
    x += (int64_t)lane_xor64<4>((uint64_t)x, lane);
    x += (int64_t)lane_xor64<8>((uint64_t)x, lane);
    x += (int64_t)lane_xor64<16>((uint64_t)x, lane);
    x += (int64_t)lane_xor64<32>((uint64_t)x, lane);
    return x;
}

// Block totals of N values per thread (no prefix), in two barriers.
// s: LDS of at least 17 * N int64.
template <int N>
__device__ void block_sum_n(int64_t (&v)[N], int64_t *s) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int waves = kPlanThreads / kWave;
    bool any = false;
#pragma unroll
    for (int i = 0; i < N; ++i) any |= v[i] != 0;
    const bool live = __ballot(any) != 0;      // all-zero waves skip the DPP sums
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int64_t x = live ? wave_sum64(v[i]) : 0;
        if (lane == 0) s[wave * N + i] = x;
    }
    __syncthreads();
    if (threadIdx.x < N) {
        int64_t run = 0;
        for (int w = 0; w < waves; ++w) run += s[w * N + threadIdx.x];
        s[waves * N + threadIdx.x] = run;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = s[waves * N + i];
    __syncthreads();
}

// Candidate chunk lengths chunk_min * 2^i, i < kChunkCands: the last is at
// least 2^31 rows, longer than any segment, so it always fits (each
// (query, slot) then has one partial and p_cap >= B*c).
constexpr int kChunkCands = 26;

// Buckets of the clusters' shorter last chunks (item order): by length
// (longest first), and within a length, clusters of more than one query tile
// (16 queries) before the others, whose items cost less per row.
constexpr int kLenBuckets = 8;
constexpr int kItemBuckets = 2 * kLenBuckets;
__device__ __forceinline__ int item_bucket(int64_t len, int lch, int64_t nq) {   // 0 < len < 2^lch
    int b = lch - 1 - (63 - __builtin_clzll((unsigned long long)len));
    b = b < kLenBuckets - 1 ? b : kLenBuckets - 1;
    return 2 * b + (nq > 16 ? 0 : 1);
}

// LDS copies of the per-cluster tables the planning step writes (fused routing).
struct PlanMirror {
    int32_t *qoff, *wstart, *gstart, *mstart;   // [G+1]
    int32_t *wlast;                             // [G]
    int64_t *pbase, *ubase;                     // [G]
};

// Chunk length and work numbering from the per-cluster query counts (read
// through cnt_of) and the segment lengths (len_of): the chunk is the
// smallest candidate length for which the partial results fit in p_cap.
// Writes qoff, wstart, wlast, gstart, mstart, pbase and ubase to the LDS
// mirror m (the fused routing uses them in the same block) and the plan.
// Clusters are split into contiguous ranges, one per thread. Returns the
// chunk length (in every thread).
template <typename CntOf, typename LenOf>
__device__ int64_t plan_chunks(const PlanArgs &pa, CntOf cnt_of, LenOf len_of, int64_t *s,
                               PlanMirror m) {
    const int t = threadIdx.x;
    const int32_t G = pa.G;
    const int32_t per = (G + kPlanThreads - 1) / kPlanThreads;
    const int32_t g0 = min((int32_t)G, t * per), g1 = min((int32_t)G, g0 + per);
    const int lmin = 63 - __builtin_clzll((unsigned long long)pa.chunk_min);   // chunk_min is a power of two
    // Partials for candidate length chunk_min * 2^i: sum over the thread's
    // clusters of (queries) x (chunks). They only fall as i grows, so the
    // first four candidates are tried together (the usual answer) and the
    // rest by bisection; the last candidate always fits.
    auto partials = [&](int i) {
        int64_t p = 0;
        for (int32_t g = g0; g < g1; ++g) {
            const int64_t c = cnt_of(g), len = len_of(g);
            if (c > 0 && len > 0) p += c * ((len + (int64_t(1) << (lmin + i)) - 1) >> (lmin + i));
        }
        return p;
    };
    int64_t q[1] = {0}, qtot[1];
    for (int32_t g = g0; g < g1; ++g) q[0] += cnt_of(g);
    block_scan_n<1>(q, qtot, s);
    constexpr int kFirst = 4;
    int64_t p4[kFirst];
#pragma unroll
    for (int i = 0; i < kFirst; ++i) p4[i] = 0;
    for (int32_t g = g0; g < g1; ++g) {        // the four in one pass over the clusters
        const int64_t c = cnt_of(g), len = len_of(g);
        if (c > 0 && len > 0) {
#pragma unroll
            for (int i = 0; i < kFirst; ++i)
                p4[i] += c * ((len + (int64_t(1) << (lmin + i)) - 1) >> (lmin + i));
        }
    }
    block_sum_n<kFirst>(p4, s);
    int cand = -1;
#pragma unroll
    for (int i = kFirst - 1; i >= 0; --i)
        if (p4[i] <= pa.p_cap) cand = i;
    if (cand < 0) {
        int lo = kFirst, hi = kChunkCands - 1;     // the answer is in [lo, hi]
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            int64_t pm[1] = {partials(mid)};
            block_sum_n<1>(pm, s);
            if (pm[0] <= pa.p_cap) hi = mid;
            else lo = mid + 1;
        }
        cand = lo;
    }
    const int lch = lmin + cand;
    const int64_t ch = int64_t(1) << lch;

    // Items: first every full-length chunk, cluster by cluster; then each
    // cluster's shorter last chunk, in buckets by length (longest first) and
    // query tiles (item_bucket), so that the dynamic work counter hands out
    // the costliest items first and the cheap ones fill the end. Length
    // bucket b holds lengths in [ch >> (b+1), ch >> b) (the last one
    // everything shorter). Counts that fit 32 bits are scanned two per 64-bit
    // value: (full items, level-one groups), bucket pairs.
    const int64_t kp = pa.kp;
    constexpr int NW = 4 + kItemBuckets / 2;
    int64_t w[NW], wt[NW];   // items | groups << 32, partials, level-one, merge list, buckets
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0;
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t c = cnt_of(g), len = len_of(g);
        const int64_t nch = (c > 0 && len > 0) ? (len + ch - 1) >> lch : 0;
        const int64_t nfull = c > 0 ? len >> lch : 0;
        const int64_t ng = group_count(nch, kp, pa.direct);
        w[0] += nfull + (ng << 32);
        w[1] += nch * c;
        w[2] += ng * c;
        w[3] += nch != 1 ? c : 0;        // empty segments are finished by the merge too
        if (nch > nfull) {
            const int b = item_bucket(len - (nfull << lch), lch, c);
#pragma unroll
            for (int i = 0; i < kItemBuckets / 2; ++i)
                if ((b >> 1) == i) w[4 + i] += int64_t(1) << (32 * (b & 1));
        }
    }
    block_scan_n<NW>(w, wt, s);
    const int64_t n_full = wt[0] & 0xffffffff;
    // next item of each bucket of last chunks, for this thread's clusters
    int32_t bnext[kItemBuckets];
    {
        int64_t at = n_full;
#pragma unroll
        for (int b = 0; b < kItemBuckets; ++b) {
            bnext[b] = (int32_t)(at + ((w[4 + b / 2] >> (32 * (b & 1))) & 0xffffffff));
            at += (wt[4 + b / 2] >> (32 * (b & 1))) & 0xffffffff;
        }
        if (t == kPlanThreads - 1) pa.plan->n_items = at;
    }
    int64_t qrun = q[0];
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t c = cnt_of(g), len = len_of(g);
        const int64_t nch = (c > 0 && len > 0) ? (len + ch - 1) >> lch : 0;
        const int64_t nfull = c > 0 ? len >> lch : 0;
        const int64_t ng = group_count(nch, kp, pa.direct);
        int32_t wl = -1;
        if (nch > nfull) {
            const int b = item_bucket(len - (nfull << lch), lch, c);
#pragma unroll
            for (int i = 0; i < kItemBuckets; ++i)
                if (b == i) wl = bnext[i]++;
        }
        m.qoff[g] = (int32_t)qrun;
        m.wstart[g] = (int32_t)(w[0] & 0xffffffff);
        m.wlast[g] = wl;
        m.pbase[g] = w[1];
        m.gstart[g] = (int32_t)(w[0] >> 32);
        m.ubase[g] = w[2];
        m.mstart[g] = (int32_t)w[3];
        qrun += c;
        w[0] += nfull + (ng << 32);
        w[1] += nch * c;
        w[2] += ng * c;
        w[3] += nch != 1 ? c : 0;
    }
    if (t == kPlanThreads - 1) {
        m.qoff[G] = (int32_t)qtot[0];
        m.wstart[G] = (int32_t)n_full;
        m.gstart[G] = (int32_t)(wt[0] >> 32);
        m.mstart[G] = (int32_t)wt[3];
        pa.plan->chunk = ch;
        pa.plan->n_parts = wt[1];
        pa.plan->n_groups = wt[0] >> 32;
        pa.plan->n_l1 = wt[2];
        pa.plan->n_merge = wt[3];
    }
    return ch;
}

struct LdsCnt {
    const int32_t *cnt;
    __device__ int64_t operator()(int32_t g) const { return cnt[g]; }
};
// Segment length of cluster g from the offsets (an LDS copy).
struct OffLen {
    const int64_t *off;
    __device__ int64_t operator()(int32_t g) const { return off[g + 1] - off[g]; }
};
// Outputs of the fine stage, for pairs the routing finishes itself: a
// selected cluster id out of range gives an empty slot (no candidates).
struct SlotOut {
    float *slot_max, *slot_sum, *cand_score;
    int32_t *cand_id;
    int32_t k;
    __device__ void empty(int64_t e) const {
        slot_max[e] = -INFINITY;
        slot_sum[e] = 0.0f;
        for (int32_t r = 0; r < k; ++r) {
            cand_score[e * k + r] = -INFINITY;
            cand_id[e * k + r] = -1;
        }
    }
};

// The bank's segment offsets (global or LDS) must partition its rows:
// off[0] = 0, nondecreasing, off[G] = N (Eq. local nodes: every record has
// one parent). Checked by the whole block before any row is indexed through
// them; returns the verdict in every thread.
__device__ __forceinline__ bool offsets_bad(const int64_t *off, int32_t G, int64_t N,
                                            const int64_t *toff) {
    int bad = 0;
    for (int32_t g = threadIdx.x; g < G; g += blockDim.x) {
        bad |= off[g] > off[g + 1];
        // the tiled copy's header must match: segments padded to 16 rows
        if (toff) bad |= toff[g + 1] - toff[g] != ((off[g + 1] - off[g] + 15) & ~int64_t(15));
    }
    if (threadIdx.x == 0) bad |= off[0] != 0 || off[G] != N || (toff && toff[0] != 0);
    return __syncthreads_or(bad) != 0;
}

// A plan with no work: nothing is streamed or merged (malformed offsets).
__device__ __forceinline__ void plan_nothing(Plan *plan) {
    plan->chunk = 1;
    plan->n_items = 0;
    plan->n_parts = 0;
    plan->n_groups = 0;
    plan->n_l1 = 0;
    plan->n_merge = 0;
    plan->next = 0;
    plan->bad_off = 1;
}

// ---- planning step of the multi-block routing -------------------------------
// route_plan: every block takes the same chunk length from the bit counts of
// route_count, then plans its own range of clusters (rounds x 256 of them;
// each wave a contiguous run, 64 at a time, one per lane, so that the
// per-cluster loads and stores are coalesced): the block-local exclusive
// prefixes of the four scanned values, and each cluster's rank among the
// block's last chunks of its length bucket; agg[block] holds the block's
// totals and its offsets check. route_emit adds the bases of the blocks
// before (a scan of agg). The plan is the one route_fused makes, table for
// table.
constexpr int kAgg = 4 + kItemBuckets + 1;   // scanned values, last chunks per bucket, bad offsets

// Per-cluster values at chunk 2^lch: v[0] = full items | level-one groups
// << 32, v[1] = partials, v[2] = level-one results, v[3] = queries |
// merge-list entries << 32 (each total below 2^31); returns the bucket of
// the cluster's shorter last chunk, or -1 if all its chunks are full-length.
__device__ __forceinline__ int plan_values(const PlanArgs &pa, int64_t c, int64_t len, int lch,
                                           int64_t (&v)[4]) {
    const int64_t ch = int64_t(1) << lch;
    const int64_t nch = (c > 0 && len > 0) ? (len + ch - 1) >> lch : 0;
    const int64_t nfull = c > 0 ? len >> lch : 0;
    const int64_t ng = group_count(nch, pa.kp, pa.direct);
    v[0] = nfull + (ng << 32);
    v[1] = nch * c;
    v[2] = ng * c;
    v[3] = c + ((nch != 1 ? c : 0) << 32);     // empty segments are finished by the merge too
    return nch > nfull ? item_bucket(len - (nfull << lch), lch, c) : -1;
}

// Chunk length (log2), the same in every block: the smallest candidate
// chunk_min * 2^i whose partial results fit in p_cap (the last always fits).
__device__ __forceinline__ int route_chunk_log2(const PlanArgs &pa, const uint32_t *bits, int32_t nb2) {
    __shared__ unsigned long long s_bits[kWave];
    __shared__ int32_t s_cand;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (t < kWave) s_bits[t] = 0;
    __syncthreads();
    constexpr int per = kCountBlocks / (kRouteThreads / kWave);
    uint32_t x[per];                           // every load in flight at once
#pragma unroll
    for (int i = 0; i < per; ++i) {
        const int32_t r = wave + i * (kRouteThreads / kWave);
        x[i] = r < nb2 ? bits[(int64_t)r * kWave + lane] : 0;
    }
    unsigned long long acc = 0;
#pragma unroll
    for (int i = 0; i < per; ++i) acc += x[i];
    if (acc) atomicAdd(&s_bits[lane], acc);
    __syncthreads();
    const int lmin = 63 - __builtin_clzll((unsigned long long)pa.chunk_min);
    if (wave == 0) {
        // candidates in order, one wave sum each (the first usually fits):
        // lane b < 63 adds its count times 2^(b-j) for b >= j, lane 63 the
        // pairs; a term above cap rules the candidate out, so the sum of at
        // most 64 terms of at most cap each cannot overflow
        const uint64_t cb = s_bits[lane], cap = (uint64_t)pa.p_cap;
        int cand = kChunkCands - 1;
#pragma unroll 1
        for (int i = 0; i < kChunkCands - 1; ++i) {
            const int j = lmin + i;
            uint64_t term = lane == kWave - 1 ? cb : 0;
            bool over = false;
            if (lane < kWave - 1 && lane >= j) {
                const int sh = lane - j;
                over = cb > (cap >> sh);
                term = over ? 0 : cb << sh;
            }
            if (__ballot(over) == 0 && (uint64_t)wave_sum64((int64_t)term) <= cap) {
                cand = i;
                break;
            }
        }
        if (lane == 0) s_cand = cand;
    }
    __syncthreads();
    return lmin + s_cand;
}

// A cluster's count and segment, and the offsets check of cluster g.
struct ClusterIn {
    int64_t c, len;
    bool bad;
};
__device__ __forceinline__ ClusterIn cluster_in(const PlanArgs &pa, const int32_t *cnt, int32_t g) {
    ClusterIn ci;
    const int64_t a0 = pa.off[g], a1 = pa.off[g + 1];
    ci.c = cnt[g];
    ci.len = a1 - a0;
    ci.bad = a0 > a1;
    // the tiled copy's header must match: segments padded to 16 rows
    if (pa.toff) ci.bad |= pa.toff[g + 1] - pa.toff[g] != ((a1 - a0 + 15) & ~int64_t(15));
    return ci;
}

__global__ __launch_bounds__(kRouteThreads) void route_plan(PlanArgs pa, const int32_t *cnt,
                                                           const uint32_t *bits, int32_t nb2,
                                                           int32_t rounds, int64_t *agg,
                                                           int32_t n_route, QCopy qc) {
    if ((int32_t)blockIdx.x >= n_route) {
        copy_queries(qc, blockIdx.x - n_route, gridDim.x - n_route);
        return;
    }
    constexpr int waves = kRouteThreads / kWave;
    __shared__ int64_t sw[waves * kAgg];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int32_t G = pa.G;
    const int32_t per_wave = rounds * kWave;
    const int32_t gw0 = min(G, (int32_t)(blockIdx.x * waves + wave) * per_wave);
    const int32_t gw1 = min(G, gw0 + per_wave);
    // the first round's cluster, loaded while the chunk length is chosen
    // (and kept for the second pass)
    ClusterIn c0{0, 0, false};
    if (gw0 + lane < gw1) c0 = cluster_in(pa, cnt, gw0 + lane);
    const int lch = route_chunk_log2(pa, bits, nb2);
    if (blockIdx.x == 0 && t == 0) pa.plan->chunk = int64_t(1) << lch;
    // pass 0: this wave's totals (lane b: its last chunks in bucket b);
    // pass 1: block-local exclusive prefixes, from the waves before this one.
    // One copy of the per-cluster code for both (it runs once per call: its
    // instructions are fetched cold)
    int64_t tot[4] = {0, 0, 0, 0}, carry[4] = {0, 0, 0, 0}, bcnt = 0, bnext = 0;
    int bad = blockIdx.x == 0 && t == 0 &&
              (pa.off[0] != 0 || pa.off[G] != pa.n_rows || (pa.toff && pa.toff[0] != 0));
    const uint64_t lt = (uint64_t(1) << lane) - 1;
#pragma unroll 1
    for (int pass = 0; pass < 2; ++pass) {
        if (pass == 1) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t x = wave_sum64(tot[i]);
                if (lane == 0) sw[wave * kAgg + i] = x;
            }
            if (lane < kItemBuckets) sw[wave * kAgg + 4 + lane] = bcnt;
            const uint64_t bm = __ballot(bad != 0);
            if (lane == 0) sw[wave * kAgg + kAgg - 1] = bm != 0;
            __syncthreads();
            if (t < kAgg) {
                int64_t x = 0;
#pragma unroll
                for (int w = 0; w < waves; ++w) x += sw[w * kAgg + t];
                agg[(int64_t)blockIdx.x * kAgg + t] = x;
            }
            for (int w = 0; w < wave; ++w) {
#pragma unroll
                for (int i = 0; i < 4; ++i) carry[i] += sw[w * kAgg + i];
                if (lane < kItemBuckets) bnext += sw[w * kAgg + 4 + lane];
            }
        }
        for (int32_t gr = gw0; gr < gw1; gr += kWave) {
            const int32_t g = gr + lane;
            const bool valid = g < gw1;
            int64_t v[4] = {0, 0, 0, 0};
            int b = -1;
            if (valid) {
                const ClusterIn ci = gr == gw0 ? c0 : cluster_in(pa, cnt, g);
                bad |= ci.bad;
                b = plan_values(pa, ci.c, ci.len, lch, v);
            }
            const bool any_last = __ballot(b >= 0) != 0;
            if (pass == 0) {
#pragma unroll
                for (int i = 0; i < 4; ++i) tot[i] += v[i];
#pragma unroll 1
                for (int bb = 0; bb < (any_last ? kItemBuckets : 0); ++bb) {
                    const uint64_t m = __ballot(b == bb);
                    if (lane == bb) bcnt += __popcll(m);
                }
                continue;
            }
            int64_t ex[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t incl = wave_scan64(v[i]);
                ex[i] = carry[i] + incl - v[i];
                carry[i] += __shfl(incl, kWave - 1);
            }
            int32_t wl = -1;                   // rank among the block's last chunks of bucket b, | b
#pragma unroll 1
            for (int bb = 0; bb < (any_last ? kItemBuckets : 0); ++bb) {
                const uint64_t m = __ballot(b == bb);
                if (m) {
                    const int64_t bn = __shfl(bnext, bb);
                    if (b == bb) wl = (int32_t)((bn + __popcll(m & lt)) << 4) | bb;
                    if (lane == bb) bnext += __popcll(m);
                }
            }
            if (valid) {
                pa.qoff[g] = (int32_t)(ex[3] & 0xffffffff);
                pa.mstart[g] = (int32_t)(ex[3] >> 32);
                pa.wstart[g] = (int32_t)(ex[0] & 0xffffffff);
                pa.gstart[g] = (int32_t)(ex[0] >> 32);
                pa.pbase[g] = ex[1];
                pa.ubase[g] = ex[2];
                pa.wlast[g] = wl;
            }
        }
    }
}

// Bytes of the LDS tables of the fused routing kernel for G clusters and n
// (query, slot) pairs: offsets, partial and level-one bases, counts, four
// starts tables, the last-chunk items, then the pairs' clusters as 16-bit ids
// and their 16-bit positions in their clusters' lists.
size_t route_fused_lds(int32_t G, int64_t n) {
    return (size_t)(3 * G + 1) * 8 + (size_t)(6 * G + 4) * 4 + (size_t)n * 4;
}

// The merge's description of pair e, position i in the list of its cluster
// (nch chunks in level-one groups of r, none if r is 0; nq queries; partials
// from pb, level-one results from ub).
__device__ __forceinline__ MergeSlot merge_slot(int64_t e, int32_t i, int64_t nch, int64_t r,
                                                int32_t nq, int64_t pb, int64_t ub) {
    MergeSlot ms;
    ms.e = (int32_t)e;
    ms.stride = nq;
    ms.level = r > 0;
    ms.n = (int32_t)(r > 0 ? div_up32(nch, r) : nch);
    ms.p0 = (r > 0 ? ub : pb) + i;
    return ms;
}

// Level-one group jg of a cluster (nch chunks, groups of r, nq queries,
// partials from pb, results from ub).
__device__ __forceinline__ MergeGroup merge_group_of(int32_t jg, int64_t nch, int64_t r,
                                                     int32_t nq, int64_t pb, int64_t ub) {
    MergeGroup mg;
    mg.p0 = pb + jg * r * nq;
    mg.u0 = ub + (int64_t)jg * nq;
    mg.npart = (int32_t)(nch - jg * r < r ? nch - jg * r : r);
    mg.nq = nq;
    return mg;
}

// Position in the item table of the w-th full-length chunk (cluster by
// cluster) among n_full: a fixed permutation (multiplication by a prime above
// any item count, modulo n_full) that spreads each cluster's chunks over the
// table, so that the blocks reach a cluster's chunks at different times and
// the later ones start from the bounds the earlier ones published.
__device__ __forceinline__ int32_t full_slot(int32_t w, int32_t n_full) {
    // w p mod n = w (p mod n) mod n; the product of two values below n <
    // 2^31 is reduced with a quotient estimated in double precision (off by
    // at most one: the quotient is below 2^31) and corrected
    const int64_t n = n_full, pm = (int64_t)(2147483629u % (uint32_t)n_full);
    const int64_t x = (int64_t)w * pm;
    int64_t r = x - (int64_t)((double)x / (double)n) * n;
    r += r < 0 ? n : 0;
    r -= r >= n ? n : 0;
    return (int32_t)r;
}

// Work item j (a chunk of ch = 2^lch rows) of cluster g, whose segment starts
// at bank row a0 and has len rows, with nq queries listed from qb and its
// partials from pb.
__device__ __forceinline__ WorkItem make_item(int32_t g, int64_t j, int64_t a0, int64_t len,
                                              int lch, int32_t qb, int32_t nq, int64_t pb) {
    const int64_t ch = int64_t(1) << lch, r = len - (j << lch);
    WorkItem wi;
    wi.r0 = a0 + (j << lch);
    wi.p0 = pb + j * nq;
    wi.len = (int32_t)(r < ch ? r : ch);
    wi.g = g;
    wi.qbeg = qb;
    wi.nq = nq;
    wi.single = len <= ch;          // the chunk is the whole segment
    wi.pad = 0;
    return wi;
}
constexpr uint16_t kNoCluster = 0xffff;   // selection out of range (G < kNoCluster in LDS)

// The whole routing in one block when the pairs are few and the per-cluster
// tables fit in LDS: count the (query, slot) pairs per cluster, plan the
// chunks, scatter the pairs into per-cluster lists, then fill the work items
// (each thread finds its items' clusters by binary search over the item starts
// in LDS), the level-one merge groups and units, and the merge list. The
// selections and every per-cluster table the later steps read are kept in
// LDS, so global memory is read once, at the start.
__global__ __launch_bounds__(kPlanThreads) void route_fused(PlanArgs pa, const int32_t *sel,
                                                            int64_t n, int32_t *qlist,
                                                            int32_t *pos, uint64_t *bound, SlotOut out,
                                                            WorkItem *items, MergeGroup *groups,
                                                            int2 *units, MergeSlot *mlist) {
    extern __shared__ int64_t lds[];
    __shared__ int64_t s[(kPlanThreads / kWave + 1) * kChunkCands];
    __shared__ int32_t s_bad;
    const int t = threadIdx.x;
    const int32_t G = pa.G;
    int64_t *loff = lds, *lpb = loff + G + 1, *lub = lpb + G;
    int32_t *lcnt = reinterpret_cast<int32_t *>(lub + G);   // counts, then fill cursors
    PlanMirror m;
    m.wstart = lcnt + G;
    m.qoff = m.wstart + G + 1;
    m.gstart = m.qoff + G + 1;
    m.mstart = m.gstart + G + 1;
    m.wlast = m.mstart + G + 1;
    m.pbase = lpb;
    m.ubase = lub;
    uint16_t *lsel = reinterpret_cast<uint16_t *>(m.wlast + G);
    uint16_t *lpos = lsel + n;                 // position of each pair in its cluster's list
    for (int64_t e0 = t; e0 < n; e0 += 8 * kPlanThreads) {   // 8 loads in flight per thread
        int32_t g[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int64_t e = e0 + r * kPlanThreads;
            g[r] = sel[e < n ? e : 0];
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int64_t e = e0 + r * kPlanThreads;
            if (e < n) lsel[e] = g[r] >= 0 && g[r] < G ? (uint16_t)g[r] : kNoCluster;
        }
    }
    for (int32_t g = t; g <= G; g += kPlanThreads) loff[g] = pa.off[g];
    for (int32_t g = t; g < G; g += kPlanThreads) lcnt[g] = 0;
    if (t == 0) s_bad = 0;
    __syncthreads();
    if (offsets_bad(loff, G, pa.n_rows, pa.toff)) {   // before any row is indexed through them
        if (t == 0) {
            plan_nothing(pa.plan);
            pa.plan->bad_sel = 0;
        }
        for (int64_t e = t; e < n; e += kPlanThreads) {
            bound[e] = 0;
            out.empty(e);
        }
        return;
    }
    int32_t bad = 0;
    for (int64_t e = t; e < n; e += kPlanThreads) {
        const uint16_t h = lsel[e];
        if (h != kNoCluster) lpos[e] = (uint16_t)atomicAdd(&lcnt[h], 1);
        else ++bad;
    }
    if (bad) atomicAdd(&s_bad, bad);
    __syncthreads();
    const int64_t ch = plan_chunks(pa, LdsCnt{lcnt}, OffLen{loff}, s, m);
    const int lch = 63 - __builtin_clzll((unsigned long long)ch);
    if (t == 0) {
        pa.plan->next = 0;
        pa.plan->bad_sel = s_bad;
        pa.plan->bad_off = 0;
    }
    __syncthreads();
    const int64_t kp = pa.kp;
    const int32_t *lwst = m.wstart;
    for (int64_t e = t; e < n; e += kPlanThreads) {
        const uint16_t h = lsel[e];
        bound[e] = 0;
        if (h != kNoCluster) {
            const int32_t g = h;
            const int32_t qb = m.qoff[g];
            const int32_t i = lpos[e];
            const int32_t at = qb + i;
            qlist[at] = (int32_t)e;
            pos[e] = i;
            const int64_t len = loff[g + 1] - loff[g];
            const int64_t nch = (len + ch - 1) >> lch;
            const int64_t r = group_span(nch, kp, pa.direct);
            if (nch != 1)
                mlist[m.mstart[g] + i] =
                    merge_slot(e, i, nch, r, m.qoff[g + 1] - qb, lpb[g], lub[g]);
            if (r > 0) {                   // this pair's level-one units, one per group
                const int32_t nq = m.qoff[g + 1] - qb, gs = m.gstart[g];
                const int32_t ng = m.gstart[g + 1] - gs;
                const int64_t ub = lub[g];
                for (int32_t jg = 0; jg < ng; ++jg)
                    units[ub + (int64_t)jg * nq + i] = make_int2(gs + jg, i);
            }
        } else {
            out.empty(e);
        }
    }
    const int32_t n_full = lwst[G];            // full-length chunks, cluster by cluster
    for (int32_t w = t; w < n_full; w += kPlanThreads) {
        int32_t lo = 0, hi = G;                // lwst[lo] <= w < lwst[hi]
        while (hi - lo > 1) {
            const int32_t mid = (lo + hi) >> 1;
            if (lwst[mid] <= w) lo = mid; else hi = mid;
        }
        const int32_t g = lo, qb = m.qoff[g];
        items[full_slot(w, n_full)] = make_item(g, w - lwst[g], loff[g], loff[g + 1] - loff[g],
                                                lch, qb, m.qoff[g + 1] - qb, lpb[g]);
    }
    for (int32_t g = t; g < G; g += kPlanThreads) {   // the shorter last chunks
        const int32_t wl = m.wlast[g];
        if (wl < 0) continue;
        const int64_t len = loff[g + 1] - loff[g];
        const int32_t qb = m.qoff[g];
        items[wl] = make_item(g, len >> lch, loff[g], len, lch, qb, m.qoff[g + 1] - qb, lpb[g]);
    }
    for (int32_t g = t; g < G; g += kPlanThreads) {
        const int32_t gs = m.gstart[g], ng = m.gstart[g + 1] - gs;
        if (ng == 0) continue;
        const int32_t nq = m.qoff[g + 1] - m.qoff[g];
        const int64_t nch = (loff[g + 1] - loff[g] + ch - 1) >> lch;
        const int64_t r = group_span(nch, kp, pa.direct);
        for (int32_t jg = 0; jg < ng; ++jg)
            groups[gs + jg] = merge_group_of(jg, nch, r, nq, lpb[g], lub[g]);
    }
}

// Finishes the routing, one thread per pair: the bases of each planning
// block (a scan of agg, one lane per block) turn its local tables into
// global ones; pair e, place i in the list of its cluster g (nq pairs), writes its list
// entry, its merge-list entry and level-one units, and the cluster's work
// items j and level-one groups jg with j, jg = i mod nq (a cluster's pairs
// share its tables). Block 0 writes the plan's totals. Malformed offsets:
// every slot is empty and the plan has no work.
__global__ __launch_bounds__(kRouteThreads) void route_emit(PlanArgs pa, const int32_t *sel, int64_t n,
                                                           const int32_t *cnt, const int32_t *pos,
                                                           const int64_t *agg, int32_t nb3,
                                                           int32_t per_block, int32_t *qlist,
                                                           uint64_t *bound, SlotOut out,
                                                           WorkItem *items, MergeGroup *groups,
                                                           int2 *units, MergeSlot *mlist,
                                                           int32_t n_route, QCopy qc) {
    if ((int32_t)blockIdx.x >= n_route) {
        copy_queries(qc, blockIdx.x - n_route, gridDim.x - n_route);
        return;
    }
    constexpr int NB = kAgg - 1;               // per-block bases: the scanned values, the buckets
    __shared__ int64_t s_base[kRouteBlocks * NB];
    __shared__ int64_t s_tot[kAgg];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int32_t G = pa.G;
    const int64_t chunk = pa.plan->chunk;
    // this thread's pair and its cluster's tables, loaded before the scan
    const int64_t e = blockIdx.x * (int64_t)kRouteThreads + t;
    const int32_t g = e < n ? sel[e] : -1;
    const bool valid = g >= 0 && g < G;
    int32_t i = 0, nq = 0, qoff = 0, mst = 0, wst = 0, gst = 0, code = -1;
    int64_t a0 = 0, len = 0, pb = 0, ub = 0;
    if (valid) {
        i = pos[e];
        nq = cnt[g];
        a0 = pa.off[g];
        len = pa.off[g + 1] - a0;
        qoff = pa.qoff[g];
        mst = pa.mstart[g];
        wst = pa.wstart[g];
        gst = pa.gstart[g];
        code = pa.wlast[g];
        pb = pa.pbase[g];
        ub = pa.ubase[g];
    }
    constexpr int per = (kAgg + kRouteThreads / kWave - 1) / (kRouteThreads / kWave);
    int64_t x[per];
#pragma unroll
    for (int j = 0; j < per; ++j) {
        const int v = wave + j * (kRouteThreads / kWave);
        x[j] = v < kAgg && lane < nb3 ? agg[(int64_t)lane * kAgg + v] : 0;
    }
#pragma unroll
    for (int j = 0; j < per; ++j) {
        const int v = wave + j * (kRouteThreads / kWave);
        if (v < kAgg) {
            const int64_t incl = wave_scan64(x[j]);
            if (v < NB) s_base[lane * NB + v] = incl - x[j];
            if (lane == kWave - 1) s_tot[v] = incl;
        }
    }
    __syncthreads();
    const int64_t n_full = s_tot[0] & 0xffffffff;
    // items: every full-length chunk, then bucket by bucket (lane b of each
    // row: the first item of bucket b)
    const int64_t bt = s_tot[4 + (lane & 15)];
    const int64_t bstart = n_full + row_scan64(bt) - bt;
    const bool bad = s_tot[kAgg - 1] != 0;
    if (blockIdx.x == 0 && t == kItemBuckets - 1) {
        if (bad) {
            plan_nothing(pa.plan);
        } else {
            pa.plan->n_items = bstart + bt;
            pa.plan->n_parts = s_tot[1];
            pa.plan->n_groups = s_tot[0] >> 32;
            pa.plan->n_l1 = s_tot[2];
            pa.plan->n_merge = s_tot[3] >> 32;
        }
    }
    const int64_t bstart_b = __shfl(bstart, code & 15);   // lanes without a last chunk: unused
    if (e >= n) return;
    bound[e] = 0;
    if (bad || !valid) {
        out.empty(e);
        return;
    }
    const int lch = 63 - __builtin_clzll((unsigned long long)chunk);
    const int64_t ch = int64_t(1) << lch, kp = pa.kp;
    const int64_t *bs = s_base + (g / per_block) * NB;
    const int32_t qb = qoff + (int32_t)(bs[3] & 0xffffffff);
    qlist[qb + i] = (int32_t)e;
    const int64_t nch = len > 0 ? (len + ch - 1) >> lch : 0;
    const int64_t r = group_span(nch, kp, pa.direct);
    pb += bs[1];
    ub += bs[2];
    if (nch != 1) mlist[mst + (int32_t)(bs[3] >> 32) + i] = merge_slot(e, i, nch, r, nq, pb, ub);
    if (r > 0) {                               // this pair's level-one units, one per group
        const int32_t gs = gst + (int32_t)(bs[0] >> 32);
        const int32_t ng = (int32_t)div_up32(nch, r);
        for (int32_t jg = 0; jg < ng; ++jg) units[ub + (int64_t)jg * nq + i] = make_int2(gs + jg, i);
        for (int32_t jg = i; jg < ng; jg += nq) groups[gs + jg] = merge_group_of(jg, nch, r, nq, pb, ub);
    }
    if (i < nch) {
        const int64_t nfull = len >> lch;
        const int32_t w0 = wst + (int32_t)(bs[0] & 0xffffffff);
        const int32_t wl =
            code < 0 ? -1 : (int32_t)(bstart_b + bs[4 + (code & 15)] + (code >> 4));
        for (int64_t j = i; j < nch; j += nq)
            items[j < nfull ? full_slot(w0 + (int32_t)j, (int32_t)n_full) : wl] =
                make_item(g, j, a0, len, lch, qb, nq, pb);
    }
}

// ---------------------------------------------------------------------------
// per-slot merge of the chunk partials
// ---------------------------------------------------------------------------
// A (query, slot) pair whose cluster has at most `group` chunks is merged
// directly from its chunk partials. Longer clusters first merge their chunks
// in groups (level one: one block per group, one wave per query), so that no
// wave has to read more than `group` partials; the pair then merges its
// level-one results.
struct MergeArgs {
    const MergeSlot *mlist;
    const uint64_t *bound;            // per pair: a key at most its k-th best (from the stream)
    const Plan *plan;
    const MergeGroup *groups;
    const int2 *units;
    const float *pm, *pz;
    const int32_t *pc;
    const uint64_t *pk;
    float *um, *uz;
    int32_t *uc;
    uint64_t *uk;
    int64_t n_pairs;
    int32_t k;
    float cexp;
    float *slot_max, *slot_sum, *cand_score;
    int32_t *cand_id;
};


// compact_select out of line for the merge loop (one copy; the loop body
// stays small).
struct MergeCompacted {
    int n;
    uint64_t theta;
};
template <int NPL>
__device__ __noinline__ MergeCompacted merge_compact(uint64_t *buf, int n, int k) {
    MergeCompacted r;
    r.theta = 0;
    r.n = compact_select<NPL>(buf, n, k, kWave, threadIdx.x & 63, r.theta);
    return r;
}

// One wave merges n partial results (m, Z, count, k keys) found at
// p0 + i * stride: (m, Z) lane-parallel; the keys 8 x 64 at a time through a
// threshold filter into the wave's LDS buffer (cap = 64 * NPL >= k + 64),
// compacted by radix select when it fills. The kept keys are left in buf
// (count returned), unsorted; M and Z are the merged statistics in every lane.
template <int NPL>
__device__ __forceinline__ int merge_partials(const float *pm, const float *pz, const int32_t *pc,
                                              const uint64_t *pk, int64_t p0, int64_t stride,
                                              int64_t n, int k, float cexp, uint64_t *buf,
                                              float &M, float &Z, uint64_t theta0 = 0) {
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63;
    const uint64_t lt_mask = (1ull << lane) - 1;
    // entries f = j * kp + r with kp = k rounded up to a power of two: the
    // partial and the key within it come from a shift and a mask
    const int lk = 31 - __builtin_clz((unsigned)(2 * k - 1));
    const int64_t kp = int64_t(1) << lk;
    const int64_t total = n * kp;
    // a batch of 8 x 64 entries, requested unconditionally (entries past the
    // end read the workspace's first key and are dropped where they are used;
    // p0 itself may lie past the partials when n is 0)
    auto request = [&](int64_t base, uint64_t (&kv)[kMergeBatch]) {
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const int64_t f = base + u * kWave + lane;
            const int64_t jj = f >> lk, r = f & (kp - 1);
            const bool ok = f < total && r < k;
            kv[u] = pk[ok ? (p0 + jj * stride) * k + r : 0];
        }
    };
    uint64_t cur[kMergeBatch], nxt[kMergeBatch];
    request(0, cur);                       // in flight with the statistics
    M = -INFINITY;
    Z = 0.0f;
    for (int64_t jj = lane; jj < n; jj += kWave)
        mz_merge(M, Z, pm[p0 + jj * stride], pz[p0 + jj * stride], cexp);
    for (int sh = 32; sh >= 1; sh >>= 1) {
        const float m2 = __shfl_xor(M, sh), z2 = __shfl_xor(Z, sh);
        mz_merge(M, Z, m2, z2, cexp);
    }
    int cnt = 0;
    uint64_t theta = theta0;
    for (int64_t base = 0; base < total; base += kWave * kMergeBatch) {
        request(base + kWave * kMergeBatch, nxt);   // the next batch while this one is filtered
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const int64_t f = base + u * kWave + lane;
            const uint64_t key = f < total && (f & (kp - 1)) < k ? cur[u] : 0;
            const bool pass = key > theta;
            const uint64_t mask = __ballot(pass);
            if (pass) buf[cnt + __popcll(mask & lt_mask)] = key;
            cnt += __popcll(mask);
            if (cnt > cap - kWave) {
                wave_lds_sync();
                const MergeCompacted mc = merge_compact<NPL>(buf, cnt, k);
                cnt = mc.n;
                theta = mc.theta > theta ? mc.theta : theta;
            }
        }
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) cur[u] = nxt[u];
    }
    (void)pc;
    wave_lds_sync();
    return cnt;
}

// Level one: one wave per unit (group, query) merges the group's chunk
// partials of that query into one result (the same form as a partial).
template <int NPL>
__global__ __launch_bounds__(kWave * kMergeWaves) void group_merge(MergeArgs a) {
    extern __shared__ __align__(16) uint64_t mbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t *buf = mbuf + wave * cap;
    const int64_t n_units = a.plan->n_l1;
    for (int64_t u = (int64_t)blockIdx.x * kMergeWaves + wave; u < n_units;
         u += (int64_t)gridDim.x * kMergeWaves) {
        const int2 un = a.units[u];
        const MergeGroup mg = a.groups[un.x];
        float M, Z;
        int cnt = merge_partials<NPL>(a.pm, a.pz, a.pc, a.pk, mg.p0 + un.y, mg.nq, mg.npart, a.k,
                                      a.cexp, buf, M, Z);
        if (cnt > a.k) {
            uint64_t th = 0;
            cnt = compact_select<NPL>(buf, cnt, a.k, cap - a.k, lane, th);
        }
        for (int r = lane; r < a.k; r += kWave) a.uk[u * a.k + r] = r < cnt ? buf[r] : 0;
        if (lane == 0) {
            a.um[u] = M;
            a.uz[u] = Z;
            a.uc[u] = cnt;
        }
        wave_lds_sync();
    }
}

// Level two (or the only level): one wave per (query, slot) pair whose
// cluster spans several chunks writes the slot's statistics and its top-k,
// sorted. Pairs of single-chunk clusters were finished by the bank stream.
template <int NPL>
__global__ __launch_bounds__(kWave * kMergeWaves) void slot_merge(MergeArgs a) {
    extern __shared__ __align__(16) uint64_t mbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t *buf = mbuf + wave * cap;
    const int64_t n_merge = a.plan->n_merge;
    for (int64_t u = (int64_t)blockIdx.x * kMergeWaves + wave; u < n_merge;
         u += (int64_t)gridDim.x * kMergeWaves) {
        const MergeSlot ms = a.mlist[u];
        const int64_t e = ms.e;
        // keys below the pair's bound cannot be in its top k; the bound itself
        // can (it may be the k-th key), hence one below it
        const uint64_t b = a.bound[e];
        const uint64_t theta0 = b ? b - 1 : 0;
        float M, Z;
        int cnt;
        if (ms.level)
            cnt = merge_partials<NPL>(a.um, a.uz, a.uc, a.uk, ms.p0, ms.stride, ms.n, a.k, a.cexp,
                                      buf, M, Z, theta0);
        else
            cnt = merge_partials<NPL>(a.pm, a.pz, a.pc, a.pk, ms.p0, ms.stride, ms.n, a.k, a.cexp,
                                      buf, M, Z, theta0);
        uint64_t v[NPL];
        sort_buffer<NPL>(buf, cnt, v, lane);
#pragma unroll
        for (int q = 0; q < NPL; ++q) {
            const int r = q * kWave + lane;
            if (r < a.k) {
                const uint64_t key = r < cnt ? v[q] : 0;
                a.cand_score[e * a.k + r] = key ? key_score(key) : -INFINITY;
                a.cand_id[e * a.k + r] = key ? key_id(key) : -1;
            }
        }
        if (lane == 0) {
            a.slot_max[e] = M;
            a.slot_sum[e] = Z;
        }
        wave_lds_sync();
    }
}

// One-level merges on a small bank (no level-one groups): the four waves of a
// block share a pair. Wave w merges the w-th quarter of its chunk partials
// into its own buffer (keys above the pair's bound, cut to k as it fills);
// wave 0 then merges the four (m, Z) and passes the other buffers' keys
// through the same filter into its own, sorts and writes the slot. A long
// cluster's merge is then about a quarter of the chain of requests.
template <int NPL>
__global__ __launch_bounds__(kWave * kMergeWaves) void slot_merge_shared(MergeArgs a) {
    extern __shared__ __align__(16) uint64_t mbuf[];
    __shared__ float s_m[kMergeWaves], s_z[kMergeWaves];
    __shared__ int32_t s_c[kMergeWaves];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt_mask = (1ull << lane) - 1;
    uint64_t *buf = mbuf + wave * cap;
    const int64_t n_merge = a.plan->n_merge;
    for (int64_t u = blockIdx.x; u < n_merge; u += gridDim.x) {      // block-uniform
        const MergeSlot ms = a.mlist[u];
        const int64_t e = ms.e;
        const uint64_t b = a.bound[e];
        const uint64_t theta0 = b ? b - 1 : 0;   // the bound itself may be the k-th key
        const int64_t per = ((int64_t)ms.n + kMergeWaves - 1) / kMergeWaves;
        const int64_t j0 = min((int64_t)ms.n, wave * per), j1 = min((int64_t)ms.n, j0 + per);
        float M, Z;
        const int cnt = merge_partials<NPL>(a.pm, a.pz, a.pc, a.pk, ms.p0 + j0 * ms.stride,
                                            ms.stride, j1 - j0, a.k, a.cexp, buf, M, Z, theta0);
        if (lane == 0) {
            s_m[wave] = M;
            s_z[wave] = Z;
            s_c[wave] = cnt;
        }
        __syncthreads();
        if (wave == 0) {
            float Mt = -INFINITY, Zt = 0.0f;
#pragma unroll
            for (int w = 0; w < kMergeWaves; ++w) mz_merge(Mt, Zt, s_m[w], s_z[w], a.cexp);
            int c0 = s_c[0];
            uint64_t theta = theta0;
            for (int w = 1; w < kMergeWaves; ++w) {
                const int cw = s_c[w];
                for (int base = 0; base < cw; base += kWave) {
                    const uint64_t key = base + lane < cw ? mbuf[w * cap + base + lane] : 0;
                    const bool pass = key > theta;
                    const uint64_t mask = __ballot(pass);
                    if (pass) buf[c0 + __popcll(mask & lt_mask)] = key;
                    c0 += __popcll(mask);
                    if (c0 > cap - kWave) {
                        wave_lds_sync();
                        const MergeCompacted mc = merge_compact<NPL>(buf, c0, a.k);
                        c0 = mc.n;
                        theta = mc.theta > theta ? mc.theta : theta;
                    }
                }
            }
            wave_lds_sync();
            uint64_t v[NPL];
            sort_buffer<NPL>(buf, c0, v, lane);
#pragma unroll
            for (int q = 0; q < NPL; ++q) {
                const int r = q * kWave + lane;
                if (r < a.k) {
                    const uint64_t key = r < c0 ? v[q] : 0;
                    a.cand_score[e * a.k + r] = key ? key_score(key) : -INFINITY;
                    a.cand_id[e * a.k + r] = key ? key_id(key) : -1;
                }
            }
            if (lane == 0) {
                a.slot_max[e] = Mt;
                a.slot_sum[e] = Zt;
            }
        }
        __syncthreads();           // the buffers and s_* are reused by the next pair
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int fine_cap(int k) { return next_pow2(k + kRowsPerStep); }

// Shortest chunk: the bank's rows spread over about one chunk per compute
// unit (a power of two between kChunkFloor and kChunkCeil rows); the planning
// kernel doubles it while the partial results would not fit. On a small bank
// (the ceiling not reached) the selected clusters' chunks then number about as
// many as the blocks the stream kernel keeps resident, so most items start at
// once and no block runs a chain of short ones.
static int64_t chunk_floor_rows(int64_t N, int n_cu) {
    const int64_t target = N / (int64_t)(n_cu > 0 ? n_cu : 1);
    int64_t ch = kChunkFloor;
    while (ch * 2 <= target && ch * 2 <= kChunkCeil) ch *= 2;
    return ch;
}

// Queries per pass of the generic kernel (its LDS holds only the top-k
// buffers and the score tiles).
static int qmax_generic(int cap) {
    int q = 16 * kMaxQueryTiles;
    while (q > 16 && fine_state_bytes(q, cap, 2) > 72 * 1024) q -= 16;
    return q;
}

// Queries per pass of the LDS kernel: the most (a multiple of 16, at most 64)
// whose B fragments, top-k buffers and one score tile fit in the LDS budget;
// 0 if 16 do not.
static int qmax_lds(int d, int cap, size_t budget) {
    for (int q = 16 * kMaxQueryTiles; q >= 16; q -= 16)
        if (fine_qs_bytes(d, q) + fine_state_bytes(q, cap, 1) <= budget) return q;
    return 0;
}

static size_t lds_budget() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    if (dev >= 0 && dev < 64 && cached[dev] > 0) return (size_t)cached[dev];
    int bytes = 0;
    if (hipDeviceGetAttribute(&bytes, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        bytes <= 0)
        bytes = 64 * 1024;
    bytes -= 256;       // static LDS of the kernels (a few words)
    if (dev >= 0 && dev < 64) cached[dev] = bytes;
    return (size_t)bytes;
}

AttendWs attend_layout(void *ws, int32_t d, int32_t G, int64_t N, int32_t key_bytes, int32_t B,
                       int32_t c, int32_t k, size_t *bytes) {
    AttendWs w{};
    Carve cv(ws);
    const int64_t bc = (int64_t)B * c;
    w.p_cap = 4 * bc;
    w.w_max = N / kChunkFloor + G + 1;
    // a cluster of nch chunks forms at most nch / 2 + 1 level-one groups
    // (groups of at least two partials, only when nch >= 2)
    w.kp = next_pow2(k);
    w.g_max = w.w_max / 2 + G + 1;
    w.u_cap = w.p_cap / 2 + bc;
    w.cnt = cv.take<int32_t>(G);
    w.qoff = cv.take<int32_t>(G + 1);
    w.wstart = cv.take<int32_t>(G + 1);
    w.wlast = cv.take<int32_t>(G);
    w.gstart = cv.take<int32_t>(G + 1);
    w.pbase = cv.take<int64_t>(G);
    w.ubase = cv.take<int64_t>(G);
    w.mstart = cv.take<int32_t>(G + 1);
    w.mlist = cv.take<MergeSlot>(bc);
    w.units = cv.take<int2>(w.u_cap);
    w.qlist = cv.take<int32_t>(bc);
    w.pos = cv.take<int32_t>(bc);
    w.bound = cv.take<uint64_t>(bc);
    w.plan = cv.take<Plan>(1);
    w.rbits = cv.take<uint32_t>(kCountBlocks * kWave);
    w.ragg = cv.take<int64_t>(kRouteBlocks * kAgg);
    w.items = cv.take<WorkItem>(w.w_max);
    w.groups = cv.take<MergeGroup>(w.g_max);
    w.pm = cv.take<float>(w.p_cap);
    w.pz = cv.take<float>(w.p_cap);
    w.pc = cv.take<int32_t>(w.p_cap);
    w.pk = cv.take<uint64_t>(w.p_cap * k);
    w.um = cv.take<float>(w.u_cap);
    w.uz = cv.take<float>(w.u_cap);
    w.uc = cv.take<int32_t>(w.u_cap);
    w.uk = cv.take<uint64_t>(w.u_cap * k);
    w.q16 = key_bytes == 4 ? cv.take<__bf16>((int64_t)B * d) : nullptr;
    if (bytes) *bytes = cv.off + 256;
    return w;
}

// Queries per pass actually provisioned: enough for about twice the mean
// number of queries per selected cluster (a cluster with more takes several
// passes), so that small query groups leave room for more blocks per CU.
static int qmax_for_load(int qmax, int64_t bc, int32_t G) {
    const int64_t mean = (bc + G - 1) / (G > 0 ? G : 1);
    int want = (int)(((2 * mean + 15) / 16) * 16);
    if (want < 16) want = 16;
    return want < qmax ? want : qmax;
}

namespace {
// fp32 queries rounded to bf16 (to nearest even, as the LDS staging rounds
// them), 8 elements per thread.
__global__ void queries_to_bf16(const float *__restrict__ q, __bf16 *__restrict__ y, int64_t n8) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n8;
         i += (int64_t)gridDim.x * blockDim.x)
        reinterpret_cast<bf16x8_t *>(y)[i] = load8(q + i * 8);
}
}  // namespace

// The streaming kernel and its launch shape for one call (nothing launched).
struct StreamChoice {
    StreamLaunch l;
    int npl;
    bool lds;          // an LDS-staged kernel (else the generic one)
    bool two;          // two blocks per CU
    bool q16;          // the split kernel with fp32 keys: stages a bf16 copy of the queries
};

static StreamChoice choose_stream(int32_t key_dtype, int32_t compute_dtype, const FineArgs &fa0,
                                  int64_t bc, int64_t n_rows, int n_cu, int64_t w_max,
                                  KernelEvents ev, hipStream_t s) {
    const size_t budget = lds_budget();
    StreamChoice c{};
    c.npl = fa0.cap / kWave;
    const int npl = c.npl;
    StreamLaunch &l = c.l;
    l.fa = fa0;
    l.ev = ev;
    l.stream = s;
    l.n_cu = n_cu > 0 ? n_cu : 1;
    l.max_grid = w_max;
    // The LDS-staged kernels need bf16 arithmetic and d % 256 == 0 (one block
    // per CU with bf16 storage reads longer units: d % 512 == 0 there).
    int ql = (compute_dtype == kBF16 && fa0.d % 256 == 0) ? qmax_lds(fa0.d, fa0.cap, budget) : 0;
    if (ql > 0) {
        ql = qmax_for_load(ql, bc, fa0.G);
        l.fa.qmax = ql;
        l.qs_bytes = (int32_t)fine_qs_bytes(fa0.d, ql);
        // two score tiles (one barrier per step) when they fit
        l.fa.ntile = l.qs_bytes + fine_state_bytes(ql, fa0.cap, 2) <= budget ? 2 : 1;
        l.smem = l.qs_bytes + fine_state_bytes(ql, fa0.cap, l.fa.ntile);
        // two blocks per CU when two blocks' LDS fits (and the buffers leave the registers)
        const bool two = npl <= 4 && 2 * (l.smem + 256) <= budget + 256;
        // two blocks per CU with half of d's query fragments staged at a time
        // (one query tile per pass: when the load needs no more), so that one
        // block's staging, epilogues and pass ends overlap the other's loads;
        // for short segments (at most two four-step row groups on average:
        // the queries are staged again for every group)
        if (!two && ql == 16 && npl <= 4 && fa0.d % (key_dtype == kF32 ? 256 : 512) == 0 &&
            n_rows <= (int64_t)fa0.G * 2 * kSplitSteps * kRowsPerStep) {
            const int32_t qs_half = (int32_t)fine_qs_bytes(fa0.d / 2, 16);
            const size_t sm2 = qs_half + fine_state_bytes(16, fa0.cap, 2);
            if (2 * (sm2 + 256) <= budget + 256) {
                // every half of every row group stages its queries: with fp32
                // keys from a bf16 copy, half the bytes and one round trip
                c.q16 = key_dtype == kF32;
                l.ksplit = true;
                l.fa.ntile = 2;
                l.qs_bytes = qs_half;
                l.smem = sm2;
                c.lds = true;
                return c;
            }
        }
        // one block per CU: producer/consumer blocks (their load units are
        // 8 k-steps for bf16 keys, 4 for fp32: d % 256 or d % 128)
        l.producer_consumer = !two && npl <= 4;
        const int unit_k = key_dtype == kF32 ? 8 : 16;
        if (two || l.producer_consumer || fa0.d % (32 * unit_k) == 0) {
            c.lds = true;
            c.two = two;
            return c;
        }
    }
    l.fa.qmax = qmax_generic(fa0.cap);
    l.fa.ntile = 2;
    l.qs_bytes = 0;
    l.smem = fine_state_bytes(l.fa.qmax, fa0.cap, 2);
    return c;
}

static hipError_t launch_stream(int32_t key_dtype, int32_t compute_dtype, const StreamChoice &c) {
    if (c.lds)
        return key_dtype == kF32 ? launch_stream_lds_f32(c.npl, c.two, c.l)
                                 : launch_stream_lds_bf16(c.npl, c.two, c.l);
    return launch_stream_generic(key_dtype, compute_dtype, c.npl, c.l);
}

// Merge grids: enough resident waves to cover the GPU several times over, or
// fewer when the bound on the work is smaller; the kernels loop over the rest.
static unsigned merge_grid(int64_t bound, int n_cu) {
    int64_t b = (bound + kMergeWaves - 1) / kMergeWaves;
    const int64_t cap = (int64_t)(n_cu > 0 ? n_cu : 1) * 16;
    if (b > cap) b = cap;
    return (unsigned)(b < 1 ? 1 : b);
}

template <int NPL>
static hipError_t launch_merge(const MergeArgs &ma, int64_t u_cap, bool groups, int n_cu,
                               hipStream_t s) {
    const size_t smem = (size_t)kMergeWaves * NPL * kWave * 8;
    const dim3 block(kWave * kMergeWaves);
    if (groups) {
        hipLaunchKernelGGL(group_merge<NPL>, dim3(merge_grid(u_cap, n_cu)), block, smem, s, ma);
        hipLaunchKernelGGL(slot_merge<NPL>, dim3(merge_grid(ma.n_pairs, n_cu)), block, smem, s, ma);
    } else {
        // one level only: the waves of a block share each pair
        hipLaunchKernelGGL(slot_merge_shared<NPL>, dim3(merge_grid(ma.n_pairs, n_cu)), block, smem,
                           s, ma);
    }
    return hipGetLastError();
}

hipError_t launch_attend(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G, int64_t N,
                         const void *fine_keys, const void *fine_keys_tiled,
                         const int64_t *seg_offsets,
                         const int32_t *transition_id, const void *q, int32_t B,
                         const int32_t *sel, int32_t c, float tau, int32_t k, float *slot_max,
                         float *slot_sum, float *cand_score, int32_t *cand_id, const AttendWs &w,
                         int n_cu, KernelEvents ev, hipStream_t s) {
    const int64_t bc = (int64_t)B * c;
    const float cexp = 1.4426950408889634f / tau;
    PlanArgs pa{};
    pa.G = G;
    pa.n_rows = N;
    pa.off = seg_offsets;
    pa.toff = static_cast<const int64_t *>(fine_keys_tiled);   // its header, or NULL
    pa.qoff = w.qoff;
    pa.wstart = w.wstart;
    pa.wlast = w.wlast;
    pa.gstart = w.gstart;
    pa.mstart = w.mstart;
    pa.pbase = w.pbase;
    pa.ubase = w.ubase;
    pa.plan = w.plan;
    pa.chunk_min = chunk_floor_rows(N, n_cu);
    pa.p_cap = w.p_cap;
    pa.kp = w.kp;
    // One merge level everywhere, and no level-one launch, when up to
    // kMergeDirectSmall requests cover even a segment of all N rows cut at
    // the shortest chunk the planner may choose (small banks); else level one
    // above kMergeDirect requests, where longer one-level chains would set
    // the merge kernel's length.
    const int64_t nch_max = (N + pa.chunk_min - 1) / pa.chunk_min;
    const int64_t req = (int64_t)kMergeBatch * kWave;
    const bool groups = group_span(nch_max, pa.kp, kMergeDirectSmall * req) > 0;
    pa.direct = (groups ? kMergeDirect : kMergeDirectSmall) * req;
    const SlotOut so{slot_max, slot_sum, cand_score, cand_id, k};
    FineArgs fa{};
    fa.keys = fine_keys;
    if (fine_keys_tiled) {          // the header of segment starts, then the tiles
        fa.toff = static_cast<const int64_t *>(fine_keys_tiled);
        fa.keys_tiled = static_cast<const char *>(fine_keys_tiled) + tile_header_bytes(G);
        fa.seg_off = seg_offsets;
    }
    fa.tid = transition_id;
    // without ids the id loads read the key array (at least N ints) and are ignored
    fa.tid_src = transition_id ? transition_id : static_cast<const int32_t *>(fine_keys);
    fa.q = q;
    fa.d = d;
    fa.c = c;
    fa.G = G;
    fa.k = k;
    fa.cap = fine_cap(k);
    fa.cexp = cexp;
    fa.qlist = w.qlist;
    fa.bound = w.bound;
    fa.items = w.items;
    fa.plan = w.plan;
    fa.pm = w.pm;
    fa.pz = w.pz;
    fa.pc = w.pc;
    fa.pk = w.pk;
    fa.slot_max = slot_max;
    fa.slot_sum = slot_sum;
    fa.cand_score = cand_score;
    fa.cand_id = cand_id;
    StreamChoice sc = choose_stream(key_dtype, compute_dtype, fa, bc, N, n_cu, w.w_max, ev, s);
    const int64_t n8 = sc.q16 ? (int64_t)B * d / 8 : 0;
    if (sc.q16) sc.l.fa.q16 = w.q16;

    const size_t route_lds = route_fused_lds(G, bc);
    static_assert((3 * (size_t)kNoCluster + 1) * 8 > kRouteLdsBytes, "fused routing keeps cluster ids in 16 bits");
    if (bc <= kFusedRoutePairs && route_lds <= kRouteLdsBytes) {
        hipError_t e0 = hipFuncSetAttribute((const void *)route_fused,
                                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)route_lds);
        if (e0 != hipSuccess) return e0;
        hipLaunchKernelGGL(route_fused, dim3(1), dim3(kPlanThreads), route_lds, s, pa, sel, bc,
                           w.qlist, w.pos, w.bound, so, w.items, w.groups, w.units, w.mlist);
        if (sc.q16) {
            const int64_t nb = (n8 + 255) / 256;
            hipLaunchKernelGGL(queries_to_bf16, dim3((unsigned)(nb < 8192 ? nb : 8192)), dim3(256),
                               0, s, static_cast<const float *>(q), w.q16, n8);
        }
    } else {
        // zero the counters, count the pairs, plan per block of clusters, then
        // emit the lists and tables pair by pair; each launch also copies a
        // quarter of the queries to bf16 on blocks past its routing grid
        QCopy qc[4];
        unsigned ncopy[4];
        for (int j = 0; j < 4; ++j) {
            qc[j] = QCopy{static_cast<const float *>(q), w.q16, n8 * j / 4, n8 * (j + 1) / 4};
            const int64_t nb = (qc[j].end - qc[j].begin + 1023) / 1024;   // 4 groups per thread
            ncopy[j] = (unsigned)(nb < 2048 ? nb : 2048);
        }
        const int64_t nz = ((int64_t)G + 255) / 256;
        hipLaunchKernelGGL(route_zero, dim3((unsigned)(nz < 1024 ? nz : 1024) + ncopy[0]), dim3(256), 0,
                           s, G, w.cnt, w.plan, qc[0]);
        const int64_t nb2 = (bc + kCountThreads - 1) / kCountThreads;
        const int32_t nc2 = (int32_t)(nb2 < kCountBlocks ? nb2 : kCountBlocks);
        const int lmin = 63 - __builtin_clzll((unsigned long long)pa.chunk_min);
        // the copy blocks of the counting kernel are 1024 threads too: a
        // quarter as many
        hipLaunchKernelGGL(route_count, dim3((unsigned)nc2 + (ncopy[1] + 3) / 4), dim3(kCountThreads), 0,
                           s, sel, bc, G, seg_offsets, lmin, w.cnt, w.pos, w.plan, w.rbits, nc2, qc[1]);
        const int32_t rounds = (int32_t)(((int64_t)G + kRouteBlocks * kRouteThreads - 1) /
                                         ((int64_t)kRouteBlocks * kRouteThreads));
        const int32_t per_block = rounds * kRouteThreads;
        const int32_t nb3 = (int32_t)(((int64_t)G + per_block - 1) / per_block);
        hipLaunchKernelGGL(route_plan, dim3((unsigned)nb3 + ncopy[2]), dim3(kRouteThreads), 0, s, pa,
                           w.cnt, w.rbits, nc2, rounds, w.ragg, nb3, qc[2]);
        const int64_t nb4 = (bc + kRouteThreads - 1) / kRouteThreads;
        hipLaunchKernelGGL(route_emit, dim3((unsigned)nb4 + ncopy[3]), dim3(kRouteThreads), 0, s, pa,
                           sel, bc, w.cnt, w.pos, w.ragg, nb3, per_block, w.qlist, w.bound, so,
                           w.items, w.groups, w.units, w.mlist, (int32_t)nb4, qc[3]);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    err = launch_stream(key_dtype, compute_dtype, sc);
    if (err != hipSuccess) return err;

    MergeArgs ma{};
    ma.plan = w.plan;
    ma.groups = w.groups;
    ma.units = w.units;
    ma.mlist = w.mlist;
    ma.bound = w.bound;
    ma.pm = w.pm;
    ma.pz = w.pz;
    ma.pc = w.pc;
    ma.pk = w.pk;
    ma.um = w.um;
    ma.uz = w.uz;
    ma.uc = w.uc;
    ma.uk = w.uk;
    ma.n_pairs = bc;
    ma.k = k;
    ma.cexp = cexp;
    ma.slot_max = slot_max;
    ma.slot_sum = slot_sum;
    ma.cand_score = cand_score;
    ma.cand_id = cand_id;
    // k >= 48: 256-key buffers (a 128-key one has at most 80 free slots
    // after each compaction; zipf_large_bf16, k = 64: merges 89 -> 56 us)
    switch (next_pow2(k + kWave) / kWave) {
        case 2: return k >= 48 ? launch_merge<4>(ma, w.u_cap, groups, n_cu, s)
                               : launch_merge<2>(ma, w.u_cap, groups, n_cu, s);
        case 4: return launch_merge<4>(ma, w.u_cap, groups, n_cu, s);
        default: return launch_merge<8>(ma, w.u_cap, groups, n_cu, s);
    }
}

}  // namespace htam
