// Online memory update on gfx950, record side (Eq. memory_update: the memory
// grows by each step's new transition record under its parent direction; Alg.
// 1, Step 4). Records are appended log-structured: new records are built into
// a small delta bank (htam_memory_build), retrieval reads the main and the
// delta bank and merges their per-slot lists, and this compaction folds the
// delta into the main bank. The result is the bank that htam_memory_build
// would make from the main bank's records followed by the delta's: segment by
// segment, the main bank's rows, then the delta's, each in their order.
//
// With both banks' offsets a partition of their rows, the destination of a
// row has a closed form: main row i of cluster g goes to i + off_delta[g]
// (the delta rows of clusters before g come first), delta row j of cluster g
// to j + off_main[g + 1] (all main rows of clusters up to g come first). One
// wave takes 64 rows: each lane finds its row's cluster by binary search over
// the offsets, then the wave copies the rows with 16-byte accesses.
//
// Statistics side (the node, edge and edge-bucket feedback the update
// refreshes, and the rule-based scorer that reads them) further down.
#include "../../include/htam.h"
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

// Both offset arrays must partition their banks' rows (off[0] = 0,
// nondecreasing, off[G] = rows); *bad = 1 otherwise. One block.
__global__ void merge_check(const int64_t *off_a, int64_t n_a, const int64_t *off_b, int64_t n_b,
                            int32_t G, int32_t *bad) {
    int b = 0;
    for (int32_t g = threadIdx.x; g < G; g += blockDim.x)
        b |= off_a[g] > off_a[g + 1] || off_b[g] > off_b[g + 1];
    if (threadIdx.x == 0) b |= off_a[0] != 0 || off_a[G] != n_a || off_b[0] != 0 || off_b[G] != n_b;
    b = __syncthreads_or(b);
    if (threadIdx.x == 0) *bad = b;
}

__global__ void merge_offsets(const int64_t *off_a, const int64_t *off_b, int32_t G,
                              const int32_t *bad, int64_t *off_out) {
    if (*bad) return;
    for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g <= G;
         g += (int64_t)gridDim.x * blockDim.x)
        off_out[g] = off_a[g] + off_b[g];
}

// Rows of one source bank to their merged positions: row r of cluster g goes
// to r + shift[g + step] (step 0: the main bank, shift = delta offsets;
// step 1: the delta bank, shift = main offsets).
typedef unsigned int ucopy_t __attribute__((ext_vector_type(4)));
constexpr int kCopyPer = 16;

__global__ __launch_bounds__(256) void merge_rows(const uint4 *__restrict__ keys,
                                                  const int32_t *__restrict__ ids,
                                                  const int64_t *__restrict__ off, int64_t n,
                                                  const int64_t *__restrict__ shift, int32_t step,
                                                  int32_t G, int32_t vpr, const int32_t *bad,
                                                  uint4 *__restrict__ keys_out,
                                                  int32_t *__restrict__ ids_out) {
    if (*bad) return;
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t r0 = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * kWave; r0 < n;
         r0 += waves * kWave) {
        const int64_t r = r0 + lane;
        int64_t dst = 0;
        if (r < n) {
            int32_t lo = 0, hi = G;                 // off[lo] <= r < off[hi]
            while (hi - lo > 1) {
                const int32_t mid = (lo + hi) >> 1;
                if (off[mid] <= r) lo = mid; else hi = mid;
            }
            dst = r + shift[lo + step];
            ids_out[dst] = ids[r];
        }
        // the wave's rows as one run of 16-byte elements, 16 per lane in
        // flight (element e: row e / vpr, its destination row from the lane
        // that holds it), with non-temporal loads and stores: each byte is
        // moved once (mixture_bf16's bank and delta: 4.46 -> 4.94 TB/s,
        // against one row at a time with ordinary loads)
        const int rows = (int)min((int64_t)kWave, n - r0);
        const int32_t total = rows * vpr;
        for (int32_t e0 = 0; e0 < total; e0 += kCopyPer * kWave) {
            ucopy_t x[kCopyPer];
            int64_t to[kCopyPer];
#pragma unroll
            for (int j = 0; j < kCopyPer; ++j) {
                const int32_t e = e0 + j * kWave + lane;
                const uint32_t ec = (uint32_t)(e < total ? e : total - 1);
                const uint32_t i = ec / (uint32_t)vpr, v = ec - i * (uint32_t)vpr;
                x[j] = __builtin_nontemporal_load(
                    reinterpret_cast<const ucopy_t *>(keys + (r0 + i) * vpr + v));
                to[j] = __shfl(dst, (int)i) * vpr + v;
            }
#pragma unroll
            for (int j = 0; j < kCopyPer; ++j)
                if (e0 + j * kWave + lane < total)
                    __builtin_nontemporal_store(x[j], reinterpret_cast<ucopy_t *>(keys_out + to[j]));
        }
    }
}

// ---------------------------------------------------------------------------
// statistics side: rule-based aggregation of step outcomes (Eq. memory_update
// refreshes the node statistics of V_G(g_t) and the edge feedback of
// E_G(g_{t-1}, g_t); App. B.6 reads them as the features z of phi = w^T z)
// ---------------------------------------------------------------------------
constexpr int kFeat = HTAM_FEEDBACK_FEATURES;
constexpr int kWords = HTAM_STATS_WORDS;
constexpr double kFixedOne = 16777216.0;   // 2^24

// One thread per (event, word): word 0 counts the observation, word 1 + f adds
// feature f in fixed point (x * 2^24 rounded to nearest even). int64 additions
// are exact and commute, so the statistics do not depend on event order.
__global__ void feedback_update(int32_t G, int32_t NB, int32_t n, const int32_t *src,
                                const int32_t *dst, const int32_t *bucket, const float *feat,
                                unsigned long long *node, unsigned long long *edge,
                                unsigned long long *edge_bucket) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < (int64_t)n * kWords;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = x / kWords;
        const int wd = (int)(x - e * kWords);
        const int32_t s = src[e], d = dst[e], k = bucket[e];
        if (d < 0 || d >= G || k < 0 || k >= NB || s >= G) continue;
        const long long v = wd == 0 ? 1LL : llrint((double)feat[e * kFeat + wd - 1] * kFixedOne);
        const unsigned long long u = (unsigned long long)v;
        atomicAdd(node + (int64_t)d * kWords + wd, u);
        if (s >= 0) {
            atomicAdd(edge + ((int64_t)s * G + d) * kWords + wd, u);
            atomicAdd(edge_bucket + (((int64_t)s * G + d) * NB + k) * kWords + wd, u);
        }
    }
}

// w^T z of one statistics record (z: means over its observations, the h_ctx
// flag in position 7, the four risk features negated; no observation: 0).
__device__ __forceinline__ double stats_utility(const long long *st, double h, const float *w) {
    const long long n = st[0];
    if (n == 0) return 0.0;
    const double inv = 1.0 / ((double)n * kFixedOne);
    double acc = 0.0;
#pragma unroll
    for (int f = 0; f < kFeat; ++f) {
        const double m = (double)st[1 + f] * inv;
        acc += (double)w[f < 7 ? f : f + 1] * (f < 7 ? m : -m);
    }
    return acc + (double)w[7] * h;
}

// score_b(g) = sum_i alpha_i phi(g_i -> g | bucket_b) over b's prefix, phi
// from the bucket's statistics when it has at least min_count observations
// (h = 1), else from the edge's (h = 0); an empty prefix scores the node
// statistics of g (h = 0). One thread per (query, direction); double inside.
__global__ void transition_scores(int32_t G, int32_t NB, int32_t B, const int32_t *prefix,
                                  int32_t lmax, const int32_t *bucket, float lambda,
                                  const float *w, int32_t min_count, const long long *node,
                                  const long long *edge, const long long *edge_bucket,
                                  float *scores) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < (int64_t)B * G;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = x / G, g = x - b * G;
        const int32_t *row = prefix + b * lmax;
        int L = 0;
        while (L < lmax && row[L] >= 0 && row[L] < G) ++L;
        double acc;
        if (L == 0) {
            acc = stats_utility(node + g * kWords, 0.0, w);
        } else {
            const int32_t k = min(max(bucket[b], 0), NB - 1);
            acc = 0.0;
            for (int i = 0; i < L; ++i) {
                const int64_t eg = (int64_t)row[i] * G + g;
                const long long *eb = edge_bucket + (eg * NB + k) * kWords;
                const double phi = (eb[0] > 0 && eb[0] >= min_count)
                                       ? stats_utility(eb, 1.0, w)
                                       : stats_utility(edge + eg * kWords, 0.0, w);
                acc += exp(-(double)lambda * (double)(L - 1 - i)) * phi;
            }
        }
        scores[x] = (float)acc;
    }
}

}  // namespace

hipError_t launch_feedback_update(int32_t G, int32_t NB, int32_t n, const int32_t *src,
                                  const int32_t *dst, const int32_t *bucket, const float *feat,
                                  int64_t *node, int64_t *edge, int64_t *edge_bucket,
                                  hipStream_t s) {
    if (n == 0) return hipSuccess;
    const int64_t t = (int64_t)n * kWords;
    hipLaunchKernelGGL(feedback_update, dim3((unsigned)((t + 255) / 256 < 8192 ? (t + 255) / 256 : 8192)),
                       dim3(256), 0, s, G, NB, n, src, dst, bucket, feat,
                       reinterpret_cast<unsigned long long *>(node),
                       reinterpret_cast<unsigned long long *>(edge),
                       reinterpret_cast<unsigned long long *>(edge_bucket));
    return hipGetLastError();
}

hipError_t launch_transition_scores(int32_t G, int32_t NB, int32_t B, const int32_t *prefix,
                                    int32_t lmax, const int32_t *bucket, float lambda,
                                    const float *w, int32_t min_count, const int64_t *node,
                                    const int64_t *edge, const int64_t *edge_bucket,
                                    float *scores, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const int64_t t = (int64_t)B * G;
    hipLaunchKernelGGL(transition_scores, dim3((unsigned)((t + 255) / 256 < 8192 ? (t + 255) / 256 : 8192)),
                       dim3(256), 0, s, G, NB, B, prefix, lmax, bucket, lambda, w, min_count,
                       reinterpret_cast<const long long *>(node),
                       reinterpret_cast<const long long *>(edge),
                       reinterpret_cast<const long long *>(edge_bucket), scores);
    return hipGetLastError();
}

hipError_t launch_merge_banks(int32_t G, int32_t row_bytes, const void *keys_a,
                              const int64_t *off_a, const int32_t *id_a, int64_t n_a,
                              const void *keys_b, const int64_t *off_b, const int32_t *id_b,
                              int64_t n_b, void *keys_out, int64_t *off_out, int32_t *id_out,
                              int32_t *bad, hipStream_t s) {
    hipLaunchKernelGGL(merge_check, dim3(1), dim3(1024), 0, s, off_a, n_a, off_b, n_b, G, bad);
    hipLaunchKernelGGL(merge_offsets, dim3((G + 256) / 256 < 1024 ? (G + 256) / 256 : 1024),
                       dim3(256), 0, s, off_a, off_b, G, bad, off_out);
    const int32_t vpr = row_bytes / 16;
    auto grid = [](int64_t n) {
        const int64_t w = (n + kWave - 1) / kWave, b = (w + 3) / 4;
        return (unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192);
    };
    if (n_a > 0)
        hipLaunchKernelGGL(merge_rows, dim3(grid(n_a)), dim3(256), 0, s,
                           static_cast<const uint4 *>(keys_a), id_a, off_a, n_a, off_b, 0, G, vpr,
                           bad, static_cast<uint4 *>(keys_out), id_out);
    if (n_b > 0)
        hipLaunchKernelGGL(merge_rows, dim3(grid(n_b)), dim3(256), 0, s,
                           static_cast<const uint4 *>(keys_b), id_b, off_b, n_b, off_a, 1, G, vpr,
                           bad, static_cast<uint4 *>(keys_out), id_out);
    return hipGetLastError();
}

}  // namespace htam
