// Prefix-aware coarse scoring on gfx950 (Sec. 4.3, Eq. score with the
// position-aware weights of Eq. prefix_weight; App. A.1, App. B.2). The score
// of global direction g for query b, whose recent directions are the prefix
// p_b = (g_1, ..., g_L), is
//     score_b(g) = sum_{i=1..L} alpha_i <q_b, E[g_i][g]>,  alpha_i = exp(-lambda (L - i)),
// read through the edge memories E[g_i][g] (the state-conditioned transition
// utility phi of App. B.6 as an inner product with an edge key); a query with
// an empty prefix (the first step, which reads no edge) is scored by the node
// keys, <q_b, c_g>.
//
// Each (query, prefix position) pair needs one row q_b E[g_i]^T over all G
// destinations, and every pair with the same source node g_i shares the edge
// slice E[g_i] ([G][d]). So the pairs are grouped by source (count, scan,
// scatter), and a grouped MFMA GEMM multiplies each group of up to 32 pairs'
// queries by its source's slice, 32 x 32 tiles per wave, every slice read once
// per group. The per-pair rows are then combined with the alpha weights in
// prefix order (fixed order, no atomics: the result does not depend on how
// the pairs were grouped), over the node scores of the queries with a
// prefix; the top-c selection is the coarse stage's.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int kGroup = 32;          // pairs per GEMM group (one 32 x 32 tile per wave)
constexpr int kScanThreads = 1024;

// Length of query b's prefix: entries up to the first outside [0, G).
__device__ __forceinline__ int prefix_len(const int32_t *row, int32_t lmax, int32_t G) {
    int L = 0;
    while (L < lmax && row[L] >= 0 && row[L] < G) ++L;
    return L;
}

__global__ void prefix_zero(int32_t G, int32_t *cnt, int32_t *cursor, int32_t *n_groups) {
    for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < G;
         g += (int64_t)gridDim.x * blockDim.x) {
        cnt[g] = 0;
        cursor[g] = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) *n_groups = 0;
}

// Pairs (b, i) with i < L_b, counted (scatter = false) or placed in their
// source's list (scatter = true).
template <bool kScatter>
__global__ void prefix_route(const int32_t *prefix, int32_t B, int32_t lmax, int32_t G,
                             int32_t *cnt, int32_t *cursor, const int32_t *off, int32_t *pairs) {
    const int64_t n = (int64_t)B * lmax;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = e / lmax;
        const int i = (int)(e - b * lmax);
        if (i >= prefix_len(prefix + b * lmax, i + 1, G)) continue;
        const int32_t src = prefix[e];
        if (kScatter) pairs[off[src] + atomicAdd(&cursor[src], 1)] = (int32_t)e;
        else atomicAdd(&cnt[src], 1);
    }
}

// Exclusive scans of the pair counts (-> off) and of the group counts
// (-> goff), one block; the number of groups to n_groups.
__global__ __launch_bounds__(kScanThreads) void prefix_scan(const int32_t *cnt, int32_t G,
                                                            int32_t *off, int32_t *goff,
                                                            int32_t *n_groups) {
    __shared__ int64_t s[2][kScanThreads];
    const int t = threadIdx.x;
    const int32_t per = (G + kScanThreads - 1) / kScanThreads;
    const int32_t g0 = min(G, t * per), g1 = min(G, g0 + per);
    int64_t a = 0, c = 0;
    for (int32_t g = g0; g < g1; ++g) {
        a += cnt[g];
        c += (cnt[g] + kGroup - 1) / kGroup;
    }
    s[0][t] = a;
    s[1][t] = c;
    __syncthreads();
    for (int o = 1; o < kScanThreads; o <<= 1) {
        const int64_t xa = t >= o ? s[0][t - o] : 0, xc = t >= o ? s[1][t - o] : 0;
        __syncthreads();
        s[0][t] += xa;
        s[1][t] += xc;
        __syncthreads();
    }
    int64_t ra = s[0][t] - a, rc = s[1][t] - c;
    for (int32_t g = g0; g < g1; ++g) {
        off[g] = (int32_t)ra;
        goff[g] = (int32_t)rc;
        ra += cnt[g];
        rc += (cnt[g] + kGroup - 1) / kGroup;
    }
    if (t == kScanThreads - 1) {
        off[G] = (int32_t)s[0][t];
        goff[G] = (int32_t)s[1][t];
        *n_groups = (int32_t)s[1][t];
    }
}

__global__ void prefix_groups(int32_t G, const int32_t *cnt, const int32_t *off,
                              const int32_t *goff, int4 *groups) {
    for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < G;
         g += (int64_t)gridDim.x * blockDim.x) {
        for (int32_t j = 0; j * kGroup < cnt[g]; ++j)
            groups[goff[g] + j] = make_int4((int32_t)g, off[g] + j * kGroup,
                                            min(kGroup, cnt[g] - j * kGroup), 0);
    }
}

// One wave per (32 destinations, group of up to 32 pairs of one source):
// part[pair][g] = <q_b, E[src][g]> for the group's pairs. bf16 arithmetic on
// v_mfma_f32_16x16x32_bf16 (fp32 storage rounded as it is loaded), or fp32 on
// v_mfma_f32_16x16x4f32. Operands are read directly in MFMA fragment layout,
// a batch of k-steps requested before any is used; rows past the group or
// past G are clamped and not written.
template <typename T, bool kF32Math>
__global__ __launch_bounds__(kWave) void prefix_gemm(const T *__restrict__ q,
                                                     const T *__restrict__ E,
                                                     const int32_t *__restrict__ pairs,
                                                     const int4 *__restrict__ groups,
                                                     const int32_t *__restrict__ n_groups,
                                                     int32_t G, int32_t d, int32_t lmax,
                                                     float *__restrict__ part) {
    const int lane = threadIdx.x & 63, r16 = lane & 15, kg = lane >> 4;
    const int64_t g0 = (int64_t)blockIdx.x * 32;
    const int32_t ng = *n_groups;
    for (int32_t gi = blockIdx.y; gi < ng; gi += gridDim.y) {
        const int4 grp = groups[gi];
        const int32_t src = grp.x, first = grp.y, np = grp.z;
        const T *ap[2], *bp[2];
        int32_t pe[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            pe[i] = pairs[first + min(16 * i + r16, np - 1)];
            ap[i] = q + (int64_t)(pe[i] / lmax) * d;
            bp[i] = E + ((int64_t)src * G + min(g0 + 16 * i + r16, (int64_t)G - 1)) * d;
        }
        f32x4_t acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if constexpr (kF32Math) {
            for (int k0 = 0; k0 < d; k0 += 4) {
                const int k = k0 + kg;
                float a[2], b[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    a[i] = (float)ap[i][k];
                    b[i] = (float)bp[i][k];
                }
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
            }
        } else {
            constexpr int kSteps = sizeof(T) == 4 ? 4 : 8;
            const int nks = (d + 31) / 32;
            for (int s0 = 0; s0 < nks; s0 += kSteps) {
                RawFrag<T> fa[kSteps][2], fb[kSteps][2];
#pragma unroll
                for (int st = 0; st < kSteps; ++st) {
                    const int k = min(32 * (s0 + st) + 8 * kg, d - 8);
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        fa[st][i].load(ap[i] + k);
                        fb[st][i].load(bp[i] + k);
                    }
                }
#pragma unroll
                for (int st = 0; st < kSteps; ++st) {
                    const bool ok = 32 * (s0 + st) + 8 * kg < d;
                    bf16x8_t a[2], b[2];
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        a[i] = ok ? fa[st][i].get() : zero8();
                        b[i] = ok ? fb[st][i].get() : zero8();
                    }
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j],
                                                                                0, 0, 0);
                }
            }
        }
        // lane (r16, kg) holds rows 4 kg + e (pairs) of column r16 (destinations)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 16 * i + 4 * kg + e;
                if (r >= np) continue;
                const int64_t pair = pairs[first + r];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int64_t g = g0 + 16 * j + r16;
                    if (g < G) part[pair * G + g] = acc[i][j][e];
                }
            }
    }
}

// score_b(g) = sum_i alpha_i part[(b, i)][g] over the prefix, in prefix
// order; queries with an empty prefix keep their node score.
__global__ void prefix_combine(const int32_t *prefix, int32_t B, int32_t lmax, int32_t G,
                               float lambda, const float *part, float *S) {
    for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < (int64_t)B * G;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = x / G, g = x - b * G;
        const int L = prefix_len(prefix + b * lmax, lmax, G);
        if (L == 0) continue;
        float acc = 0.0f;
        for (int i = 0; i < L; ++i)
            acc += expf(-lambda * (float)(L - 1 - i)) * part[(b * lmax + i) * G + g];
        S[x] = acc;
    }
}

}  // namespace

PrefixWs prefix_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                       int32_t compute_dtype, int32_t lmax, int32_t top_c, size_t *bytes) {
    PrefixWs w{};
    size_t cb = 0;
    w.c = coarse_layout(ws, B, G, d, key_dtype, compute_dtype, top_c, &cb);
    Carve cv(ws ? static_cast<char *>(ws) + cb : nullptr);
    const int64_t np = (int64_t)B * lmax;
    w.g_max = (np + kGroup - 1) / kGroup + G;
    w.part = cv.take<float>((size_t)np * G);
    w.cnt = cv.take<int32_t>(G);
    w.cursor = cv.take<int32_t>(G);
    w.off = cv.take<int32_t>(G + 1);
    w.goff = cv.take<int32_t>(G + 1);
    w.pairs = cv.take<int32_t>(np);
    w.groups = cv.take<int4>(w.g_max);
    w.n_groups = cv.take<int32_t>(1);
    if (bytes) *bytes = cb + cv.off + 256;
    return w;
}

hipError_t launch_prefix(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         const void *coarse_keys, const void *edge_keys, const int32_t *prefix,
                         int32_t lmax, float lambda, const void *q, int32_t B, int32_t top_c,
                         int32_t *sel, float *sel_score, const PrefixWs &w, int n_cu,
                         KernelEvents ev, hipStream_t s) {
    // node scores of every query (kept for the queries with an empty prefix)
    hipError_t err = launch_scores(key_dtype, compute_dtype, d, G, coarse_keys, q, B, w.c.scores,
                                   w.c.q16, w.c.c16, true, n_cu, KernelEvents{}, s);
    if (err != hipSuccess) return err;
    const int64_t np = (int64_t)B * lmax;
    const unsigned gb = (unsigned)((G + 255) / 256 < 1024 ? (G + 255) / 256 : 1024);
    const unsigned pb = (unsigned)((np + 255) / 256 < 4096 ? (np + 255) / 256 : 4096);
    hipLaunchKernelGGL(prefix_zero, dim3(gb), dim3(256), 0, s, G, w.cnt, w.cursor, w.n_groups);
    hipLaunchKernelGGL(prefix_route<false>, dim3(pb), dim3(256), 0, s, prefix, B, lmax, G, w.cnt,
                       w.cursor, w.off, w.pairs);
    hipLaunchKernelGGL(prefix_scan, dim3(1), dim3(kScanThreads), 0, s, w.cnt, G, w.off, w.goff,
                       w.n_groups);
    hipLaunchKernelGGL(prefix_route<true>, dim3(pb), dim3(256), 0, s, prefix, B, lmax, G, w.cnt,
                       w.cursor, w.off, w.pairs);
    hipLaunchKernelGGL(prefix_groups, dim3(gb), dim3(256), 0, s, G, w.cnt, w.off, w.goff,
                       w.groups);
    const dim3 grid((unsigned)((G + 31) / 32), (unsigned)(w.g_max < 4096 ? w.g_max : 4096));
    if (compute_dtype == kF32)
        launch_timed(prefix_gemm<float, true>, grid, dim3(kWave), 0, s, ev,
                     static_cast<const float *>(q), static_cast<const float *>(edge_keys), w.pairs,
                     w.groups, w.n_groups, G, d, lmax, w.part);
    else if (key_dtype == kF32)
        launch_timed(prefix_gemm<float, false>, grid, dim3(kWave), 0, s, ev,
                     static_cast<const float *>(q), static_cast<const float *>(edge_keys), w.pairs,
                     w.groups, w.n_groups, G, d, lmax, w.part);
    else
        launch_timed(prefix_gemm<__bf16, false>, grid, dim3(kWave), 0, s, ev,
                     static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(edge_keys),
                     w.pairs, w.groups, w.n_groups, G, d, lmax, w.part);
    const int64_t nc = (int64_t)B * G;
    hipLaunchKernelGGL(prefix_combine, dim3((unsigned)((nc + 255) / 256 < 8192 ? (nc + 255) / 256 : 8192)),
                       dim3(256), 0, s, prefix, B, lmax, G, lambda, w.part, w.c.scores);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    return launch_select(B, G, top_c, sel, sel_score, w.c, s);
}

}  // namespace htam
