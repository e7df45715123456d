// Fine stage of hierarchical retrieval on gfx950: candidates restricted to
// the selected clusters' child segments (Eq. local nodes), each scored by an
// inner product with the query (Eq. local policy), with temperature-softmax
// statistics and the top-k kept per (query, selected cluster).
//
// Kernels, in launch order:
//   route_init / route_count / route_plan / route_scatter
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

namespace htam {

namespace {

constexpr int kFineThreads = 256;      // 4 waves
constexpr int kFineWaves = kFineThreads / kWave;
constexpr int kRowsPerWave = 16;       // one MFMA M-tile of key rows per wave per step
constexpr int kRowsPerStep = kRowsPerWave * kFineWaves;   // rows per block per step
constexpr int kMaxQueryTiles = 4;      // at most 64 queries per pass over a chunk
constexpr int kPlanThreads = 1024;

// ---------------------------------------------------------------------------
// routing
// ---------------------------------------------------------------------------
__global__ void route_init(int32_t G, int32_t *cnt, int32_t *cursor, Plan *plan) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < G;
         i += (int64_t)gridDim.x * blockDim.x) {
        cnt[i] = 0;
        cursor[i] = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        plan->next = 0;
        plan->bad_sel = 0;
    }
}

__global__ void route_count(const int32_t *sel, int64_t n, int32_t G, int32_t *cnt, Plan *plan) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) atomicAdd(&cnt[g], 1);
        else atomicAdd(&plan->bad_sel, 1);
    }
}

// Exclusive scan of one int64 value per thread over a 1024-thread block.
__device__ int64_t block_exclusive_scan(int64_t v, int64_t *s, int64_t *total) {
    const int t = threadIdx.x;
    s[t] = v;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        const int64_t x = t >= off ? s[t - off] : 0;
        __syncthreads();
        s[t] += x;
        __syncthreads();
    }
    const int64_t incl = s[t];
    *total = s[kPlanThreads - 1];
    __syncthreads();
    return incl - v;
}

__device__ int64_t block_sum(int64_t v, int64_t *s) {
    int64_t total;
    block_exclusive_scan(v, s, &total);
    return total;
}

__device__ int64_t block_max(int64_t v, int64_t *s) {
    const int t = threadIdx.x;
    s[t] = v;
    __syncthreads();
    for (int off = kPlanThreads / 2; off > 0; off >>= 1) {
        if (t < off) s[t] = s[t] > s[t + off] ? s[t] : s[t + off];
        __syncthreads();
    }
    const int64_t r = s[0];
    __syncthreads();
    return r;
}

// Single block. qoff = exclusive scan of the per-cluster query counts; the
// chunk length is the smallest power-of-two multiple of chunk_min for which the
// partial results fit in p_cap (it always fits once a chunk spans the longest
// segment, since then each (query, slot) has one partial and p_cap >= B*c).
__global__ __launch_bounds__(kPlanThreads) void route_plan(int32_t G, const int64_t *off,
                                                           const int32_t *cnt, int32_t *qoff,
                                                           int32_t *wstart, int64_t *pbase,
                                                           Plan *plan, int64_t chunk_min,
                                                           int64_t p_cap) {
    __shared__ int64_t s[kPlanThreads];
    const int t = threadIdx.x;
    const int32_t per = (G + kPlanThreads - 1) / kPlanThreads;
    const int32_t g0 = min((int32_t)G, t * per), g1 = min((int32_t)G, g0 + per);

    int64_t local = 0, lmax = 0;
    for (int32_t g = g0; g < g1; ++g) {
        local += cnt[g];
        const int64_t len = off[g + 1] - off[g];
        lmax = len > lmax ? len : lmax;
    }
    int64_t total;
    int64_t run = block_exclusive_scan(local, s, &total);
    for (int32_t g = g0; g < g1; ++g) {
        qoff[g] = (int32_t)run;
        run += cnt[g];
    }
    if (t == kPlanThreads - 1) qoff[G] = (int32_t)total;
    const int64_t maxlen = block_max(lmax, s);

    int64_t ch = chunk_min;
    for (int it = 0; it < 48; ++it) {
        int64_t p = 0;
        for (int32_t g = g0; g < g1; ++g) {
            const int64_t len = off[g + 1] - off[g];
            if (cnt[g] > 0 && len > 0) p += (int64_t)cnt[g] * ((len + ch - 1) / ch);
        }
        const int64_t P = block_sum(p, s);
        if (P <= p_cap || ch >= maxlen) break;
        ch *= 2;
    }

    int64_t wl = 0, pl = 0;
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t len = off[g + 1] - off[g];
        const int64_t nch = (cnt[g] > 0 && len > 0) ? (len + ch - 1) / ch : 0;
        wl += nch;
        pl += nch * cnt[g];
    }
    int64_t wtot, ptot;
    int64_t wrun = block_exclusive_scan(wl, s, &wtot);
    int64_t prun = block_exclusive_scan(pl, s, &ptot);
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t len = off[g + 1] - off[g];
        const int64_t nch = (cnt[g] > 0 && len > 0) ? (len + ch - 1) / ch : 0;
        wstart[g] = (int32_t)wrun;
        pbase[g] = prun;
        wrun += nch;
        prun += nch * cnt[g];
    }
    if (t == kPlanThreads - 1) {
        wstart[G] = (int32_t)wtot;
        plan->chunk = ch;
        plan->n_items = wtot;
        plan->n_parts = ptot;
    }
}

__global__ void route_scatter(const int32_t *sel, int64_t n, int32_t G, const int32_t *qoff,
                              int32_t *cursor, int32_t *qlist, int32_t *pos) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) {
            const int32_t slot = atomicAdd(&cursor[g], 1);
            qlist[qoff[g] + slot] = (int32_t)e;
            pos[e] = slot;
        }
    }
}

// ---------------------------------------------------------------------------
// bank stream
// ---------------------------------------------------------------------------
struct FineArgs {
    const void *keys;
    const int64_t *off;
    const int32_t *tid;
    const void *q;
    int32_t d, c, G, k, cap, qmax;
    float cexp;                   // log2(e) / tau
    const int32_t *qoff, *qlist, *wstart;
    const int64_t *pbase;
    Plan *plan;
    float *pm, *pz;
    int32_t *pc;
    uint64_t *pk;
};

struct FineSmem {
    uint64_t *buf;     // [qmax][cap]
    uint64_t *theta;   // [qmax]
    uint32_t *cnt;     // [qmax]
    int32_t *qrow;     // [qmax]
    float *wm, *wz;    // [waves][qmax]
};

__host__ __device__ inline size_t fine_smem_bytes(int qmax, int cap) {
    return (size_t)qmax * cap * 8 + (size_t)qmax * (8 + 4 + 4) + (size_t)2 * kFineWaves * qmax * 4;
}

// One pass over rows [r0, r1) of a segment for nqg <= 16*NQT queries.
template <typename T, bool BF16, int NQT>
__device__ void fine_pass(const FineArgs &a, const FineSmem &sm, int32_t g, int64_t j, int64_t r0,
                          int64_t r1, int32_t qbeg, int32_t nq, int32_t qg0, int32_t nqg) {
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6, r16 = lane & 15, kg = lane >> 4;
    const int d = a.d, cap = a.cap;
    const T *K = static_cast<const T *>(a.keys);
    const T *Q = static_cast<const T *>(a.q);

    for (int n = t; n < nqg; n += kFineThreads) {
        sm.qrow[n] = a.qlist[qbeg + qg0 + n] / a.c;
        sm.cnt[n] = 0;
        sm.theta[n] = 0;
    }
    __syncthreads();

    const T *qp[NQT];
    float m[NQT], z[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        const int n = qt * 16 + r16;
        qp[qt] = Q + (int64_t)sm.qrow[n < nqg ? n : 0] * d;
        m[qt] = -INFINITY;
        z[qt] = 0.0f;
    }

    for (int64_t base = r0; base < r1; base += kRowsPerStep) {
        const int64_t rt = base + wave * kRowsPerWave;
        f32x4_t acc[NQT];
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        if (rt < r1) {
            const int64_t arow = rt + r16 < r1 ? rt + r16 : r1 - 1;
            const T *kp = K + arow * d;
            if constexpr (BF16) {
                const int full = d >> 5;
                int kk = kg * 8;
#pragma unroll 4
                for (int s = 0; s < full; ++s, kk += 32) {
                    const bf16x8_t A = load8(kp + kk);
#pragma unroll
                    for (int qt = 0; qt < NQT; ++qt)
                        acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, load8(qp[qt] + kk),
                                                                          acc[qt], 0, 0, 0);
                }
                if (d & 31) {
                    const bool ok = kk < d;
                    const bf16x8_t A = ok ? load8(kp + kk) : zero8();
#pragma unroll
                    for (int qt = 0; qt < NQT; ++qt)
                        acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            A, ok ? load8(qp[qt] + kk) : zero8(), acc[qt], 0, 0, 0);
                }
            } else {
                const int steps = d >> 2;
#pragma unroll 8
                for (int s = 0; s < steps; ++s) {
                    const int kk = 4 * s + kg;
                    const float A = (float)kp[kk];
#pragma unroll
                    for (int qt = 0; qt < NQT; ++qt)
                        acc[qt] = __builtin_amdgcn_mfma_f32_16x16x4f32(A, (float)qp[qt][kk],
                                                                       acc[qt], 0, 0, 0);
                }
            }
        }

        // D[row][query]: this lane holds rows rt + 4*kg + e, query column qt*16 + r16.
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
            const int n = qt * 16 + r16;
            const bool vq = n < nqg;
            float tm = -INFINITY;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (vq && rt + 4 * kg + e < r1) tm = fmaxf(tm, acc[qt][e]);
            if (tm != -INFINITY) {
                const float M = fmaxf(m[qt], tm);
                float zz = m[qt] == -INFINITY ? 0.0f : z[qt] * exp2f((m[qt] - M) * a.cexp);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (rt + 4 * kg + e < r1) zz += exp2f((acc[qt][e] - M) * a.cexp);
                m[qt] = M;
                z[qt] = zz;
                const uint64_t th = sm.theta[n];
                const uint32_t thi = (uint32_t)(th >> 32);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int64_t row = rt + 4 * kg + e;
                    if (row < r1) {
                        const uint32_t o = ord_of(acc[qt][e]);
                        if (o >= thi) {
                            const int32_t id = a.tid ? a.tid[row] : (int32_t)row;
                            const uint64_t key = ((uint64_t)o << 32) | (uint64_t)(~(uint32_t)id);
                            if (key > th) {
                                const uint32_t p = atomicAdd(&sm.cnt[n], 1u);
                                sm.buf[(size_t)n * cap + p] = key;
                            }
                        }
                    }
                }
            }
        }
        __syncthreads();
        for (int n = wave; n < nqg; n += kFineWaves)
            if ((int)sm.cnt[n] > cap - kRowsPerStep)
                topk_compact(TopkRow{sm.buf + (size_t)n * cap, &sm.cnt[n], &sm.theta[n]}, a.k, lane);
        __syncthreads();
    }

    // partial top-k of each query: sorted, truncated to k
    for (int n = wave; n < nqg; n += kFineWaves) {
        uint64_t *b = sm.buf + (size_t)n * cap;
        const int cn = (int)sm.cnt[n];
        const int np = next_pow2(cn < 2 ? 2 : cn);
        for (int i = cn + lane; i < np; i += kWave) b[i] = 0;
        wave_lds_sync();
        wave_sort_desc(b, np, lane);
        const int kept = cn < a.k ? cn : a.k;
        const int64_t p = a.pbase[g] + j * nq + qg0 + n;
        for (int r = lane; r < a.k; r += kWave) a.pk[p * a.k + r] = r < kept ? b[r] : 0;
        if (lane == 0) a.pc[p] = kept;
    }

    // (m, Z): lanes of one query column, then the four waves
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
        for (int sh = 16; sh <= 32; sh <<= 1) {
            const float m2 = __shfl_xor(m[qt], sh);
            const float z2 = __shfl_xor(z[qt], sh);
            mz_merge(m[qt], z[qt], m2, z2, a.cexp);
        }
        const int n = qt * 16 + r16;
        if (kg == 0 && n < nqg) {
            sm.wm[wave * a.qmax + n] = m[qt];
            sm.wz[wave * a.qmax + n] = z[qt];
        }
    }
    __syncthreads();
    for (int n = t; n < nqg; n += kFineThreads) {
        float M = -INFINITY, Z = 0.0f;
        for (int w = 0; w < kFineWaves; ++w) mz_merge(M, Z, sm.wm[w * a.qmax + n], sm.wz[w * a.qmax + n], a.cexp);
        const int64_t p = a.pbase[g] + j * nq + qg0 + n;
        a.pm[p] = M;
        a.pz[p] = Z;
    }
    __syncthreads();
}

template <typename T, bool BF16>
__global__ __launch_bounds__(kFineThreads) void fine_stream(FineArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_item;
    FineSmem sm;
    sm.buf = reinterpret_cast<uint64_t *>(smem_raw);
    sm.theta = sm.buf + (size_t)a.qmax * a.cap;
    sm.cnt = reinterpret_cast<uint32_t *>(sm.theta + a.qmax);
    sm.qrow = reinterpret_cast<int32_t *>(sm.cnt + a.qmax);
    sm.wm = reinterpret_cast<float *>(sm.qrow + a.qmax);
    sm.wz = sm.wm + kFineWaves * a.qmax;

    const int64_t W = a.plan->n_items;
    const int64_t CH = a.plan->chunk;
    for (;;) {
        if (threadIdx.x == 0) s_item = atomicAdd(&a.plan->next, 1);
        __syncthreads();
        const int64_t w = s_item;
        __syncthreads();
        if (w >= W) break;
        // cluster of work item w: the last g with wstart[g] <= w
        int32_t lo = 0, hi = a.G;          // wstart[lo] <= w < wstart[hi]
        while (hi - lo > 1) {
            const int32_t mid = (lo + hi) >> 1;
            if (a.wstart[mid] <= w) lo = mid; else hi = mid;
        }
        const int32_t g = lo;
        const int64_t j = w - a.wstart[g];
        const int64_t r0 = a.off[g] + j * CH;
        const int64_t r1 = min(a.off[g + 1], r0 + CH);
        const int32_t qbeg = a.qoff[g], nq = a.qoff[g + 1] - qbeg;
        for (int32_t qg0 = 0; qg0 < nq; qg0 += a.qmax) {
            const int32_t nqg = min(a.qmax, nq - qg0);
            switch ((nqg + 15) >> 4) {
                case 1: fine_pass<T, BF16, 1>(a, sm, g, j, r0, r1, qbeg, nq, qg0, nqg); break;
                case 2: fine_pass<T, BF16, 2>(a, sm, g, j, r0, r1, qbeg, nq, qg0, nqg); break;
                case 3: fine_pass<T, BF16, 3>(a, sm, g, j, r0, r1, qbeg, nq, qg0, nqg); break;
                default: fine_pass<T, BF16, 4>(a, sm, g, j, r0, r1, qbeg, nq, qg0, nqg); break;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// per-slot merge of the chunk partials (one wave per (query, slot))
// ---------------------------------------------------------------------------
struct MergeArgs {
    const int32_t *sel;
    const int64_t *off;
    const int32_t *qoff, *pos;
    const int64_t *pbase;
    const Plan *plan;
    const float *pm, *pz;
    const int32_t *pc;
    const uint64_t *pk;
    int32_t G, k, cap;
    float cexp;
    float *slot_max, *slot_sum, *cand_score;
    int32_t *cand_id;
};

__global__ __launch_bounds__(kWave) void slot_merge(MergeArgs a) {
    extern __shared__ __align__(16) uint64_t mbuf[];
    __shared__ uint32_t s_cnt;
    __shared__ uint64_t s_theta;
    const int lane = threadIdx.x;
    const int64_t e = blockIdx.x;
    const int32_t g = a.sel[e];
    if (lane == 0) { s_cnt = 0; s_theta = 0; }
    wave_lds_sync();
    TopkRow acc{mbuf, &s_cnt, &s_theta};
    float M = -INFINITY, Z = 0.0f;
    if (g >= 0 && g < a.G) {
        const int64_t len = a.off[g + 1] - a.off[g];
        const int64_t CH = a.plan->chunk;
        const int64_t nch = len > 0 ? (len + CH - 1) / CH : 0;
        const int64_t nq = a.qoff[g + 1] - a.qoff[g];
        const int64_t i = a.pos[e];
        for (int64_t jj = 0; jj < nch; ++jj) {
            const int64_t p = a.pbase[g] + jj * nq + i;
            mz_merge(M, Z, a.pm[p], a.pz[p], a.cexp);
            const int n = a.pc[p];
            for (int r0 = 0; r0 < n; r0 += kWave) {
                if (r0 + lane < n) topk_offer(acc, a.pk[p * a.k + r0 + lane]);
                wave_lds_sync();
                if ((int)s_cnt > a.cap - kWave) topk_compact(acc, a.k, lane);
            }
        }
    }
    const int cn = (int)s_cnt;
    const int np = next_pow2(cn < 2 ? 2 : cn);
    for (int i = cn + lane; i < np; i += kWave) mbuf[i] = 0;
    wave_lds_sync();
    wave_sort_desc(mbuf, np, lane);
    const int kept = cn < a.k ? cn : a.k;
    for (int r = lane; r < a.k; r += kWave) {
        const uint64_t key = mbuf[r];
        a.cand_score[e * a.k + r] = r < kept ? key_score(key) : -INFINITY;
        a.cand_id[e * a.k + r] = r < kept ? key_id(key) : -1;
    }
    if (lane == 0) {
        a.slot_max[e] = M;
        a.slot_sum[e] = Z;
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int fine_cap(int k) { return next_pow2(k + kRowsPerStep); }
static int fine_qmax(int k) {
    const int cap = fine_cap(k);
    int q = (72 * 1024) / (cap * 8);
    q = (q / 16) * 16;
    if (q > 16 * kMaxQueryTiles) q = 16 * kMaxQueryTiles;
    return q < 16 ? 16 : q;
}

AttendWs attend_layout(void *ws, int32_t d, int32_t G, int64_t N, int32_t key_bytes, int32_t B,
                       int32_t c, int32_t k, size_t *bytes) {
    AttendWs w{};
    Carve cv(ws);
    const int64_t bc = (int64_t)B * c;
    int64_t cm = (512 * 1024) / ((int64_t)d * key_bytes);
    int64_t ch = 64;
    while (ch * 2 <= cm) ch *= 2;
    w.chunk_min = ch;
    w.p_cap = 4 * bc;
    w.w_max = N / ch + G + 1;
    w.cnt = cv.take<int32_t>(G);
    w.cursor = cv.take<int32_t>(G);
    w.qoff = cv.take<int32_t>(G + 1);
    w.wstart = cv.take<int32_t>(G + 1);
    w.pbase = cv.take<int64_t>(G);
    w.qlist = cv.take<int32_t>(bc);
    w.pos = cv.take<int32_t>(bc);
    w.plan = cv.take<Plan>(1);
    w.pm = cv.take<float>(w.p_cap);
    w.pz = cv.take<float>(w.p_cap);
    w.pc = cv.take<int32_t>(w.p_cap);
    w.pk = cv.take<uint64_t>(w.p_cap * k);
    if (bytes) *bytes = cv.off + 256;
    return w;
}

template <typename T, bool BF16>
static hipError_t launch_fine_stream(const FineArgs &fa, int grid, size_t smem, KernelEvents ev,
                                     hipStream_t s) {
    auto kern = fine_stream<T, BF16>;
    // allow more than 64 KiB of dynamic LDS (a function attribute, not a stream operation)
    hipError_t err = hipFuncSetAttribute((const void *)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
    if (err != hipSuccess) return err;
    if (ev.before) hipEventRecord(ev.before, s);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kFineThreads), smem, s, fa);
    if (ev.after) hipEventRecord(ev.after, s);
    return hipGetLastError();
}

hipError_t launch_attend(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G, int64_t N,
                         const void *fine_keys, const int64_t *seg_offsets,
                         const int32_t *transition_id, const void *q, int32_t B,
                         const int32_t *sel, int32_t c, float tau, int32_t k, float *slot_max,
                         float *slot_sum, float *cand_score, int32_t *cand_id, const AttendWs &w,
                         int n_cu, KernelEvents ev, hipStream_t s) {
    const int64_t bc = (int64_t)B * c;
    const float cexp = 1.4426950408889634f / tau;
    const int gblocks = (int)((bc + 255) / 256 < 4096 ? (bc + 255) / 256 : 4096);
    hipLaunchKernelGGL(route_init, dim3((G + 255) / 256 < 1024 ? (G + 255) / 256 : 1024), dim3(256),
                       0, s, G, w.cnt, w.cursor, w.plan);
    hipLaunchKernelGGL(route_count, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.cnt, w.plan);
    hipLaunchKernelGGL(route_plan, dim3(1), dim3(kPlanThreads), 0, s, G, seg_offsets, w.cnt,
                       w.qoff, w.wstart, w.pbase, w.plan, w.chunk_min, w.p_cap);
    hipLaunchKernelGGL(route_scatter, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.qoff, w.cursor,
                       w.qlist, w.pos);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    FineArgs fa{};
    fa.keys = fine_keys;
    fa.off = seg_offsets;
    fa.tid = transition_id;
    fa.q = q;
    fa.d = d;
    fa.c = c;
    fa.G = G;
    fa.k = k;
    fa.cap = fine_cap(k);
    fa.qmax = fine_qmax(k);
    fa.cexp = cexp;
    fa.qoff = w.qoff;
    fa.qlist = w.qlist;
    fa.wstart = w.wstart;
    fa.pbase = w.pbase;
    fa.plan = w.plan;
    fa.pm = w.pm;
    fa.pz = w.pz;
    fa.pc = w.pc;
    fa.pk = w.pk;
    const size_t smem = fine_smem_bytes(fa.qmax, fa.cap);
    int64_t grid = (int64_t)n_cu * 2;
    if (grid > w.w_max) grid = w.w_max;
    if (grid < 1) grid = 1;
    if (compute_dtype == kF32)
        err = launch_fine_stream<float, false>(fa, (int)grid, smem, ev, s);
    else if (key_dtype == kF32)
        err = launch_fine_stream<float, true>(fa, (int)grid, smem, ev, s);
    else
        err = launch_fine_stream<__bf16, true>(fa, (int)grid, smem, ev, s);
    if (err != hipSuccess) return err;

    MergeArgs ma{};
    ma.sel = sel;
    ma.off = seg_offsets;
    ma.qoff = w.qoff;
    ma.pos = w.pos;
    ma.pbase = w.pbase;
    ma.plan = w.plan;
    ma.pm = w.pm;
    ma.pz = w.pz;
    ma.pc = w.pc;
    ma.pk = w.pk;
    ma.G = G;
    ma.k = k;
    ma.cap = next_pow2(k + kWave);
    ma.cexp = cexp;
    ma.slot_max = slot_max;
    ma.slot_sum = slot_sum;
    ma.cand_score = cand_score;
    ma.cand_id = cand_id;
    hipLaunchKernelGGL(slot_merge, dim3((unsigned)bc), dim3(kWave), (size_t)ma.cap * 8, s, ma);
    return hipGetLastError();
}

}  // namespace htam
