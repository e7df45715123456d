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
#include "stream.hpp"

namespace htam {

namespace {

constexpr int kPlanThreads = 1024;
constexpr int64_t kChunkFloor = 64;
constexpr int64_t kChunkCeil = 4096;

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
    int64_t n_pairs;
    int32_t G, k;
    float cexp;
    float *slot_max, *slot_sum, *cand_score;
    int32_t *cand_id;
};

// Partials are sorted lists of at most k keys; they are merged pairwise in
// registers (64*NPL >= k), skipping any partial whose best key cannot enter.
template <int NPL>
__global__ __launch_bounds__(256) void slot_merge(MergeArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t e = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (e >= a.n_pairs) return;
    const int32_t g = a.sel[e];
    float M = -INFINITY, Z = 0.0f;
    uint64_t acc[NPL];
#pragma unroll
    for (int jj = 0; jj < NPL; ++jj) acc[jj] = 0;
    if (g >= 0 && g < a.G) {
        const int64_t len = a.off[g + 1] - a.off[g];
        const int64_t CH = a.plan->chunk;
        const int64_t nch = len > 0 ? (len + CH - 1) / CH : 0;
        const int64_t nq = a.qoff[g + 1] - a.qoff[g];
        const int64_t i = a.pos[e];
        uint64_t kth = 0;            // k-th best key merged so far (0 while fewer)
        for (int64_t jj = 0; jj < nch; ++jj) {
            const int64_t p = a.pbase[g] + jj * nq + i;
            mz_merge(M, Z, a.pm[p], a.pz[p], a.cexp);
            const int n = a.pc[p];
            if (n == 0 || a.pk[p * a.k] <= kth) continue;
            uint64_t b[NPL];
#pragma unroll
            for (int q = 0; q < NPL; ++q)
                b[q] = (q * kWave + lane < n) ? a.pk[p * a.k + q * kWave + lane] : 0;
            wave_merge_top<NPL>(acc, b, lane);
            kth = wave_element<NPL>(acc, a.k - 1);
        }
    }
#pragma unroll
    for (int jj = 0; jj < NPL; ++jj) {
        const int r = jj * kWave + lane;
        if (r < a.k) {
            const uint64_t key = acc[jj];
            a.cand_score[e * a.k + r] = key ? key_score(key) : -INFINITY;
            a.cand_id[e * a.k + r] = key ? key_id(key) : -1;
        }
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

// Shortest chunk: the bank's rows spread over about 8 chunks per compute unit
// (a power of two between kChunkFloor and kChunkCeil rows); the planning
// kernel doubles it while the partial results would not fit.
static int64_t chunk_floor_rows(int64_t N, int n_cu) {
    const int64_t target = N / ((int64_t)(n_cu > 0 ? n_cu : 1) * 8);
    int64_t ch = kChunkFloor;
    while (ch * 2 <= target && ch * 2 <= kChunkCeil) ch *= 2;
    return ch;
}

// Queries per pass of the generic kernel (its LDS holds only the top-k state).
static int qmax_generic(int cap) {
    int q = (72 * 1024) / (cap * 8);
    q = (q / 16) * 16;
    if (q > 16 * kMaxQueryTiles) q = 16 * kMaxQueryTiles;
    return q < 16 ? 16 : q;
}

// Queries per pass of the LDS kernel: the most (a multiple of 16, at most 64)
// whose B fragments and top-k state fit in the LDS budget; 0 if 16 do not.
static int qmax_lds(int d, int cap, size_t budget) {
    for (int q = 16 * kMaxQueryTiles; q >= 16; q -= 16)
        if (fine_qs_bytes(d, q) + fine_state_bytes(q, cap) <= budget) return q;
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
    bytes -= 1024;      // static LDS of the kernels
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

// Queries per pass of the LDS kernel: the most (a multiple of 16, at most 64)
// whose B fragments and top-k state fit in the LDS budget; 0 when the LDS
// kernel does not apply (fp32 arithmetic, d not a multiple of 32 * U, or not
// even 16 queries fit).
static int qmax_for_lds(int32_t key_dtype, int32_t compute_dtype, int d, int cap, size_t budget) {
    const int U = key_dtype == kF32 ? 8 : 16;
    if (compute_dtype != kBF16 || d % (32 * U) != 0) return 0;
    return qmax_lds(d, cap, budget);
}

static hipError_t launch_stream(int32_t key_dtype, int32_t compute_dtype, const FineArgs &fa0,
                                int n_cu, int64_t w_max, KernelEvents ev, hipStream_t s) {
    const size_t budget = lds_budget();
    const int npl = fa0.cap / kWave;
    StreamLaunch l{};
    l.fa = fa0;
    l.ev = ev;
    l.stream = s;
    auto grid_for = [&](size_t smem) {
        int per_cu = (int)((budget + 1024) / (smem + 1024));
        if (per_cu < 1) per_cu = 1;
        if (per_cu > 2) per_cu = 2;
        int64_t g = (int64_t)n_cu * per_cu;
        if (g > w_max) g = w_max;
        return (int)(g < 1 ? 1 : g);
    };
    const int ql = qmax_for_lds(key_dtype, compute_dtype, fa0.d, fa0.cap, budget);
    if (ql > 0) {
        l.fa.qmax = ql;
        l.qs_bytes = (int32_t)fine_qs_bytes(fa0.d, ql);
        l.smem = l.qs_bytes + fine_state_bytes(ql, fa0.cap);
        l.grid = grid_for(l.smem);
        return key_dtype == kF32 ? launch_stream_lds_f32(npl, fa0.tid != nullptr, l)
                                 : launch_stream_lds_bf16(npl, fa0.tid != nullptr, l);
    }
    l.fa.qmax = qmax_generic(fa0.cap);
    l.qs_bytes = 0;
    l.smem = fine_state_bytes(l.fa.qmax, fa0.cap);
    l.grid = grid_for(l.smem);
    return launch_stream_generic(key_dtype, compute_dtype, npl, l);
}

template <int NPL>
static hipError_t launch_merge(const MergeArgs &ma, hipStream_t s) {
    hipLaunchKernelGGL(slot_merge<NPL>, dim3((unsigned)((ma.n_pairs + 3) / 4)), dim3(256), 0, s, ma);
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
                       w.qoff, w.wstart, w.pbase, w.plan, chunk_floor_rows(N, n_cu), w.p_cap);
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
    err = launch_stream(key_dtype, compute_dtype, fa, n_cu, w.w_max, ev, s);
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
    ma.n_pairs = bc;
    ma.G = G;
    ma.k = k;
    ma.cexp = cexp;
    ma.slot_max = slot_max;
    ma.slot_sum = slot_sum;
    ma.cand_score = cand_score;
    ma.cand_id = cand_id;
    const int kp = next_pow2(k) / kWave;
    if (kp <= 1) return launch_merge<1>(ma, s);
    if (kp == 2) return launch_merge<2>(ma, s);
    return launch_merge<4>(ma, s);
}

}  // namespace htam
