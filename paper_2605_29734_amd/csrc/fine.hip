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
constexpr size_t kRouteLdsBytes = 64 * 1024;   // per-cluster counters of the fused routing kernel
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

// Exclusive scan of one int64 value per thread over a 1024-thread block:
// wave scans through shuffles, then one wave scans the 16 wave totals.
// `s` holds at least 16 values; every thread must call it.
__device__ int64_t block_exclusive_scan(int64_t v, int64_t *s, int64_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int waves = kPlanThreads / kWave;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s[wave] = x;
    __syncthreads();
    if (wave == 0) {
        int64_t w = lane < waves ? s[lane] : 0;
#pragma unroll
        for (int o = 1; o < waves; o <<= 1) {
            const int64_t y = __shfl_up(w, o);
            if (lane >= o) w += y;
        }
        if (lane < waves) s[lane] = w;
    }
    __syncthreads();
    const int64_t before = wave > 0 ? s[wave - 1] : 0;
    *total = s[waves - 1];
    __syncthreads();
    return before + x - v;
}

__device__ int64_t block_sum(int64_t v, int64_t *s) {
    int64_t total;
    block_exclusive_scan(v, s, &total);
    return total;
}

__device__ int64_t block_max(int64_t v, int64_t *s) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int waves = kPlanThreads / kWave;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const int64_t y = __shfl_xor(v, o);
        v = v > y ? v : y;
    }
    if (lane == 0) s[wave] = v;
    __syncthreads();
    int64_t r = s[0];
    for (int w = 1; w < waves; ++w) r = r > s[w] ? r : s[w];
    __syncthreads();
    return r;
}

// Chunk length and work numbering from the per-cluster query counts (read
// through cnt_of): the chunk is the smallest power-of-two multiple of
// chunk_min for which the partial results fit in p_cap (it always fits once a
// chunk spans the longest segment: then each (query, slot) has one partial and
// p_cap >= B*c). Writes qoff, wstart, pbase and the plan.
template <typename CntOf>
__device__ void plan_chunks(int32_t G, const int64_t *off, CntOf cnt_of, int32_t *qoff,
                            int32_t *wstart, int64_t *pbase, Plan *plan, int64_t chunk_min,
                            int64_t p_cap, int64_t *s) {
    const int t = threadIdx.x;
    const int32_t per = (G + kPlanThreads - 1) / kPlanThreads;
    const int32_t g0 = min((int32_t)G, t * per), g1 = min((int32_t)G, g0 + per);
    int64_t local = 0, lmax = 0;
    for (int32_t g = g0; g < g1; ++g) {
        local += cnt_of(g);
        const int64_t len = off[g + 1] - off[g];
        lmax = len > lmax ? len : lmax;
    }
    int64_t total;
    int64_t run = block_exclusive_scan(local, s, &total);
    for (int32_t g = g0; g < g1; ++g) {
        qoff[g] = (int32_t)run;
        run += cnt_of(g);
    }
    if (t == kPlanThreads - 1) qoff[G] = (int32_t)total;
    const int64_t maxlen = block_max(lmax, s);

    int64_t ch = chunk_min;
    for (int it = 0; it < 48; ++it) {
        int64_t p = 0;
        for (int32_t g = g0; g < g1; ++g) {
            const int64_t len = off[g + 1] - off[g];
            const int64_t c = cnt_of(g);
            if (c > 0 && len > 0) p += c * ((len + ch - 1) / ch);
        }
        const int64_t P = block_sum(p, s);
        if (P <= p_cap || ch >= maxlen) break;
        ch *= 2;
    }

    int64_t wl = 0, pl = 0;
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t len = off[g + 1] - off[g];
        const int64_t c = cnt_of(g);
        const int64_t nch = (c > 0 && len > 0) ? (len + ch - 1) / ch : 0;
        wl += nch;
        pl += nch * c;
    }
    int64_t wtot, ptot;
    int64_t wrun = block_exclusive_scan(wl, s, &wtot);
    int64_t prun = block_exclusive_scan(pl, s, &ptot);
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t len = off[g + 1] - off[g];
        const int64_t c = cnt_of(g);
        const int64_t nch = (c > 0 && len > 0) ? (len + ch - 1) / ch : 0;
        wstart[g] = (int32_t)wrun;
        pbase[g] = prun;
        wrun += nch;
        prun += nch * c;
    }
    if (t == kPlanThreads - 1) {
        wstart[G] = (int32_t)wtot;
        plan->chunk = ch;
        plan->n_items = wtot;
        plan->n_parts = ptot;
    }
}

struct GlobalCnt {
    const int32_t *cnt;
    __device__ int64_t operator()(int32_t g) const { return cnt[g]; }
};
struct LdsCnt {
    const int32_t *cnt;
    __device__ int64_t operator()(int32_t g) const { return cnt[g]; }
};

// Planning step of the multi-kernel routing (counts in global memory).
__global__ __launch_bounds__(kPlanThreads) void route_plan(int32_t G, const int64_t *off,
                                                           const int32_t *cnt, int32_t *qoff,
                                                           int32_t *wstart, int64_t *pbase,
                                                           Plan *plan, int64_t chunk_min,
                                                           int64_t p_cap) {
    __shared__ int64_t s[kPlanThreads / kWave];
    plan_chunks(G, off, GlobalCnt{cnt}, qoff, wstart, pbase, plan, chunk_min, p_cap, s);
}

// The whole routing in one block when the per-cluster counters fit in LDS:
// count the (query, slot) pairs per cluster, plan the chunks, then scatter the
// pairs into per-cluster lists.
__global__ __launch_bounds__(kPlanThreads) void route_fused(const int32_t *sel, int64_t n,
                                                            int32_t G, const int64_t *off,
                                                            int32_t *qoff, int32_t *wstart,
                                                            int64_t *pbase, int32_t *qlist,
                                                            int32_t *pos, Plan *plan,
                                                            int64_t chunk_min, int64_t p_cap) {
    extern __shared__ int32_t lcnt[];       // [G]
    __shared__ int64_t s[kPlanThreads / kWave];
    __shared__ int32_t s_bad;
    const int t = threadIdx.x;
    for (int32_t g = t; g < G; g += kPlanThreads) lcnt[g] = 0;
    if (t == 0) s_bad = 0;
    __syncthreads();
    int32_t bad = 0;
    for (int64_t e = t; e < n; e += kPlanThreads) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) atomicAdd(&lcnt[g], 1);
        else ++bad;
    }
    if (bad) atomicAdd(&s_bad, bad);
    __syncthreads();
    plan_chunks(G, off, LdsCnt{lcnt}, qoff, wstart, pbase, plan, chunk_min, p_cap, s);
    __syncthreads();
    for (int32_t g = t; g < G; g += kPlanThreads) lcnt[g] = qoff[g];   // becomes the fill cursor
    if (t == 0) {
        plan->next = 0;
        plan->bad_sel = s_bad;
    }
    __syncthreads();
    for (int64_t e = t; e < n; e += kPlanThreads) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) {
            const int32_t at = atomicAdd(&lcnt[g], 1);
            qlist[at] = (int32_t)e;
            pos[e] = at - qoff[g];
        }
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

// One wave per (query, slot). The (m, Z) partials of the slot's chunks are
// merged lane-parallel; their top-k entries (k keys per chunk, zero-padded) are
// streamed 8 x 64 at a time through a threshold filter into the wave's LDS
// buffer, compacted by radix select when it fills, and sorted at the end.
constexpr int kMergeWaves = 4;
constexpr int kMergeBatch = 8;

template <int NPL>
__global__ __launch_bounds__(kWave * kMergeWaves) void slot_merge(MergeArgs a) {
    extern __shared__ __align__(16) uint64_t mbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t e = (int64_t)blockIdx.x * kMergeWaves + wave;
    if (e >= a.n_pairs) return;              // no block-wide synchronisation below
    uint64_t *buf = mbuf + wave * cap;
    const uint64_t lt_mask = (1ull << lane) - 1;
    const int32_t g = a.sel[e];
    float M = -INFINITY, Z = 0.0f;
    int cnt = 0;
    uint64_t theta = 0;
    if (g >= 0 && g < a.G) {
        const int64_t len = a.off[g + 1] - a.off[g];
        const int64_t CH = a.plan->chunk;
        const int64_t nch = len > 0 ? (len + CH - 1) / CH : 0;
        const int64_t nq = a.qoff[g + 1] - a.qoff[g];
        const int64_t p0 = a.pbase[g] + a.pos[e];
        for (int64_t jj = lane; jj < nch; jj += kWave)
            mz_merge(M, Z, a.pm[p0 + jj * nq], a.pz[p0 + jj * nq], a.cexp);
        const int64_t total = nch * a.k;
        for (int64_t base = 0; base < total; base += kWave * kMergeBatch) {
            uint64_t key[kMergeBatch];
#pragma unroll
            for (int u = 0; u < kMergeBatch; ++u) {
                const int64_t f = base + u * kWave + lane;
                const int64_t fc = f < total ? f : total - 1;
                const int64_t jj = fc / a.k, r = fc - jj * a.k;
                const uint64_t kv = a.pk[(p0 + jj * nq) * a.k + r];
                key[u] = f < total ? kv : 0;
            }
#pragma unroll
            for (int u = 0; u < kMergeBatch; ++u) {
                const bool pass = key[u] > theta;
                const uint64_t mask = __ballot(pass);
                if (pass) buf[cnt + __popcll(mask & lt_mask)] = key[u];
                cnt += __popcll(mask);
                if (cnt > cap - kWave) {
                    wave_lds_sync();
                    cnt = compact_select<NPL>(buf, cnt, a.k, kWave, lane, theta);
                }
            }
        }
    }
    for (int sh = 32; sh >= 1; sh >>= 1) {
        const float m2 = __shfl_xor(M, sh), z2 = __shfl_xor(Z, sh);
        mz_merge(M, Z, m2, z2, a.cexp);
    }
    wave_lds_sync();
    uint64_t v[NPL];
#pragma unroll
    for (int q = 0; q < NPL; ++q) v[q] = (q * kWave + lane < cnt) ? buf[q * kWave + lane] : 0;
    wave_sort_regs<NPL>(v, lane);
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

// Queries per pass actually provisioned: enough for about twice the mean
// number of queries per selected cluster (a cluster with more takes several
// passes), so that small query groups leave room for more blocks per CU.
static int qmax_for_load(int qmax, int64_t bc, int32_t G) {
    const int64_t mean = (bc + G - 1) / (G > 0 ? G : 1);
    int want = (int)(((2 * mean + 15) / 16) * 16);
    if (want < 16) want = 16;
    return want < qmax ? want : qmax;
}

static hipError_t launch_stream(int32_t key_dtype, int32_t compute_dtype, const FineArgs &fa0,
                                int64_t bc, int n_cu, int64_t w_max, KernelEvents ev,
                                hipStream_t s) {
    const size_t budget = lds_budget();
    const int npl = fa0.cap / kWave;
    StreamLaunch l{};
    l.fa = fa0;
    l.ev = ev;
    l.stream = s;
    auto grid_for = [&](size_t smem) {
        int per_cu = (int)((budget + 1024) / (smem + 1024));
        if (per_cu < 1) per_cu = 1;
        if (per_cu > 4) per_cu = 4;
        int64_t g = (int64_t)n_cu * per_cu;
        if (g > w_max) g = w_max;
        return (int)(g < 1 ? 1 : g);
    };
    int ql = qmax_for_lds(key_dtype, compute_dtype, fa0.d, fa0.cap, budget);
    if (ql > 0) {
        ql = qmax_for_load(ql, bc, fa0.G);
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
    const size_t smem = (size_t)kMergeWaves * NPL * kWave * 8;
    hipLaunchKernelGGL(slot_merge<NPL>, dim3((unsigned)((ma.n_pairs + kMergeWaves - 1) / kMergeWaves)),
                       dim3(kWave * kMergeWaves), smem, s, ma);
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
    const int64_t ch_min = chunk_floor_rows(N, n_cu);
    if ((size_t)G * 4 <= kRouteLdsBytes) {
        hipLaunchKernelGGL(route_fused, dim3(1), dim3(kPlanThreads), (size_t)G * 4, s, sel, bc, G,
                           seg_offsets, w.qoff, w.wstart, w.pbase, w.qlist, w.pos, w.plan, ch_min,
                           w.p_cap);
    } else {
        hipLaunchKernelGGL(route_init, dim3((G + 255) / 256 < 1024 ? (G + 255) / 256 : 1024),
                           dim3(256), 0, s, G, w.cnt, w.cursor, w.plan);
        hipLaunchKernelGGL(route_count, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.cnt, w.plan);
        hipLaunchKernelGGL(route_plan, dim3(1), dim3(kPlanThreads), 0, s, G, seg_offsets, w.cnt,
                           w.qoff, w.wstart, w.pbase, w.plan, ch_min, w.p_cap);
        hipLaunchKernelGGL(route_scatter, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.qoff,
                           w.cursor, w.qlist, w.pos);
    }
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
    err = launch_stream(key_dtype, compute_dtype, fa, bc, n_cu, w.w_max, ev, s);
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
    switch (next_pow2(k + kWave) / kWave) {
        case 2: return launch_merge<2>(ma, s);
        case 4: return launch_merge<4>(ma, s);
        default: return launch_merge<8>(ma, s);
    }
}

}  // namespace htam
