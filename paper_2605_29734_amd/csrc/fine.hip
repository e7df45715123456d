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
constexpr int64_t kFusedRoutePairs = 16384;     // above this many pairs, route with many blocks
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

// Inputs and outputs of the planning step (device pointers).
struct PlanArgs {
    int32_t G;
    const int64_t *off;
    int32_t *qoff;            // [G+1]
    int32_t *wstart;          // [G+1] first work item of each cluster
    int32_t *gstart;          // [G+1] first level-one merge group of each cluster
    int32_t *mstart;          // [G+1] first merge-list entry of each cluster
    int64_t *pbase;           // [G]
    int64_t *ubase;           // [G]
    Plan *plan;
    int64_t chunk_min, p_cap;
    int32_t group;            // chunk partials per level-one merge group
};

// Chunk length and work numbering from the per-cluster query counts (read
// through cnt_of): the chunk is the smallest power-of-two multiple of
// chunk_min for which the partial results fit in p_cap (it always fits once a
// chunk spans the longest segment: then each (query, slot) has one partial and
// p_cap >= B*c). Writes qoff, wstart, gstart, pbase, ubase and the plan; the
// item and group tables are filled afterwards by route_items. Clusters are
// split into contiguous ranges, one per thread.
template <typename CntOf>
__device__ void plan_chunks(const PlanArgs &pa, CntOf cnt_of, int64_t *s) {
    const int t = threadIdx.x;
    const int32_t G = pa.G;
    const int32_t per = (G + kPlanThreads - 1) / kPlanThreads;
    const int32_t g0 = min((int32_t)G, t * per), g1 = min((int32_t)G, g0 + per);
    int64_t local = 0, lmax = 0;
    for (int32_t g = g0; g < g1; ++g) {
        local += cnt_of(g);
        const int64_t len = pa.off[g + 1] - pa.off[g];
        lmax = len > lmax ? len : lmax;
    }
    int64_t total;
    int64_t run = block_exclusive_scan(local, s, &total);
    for (int32_t g = g0; g < g1; ++g) {
        pa.qoff[g] = (int32_t)run;
        run += cnt_of(g);
    }
    if (t == kPlanThreads - 1) pa.qoff[G] = (int32_t)total;
    const int64_t maxlen = block_max(lmax, s);

    int64_t ch = pa.chunk_min;
    for (int it = 0; it < 48; ++it) {
        int64_t p = 0;
        for (int32_t g = g0; g < g1; ++g) {
            const int64_t len = pa.off[g + 1] - pa.off[g];
            const int64_t c = cnt_of(g);
            if (c > 0 && len > 0) p += c * ((len + ch - 1) / ch);
        }
        const int64_t P = block_sum(p, s);
        if (P <= pa.p_cap || ch >= maxlen) break;
        ch *= 2;
    }

    const int64_t R = pa.group;
    auto chunks = [&](int32_t g) -> int64_t {
        const int64_t len = pa.off[g + 1] - pa.off[g];
        return (cnt_of(g) > 0 && len > 0) ? (len + ch - 1) / ch : 0;
    };
    auto ngroups = [&](int64_t nch) -> int64_t { return nch > R ? (nch + R - 1) / R : 0; };
    int64_t wl = 0, pl = 0, gl = 0, ul = 0, ml = 0;
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t nch = chunks(g), c = cnt_of(g);
        wl += nch;
        pl += nch * c;
        gl += ngroups(nch);
        ul += ngroups(nch) * c;
        ml += nch != 1 ? c : 0;     // empty segments are finished by the merge too
    }
    int64_t wtot, ptot, gtot, utot, mtot;
    int64_t wrun = block_exclusive_scan(wl, s, &wtot);
    int64_t prun = block_exclusive_scan(pl, s, &ptot);
    int64_t grun = block_exclusive_scan(gl, s, &gtot);
    int64_t urun = block_exclusive_scan(ul, s, &utot);
    int64_t mrun = block_exclusive_scan(ml, s, &mtot);
    for (int32_t g = g0; g < g1; ++g) {
        const int64_t nch = chunks(g), c = cnt_of(g), ng = ngroups(nch);
        pa.wstart[g] = (int32_t)wrun;
        pa.gstart[g] = (int32_t)grun;
        pa.mstart[g] = (int32_t)mrun;
        pa.pbase[g] = prun;
        pa.ubase[g] = urun;
        wrun += nch;
        prun += nch * c;
        grun += ng;
        urun += ng * c;
        mrun += nch != 1 ? c : 0;
    }
    if (t == kPlanThreads - 1) {
        pa.wstart[G] = (int32_t)wtot;
        pa.gstart[G] = (int32_t)gtot;
        pa.mstart[G] = (int32_t)mtot;
        pa.plan->n_merge = mtot;
        pa.plan->chunk = ch;
        pa.plan->n_items = wtot;
        pa.plan->n_parts = ptot;
        pa.plan->n_groups = gtot;
        pa.plan->n_l1 = utot;
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

// Planning step of the multi-kernel routing (counts in global memory).
__global__ __launch_bounds__(kPlanThreads) void route_plan(PlanArgs pa, const int32_t *cnt) {
    __shared__ int64_t s[kPlanThreads / kWave];
    plan_chunks(pa, GlobalCnt{cnt}, s);
}

// The whole routing in one block when the pairs are few and the per-cluster
// counters fit in LDS: count the (query, slot) pairs per cluster, plan the
// chunks, then scatter the pairs into per-cluster lists.
__global__ __launch_bounds__(kPlanThreads) void route_fused(PlanArgs pa, const int32_t *sel,
                                                            int64_t n, int32_t *qlist,
                                                            int32_t *pos, SlotOut out) {
    extern __shared__ int32_t lcnt[];       // [G]
    __shared__ int64_t s[kPlanThreads / kWave];
    __shared__ int32_t s_bad;
    const int t = threadIdx.x;
    const int32_t G = pa.G;
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
    plan_chunks(pa, LdsCnt{lcnt}, s);
    __syncthreads();
    for (int32_t g = t; g < G; g += kPlanThreads) lcnt[g] = pa.qoff[g];   // becomes the fill cursor
    if (t == 0) {
        pa.plan->next = 0;
        pa.plan->bad_sel = s_bad;
    }
    __syncthreads();
    for (int64_t e = t; e < n; e += kPlanThreads) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) {
            const int32_t at = atomicAdd(&lcnt[g], 1);
            qlist[at] = (int32_t)e;
            pos[e] = at - pa.qoff[g];
        } else {
            out.empty(e);
        }
    }
}

// Fills, from the plan and the per-cluster query lists, the item table of the
// bank stream, the level-one merge groups and their work units, and the list
// of pairs the merge finishes (clusters of several chunks, and empty ones):
// one wave per cluster, spread over the lanes.
__global__ __launch_bounds__(256) void route_items(PlanArgs pa, const int32_t *qlist,
                                                   WorkItem *items, MergeGroup *groups,
                                                   int2 *units, int32_t *mlist) {
    const int lane = threadIdx.x & 63;
    const int64_t ch = pa.plan->chunk;
    const int64_t R = pa.group;
    for (int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); g < pa.G;
         g += (int64_t)gridDim.x * 4) {
        const int32_t w0 = pa.wstart[g], nch = pa.wstart[g + 1] - w0;
        const int32_t qb = pa.qoff[g], nq = pa.qoff[g + 1] - qb;
        if (nq == 0) continue;
        if (nch != 1) {
            const int32_t m0 = pa.mstart[g];
            for (int32_t i = lane; i < nq; i += kWave) mlist[m0 + i] = qlist[qb + i];
        }
        if (nch == 0) continue;
        const int32_t gs = pa.gstart[g], ng = pa.gstart[g + 1] - gs;
        const int64_t a = pa.off[g], len = pa.off[g + 1] - a;
        const int64_t pb = pa.pbase[g], ub = pa.ubase[g];
        for (int32_t j = lane; j < nch; j += kWave) {
            WorkItem wi;
            wi.r0 = a + j * ch;
            wi.p0 = pb + (int64_t)j * nq;
            wi.len = (int32_t)(len - j * ch < ch ? len - j * ch : ch);
            wi.g = (int32_t)g;
            wi.qbeg = qb;
            wi.nq = nq;
            wi.single = nch == 1;
            wi.pad = 0;
            items[w0 + j] = wi;
        }
        for (int32_t jg = lane; jg < ng; jg += kWave) {
            MergeGroup mg;
            mg.p0 = pb + jg * R * nq;
            mg.u0 = ub + (int64_t)jg * nq;
            mg.npart = (int32_t)(nch - jg * R < R ? nch - jg * R : R);
            mg.nq = nq;
            groups[gs + jg] = mg;
        }
        for (int64_t x = lane; x < (int64_t)ng * nq; x += kWave) {
            const int32_t jg = (int32_t)(x / nq), i = (int32_t)(x - (int64_t)jg * nq);
            units[ub + x] = make_int2(gs + jg, i);
        }
    }
}

__global__ void route_scatter(const int32_t *sel, int64_t n, int32_t G, const int32_t *qoff,
                              int32_t *cursor, int32_t *qlist, int32_t *pos, SlotOut out) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t g = sel[e];
        if (g >= 0 && g < G) {
            const int32_t slot = atomicAdd(&cursor[g], 1);
            qlist[qoff[g] + slot] = (int32_t)e;
            pos[e] = slot;
        } else {
            out.empty(e);
        }
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
    const int32_t *sel;
    const int64_t *off;
    const int32_t *qoff, *pos, *mlist;
    const int64_t *pbase, *ubase;
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
    int32_t G, k, group;
    float cexp;
    float *slot_max, *slot_sum, *cand_score;
    int32_t *cand_id;
};

constexpr int kMergeWaves = 4;
constexpr int kMergeBatch = 8;

// One wave merges n partial results (m, Z, count, k keys) found at
// p0 + i * stride: (m, Z) lane-parallel; the keys 8 x 64 at a time through a
// threshold filter into the wave's LDS buffer (cap = 64 * NPL >= k + 64),
// compacted by radix select when it fills. The kept keys are left in buf
// (count returned), unsorted; M and Z are the merged statistics in every lane.
template <int NPL>
__device__ __forceinline__ int merge_partials(const float *pm, const float *pz, const int32_t *pc,
                                              const uint64_t *pk, int64_t p0, int64_t stride,
                                              int64_t n, int k, float cexp, uint64_t *buf,
                                              float &M, float &Z) {
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63;
    const uint64_t lt_mask = (1ull << lane) - 1;
    M = -INFINITY;
    Z = 0.0f;
    for (int64_t jj = lane; jj < n; jj += kWave)
        mz_merge(M, Z, pm[p0 + jj * stride], pz[p0 + jj * stride], cexp);
    for (int sh = 32; sh >= 1; sh >>= 1) {
        const float m2 = __shfl_xor(M, sh), z2 = __shfl_xor(Z, sh);
        mz_merge(M, Z, m2, z2, cexp);
    }
    int cnt = 0;
    uint64_t theta = 0;
    // entries f = j * kp + r with kp = k rounded up to a power of two: the
    // partial and the key within it come from a shift and a mask
    const int lk = 31 - __builtin_clz((unsigned)(2 * k - 1));
    const int64_t kp = int64_t(1) << lk;
    const int64_t total = n * kp;
    for (int64_t base = 0; base < total; base += kWave * kMergeBatch) {
        uint64_t key[kMergeBatch];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const int64_t f = base + u * kWave + lane;
            const int64_t jj = f >> lk, r = f & (kp - 1);
            const bool ok = f < total && r < k;
            const int64_t src = ok ? (p0 + jj * stride) * k + r : p0 * k;
            const uint64_t kv = pk[src];
            key[u] = ok ? kv : 0;
        }
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            const bool pass = key[u] > theta;
            const uint64_t mask = __ballot(pass);
            if (pass) buf[cnt + __popcll(mask & lt_mask)] = key[u];
            cnt += __popcll(mask);
            if (cnt > cap - kWave) {
                wave_lds_sync();
                cnt = compact_select<NPL>(buf, cnt, k, kWave, lane, theta);
            }
        }
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
        const int64_t e = a.mlist[u];
        const int32_t g = a.sel[e];
        const int64_t len = a.off[g + 1] - a.off[g];
        const int64_t CH = a.plan->chunk;
        const int64_t nch = (len + CH - 1) / CH;
        const int64_t nq = a.qoff[g + 1] - a.qoff[g];
        float M, Z;
        int cnt;
        if (nch > a.group)
            cnt = merge_partials<NPL>(a.um, a.uz, a.uc, a.uk, a.ubase[g] + a.pos[e], nq,
                                      (nch + a.group - 1) / a.group, a.k, a.cexp, buf, M, Z);
        else
            cnt = merge_partials<NPL>(a.pm, a.pz, a.pc, a.pk, a.pbase[g] + a.pos[e], nq, nch, a.k,
                                      a.cexp, buf, M, Z);
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
        wave_lds_sync();
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int fine_cap(int k) { return next_pow2(k + kRowsPerStep); }

// Shortest chunk: the bank's rows spread over about 4 chunks per compute unit
// (a power of two between kChunkFloor and kChunkCeil rows); the planning
// kernel doubles it while the partial results would not fit.
static int64_t chunk_floor_rows(int64_t N, int n_cu) {
    const int64_t target = N / ((int64_t)(n_cu > 0 ? n_cu : 1) * 4);
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

// Chunk partials per level-one merge group: about 2048 keys per wave.
static int merge_group(int k) {
    int r = 8;
    while (r * 2 * k <= 2048 && r < 128) r *= 2;
    return r;
}

AttendWs attend_layout(void *ws, int32_t d, int32_t G, int64_t N, int32_t key_bytes, int32_t B,
                       int32_t c, int32_t k, size_t *bytes) {
    (void)d;
    (void)key_bytes;
    AttendWs w{};
    Carve cv(ws);
    const int64_t bc = (int64_t)B * c;
    w.p_cap = 4 * bc;
    w.w_max = N / kChunkFloor + G + 1;
    w.group = merge_group(k);
    w.g_max = 2 * w.w_max / w.group + 1;
    w.u_cap = 2 * w.p_cap / w.group + 1;
    w.cnt = cv.take<int32_t>(G);
    w.cursor = cv.take<int32_t>(G);
    w.qoff = cv.take<int32_t>(G + 1);
    w.wstart = cv.take<int32_t>(G + 1);
    w.gstart = cv.take<int32_t>(G + 1);
    w.pbase = cv.take<int64_t>(G);
    w.ubase = cv.take<int64_t>(G);
    w.mstart = cv.take<int32_t>(G + 1);
    w.mlist = cv.take<int32_t>(bc);
    w.units = cv.take<int2>(w.u_cap);
    w.qlist = cv.take<int32_t>(bc);
    w.pos = cv.take<int32_t>(bc);
    w.plan = cv.take<Plan>(1);
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

static hipError_t launch_stream(int32_t key_dtype, int32_t compute_dtype, const FineArgs &fa0,
                                int64_t bc, int n_cu, int64_t w_max, KernelEvents ev,
                                hipStream_t s) {
    const size_t budget = lds_budget();
    const int npl = fa0.cap / kWave;
    StreamLaunch l{};
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
        const int unit_k = key_dtype == kF32 ? 8 : 16;
        if (two || fa0.d % (32 * unit_k) == 0)
            return key_dtype == kF32 ? launch_stream_lds_f32(npl, two, l)
                                     : launch_stream_lds_bf16(npl, two, l);
    }
    l.fa.qmax = qmax_generic(fa0.cap);
    l.fa.ntile = 2;
    l.qs_bytes = 0;
    l.smem = fine_state_bytes(l.fa.qmax, fa0.cap, 2);
    return launch_stream_generic(key_dtype, compute_dtype, npl, l);
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
static hipError_t launch_merge(const MergeArgs &ma, int64_t u_cap, int n_cu, hipStream_t s) {
    const size_t smem = (size_t)kMergeWaves * NPL * kWave * 8;
    hipLaunchKernelGGL(group_merge<NPL>, dim3(merge_grid(u_cap, n_cu)), dim3(kWave * kMergeWaves),
                       smem, s, ma);
    hipLaunchKernelGGL(slot_merge<NPL>, dim3(merge_grid(ma.n_pairs, n_cu)),
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
    PlanArgs pa{};
    pa.G = G;
    pa.off = seg_offsets;
    pa.qoff = w.qoff;
    pa.wstart = w.wstart;
    pa.gstart = w.gstart;
    pa.mstart = w.mstart;
    pa.pbase = w.pbase;
    pa.ubase = w.ubase;
    pa.plan = w.plan;
    pa.chunk_min = chunk_floor_rows(N, n_cu);
    pa.p_cap = w.p_cap;
    pa.group = w.group;
    const SlotOut so{slot_max, slot_sum, cand_score, cand_id, k};
    if (bc <= kFusedRoutePairs && (size_t)G * 4 <= kRouteLdsBytes) {
        hipLaunchKernelGGL(route_fused, dim3(1), dim3(kPlanThreads), (size_t)G * 4, s, pa, sel, bc,
                           w.qlist, w.pos, so);
    } else {
        hipLaunchKernelGGL(route_init, dim3((G + 255) / 256 < 1024 ? (G + 255) / 256 : 1024),
                           dim3(256), 0, s, G, w.cnt, w.cursor, w.plan);
        hipLaunchKernelGGL(route_count, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.cnt, w.plan);
        hipLaunchKernelGGL(route_plan, dim3(1), dim3(kPlanThreads), 0, s, pa, w.cnt);
        hipLaunchKernelGGL(route_scatter, dim3(gblocks), dim3(256), 0, s, sel, bc, G, w.qoff,
                           w.cursor, w.qlist, w.pos, so);
    }
    hipLaunchKernelGGL(route_items, dim3((G + 3) / 4 < 2048 ? (G + 3) / 4 : 2048), dim3(256), 0, s,
                       pa, w.qlist, w.items, w.groups, w.units, w.mlist);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    FineArgs fa{};
    fa.keys = fine_keys;
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
    err = launch_stream(key_dtype, compute_dtype, fa, bc, n_cu, w.w_max, ev, s);
    if (err != hipSuccess) return err;

    MergeArgs ma{};
    ma.sel = sel;
    ma.off = seg_offsets;
    ma.qoff = w.qoff;
    ma.pos = w.pos;
    ma.pbase = w.pbase;
    ma.ubase = w.ubase;
    ma.plan = w.plan;
    ma.groups = w.groups;
    ma.units = w.units;
    ma.mlist = w.mlist;
    ma.pm = w.pm;
    ma.pz = w.pz;
    ma.pc = w.pc;
    ma.pk = w.pk;
    ma.um = w.um;
    ma.uz = w.uz;
    ma.uc = w.uc;
    ma.uk = w.uk;
    ma.n_pairs = bc;
    ma.G = G;
    ma.k = k;
    ma.group = w.group;
    ma.cexp = cexp;
    ma.slot_max = slot_max;
    ma.slot_sum = slot_sum;
    ma.cand_score = cand_score;
    ma.cand_id = cand_id;
    switch (next_pow2(k + kWave) / kWave) {
        case 2: return launch_merge<2>(ma, w.u_cap, n_cu, s);
        case 4: return launch_merge<4>(ma, w.u_cap, n_cu, s);
        default: return launch_merge<8>(ma, w.u_cap, n_cu, s);
    }
}

}  // namespace htam
