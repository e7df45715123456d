// Bank-streaming kernels of the fine stage (shared by the translation units
// that instantiate them).
//
// Work item = (selected cluster g, chunk j of g's segment). A block of four
// waves streams the chunk's key rows from HBM exactly once per pass, scoring
// them on MFMA (v_mfma_f32_16x16x32_bf16, keys as the 16-row A operand,
// queries as the 16-column B operand) against every query that selected g
// (the children of Eq. local nodes, scored as in Eq. local policy).
//
// A step covers 64 rows: each wave multiplies 16 of them against all the
// pass's queries and writes the scores to an LDS tile (query-major). After one
// barrier each wave reads the whole step for the queries it owns (n = wave,
// wave + 4, ...), one row per lane, and keeps for them
//   - online softmax statistics per lane (max, sum of exp((s - max)/tau)),
//     reduced across the lanes when the pass ends;
//   - a top-k of (score, caller id) keys in an LDS buffer private to the
//     wave, behind a threshold filter; candidates are appended at ballot
//     prefix positions and the buffer is cut down by a radix select when it
//     could not take another step.
// No LDS atomics and no other barrier are involved. With room for two score
// tiles the steps alternate between them; with one, a second barrier per step
// keeps a step's writes behind the previous step's reads.
//
// At the end of a pass each query writes its result: the final sorted top-k
// and statistics of its (query, slot) pair when the chunk is the cluster's
// whole segment, else one partial (m, Z, the chunk's top-k keys unsorted).
//
// Two variants:
//   stream_lds      queries staged once per pass in LDS as B fragments; key
//                   fragments prefetched through a ring of three load units with
//                   branch-free loads (needs d % (32 * U) == 0);
//   stream_generic  query fragments read from global memory (any d, and the
//                   fp32-arithmetic path).
#pragma once
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

constexpr int kFineThreads = 256;      // 4 waves
constexpr int kFineWaves = kFineThreads / kWave;
constexpr int kRowsPerWave = 16;       // one MFMA tile of key rows per wave per step
constexpr int kRowsPerStep = kRowsPerWave * kFineWaves;   // rows per block per step

// The wave's index among the four waves of its role: the block's waves in
// the four-wave kernels; in the producer/consumer kernel each role has four
// (waves 0-3 stream keys, waves 4-7 keep the top-k buffers).
__device__ __forceinline__ int fine_wave() { return (threadIdx.x >> 6) & (kFineWaves - 1); }
constexpr int kMaxQueryTiles = 4;      // at most 64 queries per pass over a chunk
constexpr int kRing = 3;               // key load units in the LDS kernel's prefetch ring

struct FineArgs {
    const void *keys;
    const void *keys_tiled;       // the tiles of the keys' tiled copy, or NULL (split kernel)
    const int64_t *toff;          // the tiled copy's segment starts (its header)
    const int64_t *seg_off;       // the bank's segment offsets
    const int32_t *tid;           // caller ids, or NULL: ids are bank rows
    const int32_t *tid_src;       // tid, or (when NULL) any readable array of >= N ints
    const void *q;
    const __bf16 *q16;            // the queries rounded to bf16 ([B][d]) when the split
                                  // kernel streams fp32 keys, else NULL
    int32_t d, c, G, k, cap, qmax;
    int32_t ntile;                // score tiles in LDS (1 or 2)
    float cexp;                   // log2(e) / tau
    const int32_t *qlist;
    const WorkItem *items;
    Plan *plan;
    float *pm, *pz;
    int32_t *pc;
    uint64_t *pk;
    uint64_t *bound;   // [B*c] per pair: a key at most its k-th best (shared by its chunks)
    float *slot_max, *slot_sum, *cand_score;   // final per-slot outputs (single-chunk clusters)
    int32_t *cand_id;
};

// Epilogue lane map. A wave owns a contiguous run of qw = ceil(nqg / 4)
// queries (n = wave * qw + jq). Each owned query gets a group of RG lanes
// (jq = lane / RG, rg = lane % RG), and lane rg of the group takes the QP
// consecutive rows rg*QP .. rg*QP + QP-1 of the step (QP = 64 / RG,
// QP >= 4 * NQT >= qw), read four at a time. A query's row of the score tile
// holds kTileRow = 68 floats, which spreads every 16-lane phase of those
// 16-byte reads over all 64 banks.
constexpr int kTileRow = kRowsPerStep + 4;
template <int NQT>
struct OwnerMap {
    static constexpr int QP = NQT == 1 ? 4 : NQT == 2 ? 8 : 16;
    static constexpr int RG = kWave / QP;
};

// Floats of one score tile for passes of up to qmax queries: the step's 64
// caller ids, then one row per query.
__host__ __device__ inline size_t fine_tile_floats(int qmax) {
    return (size_t)kWave + (size_t)qmax * kTileRow;
}

// LDS of one block besides the staged queries: top-k buffers, score tiles,
// per-query hand-over slots (threshold, count) and the query rows. The
// end-of-pass softmax statistics reuse the first score tile.
__host__ __device__ inline size_t fine_state_bytes(int qmax, int cap, int ntile) {
    return (size_t)qmax * cap * 8 + (size_t)ntile * fine_tile_floats(qmax) * 4 +
           (size_t)qmax * (8 + 4 + 4 + 4);
}
__host__ __device__ inline size_t fine_qs_bytes(int d, int qmax) {
    return (size_t)((d + 31) / 32) * (qmax / 16) * kWave * 16;
}

// Launch description handed from the host code of the fine stage to the
// translation unit that holds a kernel.
struct StreamLaunch {
    FineArgs fa;
    int n_cu;                     // compute units
    int64_t max_grid;             // no more blocks than work items
    size_t smem;
    int32_t qs_bytes;
    bool producer_consumer;       // eight-wave producer/consumer blocks (one block per CU)
    bool ksplit;                  // two blocks per CU, half the query fragments staged at a time
    KernelEvents ev;
    hipStream_t stream;
};
hipError_t launch_stream_lds_bf16(int npl, bool two_per_cu, const StreamLaunch &l);
hipError_t launch_stream_lds_f32(int npl, bool two_per_cu, const StreamLaunch &l);
hipError_t launch_stream_generic(int key_dtype, int compute_dtype, int npl, const StreamLaunch &l);

namespace {

struct FineSmem {
    bf16x8_t *qs;      // [d/32][16-query tiles][64 lanes] query B fragments (LDS kernel)
    uint64_t *buf;     // [qmax][cap] top-k buffers
    float *st;         // [ntile][fine_tile_floats(qmax)] a step's caller ids, then its scores
    uint64_t *otheta;  // [qmax] owner-wave hand-over of a query's threshold
    int32_t *ocnt;     //        and buffer count
    float *wm, *wz;    // [waves][qmax] per-wave softmax statistics at the end of a pass,
    float *om, *oz;    // [qmax] and merged (both in the first score tile, then free)
    int32_t *qrow;     // [qmax] query row of each of the pass's queries
    int32_t *qpair;    // [qmax] and its (query, slot) pair index
};

__device__ __forceinline__ FineSmem fine_carve(unsigned char *raw, size_t qs_bytes, int qmax,
                                               int cap, int ntile) {
    FineSmem sm;
    sm.qs = reinterpret_cast<bf16x8_t *>(raw);
    sm.buf = reinterpret_cast<uint64_t *>(raw + qs_bytes);
    sm.st = reinterpret_cast<float *>(sm.buf + (size_t)qmax * cap);
    sm.otheta = reinterpret_cast<uint64_t *>(sm.st + (size_t)ntile * fine_tile_floats(qmax));
    sm.ocnt = reinterpret_cast<int32_t *>(sm.otheta + qmax);
    sm.qrow = sm.ocnt + qmax;
    sm.qpair = sm.qrow + qmax;
    // 2 * 4 * qmax + 2 * qmax floats <= 64 + 68 * qmax: they fit in one tile
    sm.wm = sm.st;
    sm.wz = sm.wm + kFineWaves * qmax;
    sm.om = sm.wz + kFineWaves * qmax;
    sm.oz = sm.om + qmax;
    return sm;
}

// Per-lane state of the owned query of the lane's group during a pass: the
// query's top-k buffer count and threshold (the same in every lane of the
// group).
struct OwnedLane {
    int cnt;
    uint64_t theta;
};

// Softmax statistics in the MFMA result layout: lane (r16, kg) keeps, for
// query column qt*16 + r16, the running max and sum of exp((s - max)/tau)
// over its rows (4 kg + e of each of the wave's 16-row tiles). The rows a
// lane sees do not depend on how many queries share the pass, and the lanes
// and waves are merged in a fixed order, so a query's statistics are the same
// bits whichever pass it falls in.
template <int NQT>
struct Stats {
    float m[NQT], z[NQT];
};

template <int NQT>
__device__ __forceinline__ void stats_reset(Stats<NQT> &st) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        st.m[qt] = -INFINITY;
        st.z[qt] = 0.0f;
    }
}

// Folds one step's scores (this wave's 16 rows starting at rt) into the stats.
template <int NQT>
__device__ __forceinline__ void stats_update(Stats<NQT> &st, const f32x4_t (&acc)[NQT],
                                             int64_t rt, int64_t r1, float cexp) {
#pragma clang fp contract(off)
    const int kg = (threadIdx.x & 63) >> 4;
    const int64_t nvalid = r1 - (rt + 4 * kg);    // rows of this lane's four that exist
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        float tm = -INFINITY;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (e < nvalid) tm = fmaxf(tm, acc[qt][e]);
        if (tm != -INFINITY) {
            const float M = fmaxf(st.m[qt], tm);
            float zz = st.m[qt] == -INFINITY ? 0.0f : st.z[qt] * fast_exp2((st.m[qt] - M) * cexp);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (e < nvalid) zz += fast_exp2((acc[qt][e] - M) * cexp);
            st.m[qt] = M;
            st.z[qt] = zz;
        }
    }
}

// Per-pass set-up: the (query, slot) pairs of the pass and their query rows.
// A query's shared bound as loaded by pass_begin, for pass_bound to store.
struct PassBound {
    uint64_t v = 0;
    int n = -1;            // the query whose bound this thread holds, -1: none
};

// Start of a pass: the pass's pair indices and query rows into LDS, and each
// query's starting threshold: 0 for a cluster that is one chunk, else the
// pair's shared bound (a chunk of a longer segment starts from it). Thread n
// handles query n (nqg <= qmax <= blocks' thread count). With kDefer the
// bound load is left in flight (the barrier here waits for LDS only) and the
// caller stores it with pass_bound before its next block-wide barrier, so
// that the load overlaps the query staging.
template <bool kDefer>
__device__ __forceinline__ PassBound pass_begin(const FineArgs &a, const FineSmem &sm,
                                                int32_t qbeg, int32_t qg0, int32_t nqg,
                                                bool single) {
    PassBound pb;
    if (qg0 > 0) {
        // a later pass over the same item: every wave must be done writing
        // the previous pass's results out, which reads these same slots
        block_lds_barrier();
    }
    const int n = threadIdx.x;
    if (n < nqg) {
        const int32_t e = a.qlist[qbeg + qg0 + n];
        sm.qpair[n] = e;
        sm.qrow[n] = e / a.c;
        pb.v = single ? 0 : __hip_atomic_load(a.bound + e, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
        pb.n = n;
        if constexpr (!kDefer) sm.otheta[n] = pb.v;
    }
    if constexpr (kDefer) {
        block_lds_barrier();
    } else {
        __syncthreads();
    }
    return pb;
}

__device__ __forceinline__ void pass_bound(const FineSmem &sm, const PassBound &pb) {
    if (pb.n >= 0) sm.otheta[pb.n] = pb.v;
}

// The owned query's buffer starts empty, with the threshold handed over from
// the pair's shared bound.
template <int NQT>
__device__ __forceinline__ void owned_begin(const FineSmem &sm, int nqg, OwnedLane &o) {
    constexpr int RG = OwnerMap<NQT>::RG;
    const int lane = threadIdx.x & 63, wave = fine_wave(), jq = lane / RG;
    const int qw = (nqg + kFineWaves - 1) / kFineWaves;
    const int n = wave * qw + jq;
    o.cnt = 0;
    o.theta = jq < qw && n < nqg ? sm.otheta[n] : 0;
}

// This wave's MFMA results for one step into the score tile: the lane holds
// rows 4 kg + e (e = 0..3) of the wave's 16 for query column qt*16 + r16.
// Wave 0 also stores the step's caller ids (lane = row) ahead of the scores.
template <int NQT>
__device__ __forceinline__ void tile_write(float *tile, const f32x4_t (&acc)[NQT], int32_t tid) {
    constexpr int ROW = kTileRow;
    const int lane = threadIdx.x & 63, wave = fine_wave(), r16 = lane & 15, kg = lane >> 4;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
        *reinterpret_cast<f32x4_t *>(tile + kWave + (qt * 16 + r16) * ROW + wave * kRowsPerWave +
                                     4 * kg) = acc[qt];
    if (wave == 0) reinterpret_cast<int32_t *>(tile)[lane] = tid;
}

// Sum over the RG lanes of this lane's group (the same in all of them).
template <int RG>
__device__ __forceinline__ int group_sum(int x, int lane) {
    if constexpr (RG > 1) x += (int)lane_xor32<1>((uint32_t)x, lane);
    if constexpr (RG > 2) x += (int)lane_xor32<2>((uint32_t)x, lane);
    if constexpr (RG > 4) x += (int)lane_xor32<4>((uint32_t)x, lane);
    if constexpr (RG > 8) x += (int)lane_xor32<8>((uint32_t)x, lane);
    return x;
}

// compact_select kept out of line: the stream kernels are far larger than the
// instruction cache, and a rarely taken path inlined at every step end is
// fetched from L2 each time it runs; one shared copy stays warmer.
struct Compacted {
    int n;
    uint64_t theta;
};
template <int NPL>
__device__ __noinline__ Compacted compact_cold(uint64_t *buf, int n, int k, int room) {
    Compacted r;
    r.theta = 0;
    r.n = compact_select<NPL>(buf, n, k, room, threadIdx.x & 63, r.theta);
    return r;
}

// The owned queries' share of one step (see OwnerMap). Rows at or beyond r1
// are not candidates. Each lane counts its candidates above the threshold;
// a buffer that cannot take its group's candidates is compacted (one query at
// a time by the whole wave, raising its threshold); then each lane appends
// the candidates still above the threshold at its place in the group (an
// exclusive scan of the counts over the group's lanes).
template <int NQT, int NPL>
__device__ __forceinline__ void owner_epilogue(const FineArgs &a, const FineSmem &sm,
                                               const float *tile, int64_t base, int64_t r1,
                                               int nqg, OwnedLane &o) {
    constexpr int QP = OwnerMap<NQT>::QP, RG = OwnerMap<NQT>::RG;
    const int lane = threadIdx.x & 63, wave = fine_wave();
    const int jq = lane / RG, rg = lane % RG;
    const int qw = (nqg + kFineWaves - 1) / kFineWaves;
    const int n = wave * qw + jq;
    const bool active = jq < qw && n < nqg;
    const int nn = active ? n : 0;
    const float *trow = tile + kWave + nn * kTileRow + rg * QP;
    const int32_t *tids = reinterpret_cast<const int32_t *>(tile) + rg * QP;
    const int64_t valid = active ? r1 - base - rg * QP : 0;   // of this lane's rows, those that exist
    f32x4_t s4[QP / 4];
    float mx = -INFINITY;
#pragma unroll
    for (int i4 = 0; i4 < QP; i4 += 4) {
        s4[i4 / 4] = *reinterpret_cast<const f32x4_t *>(trow + i4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (i4 + e < valid) mx = fmaxf(mx, s4[i4 / 4][e]);
    }
    // Past a buffer's first steps few rows beat its threshold: a lane whose
    // best score is below the threshold's score has no candidate (keys order
    // by score first), and a wave with no such lane is done with the step.
    if (!__ballot(mx != -INFINITY && ord_of(mx) >= (uint32_t)(o.theta >> 32))) return;
    uint64_t key[QP];
    int mine = 0;
#pragma unroll
    for (int i4 = 0; i4 < QP; i4 += 4) {
        const int4 t4 = *reinterpret_cast<const int4 *>(tids + i4);
        const int32_t tv[4] = {t4.x, t4.y, t4.z, t4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = i4 + e;
            const uint64_t kk =
                ((uint64_t)ord_of(s4[i4 / 4][e]) << 32) | (uint64_t)(~(uint32_t)tv[e]);
            key[i] = i < valid ? kk : 0;
            mine += key[i] > o.theta;
        }
    }
    if (!__ballot(mine > 0)) return;
    const int count = group_sum<RG>(mine, lane);
    uint64_t full = __ballot(active && rg == 0 && o.cnt + count > a.cap);
    if (full) {
        wave_lds_sync();
        for (; full; full &= full - 1) {
            const int l0 = __builtin_ctzll(full);
            const int n0 = wave * qw + l0 / RG;
            const int c0 = __shfl(o.cnt, l0);
            const Compacted c1 = compact_cold<NPL>(sm.buf + (size_t)n0 * a.cap, c0, a.k, kWave);
            if (jq == l0 / RG) {
                o.cnt = c1.n;
                o.theta = c1.theta > o.theta ? c1.theta : o.theta;
            }
        }
        mine = 0;
#pragma unroll
        for (int i = 0; i < QP; ++i) mine += key[i] > o.theta;
    }
    // exclusive scan of the lanes' counts within the group
    int incl = mine;
#pragma unroll
    for (int off = 1; off < RG; off <<= 1) {
        const int y = __shfl_up(incl, off, RG);
        if (rg >= off) incl += y;
    }
    const int total = __shfl(incl, jq * RG + RG - 1);
    uint64_t *b = sm.buf + (size_t)nn * a.cap + o.cnt + (incl - mine);
    int w = 0;
#pragma unroll
    for (int i = 0; i < QP; ++i) {
        if (key[i] > o.theta) b[w++] = key[i];
    }
    o.cnt += total;
}

// One step's end, common to both kernels: scores to the tile, barrier(s),
// then the owned queries' epilogue. Every wave of the block calls it the same
// number of times. tid: caller id of row base + lane (loaded with the step's
// keys, so that no load is waited for here).
template <int NQT, int NPL>
__device__ __forceinline__ void step_end(const FineArgs &a, const FineSmem &sm,
                                         const f32x4_t (&acc)[NQT], int step, int64_t base,
                                         int64_t r1, int nqg, int32_t tid, OwnedLane &o,
                                         Stats<NQT> &st) {
    stats_update<NQT>(st, acc, base + fine_wave() * kRowsPerWave, r1, a.cexp);
    float *tile = sm.st + (size_t)(a.ntile == 2 ? step & 1 : 0) * fine_tile_floats(a.qmax);
    if (a.ntile == 1) __syncthreads();      // the previous step's reads are done
    tile_write<NQT>(tile, acc, tid);
    __syncthreads();
    owner_epilogue<NQT, NPL>(a, sm, tile, base, r1, nqg, o);
}

// A producer wave's share of a step's end in the producer/consumer kernel:
// statistics, then the scores into the tile for the consumer waves (after the
// consumers are done with the tile when only one fits). The consumers make
// the same barriers in the same order, once per step.
template <int NQT>
__device__ __forceinline__ void producer_step_end(const FineArgs &a, const FineSmem &sm,
                                                  const f32x4_t (&acc)[NQT], int step,
                                                  int64_t base, int64_t r1, int32_t tid,
                                                  Stats<NQT> &st) {
    stats_update<NQT>(st, acc, base + fine_wave() * kRowsPerWave, r1, a.cexp);
    float *tile = sm.st + (size_t)(a.ntile == 2 ? step & 1 : 0) * fine_tile_floats(a.qmax);
    if (a.ntile == 1) __syncthreads();      // the consumers are done with the previous step
    tile_write<NQT>(tile, acc, tid);
    __syncthreads();
}

// Caller id of row base + lane of a step (rows past the chunk clamped). The
// load is unconditional, so that the compiler can count outstanding loads
// exactly: a bank without an id array (ids = bank rows) passes any readable
// array of at least N ints as `src`, and tid_value() replaces the loaded
// value by the row where the step uses it (a select on the loaded value at
// load time would make the compiler wait for every load in flight).
__device__ __forceinline__ int32_t step_tid_load(const int32_t *__restrict__ src, int64_t base,
                                                 int64_t r1) {
    return src[min(base + (int64_t)(threadIdx.x & 63), r1 - 1)];
}
__device__ __forceinline__ int32_t tid_value(int32_t loaded, bool identity, int64_t base,
                                             int64_t r1) {
    return identity ? (int32_t)min(base + (int64_t)(threadIdx.x & 63), r1 - 1) : loaded;
}

// End of a pass: for each owned query, the final sorted top-k and statistics
// of its (query, slot) pair when the chunk is the cluster's whole segment
// (passes over an item cover disjoint queries), else one partial: the
// chunk's best k keys unsorted and zero-padded, and (max, sum). The lanes'
// statistics are merged within each group and handed over through LDS with
// the counts, then the buffers are written out query by query.
// PC: producer/consumer block (waves 0-3 hold the statistics, waves 4-7 the
// buffers); otherwise every wave holds both.
template <int NQT, int NPL, bool PC = false>
__device__ __forceinline__ void pass_end(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                         int32_t qbeg, bool single, int32_t qg0, int32_t nqg,
                                         OwnedLane &o, Stats<NQT> &st) {
    constexpr int RG = OwnerMap<NQT>::RG;
    const int t = threadIdx.x, lane = t & 63, wave = fine_wave(), r16 = lane & 15, kg = lane >> 4;
    const bool stats_here = !PC || t < kFineThreads, buffers_here = !PC || t >= kFineThreads;
    const int jq = lane / RG, rg = lane % RG;
    const int qw = (nqg + kFineWaves - 1) / kFineWaves;
    const int n = wave * qw + jq;
    if (buffers_here && jq < qw && n < nqg && rg == 0) {
        sm.ocnt[n] = o.cnt;
        sm.otheta[n] = o.theta;
    }
    __syncthreads();           // every wave is done with the score tile, which the statistics reuse
    // statistics: the four row groups of a lane column, then the waves in order
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
        for (int sh = 16; sh <= 32; sh <<= 1) {
            const float m2 = __shfl_xor(st.m[qt], sh), z2 = __shfl_xor(st.z[qt], sh);
            mz_merge(st.m[qt], st.z[qt], m2, z2, a.cexp);
        }
        const int q = qt * 16 + r16;
        if (stats_here && kg == 0 && q < nqg) {
            sm.wm[wave * a.qmax + q] = st.m[qt];
            sm.wz[wave * a.qmax + q] = st.z[qt];
        }
    }
    __syncthreads();
    for (int q = t; q < nqg; q += blockDim.x) {
        float M = -INFINITY, Z = 0.0f;
        for (int w = 0; w < kFineWaves; ++w)
            mz_merge(M, Z, sm.wm[w * a.qmax + q], sm.wz[w * a.qmax + q], a.cexp);
        sm.om[q] = M;
        sm.oz[q] = Z;
    }
    __syncthreads();
    // the buffers are written out by every wave of the block
    const int nw = blockDim.x >> 6, wo = t >> 6, qwo = (nqg + nw - 1) / nw;
    const int n1 = min(nqg, (wo + 1) * qwo);
    if (single) {
        // final sorted results
        for (int q = wo * qwo; q < n1; ++q) {
            int cn = sm.ocnt[q];
            uint64_t *b = sm.buf + (size_t)q * a.cap;
            const int64_t e = sm.qpair[q];
            uint64_t v[NPL];
            if constexpr (NPL == 2) {
                // k <= 64: cut the buffer to at most 64 keys (all the top k)
                // when it holds more, then sort one 64-key register
                if (cn > kWave) cn = compact_cold<NPL>(b, cn, a.k, a.cap - kWave).n;
                v[0] = lane < cn ? b[lane] : 0;
                v[1] = 0;
                uint64_t(&v1)[1] = *reinterpret_cast<uint64_t(*)[1]>(&v[0]);
                wave_sort_regs<1>(v1, lane);
            } else {
#pragma unroll
                for (int j = 0; j < NPL; ++j) v[j] = (j * kWave + lane < cn) ? b[j * kWave + lane] : 0;
                wave_sort_regs<NPL>(v, lane);
            }
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                const int r = j * kWave + lane;
                if (r < a.k) {
                    const uint64_t key = r < cn ? v[j] : 0;
                    a.cand_score[e * a.k + r] = key ? key_score(key) : -INFINITY;
                    a.cand_id[e * a.k + r] = key ? key_id(key) : -1;
                }
            }
            if (lane == 0) {
                a.slot_max[e] = sm.om[q];
                a.slot_sum[e] = sm.oz[q];
            }
            wave_lds_sync();
        }
        return;
    }
    for (int q = wo * qwo; q < n1; ++q) {
        uint64_t *b = sm.buf + (size_t)q * a.cap;
        int cn = sm.ocnt[q];
        const float Mq = sm.om[q], Zq = sm.oz[q];
        uint64_t th = sm.otheta[q];
        if (cn > a.k) {
            const Compacted c = compact_cold<NPL>(b, cn, a.k, a.cap - a.k);
            cn = c.n;
            th = c.theta > th ? c.theta : th;
        }
        // At least k keys of this partial (or of the one the bound came
        // from) are at or above th, so no key below it can be among the
        // pair's top k: later chunks of the segment start from it.
        if (lane == 0 && th != 0) atomicMax(a.bound + sm.qpair[q], th);
        const int64_t p = p0 + qg0 + q;
        for (int i = lane; i < a.k; i += kWave) a.pk[p * a.k + i] = i < cn ? b[i] : 0;
        if (lane == 0) {
            a.pc[p] = cn;
            a.pm[p] = Mq;
            a.pz[p] = Zq;
        }
        wave_lds_sync();
    }
}

// ---- generic pass: query fragments read from global memory ------------------
template <typename T, bool BF16, int NQT, int NPL>
__device__ __forceinline__ void pass_generic(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                             bool single, int64_t r0, int64_t r1, int32_t qbeg,
                                             int32_t qg0, int32_t nqg) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, kg = lane >> 4;
    const int d = a.d;
    const T *K = static_cast<const T *>(a.keys);
    const T *Q = static_cast<const T *>(a.q);
    pass_begin<false>(a, sm, qbeg, qg0, nqg, single);
    const T *qp[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        const int n = qt * 16 + r16;
        qp[qt] = Q + (int64_t)sm.qrow[n < nqg ? n : 0] * d;
    }
    OwnedLane o;
    owned_begin<NQT>(sm, nqg, o);
    Stats<NQT> st;
    stats_reset<NQT>(st);
    int step = 0;
    for (int64_t base = r0; base < r1; base += kRowsPerStep, ++step) {
        const int64_t rt = base + wave * kRowsPerWave;
        const int32_t tid = tid_value(step_tid_load(a.tid_src, base, r1), a.tid == nullptr, base, r1);
        f32x4_t acc[NQT];
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (rt < r1) {
            const int64_t arow = rt + r16 < r1 ? rt + r16 : r1 - 1;
            const T *kp = K + arow * d;
            if constexpr (BF16) {
                for (int kk = kg * 8; kk - kg * 8 < d; kk += 32) {
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
        step_end<NQT, NPL>(a, sm, acc, step, base, r1, nqg, tid, o, st);
    }
    pass_end<NQT, NPL>(a, sm, p0, qbeg, single, qg0, nqg, o, st);
}

// ---- LDS pass: query fragments staged in LDS, key fragments prefetched -------
// A key fragment (8 elements of one row) as it is loaded: bf16 storage is used
// as is, fp32 storage is rounded to bf16 when the fragment is consumed.
// Key loads are non-temporal (streaming cache policy): a call reads each key
// row once, and HBM delivers such reads faster (a read probe of the stream's
// tiled units: 6.23 -> 6.70 TB/s; the stream 5.69 -> 5.36 ms on
// before_after_f32, 3.20 -> 3.02 ms on zipf_large_bf16).
typedef unsigned int ntu32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 nt_load16(const void *p) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const ntu32x4 *>(p)));
}
__device__ __forceinline__ float4 nt_load16f(const void *p) {
    return __builtin_bit_cast(float4, __builtin_nontemporal_load(reinterpret_cast<const ntu32x4 *>(p)));
}

template <typename KT>
struct AFrag;
template <>
struct AFrag<__bf16> {
    static constexpr int U = 16;   // k-steps per load unit (one-block-per-CU kernels): 16 x 16 B per lane
    uint4 v;
    __device__ __forceinline__ void load(const __bf16 *p) { v = nt_load16(p); }
    // in the tiled copy a fragment is one 16-byte piece
    __device__ __forceinline__ void load_tiled(const __bf16 *p) { load(p); }
    __device__ __forceinline__ bf16x8_t bf16() const { return __builtin_bit_cast(bf16x8_t, v); }
};
template <>
struct AFrag<float> {
    static constexpr int U = 8;    // k-steps per load unit: 8 x 32 B per lane
    float4 lo, hi;
    __device__ __forceinline__ void load(const float *p) {
        lo = nt_load16f(p);
        hi = nt_load16f(p + 4);
    }
    // in the tiled copy the fragment's second piece is 64 pieces (256 floats)
    // after the first
    __device__ __forceinline__ void load_tiled(const float *p) {
        lo = nt_load16f(p);
        hi = nt_load16f(p + 256);
    }
    __device__ __forceinline__ bf16x8_t bf16() const {
        bf16x8_t r;
        r[0] = (__bf16)lo.x; r[1] = (__bf16)lo.y; r[2] = (__bf16)lo.z; r[3] = (__bf16)lo.w;
        r[4] = (__bf16)hi.x; r[5] = (__bf16)hi.y; r[6] = (__bf16)hi.z; r[7] = (__bf16)hi.w;
        return r;
    }
};

// One load unit: U k-steps of one 16-row tile for this lane, and the caller
// id of row lane of the unit's step (used by the step's epilogue).
template <typename KT, int U>
struct LoadUnit {
    AFrag<KT> f[U];
    int32_t tid;
};

// Unconditional loads only (rows clamped into the chunk), so that the compiler
// can count outstanding loads exactly and wait for one unit at a time.
// The lane's first fragment in the keys' tiled copy for the 16 rows from bank
// row `base + 16 * wave` of a segment (copy row = bank row + shift; the 16
// rows are one tile) at k-step ks0. Rows past the item's last row read that
// row, as in the row-major layout, so that no row outside the item is read
// from memory; the tile index is then wave-uniform (scalar arithmetic) and
// the lane adds its place in the block, (kg * 16 + row % 16) * P.
template <typename KT>
__device__ __forceinline__ const KT *tiled_frag(const KT *__restrict__ K, int d, int64_t base,
                                                int64_t r1, int64_t shift, int ks0) {
    constexpr int P = 16 / (int)sizeof(KT);
    const int lane = threadIdx.x & 63, r16 = lane & 15, kg = lane >> 4;
    const int64_t wave = __builtin_amdgcn_readfirstlane(fine_wave());
    const int64_t t = min((base + shift) / 16 + wave, (r1 - 1 + shift) / 16);
    const int i = (int)((min(base + 16 * wave + r16, r1 - 1) + shift) & 15);
    return K + (t * (d >> 5) + ks0) * 512 + (kg * 16 + i) * P;
}

// The lane's first key fragment of unit u. With TILED, K is the keys' tiled
// copy, where bank row r of the item's segment is row r + shift and the unit's
// k-steps are blocks of 512 elements (unit_frag reads fragment uu).
template <typename KT, int U, bool TILED>
__device__ __forceinline__ const KT *unit_keys(const KT *__restrict__ K, int d, int NG, int u,
                                               int64_t r0, int64_t r1, int64_t shift,
                                               int64_t &base) {
    const int lane = threadIdx.x & 63, wave = fine_wave(), r16 = lane & 15, kg = lane >> 4;
    const int tt = u / NG, gi = u - tt * NG;
    base = r0 + (int64_t)tt * kRowsPerStep;
    if constexpr (TILED) {
        return tiled_frag<KT>(K, d, base, r1, shift, U * gi);
    } else {
        const int64_t row = min(base + wave * kRowsPerWave + r16, r1 - 1);
        return K + row * d + 32 * U * gi + 8 * kg;
    }
}
template <typename KT, int U, bool TILED>
__device__ __forceinline__ void unit_frag(AFrag<KT> &f, const KT *kp, int uu) {
    if constexpr (TILED) f.load_tiled(kp + 512 * uu);
    else f.load(kp + 32 * uu);
}

template <typename KT, int U, bool TILED>
__device__ __forceinline__ void lds_load_unit(LoadUnit<KT, U> &lu, const KT *__restrict__ K,
                                              const int32_t *__restrict__ tid_src, int d, int NG,
                                              int u, int64_t r0, int64_t r1, int64_t shift) {
    int64_t base;
    const KT *kp = unit_keys<KT, U, TILED>(K, d, NG, u, r0, r1, shift, base);
#pragma unroll
    for (int uu = 0; uu < U; ++uu) unit_frag<KT, U, TILED>(lu.f[uu], kp, uu);
    lu.tid = step_tid_load(tid_src, base, r1);
}

// Multiplies unit u (in lu) and requests unit nu into nx. With SPREAD the
// loads are spread between the MFMAs, one fragment per k-step, so that a wave
// that is alone on its SIMD keeps refilling its share of the memory pipeline
// while it multiplies, instead of issuing a whole unit at once and leaving
// the pipeline to drain; without it (two blocks per CU, whose waves cover for
// each other) the unit is requested before the MFMAs.
template <typename KT, int U, int NQT, int NPL, bool SPREAD, bool PC, bool TILED>
__device__ __forceinline__ void lds_compute_unit(const FineArgs &a, const FineSmem &sm,
                                                 const LoadUnit<KT, U> &lu, LoadUnit<KT, U> &nx,
                                                 const KT *__restrict__ K, int nu, int NG, int u,
                                                 bool valid, int64_t r0, int64_t r1, int64_t shift,
                                                 int nqg, f32x4_t (&acc)[NQT], OwnedLane &o,
                                                 Stats<NQT> &st) {
    const int lane = threadIdx.x & 63;
    const int tt = u / NG, gi = u - tt * NG;
    const float keep = gi == 0 ? 0.0f : 1.0f;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) acc[qt] *= keep;
    int64_t nbase;
    const KT *nkp = unit_keys<KT, U, TILED>(K, a.d, NG, nu, r0, r1, shift, nbase);
    nx.tid = step_tid_load(a.tid_src, nbase, r1);
    if (!SPREAD) {
#pragma unroll
        for (int uu = 0; uu < U; ++uu) unit_frag<KT, U, TILED>(nx.f[uu], nkp, uu);
    }
    const bf16x8_t *qs = sm.qs + (size_t)gi * U * NQT * kWave + lane;
    // Query fragments are read from LDS a few k-steps ahead of their MFMAs;
    // the scheduling barriers keep the compiler from hoisting all of them
    // (4 registers each), or the next unit's loads, to the top of the unit.
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
        if (SPREAD) unit_frag<KT, U, TILED>(nx.f[uu], nkp, uu);
        const bf16x8_t A = lu.f[uu].bf16();
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
            acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, qs[(uu * NQT + qt) * kWave],
                                                              acc[qt], 0, 0, 0);
        if ((uu & 3) == 3) __builtin_amdgcn_sched_barrier(0);
    }
    if (valid && gi == NG - 1) {
        const int64_t base = r0 + (int64_t)tt * kRowsPerStep;
        const int32_t tid = tid_value(lu.tid, a.tid == nullptr, base, r1);
        if constexpr (PC) producer_step_end<NQT>(a, sm, acc, tt, base, r1, tid, st);
        else step_end<NQT, NPL>(a, sm, acc, tt, base, r1, nqg, tid, o, st);
    }
}
// PC: producer/consumer block of eight waves. Waves 0-3 stream the keys
// (loads, MFMAs, statistics, score tiles) and never stop to keep top-k
// buffers; waves 4-7 run the owner epilogue of each step's tile while the
// producers multiply the next. Both sides meet once per step at a barrier
// (twice when only one score tile fits in LDS).
template <typename KT, int U, int NQT, int NPL, bool SPREAD, bool PC, bool TILED>
__device__ __forceinline__ void pass_lds(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                         bool single, int64_t r0, int64_t r1, int32_t qbeg,
                                         int32_t qg0, int32_t nqg, int32_t g) {
    const int t = threadIdx.x;
    const bool producer = !PC || t < kFineThreads;
    const int d = a.d;
    const KT *__restrict__ K = static_cast<const KT *>(TILED ? a.keys_tiled : a.keys);
    // the tiled copy's row of bank row r of segment g is r + shift
    const int64_t shift = TILED ? a.toff[g] - a.seg_off[g] : 0;
    const KT *__restrict__ Q = static_cast<const KT *>(a.q);
    const int KS = d >> 5;
    const int NG = KS / U;
    const int T = (int)((r1 - r0 + kRowsPerStep - 1) / kRowsPerStep);
    const int total = T * NG;

    // A ring of kRing load units: while unit u is multiplied (and its step's
    // epilogue runs) the loads of the next kRing - 1 units are in flight. Past
    // the end, the last unit is loaded again (an L2 hit) so that every load
    // stays unconditional and the compiler can wait for exactly one unit at a
    // time. The first units are requested before the queries are staged.
    // the largest top-k buffers leave fewer registers for the ring
    constexpr int R = PC ? (sizeof(KT) == 4 ? 3 : 4) : NPL < 8 ? kRing : (sizeof(KT) == 4 ? 2 : 3);
    LoadUnit<KT, U> ring[R];
    if (producer) {
#pragma unroll
        for (int j = 0; j < R - 1; ++j)
            lds_load_unit<KT, U, TILED>(ring[j], K, a.tid_src, d, NG, min(j, total - 1), r0, r1,
                                        shift);
    }

    const PassBound pb = pass_begin<true>(a, sm, qbeg, qg0, nqg, single);
    // stage the queries as MFMA B fragments: [k-step][query tile][lane], eight
    // fragments per thread loaded before any is stored. Indices past the end
    // load and store the last fragment again (the same value), so that every
    // load is consumed on every path: a load left pending on one path would
    // make the compiler drain all loads in flight at the head of the unit loop.
    {
        constexpr int kBatch = 8;
        const int nfrag = KS * NQT * kWave;
        const int nt = blockDim.x;
        for (int i0 = t; i0 < nfrag; i0 += nt * kBatch) {
            bf16x8_t f[kBatch];
#pragma unroll
            for (int b = 0; b < kBatch; ++b) {
                const int idx = min(i0 + b * nt, nfrag - 1);
                const int s = idx / (NQT * kWave), rem = idx - s * NQT * kWave;
                const int qt = rem >> 6, ln = rem & 63;
                const int n = qt * 16 + (ln & 15), k = 32 * s + 8 * (ln >> 4);
                f[b] = load8(Q + (int64_t)sm.qrow[n < nqg ? n : 0] * d + k);
            }
            // padding columns (no query) are zeroed at the store: a select on
            // a loaded value where it is loaded would wait for every load
#pragma unroll
            for (int b = 0; b < kBatch; ++b) {
                const int idx = min(i0 + b * nt, nfrag - 1);
                const int rem = idx % (NQT * kWave);
                const int n = (rem >> 6) * 16 + (rem & 15);
                sm.qs[idx] = n < nqg ? f[b] : zero8();
            }
        }
    }
    pass_bound(sm, pb);
    // The first ring units are in: no path enters the unit loop with a load
    // outstanding.
    wait_vmcnt<0>();
    __syncthreads();

    OwnedLane o;
    owned_begin<NQT>(sm, nqg, o);
    Stats<NQT> st;
    stats_reset<NQT>(st);
    f32x4_t acc[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // Whole iterations only: units past the end are multiplied too (on the
    // last unit's keys, loaded again) and have no step end. On the way back
    // to the loop head every ring slot loaded in an iteration has then been
    // consumed in it on every path; a slot still loading on some path would
    // make the compiler wait for every load in flight at each iteration.
    if (producer) {
        for (int u = 0; u < total; u += R) {
#pragma unroll
            for (int j = 0; j < R; ++j)
                lds_compute_unit<KT, U, NQT, NPL, SPREAD, PC, TILED>(
                    a, sm, ring[j], ring[(j + R - 1) % R], K, min(u + j + R - 1, total - 1), NG,
                    u + j, u + j < total, r0, r1, shift, nqg, acc, o, st);
        }
    } else {
        // consumers: one step's tile at a time, in step order
        for (int step = 0; step < T; ++step) {
            const float *tile =
                sm.st + (size_t)(a.ntile == 2 ? step & 1 : 0) * fine_tile_floats(a.qmax);
            if (a.ntile == 1) __syncthreads();
            __syncthreads();
            owner_epilogue<NQT, NPL>(a, sm, tile, r0 + (int64_t)step * kRowsPerStep, r1, nqg, o);
        }
    }
    // the ring's last loads (re-reads of the last unit) are not used: wait for
    // them here, so that no path reaches the next pass's unit loop with ring
    // registers still loading
    wait_vmcnt<0>();
    pass_end<NQT, NPL, PC>(a, sm, p0, qbeg, single, qg0, nqg, o, st);
}

// Work loop shared by both kernels: items (cluster, chunk) from the planned
// item table, the first one by block index and the rest from a dynamic
// counter, whose next value is requested when an item starts and read when it
// ends; the queries of an item in passes of at most qmax.
struct ItemPass {
    int64_t p0, r0, r1;
    int32_t qbeg, nq, g;
    bool single;
};

__device__ __forceinline__ ItemPass item_pass(const WorkItem &wi) {
    ItemPass it;
    it.p0 = wi.p0;
    it.r0 = wi.r0;
    it.r1 = wi.r0 + wi.len;
    it.qbeg = wi.qbeg;
    it.nq = wi.nq;
    it.g = wi.g;
    // passes over one item cover disjoint queries, so a single-chunk item's results are final
    it.single = wi.single != 0;
    return it;
}

// Runs body(item) for every item this block takes. s_next: two LDS words.
template <typename Body>
__device__ __forceinline__ void for_each_item(const FineArgs &a, int32_t *s_next, Body &&body) {
    // The block's own first item (the grid is at most the item table's
    // capacity) is requested together with the item count, not after it.
    // The counter is used only when there are more items than blocks:
    // otherwise no block takes a second item, and the blocks' atomics on the
    // one counter at start would hold up each block's first loads (the
    // loads complete in order behind its contended atomic).
    const int64_t n_items = a.plan->n_items;
    const WorkItem first = a.items[blockIdx.x];
    const bool more = n_items > (int64_t)gridDim.x;
    int64_t w = blockIdx.x;
    for (int parity = 0; w < n_items; parity ^= 1) {
        int32_t nxt = 0;
        if (more && threadIdx.x == 0) nxt = atomicAdd(&a.plan->next, 1);   // consumed after the item
        body(item_pass(w == (int64_t)blockIdx.x ? first : a.items[w]));
        if (threadIdx.x == 0) s_next[parity] = more ? (int32_t)gridDim.x + nxt : (int32_t)n_items;
        __syncthreads();
        // uniform: the item is then read with scalar loads, which do not
        // count against the vector loads the unit loop waits for
        w = __builtin_amdgcn_readfirstlane(s_next[parity]);
    }
}

template <typename KT, int U, int NPL, bool SPREAD, bool PC = false, bool TILED = false>
__device__ __forceinline__ void stream_lds_body(const FineArgs &a, int32_t qs_bytes,
                                                unsigned char *smem_raw, int32_t *s_next) {
    const FineSmem sm = fine_carve(smem_raw, qs_bytes, a.qmax, a.cap, a.ntile);
    for_each_item(a, s_next, [&](const ItemPass &it) {
        for (int32_t qg0 = 0; qg0 < it.nq; qg0 += a.qmax) {
            const int32_t nqg = min(a.qmax, it.nq - qg0);
            switch ((nqg + 15) >> 4) {
                case 1: pass_lds<KT, U, 1, NPL, SPREAD, PC, TILED>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg, it.g); break;
                case 2: pass_lds<KT, U, 2, NPL, SPREAD, PC, TILED>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg, it.g); break;
                case 3: pass_lds<KT, U, 3, NPL, SPREAD, PC, TILED>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg, it.g); break;
                default: pass_lds<KT, U, 4, NPL, SPREAD, PC, TILED>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg, it.g); break;
            }
        }
    });
}

// One block per CU (LDS-bound launches): all registers, long load units.
template <typename KT, int NPL>
__global__ __launch_bounds__(kFineThreads) void stream_lds(FineArgs a, int32_t qs_bytes) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_next[2];
    stream_lds_body<KT, AFrag<KT>::U, NPL, true>(a, qs_bytes, smem_raw, s_next);
}

// Two blocks per CU when their LDS fits (small query groups): registers
// capped at two waves per SIMD, so that one block's latency-bound steps
// (staging, epilogue, pass end) overlap the other's; shorter load units keep
// the ring within that budget (d must be a multiple of 256).
template <typename KT, int NPL, bool TILED>
__global__ __launch_bounds__(kFineThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void stream_lds2(FineArgs a, int32_t qs_bytes) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_next[2];
    // fp32 fragments take twice the registers: half-length units
    stream_lds_body<KT, sizeof(KT) == 4 ? 4 : 8, NPL, false, false, TILED>(a, qs_bytes, smem_raw,
                                                                         s_next);
}

// Producer/consumer blocks of eight waves, one per CU (LDS-bound launches):
// four waves stream the keys with 8-k-step units (4 for fp32 keys, whose
// fragments take twice the registers) in a ring of four (spread between the
// MFMAs), four keep the top-k buffers. Registers are capped at two waves per
// SIMD, which the two roles share.
template <typename KT, int NPL, bool TILED>
__global__ __launch_bounds__(2 * kFineThreads) void stream_pc(FineArgs a, int32_t qs_bytes) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_next[2];
    stream_lds_body<KT, sizeof(KT) == 4 ? 4 : 8, NPL, true, true, TILED>(a, qs_bytes, smem_raw,
                                                                       s_next);
}

// ---- split pass: the query fragments staged half of d at a time ------------
// When two blocks fit on a CU only with half the query fragments in LDS, a
// pass runs over its rows in groups of up to kSplitSteps steps, each group
// twice: first over the k-steps of the first half of d, keeping every step's
// partial scores in registers, then over the second half, which completes
// the scores and runs the step ends. Each half of every key row is read once;
// the queries are staged twice per group. With two blocks per CU, one
// block's staging, epilogues and pass ends overlap the other's key loads.
constexpr int kSplitSteps = 4;

// Unit u of a half (NGH units of U k-steps per step, k-steps from k0) of the
// row group starting at bank row g0: loads clamped into the chunk.
template <typename KT, int U, bool TILED>
__device__ __forceinline__ void split_load_unit(LoadUnit<KT, U> &lu, const KT *__restrict__ K,
                                                const int32_t *__restrict__ tid_src, int d,
                                                int NGH, int k0, int u, int64_t g0, int64_t r1,
                                                int64_t shift) {
    const int lane = threadIdx.x & 63, wave = fine_wave(), r16 = lane & 15, kg = lane >> 4;
    const int tt = u / NGH, gi = u - tt * NGH;
    const int64_t base = g0 + (int64_t)tt * kRowsPerStep;
    const int64_t row = min(base + wave * kRowsPerWave + r16, r1 - 1);
    const int ks0 = k0 + U * gi;
    if constexpr (TILED) {
        // K is the tiled copy, where bank row r of this segment is row r +
        // shift (a segment starts on a tile, and so does a wave's 16 rows):
        // block (row / 16, k-step) of 512 elements, this lane's first piece
        // at (kg * 16 + row % 16) * P, P = 16 / element bytes. (Per-lane
        // arithmetic here: with tiled_frag's scalar tile index this kernel
        // ran 1% slower.)
        constexpr int P = 16 / (int)sizeof(KT);
        const int64_t tr = row + shift;
        const KT *kp = K + ((tr >> 4) * (d >> 5) + ks0) * 512 + (kg * 16 + (int)(tr & 15)) * P;
#pragma unroll
        for (int uu = 0; uu < U; ++uu) lu.f[uu].load_tiled(kp + 512 * uu);
    } else {
        const KT *kp = K + row * d + 32 * ks0 + 8 * kg;
#pragma unroll
        for (int uu = 0; uu < U; ++uu) lu.f[uu].load(kp + 32 * uu);
    }
    lu.tid = step_tid_load(tid_src, base, r1);
}

// Multiplies unit u (in lu) of half h and requests unit nu into nx. A step
// starts from zero in the first half and from its partial scores in the
// second; it ends by saving them (first half) or with the step end.
template <typename KT, int U, int NQT, int NPL, bool TILED>
__device__ __forceinline__ void split_compute_unit(
    const FineArgs &a, const FineSmem &sm, const LoadUnit<KT, U> &lu, LoadUnit<KT, U> &nx,
    const KT *__restrict__ K, int nu, int NGH, int k0, int u, bool valid, int h, int64_t g0,
    int64_t r1, int64_t shift, int step0, int nqg, f32x4_t (&acc)[NQT],
    f32x4_t (&part)[kSplitSteps][NQT], OwnedLane &o, Stats<NQT> &st) {
    const int lane = threadIdx.x & 63;
    const int tt = u / NGH, gi = u - tt * NGH;
    if (gi == 0) {
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (h == 1) {
#pragma unroll
            for (int i = 0; i < kSplitSteps; ++i)
                if (i == tt) {
#pragma unroll
                    for (int qt = 0; qt < NQT; ++qt) acc[qt] = part[i][qt];
                }
        }
    }
    split_load_unit<KT, U, TILED>(nx, K, a.tid_src, a.d, NGH, k0, nu, g0, r1, shift);
    const bf16x8_t *qs = sm.qs + (size_t)gi * U * NQT * kWave + lane;
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
        const bf16x8_t A = lu.f[uu].bf16();
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
            acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, qs[(uu * NQT + qt) * kWave],
                                                              acc[qt], 0, 0, 0);
        if ((uu & 3) == 3) __builtin_amdgcn_sched_barrier(0);
    }
    if (valid && gi == NGH - 1) {
        if (h == 0) {
#pragma unroll
            for (int i = 0; i < kSplitSteps; ++i)
                if (i == tt) {
#pragma unroll
                    for (int qt = 0; qt < NQT; ++qt) part[i][qt] = acc[qt];
                }
        } else {
            const int64_t base = g0 + (int64_t)tt * kRowsPerStep;
            const int32_t tid = tid_value(lu.tid, a.tid == nullptr, base, r1);
            step_end<NQT, NPL>(a, sm, acc, step0 + tt, base, r1, nqg, tid, o, st);
        }
    }
}

template <typename KT, int U, int NQT, int NPL, bool TILED>
__device__ __forceinline__ void pass_split(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                           bool single, int64_t r0, int64_t r1, int32_t qbeg,
                                           int32_t qg0, int32_t nqg, int32_t g) {
    const int t = threadIdx.x;
    // the tiled copy's row of bank row r of segment g is r + shift
    const int64_t shift = TILED ? a.toff[g] - a.seg_off[g] : 0;
    const int d = a.d;
    const KT *__restrict__ K = static_cast<const KT *>(TILED ? a.keys_tiled : a.keys);
    // the queries in bf16: fp32 ones were rounded once per call (as the
    // staging would round them), so each half is staged in one round trip
    const __bf16 *__restrict__ Q =
        sizeof(KT) == 4 ? a.q16 : reinterpret_cast<const __bf16 *>(a.q);
    const int KH = d >> 6;             // k-steps per half of d
    const int NGH = KH / U;            // units per step and half
    const int T = (int)((r1 - r0 + kRowsPerStep - 1) / kRowsPerStep);
    constexpr int R = kRing;
    const PassBound pb = pass_begin<true>(a, sm, qbeg, qg0, nqg, single);
    OwnedLane o;
    Stats<NQT> st;
    stats_reset<NQT>(st);
    for (int tg = 0; tg < T; tg += kSplitSteps) {
        const int Tg = min(kSplitSteps, T - tg);
        const int64_t g0 = r0 + (int64_t)tg * kRowsPerStep;
        f32x4_t part[kSplitSteps][NQT];
#pragma unroll
        for (int i = 0; i < kSplitSteps; ++i)
#pragma unroll
            for (int qt = 0; qt < NQT; ++qt) part[i][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int h = 0; h < 2; ++h) {
            const int k0 = h * KH;
            const int total = Tg * NGH;
            LoadUnit<KT, U> ring[R];
            // this half's query fragments: [k-step][query tile][lane], as in
            // the full staging (padding columns zeroed at the store). The
            // ring's first units are requested behind the first batch, so that
            // the staging waits for its own loads only, and the barrier after
            // it waits for LDS only: the key loads stay in flight.
            {
                constexpr int kBatch = 8;
                const int nfrag = KH * NQT * kWave;
                const int nt = blockDim.x;
                for (int i0 = t; i0 < nfrag; i0 += nt * kBatch) {
                    bf16x8_t f[kBatch];
#pragma unroll
                    for (int b = 0; b < kBatch; ++b) {
                        const int idx = min(i0 + b * nt, nfrag - 1);
                        const int s2 = idx / (NQT * kWave), rem = idx - s2 * NQT * kWave;
                        const int qt = rem >> 6, ln = rem & 63;
                        const int n = qt * 16 + (ln & 15), k = 32 * (k0 + s2) + 8 * (ln >> 4);
                        f[b] = load8(Q + (int64_t)sm.qrow[n < nqg ? n : 0] * d + k);
                    }
                    if (i0 == t) {
#pragma unroll
                        for (int j = 0; j < R - 1; ++j)
                            split_load_unit<KT, U, TILED>(ring[j], K, a.tid_src, d, NGH, k0,
                                                          min(j, total - 1), g0, r1, shift);
                        // every wave is done with the fragments of the previous half
                        block_lds_barrier();
                    }
#pragma unroll
                    for (int b = 0; b < kBatch; ++b) {
                        const int idx = min(i0 + b * nt, nfrag - 1);
                        const int rem = idx % (NQT * kWave);
                        const int n = (rem >> 6) * 16 + (rem & 15);
                        sm.qs[idx] = n < nqg ? f[b] : zero8();
                    }
                }
            }
            if (tg == 0 && h == 0) pass_bound(sm, pb);
            block_lds_barrier();
            if (tg == 0 && h == 0) owned_begin<NQT>(sm, nqg, o);
            f32x4_t acc[NQT];
#pragma unroll
            for (int qt = 0; qt < NQT; ++qt) acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            for (int u = 0; u < total; u += R) {
#pragma unroll
                for (int j = 0; j < R; ++j)
                    split_compute_unit<KT, U, NQT, NPL, TILED>(
                        a, sm, ring[j], ring[(j + R - 1) % R], K, min(u + j + R - 1, total - 1),
                        NGH, k0, u + j, u + j < total, h, g0, r1, shift, tg, nqg, acc, part, o,
                        st);
            }
        }
    }
    // the ring's last loads (re-reads of the last unit) are not used
    wait_vmcnt<0>();
    pass_end<NQT, NPL, false>(a, sm, p0, qbeg, single, qg0, nqg, o, st);
}

// Two blocks per CU with half the query fragments staged at a time (see
// pass_split): registers capped at two waves per SIMD (the partial scores of
// a group take 16 of them: one query tile per pass, qmax == 16);
// d % (64 U) == 0.
template <typename KT, int NPL, bool TILED>
__global__ __launch_bounds__(kFineThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void stream_split(FineArgs a, int32_t qs_bytes) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_next[2];
    constexpr int U = sizeof(KT) == 4 ? 4 : 8;
    const FineSmem sm = fine_carve(smem_raw, qs_bytes, a.qmax, a.cap, a.ntile);
    for_each_item(a, s_next, [&](const ItemPass &it) {
        for (int32_t qg0 = 0; qg0 < it.nq; qg0 += a.qmax)
            pass_split<KT, U, 1, NPL, TILED>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0,
                                             min(a.qmax, it.nq - qg0), it.g);
    });
}

template <typename T, bool BF16, int NPL>
__global__ __launch_bounds__(kFineThreads) void stream_generic(FineArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_next[2];
    const FineSmem sm = fine_carve(smem_raw, 0, a.qmax, a.cap, a.ntile);
    for_each_item(a, s_next, [&](const ItemPass &it) {
        for (int32_t qg0 = 0; qg0 < it.nq; qg0 += a.qmax) {
            const int32_t nqg = min(a.qmax, it.nq - qg0);
            switch ((nqg + 15) >> 4) {
                case 1: pass_generic<T, BF16, 1, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 2: pass_generic<T, BF16, 2, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 3: pass_generic<T, BF16, 3, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                default: pass_generic<T, BF16, 4, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
            }
        }
    });
}

template <typename Kern, typename... Args>
hipError_t launch_stream_kernel_n(Kern kern, int threads, const StreamLaunch &l, Args... args) {
    // allow more than 64 KiB of dynamic LDS (a function attribute, not a stream operation)
    hipError_t err = hipFuncSetAttribute((const void *)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)l.smem);
    if (err != hipSuccess) return err;
    // as many blocks as are resident at once (registers and LDS), no more:
    // the rest of the work is handed out by the item counter
    int per_cu = 0;
    err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, l.smem);
    if (err != hipSuccess) return err;
    int64_t grid = (int64_t)l.n_cu * (per_cu > 0 ? per_cu : 1);
    if (grid > l.max_grid) grid = l.max_grid;
    if (grid < 1) grid = 1;
    launch_timed(kern, dim3((unsigned)grid), dim3(threads), l.smem, l.stream, l.ev, args...);
    return hipGetLastError();
}
template <typename Kern, typename... Args>
hipError_t launch_stream_kernel(Kern kern, const StreamLaunch &l, Args... args) {
    return launch_stream_kernel_n(kern, kFineThreads, l, args...);
}

template <typename KT>
hipError_t launch_stream_lds_t(int npl, bool two_per_cu, const StreamLaunch &l) {
    if (l.ksplit) {
        switch (npl) {
            case 2: return l.fa.keys_tiled
                               ? launch_stream_kernel(stream_split<KT, 2, true>, l, l.fa, l.qs_bytes)
                               : launch_stream_kernel(stream_split<KT, 2, false>, l, l.fa, l.qs_bytes);
            case 4: return l.fa.keys_tiled
                               ? launch_stream_kernel(stream_split<KT, 4, true>, l, l.fa, l.qs_bytes)
                               : launch_stream_kernel(stream_split<KT, 4, false>, l, l.fa, l.qs_bytes);
        }
        return hipErrorInvalidValue;
    }
    // the kernels that read the tiled copy of the keys when the bank has one
    const bool tiled = l.fa.keys_tiled != nullptr;
    if (l.producer_consumer) {
        const int th = 2 * kFineThreads;
        switch (npl) {
            case 2: return tiled ? launch_stream_kernel_n(stream_pc<KT, 2, true>, th, l, l.fa, l.qs_bytes)
                                 : launch_stream_kernel_n(stream_pc<KT, 2, false>, th, l, l.fa, l.qs_bytes);
            case 4: return tiled ? launch_stream_kernel_n(stream_pc<KT, 4, true>, th, l, l.fa, l.qs_bytes)
                                 : launch_stream_kernel_n(stream_pc<KT, 4, false>, th, l, l.fa, l.qs_bytes);
        }
        return hipErrorInvalidValue;
    }
    if (two_per_cu) {
        switch (npl) {
            case 2: return tiled ? launch_stream_kernel(stream_lds2<KT, 2, true>, l, l.fa, l.qs_bytes)
                                 : launch_stream_kernel(stream_lds2<KT, 2, false>, l, l.fa, l.qs_bytes);
            case 4: return tiled ? launch_stream_kernel(stream_lds2<KT, 4, true>, l, l.fa, l.qs_bytes)
                                 : launch_stream_kernel(stream_lds2<KT, 4, false>, l, l.fa, l.qs_bytes);
        }
        return hipErrorInvalidValue;
    }
    switch (npl) {
        case 2: return launch_stream_kernel(stream_lds<KT, 2>, l, l.fa, l.qs_bytes);
        case 4: return launch_stream_kernel(stream_lds<KT, 4>, l, l.fa, l.qs_bytes);
        case 8: return launch_stream_kernel(stream_lds<KT, 8>, l, l.fa, l.qs_bytes);
    }
    return hipErrorInvalidValue;
}

}  // namespace
}  // namespace htam
