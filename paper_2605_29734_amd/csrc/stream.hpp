// Bank-streaming kernels of the fine stage (shared by the translation units
// that instantiate them).
//
// Work item = (selected cluster g, chunk j of g's segment). One block takes an
// item from a dynamic counter and streams the chunk's key rows from HBM
// exactly once per pass, scoring them on MFMA (v_mfma_f32_16x16x32_bf16,
// keys as the 16-row A operand, queries as the 16-column B operand) against
// every query that selected g (the children of Eq. local nodes, scored as in
// Eq. local policy). Per query it keeps the online softmax statistics
// (max, sum of exp((s - max)/tau)) and a top-k of (score, caller id) keys in
// an LDS buffer behind a threshold filter. At the end of a pass it writes one
// partial (m, Z, the chunk's top-k keys unsorted) per (query, chunk).
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
constexpr int kMaxQueryTiles = 4;      // at most 64 queries per pass over a chunk

struct FineArgs {
    const void *keys;
    const int32_t *tid;
    const void *q;
    int32_t d, c, G, k, cap, qmax;
    float cexp;                   // log2(e) / tau
    const int32_t *qlist;
    const WorkItem *items;
    Plan *plan;
    float *pm, *pz;
    int32_t *pc;
    uint64_t *pk;
    float *slot_max, *slot_sum, *cand_score;   // final per-slot outputs (single-chunk clusters)
    int32_t *cand_id;
};

__host__ __device__ inline size_t fine_state_bytes(int qmax, int cap) {
    return (size_t)qmax * cap * 8 + (size_t)qmax * (8 + 4 + 4 + 4) + (size_t)2 * kFineWaves * qmax * 4;
}
__host__ __device__ inline size_t fine_qs_bytes(int d, int qmax) {
    return (size_t)((d + 31) / 32) * (qmax / 16) * kWave * 16;
}

// Launch description handed from the host code of the fine stage to the
// translation unit that holds a kernel.
struct StreamLaunch {
    FineArgs fa;
    int grid;
    size_t smem;
    int32_t qs_bytes;
    KernelEvents ev;
    hipStream_t stream;
};
hipError_t launch_stream_lds_bf16(int npl, bool has_tid, const StreamLaunch &l);
hipError_t launch_stream_lds_f32(int npl, bool has_tid, const StreamLaunch &l);
hipError_t launch_stream_generic(int key_dtype, int compute_dtype, int npl, const StreamLaunch &l);

namespace {

struct FineSmem {
    bf16x8_t *qs;      // [d/32][16-query tiles][64 lanes] query B fragments (LDS kernel)
    uint64_t *buf;     // [qmax][cap]
    uint64_t *theta;   // [qmax]
    uint32_t *cnt;     // [qmax]
    uint32_t *pend;    // [qmax] candidates counted in the current step
    int32_t *qrow;     // [qmax]
    float *wm, *wz;    // [waves][qmax]
};

__device__ __forceinline__ FineSmem fine_carve(unsigned char *raw, size_t qs_bytes, int qmax,
                                               int cap) {
    FineSmem sm;
    sm.qs = reinterpret_cast<bf16x8_t *>(raw);
    sm.buf = reinterpret_cast<uint64_t *>(raw + qs_bytes);
    sm.theta = sm.buf + (size_t)qmax * cap;
    sm.cnt = reinterpret_cast<uint32_t *>(sm.theta + qmax);
    sm.pend = sm.cnt + qmax;
    sm.qrow = reinterpret_cast<int32_t *>(sm.pend + qmax);
    sm.wm = reinterpret_cast<float *>(sm.qrow + qmax);
    sm.wz = sm.wm + kFineWaves * qmax;
    return sm;
}

// Per-pass state: the rows of the pass's queries, empty top-k buffers.
__device__ __forceinline__ void pass_begin(const FineArgs &a, const FineSmem &sm, int32_t qbeg,
                                           int32_t qg0, int32_t nqg) {
    for (int n = threadIdx.x; n < nqg; n += kFineThreads) {
        sm.qrow[n] = a.qlist[qbeg + qg0 + n] / a.c;
        sm.cnt[n] = 0;
        sm.pend[n] = 0;
        sm.theta[n] = 0;
    }
    __syncthreads();
}

// Compact the top-k buffers of this wave's queries (n = wave, wave + 4, ...)
// that cannot take their pending candidates (cnt[n] + pend[n] > cap), and
// reset pend[n] for every query of the wave. The queries are checked
// lane-parallel (lane i looks at query wave + 4 i); only the full ones are
// compacted, one after the other.
template <int NPL>
__device__ __forceinline__ void compact_wave_queries(const FineArgs &a, const FineSmem &sm, int nqg) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n_mine = lane * kFineWaves + wave;
    bool full = false;
    if (n_mine < nqg) {
        full = (int)sm.cnt[n_mine] + (int)sm.pend[n_mine] > a.cap;
        sm.pend[n_mine] = 0;
    }
    uint64_t mask = __ballot(full);
    while (mask) {
        const int i = __builtin_ctzll(mask);
        mask &= mask - 1;
        const int n = i * kFineWaves + wave;
        uint64_t th = 0;
        const int kept = compact_select<NPL>(sm.buf + (size_t)n * a.cap, (int)sm.cnt[n], a.k,
                                             kRowsPerStep, lane, th);
        if (lane == 0) {
            sm.cnt[n] = (uint32_t)kept;
            sm.theta[n] = th;
        }
        wave_lds_sync();
    }
}

// Scores of one 64-row step are in acc: this lane holds rows rt + 4*kg + e
// (e = 0..3) for query column qt*16 + r16, with caller ids tidv[e]. Folds them
// into the online (max, sum), then offers them to the queries' top-k buffers
// in three phases: count the candidates above each threshold; compact the
// buffers that could not take them (the threshold rises); append the
// candidates still above the threshold (one LDS atomic per lane and query
// tile). A buffer is compacted only when it would otherwise overflow (at most
// 64 candidates per step, and a compaction leaves at least 64 free slots).
template <int NQT, int NPL>
__device__ __forceinline__ void tile_epilogue(const FineArgs &a, const FineSmem &sm,
                                              const f32x4_t (&acc)[NQT], int64_t rt, int64_t r1,
                                              int nqg, const int32_t (&tidv)[4], float (&m)[NQT],
                                              float (&z)[NQT]) {
    const int lane = threadIdx.x & 63, r16 = lane & 15, kg = lane >> 4;
    const int cap = a.cap;
    uint64_t key[NQT][4];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        const int n = qt * 16 + r16;
        const bool vq = n < nqg;
        float tm = -INFINITY;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (vq && rt + 4 * kg + e < r1) tm = fmaxf(tm, acc[qt][e]);
        int pending = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) key[qt][e] = 0;
        if (tm != -INFINITY) {
            const float M = fmaxf(m[qt], tm);
            float zz = m[qt] == -INFINITY ? 0.0f : z[qt] * exp2f((m[qt] - M) * a.cexp);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (rt + 4 * kg + e < r1) zz += exp2f((acc[qt][e] - M) * a.cexp);
            m[qt] = M;
            z[qt] = zz;
            const uint64_t th = sm.theta[n];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (rt + 4 * kg + e < r1) {
                    const uint64_t kk = ((uint64_t)ord_of(acc[qt][e]) << 32) |
                                        (uint64_t)(~(uint32_t)tidv[e]);
                    if (kk > th) {
                        key[qt][e] = kk;
                        ++pending;
                    }
                }
            }
        }
        if (pending) atomicAdd(&sm.pend[n], (uint32_t)pending);
    }
    __syncthreads();
    compact_wave_queries<NPL>(a, sm, nqg);
    __syncthreads();
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        const int n = qt * 16 + r16;
        if (n < nqg && (key[qt][0] | key[qt][1] | key[qt][2] | key[qt][3])) {
            const uint64_t th = sm.theta[n];
            int c = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) c += key[qt][e] > th;
            if (c) {
                uint64_t *dst = sm.buf + (size_t)n * cap + atomicAdd(&sm.cnt[n], (uint32_t)c);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (key[qt][e] > th) *dst++ = key[qt][e];
            }
        }
    }
}

// End of a pass. For a chunk that is its cluster's whole segment, each query's
// (query, slot) result is final: the top-k sorted into the slot's outputs and
// the (max, sum) into slot_max / slot_sum. Otherwise each query writes one
// partial: its chunk's best k keys, in no particular order (the merge that
// reads them selects again), zero-padded to k, and the chunk's (max, sum).
template <int NQT, int NPL>
__device__ __forceinline__ void pass_end(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                         int32_t qbeg, bool single, int32_t qg0, int32_t nqg,
                                         float (&m)[NQT], float (&z)[NQT]) {
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6, r16 = lane & 15, kg = lane >> 4;
    __syncthreads();           // the last step's appends are complete
    for (int n = wave; n < nqg; n += kFineWaves) {
        uint64_t *b = sm.buf + (size_t)n * a.cap;
        int cn = (int)sm.cnt[n];
        if (single) {
            const int64_t e = a.qlist[qbeg + qg0 + n];
            uint64_t v[NPL];
#pragma unroll
            for (int q = 0; q < NPL; ++q) v[q] = (q * kWave + lane < cn) ? b[q * kWave + lane] : 0;
            wave_sort_regs<NPL>(v, lane);
#pragma unroll
            for (int q = 0; q < NPL; ++q) {
                const int r = q * kWave + lane;
                if (r < a.k) {
                    const uint64_t key = r < cn ? v[q] : 0;
                    a.cand_score[e * a.k + r] = key ? key_score(key) : -INFINITY;
                    a.cand_id[e * a.k + r] = key ? key_id(key) : -1;
                }
            }
            continue;
        }
        if (cn > a.k) {
            uint64_t th = 0;
            cn = compact_select<NPL>(b, cn, a.k, a.cap - a.k, lane, th);
        }
        const int64_t p = p0 + qg0 + n;
        for (int i = lane; i < a.k; i += kWave) a.pk[p * a.k + i] = i < cn ? b[i] : 0;
        if (lane == 0) a.pc[p] = cn;
    }
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
        for (int w = 0; w < kFineWaves; ++w)
            mz_merge(M, Z, sm.wm[w * a.qmax + n], sm.wz[w * a.qmax + n], a.cexp);
        if (single) {
            const int64_t e = a.qlist[qbeg + qg0 + n];
            a.slot_max[e] = M;
            a.slot_sum[e] = Z;
        } else {
            const int64_t p = p0 + qg0 + n;
            a.pm[p] = M;
            a.pz[p] = Z;
        }
    }
    __syncthreads();
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
    pass_begin(a, sm, qbeg, qg0, nqg);
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
        int32_t tidv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t row = rt + 4 * kg + e;
            tidv[e] = row < r1 ? (a.tid ? a.tid[row] : (int32_t)row) : -1;
        }
        tile_epilogue<NQT, NPL>(a, sm, acc, rt, r1, nqg, tidv, m, z);
    }
    pass_end<NQT, NPL>(a, sm, p0, qbeg, single, qg0, nqg, m, z);
}

// ---- LDS pass: query fragments staged in LDS, key fragments prefetched -------
// A key fragment (8 elements of one row) as it is loaded: bf16 storage is used
// as is, fp32 storage is rounded to bf16 when the fragment is consumed.
template <typename KT>
struct AFrag;
template <>
struct AFrag<__bf16> {
    static constexpr int U = 16;   // k-steps per load unit: 16 x 16 B per lane
    uint4 v;
    __device__ __forceinline__ void load(const __bf16 *p) { v = *reinterpret_cast<const uint4 *>(p); }
    __device__ __forceinline__ bf16x8_t bf16() const { return __builtin_bit_cast(bf16x8_t, v); }
};
template <>
struct AFrag<float> {
    static constexpr int U = 8;    // 8 x 32 B per lane
    float4 lo, hi;
    __device__ __forceinline__ void load(const float *p) {
        lo = reinterpret_cast<const float4 *>(p)[0];
        hi = reinterpret_cast<const float4 *>(p)[1];
    }
    __device__ __forceinline__ bf16x8_t bf16() const {
        bf16x8_t r;
        r[0] = (__bf16)lo.x; r[1] = (__bf16)lo.y; r[2] = (__bf16)lo.z; r[3] = (__bf16)lo.w;
        r[4] = (__bf16)hi.x; r[5] = (__bf16)hi.y; r[6] = (__bf16)hi.z; r[7] = (__bf16)hi.w;
        return r;
    }
};

// One load unit: U k-steps of one 16-row tile for this lane, and the caller
// ids of the lane's 4 output rows of that tile.
template <typename KT>
struct LoadUnit {
    AFrag<KT> f[AFrag<KT>::U];
    int32_t tid[4];
};

// Unconditional loads only (rows clamped into the chunk), so that the compiler
// can count outstanding loads exactly and wait for one unit at a time.
template <typename KT, bool HAS_TID>
__device__ __forceinline__ void lds_load_unit(LoadUnit<KT> &lu, const KT *__restrict__ K,
                                              const int32_t *__restrict__ tid, int d, int NG, int u,
                                              int64_t r0, int64_t r1) {
    constexpr int U = AFrag<KT>::U;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, kg = lane >> 4;
    const int tt = u / NG, gi = u - tt * NG;
    const int64_t rt = r0 + (int64_t)tt * kRowsPerStep + wave * kRowsPerWave;
    const int64_t row = min(rt + r16, r1 - 1);
    const KT *kp = K + row * d + 32 * U * gi + 8 * kg;
#pragma unroll
    for (int uu = 0; uu < U; ++uu) lu.f[uu].load(kp + 32 * uu);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int64_t rr = min(rt + 4 * kg + e, r1 - 1);
        lu.tid[e] = HAS_TID ? tid[rr] : (int32_t)rr;
    }
}

template <typename KT, int NQT, int NPL>
__device__ __forceinline__ void lds_compute_unit(const FineArgs &a, const FineSmem &sm,
                                                 const LoadUnit<KT> &lu, int NG, int u, int64_t r0,
                                                 int64_t r1, int nqg, f32x4_t (&acc)[NQT],
                                                 float (&m)[NQT], float (&z)[NQT]) {
    constexpr int U = AFrag<KT>::U;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int tt = u / NG, gi = u - tt * NG;
    const float keep = gi == 0 ? 0.0f : 1.0f;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) acc[qt] *= keep;
    const bf16x8_t *qs = sm.qs + (size_t)gi * U * NQT * kWave + lane;
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
        const bf16x8_t A = lu.f[uu].bf16();
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
            acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, qs[(uu * NQT + qt) * kWave],
                                                              acc[qt], 0, 0, 0);
    }
    if (gi == NG - 1) {
        const int64_t rt = r0 + (int64_t)tt * kRowsPerStep + wave * kRowsPerWave;
        tile_epilogue<NQT, NPL>(a, sm, acc, rt, r1, nqg, lu.tid, m, z);
    }
}

template <typename KT, bool HAS_TID, int NQT, int NPL>
__device__ __forceinline__ void pass_lds(const FineArgs &a, const FineSmem &sm, int64_t p0,
                                         bool single, int64_t r0, int64_t r1, int32_t qbeg,
                                         int32_t qg0, int32_t nqg) {
    constexpr int U = AFrag<KT>::U;
    const int t = threadIdx.x;
    const int d = a.d;
    const KT *__restrict__ K = static_cast<const KT *>(a.keys);
    const KT *__restrict__ Q = static_cast<const KT *>(a.q);
    pass_begin(a, sm, qbeg, qg0, nqg);

    // stage the queries as MFMA B fragments: [k-step][query tile][lane]
    const int KS = d >> 5;
    for (int idx = t; idx < KS * NQT * kWave; idx += kFineThreads) {
        const int s = idx / (NQT * kWave), rem = idx - s * NQT * kWave;
        const int qt = rem >> 6, ln = rem & 63;
        const int n = qt * 16 + (ln & 15), k = 32 * s + 8 * (ln >> 4);
        sm.qs[idx] = n < nqg ? load8(Q + (int64_t)sm.qrow[n] * d + k) : zero8();
    }
    __syncthreads();

    const int NG = KS / U;
    const int T = (int)((r1 - r0 + kRowsPerStep - 1) / kRowsPerStep);
    const int total = T * NG;
    float m[NQT], z[NQT];
    f32x4_t acc[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
        m[qt] = -INFINITY;
        z[qt] = 0.0f;
        acc[qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    // A ring of three load units: while unit u is multiplied (and its step's
    // epilogue runs) the loads of units u+1 and u+2 are in flight. Past the
    // end, the last unit is loaded again (an L2 hit) so that every load stays
    // unconditional and the compiler can wait for exactly one unit at a time.
    LoadUnit<KT> s0, s1, s2;
    lds_load_unit<KT, HAS_TID>(s0, K, a.tid, d, NG, 0, r0, r1);
    lds_load_unit<KT, HAS_TID>(s1, K, a.tid, d, NG, min(1, total - 1), r0, r1);
    for (int u = 0; u < total; u += 3) {
        lds_load_unit<KT, HAS_TID>(s2, K, a.tid, d, NG, min(u + 2, total - 1), r0, r1);
        lds_compute_unit<KT, NQT, NPL>(a, sm, s0, NG, u, r0, r1, nqg, acc, m, z);
        lds_load_unit<KT, HAS_TID>(s0, K, a.tid, d, NG, min(u + 3, total - 1), r0, r1);
        if (u + 1 < total) lds_compute_unit<KT, NQT, NPL>(a, sm, s1, NG, u + 1, r0, r1, nqg, acc, m, z);
        lds_load_unit<KT, HAS_TID>(s1, K, a.tid, d, NG, min(u + 4, total - 1), r0, r1);
        if (u + 2 < total) lds_compute_unit<KT, NQT, NPL>(a, sm, s2, NG, u + 2, r0, r1, nqg, acc, m, z);
    }
    pass_end<NQT, NPL>(a, sm, p0, qbeg, single, qg0, nqg, m, z);
}

// Work loop shared by both kernels: items (cluster, chunk) from the planned
// item table, the first one by block index and the rest from a dynamic
// counter; the queries of an item in passes of at most qmax.
struct ItemPass {
    int64_t p0, r0, r1;
    int32_t qbeg, nq;
    bool single;
};

__device__ __forceinline__ bool next_item(const FineArgs &a, int32_t *s_item, bool first,
                                          ItemPass &it) {
    if (threadIdx.x == 0)
        *s_item = first ? (int32_t)blockIdx.x : (int32_t)gridDim.x + atomicAdd(&a.plan->next, 1);
    __syncthreads();
    const int64_t w = *s_item;
    __syncthreads();
    if (w >= a.plan->n_items) return false;
    const WorkItem wi = a.items[w];
    it.p0 = wi.p0;
    it.r0 = wi.r0;
    it.r1 = wi.r0 + wi.len;
    it.qbeg = wi.qbeg;
    it.nq = wi.nq;
    // passes over one item cover disjoint queries, so a single-chunk item's results are final
    it.single = wi.single != 0;
    return true;
}

template <typename KT, bool HAS_TID, int NPL>
__global__ __launch_bounds__(kFineThreads) void stream_lds(FineArgs a, int32_t qs_bytes) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_item;
    const FineSmem sm = fine_carve(smem_raw, qs_bytes, a.qmax, a.cap);
    ItemPass it;
    for (bool first = true; next_item(a, &s_item, first, it); first = false) {
        for (int32_t qg0 = 0; qg0 < it.nq; qg0 += a.qmax) {
            const int32_t nqg = min(a.qmax, it.nq - qg0);
            switch ((nqg + 15) >> 4) {
                case 1: pass_lds<KT, HAS_TID, 1, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 2: pass_lds<KT, HAS_TID, 2, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 3: pass_lds<KT, HAS_TID, 3, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                default: pass_lds<KT, HAS_TID, 4, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
            }
        }
    }
}

template <typename T, bool BF16, int NPL>
__global__ __launch_bounds__(kFineThreads) void stream_generic(FineArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int32_t s_item;
    const FineSmem sm = fine_carve(smem_raw, 0, a.qmax, a.cap);
    ItemPass it;
    for (bool first = true; next_item(a, &s_item, first, it); first = false) {
        for (int32_t qg0 = 0; qg0 < it.nq; qg0 += a.qmax) {
            const int32_t nqg = min(a.qmax, it.nq - qg0);
            switch ((nqg + 15) >> 4) {
                case 1: pass_generic<T, BF16, 1, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 2: pass_generic<T, BF16, 2, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                case 3: pass_generic<T, BF16, 3, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
                default: pass_generic<T, BF16, 4, NPL>(a, sm, it.p0, it.single, it.r0, it.r1, it.qbeg, qg0, nqg); break;
            }
        }
    }
}

template <typename Kern, typename... Args>
hipError_t launch_stream_kernel(Kern kern, const StreamLaunch &l, Args... args) {
    // allow more than 64 KiB of dynamic LDS (a function attribute, not a stream operation)
    hipError_t err = hipFuncSetAttribute((const void *)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)l.smem);
    if (err != hipSuccess) return err;
    if (l.ev.before) hipEventRecord(l.ev.before, l.stream);
    hipLaunchKernelGGL(kern, dim3(l.grid), dim3(kFineThreads), l.smem, l.stream, args...);
    if (l.ev.after) hipEventRecord(l.ev.after, l.stream);
    return hipGetLastError();
}

template <typename KT>
hipError_t launch_stream_lds_t(int npl, bool has_tid, const StreamLaunch &l) {
    switch (npl * 2 + (has_tid ? 1 : 0)) {
        case 4: return launch_stream_kernel(stream_lds<KT, false, 2>, l, l.fa, l.qs_bytes);
        case 5: return launch_stream_kernel(stream_lds<KT, true, 2>, l, l.fa, l.qs_bytes);
        case 8: return launch_stream_kernel(stream_lds<KT, false, 4>, l, l.fa, l.qs_bytes);
        case 9: return launch_stream_kernel(stream_lds<KT, true, 4>, l, l.fa, l.qs_bytes);
        case 16: return launch_stream_kernel(stream_lds<KT, false, 8>, l, l.fa, l.qs_bytes);
        case 17: return launch_stream_kernel(stream_lds<KT, true, 8>, l, l.fa, l.qs_bytes);
    }
    return hipErrorInvalidValue;
}

}  // namespace
}  // namespace htam
