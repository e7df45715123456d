// Internal interface between the host API (htam_api.cpp) and the kernel
// translation units: workspace layouts and kernel launchers.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace htam {

enum DType : int32_t { kF32 = 0, kBF16 = 1 };

// Optional events stamped at the start and the end of one kernel (timing
// hooks of the C ABI).
struct KernelEvents {
    hipEvent_t before = nullptr, after = nullptr;
};

// Launches kern; with events, through hipExtLaunchKernel, which stamps them
// from the kernel's own dispatch (no marker packets of their own around it).
template <typename Kern, typename... Args>
inline void launch_timed(Kern kern, dim3 grid, dim3 block, size_t smem, hipStream_t s,
                         KernelEvents ev, Args... args) {
    if (ev.before || ev.after)
        hipExtLaunchKernelGGL(kern, grid, block, (std::uint32_t)smem, s, ev.before, ev.after, 0u,
                              args...);
    else
        hipLaunchKernelGGL(kern, grid, block, smem, s, args...);
}

// Routing plan written on the device by the planning kernel of the fine stage.
struct Plan {
    int64_t chunk;     // rows per work item (chunk of a segment)
    int64_t n_items;   // work items (cluster, chunk) with at least one query
    int64_t n_parts;   // partial results (query, chunk)
    int64_t n_groups;  // level-one merge groups (clusters with more chunks than one group)
    int64_t n_l1;      // level-one merge results (query, group)
    int64_t n_merge;   // (query, slot) pairs whose cluster spans more than one chunk
    int32_t next;      // dynamic work counter of the streaming kernel
    int32_t bad_sel;   // count of selected cluster ids out of range
    int32_t bad_off;   // 1 if the bank's segment offsets are not a partition of [0, N)
    int32_t pad;
};

// One work item of the bank stream: a chunk of one selected cluster's segment,
// scored against every query that selected the cluster. The item table holds
// every full-length chunk first, then the clusters' shorter last chunks,
// longest first.
struct WorkItem {
    int64_t r0;        // first bank row
    int64_t p0;        // partial result of the item's first query (query i: p0 + i)
    int32_t len;       // rows
    int32_t g;         // cluster
    int32_t qbeg;      // first entry of the cluster's query list
    int32_t nq;        // queries that selected the cluster
    int32_t single;    // 1 if this chunk is the cluster's whole segment
    int32_t pad;
};

// Level-one merge group: up to `group` consecutive chunk partials of one
// cluster, merged for each of its queries into one result.
struct MergeGroup {
    int64_t p0;        // partial of the group's first chunk for query 0 (query i, chunk j: p0 + j*nq + i)
    int64_t u0;        // level-one result for query 0 (query i: u0 + i)
    int32_t npart;     // chunks in the group
    int32_t nq;        // queries of the cluster
};

// One (query, slot) pair the merge finishes (its cluster has more chunks than
// one, or none): n partial results at p0 + j * stride, from the chunk
// partials or, for clusters with level-one groups, from the group results.
struct MergeSlot {
    int64_t p0;
    int32_t e;         // pair index (query * c + slot)
    int32_t n;         // partial results to merge
    int32_t stride;    // queries of the cluster
    int32_t level;     // 1: the partials are level-one group results
};

// Carves a workspace into 256-byte aligned pieces; with base == nullptr it
// only measures.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *b) : base(static_cast<char *>(b)) {}
    template <typename T>
    T *take(size_t count) {
        off = (off + 255) & ~size_t(255);
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

// ---- memory build --------------------------------------------------------
struct BuildWs {
    int64_t chunk, n_chunks;
    int32_t *cnt;      // [n_chunks][G] per-chunk cluster counts, then exclusive column prefix
    int64_t *len;      // [G] segment lengths
    int32_t *err;      // [1] count of out-of-range cluster ids
};
BuildWs build_layout(void *ws, int64_t n, int32_t G, size_t *bytes);
// The tiled copy of a bank's fine keys (d % 32 == 0): a header of G + 1
// int64 segment starts in the copy (tile_header_bytes), then the tiles.
size_t tile_header_bytes(int32_t G);
hipError_t launch_tile_keys(int64_t n_rows, int32_t G, int32_t d, int32_t elem_bytes,
                            const void *keys, const int64_t *seg_offsets, void *out,
                            hipStream_t s);
hipError_t launch_build(int64_t n, int32_t G, int32_t row_bytes, const int32_t *cluster_of,
                        const void *keys_in, void *keys_out, int64_t *seg_offsets,
                        int32_t *transition_id, const BuildWs &w, hipStream_t s);

// ---- coarse scoring --------------------------------------------------------
struct CoarseWs {
    float *scores;     // [B][G]
    __bf16 *q16;       // [B][d] bf16 copy of fp32 queries (bf16 arithmetic on fp32 storage)
    __bf16 *c16;       // [G][d] bf16 copy of fp32 coarse keys
    int32_t n_seg;     // segments per score row in the top-c selection
    float *p_score;    // [B][n_seg][top_c] per-segment selections (n_seg > 1)
    int32_t *p_id;
    float *tmax;       // [B][n_tile] each row's maximum over each 64-column tile (n_seg > 1)
    int32_t n_tile;
};
CoarseWs coarse_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                       int32_t compute_dtype, int32_t top_c, size_t *bytes);
// fp32 -> bf16, round to nearest even (n % 8 == 0).
hipError_t launch_round_bf16(const float *x, __bf16 *y, int64_t n, hipStream_t s);
hipError_t launch_coarse(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         const void *coarse_keys, const void *coarse_keys_bf16, const void *q,
                         int32_t B, int32_t top_c, int32_t *sel, float *sel_score,
                         const CoarseWs &w, int n_cu, KernelEvents ev, hipStream_t s);

// The top_c of each score row of w.scores [B][G] (descending, ties to the lower id).
// With tmax (the rows' 256-column tile maxima of these scores) only the tiles
// that can hold a row's top_c are read.
hipError_t launch_select(int32_t B, int32_t G, int32_t top_c, int32_t *sel, float *sel_score,
                         const CoarseWs &w, hipStream_t s, const float *tmax = nullptr);

// ---- prefix-aware coarse scoring ----------------------------------------------
struct PrefixWs {
    CoarseWs c;        // node scores, then the combined scores, and the selection
    float *part;       // [B * Lmax][G] per (query, prefix position) edge scores
    int32_t *cnt;      // [G] pairs per source node
    int32_t *cursor;   // [G]
    int32_t *off;      // [G+1] first pair of each source in `pairs`
    int32_t *goff;     // [G+1] first group of each source
    int32_t *pairs;    // [B * Lmax] (query, position) pairs grouped by source
    int4 *groups;      // [g_max] (source, first pair, pairs, -)
    int32_t *n_groups; // [1]
    int64_t g_max;
};
PrefixWs prefix_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                       int32_t compute_dtype, int32_t lmax, int32_t top_c, size_t *bytes);
hipError_t launch_prefix(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         const void *coarse_keys, const void *edge_keys, const int32_t *prefix,
                         int32_t lmax, float lambda, const void *q, int32_t B, int32_t top_c,
                         int32_t *sel, float *sel_score, const PrefixWs &w, int n_cu,
                         KernelEvents ev, hipStream_t s);

// ---- online memory update: log-structured compaction -----------------------------
// Merged bank of (a then b) per cluster; *bad (device) is set when either
// bank's offsets are not a partition of its rows, and nothing is written then.
hipError_t launch_merge_banks(int32_t G, int32_t row_bytes, const void *keys_a,
                              const int64_t *off_a, const int32_t *id_a, int64_t n_a,
                              const void *keys_b, const int64_t *off_b, const int32_t *id_b,
                              int64_t n_b, void *keys_out, int64_t *off_out, int32_t *id_out,
                              int32_t *bad, hipStream_t s);

// Feedback statistics (record: count, then fixed-point feature sums) and the
// rule-based transition scores over them.
hipError_t launch_feedback_update(int32_t G, int32_t NB, int32_t n, const int32_t *src,
                                  const int32_t *dst, const int32_t *bucket, const float *feat,
                                  int64_t *node, int64_t *edge, int64_t *edge_bucket,
                                  hipStream_t s);
hipError_t launch_transition_scores(int32_t G, int32_t NB, int32_t B, const int32_t *prefix,
                                    int32_t lmax, const int32_t *bucket, float lambda,
                                    const float *w, int32_t min_count, const int64_t *node,
                                    const int64_t *edge, const int64_t *edge_bucket,
                                    float *scores, hipStream_t s);

// ---- sampled direction choice (Gumbel-top-k of the policy) ---------------------
struct SampledWs {
    CoarseWs c;        // scores and the selection's buffers
    float *keys;       // [B][G] perturbed log-policy keys
    float *sel_key;    // [B][top_c] keys of the selection
};
SampledWs sampled_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                         int32_t compute_dtype, int32_t top_c, size_t *bytes);
hipError_t launch_sampled(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                          const void *coarse_keys, const void *q, int32_t B, int32_t top_c,
                          float eps, float tau_g, const uint32_t *noise, uint64_t seed,
                          uint64_t offset, int32_t *sel, float *sel_score, const SampledWs &w,
                          int n_cu, KernelEvents ev, hipStream_t s);

// ---- fine stage (routing + bank stream + per-slot merge) ----------------------
struct AttendWs {
    int32_t *cnt;      // [G] queries per cluster
    // per-cluster tables of the routing (block-local prefixes on the
    // multi-block path, which adds the planning blocks' bases as it reads them)
    int32_t *qoff;     // [G+1]
    int32_t *wstart;   // [G+1] first full-length chunk item of each cluster
    int32_t *wlast;    // [G]   the cluster's shorter last chunk (-1: none)
    int32_t *gstart;   // [G+1] first level-one merge group of each cluster
    int64_t *pbase;    // [G]   first partial of each cluster
    int64_t *ubase;    // [G]   first level-one merge result of each cluster
    int32_t *mstart;   // [G+1] first entry of each cluster in mlist
    MergeSlot *mlist;  // [B*c] pairs to merge (their cluster has several chunks, or none)
    int2 *units;       // [u_cap] level-one work: (group, query position)
    int32_t *qlist;    // [B*c] (query, slot) entries grouped by cluster
    int32_t *pos;      // [B*c] position of each entry inside its cluster's list
    uint64_t *bound;   // [B*c] per pair: a key at or below its k-th best, raised as chunks finish
    Plan *plan;
    uint32_t *rbits;   // multi-block routing: per counting block, bit counts of segment lengths
    int64_t *ragg;     //   and per planning block, its totals
    WorkItem *items;   // [w_max]
    MergeGroup *groups;// [g_max]
    float *pm;         // [p_cap] partial max
    float *pz;         // [p_cap] partial sum
    int32_t *pc;       // [p_cap] partial kept count
    uint64_t *pk;      // [p_cap][k] partial keys (a chunk's top-k, unsorted, zero-padded)
    float *um, *uz;    // [u_cap] level-one merge results, same form as the partials
    int32_t *uc;
    uint64_t *uk;      // [u_cap][k]
    __bf16 *q16;       // [B][d] the queries rounded to bf16 (fp32 keys; the split stream kernel)
    int64_t p_cap;     // partial results the workspace holds (>= B*c)
    int64_t w_max;     // bound on work items
    int64_t g_max;     // bound on level-one groups
    int64_t u_cap;     // bound on level-one results
    int32_t kp;        // key slots per partial (k rounded up to a power of two)
};
AttendWs attend_layout(void *ws, int32_t d, int32_t G, int64_t N, int32_t key_bytes, int32_t B,
                       int32_t c, int32_t k, size_t *bytes);
hipError_t launch_attend(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         int64_t N, const void *fine_keys, const void *fine_keys_tiled,
                         const int64_t *seg_offsets,
                         const int32_t *transition_id, const void *q, int32_t B,
                         const int32_t *sel, int32_t c, float tau, int32_t k, float *slot_max,
                         float *slot_sum, float *cand_score, int32_t *cand_id, const AttendWs &w,
                         int n_cu, KernelEvents ev, hipStream_t s);

// Segmented row top-k: rows of n scores (row_stride apart) cut into n_seg
// segments of seg_topk_cols() columns; segment s of row r writes a list of
// seg_topk_slots(top_k) (score, id) entries holding its top_k (unsorted,
// padded with (-inf, -1)) as list r * o_lists + o_seg0 + s of o_score/o_id
// [rows][o_lists][slots], and with o_m/o_z non-null its softmax statistics
// there too. Column j's id is col_id[j] (or id_base + j without col_id).
int32_t seg_topk_cols();
int32_t seg_topk_slots(int32_t top_k);

// Row top-k over score rows [rows][n] that come with their 64-column tile
// maxima tmax [rows][ceil(n / 64)] (top_k <= 64): the top_k-th largest
// tile maximum bounds the row's top_k from below, so only the tiles whose
// maximum reaches it are read. Writes out_id / out_score [rows][top_k]
// (descending, ties to the lower column), padded with (-1, -inf).
hipError_t launch_tile_topk(int64_t rows, int64_t n, const float *score, const float *tmax,
                            int32_t top_k, int32_t *out_id, float *out_score, hipStream_t s);
hipError_t launch_seg_topk(int64_t rows, int64_t row_stride, int64_t n, const float *score,
                           const int32_t *col_id, int64_t id_base, int32_t top_k, float tau,
                           float *o_score, int32_t *o_id, float *o_m, float *o_z, int64_t o_lists,
                           int64_t o_seg0, hipStream_t s);

// S[B][n] = Q K^T over n key rows (row stride n), on the coarse GEMM kernels.
// With fp32 storage and bf16 arithmetic the 256 x 256-tile kernel reads bf16
// copies: k16 [n][d] is made here, q16 [B][d] too when convert_q. Given tmax
// ([B][ceil(n / 64)]), the 256 x 256-tile kernel also writes each row's
// maximum over each 64-column tile there and sets *tiled (else false).
hipError_t launch_scores(int32_t key_dtype, int32_t compute_dtype, int32_t d, int64_t n,
                         const void *keys, const void *q, int32_t B, float *S, __bf16 *q16,
                         __bf16 *k16, bool convert_q, int n_cu, KernelEvents ev, hipStream_t s,
                         float *tmax = nullptr, bool *tiled = nullptr,
                         const __bf16 *keys16 = nullptr);

// ---- flat retrieval (every record a candidate) --------------------------------
struct FlatWs {
    int64_t band;      // key rows scored per GEMM launch (a multiple of the segment length)
    int64_t n_lists;   // per-query partial lists over all bands
    float *scores;     // [B][band]
    __bf16 *q16, *k16; // bf16 copies (fp32 storage, bf16 arithmetic)
    float *p_score;    // [B][n_lists][k]
    int32_t *p_id;
    float *pm, *pz;    // [B][n_lists]
};
FlatWs flat_layout(void *ws, int32_t d, int64_t N, int32_t key_dtype, int32_t compute_dtype,
                   int32_t B, int32_t k, size_t *bytes);
hipError_t launch_flat(int32_t key_dtype, int32_t compute_dtype, int32_t d, int64_t N,
                       const void *fine_keys, const int32_t *transition_id, const void *q,
                       int32_t B, float tau, int32_t k, int32_t *out_id, float *out_score,
                       float *out_weight, float *row_max, float *row_sum, int32_t *out_count,
                       const FlatWs &w, int n_cu, KernelEvents ev, hipStream_t s);

// Records msg as the calling thread's last error (htam_last_error) and returns status.
int32_t report_error(int32_t status, const char *msg);

// ---- top-k merge -----------------------------------------------------------
// sorted_lists: every list is sorted by descending (score, lower id) with its
// padding at the end (htam_attend_transitions' per-slot lists), so a row
// reads each list only as far as its entries can still reach the top_k.
hipError_t launch_topk(int32_t rows, int32_t lists, int32_t k_in, const float *score,
                       const int32_t *id, const float *slot_max, const float *slot_sum, float tau,
                       int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                       float *row_max, float *row_sum, int32_t *out_count, hipStream_t s,
                       bool sorted_lists = false);

}  // namespace htam
