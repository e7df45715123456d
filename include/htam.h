/*
 * htam.h -- C ABI of the MI355X (gfx950) library for HTAM's hierarchical
 * transition-attended memory retrieval.
 *
 * Paper: "HTAM: Hierarchical Transition-Attended Memory for Operator
 * Optimization" (arXiv 2605.29734). The memory is a two-level graph
 * M = (V_G, V_GL, E_G) (Sec. 4.1, Eq. HTG): coarse global nodes, and local
 * records grouped under a parent global node. One retrieval step (Alg. 1,
 * Steps 2-3) scores every global node against the current state, picks a
 * direction (Eq. global direction), restricts the candidates to that node's
 * children (Eq. local nodes) and keeps the best-scoring children
 * (Eq. local policy), whose memories are injected into the next generation
 * (Eq. generation). This library runs that read path batched and in
 * embedding space: a state is a query vector, a global node a coarse key, a
 * local record (a before-state -> after-state transition, Eq. memory_update)
 * a fine key, and every score an inner product (the linear scorer
 * phi = w^T z of App. B.6).
 *
 * Conventions for every call:
 *   - Array arguments are DEVICE pointers (memory of the current HIP device)
 *     unless a comment says "host". Matrices are row-major and contiguous.
 *   - The caller owns every buffer, including the workspace; the library
 *     never allocates or frees device memory and keeps no pointer after a
 *     call returns.
 *   - Every call validates its arguments on the host first. On an invalid
 *     argument it returns a negative status and enqueues nothing. Otherwise it
 *     enqueues its kernels on `stream` (NULL = the null stream) and returns
 *     without waiting (htam_memory_build excepted, see there). Outputs are
 *     valid once the stream has reached that point.
 *   - HTAM_ERR_DEVICE reports a HIP error seen while enqueueing; the message
 *     is available from htam_last_error() on the calling thread.
 *   - Inputs must be finite. NaN or infinite scores give unspecified rankings.
 *   - The bank's segment offsets are checked on the device by the first kernel
 *     that reads them, before any record is indexed through them: offsets
 *     that are not a partition of the rows (off[0] = 0, nondecreasing,
 *     off[G] = N) give empty slots and no bank read. With the environment
 *     variable HTAM_VALIDATE set (to anything but "" or "0"),
 *     htam_attend_transitions waits for that check and returns
 *     HTAM_ERR_VALUE for malformed offsets or for selected cluster ids
 *     outside [0, G); this is the only case in which it synchronises.
 *   - Calls are stateless: concurrent calls on distinct streams with
 *     distinct output and workspace buffers are safe.
 */
#ifndef HTAM_H
#define HTAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;
typedef struct ihipStream_t *hipStream_t;

/* Element types. */
typedef enum { HTAM_F32 = 0, HTAM_BF16 = 1 } htam_dtype;

typedef enum {
    HTAM_OK = 0,
    HTAM_ERR_NULL = -1,      /* a required pointer is NULL                        */
    HTAM_ERR_SHAPE = -2,     /* a size or count is out of its documented range    */
    HTAM_ERR_DTYPE = -3,     /* unsupported dtype or dtype combination            */
    HTAM_ERR_VALUE = -4,     /* bad value: tau, invalid records found in build,
                                bad offsets or selections (HTAM_VALIDATE)          */
    HTAM_ERR_WORKSPACE = -5, /* workspace NULL or smaller than the size asked for */
    HTAM_ERR_ALIGN = -6,     /* a pointer is not 16-byte aligned                  */
    HTAM_ERR_DEVICE = -7     /* HIP runtime error (see htam_last_error)           */
} htam_status;

/* Limits checked by the calls. */
#define HTAM_MAX_TOP_K 256   /* 1 <= top_k <= HTAM_MAX_TOP_K                      */
#define HTAM_MAX_TOP_C 256   /* 1 <= top_c <= min(n_clusters, HTAM_MAX_TOP_C);
                                selecting every cluster of a larger bank is
                                htam_retrieve_flat                              */
#define HTAM_MAX_DIM 8192    /* 8 <= d <= HTAM_MAX_DIM, d % 8 == 0                */

/*
 * A built memory bank: the two-level memory of Sec. 4.1 (Eq. HTG) as flat
 * device arrays. Plain descriptor filled by the caller; the library reads it
 * during a call and keeps no reference.
 *
 *   d              embedding width.
 *   n_clusters     G, the number of coarse keys (global nodes V_G).
 *   n_transitions  N, the number of fine keys (local records V_GL), N < 2^31.
 *   key_dtype      storage type of coarse_keys and fine_keys.
 *   compute_dtype  arithmetic of the scores: HTAM_F32 (requires key_dtype
 *                  HTAM_F32) or HTAM_BF16 (fp32 inputs are rounded to bf16,
 *                  to nearest even, as they are loaded). Products are
 *                  accumulated in fp32 either way.
 *   coarse_keys    [G][d]  one key per cluster.
 *   fine_keys      [N][d]  records grouped by cluster: the records of cluster
 *                  g occupy rows seg_offsets[g] .. seg_offsets[g+1]-1.
 *   seg_offsets    [G+1] int64, seg_offsets[0] = 0, nondecreasing,
 *                  seg_offsets[G] = N (the children sets of Eq. local nodes).
 *   transition_id  [N] int32 caller id of each row of fine_keys, or NULL for
 *                  the row index itself. Outputs report these ids, and ties
 *                  between equal scores go to the lower id.
 *   fine_keys_tiled  NULL, or the copy written by htam_memory_tile for this
 *                  bank (fine_keys and seg_offsets as they are now): an
 *                  optional second copy of the keys that the bank stream of
 *                  htam_attend_transitions reads instead of fine_keys where
 *                  it can; results are identical either way. Requires
 *                  d % 32 == 0; 16-byte aligned.
 *   coarse_keys_bf16  NULL, or (fp32 banks computed in bf16) coarse_keys
 *                  rounded to bf16 as htam_coarse_keys_bf16 writes them:
 *                  the coarse scoring then rounds only the queries per call.
 *                  Ignored for bf16 banks; 16-byte aligned.
 */
typedef struct htam_bank {
    int32_t d;
    int32_t n_clusters;
    int64_t n_transitions;
    int32_t key_dtype;
    int32_t compute_dtype;
    const void *coarse_keys;
    const void *fine_keys;
    const int64_t *seg_offsets;
    const int32_t *transition_id;
    const void *fine_keys_tiled;
    const void *coarse_keys_bf16;
} htam_bank;

/*
 * htam_memory_build -- group transition records under their parent cluster.
 *
 * Follows Eq. HTG (each local record belongs to one global node, par(l) in
 * Eq. local nodes) and the memory append of Sec. 3 / Eq. memory_update: the
 * records arrive in any order and are laid out cluster by cluster so that a
 * cluster's children form one contiguous segment. The sort is stable: within
 * a cluster, records keep their input order.
 *
 *   n            number of records, 0 <= n < 2^31.
 *   n_clusters   G >= 1.
 *   d            key width (ignored when keys_in is NULL).
 *   key_dtype    element type of keys_in / keys_out.
 *   cluster_of   [n] int32 parent cluster of each input record, in [0, G).
 *   keys_in      [n][d] input keys in record order, or NULL to build only the
 *                offsets and ids.
 *   keys_out     [n][d] receives the keys in segment order (required iff
 *                keys_in is given; must not overlap keys_in).
 *   seg_offsets  [G+1] int64 out: segment bounds.
 *   transition_id [n] int32 out: input record index of each output row.
 *   ws, ws_bytes workspace of at least htam_memory_build_workspace_size(n, G)
 *                bytes, 256-byte aligned.
 *
 * Unlike the other calls this one waits for the stream before returning, so
 * that it can report records whose cluster id is out of range
 * (HTAM_ERR_VALUE; those records are left out of the outputs).
 */
htam_status htam_memory_build(int64_t n, int32_t n_clusters, int32_t d, int32_t key_dtype,
                              const int32_t *cluster_of, const void *keys_in, void *keys_out,
                              int64_t *seg_offsets, int32_t *transition_id, void *ws,
                              size_t ws_bytes, hipStream_t stream);
size_t htam_memory_build_workspace_size(int64_t n, int32_t n_clusters);

/*
 * htam_memory_tile -- a copy of a bank's fine keys in the order the bank
 * stream reads them (Eq. local policy scores every child of a selected
 * cluster; this only changes where each key element is stored).
 *
 * The copy starts with a header of G + 1 int64: toff[g], the copy's row of
 * segment g's first record (each segment padded to a multiple of 16 rows, so
 * toff[g] % 16 == 0 and toff[G] is the padded total), the header padded to a
 * multiple of 256 bytes. Then come the rows of the copy in tiles of 16, d cut
 * into steps of 32: block (tile t, step s) holds copy rows 16 t .. 16 t + 15,
 * elements 32 s .. 32 s + 31, at element offset (t * d / 32 + s) * 512 after
 * the header. Inside a block, element 32 s + 8 c + e of copy row 16 t + i
 * (c < 4, e < 8) sits at ((e / P) * 64 + c * 16 + i) * P + e % P, P = 16 /
 * element bytes (4 for fp32, 8 for bf16): the 16-byte pieces of one
 * matrix-core operand load of 16 rows lie next to each other, so a wave's
 * load instruction reads 1 KB of consecutive bytes instead of 16 pieces of
 * 16 rows. Copy row toff[g] + j holds bank row seg_offsets[g] + j (j below
 * the segment's length); padding rows are zero.
 *
 *   bank         a bank with fine_keys (key_dtype HTAM_F32 or HTAM_BF16),
 *                d % 32 == 0 and valid seg_offsets; its fine_keys_tiled is
 *                ignored.
 *   tiled_out    htam_memory_tile_bytes(bank) bytes (an upper bound:
 *                N / 16 + G tiles), 16-byte aligned, not overlapping
 *                fine_keys; receives the copy.
 * Asynchronous on stream; allocates nothing.
 */
htam_status htam_memory_tile(const htam_bank *bank, void *tiled_out, hipStream_t stream);
size_t htam_memory_tile_bytes(const htam_bank *bank);

/*
 * htam_coarse_keys_bf16 -- the bank's fp32 coarse keys rounded to bf16 (to
 * nearest even), the operand of the bf16 coarse scores of Eq. score, for
 * htam_bank.coarse_keys_bf16 (so that htam_retrieve_coarse does not round
 * them on every call; its results are the same either way).
 *
 *   bank   a bank with key_dtype HTAM_F32; its coarse_keys_bf16 is ignored.
 *   out    [G][d] bf16, 16-byte aligned, not overlapping coarse_keys.
 * Asynchronous on stream; allocates nothing.
 */
htam_status htam_coarse_keys_bf16(const htam_bank *bank, void *out, hipStream_t stream);

/*
 * htam_memory_merge -- online memory update, record side: fold a delta bank
 * of newly appended records into the main bank (the memory growth of
 * Eq. memory_update, Alg. 1 Step 4, kept log-structured). New records are
 * built into a small delta bank with htam_memory_build; retrieval reads both
 * banks (htam_attend_transitions on each, the per-slot lists merged by
 * htam_topk, which gives exactly the union's softmax and top-k); this call
 * compacts them into one bank: the bank htam_memory_build would make from the
 * main bank's records followed by the delta's. Per cluster g the output
 * segment holds main's rows of g, then delta's, each in their order, and
 * off_out[g] = off_a[g] + off_b[g].
 *
 *   n_clusters   G >= 1 (both banks have G segments).
 *   d, key_dtype key width and element type of both banks and of keys_out.
 *   keys_a, off_a, id_a, n_a   main bank: [n_a][d] keys, [G+1] offsets,
 *                [n_a] caller ids (required).
 *   keys_b, off_b, id_b, n_b   delta bank, the same.
 *   keys_out [n_a + n_b][d], off_out [G+1], id_out [n_a + n_b] out; keys_out
 *                must not overlap the inputs.
 *   ws, ws_bytes workspace of htam_memory_merge_workspace_size() bytes.
 * Offsets that are not a partition of their bank's rows are detected on the
 * device before any row is moved, and then nothing is written; under
 * HTAM_VALIDATE the call waits and returns HTAM_ERR_VALUE for them.
 */
htam_status htam_memory_merge(int32_t n_clusters, int32_t d, int32_t key_dtype,
                              const void *keys_a, const int64_t *off_a, const int32_t *id_a,
                              int64_t n_a, const void *keys_b, const int64_t *off_b,
                              const int32_t *id_b, int64_t n_b, void *keys_out, int64_t *off_out,
                              int32_t *id_out, void *ws, size_t ws_bytes, hipStream_t stream);
size_t htam_memory_merge_workspace_size(void);

/*
 * htam_feedback_update -- online memory update, statistics side: the
 * rule-based aggregation of step outcomes (Eq. memory_update refreshes the
 * node statistics of V_G(g_t) and the transition-edge feedback of
 * E_G(g_{t-1}, g_t), t > 1; App. B.2, B.6). A statistics record is
 * HTAM_STATS_WORDS int64: the count of observations, then the sum of each of
 * the HTAM_FEEDBACK_FEATURES outcome features in fixed point (x * 2^24,
 * rounded to nearest even). Features, in order: r_imm and r_fut (log-runtime
 * gains), then the indicators pos, succ, comp, corr, safe, cfail, corfail,
 * neg (0 or 1, or rates), then risk. Event e adds one observation to
 * node_stats[dst[e]] and, when src[e] >= 0 (not a first step), to
 * edge_stats[src][dst] and edge_bucket_stats[src][dst][bucket[e]]. The sums
 * are exact integer additions: the result does not depend on event order.
 * Events with dst or bucket out of range, or src >= G, are skipped.
 * Features must be finite with |x| < 2^38.
 *
 *   src, dst, bucket [n_events] int32; features [n_events][11] fp32;
 *   node_stats [G][12], edge_stats [G][G][12],
 *   edge_bucket_stats [G][G][n_buckets][12] int64, caller-owned, updated in
 *   place (zero them to start an empty memory).
 */
#define HTAM_FEEDBACK_FEATURES 11
#define HTAM_STATS_WORDS 12
htam_status htam_feedback_update(int32_t n_clusters, int32_t n_buckets, int32_t n_events,
                                 const int32_t *src, const int32_t *dst, const int32_t *bucket,
                                 const float *features, int64_t *node_stats, int64_t *edge_stats,
                                 int64_t *edge_bucket_stats, hipStream_t stream);

/*
 * htam_transition_scores -- the rule-based direction scores over those
 * statistics: score_b(g) = sum_{i=1..L} alpha_i phi(g_i -> g | bucket_b),
 * alpha_i = exp(-lambda (L - i)) (Eq. score, Eq. prefix_weight), with
 * phi = w^T z (App. B.6, Eq. transition_phi, Eq. transition_feature_vector):
 * z = [r_imm, r_fut, p_pos, p_succ, p_comp, p_corr, p_safe, h_ctx, -p_cfail,
 * -p_corfail, -p_neg, -rho_risk], the means of the features over the state
 * bucket's observations when it has at least min_count of them (h_ctx = 1),
 * else over all of the edge's (h_ctx = 0); an edge never observed scores 0
 * (the default prior). A query with an empty prefix scores w^T z of the node
 * statistics of g (h_ctx = 0), as the first step does.
 *
 *   prefix [n_queries][max_prefix] (ends at the first entry outside [0, G)),
 *   bucket [n_queries] the state bucket of each query (clamped into range),
 *   w [12] fp32, scores [n_queries][G] fp32 out (select from them with
 *   htam_topk, cand_id NULL). Arithmetic in double.
 */
htam_status htam_transition_scores(int32_t n_clusters, int32_t n_buckets, int32_t n_queries,
                                   const int32_t *prefix, int32_t max_prefix,
                                   const int32_t *bucket, float lambda, const float *w,
                                   int32_t min_count, const int64_t *node_stats,
                                   const int64_t *edge_stats, const int64_t *edge_bucket_stats,
                                   float *scores, hipStream_t stream);

/*
 * htam_retrieve_coarse -- score every cluster and keep the best top_c.
 *
 * Alg. 1, Step 2: the score of each global node for the current state
 * (Eq. score, with a one-term prefix and the linear scorer of App. B.6, so
 * score = <q_b, c_g>), followed by the direction choice of Eq. global
 * direction in its greedy limit (epsilon = 0), widened from one direction to
 * the top_c best.
 *
 *   q            [n_queries][d] query embeddings, element type q_dtype
 *                (HTAM_BF16 queries require compute_dtype HTAM_BF16).
 *   top_c        1 <= top_c <= min(G, HTAM_MAX_TOP_C).
 *   sel_cluster  [n_queries][top_c] int32 out: cluster ids by descending
 *                score, ties to the lower cluster id.
 *   sel_score    [n_queries][top_c] fp32 out (may be NULL): their scores.
 *   ws, ws_bytes workspace of htam_retrieve_coarse_workspace_size() bytes.
 */
htam_status htam_retrieve_coarse(const htam_bank *bank, const void *q, int32_t q_dtype,
                                 int32_t n_queries, int32_t top_c, int32_t *sel_cluster,
                                 float *sel_score, void *ws, size_t ws_bytes, hipStream_t stream);
size_t htam_retrieve_coarse_workspace_size(const htam_bank *bank, int32_t n_queries, int32_t top_c);

/*
 * htam_retrieve_coarse_sampled -- the stochastic direction choice of Alg. 1,
 * Step 2 (g_t ~ mu_g), drawn top_c times without replacement. The policy of
 * Eq. global direction over every cluster,
 *     mu(g) = epsilon / G + (1 - epsilon) softmax(score / tau_g)(g),
 * (epsilon-uniform exploration plus the temperature softmax of the one-term
 * coarse scores <q_b, c_g>) is sampled by the Gumbel-top-k construction:
 * cluster g's key is log mu(g) + Gumbel(u_bg), and the top_c keys are a draw
 * of top_c clusters one after another without replacement from mu.
 *
 *   epsilon      exploration weight, 0 <= epsilon <= 1.
 *   tau_g        policy temperature, finite and > 0 (as tau_g -> 0 with
 *                epsilon = 0 the draw becomes the greedy top_c).
 *   noise        [n_queries][G] uint32 uniform words (u = (x + 1/2) / 2^32),
 *                or NULL: the library draws them from Philox4x32-10 with key
 *                (seed low, seed high) and counter (g / 4, b, offset low,
 *                offset high), word g % 4, so a draw depends only on
 *                (seed, offset, b, g) (use a new offset for a new draw).
 *   sel_cluster  [n_queries][top_c] out: the drawn clusters in draw order
 *                (descending key; ties to the lower cluster id).
 *   sel_score    [n_queries][top_c] out or NULL: their coarse scores.
 *   ws, ws_bytes workspace of htam_retrieve_coarse_sampled_workspace_size().
 */
htam_status htam_retrieve_coarse_sampled(const htam_bank *bank, const void *q, int32_t q_dtype,
                                         int32_t n_queries, int32_t top_c, float epsilon,
                                         float tau_g, const uint32_t *noise, uint64_t seed,
                                         uint64_t offset, int32_t *sel_cluster, float *sel_score,
                                         void *ws, size_t ws_bytes, hipStream_t stream);
size_t htam_retrieve_coarse_sampled_workspace_size(const htam_bank *bank, int32_t n_queries,
                                                   int32_t top_c);

/*
 * htam_retrieve_coarse_prefix -- prefix-aware scoring of every cluster, then
 * the best top_c: htam_retrieve_coarse with the transition-attended score of
 * Sec. 4.3 (Eq. score, with the position-aware weights of Eq. prefix_weight;
 * the edge memories of App. A.1 and App. B.2). For query b with prefix
 * p_b = (g_1, ..., g_L) of previously chosen directions (g_L the most
 * recent), the score of cluster g is
 *     sum_{i=1..L} alpha_i <q_b, E[g_i][g]>,  alpha_i = exp(-lambda (L - i)),
 * each term the state-conditioned transition utility of the edge g_i -> g
 * (the linear scorer of App. B.6 as an inner product with an edge key). A
 * query with an empty prefix (the first step, which reads no edge) is scored
 * by the node keys, <q_b, c_g>, as in htam_retrieve_coarse.
 *
 *   edge_keys    [G][G][d] edge keys E[src][dst], element type key_dtype,
 *                16-byte aligned (the complete directed pair space of App. B.2).
 *   prefix       [n_queries][max_prefix] int32: row b lists g_1, ..., g_L and
 *                ends at its first entry outside [0, G) (pad with -1).
 *   max_prefix   1 <= max_prefix <= HTAM_MAX_PREFIX.
 *   lambda       recency decay, finite and >= 0 (0: every edge weighs 1).
 *   q, q_dtype, n_queries, top_c, sel_cluster, sel_score as in
 *                htam_retrieve_coarse (ties to the lower cluster id).
 *   ws, ws_bytes workspace of htam_retrieve_coarse_prefix_workspace_size()
 *                bytes.
 * The kernel timing hook HTAM_KERNEL_COARSE stamps the edge-score GEMM.
 */
#define HTAM_MAX_PREFIX 16
htam_status htam_retrieve_coarse_prefix(const htam_bank *bank, const void *edge_keys,
                                        const int32_t *prefix, int32_t max_prefix, float lambda,
                                        const void *q, int32_t q_dtype, int32_t n_queries,
                                        int32_t top_c, int32_t *sel_cluster, float *sel_score,
                                        void *ws, size_t ws_bytes, hipStream_t stream);
size_t htam_retrieve_coarse_prefix_workspace_size(const htam_bank *bank, int32_t n_queries,
                                                  int32_t max_prefix, int32_t top_c);

/*
 * htam_attend_transitions -- stream the selected clusters' transition
 * segments, with softmax statistics and top-k per selected cluster.
 *
 * Alg. 1, Step 3: the candidates of a query are the children of its selected
 * clusters (Eq. local nodes). Each candidate is scored by <q_b, k_j> (the
 * preference score of Eq. local policy, as an inner product), and for every
 * (query b, slot s) with cluster g = sel_cluster[b][s] this call returns:
 *   slot_max[b][s]  m = max of the scores over segment g (-inf if empty);
 *   slot_sum[b][s]  Z = sum over segment g of exp((score - m) / tau)
 *                   (0 if empty): the temperature softmax of Eq. global
 *                   direction applied to the transitions, in a form that
 *                   merges across slots;
 *   cand_score[b][s][0..top_k-1], cand_id[b][s][...]: the top_k records of
 *                   segment g by descending score, ties to the lower caller
 *                   id; padded with score -inf and id -1 when the segment is
 *                   shorter than top_k.
 * Scores are raw inner products (not divided by tau).
 *
 *   sel_cluster  [n_queries][top_c] int32, each in [0, G) (as produced by
 *                htam_retrieve_coarse; a query's clusters must be distinct
 *                for the union of htam_topk to be a set). An id outside
 *                [0, G) gives an empty slot (HTAM_ERR_VALUE under
 *                HTAM_VALIDATE).
 *   tau          temperature, finite and > 0.
 *   top_k        1 <= top_k <= HTAM_MAX_TOP_K.
 *   ws, ws_bytes workspace of htam_attend_transitions_workspace_size() bytes.
 */
htam_status htam_attend_transitions(const htam_bank *bank, const void *q, int32_t q_dtype,
                                    int32_t n_queries, const int32_t *sel_cluster, int32_t top_c,
                                    float tau, int32_t top_k, float *slot_max, float *slot_sum,
                                    float *cand_score, int32_t *cand_id, void *ws,
                                    size_t ws_bytes, hipStream_t stream);
size_t htam_attend_transitions_workspace_size(const htam_bank *bank, int32_t n_queries,
                                              int32_t top_c, int32_t top_k);

/*
 * htam_topk -- merge candidate lists into the memories to inject.
 *
 * The argmax of Eq. local policy widened to top_k injected memories, taken
 * over the union of a query's selected segments (the weights are the
 * temperature softmax over that union). With the App. B.7 fallback read as:
 * a row with fewer than top_k candidates is padded, an empty row is invalid
 * (count 0, row_max -inf, row_sum 0).
 *
 * Row b's candidates are the n_lists * k_in entries cand_score[b][..][..] with
 * cand_id >= 0 (entries with id < 0 are padding and are skipped). If cand_id
 * is NULL, every entry is a candidate and its id is its position
 * 0 .. n_lists*k_in-1 within the row (a plain row-wise top-k over a dense
 * score matrix). Entries need not be sorted.
 *
 *   slot_max, slot_sum  [n_rows][n_lists] per-list softmax statistics as
 *                returned by htam_attend_transitions, or both NULL. When given,
 *                the row's statistics are merged from them:
 *                row_max = max_l m_l, row_sum = sum_l Z_l exp((m_l - row_max)/tau),
 *                and out_weight = exp((score - row_max)/tau) / row_sum.
 *                When NULL, row_max, row_sum and out_weight must be NULL too.
 *   out_id, out_score [n_rows][top_k] out: by descending score, ties to the
 *                lower id, padded with (-1, -inf).
 *   out_weight   [n_rows][top_k] out or NULL (padding weight 0).
 *   row_max, row_sum [n_rows] out or NULL.
 *   out_count    [n_rows] out or NULL: min(top_k, number of candidates).
 *   tau          finite and > 0 (unused without slot statistics).
 *   top_k        1 <= top_k <= HTAM_MAX_TOP_K.
 */
htam_status htam_topk(int32_t n_rows, int32_t n_lists, int32_t k_in, const float *cand_score,
                      const int32_t *cand_id, const float *slot_max, const float *slot_sum,
                      float tau, int32_t top_k, int32_t *out_id, float *out_score,
                      float *out_weight, float *row_max, float *row_sum, int32_t *out_count,
                      hipStream_t stream);

/*
 * htam_topk_sorted -- htam_topk for lists that are each sorted, as
 * htam_attend_transitions returns its per-slot lists: by descending score,
 * ties to the lower id, padding (id -1) only at the end of a list (with
 * cand_id NULL: by descending score, ties to the lower position). The same
 * arguments and the same outputs as htam_topk on such lists, bit for bit.
 * With m = ceil(top_k / n_lists), at least top_k entries score at least the
 * lowest of the lists' m-th entries, so no entry below it can be among the
 * top_k (the argmax of Eq. local policy widened to top_k needs only the best
 * entries of each list); each list is read only as far as its entries can
 * still reach the row's top_k. Lists that are not sorted give undefined
 * (but in-bounds) results. Rows of more than 64 lists, or of lists shorter
 * than 128 entries, are merged as by htam_topk.
 */
htam_status htam_topk_sorted(int32_t n_rows, int32_t n_lists, int32_t k_in,
                             const float *cand_score, const int32_t *cand_id,
                             const float *slot_max, const float *slot_sum, float tau,
                             int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                             float *row_max, float *row_sum, int32_t *out_count,
                             hipStream_t stream);

/*
 * htam_retrieve_flat -- flat memory retrieval: the baseline without a
 * hierarchy, in which every record of the memory is a candidate of every
 * query (the "Flat Memory Retrieval" row of Table 1 and App. C.4; the
 * "w/o hierarchy" ablation of Sec. 5.5). Scores are <q_b, k_j> over all N
 * rows of fine_keys (seg_offsets and coarse_keys are not read), the weights
 * the temperature softmax over all N, and the result the top_k records by
 * descending score, ties to the lower caller id. It equals the row outputs of
 * the hierarchical path when every cluster is selected.
 *
 *   q            [n_queries][d], element type q_dtype (as in the other calls).
 *   tau          temperature, finite and > 0.
 *   top_k        1 <= top_k <= HTAM_MAX_TOP_K.
 *   out_id, out_score [n_queries][top_k] out: by descending score, ties to
 *                the lower caller id, padded with (-1, -inf) when N < top_k.
 *   out_weight   [n_queries][top_k] out or NULL: exp((s - row_max)/tau)/row_sum
 *                (padding 0).
 *   row_max, row_sum [n_queries] out or NULL: max over all N scores, and the
 *                sum of exp((s - row_max)/tau) (-inf and 0 when N = 0).
 *   out_count    [n_queries] out or NULL: min(top_k, N).
 *   ws, ws_bytes workspace of htam_retrieve_flat_workspace_size() bytes
 *                (the score buffer is bounded: the bank is scored in bands).
 * The kernel timing hook HTAM_KERNEL_COARSE stamps this call's score GEMM
 * launches (the last band's when there are several).
 */
htam_status htam_retrieve_flat(const htam_bank *bank, const void *q, int32_t q_dtype,
                               int32_t n_queries, float tau, int32_t top_k, int32_t *out_id,
                               float *out_score, float *out_weight, float *row_max,
                               float *row_sum, int32_t *out_count, void *ws, size_t ws_bytes,
                               hipStream_t stream);
size_t htam_retrieve_flat_workspace_size(const htam_bank *bank, int32_t n_queries, int32_t top_k);

/*
 * htam_attend_transitions_noalloc -- htam_attend_transitions without a caller
 * workspace, for callers that cannot allocate device memory (code under
 * stream capture, serving loops that must not allocate, harnesses that forbid
 * it). Same arguments, outputs, checks and results as htam_attend_transitions
 * (same kernels), with the workspace taken from a file-scope device array of
 * HTAM_NOALLOC_SCRATCH_MIB MiB that each GPU the library runs on holds until
 * the process ends. Calls that need more workspace than that (see
 * htam_attend_transitions_workspace_size) return HTAM_ERR_WORKSPACE and
 * enqueue nothing. The call allocates nothing. All calls on one GPU share its
 * array: calls that overlap in time on one GPU (on different streams, or from
 * different threads) race and must be serialised by the caller.
 */
#define HTAM_NOALLOC_SCRATCH_MIB 64
htam_status htam_attend_transitions_noalloc(const htam_bank *bank, const void *q, int32_t q_dtype,
                                            int32_t n_queries, const int32_t *sel_cluster,
                                            int32_t top_c, float tau, int32_t top_k,
                                            float *slot_max, float *slot_sum, float *cand_score,
                                            int32_t *cand_id, hipStream_t stream);

/*
 * Diagnostics: kernel timing hooks. After htam_set_kernel_events(which, before,
 * after) with two hipEvent_t handles (passed as void *), every later call on
 * the calling thread that launches kernel `which` has `before` stamped at that
 * kernel's start and `after` at its end (by the kernel's own dispatch, through
 * hipExtLaunchKernel), so that hipEventElapsedTime gives the kernel's own
 * duration. NULL handles switch the hook off. The events are owned by the
 * caller.
 *   HTAM_KERNEL_COARSE  the coarse scoring kernel (htam_retrieve_coarse);
 *   HTAM_KERNEL_STREAM  the bank-streaming kernel (htam_attend_transitions).
 */
#define HTAM_KERNEL_COARSE 0
#define HTAM_KERNEL_STREAM 1
htam_status htam_set_kernel_events(int32_t which, void *before, void *after);

/* Human-readable name of a status, and the last error message of the calling thread. */
const char *htam_status_string(htam_status status);
const char *htam_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HTAM_H */
