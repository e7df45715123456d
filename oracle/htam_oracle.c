/*
 * Plain CPU oracle for HTAM's hierarchical transition-attended retrieval.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or
 * call this file: it exists so that tests, the smoke check and the bench's
 * CPU baseline can check the GPU library against an independent, slow and
 * obviously correct definition. It shares no code, header, table or helper
 * with the HIP library.
 *
 * Paper: "HTAM: Hierarchical Transition-Attended Memory for Operator
 * Optimization" (arXiv 2605.29734).
 *
 * What is computed (each step cites the passage it follows):
 *   O0  operand quantisation to bfloat16 (round to nearest, ties to even) when
 *       the bank computes in bf16 -- the paper fixes no precision; this is the
 *       bf16-compute reading of the batched retrieval problem.
 *   O1  coarse scores  S[b][g] = <q_b, c_g>: the global-direction score of
 *       Sec. 4.3 (Eq. score) with a one-term prefix and the linear scorer
 *       phi = w^T z of App. B.6 (Eq. transition_phi), so a score is an inner
 *       product of a state embedding with a key.
 *   O2  coarse selection: the c best clusters by descending score, ties to the
 *       lower cluster id -- the greedy (epsilon = 0) limit of the softmax
 *       direction policy (Sec. 4.3, Eq. global direction; Alg. 1, Step 2),
 *       widened from one direction to c.
 *   O3  candidate set: the union of the selected clusters' child segments
 *       (Sec. 4.3, Eq. local nodes; Alg. 1, Step 3).
 *   O4  fine scores s_j = <q_b, k_j> over the candidates (Eq. local policy,
 *       with the preference score replaced by an inner product).
 *   O5  temperature softmax over the candidate set: m = max s,
 *       Z = sum exp((s - m)/tau), w_j = exp((s_j - m)/tau) / Z (the softmax
 *       form of Eq. global direction, applied to the transitions).
 *   O6  top-k: candidates ordered by descending score, ties to the lower
 *       caller transition id; the first min(k, |M_b|) kept, the rest padded
 *       with (id -1, score -inf, weight 0) -- the argmax of Eq. local policy
 *       widened to k injected memories, with the "no valid local node"
 *       fallback of App. B.7 read as an empty row.
 *   B   memory build: a stable counting sort of transition records by their
 *       parent cluster (Eq. HTG; par(l) in Eq. local nodes).
 *
 * All accumulation is in double. Products of two bf16 or two fp32 values are
 * exact in double, so O1 and O4 differ from the exact real inner product only
 * by the rounding of the double sum.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- O0: fp32 -> bf16, round to nearest even (finite inputs) ------------ */
static float oracle_bf16_of(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if ((u & 0x7f800000u) == 0x7f800000u) {
        /* inf stays inf; NaN stays NaN (quiet bit set) */
        if (u & 0x007fffffu)
            u |= 0x00400000u;
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u = (u + 0x7fffu + lsb) & 0xffff0000u;
    }
    memcpy(&x, &u, sizeof u);
    return x;
}

void htam_oracle_round_bf16(const float *x, float *y, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        y[i] = oracle_bf16_of(x[i]);
}

/* ---- O1 / O4: inner products in double ---------------------------------- */
static double oracle_dot(const float *a, const float *b, int32_t d)
{
    double s = 0.0;
    for (int32_t i = 0; i < d; ++i)
        s += (double)a[i] * (double)b[i];
    return s;
}

/* out[i][j] = <q_i, k_j> for nq queries and nk keys, row-major [nq][nk]. */
void htam_oracle_scores(int32_t nq, int64_t nk, int32_t d, const float *q,
                        const float *k, double *out)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < (int64_t)nq * nk; ++t) {
        int64_t i = t / nk, j = t % nk;
        out[t] = oracle_dot(q + i * (int64_t)d, k + j * (int64_t)d, d);
    }
}

/* ---- ordering: descending score, then ascending id ----------------------- */
typedef struct {
    double s;
    int32_t id;
} oracle_entry;

static int oracle_cmp(const void *pa, const void *pb)
{
    const oracle_entry *a = (const oracle_entry *)pa;
    const oracle_entry *b = (const oracle_entry *)pb;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    if (a->id < b->id) return -1;
    if (a->id > b->id) return 1;
    return 0;
}

/* ---- O1 + O2: coarse scores and top-c selection -------------------------- */
void htam_oracle_coarse(int32_t B, int32_t G, int32_t d, const float *q,
                        const float *ck, int32_t top_c, int32_t *sel,
                        double *sel_score)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t b = 0; b < B; ++b) {
        oracle_entry *e = (oracle_entry *)malloc(sizeof(oracle_entry) * (size_t)G);
        for (int32_t g = 0; g < G; ++g) {
            e[g].s = oracle_dot(q + (int64_t)b * d, ck + (int64_t)g * d, d);
            e[g].id = g;
        }
        qsort(e, (size_t)G, sizeof *e, oracle_cmp);
        for (int32_t j = 0; j < top_c; ++j) {
            sel[(int64_t)b * top_c + j] = e[j].id;
            sel_score[(int64_t)b * top_c + j] = e[j].s;
        }
        free(e);
    }
}

/* ---- O5 + O6 on one candidate set ----------------------------------------
 * s[n], id[n]: the candidate scores and caller ids of one row (any order).
 * Outputs: the first min(top_k, n) candidates in (-s, id) order, padded with
 * (-1, -inf, 0); *m and *Z as defined in O5 (m = -inf, Z = 0 when n = 0);
 * if w_full is not NULL it receives every candidate's weight, aligned with s.
 */
void htam_oracle_attend(int64_t n, const double *s, const int32_t *id,
                        double tau, int32_t top_k, int32_t *out_id,
                        double *out_score, double *out_weight, double *m,
                        double *Z, double *w_full)
{
    double mx = -INFINITY;
    for (int64_t j = 0; j < n; ++j)
        if (s[j] > mx) mx = s[j];
    double z = 0.0;
    for (int64_t j = 0; j < n; ++j)
        z += exp((s[j] - mx) / tau);
    *m = mx;
    *Z = z;
    if (w_full)
        for (int64_t j = 0; j < n; ++j)
            w_full[j] = exp((s[j] - mx) / tau) / z;

    oracle_entry *e = (oracle_entry *)malloc(sizeof(oracle_entry) * (size_t)(n > 0 ? n : 1));
    for (int64_t j = 0; j < n; ++j) {
        e[j].s = s[j];
        e[j].id = id[j];
    }
    qsort(e, (size_t)n, sizeof *e, oracle_cmp);
    for (int32_t r = 0; r < top_k; ++r) {
        if (r < n) {
            out_id[r] = e[r].id;
            out_score[r] = e[r].s;
            out_weight[r] = exp((e[r].s - mx) / tau) / z;
        } else {
            out_id[r] = -1;
            out_score[r] = -INFINITY;
            out_weight[r] = 0.0;
        }
    }
    free(e);
}

/* Many independent rows at once (OpenMP over rows). Row r's candidates are
 * s[off[r] .. off[r+1]) with ids id[...]; outputs are [rows][top_k] and [rows]. */
void htam_oracle_attend_rows(int64_t rows, const int64_t *off, const double *s,
                             const int32_t *id, double tau, int32_t top_k,
                             int32_t *out_id, double *out_score,
                             double *out_weight, double *m, double *Z)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r)
        htam_oracle_attend(off[r + 1] - off[r], s + off[r], id + off[r], tau,
                           top_k, out_id + r * top_k, out_score + r * top_k,
                           out_weight + r * top_k, m + r, Z + r, NULL);
}

/* ---- B: memory build (stable counting sort by parent cluster) ------------
 * seg_offsets[g] = #records whose cluster is < g  (g = 0..G);
 * transition_id lists, for g = 0, 1, ..., the input positions i with
 * cluster_of[i] == g in increasing i. Returns 0, or -1 if a cluster id is out
 * of [0, G). */
int htam_oracle_build(int64_t n, int32_t G, const int32_t *cluster_of,
                      int64_t *seg_offsets, int32_t *transition_id)
{
    for (int32_t g = 0; g <= G; ++g)
        seg_offsets[g] = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (cluster_of[i] < 0 || cluster_of[i] >= G)
            return -1;
        seg_offsets[cluster_of[i] + 1] += 1;
    }
    for (int32_t g = 0; g < G; ++g)
        seg_offsets[g + 1] += seg_offsets[g];
    int64_t *cursor = (int64_t *)malloc(sizeof(int64_t) * (size_t)(G > 0 ? G : 1));
    for (int32_t g = 0; g < G; ++g)
        cursor[g] = seg_offsets[g];
    for (int64_t i = 0; i < n; ++i)
        transition_id[cursor[cluster_of[i]]++] = (int32_t)i;
    free(cursor);
    return 0;
}
