// Host side of the C ABI declared in include/htam.h: argument validation
// (before anything is enqueued), workspace sizing, and kernel sequencing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <string>

#include "../../include/htam.h"
#include "internal.hpp"

#define HTAM_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_last_error;
thread_local htam::KernelEvents g_events[2];

htam_status fail(htam_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
htam_status fail(htam_status st, const char *fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(msg, sizeof msg, fmt, ap);
    va_end(ap);
    g_last_error = msg;
    return st;
}

htam_status ok() {
    g_last_error.clear();
    return HTAM_OK;
}

htam_status device_status(hipError_t e, const char *where) {
    if (e == hipSuccess) return ok();
    return fail(HTAM_ERR_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned256(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }
int dtype_bytes(int32_t t) { return t == HTAM_BF16 ? 2 : 4; }
bool valid_dtype(int32_t t) { return t == HTAM_F32 || t == HTAM_BF16; }

htam_status check_bank(const htam_bank *b) {
    if (!b) return fail(HTAM_ERR_NULL, "bank is NULL");
    if (b->d < 8 || b->d > HTAM_MAX_DIM || b->d % 8 != 0)
        return fail(HTAM_ERR_SHAPE, "d = %d: need 8 <= d <= %d and d %% 8 == 0", b->d, HTAM_MAX_DIM);
    if (b->n_clusters < 1) return fail(HTAM_ERR_SHAPE, "n_clusters = %d < 1", b->n_clusters);
    if (b->n_transitions < 0 || b->n_transitions >= (int64_t(1) << 31))
        return fail(HTAM_ERR_SHAPE, "n_transitions = %lld out of [0, 2^31)",
                    (long long)b->n_transitions);
    if (!valid_dtype(b->key_dtype) || !valid_dtype(b->compute_dtype))
        return fail(HTAM_ERR_DTYPE, "unknown dtype (key %d, compute %d)", b->key_dtype,
                    b->compute_dtype);
    if (b->key_dtype == HTAM_BF16 && b->compute_dtype == HTAM_F32)
        return fail(HTAM_ERR_DTYPE, "bf16 keys with fp32 compute is not supported");
    if (!b->coarse_keys) return fail(HTAM_ERR_NULL, "bank->coarse_keys is NULL");
    if (!b->seg_offsets) return fail(HTAM_ERR_NULL, "bank->seg_offsets is NULL");
    if (b->n_transitions > 0 && !b->fine_keys) return fail(HTAM_ERR_NULL, "bank->fine_keys is NULL");
    if (!aligned16(b->coarse_keys) || !aligned16(b->fine_keys) || !aligned16(b->fine_keys_tiled) ||
        !aligned16(b->coarse_keys_bf16))
        return fail(HTAM_ERR_ALIGN, "bank key arrays must be 16-byte aligned");
    if (b->fine_keys_tiled && b->d % 32 != 0)
        return fail(HTAM_ERR_SHAPE, "bank->fine_keys_tiled needs d %% 32 == 0 (d = %d)", b->d);
    return HTAM_OK;
}

htam_status check_query(const htam_bank *b, const void *q, int32_t q_dtype, int32_t B) {
    if (B < 0) return fail(HTAM_ERR_SHAPE, "n_queries = %d < 0", B);
    if (!valid_dtype(q_dtype)) return fail(HTAM_ERR_DTYPE, "unknown q_dtype %d", q_dtype);
    if (q_dtype != b->key_dtype)
        return fail(HTAM_ERR_DTYPE, "q_dtype %d differs from the bank's key_dtype %d", q_dtype,
                    b->key_dtype);
    if (B > 0 && !q) return fail(HTAM_ERR_NULL, "q is NULL");
    if (!aligned16(q)) return fail(HTAM_ERR_ALIGN, "q must be 16-byte aligned");
    return HTAM_OK;
}

htam_status check_ws(void *ws, size_t have, size_t need) {
    if (!ws) return fail(HTAM_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
    if (have < need)
        return fail(HTAM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than %zu", have, need);
    if (!aligned256(ws)) return fail(HTAM_ERR_ALIGN, "workspace must be 256-byte aligned");
    return HTAM_OK;
}

htam_status check_tau(float tau) {
    if (!std::isfinite(tau) || !(tau > 0.0f))
        return fail(HTAM_ERR_VALUE, "tau = %g: need a finite tau > 0", (double)tau);
    return HTAM_OK;
}

// HTAM_VALIDATE set to anything but "" or "0": the fine stage waits for its
// planning step and reports malformed bank offsets and out-of-range selected
// cluster ids as HTAM_ERR_VALUE (read at every call).
bool validate_mode() {
    const char *v = std::getenv("HTAM_VALIDATE");
    return v && v[0] && !(v[0] == '0' && v[1] == 0);
}

// Compute units of the current device (cached per device).
int device_cus(int *dev_out) {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    if (dev_out) *dev_out = dev;
    if (dev >= 0 && dev < 64 && cached[dev] > 0) return cached[dev];
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    if (dev >= 0 && dev < 64) cached[dev] = n;
    return n;
}

}  // namespace

int32_t htam::report_error(int32_t status, const char *msg) {
    g_last_error = msg ? msg : "";
    return status;
}

#define HTAM_TRY(x)                                    \
    do {                                               \
        htam_status _st = (x);                         \
        if (_st != HTAM_OK) return _st;                \
    } while (0)

// ---------------------------------------------------------------------------
HTAM_API size_t htam_memory_build_workspace_size(int64_t n, int32_t n_clusters) {
    if (n < 0 || n_clusters < 1) return 0;
    size_t bytes = 0;
    htam::build_layout(nullptr, n, n_clusters, &bytes);
    return bytes;
}

HTAM_API htam_status htam_memory_build(int64_t n, int32_t n_clusters, int32_t d, int32_t key_dtype,
                                       const int32_t *cluster_of, const void *keys_in,
                                       void *keys_out, int64_t *seg_offsets,
                                       int32_t *transition_id, void *ws, size_t ws_bytes,
                                       hipStream_t stream) {
    if (n < 0 || n >= (int64_t(1) << 31)) return fail(HTAM_ERR_SHAPE, "n = %lld out of [0, 2^31)", (long long)n);
    if (n_clusters < 1) return fail(HTAM_ERR_SHAPE, "n_clusters = %d < 1", n_clusters);
    if (!seg_offsets) return fail(HTAM_ERR_NULL, "seg_offsets is NULL");
    if (n > 0 && (!cluster_of || !transition_id))
        return fail(HTAM_ERR_NULL, "cluster_of / transition_id is NULL");
    if (keys_in) {
        if (!keys_out) return fail(HTAM_ERR_NULL, "keys_out is NULL while keys_in is given");
        if (!valid_dtype(key_dtype)) return fail(HTAM_ERR_DTYPE, "unknown key_dtype %d", key_dtype);
        if (d < 8 || d > HTAM_MAX_DIM || d % 8 != 0)
            return fail(HTAM_ERR_SHAPE, "d = %d: need 8 <= d <= %d and d %% 8 == 0", d, HTAM_MAX_DIM);
        if (!aligned16(keys_in) || !aligned16(keys_out))
            return fail(HTAM_ERR_ALIGN, "key arrays must be 16-byte aligned");
        const char *a = static_cast<const char *>(keys_in), *b = static_cast<const char *>(keys_out);
        const size_t bytes = (size_t)n * d * dtype_bytes(key_dtype);
        if (n > 0 && a < b + bytes && b < a + bytes)
            return fail(HTAM_ERR_VALUE, "keys_in and keys_out overlap");
    }
    HTAM_TRY(check_ws(ws, ws_bytes, htam_memory_build_workspace_size(n, n_clusters)));

    const htam::BuildWs w = htam::build_layout(ws, n, n_clusters, nullptr);
    hipError_t e = htam::launch_build(n, n_clusters, keys_in ? d * dtype_bytes(key_dtype) : 0,
                                      cluster_of, keys_in, keys_out, seg_offsets, transition_id, w,
                                      stream);
    if (e != hipSuccess) return device_status(e, "htam_memory_build launch");
    int32_t bad = 0;
    e = hipMemcpyAsync(&bad, w.err, sizeof bad, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return device_status(e, "htam_memory_build");
    if (bad) return fail(HTAM_ERR_VALUE, "%d records have a cluster id outside [0, %d)", bad, n_clusters);
    return ok();
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_memory_tile_bytes(const htam_bank *bank) {
    if (!bank || bank->d < 32 || bank->d > HTAM_MAX_DIM || bank->d % 32 != 0 ||
        bank->n_transitions < 0 || !valid_dtype(bank->key_dtype))
        return 0;
    if (bank->n_clusters < 1) return 0;
    // the header, then at most N / 16 + G tiles (each segment padded to 16 rows)
    const size_t tiles = (size_t)((bank->n_transitions + 15) / 16) + (size_t)bank->n_clusters;
    return htam::tile_header_bytes(bank->n_clusters) +
           tiles * 16 * bank->d * dtype_bytes(bank->key_dtype);
}

HTAM_API htam_status htam_memory_tile(const htam_bank *bank, void *tiled_out, hipStream_t stream) {
    if (!bank) return fail(HTAM_ERR_NULL, "bank is NULL");
    htam_bank b = *bank;
    b.fine_keys_tiled = nullptr;               // ignored here
    HTAM_TRY(check_bank(&b));
    if (b.d % 32 != 0) return fail(HTAM_ERR_SHAPE, "d = %d: the tiled copy needs d %% 32 == 0", b.d);
    if (!tiled_out) return fail(HTAM_ERR_NULL, "tiled_out is NULL");
    if (!aligned16(tiled_out)) return fail(HTAM_ERR_ALIGN, "tiled_out must be 16-byte aligned");
    const size_t in_bytes = (size_t)b.n_transitions * b.d * dtype_bytes(b.key_dtype);
    const char *a = static_cast<const char *>(b.fine_keys), *o = static_cast<const char *>(tiled_out);
    if (a < o + htam_memory_tile_bytes(&b) && o < a + in_bytes)
        return fail(HTAM_ERR_VALUE, "tiled_out overlaps bank->fine_keys");
    return device_status(htam::launch_tile_keys(b.n_transitions, b.n_clusters, b.d,
                                                dtype_bytes(b.key_dtype), b.fine_keys,
                                                b.seg_offsets, tiled_out, stream),
                         "htam_memory_tile");
}

HTAM_API htam_status htam_coarse_keys_bf16(const htam_bank *bank, void *out, hipStream_t stream) {
    if (!bank) return fail(HTAM_ERR_NULL, "bank is NULL");
    htam_bank b = *bank;
    b.coarse_keys_bf16 = nullptr;              // ignored here
    HTAM_TRY(check_bank(&b));
    if (b.key_dtype != HTAM_F32) return fail(HTAM_ERR_DTYPE, "the bank's keys are not fp32");
    if (!out) return fail(HTAM_ERR_NULL, "out is NULL");
    if (!aligned16(out)) return fail(HTAM_ERR_ALIGN, "out must be 16-byte aligned");
    const size_t n = (size_t)b.n_clusters * b.d;
    const char *a = static_cast<const char *>(b.coarse_keys), *o = static_cast<const char *>(out);
    if (a < o + 2 * n && o < a + 4 * n) return fail(HTAM_ERR_VALUE, "out overlaps bank->coarse_keys");
    return device_status(htam::launch_round_bf16(static_cast<const float *>(b.coarse_keys),
                                                 static_cast<__bf16 *>(out), (int64_t)n, stream),
                         "htam_coarse_keys_bf16");
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_retrieve_coarse_workspace_size(const htam_bank *bank, int32_t n_queries,
                                                    int32_t top_c) {
    if (!bank || n_queries < 0 || bank->n_clusters < 1 || top_c < 1) return 0;
    size_t bytes = 0;
    htam::coarse_layout(nullptr, n_queries, bank->n_clusters, bank->d, bank->key_dtype,
                        bank->compute_dtype, top_c, &bytes);
    return bytes;
}

HTAM_API htam_status htam_retrieve_coarse(const htam_bank *bank, const void *q, int32_t q_dtype,
                                          int32_t n_queries, int32_t top_c, int32_t *sel_cluster,
                                          float *sel_score, void *ws, size_t ws_bytes,
                                          hipStream_t stream) {
    HTAM_TRY(check_bank(bank));
    HTAM_TRY(check_query(bank, q, q_dtype, n_queries));
    const int32_t cmax = bank->n_clusters < HTAM_MAX_TOP_C ? bank->n_clusters : HTAM_MAX_TOP_C;
    if (top_c < 1 || top_c > cmax)
        return fail(HTAM_ERR_SHAPE, "top_c = %d out of [1, %d]", top_c, cmax);
    if (n_queries > 0 && !sel_cluster) return fail(HTAM_ERR_NULL, "sel_cluster is NULL");
    if (n_queries == 0) return ok();
    HTAM_TRY(check_ws(ws, ws_bytes, htam_retrieve_coarse_workspace_size(bank, n_queries, top_c)));
    const int n_cu = device_cus(nullptr);
    if (n_cu <= 0) return fail(HTAM_ERR_DEVICE, "no HIP device");
    const htam::CoarseWs w = htam::coarse_layout(ws, n_queries, bank->n_clusters, bank->d,
                                                 bank->key_dtype, bank->compute_dtype, top_c,
                                                 nullptr);
    const void *ck16 = bank->key_dtype == HTAM_F32 ? bank->coarse_keys_bf16 : nullptr;
    return device_status(htam::launch_coarse(bank->key_dtype, bank->compute_dtype, bank->d,
                                             bank->n_clusters, bank->coarse_keys, ck16, q,
                                             n_queries, top_c, sel_cluster, sel_score, w, n_cu,
                                             g_events[HTAM_KERNEL_COARSE], stream),
                         "htam_retrieve_coarse");
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_attend_transitions_workspace_size(const htam_bank *bank, int32_t n_queries,
                                                       int32_t top_c, int32_t top_k) {
    if (!bank || n_queries < 0 || top_c < 1 || top_k < 1 || bank->n_clusters < 1 || bank->d < 8)
        return 0;
    size_t bytes = 0;
    htam::attend_layout(nullptr, bank->d, bank->n_clusters, bank->n_transitions,
                        dtype_bytes(bank->key_dtype), n_queries, top_c, top_k, &bytes);
    return bytes;
}

HTAM_API htam_status htam_attend_transitions(const htam_bank *bank, const void *q, int32_t q_dtype,
                                             int32_t n_queries, const int32_t *sel_cluster,
                                             int32_t top_c, float tau, int32_t top_k,
                                             float *slot_max, float *slot_sum, float *cand_score,
                                             int32_t *cand_id, void *ws, size_t ws_bytes,
                                             hipStream_t stream) {
    HTAM_TRY(check_bank(bank));
    HTAM_TRY(check_query(bank, q, q_dtype, n_queries));
    const int32_t cmax = bank->n_clusters < HTAM_MAX_TOP_C ? bank->n_clusters : HTAM_MAX_TOP_C;
    if (top_c < 1 || top_c > cmax)
        return fail(HTAM_ERR_SHAPE, "top_c = %d out of [1, %d]", top_c, cmax);
    if (top_k < 1 || top_k > HTAM_MAX_TOP_K)
        return fail(HTAM_ERR_SHAPE, "top_k = %d out of [1, %d]", top_k, HTAM_MAX_TOP_K);
    HTAM_TRY(check_tau(tau));
    if ((int64_t)n_queries * top_c >= (int64_t(1) << 31))
        return fail(HTAM_ERR_SHAPE, "n_queries * top_c must be < 2^31");
    if (n_queries == 0) return ok();
    if (!sel_cluster || !slot_max || !slot_sum || !cand_score || !cand_id)
        return fail(HTAM_ERR_NULL, "an output or sel_cluster is NULL");
    HTAM_TRY(check_ws(ws, ws_bytes,
                      htam_attend_transitions_workspace_size(bank, n_queries, top_c, top_k)));
    const int n_cu = device_cus(nullptr);
    if (n_cu <= 0) return fail(HTAM_ERR_DEVICE, "no HIP device");
    const htam::AttendWs w =
        htam::attend_layout(ws, bank->d, bank->n_clusters, bank->n_transitions,
                            dtype_bytes(bank->key_dtype), n_queries, top_c, top_k, nullptr);
    const htam_status st = device_status(
        htam::launch_attend(bank->key_dtype, bank->compute_dtype, bank->d, bank->n_clusters,
                            bank->n_transitions, bank->fine_keys, bank->fine_keys_tiled,
                            bank->seg_offsets, bank->transition_id, q, n_queries, sel_cluster,
                            top_c, tau, top_k,
                            slot_max, slot_sum, cand_score, cand_id, w, n_cu,
                            g_events[HTAM_KERNEL_STREAM], stream),
        "htam_attend_transitions");
    if (st != HTAM_OK || !validate_mode()) return st;
    htam::Plan plan{};
    hipError_t e = hipMemcpyAsync(&plan, w.plan, sizeof plan, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return device_status(e, "htam_attend_transitions (validation)");
    if (plan.bad_off)
        return fail(HTAM_ERR_VALUE, "bank->seg_offsets is not a partition of [0, %lld): need "
                    "off[0] = 0, nondecreasing, off[G] = N; or the header of "
                    "bank->fine_keys_tiled does not match them (no record was read)",
                    (long long)bank->n_transitions);
    if (plan.bad_sel)
        return fail(HTAM_ERR_VALUE, "%d selected cluster ids lie outside [0, %d) (their slots are empty)",
                    plan.bad_sel, bank->n_clusters);
    return ok();
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_memory_merge_workspace_size(void) { return 256; }

HTAM_API htam_status htam_memory_merge(int32_t n_clusters, int32_t d, int32_t key_dtype,
                                       const void *keys_a, const int64_t *off_a,
                                       const int32_t *id_a, int64_t n_a, const void *keys_b,
                                       const int64_t *off_b, const int32_t *id_b, int64_t n_b,
                                       void *keys_out, int64_t *off_out, int32_t *id_out,
                                       void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n_clusters < 1) return fail(HTAM_ERR_SHAPE, "n_clusters = %d < 1", n_clusters);
    if (n_a < 0 || n_b < 0 || n_a + n_b >= (int64_t(1) << 31))
        return fail(HTAM_ERR_SHAPE, "n_a = %lld, n_b = %lld: need n_a, n_b >= 0 and n_a + n_b < 2^31",
                    (long long)n_a, (long long)n_b);
    if (!valid_dtype(key_dtype)) return fail(HTAM_ERR_DTYPE, "unknown key_dtype %d", key_dtype);
    if (d < 8 || d > HTAM_MAX_DIM || d % 8 != 0)
        return fail(HTAM_ERR_SHAPE, "d = %d: need 8 <= d <= %d and d %% 8 == 0", d, HTAM_MAX_DIM);
    if (!off_a || !off_b || !off_out) return fail(HTAM_ERR_NULL, "an offset array is NULL");
    if ((n_a > 0 && (!keys_a || !id_a)) || (n_b > 0 && (!keys_b || !id_b)) ||
        (n_a + n_b > 0 && (!keys_out || !id_out)))
        return fail(HTAM_ERR_NULL, "a key or id array is NULL");
    if (!aligned16(keys_a) || !aligned16(keys_b) || !aligned16(keys_out))
        return fail(HTAM_ERR_ALIGN, "key arrays must be 16-byte aligned");
    const size_t rb = (size_t)d * dtype_bytes(key_dtype);
    auto overlap = [](const void *p, size_t np, const void *q, size_t nq) {
        const char *a = static_cast<const char *>(p), *b = static_cast<const char *>(q);
        return np && nq && a < b + nq && b < a + np;
    };
    if (overlap(keys_out, (n_a + n_b) * rb, keys_a, n_a * rb) ||
        overlap(keys_out, (n_a + n_b) * rb, keys_b, n_b * rb))
        return fail(HTAM_ERR_VALUE, "keys_out overlaps an input bank");
    HTAM_TRY(check_ws(ws, ws_bytes, htam_memory_merge_workspace_size()));
    int32_t *bad = static_cast<int32_t *>(ws);
    hipError_t e = htam::launch_merge_banks(n_clusters, (int32_t)rb, keys_a, off_a, id_a, n_a,
                                            keys_b, off_b, id_b, n_b, keys_out, off_out, id_out,
                                            bad, stream);
    if (e != hipSuccess) return device_status(e, "htam_memory_merge");
    if (!validate_mode()) return ok();
    int32_t hb = 0;
    e = hipMemcpyAsync(&hb, bad, sizeof hb, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return device_status(e, "htam_memory_merge (validation)");
    if (hb) return fail(HTAM_ERR_VALUE, "an input bank's offsets are not a partition of its rows "
                        "(nothing was written)");
    return ok();
}

// ---------------------------------------------------------------------------
HTAM_API htam_status htam_feedback_update(int32_t n_clusters, int32_t n_buckets, int32_t n_events,
                                          const int32_t *src, const int32_t *dst,
                                          const int32_t *bucket, const float *features,
                                          int64_t *node_stats, int64_t *edge_stats,
                                          int64_t *edge_bucket_stats, hipStream_t stream) {
    if (n_clusters < 1 || n_buckets < 1 || n_events < 0)
        return fail(HTAM_ERR_SHAPE, "n_clusters %d, n_buckets %d, n_events %d: need >= 1, >= 1, >= 0",
                    n_clusters, n_buckets, n_events);
    if ((int64_t)n_clusters * n_clusters * n_buckets * HTAM_STATS_WORDS >= (int64_t(1) << 40))
        return fail(HTAM_ERR_SHAPE, "the edge-bucket statistics would exceed 2^40 words");
    if (!node_stats || !edge_stats || !edge_bucket_stats)
        return fail(HTAM_ERR_NULL, "a statistics array is NULL");
    if (n_events == 0) return ok();
    if (!src || !dst || !bucket || !features) return fail(HTAM_ERR_NULL, "an event array is NULL");
    return device_status(htam::launch_feedback_update(n_clusters, n_buckets, n_events, src, dst,
                                                      bucket, features, node_stats, edge_stats,
                                                      edge_bucket_stats, stream),
                         "htam_feedback_update");
}

HTAM_API htam_status htam_transition_scores(int32_t n_clusters, int32_t n_buckets,
                                            int32_t n_queries, const int32_t *prefix,
                                            int32_t max_prefix, const int32_t *bucket, float lambda,
                                            const float *w, int32_t min_count,
                                            const int64_t *node_stats, const int64_t *edge_stats,
                                            const int64_t *edge_bucket_stats, float *scores,
                                            hipStream_t stream) {
    if (n_clusters < 1 || n_buckets < 1 || n_queries < 0)
        return fail(HTAM_ERR_SHAPE, "n_clusters %d, n_buckets %d, n_queries %d", n_clusters,
                    n_buckets, n_queries);
    if (max_prefix < 1 || max_prefix > HTAM_MAX_PREFIX)
        return fail(HTAM_ERR_SHAPE, "max_prefix = %d out of [1, %d]", max_prefix, HTAM_MAX_PREFIX);
    if (!std::isfinite(lambda) || lambda < 0.0f)
        return fail(HTAM_ERR_VALUE, "lambda = %g: need a finite lambda >= 0", (double)lambda);
    if (min_count < 0) return fail(HTAM_ERR_VALUE, "min_count = %d < 0", min_count);
    if (n_queries == 0) return ok();
    if (!prefix || !bucket || !w || !node_stats || !edge_stats || !edge_bucket_stats || !scores)
        return fail(HTAM_ERR_NULL, "an input or output array is NULL");
    return device_status(htam::launch_transition_scores(n_clusters, n_buckets, n_queries, prefix,
                                                        max_prefix, bucket, lambda, w, min_count,
                                                        node_stats, edge_stats, edge_bucket_stats,
                                                        scores, stream),
                         "htam_transition_scores");
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_retrieve_coarse_sampled_workspace_size(const htam_bank *bank,
                                                            int32_t n_queries, int32_t top_c) {
    if (!bank || n_queries < 0 || bank->n_clusters < 1 || top_c < 1) return 0;
    size_t bytes = 0;
    htam::sampled_layout(nullptr, n_queries, bank->n_clusters, bank->d, bank->key_dtype,
                         bank->compute_dtype, top_c, &bytes);
    return bytes;
}

HTAM_API htam_status htam_retrieve_coarse_sampled(const htam_bank *bank, const void *q,
                                                  int32_t q_dtype, int32_t n_queries, int32_t top_c,
                                                  float epsilon, float tau_g,
                                                  const uint32_t *noise, uint64_t seed,
                                                  uint64_t offset, int32_t *sel_cluster,
                                                  float *sel_score, void *ws, size_t ws_bytes,
                                                  hipStream_t stream) {
    HTAM_TRY(check_bank(bank));
    HTAM_TRY(check_query(bank, q, q_dtype, n_queries));
    const int32_t cmax = bank->n_clusters < HTAM_MAX_TOP_C ? bank->n_clusters : HTAM_MAX_TOP_C;
    if (top_c < 1 || top_c > cmax)
        return fail(HTAM_ERR_SHAPE, "top_c = %d out of [1, %d]", top_c, cmax);
    if (!std::isfinite(epsilon) || epsilon < 0.0f || epsilon > 1.0f)
        return fail(HTAM_ERR_VALUE, "epsilon = %g: need 0 <= epsilon <= 1", (double)epsilon);
    if (!std::isfinite(tau_g) || !(tau_g > 0.0f))
        return fail(HTAM_ERR_VALUE, "tau_g = %g: need a finite tau_g > 0", (double)tau_g);
    if (n_queries == 0) return ok();
    if (!sel_cluster) return fail(HTAM_ERR_NULL, "sel_cluster is NULL");
    HTAM_TRY(check_ws(ws, ws_bytes,
                      htam_retrieve_coarse_sampled_workspace_size(bank, n_queries, top_c)));
    const int n_cu = device_cus(nullptr);
    if (n_cu <= 0) return fail(HTAM_ERR_DEVICE, "no HIP device");
    const htam::SampledWs w = htam::sampled_layout(ws, n_queries, bank->n_clusters, bank->d,
                                                   bank->key_dtype, bank->compute_dtype, top_c,
                                                   nullptr);
    return device_status(htam::launch_sampled(bank->key_dtype, bank->compute_dtype, bank->d,
                                              bank->n_clusters, bank->coarse_keys, q, n_queries,
                                              top_c, epsilon, tau_g, noise, seed, offset,
                                              sel_cluster, sel_score, w, n_cu,
                                              g_events[HTAM_KERNEL_COARSE], stream),
                         "htam_retrieve_coarse_sampled");
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_retrieve_coarse_prefix_workspace_size(const htam_bank *bank,
                                                           int32_t n_queries, int32_t max_prefix,
                                                           int32_t top_c) {
    if (!bank || n_queries < 0 || bank->n_clusters < 1 || top_c < 1 || max_prefix < 1 ||
        max_prefix > HTAM_MAX_PREFIX)
        return 0;
    size_t bytes = 0;
    htam::prefix_layout(nullptr, n_queries, bank->n_clusters, bank->d, bank->key_dtype,
                        bank->compute_dtype, max_prefix, top_c, &bytes);
    return bytes;
}

HTAM_API htam_status htam_retrieve_coarse_prefix(const htam_bank *bank, const void *edge_keys,
                                                 const int32_t *prefix, int32_t max_prefix,
                                                 float lambda, const void *q, int32_t q_dtype,
                                                 int32_t n_queries, int32_t top_c,
                                                 int32_t *sel_cluster, float *sel_score, void *ws,
                                                 size_t ws_bytes, hipStream_t stream) {
    HTAM_TRY(check_bank(bank));
    HTAM_TRY(check_query(bank, q, q_dtype, n_queries));
    const int32_t cmax = bank->n_clusters < HTAM_MAX_TOP_C ? bank->n_clusters : HTAM_MAX_TOP_C;
    if (top_c < 1 || top_c > cmax)
        return fail(HTAM_ERR_SHAPE, "top_c = %d out of [1, %d]", top_c, cmax);
    if (max_prefix < 1 || max_prefix > HTAM_MAX_PREFIX)
        return fail(HTAM_ERR_SHAPE, "max_prefix = %d out of [1, %d]", max_prefix, HTAM_MAX_PREFIX);
    if (!std::isfinite(lambda) || lambda < 0.0f)
        return fail(HTAM_ERR_VALUE, "lambda = %g: need a finite lambda >= 0", (double)lambda);
    if ((int64_t)n_queries * max_prefix >= (int64_t(1) << 31))
        return fail(HTAM_ERR_SHAPE, "n_queries * max_prefix must be < 2^31");
    if (!edge_keys) return fail(HTAM_ERR_NULL, "edge_keys is NULL");
    if (!aligned16(edge_keys)) return fail(HTAM_ERR_ALIGN, "edge_keys must be 16-byte aligned");
    if (n_queries == 0) return ok();
    if (!prefix || !sel_cluster) return fail(HTAM_ERR_NULL, "prefix / sel_cluster is NULL");
    HTAM_TRY(check_ws(ws, ws_bytes, htam_retrieve_coarse_prefix_workspace_size(
                                         bank, n_queries, max_prefix, top_c)));
    const int n_cu = device_cus(nullptr);
    if (n_cu <= 0) return fail(HTAM_ERR_DEVICE, "no HIP device");
    const htam::PrefixWs w =
        htam::prefix_layout(ws, n_queries, bank->n_clusters, bank->d, bank->key_dtype,
                            bank->compute_dtype, max_prefix, top_c, nullptr);
    return device_status(htam::launch_prefix(bank->key_dtype, bank->compute_dtype, bank->d,
                                             bank->n_clusters, bank->coarse_keys, edge_keys,
                                             prefix, max_prefix, lambda, q, n_queries, top_c,
                                             sel_cluster, sel_score, w, n_cu,
                                             g_events[HTAM_KERNEL_COARSE], stream),
                         "htam_retrieve_coarse_prefix");
}

// ---------------------------------------------------------------------------
HTAM_API size_t htam_retrieve_flat_workspace_size(const htam_bank *bank, int32_t n_queries,
                                                  int32_t top_k) {
    if (!bank || n_queries < 0 || top_k < 1 || bank->d < 8 || bank->n_transitions < 0) return 0;
    size_t bytes = 0;
    htam::flat_layout(nullptr, bank->d, bank->n_transitions, bank->key_dtype, bank->compute_dtype,
                      n_queries, top_k, &bytes);
    return bytes;
}

HTAM_API htam_status htam_retrieve_flat(const htam_bank *bank, const void *q, int32_t q_dtype,
                                        int32_t n_queries, float tau, int32_t top_k,
                                        int32_t *out_id, float *out_score, float *out_weight,
                                        float *row_max, float *row_sum, int32_t *out_count,
                                        void *ws, size_t ws_bytes, hipStream_t stream) {
    HTAM_TRY(check_bank(bank));
    HTAM_TRY(check_query(bank, q, q_dtype, n_queries));
    if (top_k < 1 || top_k > HTAM_MAX_TOP_K)
        return fail(HTAM_ERR_SHAPE, "top_k = %d out of [1, %d]", top_k, HTAM_MAX_TOP_K);
    HTAM_TRY(check_tau(tau));
    if (n_queries == 0) return ok();
    if (!out_id || !out_score) return fail(HTAM_ERR_NULL, "out_id / out_score is NULL");
    HTAM_TRY(check_ws(ws, ws_bytes, htam_retrieve_flat_workspace_size(bank, n_queries, top_k)));
    const int n_cu = device_cus(nullptr);
    if (n_cu <= 0) return fail(HTAM_ERR_DEVICE, "no HIP device");
    const htam::FlatWs w = htam::flat_layout(ws, bank->d, bank->n_transitions, bank->key_dtype,
                                             bank->compute_dtype, n_queries, top_k, nullptr);
    return device_status(htam::launch_flat(bank->key_dtype, bank->compute_dtype, bank->d,
                                           bank->n_transitions, bank->fine_keys,
                                           bank->transition_id, q, n_queries, tau, top_k, out_id,
                                           out_score, out_weight, row_max, row_sum, out_count, w,
                                           n_cu, g_events[HTAM_KERNEL_COARSE], stream),
                         "htam_retrieve_flat");
}

// ---------------------------------------------------------------------------
static htam_status topk_entry(int32_t n_rows, int32_t n_lists, int32_t k_in,
                              const float *cand_score, const int32_t *cand_id,
                              const float *slot_max, const float *slot_sum, float tau,
                              int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                              float *row_max, float *row_sum, int32_t *out_count,
                              hipStream_t stream, bool sorted_lists, const char *name) {
    if (n_rows < 0 || n_lists < 1 || k_in < 1)
        return fail(HTAM_ERR_SHAPE, "n_rows %d, n_lists %d, k_in %d: need n_rows >= 0, n_lists >= 1, k_in >= 1",
                    n_rows, n_lists, k_in);
    if ((int64_t)n_lists * k_in >= (int64_t(1) << 31))
        return fail(HTAM_ERR_SHAPE, "n_lists * k_in must be < 2^31");
    if (top_k < 1 || top_k > HTAM_MAX_TOP_K)
        return fail(HTAM_ERR_SHAPE, "top_k = %d out of [1, %d]", top_k, HTAM_MAX_TOP_K);
    if ((slot_max == nullptr) != (slot_sum == nullptr))
        return fail(HTAM_ERR_NULL, "slot_max and slot_sum must be given together");
    if (!slot_max && (out_weight || row_max || row_sum))
        return fail(HTAM_ERR_VALUE, "out_weight / row_max / row_sum need slot_max and slot_sum");
    if (slot_max) HTAM_TRY(check_tau(tau));
    if (n_rows == 0) return ok();
    if (!cand_score || !out_id || !out_score) return fail(HTAM_ERR_NULL, "an input or output is NULL");
    return device_status(htam::launch_topk(n_rows, n_lists, k_in, cand_score, cand_id, slot_max,
                                           slot_sum, slot_max ? tau : 1.0f, top_k, out_id,
                                           out_score, out_weight, row_max, row_sum, out_count,
                                           stream, sorted_lists),
                         name);
}

HTAM_API htam_status htam_topk(int32_t n_rows, int32_t n_lists, int32_t k_in,
                               const float *cand_score, const int32_t *cand_id,
                               const float *slot_max, const float *slot_sum, float tau,
                               int32_t top_k, int32_t *out_id, float *out_score,
                               float *out_weight, float *row_max, float *row_sum,
                               int32_t *out_count, hipStream_t stream) {
    return topk_entry(n_rows, n_lists, k_in, cand_score, cand_id, slot_max, slot_sum, tau, top_k,
                      out_id, out_score, out_weight, row_max, row_sum, out_count, stream, false,
                      "htam_topk");
}

HTAM_API htam_status htam_topk_sorted(int32_t n_rows, int32_t n_lists, int32_t k_in,
                                      const float *cand_score, const int32_t *cand_id,
                                      const float *slot_max, const float *slot_sum, float tau,
                                      int32_t top_k, int32_t *out_id, float *out_score,
                                      float *out_weight, float *row_max, float *row_sum,
                                      int32_t *out_count, hipStream_t stream) {
    return topk_entry(n_rows, n_lists, k_in, cand_score, cand_id, slot_max, slot_sum, tau, top_k,
                      out_id, out_score, out_weight, row_max, row_sum, out_count, stream, true,
                      "htam_topk_sorted");
}

// ---------------------------------------------------------------------------
HTAM_API const char *htam_status_string(htam_status st) {
    switch (st) {
        case HTAM_OK: return "HTAM_OK";
        case HTAM_ERR_NULL: return "HTAM_ERR_NULL";
        case HTAM_ERR_SHAPE: return "HTAM_ERR_SHAPE";
        case HTAM_ERR_DTYPE: return "HTAM_ERR_DTYPE";
        case HTAM_ERR_VALUE: return "HTAM_ERR_VALUE";
        case HTAM_ERR_WORKSPACE: return "HTAM_ERR_WORKSPACE";
        case HTAM_ERR_ALIGN: return "HTAM_ERR_ALIGN";
        case HTAM_ERR_DEVICE: return "HTAM_ERR_DEVICE";
    }
    return "HTAM_UNKNOWN_STATUS";
}

HTAM_API const char *htam_last_error(void) { return g_last_error.c_str(); }

HTAM_API htam_status htam_set_kernel_events(int32_t which, void *before, void *after) {
    if (which != HTAM_KERNEL_COARSE && which != HTAM_KERNEL_STREAM)
        return fail(HTAM_ERR_VALUE, "unknown kernel %d", which);
    if ((before == nullptr) != (after == nullptr))
        return fail(HTAM_ERR_NULL, "give both events or neither");
    g_events[which].before = static_cast<hipEvent_t>(before);
    g_events[which].after = static_cast<hipEvent_t>(after);
    return ok();
}
