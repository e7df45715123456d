// Row-wise top-k merge on gfx950 (htam_topk, and the coarse top-c selection):
// the argmax of Eq. local policy widened to k injected memories, over the
// union of a query's candidate lists, with the temperature-softmax statistics
// of the lists merged into the row's (max, sum) and per-candidate weights.
//
// One wave per row. Candidates are read 8 x 64 at a time; those above the
// row's threshold are appended to the wave's LDS buffer (positions from a
// ballot prefix count, no atomics). When fewer than 64 free slots remain the
// buffer is cut down by a radix select (compact_select), which raises the
// threshold to the k-th best score.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int kTopkWaves = 4;
constexpr int kTopkBatch = 8;          // 64-entry groups loaded before they are offered
constexpr int kTopkStatLists = 1;      // 64-list groups of statistics loaded with the keys

struct TopkArgs {
    int64_t rows, n;              // entries per row = lists * k_in
    int32_t lists, top_k;
    float cexp;                   // log2(e) / tau
    const float *score;
    const int32_t *id;            // nullable: id = position in the row
    const float *slot_max, *slot_sum;
    int32_t *out_id;
    float *out_score, *out_weight, *row_max, *row_sum;
    int32_t *out_count;
};

// cap = 64 * NPL >= top_k + 64 keys of LDS per wave.
template <int NPL>
__global__ __launch_bounds__(kWave * kTopkWaves) void topk_rows(TopkArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t row = (int64_t)blockIdx.x * kTopkWaves + wave;
    if (row >= a.rows) return;              // no block-wide synchronisation below
    uint64_t *buf = tbuf + wave * cap;
    const float *sc = a.score + row * a.n;
    const int32_t *ids = a.id ? a.id + row * a.n : nullptr;
    const uint64_t lt_mask = (1ull << lane) - 1;

    // the row's list statistics, requested with the first keys
    float lm[kTopkStatLists], lz[kTopkStatLists];
#pragma unroll
    for (int i = 0; i < kTopkStatLists; ++i) {
        const int l = i * kWave + lane;
        const bool ok = a.slot_max && l < a.lists;
        lm[i] = ok ? a.slot_max[row * a.lists + l] : -INFINITY;
        lz[i] = ok ? a.slot_sum[row * a.lists + l] : 0.0f;
    }

    int cnt = 0, total = 0;
    uint64_t theta = 0;
    for (int64_t base = 0; base < a.n; base += kWave * kTopkBatch) {
        float s[kTopkBatch];
        int32_t cid[kTopkBatch];
#pragma unroll
        for (int u = 0; u < kTopkBatch; ++u) {
            const int64_t i = base + u * kWave + lane;
            const int64_t ic = i < a.n ? i : a.n - 1;
            s[u] = sc[ic];
            cid[u] = i < a.n ? (ids ? ids[ic] : (int32_t)i) : -1;
        }
#pragma unroll
        for (int u = 0; u < kTopkBatch; ++u) {
            const bool ok = cid[u] >= 0;
            total += __popcll(__ballot(ok));
            const uint64_t key = ok ? make_key(s[u], cid[u]) : 0;
            const bool pass = ok && key > theta;
            const uint64_t mask = __ballot(pass);
            if (pass) buf[cnt + __popcll(mask & lt_mask)] = key;
            cnt += __popcll(mask);
            if (cnt > cap - kWave) {
                wave_lds_sync();
                cnt = compact_select<NPL>(buf, cnt, a.top_k, kWave, lane, theta);
            }
        }
    }

    // merged softmax statistics of the row's lists
    float M = -INFINITY, Z = 0.0f;
    if (a.slot_max) {
#pragma unroll
        for (int i = 0; i < kTopkStatLists; ++i) mz_merge(M, Z, lm[i], lz[i], a.cexp);
        for (int l = kTopkStatLists * kWave + lane; l < a.lists; l += kWave)
            mz_merge(M, Z, a.slot_max[row * a.lists + l], a.slot_sum[row * a.lists + l], a.cexp);
        for (int sh = 32; sh >= 1; sh >>= 1) {
            const float m2 = __shfl_xor(M, sh), z2 = __shfl_xor(Z, sh);
            mz_merge(M, Z, m2, z2, a.cexp);
        }
    }

    wave_lds_sync();
    uint64_t v[NPL];
    sort_buffer<NPL>(buf, cnt, v, lane);
    const int kept = cnt < a.top_k ? cnt : a.top_k;
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
        const int r = q * kWave + lane;
        if (r < a.top_k) {
            const bool ok = r < kept;
            const float sv = ok ? key_score(v[q]) : -INFINITY;
            a.out_id[row * a.top_k + r] = ok ? key_id(v[q]) : -1;
            if (a.out_score) a.out_score[row * a.top_k + r] = sv;
            if (a.out_weight)
                a.out_weight[row * a.top_k + r] = ok ? exp2f((sv - M) * a.cexp) / Z : 0.0f;
        }
    }
    if (lane == 0) {
        if (a.row_max) a.row_max[row] = M;
        if (a.row_sum) a.row_sum[row] = Z;
        if (a.out_count) a.out_count[row] = total < a.top_k ? total : a.top_k;
    }
}

}  // namespace

hipError_t launch_topk(int32_t rows, int32_t lists, int32_t k_in, const float *score,
                       const int32_t *id, const float *slot_max, const float *slot_sum, float tau,
                       int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                       float *row_max, float *row_sum, int32_t *out_count, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    TopkArgs a{};
    a.rows = rows;
    a.n = (int64_t)lists * k_in;
    a.lists = lists;
    a.top_k = top_k;
    a.cexp = 1.4426950408889634f / tau;
    a.score = score;
    a.id = id;
    a.slot_max = slot_max;
    a.slot_sum = slot_sum;
    a.out_id = out_id;
    a.out_score = out_score;
    a.out_weight = out_weight;
    a.row_max = row_max;
    a.row_sum = row_sum;
    a.out_count = out_count;
    const int npl = next_pow2(top_k + kWave) / kWave;
    const dim3 grid((unsigned)((rows + kTopkWaves - 1) / kTopkWaves)), block(kWave * kTopkWaves);
    const size_t smem = (size_t)kTopkWaves * npl * kWave * 8;
    switch (npl) {
        case 2: hipLaunchKernelGGL(topk_rows<2>, grid, block, smem, s, a); break;
        case 4: hipLaunchKernelGGL(topk_rows<4>, grid, block, smem, s, a); break;
        case 8: hipLaunchKernelGGL(topk_rows<8>, grid, block, smem, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace htam
