// Row-wise top-k merge on gfx950 (htam_topk, and the coarse top-c selection):
// the argmax of Eq. local policy widened to k injected memories, over the
// union of a query's candidate lists, with the temperature-softmax statistics
// of the lists merged into the row's (max, sum) and per-candidate weights.
//
// One block of 256 threads per row. Candidates stream through a threshold
// filter into an LDS buffer (see TopkRow); the buffer is compacted by one wave
// whenever the next round of 256 offers might not fit.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int kTopkThreads = 256;
constexpr int kTopkWaves = kTopkThreads / kWave;

struct TopkArgs {
    int64_t n;                    // entries per row = lists * k_in
    int32_t lists, top_k, cap;
    float cexp;                   // log2(e) / tau
    const float *score;
    const int32_t *id;            // nullable: id = position in the row
    const float *slot_max, *slot_sum;
    int32_t *out_id;
    float *out_score, *out_weight, *row_max, *row_sum;
    int32_t *out_count;
};

__global__ __launch_bounds__(kTopkThreads) void topk_rows(TopkArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    __shared__ uint32_t s_cnt, s_total;
    __shared__ uint64_t s_theta;
    __shared__ float s_m[kTopkWaves], s_z[kTopkWaves];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t row = blockIdx.x;
    const float *sc = a.score + row * a.n;
    const int32_t *ids = a.id ? a.id + row * a.n : nullptr;
    if (t == 0) { s_cnt = 0; s_total = 0; s_theta = 0; }
    __syncthreads();
    TopkRow acc{tbuf, &s_cnt, &s_theta};

    uint32_t mine = 0;
    for (int64_t base = 0; base < a.n; base += kTopkThreads) {
        const int64_t i = base + t;
        if (i < a.n) {
            const int32_t cid = ids ? ids[i] : (int32_t)i;
            if (cid >= 0) {
                ++mine;
                const float s = sc[i];
                if (ord_of(s) >= (uint32_t)(s_theta >> 32)) topk_offer(acc, make_key(s, cid));
            }
        }
        __syncthreads();
        if ((int)s_cnt > a.cap - kTopkThreads) {
            if (wave == 0) topk_compact(acc, a.top_k, lane);
        }
        __syncthreads();
    }
    atomicAdd(&s_total, mine);

    // merged softmax statistics of the row's lists
    float M = -INFINITY, Z = 0.0f;
    if (a.slot_max) {
        for (int l = t; l < a.lists; l += kTopkThreads)
            mz_merge(M, Z, a.slot_max[row * a.lists + l], a.slot_sum[row * a.lists + l], a.cexp);
        for (int sh = 32; sh >= 1; sh >>= 1) {
            const float m2 = __shfl_xor(M, sh), z2 = __shfl_xor(Z, sh);
            mz_merge(M, Z, m2, z2, a.cexp);
        }
        if (lane == 0) { s_m[wave] = M; s_z[wave] = Z; }
    }
    __syncthreads();
    if (a.slot_max) {
        M = -INFINITY;
        Z = 0.0f;
        for (int w = 0; w < kTopkWaves; ++w) mz_merge(M, Z, s_m[w], s_z[w], a.cexp);
    }

    if (wave == 0) {
        const int cn = (int)s_cnt;
        const int np = next_pow2(cn < 2 ? 2 : cn);
        for (int i = cn + lane; i < np; i += kWave) tbuf[i] = 0;
        wave_lds_sync();
        wave_sort_desc(tbuf, np, lane);
        const int kept = cn < a.top_k ? cn : a.top_k;
        for (int r = lane; r < a.top_k; r += kWave) {
            const uint64_t key = tbuf[r];
            const bool ok = r < kept;
            const float s = ok ? key_score(key) : -INFINITY;
            a.out_id[row * a.top_k + r] = ok ? key_id(key) : -1;
            if (a.out_score) a.out_score[row * a.top_k + r] = s;
            if (a.out_weight)
                a.out_weight[row * a.top_k + r] = ok ? exp2f((s - M) * a.cexp) / Z : 0.0f;
        }
        if (lane == 0) {
            if (a.row_max) a.row_max[row] = M;
            if (a.row_sum) a.row_sum[row] = Z;
            if (a.out_count) {
                const uint32_t tot = s_total;
                a.out_count[row] = (int32_t)(tot < (uint32_t)a.top_k ? tot : (uint32_t)a.top_k);
            }
        }
    }
}

}  // namespace

hipError_t launch_topk(int32_t rows, int32_t lists, int32_t k_in, const float *score,
                       const int32_t *id, const float *slot_max, const float *slot_sum, float tau,
                       int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                       float *row_max, float *row_sum, int32_t *out_count, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    TopkArgs a{};
    a.n = (int64_t)lists * k_in;
    a.lists = lists;
    a.top_k = top_k;
    a.cap = next_pow2(top_k + kTopkThreads);
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
    hipLaunchKernelGGL(topk_rows, dim3(rows), dim3(kTopkThreads), (size_t)a.cap * 8, s, a);
    return hipGetLastError();
}

}  // namespace htam
