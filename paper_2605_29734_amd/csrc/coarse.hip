// Coarse stage on gfx950: the global-direction score of every cluster for
// every query (Alg. 1 Step 2; Eq. score with a one-term prefix and the linear
// scorer of App. B.6: an inner product), S = Q C^T on MFMA, then the top_c
// clusters of each row (greedy limit of Eq. global direction).
//
// Block tile 64 queries x 64 clusters (4 waves, each 32 x 32 = 2 x 2 MFMA
// 16x16 tiles), operands loaded straight from global memory in MFMA fragment
// layout; scores go to a [B][G] fp32 workspace and the top-c selection runs
// the row-wise top-k kernel over it with implicit ids.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

template <typename T, bool BF16>
__global__ __launch_bounds__(256) void coarse_scores(const T *__restrict__ q,
                                                     const T *__restrict__ ck, int32_t B,
                                                     int32_t G, int32_t d, float *__restrict__ S) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, kg = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.y * 64 + (wave >> 1) * 32;
    const int64_t col0 = (int64_t)blockIdx.x * 64 + (wave & 1) * 32;
    const T *qp[2], *cp[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t r = row0 + 16 * i + r16, c = col0 + 16 * i + r16;
        qp[i] = q + (r < B ? r : B - 1) * d;
        cp[i] = ck + (c < G ? c : G - 1) * d;
    }
    f32x4_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if constexpr (BF16) {
        for (int k0 = 0; k0 < d; k0 += 32) {
            const int k = k0 + kg * 8;
            const bool ok = k < d;
            bf16x8_t a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                a[i] = ok ? load8(qp[i] + k) : zero8();
                b[i] = ok ? load8(cp[i] + k) : zero8();
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    } else {
        for (int k0 = 0; k0 < d; k0 += 4) {
            const int k = k0 + kg;
            float a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                a[i] = (float)qp[i][k];
                b[i] = (float)cp[i][k];
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }
    // D[m][n]: this lane holds rows 4*kg + e of the 16x16 tile, column r16.
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t r = row0 + 16 * i + 4 * kg + e, c = col0 + 16 * j + r16;
                if (r < B && c < G) S[r * G + c] = acc[i][j][e];
            }
}

}  // namespace

CoarseWs coarse_layout(void *ws, int32_t B, int32_t G, size_t *bytes) {
    Carve cv(ws);
    CoarseWs w{};
    w.scores = cv.take<float>((size_t)B * G);
    if (bytes) *bytes = cv.off + 256;
    return w;
}

hipError_t launch_coarse(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         const void *coarse_keys, const void *q, int32_t B, int32_t top_c,
                         int32_t *sel, float *sel_score, const CoarseWs &w, KernelEvents ev,
                         hipStream_t s) {
    const dim3 grid((G + 63) / 64, (B + 63) / 64);
    if (ev.before) hipEventRecord(ev.before, s);
    if (compute_dtype == kF32)
        hipLaunchKernelGGL((coarse_scores<float, false>), grid, dim3(256), 0, s,
                           static_cast<const float *>(q), static_cast<const float *>(coarse_keys),
                           B, G, d, w.scores);
    else if (key_dtype == kF32)
        hipLaunchKernelGGL((coarse_scores<float, true>), grid, dim3(256), 0, s,
                           static_cast<const float *>(q), static_cast<const float *>(coarse_keys),
                           B, G, d, w.scores);
    else
        hipLaunchKernelGGL((coarse_scores<__bf16, true>), grid, dim3(256), 0, s,
                           static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(coarse_keys),
                           B, G, d, w.scores);
    if (ev.after) hipEventRecord(ev.after, s);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    return launch_topk(B, 1, G, w.scores, nullptr, nullptr, nullptr, 1.0f, top_c, sel, sel_score,
                       nullptr, nullptr, nullptr, nullptr, s);
}

}  // namespace htam
