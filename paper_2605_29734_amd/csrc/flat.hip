// Flat memory retrieval on gfx950: every record of the memory is a candidate
// of every query, with no coarse level (the "Flat Memory Retrieval" baseline
// of Table 1 and App. C.4, the "w/o hierarchy" ablation of Sec. 5.5). Scores
// are inner products (Eq. local policy), weights the temperature softmax over
// all N records, and the result the top-k by descending score, ties to the
// lower caller id.
//
// The bank is scored in bands of rows: per band one launch of the coarse
// GEMM kernels writes S = Q K_band^T (a dense B x band contraction on bf16
// MFMA, the flat path's MFMA-bound bulk), then the segmented top-k cuts every
// score row into 2048-column segments and keeps, per (query, segment), the
// segment's best k and its softmax statistics (max, sum). A final row merge
// (htam_topk's kernel) combines the segments' statistics and lists into the
// row's top-k, weights, max and sum. The score buffer is bounded (256 MiB),
// so the bank can be any size.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int64_t kFlatBufBytes = int64_t(256) << 20;

// Rows of one band: the score buffer [B][band] and the bf16 copy of the band's
// keys each within kFlatBufBytes, a multiple of the segment length.
int64_t flat_band(int32_t B, int32_t d, int64_t N, bool convert) {
    const int64_t kFlatSeg = seg_topk_cols();
    int64_t band = kFlatBufBytes / (4 * (int64_t)(B > 0 ? B : 1));
    if (convert) band = band < kFlatBufBytes / (2 * (int64_t)d) ? band : kFlatBufBytes / (2 * (int64_t)d);
    band = band / kFlatSeg * kFlatSeg;
    if (band < kFlatSeg) band = kFlatSeg;
    const int64_t all = (N + kFlatSeg - 1) / kFlatSeg * kFlatSeg;
    return band < all ? band : (all > 0 ? all : kFlatSeg);
}

// An empty bank: one list per query holding nothing.
__global__ void flat_empty(int32_t B, int32_t k, float *ps, int32_t *pi, float *pm, float *pz) {
    // k: slots per list
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < (int64_t)B * k;
         i += (int64_t)gridDim.x * blockDim.x) {
        ps[i] = -INFINITY;
        pi[i] = -1;
        if (i < B) {
            pm[i] = -INFINITY;
            pz[i] = 0.0f;
        }
    }
}

}  // namespace

FlatWs flat_layout(void *ws, int32_t d, int64_t N, int32_t key_dtype, int32_t compute_dtype,
                   int32_t B, int32_t k, size_t *bytes) {
    Carve cv(ws);
    FlatWs w{};
    const bool convert = key_dtype == kF32 && compute_dtype == kBF16;
    w.band = flat_band(B, d, N, convert);
    const int64_t seg = seg_topk_cols();
    w.n_lists = N > 0 ? (N + seg - 1) / seg : 1;
    w.scores = cv.take<float>((size_t)B * w.band);
    w.q16 = convert ? cv.take<__bf16>((size_t)B * d) : nullptr;
    w.k16 = convert ? cv.take<__bf16>((size_t)w.band * d) : nullptr;
    w.p_score = cv.take<float>((size_t)B * w.n_lists * seg_topk_slots(k));
    w.p_id = cv.take<int32_t>((size_t)B * w.n_lists * seg_topk_slots(k));
    w.pm = cv.take<float>((size_t)B * w.n_lists);
    w.pz = cv.take<float>((size_t)B * w.n_lists);
    if (bytes) *bytes = cv.off + 256;
    return w;
}

hipError_t launch_flat(int32_t key_dtype, int32_t compute_dtype, int32_t d, int64_t N,
                       const void *fine_keys, const int32_t *transition_id, const void *q,
                       int32_t B, float tau, int32_t k, int32_t *out_id, float *out_score,
                       float *out_weight, float *row_max, float *row_sum, int32_t *out_count,
                       const FlatWs &w, int n_cu, KernelEvents ev, hipStream_t s) {
    const int64_t kb = key_dtype == kF32 ? 4 : 2;
    if (N == 0) {
        hipLaunchKernelGGL(flat_empty, dim3(64), dim3(256), 0, s, B, seg_topk_slots(k), w.p_score,
                           w.p_id, w.pm, w.pz);
    }
    for (int64_t r0 = 0; r0 < N; r0 += w.band) {
        const int64_t nb = N - r0 < w.band ? N - r0 : w.band;
        hipError_t err = launch_scores(key_dtype, compute_dtype, d, nb,
                                       static_cast<const char *>(fine_keys) + r0 * d * kb, q, B,
                                       w.scores, w.q16, w.k16, r0 == 0, n_cu, ev, s);
        if (err != hipSuccess) return err;
        err = launch_seg_topk(B, nb, nb, w.scores, transition_id ? transition_id + r0 : nullptr,
                              r0, k, tau, w.p_score, w.p_id, w.pm, w.pz, w.n_lists,
                              r0 / seg_topk_cols(), s);
        if (err != hipSuccess) return err;
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    return launch_topk(B, (int32_t)w.n_lists, seg_topk_slots(k), w.p_score, w.p_id, w.pm, w.pz,
                       tau, k, out_id, out_score, out_weight, row_max, row_sum, out_count, s);
}

}  // namespace htam
