// Coarse stage on gfx950: the global-direction score of every cluster for
// every query (Alg. 1 Step 2; Eq. score with a one-term prefix and the linear
// scorer of App. B.6: an inner product), S = Q C^T, then the top_c clusters
// of each row (the greedy limit of Eq. global direction).
//
// bf16 arithmetic: an LDS-tiled MFMA GEMM (v_mfma_f32_16x16x32_bf16).
//   block tile 256 queries x 256 clusters, 8 waves (2 x 4), each wave
//   128 x 64 = 8 x 4 MFMA tiles; K in stages of 32 loaded straight from global
//   memory into LDS (global_load_lds_dwordx4, no register staging), four
//   stages in flight, rows swizzled so that fragment reads are free of bank
//   conflicts (d % 32 == 0); tiles ordered so that the blocks of one XCD share
//   query rows in their L2. fp32 inputs are rounded to bf16 once per call.
// Too few 256 x 256 tiles to fill the GPU, or d not a multiple of 32: one wave
//   per 32 x 32 tile, operands read directly from global memory in MFMA
//   fragment layout, eight k-steps requested at a time.
// fp32 arithmetic (small configurations): a direct MFMA kernel on
//   v_mfma_f32_16x16x4f32.
// The scores go to a [B][G] fp32 workspace; the top-c selection is the
// row-wise top-k kernel with implicit ids; rows longer than 2048 clusters go
// through the segmented top-k first (2048 clusters per wave, held in
// registers) and then a merge of the segments' lists.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int kGemmThreads = 512;
constexpr int kStages = 4;                                // LDS stages in flight
constexpr int kStageBytes = (BM + BN) * BK * 2;           // 32 KiB: 512 rows x 64 bytes
constexpr size_t kGemmLds = (size_t)kStages * kStageBytes;
constexpr int kLoadsPerWave = (BM + BN) * BK / 8 / kWave / (kGemmThreads / kWave);   // 4

// fp32 -> bf16 (round to nearest even) of two arrays in one launch (the
// queries and the coarse keys), 8 elements per thread.
__global__ void to_bf16(const float *__restrict__ x0, __bf16 *__restrict__ y0, int64_t n0,
                        const float *__restrict__ x1, __bf16 *__restrict__ y1, int64_t n1) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n0 + n1;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i < n0) reinterpret_cast<bf16x8_t *>(y0)[i] = load8(x0 + i * 8);
        else reinterpret_cast<bf16x8_t *>(y1)[i - n0] = load8(x1 + (i - n0) * 8);
    }
}

// Tile of block b: the blocks that run on one XCD (b % 8) take consecutive
// tiles, and within that range tiles go column-major in groups of 8 row tiles.
__device__ __forceinline__ void gemm_tile(int b, int nb, int tm, int tn, int &mt, int &nt) {
    const int xcd = b % 8, per = (nb + 7) / 8;
    int lin = xcd * per + b / 8;
    if (lin >= nb) lin = b;                       // nb not a multiple of 8: keep a bijection
    const int group = 8 * tn;
    const int g = lin / group, first_m = g * 8;
    const int gm = min(tm - first_m, 8);
    const int in = lin - g * group;
    mt = first_m + in % gm;
    nt = in / gm;
}

// x from the lane N places before this one within its 16-lane row, rotating
// (DPP row_ror).
template <int N>
__device__ __forceinline__ float row_ror_f32(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + N, 0xF, 0xF, false));
}

// Stage layout in LDS: the stacked [Q tile; C tile] rows (512 of them), 64
// bytes each = four 16-byte chunks, chunk c of row r stored in slot
// c ^ ((r >> 2) & 3). A fragment read (16 rows, one chunk each) then touches
// 16 distinct (row % 4, slot) pairs: all 64 banks once.
__device__ __forceinline__ int gemm_slot(int row, int c) { return c ^ ((row >> 2) & 3); }

// Requests one stage straight into LDS (global_load_lds_dwordx4: lane i of an
// instruction writes bytes 16 i .. 16 i + 15 after the instruction's base).
// Instruction i of wave w covers rows 16 (4 w + i) .. + 15; its lane l loads
// row + l / 4, slot l % 4, i.e. the chunk gemm_slot(row, l % 4) of global
// memory. Rows are clamped into the matrices; d % BK == 0.
__device__ __forceinline__ void gemm_issue_stage(const __bf16 *__restrict__ q,
                                                 const __bf16 *__restrict__ ck, int64_t m0,
                                                 int64_t n0, int32_t B, int32_t G, int32_t d,
                                                 int k0, unsigned char *stage_base) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
        const int r0 = 16 * (kLoadsPerWave * wave + i);
        const int row = r0 + (lane >> 2);
        const int c = gemm_slot(row, lane & 3);
        const __bf16 *p = row < BM ? q + min(m0 + row, (int64_t)B - 1) * d
                                   : ck + min(n0 + row - BM, (int64_t)G - 1) * d;
        __builtin_amdgcn_global_load_lds((const void *)(p + k0 + 8 * c),
                                         (__attribute__((address_space(3))) void *)(stage_base + r0 * 64),
                                         16, 0, 0);
    }
}

__global__ __launch_bounds__(kGemmThreads) void coarse_gemm(const __bf16 *__restrict__ q,
                                                            const __bf16 *__restrict__ ck,
                                                            int32_t B, int32_t G, int32_t d,
                                                            float *__restrict__ S,
                                                            float *__restrict__ tmax) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r16 = lane & 15, kg = lane >> 4;
    const int wm = wave >> 2, wn = wave & 3;
    const int tm = (B + BM - 1) / BM, tn = (G + BN - 1) / BN;
    int mt, nt;
    if (tm * tn % 8 == 0) gemm_tile(blockIdx.x, tm * tn, tm, tn, mt, nt);
    else { mt = blockIdx.x / tn; nt = blockIdx.x % tn; }
    const int64_t m0 = (int64_t)mt * BM, n0 = (int64_t)nt * BN;
    const int nk = d / BK;

    f32x4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Software pipeline over K stages of 32: while the MFMAs of stage ks run
    // (its fragments already in registers), the fragments of stage ks + 1 are
    // read from LDS between them, and stages ks + 1 .. ks + 4 are in flight
    // or landed in the four LDS buffers. Past the end the last stage is
    // requested again into a buffer nobody reads, so that every wave issues
    // the same loads and the counts below stay exact.
    auto read_frags = [&](int ks, bf16x8_t (&a)[8], bf16x8_t (&b)[4]) {
        const unsigned char *st = lds + (ks % kStages) * kStageBytes;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = wm * 128 + i * 16 + r16;
            a[i] = *reinterpret_cast<const bf16x8_t *>(st + row * 64 + 16 * gemm_slot(row, kg));
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int row = BM + wn * 64 + j * 16 + r16;
            b[j] = *reinterpret_cast<const bf16x8_t *>(st + row * 64 + 16 * gemm_slot(row, kg));
        }
    };
    // One stage: wait until stage ks + 1 has landed for every wave and every
    // wave's reads of stage ks are done, refill stage ks's buffer with stage
    // ks + 4, then multiply stage ks while reading stage ks + 1.
    auto stage = [&](int ks, const bf16x8_t (&a)[8], const bf16x8_t (&b)[4], bf16x8_t (&na)[8],
                     bf16x8_t (&nb)[4]) {
        wait_vmcnt<(kStages - 2) * kLoadsPerWave>();
        __builtin_amdgcn_s_waitcnt(0xC07F);               // lgkmcnt(0): this wave's LDS reads are in
        __builtin_amdgcn_s_barrier();
        gemm_issue_stage(q, ck, m0, n0, B, G, d, min(ks + kStages, nk - 1) * BK,
                         lds + (ks % kStages) * kStageBytes);
        const unsigned char *st = lds + ((ks + 1) % kStages) * kStageBytes;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
            const int row = wm * 128 + i * 16 + r16;
            na[i] = *reinterpret_cast<const bf16x8_t *>(st + row * 64 + 16 * gemm_slot(row, kg));
            if (i < 4) {
                const int rb = BM + wn * 64 + i * 16 + r16;
                nb[i] = *reinterpret_cast<const bf16x8_t *>(st + rb * 64 + 16 * gemm_slot(rb, kg));
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
#pragma unroll
    for (int s0 = 0; s0 < kStages; ++s0)
        gemm_issue_stage(q, ck, m0, n0, B, G, d, min(s0, nk - 1) * BK, lds + s0 * kStageBytes);
    wait_vmcnt<(kStages - 1) * kLoadsPerWave>();          // stage 0 has landed for this wave
    __builtin_amdgcn_s_barrier();
    bf16x8_t a0[8], b0[4], a1[8], b1[4];
    read_frags(0, a0, b0);
    int ks = 0;
    for (; ks + 2 <= nk; ks += 2) {
        stage(ks, a0, b0, a1, b1);
        stage(ks + 1, a1, b1, a0, b0);
    }
    if (ks < nk) stage(ks, a0, b0, a1, b1);
    // No load may still be writing LDS when the block ends. Waiting here,
    // before the stores (the counter covers both), lets the block end while
    // its stores drain and the next block on the CU starts.
    wait_vmcnt<0>();
    // D[m][n]: this lane holds rows 4*kg + e of each 16x16 tile, column r16.
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t r = m0 + wm * 128 + i * 16 + 4 * kg + e;
                const int64_t c = n0 + wn * 64 + j * 16 + r16;
                if (r < B && c < G) S[r * G + c] = acc[i][j][e];
            }
    if (tmax) {
        // Each row's maximum over this wave's 64 columns (a 64-column tile of
        // the score row): over the lane's four columns, then the 16 lanes of
        // its row group (lanes 16 kg .. 16 kg + 15 hold one row's 16-column
        // slices) by DPP row rotations; no LDS, no barrier. Lane r16 of a row
        // group keeps the maxima of its rows r16 and 16 + r16 (in the order
        // i * 4 + e), so that the wave stores them in two instructions.
        const int n64 = (G + 63) / 64;
        const int tcol = nt * (BN / 64) + wn;
        if (tcol < n64) {
            bool ok[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) ok[j] = (int)n0 + wn * 64 + j * 16 + r16 < G;
            float keep[2] = {-INFINITY, -INFINITY};
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float m = fmaxf(fmaxf(ok[0] ? acc[i][0][e] : -INFINITY,
                                          ok[1] ? acc[i][1][e] : -INFINITY),
                                    fmaxf(ok[2] ? acc[i][2][e] : -INFINITY,
                                          ok[3] ? acc[i][3][e] : -INFINITY));
                    m = fmaxf(m, row_ror_f32<8>(m));
                    m = fmaxf(m, row_ror_f32<4>(m));
                    m = fmaxf(m, row_ror_f32<2>(m));
                    m = fmaxf(m, row_ror_f32<1>(m));
                    const int idx = i * 4 + e;
                    if ((idx & 15) == r16) keep[idx >> 4] = m;
                }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int idx = 16 * h + r16, i = idx >> 2, e = idx & 3;
                const int64_t r = m0 + wm * 128 + i * 16 + 4 * kg + e;
                if (r < B) tmax[r * n64 + tcol] = keep[h];
            }
        }
    }
}

// Small problems (fewer 256 x 256 tiles than compute units): one wave per
// TM*16 x TM*16 tile, operands read directly in MFMA fragment layout. A batch
// of k-steps is requested before any is used (addresses clamped into the
// row, past-the-end fragments zeroed where they are used), so a batch costs
// one memory round trip rather than one per k-step. TM = 1 (16 x 16 tiles,
// twice the k-steps per batch) when 32 x 32 tiles would leave compute units
// idle: four times the waves, and half the round trips each.
template <typename T, int TM>
__global__ __launch_bounds__(kWave) void coarse_small_bf16(const T *__restrict__ q,
                                                           const T *__restrict__ ck, int32_t B,
                                                           int32_t G, int32_t d,
                                                           float *__restrict__ S) {
    constexpr int kSteps = (sizeof(T) == 4 ? 4 : 8) * (TM == 1 ? 2 : 1);
    const int lane = threadIdx.x & 63;
    const int r16 = lane & 15, kg = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.y * 16 * TM, col0 = (int64_t)blockIdx.x * 16 * TM;
    const T *qp[TM], *cp[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int64_t r = row0 + 16 * i + r16, c = col0 + 16 * i + r16;
        qp[i] = q + (r < B ? r : B - 1) * d;
        cp[i] = ck + (c < G ? c : G - 1) * d;
    }
    f32x4_t acc[TM][TM];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int nks = (d + 31) / 32;
    for (int s0 = 0; s0 < nks; s0 += kSteps) {
        RawFrag<T> fa[kSteps][TM], fb[kSteps][TM];
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int k = min(32 * (s0 + st) + 8 * kg, d - 8);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                fa[st][i].load(qp[i] + k);
                fb[st][i].load(cp[i] + k);
            }
        }
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            // steps past the end multiply zeros: no branch for the compiler to
            // sink the loads into
            const bool ok = 32 * (s0 + st) + 8 * kg < d;
            bf16x8_t a[TM], b[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                a[i] = ok ? fa[st][i].get() : zero8();
                b[i] = ok ? fb[st][i].get() : zero8();
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t r = row0 + 16 * i + 4 * kg + e, c = col0 + 16 * j + r16;
                if (r < B && c < G) S[r * G + c] = acc[i][j][e];
            }
}

// fp32 arithmetic: 64 x 64 block tiles, operands read directly in MFMA layout.
__global__ __launch_bounds__(256) void coarse_f32(const float *__restrict__ q,
                                                  const float *__restrict__ ck, int32_t B,
                                                  int32_t G, int32_t d, float *__restrict__ S) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, kg = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.y * 64 + (wave >> 1) * 32;
    const int64_t col0 = (int64_t)blockIdx.x * 64 + (wave & 1) * 32;
    const float *qp[2], *cp[2];
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
    for (int k0 = 0; k0 < d; k0 += 4) {
        const int k = k0 + kg;
        float a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            a[i] = qp[i][k];
            b[i] = cp[i][k];
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
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


CoarseWs coarse_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                       int32_t compute_dtype, int32_t top_c, size_t *bytes) {
    Carve cv(ws);
    CoarseWs w{};
    w.scores = cv.take<float>((size_t)B * G);
    const bool convert = compute_dtype == kBF16 && key_dtype == kF32;
    w.q16 = convert ? cv.take<__bf16>((size_t)B * d) : nullptr;
    w.c16 = convert ? cv.take<__bf16>((size_t)G * d) : nullptr;
    // score rows longer than one segment of the segmented top-k are cut into
    // segments (one wave each, then a merge of the segments' lists): many
    // short units keep far more loads in flight than one wave per row
    const int32_t seg = seg_topk_cols();
    w.n_seg = G > seg ? (G + seg - 1) / seg : 1;
    const size_t np = w.n_seg > 1 ? (size_t)B * w.n_seg * seg_topk_slots(top_c) : 0;
    w.p_score = np ? cv.take<float>(np) : nullptr;
    w.p_id = np ? cv.take<int32_t>(np) : nullptr;
    // 64-column tile maxima for the selection that reads only the tiles that matter
    w.n_tile = (G + 63) / 64;
    w.tmax = w.n_seg > 1 && compute_dtype == kBF16 ? cv.take<float>((size_t)B * w.n_tile) : nullptr;
    if (bytes) *bytes = cv.off + 256;
    return w;
}

hipError_t launch_scores(int32_t key_dtype, int32_t compute_dtype, int32_t d, int64_t n,
                         const void *keys, const void *q, int32_t B, float *S, __bf16 *q16,
                         __bf16 *k16, bool convert_q, int n_cu, KernelEvents ev, hipStream_t s,
                         float *tmax, bool *tiled, const __bf16 *keys16) {
    const int32_t G = (int32_t)n;
    if (tiled) *tiled = false;
    if (compute_dtype == kF32) {
        launch_timed(coarse_f32, dim3((G + 63) / 64, (B + 63) / 64), dim3(256), 0, s, ev,
                     static_cast<const float *>(q), static_cast<const float *>(keys), B, G, d, S);
    } else if ((int64_t)((B + BM - 1) / BM) * ((G + BN - 1) / BN) < n_cu || d % BK != 0) {
        const bool small_tiles = (int64_t)((G + 31) / 32) * ((B + 31) / 32) < n_cu;
        const int tile = small_tiles ? 16 : 32;
        const dim3 grid((G + tile - 1) / tile, (B + tile - 1) / tile);
        const float *qf = static_cast<const float *>(q), *cf = static_cast<const float *>(keys);
        const __bf16 *qb = static_cast<const __bf16 *>(q);
        const __bf16 *cb = static_cast<const __bf16 *>(keys);
        if (key_dtype == kF32 && small_tiles)
            launch_timed(coarse_small_bf16<float, 1>, grid, dim3(kWave), 0, s, ev, qf, cf, B, G, d, S);
        else if (key_dtype == kF32)
            launch_timed(coarse_small_bf16<float, 2>, grid, dim3(kWave), 0, s, ev, qf, cf, B, G, d, S);
        else if (small_tiles)
            launch_timed(coarse_small_bf16<__bf16, 1>, grid, dim3(kWave), 0, s, ev, qb, cb, B, G, d, S);
        else
            launch_timed(coarse_small_bf16<__bf16, 2>, grid, dim3(kWave), 0, s, ev, qb, cb, B, G, d, S);
    } else {
        const __bf16 *qa = static_cast<const __bf16 *>(q);
        const __bf16 *ka = static_cast<const __bf16 *>(keys);
        if (key_dtype == kF32) {
            // the keys are rounded here unless the caller's bf16 copy is given
            const int64_t nq = convert_q ? (int64_t)B * d / 8 : 0;
            const int64_t nc = keys16 ? 0 : (int64_t)G * d / 8;
            const int64_t nb = (nq + nc + 255) / 256;
            if (nb > 0)
                hipLaunchKernelGGL(to_bf16, dim3((unsigned)(nb < 8192 ? nb : 8192)), dim3(256), 0,
                                   s, static_cast<const float *>(q), q16, nq,
                                   static_cast<const float *>(keys), k16, nc);
            qa = q16;
            ka = keys16 ? keys16 : k16;
        }
        hipError_t err = hipFuncSetAttribute((const void *)coarse_gemm,
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)kGemmLds);
        if (err != hipSuccess) return err;
        const int tiles = ((B + BM - 1) / BM) * ((G + BN - 1) / BN);
        launch_timed(coarse_gemm, dim3(tiles), dim3(kGemmThreads), kGemmLds, s, ev, qa, ka, B, G,
                     d, S, tmax);
        if (tiled) *tiled = tmax != nullptr;
    }
    return hipGetLastError();
}

hipError_t launch_round_bf16(const float *x, __bf16 *y, int64_t n, hipStream_t s) {
    const int64_t n8 = n / 8, nb = (n8 + 255) / 256;
    if (nb > 0)
        hipLaunchKernelGGL(to_bf16, dim3((unsigned)(nb < 8192 ? nb : 8192)), dim3(256), 0, s, x, y,
                           n8, nullptr, nullptr, (int64_t)0);
    return hipGetLastError();
}

hipError_t launch_coarse(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                         const void *coarse_keys, const void *coarse_keys_bf16, const void *q,
                         int32_t B, int32_t top_c, int32_t *sel, float *sel_score,
                         const CoarseWs &w, int n_cu, KernelEvents ev, hipStream_t s) {
    // tile maxima only where the selection can prune with them
    bool tiled = false;
    float *tmax = top_c <= kWave && top_c < w.n_tile ? w.tmax : nullptr;
    hipError_t err = launch_scores(key_dtype, compute_dtype, d, G, coarse_keys, q, B, w.scores,
                                   w.q16, w.c16, true, n_cu, ev, s, tmax, &tiled,
                                   static_cast<const __bf16 *>(coarse_keys_bf16));
    if (err != hipSuccess) return err;
    return launch_select(B, G, top_c, sel, sel_score, w, s, tiled ? tmax : nullptr);
}

hipError_t launch_select(int32_t B, int32_t G, int32_t top_c, int32_t *sel, float *sel_score,
                         const CoarseWs &w, hipStream_t s, const float *tmax) {
    hipError_t err = hipSuccess;
    // enough tiles for the bound to prune: read only the tiles that can hold the top_c
    if (tmax && top_c <= kWave && top_c < (G + 63) / 64)
        return launch_tile_topk(B, G, w.scores, tmax, top_c, sel, sel_score, s);
    if (w.n_seg == 1)
        return launch_topk(B, 1, G, w.scores, nullptr, nullptr, nullptr, 1.0f, top_c, sel,
                           sel_score, nullptr, nullptr, nullptr, nullptr, s);
    // each (query, segment) keeps its best top_c, then the segments' lists are merged
    err = launch_seg_topk(B, G, G, w.scores, nullptr, 0, top_c, 1.0f, w.p_score, w.p_id, nullptr,
                          nullptr, w.n_seg, 0, s);
    if (err != hipSuccess) return err;
    return launch_topk(B, w.n_seg, seg_topk_slots(top_c), w.p_score, w.p_id, nullptr, nullptr,
                       1.0f, top_c, sel, sel_score, nullptr, nullptr, nullptr, nullptr, s);
}

}  // namespace htam
