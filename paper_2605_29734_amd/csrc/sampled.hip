// Sampled direction choice on gfx950: Alg. 1 Step 2 draws the global
// direction from the policy of Eq. global direction,
//     mu(g) = eps / G + (1 - eps) exp(score_g / tau_g) / sum_g' exp(score_g' / tau_g),
// here c times without replacement, by the Gumbel-top-k construction (Kool,
// van Hoof and Welling, ICML 2019): each cluster's key is log mu(g) plus an
// independent standard Gumbel variate, and the c largest keys are the draw.
//
// Scores are the coarse stage's (<q_b, c_g>, the same GEMM kernels). One wave
// per query row takes the row's maximum and softmax sum, then writes every
// cluster's key; the top-c of the keys is the coarse stage's selection. The
// uniform words come from the caller, or from Philox4x32-10 (Salmon, Moraes,
// Dror and Shaw, SC'11) keyed by (seed, offset): counter
// (g / 4, b, offset_lo, offset_hi), key (seed_lo, seed_hi), word g % 4 of the
// output, so a draw depends only on (seed, offset, b, g).
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int kPolicyWaves = 4;

// Philox4x32 with 10 rounds: each round multiplies counter words 0 and 2 by
// the round constants (high and low halves of the 64-bit products), mixes in
// words 1 and 3 and the key, and the key advances by the Weyl increments
// between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const uint32_t hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
        const uint32_t hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    }
    return c;
}

// Standard Gumbel variate of the uniform word x, u = (x + 1/2) / 2^32:
// -log(-log u), with -log u taken as -log1p(-(1 - u)) when u >= 1/2 so that
// words near 2^32 keep their precision.
__device__ __forceinline__ float gumbel(uint32_t x) {
    const float two32 = 2.3283064365386963e-10f;    // 2^-32
    float w;
    if (x < 0x80000000u) w = -logf(((float)x + 0.5f) * two32);
    else w = -log1pf(-(((float)(0xFFFFFFFFu - x) + 0.5f) * two32));
    return -logf(w);
}

struct PolicyArgs {
    int64_t B, G;
    const float *S;        // [B][G] scores
    float *keys;           // [B][G] out
    float inv_tau, log_eps_g, log_1m_eps;   // 1/tau_g, log(eps/G), log(1 - eps)
    const uint32_t *noise; // [B][G] or NULL (Philox)
    uint32_t seed_lo, seed_hi, off_lo, off_hi;
};

__global__ __launch_bounds__(kWave * kPolicyWaves) void policy_keys(PolicyArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t b = (int64_t)blockIdx.x * kPolicyWaves + (threadIdx.x >> 6);
    if (b >= a.B) return;
    const float *s = a.S + b * a.G;
    float m = -INFINITY;
    for (int64_t g = lane; g < a.G; g += kWave) m = fmaxf(m, s[g]);
    for (int sh = 32; sh >= 1; sh >>= 1) m = fmaxf(m, __shfl_xor(m, sh));
    float z = 0.0f;
    for (int64_t g = lane; g < a.G; g += kWave) z += expf((s[g] - m) * a.inv_tau);
    for (int sh = 32; sh >= 1; sh >>= 1) z += __shfl_xor(z, sh);
    const float logz = logf(z);
    // four consecutive clusters per lane and Philox call
    for (int64_t g0 = 4 * (int64_t)lane; g0 < a.G; g0 += 4 * kWave) {
        uint4 words;
        if (a.noise) {
            const uint32_t *nz = a.noise + b * a.G + g0;
            words = make_uint4(nz[0], g0 + 1 < a.G ? nz[1] : 0u, g0 + 2 < a.G ? nz[2] : 0u,
                               g0 + 3 < a.G ? nz[3] : 0u);
        } else {
            words = philox4x32_10(make_uint4((uint32_t)(g0 >> 2), (uint32_t)b, a.off_lo, a.off_hi),
                                  a.seed_lo, a.seed_hi);
        }
        const uint32_t wv[4] = {words.x, words.y, words.z, words.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t g = g0 + e;
            if (g >= a.G) break;
            // log mu(g) = logaddexp(log(eps / G), log(1 - eps) + log softmax(g))
            const float x = a.log_eps_g, y = a.log_1m_eps + (s[g] - m) * a.inv_tau - logz;
            const float hi = fmaxf(x, y), lo = fminf(x, y);
            const float lmu = lo == -INFINITY ? hi : hi + log1pf(expf(lo - hi));
            a.keys[b * a.G + g] = lmu + gumbel(wv[e]);
        }
    }
}

__global__ void gather_scores(int64_t B, int32_t G, int32_t c, const float *S, const int32_t *sel,
                              float *out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < B * c;
         i += (int64_t)gridDim.x * blockDim.x)
        out[i] = S[(i / c) * G + sel[i]];
}

}  // namespace

SampledWs sampled_layout(void *ws, int32_t B, int32_t G, int32_t d, int32_t key_dtype,
                         int32_t compute_dtype, int32_t top_c, size_t *bytes) {
    SampledWs w{};
    size_t cb = 0;
    w.c = coarse_layout(ws, B, G, d, key_dtype, compute_dtype, top_c, &cb);
    Carve cv(ws ? static_cast<char *>(ws) + cb : nullptr);
    w.keys = cv.take<float>((size_t)B * G);
    w.sel_key = cv.take<float>((size_t)B * top_c);
    if (bytes) *bytes = cb + cv.off + 256;
    return w;
}

hipError_t launch_sampled(int32_t key_dtype, int32_t compute_dtype, int32_t d, int32_t G,
                          const void *coarse_keys, const void *q, int32_t B, int32_t top_c,
                          float eps, float tau_g, const uint32_t *noise, uint64_t seed,
                          uint64_t offset, int32_t *sel, float *sel_score, const SampledWs &w,
                          int n_cu, KernelEvents ev, hipStream_t s) {
    hipError_t err = launch_scores(key_dtype, compute_dtype, d, G, coarse_keys, q, B, w.c.scores,
                                   w.c.q16, w.c.c16, true, n_cu, ev, s);
    if (err != hipSuccess) return err;
    PolicyArgs a{};
    a.B = B;
    a.G = G;
    a.S = w.c.scores;
    a.keys = w.keys;
    a.inv_tau = 1.0f / tau_g;
    a.log_eps_g = eps > 0.0f ? logf(eps / (float)G) : -INFINITY;
    a.log_1m_eps = eps < 1.0f ? log1pf(-eps) : -INFINITY;
    a.noise = noise;
    a.seed_lo = (uint32_t)seed;
    a.seed_hi = (uint32_t)(seed >> 32);
    a.off_lo = (uint32_t)offset;
    a.off_hi = (uint32_t)(offset >> 32);
    hipLaunchKernelGGL(policy_keys, dim3((unsigned)((B + kPolicyWaves - 1) / kPolicyWaves)),
                       dim3(kWave * kPolicyWaves), 0, s, a);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    CoarseWs wk = w.c;
    wk.scores = w.keys;          // select on the perturbed keys
    err = launch_select(B, G, top_c, sel, w.sel_key, wk, s);
    if (err != hipSuccess) return err;
    if (sel_score) {
        const int64_t n = (int64_t)B * top_c;
        hipLaunchKernelGGL(gather_scores, dim3((unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096)),
                           dim3(256), 0, s, (int64_t)B, G, top_c, w.c.scores, sel, sel_score);
    }
    return hipGetLastError();
}

}  // namespace htam
