// Device helpers shared by the gfx950 kernels: MFMA fragment loads, ordered
// 64-bit ranking keys, softmax-statistic merges and wave-level LDS sorting.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace htam {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Ranking keys. A candidate (score s, caller id) maps to one uint64 whose
// unsigned order is "descending score, then ascending id": the high half is
// the float's bits made monotone (negative floats inverted, positive floats
// with the sign bit set), the low half is ~id. -0.0 is folded into +0.0 first
// so that the two zeros tie, as they do in real arithmetic. Key 0 is below
// every real candidate and marks "empty".
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ord_of(float s) {
    uint32_t u = __float_as_uint(s + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float score_of_ord(uint32_t o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__device__ __forceinline__ uint64_t make_key(float s, int32_t id) {
    return ((uint64_t)ord_of(s) << 32) | (uint64_t)(~(uint32_t)id);
}
__device__ __forceinline__ float key_score(uint64_t k) { return score_of_ord((uint32_t)(k >> 32)); }
__device__ __forceinline__ int32_t key_id(uint64_t k) { return (int32_t)(~(uint32_t)k); }

// ---------------------------------------------------------------------------
// Online softmax statistics with temperature: (m, Z) with
// Z = sum exp((s - m) / tau). Evaluated as exp2((s - m) * c), c = log2(e)/tau.
// (m, Z) (+) (m', Z') = (M, Z e^{(m-M)/tau} + Z' e^{(m'-M)/tau}), M = max(m, m').
// An empty set is (-inf, 0).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void mz_merge(float &m, float &z, float m2, float z2, float c) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; z = z2; return; }
    float M = fmaxf(m, m2);
    z = z * exp2f((m - M) * c) + z2 * exp2f((m2 - M) * c);
    m = M;
}

// ---------------------------------------------------------------------------
// Fragment loads for v_mfma_f32_16x16x32_bf16: 8 consecutive elements of one
// row starting at p, as bf16 (fp32 storage is rounded to nearest even by the
// hardware conversion). p must be 16-byte aligned.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bf16x8_t load8(const __bf16 *p) {
    return *reinterpret_cast<const bf16x8_t *>(p);
}
__device__ __forceinline__ bf16x8_t load8(const float *p) {
    const float4 a = reinterpret_cast<const float4 *>(p)[0];
    const float4 b = reinterpret_cast<const float4 *>(p)[1];
    bf16x8_t r;
    r[0] = (__bf16)a.x; r[1] = (__bf16)a.y; r[2] = (__bf16)a.z; r[3] = (__bf16)a.w;
    r[4] = (__bf16)b.x; r[5] = (__bf16)b.y; r[6] = (__bf16)b.z; r[7] = (__bf16)b.w;
    return r;
}
__device__ __forceinline__ bf16x8_t zero8() {
    bf16x8_t r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (__bf16)0.0f;
    return r;
}

// Wait for this wave's LDS traffic and stop the compiler from moving memory
// operations across this point (LDS operations of one wave complete in order).
__device__ __forceinline__ void wave_lds_sync() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Descending bitonic sort of n = 2^j (2 <= n) 64-bit keys in LDS by one wave.
__device__ __forceinline__ void wave_sort_desc(uint64_t *a, int n, int lane) {
    for (int size = 2; size <= n; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = lane; i < (n >> 1); i += kWave) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const uint64_t x = a[lo], y = a[hi];
                const bool desc = (lo & size) == 0;
                if (desc ? (x < y) : (x > y)) { a[lo] = y; a[hi] = x; }
            }
            wave_lds_sync();
        }
    }
}

__host__ __device__ constexpr int next_pow2(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// ---------------------------------------------------------------------------
// Top-k accumulator of one row in LDS: a buffer of `cap` (a power of two)
// keys, a fill count and a threshold (the k-th best key seen once at least k
// keys were kept; 0 before). Keys above the threshold are appended with an LDS
// atomic; a compaction sorts the buffer and keeps the k best. The caller
// compacts whenever fewer free slots remain than it may append before the
// next compaction point, so an append never overflows.
// ---------------------------------------------------------------------------
struct TopkRow {
    uint64_t *buf;
    uint32_t *cnt;
    uint64_t *theta;
};

__device__ __forceinline__ void topk_offer(const TopkRow &r, uint64_t key) {
    if (key > *r.theta) {
        const uint32_t p = atomicAdd(r.cnt, 1u);
        r.buf[p] = key;
    }
}

// Compact (one wave): sort the kept keys and keep the best k.
__device__ __forceinline__ void topk_compact(const TopkRow &r, int k, int lane) {
    const int n = (int)*r.cnt;
    const int np = next_pow2(n < 2 ? 2 : n);
    for (int i = n + lane; i < np; i += kWave) r.buf[i] = 0;
    wave_lds_sync();
    wave_sort_desc(r.buf, np, lane);
    if (lane == 0) {
        if (n >= k) { *r.cnt = (uint32_t)k; *r.theta = r.buf[k - 1]; }
    }
    wave_lds_sync();
}

}  // namespace htam
