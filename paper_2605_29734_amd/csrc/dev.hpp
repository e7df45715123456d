// Device helpers shared by the gfx950 kernels: MFMA fragment loads, ordered
// 64-bit ranking keys, softmax-statistic merges, and wave-level sorting and
// top-k compaction in registers.
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
// Contraction into fused multiply-adds is off here and in the stream's
// statistics update: every product and sum is rounded on its own, in source
// order, so the bits of a (query, slot)'s statistics do not depend on which
// inlined or templated copy of the code computed them (a query's place in its
// cluster's list, and so its pass and query tile, depends on atomic order).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void mz_merge(float &m, float &z, float m2, float z2, float c) {
#pragma clang fp contract(off)
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; z = z2; return; }
    float M = fmaxf(m, m2);
    z = z * exp2f((m - M) * c) + z2 * exp2f((m2 - M) * c);
    m = M;
}

// 2^x by the hardware instruction (v_exp_f32, about 1 ulp), without the
// denormal-range handling of exp2f: results below the smallest normal float
// may come out as zero. Used for softmax terms exp((s - m)/tau) <= 1 summed
// next to the maximum's own term 1, where such terms do not change the sum.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// s_waitcnt with only a vector-memory count (the other counters left free):
// at most N of this wave's vector memory loads still outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
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

// A fragment as loaded (bf16 as is; fp32 rounded to bf16 when used).
template <typename T>
struct RawFrag;
template <>
struct RawFrag<__bf16> {
    uint4 v;
    __device__ __forceinline__ void load(const __bf16 *p) { v = *reinterpret_cast<const uint4 *>(p); }
    __device__ __forceinline__ bf16x8_t get() const { return __builtin_bit_cast(bf16x8_t, v); }
};
template <>
struct RawFrag<float> {
    float4 lo, hi;
    __device__ __forceinline__ void load(const float *p) {
        lo = reinterpret_cast<const float4 *>(p)[0];
        hi = reinterpret_cast<const float4 *>(p)[1];
    }
    __device__ __forceinline__ bf16x8_t get() const {
        bf16x8_t r;
        r[0] = (__bf16)lo.x; r[1] = (__bf16)lo.y; r[2] = (__bf16)lo.z; r[3] = (__bf16)lo.w;
        r[4] = (__bf16)hi.x; r[5] = (__bf16)hi.y; r[6] = (__bf16)hi.z; r[7] = (__bf16)hi.w;
        return r;
    }
};

// Wait for this wave's LDS traffic and stop the compiler from moving memory
// operations across this point (LDS operations of one wave complete in order).
__device__ __forceinline__ void wave_lds_sync() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Block barrier for LDS only: this thread's LDS operations complete, then the
// workgroup barrier; its global loads stay in flight (__syncthreads would wait
// for them). The memory clobber keeps the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void block_lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}


// ---------------------------------------------------------------------------
// Register-resident sorting networks over one wave. A list of 64*NPL keys is
// held as v[j] on every lane, element index i = j*64 + lane. Every stage's
// stride is a compile-time constant: strides >= 64 exchange registers within a
// lane; strides 1..32 exchange across lanes without going through LDS:
//   1, 2   quad permutations (DPP);
//   4      two row rotations by 4 and 12 (DPP), one of them selected per lane;
//   8      row rotation by 8 (DPP);
//   16, 32 v_permlane16_swap / v_permlane32_swap (gfx950).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    const uint32_t lo = __shfl((uint32_t)v, src);
    const uint32_t hi = __shfl((uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}

// The value held by lane (lane ^ M).
template <int M>
__device__ __forceinline__ uint32_t lane_xor32(uint32_t x, int lane) {
    if constexpr (M == 1) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);   // [1,0,3,2]
    } else if constexpr (M == 2) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);   // [2,3,0,1]
    } else if constexpr (M == 4) {
        const uint32_t a = (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x124, 0xF, 0xF, false);
        const uint32_t b = (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x12C, 0xF, 0xF, false);
        return (lane & 4) ? a : b;
    } else if constexpr (M == 8) {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x128, 0xF, 0xF, false);
    } else if constexpr (M == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return (lane & 16) ? r[0] : r[1];
    } else {
        static_assert(M == 32, "lane_xor32: mask must be a power of two below 64");
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (lane & 32) ? r[0] : r[1];
    }
}
template <int M>
__device__ __forceinline__ uint64_t lane_xor64(uint64_t v, int lane) {
    const uint32_t lo = lane_xor32<M>((uint32_t)v, lane);
    const uint32_t hi = lane_xor32<M>((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

template <int NPL>
struct Log2Npl {
    static constexpr int value = NPL == 1 ? 6 : NPL == 2 ? 7 : NPL == 4 ? 8 : NPL == 8 ? 9 : -1;
};

// One compare-exchange stage: elements i and i ^ STRIDE, the pair ordered
// descending when desc_all, else by the bitonic-sort rule for block `size`.
template <int NPL, int STRIDE>
__device__ __forceinline__ void wave_cx(uint64_t (&v)[NPL], int lane, int size, bool desc_all) {
    if constexpr (STRIDE >= kWave) {
        constexpr int js = STRIDE / kWave;
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            if ((j & js) == 0) {
                const int j2 = j | js;
                const bool desc = desc_all || ((j * kWave) & size) == 0;
                const uint64_t x = v[j], y = v[j2];
                const bool sw = desc ? (x < y) : (x > y);
                v[j] = sw ? y : x;
                v[j2] = sw ? x : y;
            }
        }
    } else {
        const bool lo = (lane & STRIDE) == 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const uint64_t y = lane_xor64<STRIDE>(v[j], lane);
            const bool desc = desc_all || ((j * kWave + lane) & size) == 0;
            const uint64_t mx = v[j] > y ? v[j] : y, mn = v[j] > y ? y : v[j];
            v[j] = (lo == desc) ? mx : mn;
        }
    }
}

// Stages of block size 2^LS with strides 2^LT, 2^(LT-1), ..., 1, on NB lists
// side by side (independent exchanges overlap).
template <int NB, int NPL, int LS, int LT>
struct BitonicStages {
    __device__ static __forceinline__ void run(uint64_t (&v)[NB][NPL], int lane) {
#pragma unroll
        for (int b = 0; b < NB; ++b) wave_cx<NPL, (1 << LT)>(v[b], lane, 1 << LS, false);
        if constexpr (LT > 0) BitonicStages<NB, NPL, LS, LT - 1>::run(v, lane);
    }
};
template <int NB, int NPL, int LS>
struct BitonicSort {
    __device__ static __forceinline__ void run(uint64_t (&v)[NB][NPL], int lane) {
        if constexpr (LS > 1) BitonicSort<NB, NPL, LS - 1>::run(v, lane);
        BitonicStages<NB, NPL, LS, LS - 1>::run(v, lane);
    }
};
template <int NPL, int LT>
struct MergeStages {
    __device__ static __forceinline__ void run(uint64_t (&v)[NPL], int lane) {
        wave_cx<NPL, (1 << LT)>(v, lane, 0, true);
        if constexpr (LT > 0) MergeStages<NPL, LT - 1>::run(v, lane);
    }
};

// Sort NB lists of 64*NPL keys each, descending, side by side.
template <int NB, int NPL>
__device__ __forceinline__ void wave_sort_multi(uint64_t (&v)[NB][NPL], int lane) {
    BitonicSort<NB, NPL, Log2Npl<NPL>::value>::run(v, lane);
}

// Sort 64*NPL keys descending.
template <int NPL>
__device__ __forceinline__ void wave_sort_regs(uint64_t (&v)[NPL], int lane) {
    uint64_t(&w)[1][NPL] = *reinterpret_cast<uint64_t(*)[1][NPL]>(&v);
    BitonicSort<1, NPL, Log2Npl<NPL>::value>::run(w, lane);
}

// Loads the n keys of an LDS buffer (n wave-uniform, at most 64 NPL) into v
// sorted descending (register j holds ranks 64 j + lane; empty slots 0).
// Up to 64 keys are sorted as one register, a fraction of the cost of all NPL.
template <int NPL>
__device__ __forceinline__ void sort_buffer(const uint64_t *buf, int n, uint64_t (&v)[NPL],
                                            int lane) {
    n = __builtin_amdgcn_readfirstlane(n);
    if (NPL > 1 && n <= kWave) {
        uint64_t one[1] = {lane < n ? buf[lane] : 0};
        wave_sort_regs<1>(one, lane);
        v[0] = one[0];
#pragma unroll
        for (int q = 1; q < NPL; ++q) v[q] = 0;
    } else {
#pragma unroll
        for (int q = 0; q < NPL; ++q) v[q] = (q * kWave + lane < n) ? buf[q * kWave + lane] : 0;
        wave_sort_regs<NPL>(v, lane);
    }
}

// a, b: sorted descending. Leaves in a the 64*NPL largest of a and b, sorted.
template <int NPL>
__device__ __forceinline__ void wave_merge_top(uint64_t (&a)[NPL], const uint64_t (&b)[NPL],
                                               int lane) {
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const uint64_t rb = shfl64(b[NPL - 1 - j], kWave - 1 - lane);
        a[j] = a[j] > rb ? a[j] : rb;      // bitonic: the top half of a u b
    }
    MergeStages<NPL, Log2Npl<NPL>::value - 1>::run(a, lane);
}

// Element i (held by lane i % 64 as v[i / 64]) broadcast to the whole wave.
template <int NPL>
__device__ __forceinline__ uint64_t wave_element(const uint64_t (&v)[NPL], int i) {
    uint64_t x = 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j)
        if (j == i / kWave) x = v[j];
    return shfl64(x, i % kWave);
}

// Compaction of a top-k buffer of n keys (n > k, capacity 64*NPL) by one wave.
// A radix select over the keys' high halves (the ordered scores) looks for T,
// the k-th largest score in the buffer, one bit at a time from the highest bit
// in which the buffer's scores differ (the bits above are the same in all of
// them and so in T). Every prefix found on the way is at most T, so keeping
// all keys scoring >= the current prefix keeps the true top k; the select
// stops as soon as that keeps few enough keys to leave `room` free slots
// (most buffers need only the first several bits), and the threshold becomes
// the prefix: later keys must score at least that much. If even the full T
// leaves fewer than `room` free slots (ties at T), the buffer is sorted
// instead and cut to exactly k keys (threshold = the k-th key). Returns the
// new count.
template <int NPL>
__device__ __forceinline__ int compact_select(uint64_t *gbuf, int n, int k, int room, int lane,
                                              uint64_t &theta) {
    constexpr int cap = NPL * kWave;
    // The buffer is in LDS (every caller's is): addressed as such, its reads
    // and writes are LDS operations even where address-space inference does
    // not reach (flat ones would also wait for the wave's global loads).
    typedef __attribute__((address_space(3))) uint64_t lds_u64;
    lds_u64 *buf = (lds_u64 *)gbuf;
    n = __builtin_amdgcn_readfirstlane(n);     // wave-uniform arguments, held as such
    k = __builtin_amdgcn_readfirstlane(k);
    room = __builtin_amdgcn_readfirstlane(room);
    uint64_t v[NPL];
    uint32_t hi[NPL];
    uint64_t vm[NPL];             // lanes holding a key, per register (wave-uniform masks)
    uint32_t hand = 0xffffffffu, hor = 0;
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
        const bool ok = q * kWave + lane < n;
        v[q] = ok ? buf[q * kWave + lane] : 0;
        hi[q] = (uint32_t)(v[q] >> 32);
        vm[q] = __ballot(v[q] != 0);
        if (ok) {
            hand &= hi[q];
            hor |= hi[q];
        }
    }
    hand &= lane_xor32<1>(hand, lane);
    hor |= lane_xor32<1>(hor, lane);
    hand &= lane_xor32<2>(hand, lane);
    hor |= lane_xor32<2>(hor, lane);
    hand &= lane_xor32<4>(hand, lane);
    hor |= lane_xor32<4>(hor, lane);
    hand &= lane_xor32<8>(hand, lane);
    hor |= lane_xor32<8>(hor, lane);
    hand &= lane_xor32<16>(hand, lane);
    hor |= lane_xor32<16>(hor, lane);
    hand &= lane_xor32<32>(hand, lane);
    hor |= lane_xor32<32>(hor, lane);
    // the same in every lane: made explicit, so that the select below is a
    // scalar loop (ballots and their counts) rather than a lane-masked one
    hand = __builtin_amdgcn_readfirstlane(hand);
    hor = __builtin_amdgcn_readfirstlane(hor);
    const uint32_t diff = hand ^ hor;
    const int top = diff ? 31 - __builtin_clz(diff) : -1;
    uint32_t T = top < 0 ? hand : (top == 31 ? 0u : hand & ~((2u << top) - 1u));
    int keep = n;                 // keys scoring >= T (all of them at the common prefix)
    for (int bit = top; bit >= 0 && keep > cap - room; --bit) {
        const uint32_t cand = T | (1u << bit);
        int c = 0;
#pragma unroll
        for (int q = 0; q < NPL; ++q) c += __popcll(__ballot(hi[q] >= cand) & vm[q]);
        if (c >= k) {
            T = cand;
            keep = c;
        }
    }
    const uint64_t lt_mask = (1ull << lane) - 1;
    wave_lds_sync();
    if (keep <= cap - room) {
        int base = 0;
#pragma unroll
        for (int q = 0; q < NPL; ++q) {
            const uint64_t mask = __ballot(hi[q] >= T) & vm[q];
            if ((mask >> lane) & 1) buf[base + __popcll(mask & lt_mask)] = v[q];
            base += __popcll(mask);
        }
        theta = (uint64_t)T << 32;
        wave_lds_sync();
        return keep;
    }
    wave_sort_regs<NPL>(v, lane);
#pragma unroll
    for (int q = 0; q < NPL; ++q)
        if (q * kWave + lane < k) buf[q * kWave + lane] = v[q];
    theta = wave_element<NPL>(v, k - 1);
    wave_lds_sync();
    return k;
}

__host__ __device__ constexpr int next_pow2(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

}  // namespace htam
