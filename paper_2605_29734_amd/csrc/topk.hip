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

// The end of a row's merge, common to the row kernels: the merged softmax
// statistics of the row's lists (lane l holds list l's (lm, lz) for l < 64;
// more lists are read here), then the buffer's top_k sorted and written with
// their weights.
template <int NPL>
__device__ __forceinline__ void finish_row(const TopkArgs &a, int64_t row, uint64_t *buf, int cnt,
                                           int total, float lm, float lz, int lane) {
    static_assert(kTopkStatLists == 1, "one 64-list group of statistics loaded with the keys");
    float M = -INFINITY, Z = 0.0f;
    if (a.slot_max) {
        mz_merge(M, Z, lm, lz, a.cexp);
        for (int l = kWave + lane; l < a.lists; l += kWave)
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

// cap = 64 * NPL >= top_k + 64 keys of LDS per wave.
template <int NPL>
__global__ __launch_bounds__(kWave * kTopkWaves) void topk_rows(TopkArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63;
    // the wave index as a uniform value: the unit's row, segment and bounds,
    // and every address derived from them, then live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

    finish_row<NPL>(a, row, buf, cnt, total, lm[0], lz[0], lane);
}

// Row top-k over lists that are each sorted by descending key (score, then
// the lower id) with their padding (id < 0) at the end, as
// htam_attend_transitions writes them. With m = ceil(top_k / lists), each
// list's first m keys are at least its m-th key, so at least lists x m >=
// top_k keys are at least th, the smallest of the lists' m-th keys, and no
// key below th is in the top-k (th = 0, no bound, when a list is shorter
// than m). A list is read 16 entries at a time, four lists per 64-lane load,
// and only while the last key read from it is above the running threshold,
// which starts just below th and rises with every compaction: a row of
// sorted lists reads a few entries past each list's share of the top-k
// instead of every entry. The result is topk_rows' (the same keys are kept:
// the exact top_k). Up to 64 lists of at least 128 entries (the launcher
// sends other rows to topk_rows).
constexpr int kSortedMaxLists = 64;
constexpr int kSortedMinLen = 128;
constexpr int kSortedChunk = 16;

// compact_select out of line (one copy: the unrolled loop over the lists
// stays small; the row kernels run once per row, their code fetched cold).
struct TopkCompacted {
    int n;
    uint64_t theta;
};
template <int NPL>
__device__ __noinline__ TopkCompacted topk_compact(uint64_t *buf, int n, int k) {
    TopkCompacted r;
    r.theta = 0;
    r.n = compact_select<NPL>(buf, n, k, kWave, threadIdx.x & 63, r.theta);
    return r;
}

template <int NPL>
__global__ __launch_bounds__(kWave * kTopkWaves) void topk_sorted_rows(TopkArgs a, int32_t k_in) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    constexpr int kGroups = kSortedMaxLists / (kWave / kSortedChunk);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * kTopkWaves + wave;
    if (row >= a.rows) return;              // no block-wide synchronisation below
    uint64_t *buf = tbuf + wave * cap;
    const float *sc = a.score + row * a.n;
    const int32_t *ids = a.id ? a.id + row * a.n : nullptr;
    const uint64_t lt_mask = (1ull << lane) - 1;
    const int L = a.lists, sub = lane / kSortedChunk, pos = lane % kSortedChunk;
    auto key_at = [&](int64_t i) -> uint64_t {
        const int32_t id = ids ? ids[i] : (int32_t)i;
        return id >= 0 ? make_key(sc[i], id) : 0ull;
    };
    // statistics, the lists' m-th keys and every list's first chunk, all
    // requested before any is used
    const bool okl = a.slot_max && lane < L;
    const float lm = okl ? a.slot_max[row * L + lane] : -INFINITY;
    const float lz = okl ? a.slot_sum[row * L + lane] : 0.0f;
    const int m = (a.top_k + L - 1) / L;
    uint64_t th = m <= k_in && lane < L ? key_at((int64_t)lane * k_in + m - 1) : ~0ull;
    uint64_t key[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const int l = g * (kWave / kSortedChunk) + sub;
        key[g] = l < L && pos < k_in ? key_at((int64_t)l * k_in + pos) : 0ull;
    }
    th = m <= k_in ? th : 0ull;
#pragma unroll
    for (int sh = 1; sh < kWave; sh <<= 1) {
        uint64_t o;
        switch (sh) {
            case 1: o = lane_xor64<1>(th, lane); break;
            case 2: o = lane_xor64<2>(th, lane); break;
            case 4: o = lane_xor64<4>(th, lane); break;
            case 8: o = lane_xor64<8>(th, lane); break;
            case 16: o = lane_xor64<16>(th, lane); break;
            default: o = lane_xor64<32>(th, lane); break;
        }
        th = o < th ? o : th;
    }
    uint64_t theta = th ? th - 1 : 0;       // offered: keys above theta, i.e. at least th

    int cnt = 0, total = 0;
    for (int c0 = 0;;) {
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            if (g * (kWave / kSortedChunk) < L) {       // groups past the lists: nothing
                const uint64_t k = key[g];
                total += __popcll(__ballot(k != 0));
                const bool pass = k > theta;
                const uint64_t mask = __ballot(pass);
                if (pass) buf[cnt + __popcll(mask & lt_mask)] = k;
                cnt += __popcll(mask);
                if (cnt > cap - kWave) {
                    wave_lds_sync();
                    const TopkCompacted tc = topk_compact<NPL>(buf, cnt, a.top_k);
                    cnt = tc.n;
                    theta = tc.theta > theta ? tc.theta : theta;
                }
            }
        }
        // a list goes on while the last key of its chunk is above the
        // threshold the whole round has raised
        uint64_t live = 0;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            if (g * (kWave / kSortedChunk) < L) {
                const uint64_t cm = __ballot(pos == kSortedChunk - 1 && key[g] > theta);
#pragma unroll
                for (int j = 0; j < kWave / kSortedChunk; ++j)
                    live |= ((cm >> (j * kSortedChunk + kSortedChunk - 1)) & 1ull)
                            << (g * (kWave / kSortedChunk) + j);
            }
        }
        c0 += kSortedChunk;
        if (c0 >= k_in || live == 0) break;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const int l = g * (kWave / kSortedChunk) + sub;
            key[g] = l < L && ((live >> l) & 1) && c0 + pos < k_in
                         ? key_at((int64_t)l * k_in + c0 + pos) : 0ull;
        }
    }
    finish_row<NPL>(a, row, buf, cnt, total, lm, lz, lane);
}

// Segmented row top-k with optional softmax statistics. A unit is one
// segment of kSegCols consecutive columns of one score row, handled by one
// wave that loads the whole segment into registers at once (kSegPer scores
// per lane, every load in flight together; with caller ids, those too).
//
// Candidates: with top_k <= 64, only scores at or above T, the top_k-th
// largest of the 64 lanes' maximum scores, can be in the segment's top-k
// (those maxima are top_k entries scoring at least T). T comes from a radix
// select over the lane maxima, one ballot per bit. Random scores leave a few
// more than top_k candidates; each is written straight to the unit's output
// list (k_slot >= top_k slots, unsorted, padded with (-inf, -1)) at its
// lane's place (a prefix sum of the lanes' counts) in register order. A
// superset of the segment's top-k is all the row
// merge (topk_rows) needs. Only if the candidates overflow the list (many
// ties, or top_k > 64 where no bound is taken) does the unit fall back to
// the LDS buffer with radix-select compaction of topk_rows and write its
// exact top_k, sorted.
//
// Statistics: the segment's maximum (the largest lane maximum), then one sum
// of exp((s - max)/tau) per lane, written for the row merge.
//
// The work per score is a compare and a ballot for most scores: a wave64
// VALU instruction issues over four cycles, so the instruction count, not
// the memory traffic, decides whether this kernel keeps up with HBM.
constexpr int kSegCols = 2048;
constexpr int kSegPer = kSegCols / kWave;  // 32 scores per lane

struct SegArgs {
    int64_t rows, row_stride;      // score rows and the elements between them
    int64_t n;                     // columns per row
    int64_t units;                 // rows * n_seg
    int32_t n_seg, top_k, k_slot;
    int32_t stats;                 // 1: also the segment's softmax statistics
    float cexp;                    // log2(e) / tau
    const float *score;
    const int32_t *col_id;         // column j's id is col_id[j] (IDS), else id_base + j
    int64_t id_base;
    float *o_score;                // [rows][o_lists][k_slot], this call's lists from o_seg0
    int32_t *o_id;
    float *o_m, *o_z;              // [rows][o_lists] (stats only)
    int64_t o_lists, o_seg0;
};

struct SegCompacted {
    int n;
    uint64_t theta;
};
template <int NPL>
__device__ __noinline__ SegCompacted seg_compact(uint64_t *buf, int n, int k) {
    SegCompacted r;
    r.theta = 0;
    r.n = compact_select<NPL>(buf, n, k, kWave, threadIdx.x & 63, r.theta);
    return r;
}

template <int NPL, bool IDS>
__global__ __launch_bounds__(kWave * kTopkWaves) void seg_topk(SegArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63;
    // the wave index as a uniform value: the unit's row, segment and bounds,
    // and every address derived from them, then live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t u = (int64_t)blockIdx.x * kTopkWaves + wave;
    if (u >= a.units) return;               // no block-wide synchronisation below
    const int64_t row = u / a.n_seg, seg = u - row * a.n_seg;
    const int64_t ol = row * a.o_lists + a.o_seg0 + seg;    // output list
    const int64_t c0 = seg * kSegCols;
    const int len = (int)min((int64_t)kSegCols, a.n - c0);
    const float *sc = a.score + row * a.row_stride + c0;
    const uint64_t lt_mask = (1ull << lane) - 1;
    float *os = a.o_score + ol * a.k_slot;
    int32_t *oi = a.o_id + ol * a.k_slot;

    // column j * 64 + lane in register j (unconditional loads clamped into
    // the segment; past-the-end columns become -inf and are never candidates)
    float s[kSegPer];
    int32_t id[IDS ? kSegPer : 1];
    if (len == kSegCols) {
        // a whole segment: one base address, the rest are instruction offsets
        const float *sl = sc + lane;
#pragma unroll
        for (int j = 0; j < kSegPer; ++j) s[j] = sl[j * kWave];
        if constexpr (IDS) {
            const int32_t *il = a.col_id + c0 + lane;
#pragma unroll
            for (int j = 0; j < kSegPer; ++j) id[j] = il[j * kWave];
        }
    } else {
#pragma unroll
        for (int j = 0; j < kSegPer; ++j) s[j] = sc[min(j * kWave + lane, len - 1)];
        if constexpr (IDS) {
#pragma unroll
            for (int j = 0; j < kSegPer; ++j) id[j] = a.col_id[c0 + min(j * kWave + lane, len - 1)];
        }
        // past-the-end columns
#pragma unroll
        for (int j = 0; j < kSegPer; ++j)
            if (j * kWave + lane >= len) s[j] = -INFINITY;
    }
    if constexpr (IDS) {
#pragma unroll
        for (int j = 0; j < kSegPer; ++j)
            if (id[j] < 0) s[j] = -INFINITY;          // not a record
    }
    float lmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < kSegPer; ++j) lmax = fmaxf(lmax, s[j]);

    // T: the top_k-th largest lane maximum, bit by bit on the ordered bits
    float T = -INFINITY;
    if (a.top_k <= kWave) {
        const uint32_t o = lmax == -INFINITY ? 0u : ord_of(lmax);
        uint32_t t = 0;
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t cand = t | (1u << bit);
            if (__popcll(__ballot(o >= cand)) >= a.top_k) t = cand;
        }
        if (t) T = score_of_ord(t);
    }
    // candidates straight to the output list: a lane's passing registers as
    // a bit mask, its first place the sum of the counts of the lanes below
    // it (one ballot per bit of the counts, which are at most 32)
    uint32_t pm = 0;
#pragma unroll
    for (int j = 0; j < kSegPer; ++j) pm |= (s[j] >= T && s[j] != -INFINITY) ? (1u << j) : 0u;
    const int mine = __popc(pm);
    int first = 0, cnt = 0;
#pragma unroll
    for (int b = 0; b < 6; ++b) {
        const uint64_t mb = __ballot((mine >> b) & 1);
        first += __popcll(mb & lt_mask) << b;
        cnt += __popcll(mb) << b;
    }
    if (cnt <= a.k_slot) {
        int pos = first;
#pragma unroll
        for (int j = 0; j < kSegPer; ++j) {
            if ((pm >> j) & 1) {
                os[pos] = s[j];
                oi[pos] = IDS ? id[j] : (int32_t)(a.id_base + c0 + j * kWave + lane);
                ++pos;
            }
        }
        for (int r = cnt + lane; r < a.k_slot; r += kWave) {
            os[r] = -INFINITY;
            oi[r] = -1;
        }
    } else {
        // overflow: the exact top_k through the LDS buffer, sorted
        uint64_t *buf = tbuf + wave * cap;
        int bc = 0;
        uint64_t theta = 0;
#pragma unroll
        for (int j = 0; j < kSegPer; ++j) {
            const bool ok = s[j] >= T && s[j] != -INFINITY;
            const int32_t cid = IDS ? id[j] : (int32_t)(a.id_base + c0 + j * kWave + lane);
            const uint64_t key = ok ? make_key(s[j], cid) : 0;
            const bool in = key > theta;
            const uint64_t mask = __ballot(in);
            if (in) buf[bc + __popcll(mask & lt_mask)] = key;
            bc += __popcll(mask);
            if (bc > cap - kWave) {
                wave_lds_sync();
                const SegCompacted c = seg_compact<NPL>(buf, bc, a.top_k);
                bc = c.n;
                theta = c.theta > theta ? c.theta : theta;
            }
        }
        wave_lds_sync();
        uint64_t v[NPL];
        sort_buffer<NPL>(buf, bc, v, lane);
#pragma unroll
        for (int q = 0; q < NPL; ++q) {
            const int r = q * kWave + lane;
            if (r < a.top_k) {
                const bool ok = r < bc;
                oi[r] = ok ? key_id(v[q]) : -1;
                os[r] = ok ? key_score(v[q]) : -INFINITY;
            }
        }
        for (int r = a.top_k + lane; r < a.k_slot; r += kWave) {
            os[r] = -INFINITY;
            oi[r] = -1;
        }
    }
    if (a.stats) {
        float M = lmax;
        for (int sh = 32; sh >= 1; sh >>= 1) M = fmaxf(M, __shfl_xor(M, sh));
        float z = 0.0f;
        if (M != -INFINITY) {
#pragma clang fp contract(off)
#pragma unroll
            for (int j = 0; j < kSegPer; ++j)
                if (s[j] != -INFINITY) z += fast_exp2((s[j] - M) * a.cexp);
        }
        for (int sh = 32; sh >= 1; sh >>= 1) z += __shfl_xor(z, sh);
        if (lane == 0) {
            a.o_m[ol] = M;
            a.o_z[ol] = z;
        }
    }
}

// Row top-k with tile maxima (the coarse selection after the 256 x 256-tile
// GEMM, which writes each row's maximum over each 64-column tile). One wave
// per row. T, the top_k-th largest of the lanes' maxima of the row's tile
// maxima (lane l holds tiles l, l + 64, ...), is the maximum of top_k
// distinct entries, so at most the row's top_k-th score: the top_k lie in
// the tiles whose maximum reaches T and score at least T. Those tiles are
// read four at a time (one score per lane each) and their entries of at
// least T appended to the wave's LDS buffer as in topk_rows, compacted when
// it fills.
constexpr int kTileCols = 64;

struct TileArgs {
    int64_t rows, n;
    int32_t n_tile, top_k;
    const float *score, *tmax;
    int32_t *out_id;
    float *out_score;
};

template <int NPL>
__global__ __launch_bounds__(kWave * kTopkWaves) void tile_topk(TileArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    constexpr int kTilesPerRound = 4;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * kTopkWaves + wave;
    if (row >= a.rows) return;              // no block-wide synchronisation below
    uint64_t *buf = tbuf + wave * cap;
    const uint64_t lt_mask = (1ull << lane) - 1;
    const float *tm = a.tmax + row * a.n_tile;
    const float *sc = a.score + row * a.n;

    float lm = -INFINITY;
    for (int t = lane; t < a.n_tile; t += kWave) lm = fmaxf(lm, tm[t]);
    float T = -INFINITY;
    {
        const uint32_t o = lm == -INFINITY ? 0u : ord_of(lm);
        uint32_t th = 0;
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t cand = th | (1u << bit);
            if (__popcll(__ballot(o >= cand)) >= a.top_k) th = cand;
        }
        if (th) T = score_of_ord(th);
    }

    int cnt = 0;
    uint64_t theta = 0;
    for (int tb = 0; tb < a.n_tile; tb += kWave) {
        const int t = tb + lane;
        const float mt = t < a.n_tile ? tm[t] : -INFINITY;
        uint64_t pending = __ballot(mt >= T && mt != -INFINITY);
        while (pending) {
            // up to four qualifying tiles: every load issued before any is used
            int tile[kTilesPerRound];
#pragma unroll
            for (int r = 0; r < kTilesPerRound; ++r) {
                tile[r] = pending ? tb + __builtin_ctzll(pending) : -1;
                pending &= pending ? pending - 1 : 0;
            }
            float v[kTilesPerRound];
#pragma unroll
            for (int r = 0; r < kTilesPerRound; ++r) {
                const int64_t c = (int64_t)(tile[r] < 0 ? tile[0] : tile[r]) * kTileCols + lane;
                v[r] = sc[c < a.n ? c : a.n - 1];
            }
#pragma unroll
            for (int r = 0; r < kTilesPerRound; ++r) {
                const int64_t c = (int64_t)tile[r] * kTileCols + lane;
                const bool ok = tile[r] >= 0 && c < a.n && v[r] >= T;
                const uint64_t key = ok ? make_key(v[r], (int32_t)c) : 0;
                const bool pass = key > theta;
                const uint64_t mask = __ballot(pass);
                if (pass) buf[cnt + __popcll(mask & lt_mask)] = key;
                cnt += __popcll(mask);
                if (cnt > cap - kWave) {
                    wave_lds_sync();
                    cnt = compact_select<NPL>(buf, cnt, a.top_k, kWave, lane, theta);
                }
            }
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
            a.out_id[row * a.top_k + r] = ok ? key_id(v[q]) : -1;
            a.out_score[row * a.top_k + r] = ok ? key_score(v[q]) : -INFINITY;
        }
    }
}

// The same selection for rows of 65 to 512 tiles, in about three memory
// round trips instead of one per round of tile maxima and per four tiles:
// every tile maximum is held in registers (eight per lane), T is the exact
// top_k-th largest of them (a radix select, one ballot per register and
// bit), so that hardly more than top_k tiles reach it; their ids are listed
// in LDS and the tiles read sixteen at a time.
constexpr int kHeldPer = 8;
constexpr int kHeldTiles = kHeldPer * kWave;
constexpr int kHeldBatch = 16;

template <int NPL>
__global__ __launch_bounds__(kWave * kTopkWaves) void tile_topk_held(TileArgs a) {
    extern __shared__ __align__(16) uint64_t tbuf[];
    constexpr int cap = NPL * kWave;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * kTopkWaves + wave;
    if (row >= a.rows) return;              // no block-wide synchronisation below
    uint64_t *buf = tbuf + wave * cap;
    int32_t *list = reinterpret_cast<int32_t *>(tbuf + kTopkWaves * cap) + wave * kHeldTiles;
    const uint64_t lt_mask = (1ull << lane) - 1;
    const float *tm = a.tmax + row * a.n_tile;
    const float *sc = a.score + row * a.n;
    const int R = (a.n_tile + kWave - 1) / kWave;        // registers in use, at most kHeldPer
    uint32_t o[kHeldPer];                                // ordered tile maxima, 0: none
#pragma unroll
    for (int r = 0; r < kHeldPer; ++r) {
        const int t = r * kWave + lane;
        const float m = r < R && t < a.n_tile ? tm[t] : -INFINITY;
        o[r] = m == -INFINITY ? 0u : ord_of(m);
    }
    uint32_t th = 0;                                     // the top_k-th largest (0: fewer tiles)
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t cand = th | (1u << bit);
        int c = 0;
#pragma unroll
        for (int r = 0; r < kHeldPer; ++r)
            if (r < R) c += __popcll(__ballot(o[r] >= cand));
        if (c >= a.top_k) th = cand;
    }
    const float T = th ? score_of_ord(th) : -INFINITY;
    const uint32_t lo = th ? th : 1u;
    int n_list = 0;
#pragma unroll
    for (int r = 0; r < kHeldPer; ++r) {
        if (r < R) {
            const bool q = o[r] >= lo;
            const uint64_t m = __ballot(q);
            if (q) list[n_list + __popcll(m & lt_mask)] = r * kWave + lane;
            n_list += __popcll(m);
        }
    }
    wave_lds_sync();

    int cnt = 0;
    uint64_t theta = 0;
    for (int b0 = 0; b0 < n_list; b0 += kHeldBatch) {
        int tile[kHeldBatch];
        float v[kHeldBatch];
#pragma unroll
        for (int j = 0; j < kHeldBatch; ++j) tile[j] = b0 + j < n_list ? list[b0 + j] : -1;
#pragma unroll
        for (int j = 0; j < kHeldBatch; ++j) {           // every load in flight at once
            const int64_t c = (int64_t)(tile[j] < 0 ? tile[0] : tile[j]) * kTileCols + lane;
            v[j] = sc[c < a.n ? c : a.n - 1];
        }
#pragma unroll
        for (int j = 0; j < kHeldBatch; ++j) {
            const int64_t c = (int64_t)tile[j] * kTileCols + lane;
            const bool ok = tile[j] >= 0 && c < a.n && v[j] >= T;
            const uint64_t key = ok ? make_key(v[j], (int32_t)c) : 0;
            const bool pass = key > theta;
            const uint64_t mask = __ballot(pass);
            if (pass) buf[cnt + __popcll(mask & lt_mask)] = key;
            cnt += __popcll(mask);
            if (cnt > cap - kWave) {
                wave_lds_sync();
                const TopkCompacted tc = topk_compact<NPL>(buf, cnt, a.top_k);
                cnt = tc.n;
                theta = tc.theta > theta ? tc.theta : theta;
            }
        }
    }
    wave_lds_sync();
    uint64_t w[NPL];
    sort_buffer<NPL>(buf, cnt, w, lane);
    const int kept = cnt < a.top_k ? cnt : a.top_k;
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
        const int r = q * kWave + lane;
        if (r < a.top_k) {
            const bool ok = r < kept;
            a.out_id[row * a.top_k + r] = ok ? key_id(w[q]) : -1;
            a.out_score[row * a.top_k + r] = ok ? key_score(w[q]) : -INFINITY;
        }
    }
}

}  // namespace

int32_t seg_topk_cols() { return kSegCols; }
int32_t seg_topk_slots(int32_t top_k) { return top_k < kWave ? kWave : top_k; }

hipError_t launch_seg_topk(int64_t rows, int64_t row_stride, int64_t n, const float *score,
                           const int32_t *col_id, int64_t id_base, int32_t top_k, float tau,
                           float *o_score, int32_t *o_id, float *o_m, float *o_z, int64_t o_lists,
                           int64_t o_seg0, hipStream_t s) {
    if (rows == 0 || n == 0) return hipSuccess;
    SegArgs a{};
    a.rows = rows;
    a.row_stride = row_stride;
    a.n = n;
    a.n_seg = (int32_t)((n + kSegCols - 1) / kSegCols);
    a.units = rows * a.n_seg;
    a.top_k = top_k;
    a.k_slot = seg_topk_slots(top_k);
    a.stats = o_m != nullptr;
    a.cexp = 1.4426950408889634f / tau;
    a.score = score;
    a.col_id = col_id;
    a.id_base = id_base;
    a.o_score = o_score;
    a.o_id = o_id;
    a.o_m = o_m;
    a.o_z = o_z;
    a.o_lists = o_lists;
    a.o_seg0 = o_seg0;
    const int npl = next_pow2(top_k + kWave) / kWave;
    const dim3 grid((unsigned)((a.units + kTopkWaves - 1) / kTopkWaves)), block(kWave * kTopkWaves);
    const size_t smem = (size_t)kTopkWaves * npl * kWave * 8;
    const bool ids = col_id != nullptr;
    switch (npl * 2 + (ids ? 1 : 0)) {
        case 4: hipLaunchKernelGGL((seg_topk<2, false>), grid, block, smem, s, a); break;
        case 5: hipLaunchKernelGGL((seg_topk<2, true>), grid, block, smem, s, a); break;
        case 8: hipLaunchKernelGGL((seg_topk<4, false>), grid, block, smem, s, a); break;
        case 9: hipLaunchKernelGGL((seg_topk<4, true>), grid, block, smem, s, a); break;
        case 16: hipLaunchKernelGGL((seg_topk<8, false>), grid, block, smem, s, a); break;
        case 17: hipLaunchKernelGGL((seg_topk<8, true>), grid, block, smem, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_tile_topk(int64_t rows, int64_t n, const float *score, const float *tmax,
                            int32_t top_k, int32_t *out_id, float *out_score, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (top_k > kWave) return hipErrorInvalidValue;
    TileArgs a{};
    a.rows = rows;
    a.n = n;
    a.n_tile = (int32_t)((n + kTileCols - 1) / kTileCols);
    a.top_k = top_k;
    a.score = score;
    a.tmax = tmax;
    a.out_id = out_id;
    a.out_score = out_score;
    const dim3 grid((unsigned)((rows + kTopkWaves - 1) / kTopkWaves)), block(kWave * kTopkWaves);
    // buffers of top_k + 64 keys at least (compaction when fewer than 64 slots remain)
    const int npl = next_pow2(top_k + kWave) / kWave;
    const size_t smem = (size_t)kTopkWaves * npl * kWave * 8;
    // more tiles than lanes: a lane's maximum merges several tiles and its
    // bound admits more tiles than the exact one (before_after_f32, 256
    // tiles: 32 -> 28 us); up to 64 tiles both bounds are the same and the
    // exact one costs its radix select (zipf_large_bf16: 16.5 -> 19 us)
    if (a.n_tile > kWave && a.n_tile <= kHeldTiles) {
        const size_t sm2 = smem + (size_t)kTopkWaves * kHeldTiles * 4;   // and the tile lists
        switch (npl) {
            case 2: hipLaunchKernelGGL(tile_topk_held<2>, grid, block, sm2, s, a); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    switch (npl) {
        case 2: hipLaunchKernelGGL(tile_topk<2>, grid, block, smem, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_topk(int32_t rows, int32_t lists, int32_t k_in, const float *score,
                       const int32_t *id, const float *slot_max, const float *slot_sum, float tau,
                       int32_t top_k, int32_t *out_id, float *out_score, float *out_weight,
                       float *row_max, float *row_sum, int32_t *out_count, hipStream_t s,
                       bool sorted_lists) {
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
    // the smallest buffer that holds top_k + 64 keys; twice that when a row
    // offers at least 16 times as many entries (zipf_large_bf16's final merge:
    // 2048 entries, k = 64: 64 -> 39 us): a compaction every 64 entries that
    // pass the threshold becomes one every 192, while for shorter rows the
    // larger sort costs more than it saves
    const int npl0 = next_pow2(top_k + kWave) / kWave;
    const int npl = npl0 < 8 && a.n >= (int64_t)16 * kWave * npl0 ? 2 * npl0 : npl0;
    const dim3 grid((unsigned)((rows + kTopkWaves - 1) / kTopkWaves)), block(kWave * kTopkWaves);
    const size_t smem = (size_t)kTopkWaves * npl * kWave * 8;
    // sorted lists of at least 128 entries: a row reads a chunk or two of
    // each instead of all (before_after_f32's final merge, 16 lists of 128:
    // 63 -> 51 us); on shorter lists the rounds of chunks cost more than the
    // entries they skip (zipf_large_bf16, 32 lists of 64: 36 -> 54 us)
    if (sorted_lists && lists <= kSortedMaxLists && k_in >= kSortedMinLen) {
        switch (npl) {
            case 2: hipLaunchKernelGGL(topk_sorted_rows<2>, grid, block, smem, s, a, k_in); break;
            case 4: hipLaunchKernelGGL(topk_sorted_rows<4>, grid, block, smem, s, a, k_in); break;
            case 8: hipLaunchKernelGGL(topk_sorted_rows<8>, grid, block, smem, s, a, k_in); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    switch (npl) {
        case 2: hipLaunchKernelGGL(topk_rows<2>, grid, block, smem, s, a); break;
        case 4: hipLaunchKernelGGL(topk_rows<4>, grid, block, smem, s, a); break;
        case 8: hipLaunchKernelGGL(topk_rows<8>, grid, block, smem, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace htam
