// Memory build on gfx950: lay transition records out cluster by cluster
// (Eq. HTG, par(l) of Eq. local nodes; the memory append of Eq. memory_update
// collects records in arrival order). A stable counting sort:
//
//   build_zero     clear the per-chunk counts and the error counter;
//   build_count    count the records of each (input chunk, cluster);
//   build_colscan  per cluster, exclusive prefix of the counts over chunks, and
//                  the segment length;
//   build_offsets  exclusive scan of the segment lengths -> seg_offsets;
//   build_scatter  per chunk, sort (cluster, local index) in LDS; a record's
//                  rank inside its cluster within the chunk is its distance to
//                  the start of its run, which gives its output row;
//   build_gather   copy each key row to its output position.
#include "dev.hpp"
#include "internal.hpp"

namespace htam {

namespace {

constexpr int kBuildThreads = 256;
constexpr int kBuildChunk = 4096;      // records per chunk (one LDS sort of 32 KB)
constexpr int kScanThreads = 1024;

__global__ void build_zero(int32_t *cnt, int64_t n, int32_t *err) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        cnt[i] = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *err = 0;
}

__global__ __launch_bounds__(kBuildThreads) void build_count(const int32_t *cluster_of, int64_t n,
                                                             int32_t G, int32_t *cnt, int32_t *err) {
    const int64_t c = blockIdx.x;
    const int64_t i0 = c * kBuildChunk;
    const int64_t i1 = i0 + kBuildChunk < n ? i0 + kBuildChunk : n;
    for (int64_t i = i0 + threadIdx.x; i < i1; i += kBuildThreads) {
        const int32_t g = cluster_of[i];
        if (g >= 0 && g < G) atomicAdd(&cnt[c * G + g], 1);
        else atomicAdd(err, 1);
    }
}

__global__ void build_colscan(int32_t *cnt, int64_t n_chunks, int32_t G, int64_t *len) {
    const int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (g >= G) return;
    int64_t run = 0;
    for (int64_t c = 0; c < n_chunks; ++c) {
        const int32_t v = cnt[c * G + g];
        cnt[c * G + g] = (int32_t)run;
        run += v;
    }
    len[g] = run;
}

__global__ __launch_bounds__(kScanThreads) void build_offsets(const int64_t *len, int32_t G,
                                                              int64_t *off) {
    __shared__ int64_t s[kScanThreads];
    const int t = threadIdx.x;
    const int32_t per = (G + kScanThreads - 1) / kScanThreads;
    const int32_t g0 = min(G, t * per), g1 = min(G, g0 + per);
    int64_t local = 0;
    for (int32_t g = g0; g < g1; ++g) local += len[g];
    s[t] = local;
    __syncthreads();
    for (int o = 1; o < kScanThreads; o <<= 1) {
        const int64_t x = t >= o ? s[t - o] : 0;
        __syncthreads();
        s[t] += x;
        __syncthreads();
    }
    int64_t run = s[t] - local;
    for (int32_t g = g0; g < g1; ++g) {
        off[g] = run;
        run += len[g];
    }
    if (t == kScanThreads - 1) off[G] = s[t];
}

__global__ __launch_bounds__(kBuildThreads) void build_scatter(const int32_t *cluster_of, int64_t n,
                                                               int32_t G, const int32_t *cnt,
                                                               const int64_t *off,
                                                               int32_t *transition_id) {
    __shared__ uint64_t key[kBuildChunk];
    const int t = threadIdx.x;
    const int64_t c = blockIdx.x;
    const int64_t i0 = c * kBuildChunk;
    const int len = (int)((i0 + kBuildChunk < n ? i0 + kBuildChunk : n) - i0);
    for (int li = t; li < kBuildChunk; li += kBuildThreads) {
        uint64_t k = ~0ull;
        if (li < len) {
            const int32_t g = cluster_of[i0 + li];
            const uint32_t hi = (g >= 0 && g < G) ? (uint32_t)g : 0xffffffffu;
            k = ((uint64_t)hi << 32) | (uint32_t)li;
        }
        key[li] = k;
    }
    __syncthreads();
    // ascending bitonic sort of (cluster, local index)
    for (int size = 2; size <= kBuildChunk; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = t; i < kBuildChunk / 2; i += kBuildThreads) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const uint64_t x = key[lo], y = key[hi];
                const bool asc = (lo & size) == 0;
                if (asc ? (x > y) : (x < y)) { key[lo] = y; key[hi] = x; }
            }
            __syncthreads();
        }
    }
    for (int p = t; p < len; p += kBuildThreads) {
        const uint64_t k = key[p];
        const uint32_t g = (uint32_t)(k >> 32);
        if (g == 0xffffffffu) continue;
        // first position of this cluster's run
        int lo = 0, hi = p;
        const uint64_t first = (uint64_t)g << 32;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (key[mid] < first) lo = mid + 1; else hi = mid;
        }
        const int64_t dst = off[g] + cnt[c * G + g] + (p - lo);
        transition_id[dst] = (int32_t)(i0 + (uint32_t)k);
    }
}

// Rows past seg_offsets[G] (the count of valid records) are left untouched.
__global__ void build_gather(const uint4 *keys_in, uint4 *keys_out, const int32_t *transition_id,
                             const int64_t *off, int32_t G, int32_t vec_per_row) {
    const int64_t total = off[G] * vec_per_row;
    for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < total;
         v += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = v / vec_per_row;
        const int32_t e = (int32_t)(v - p * vec_per_row);
        keys_out[v] = keys_in[(int64_t)transition_id[p] * vec_per_row + e];
    }
}

// The tiled copy of the keys (htam_memory_tile). Its header holds each
// segment's first row in the copy, toff[g]: segments padded to multiples of
// 16 rows, so that every segment, and every chunk of one (chunks are
// multiples of 64 rows), starts on a tile.
__global__ __launch_bounds__(kScanThreads) void tile_offsets(const int64_t *off, int32_t G,
                                                             int64_t *toff) {
    __shared__ int64_t s[kScanThreads];
    const int t = threadIdx.x;
    const int32_t per = (G + kScanThreads - 1) / kScanThreads;
    const int32_t g0 = min(G, t * per), g1 = min(G, g0 + per);
    int64_t local = 0;
    for (int32_t g = g0; g < g1; ++g) local += (off[g + 1] - off[g] + 15) & ~int64_t(15);
    s[t] = local;
    __syncthreads();
    for (int o = 1; o < kScanThreads; o <<= 1) {
        const int64_t x = t >= o ? s[t - o] : 0;
        __syncthreads();
        s[t] += x;
        __syncthreads();
    }
    int64_t run = s[t] - local;
    for (int32_t g = g0; g < g1; ++g) {
        toff[g] = run;
        run += (off[g + 1] - off[g] + 15) & ~int64_t(15);
    }
    if (t == kScanThreads - 1) toff[G] = s[t];
}

// Blocks take the tiles of the copy in turn (tile = block index, then every
// grid-th). A tile's segment g is found once, by binary search over toff;
// then every 16-byte piece of the tile, in the copy's order: piece w of block
// (tile, step) (`parts` pieces per 8-element fragment) is part h = w / 64 of
// the fragment of group c = (w / 16) % 4 of the tile's row i = w % 16, read
// from bank row off[g] + 16 tile + i - toff[g] of the row-major keys, or zero
// past the segment's end. Malformed offsets give a wrong copy (the stream's
// offset check rejects it) but no access outside the keys or the copy's
// max_tiles tiles.
__global__ __launch_bounds__(256) void tile_keys(const uint4 *__restrict__ keys, int64_t n_rows,
                                                 const int64_t *__restrict__ off,
                                                 const int64_t *__restrict__ toff, int32_t G,
                                                 int32_t steps, int32_t parts, int64_t max_tiles,
                                                 uint4 *__restrict__ tiles) {
    __shared__ int32_t s_g;
    const int64_t n_tiles = min(toff[G] / 16, max_tiles);
    const int64_t per_block = (int64_t)parts * 64, per_row = (int64_t)steps * 4 * parts;
    const int64_t n = (int64_t)steps * per_block;
    for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {   // uniform bounds
        const int64_t row0 = tile * 16;
        __syncthreads();                         // the previous tile is done with s_g
        if (threadIdx.x == 0) {
            int32_t lo = 0, hi = G - 1;          // last g with toff[g] <= row0
            while (lo < hi) {
                const int32_t mid = (lo + hi + 1) >> 1;
                if (toff[mid] <= row0) lo = mid; else hi = mid - 1;
            }
            s_g = lo;
        }
        __syncthreads();
        const int32_t g = s_g;
        const int64_t j0 = row0 - toff[g], len = off[g + 1] - off[g], src0 = off[g];
        uint4 *out = tiles + tile * n;
        for (int64_t p = threadIdx.x; p < n; p += blockDim.x) {
            const int64_t st = p / per_block;
            const int w = (int)(p - st * per_block);
            const int h = w >> 6, c = (w >> 4) & 3, i = w & 15;
            const int64_t j = j0 + i;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (j < len && src0 + j >= 0 && src0 + j < n_rows)
                v = keys[(src0 + j) * per_row + st * 4 * parts + c * parts + h];
            out[p] = v;
        }
    }
}

}  // namespace

size_t tile_header_bytes(int32_t G) { return ((size_t)(G + 1) * 8 + 255) / 256 * 256; }

hipError_t launch_tile_keys(int64_t n_rows, int32_t G, int32_t d, int32_t elem_bytes,
                            const void *keys, const int64_t *seg_offsets, void *out,
                            hipStream_t s) {
    int64_t *toff = static_cast<int64_t *>(out);
    uint4 *tiles = reinterpret_cast<uint4 *>(static_cast<char *>(out) + tile_header_bytes(G));
    hipLaunchKernelGGL(tile_offsets, dim3(1), dim3(kScanThreads), 0, s, seg_offsets, G, toff);
    const int64_t max_tiles = (n_rows + 15) / 16 + G;
    if (n_rows > 0)
        hipLaunchKernelGGL(tile_keys, dim3((unsigned)(max_tiles < 65536 ? max_tiles : 65536)),
                           dim3(256), 0, s,
                           static_cast<const uint4 *>(keys), n_rows, seg_offsets, toff, G, d / 32,
                           elem_bytes == 4 ? 2 : 1, max_tiles, tiles);
    return hipGetLastError();
}

BuildWs build_layout(void *ws, int64_t n, int32_t G, size_t *bytes) {
    Carve cv(ws);
    BuildWs w{};
    w.chunk = kBuildChunk;
    w.n_chunks = (n + kBuildChunk - 1) / kBuildChunk;
    w.cnt = cv.take<int32_t>((size_t)(w.n_chunks > 0 ? w.n_chunks : 1) * G);
    w.len = cv.take<int64_t>(G);
    w.err = cv.take<int32_t>(1);
    if (bytes) *bytes = cv.off + 256;
    return w;
}

hipError_t launch_build(int64_t n, int32_t G, int32_t row_bytes, const int32_t *cluster_of,
                        const void *keys_in, void *keys_out, int64_t *seg_offsets,
                        int32_t *transition_id, const BuildWs &w, hipStream_t s) {
    const int64_t ncnt = (w.n_chunks > 0 ? w.n_chunks : 1) * (int64_t)G;
    const int zb = (int)((ncnt + 255) / 256 < 4096 ? (ncnt + 255) / 256 : 4096);
    hipLaunchKernelGGL(build_zero, dim3(zb), dim3(256), 0, s, w.cnt, ncnt, w.err);
    if (n > 0)
        hipLaunchKernelGGL(build_count, dim3((unsigned)w.n_chunks), dim3(kBuildThreads), 0, s,
                           cluster_of, n, G, w.cnt, w.err);
    hipLaunchKernelGGL(build_colscan, dim3((G + 255) / 256), dim3(256), 0, s, w.cnt, w.n_chunks, G,
                       w.len);
    hipLaunchKernelGGL(build_offsets, dim3(1), dim3(kScanThreads), 0, s, w.len, G, seg_offsets);
    if (n > 0) {
        hipLaunchKernelGGL(build_scatter, dim3((unsigned)w.n_chunks), dim3(kBuildThreads), 0, s,
                           cluster_of, n, G, w.cnt, seg_offsets, transition_id);
        if (keys_in) {
            const int32_t vpr = row_bytes / 16;
            const int64_t total = n * vpr;
            const int gb = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
            hipLaunchKernelGGL(build_gather, dim3(gb), dim3(256), 0, s,
                               static_cast<const uint4 *>(keys_in), static_cast<uint4 *>(keys_out),
                               transition_id, seg_offsets, G, vpr);
        }
    }
    return hipGetLastError();
}

}  // namespace htam
