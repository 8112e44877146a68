// Sum of clipped gradients of an embedding layer (Algorithm 1 applied to a
// layer whose input is the one-hot encoding of token ids):
//
//   G[v, :] = sum_i C_i sum_{t : x_it = v} g_it        for every v in [0, V).
//
// Deterministic grouping, no floating-point atomics, any number of tokens:
//  1. the n = B*T keys (id << 32 | flat token index) are sorted by id with a
//     stable least-significant-digit radix sort (8-bit digits, as many passes
//     as V needs), so equal ids keep ascending token order.  An id outside
//     [0, V) is replaced by V, which sorts after every valid id and is never
//     written (the token's one-hot row is zero).  Each pass: per-tile digit
//     histograms (1024 keys per tile), one exclusive scan over (digit, tile),
//     then each tile ranks its keys within their digit stably and scatters
//     them.  The rank comes from wave ballots: eight ballots of the digit's
//     bits give each lane the mask of the lanes with the same digit, whose
//     lower lanes it counts; the counts of the earlier (round, wave) groups
//     of the tile come from a small LDS table;
//  2. without accumulation every row of G is zeroed (a streaming fill);
//  3. the sorted positions are cut into chunks of kChunk; one workgroup per
//     (chunk, 256 columns) walks its chunk in order, each thread summing its
//     column of C_i g_it run by run.  A run that lies inside the chunk is
//     written to its row; the first run of a chunk that began in an earlier
//     chunk and the last run that goes on into the next leave partial rows;
//  4. one workgroup per (chunk boundary crossed by a run that starts before
//     it, 256 columns) adds that run's partials in chunk order and writes the
//     row.  Every present row is written exactly once, from sums taken in
//     ascending token order, and the work per workgroup is bounded by the
//     chunk length whatever the id frequencies.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kTile = kEmbedTileKeys;   // keys per radix tile
constexpr int kTileThreads = 256;
constexpr int kPer = kTile / kTileThreads;   // rounds of one key per thread
constexpr int kChunk = kEmbedChunk;     // sorted positions per reduction chunk
constexpr int kCols = 256;          // columns per reduction workgroup

size_t ws_align(size_t x) { return embed_ws_align(x); }
int64_t tiles_of(int64_t n) { return embed_tiles_of(n); }
int64_t chunks_of(int64_t n) { return embed_chunks_of(n); }

// Workspace for n tokens and rows of p columns: two key buffers [n] uint64,
// the digit histograms [256 x tiles] int32, the partial rows of the chunks
// (first and last run, [chunks x 2 x p] float32) and each chunk's flag
// (its first run goes on into the next chunk) [chunks] int32.
struct EmbedWs {
    uint64_t* keys[2];
    int32_t* hist;
    float* part;
    int32_t* through;
};
EmbedWs carve(void* ws, int64_t n, int64_t p) {
    char* w = static_cast<char*>(ws);
    EmbedWs e;
    for (int b = 0; b < 2; ++b) {
        e.keys[b] = reinterpret_cast<uint64_t*>(w);
        w += ws_align((size_t)n * sizeof(uint64_t));
    }
    e.hist = reinterpret_cast<int32_t*>(w);
    w += ws_align((size_t)(256 * tiles_of(n)) * sizeof(int32_t));
    e.part = reinterpret_cast<float*>(w);
    w += ws_align((size_t)(2 * chunks_of(n) * p) * sizeof(float));
    e.through = reinterpret_cast<int32_t*>(w);
    return e;
}

// Key of token s: (id if 0 <= id < V, else V) << 32 | s.
__device__ __forceinline__ uint64_t make_key(const int64_t* ids, int s, int64_t V) {
    const int64_t id = ids[s];
    const uint64_t v = (id >= 0 && id < V) ? (uint64_t)id : (uint64_t)V;
    return (v << 32) | (uint32_t)s;
}

__device__ __forceinline__ uint64_t tile_key(const int64_t* ids, const uint64_t* in, int s, int64_t V) {
    return in ? in[s] : make_key(ids, s, V);
}

// Digit histogram of one tile: hist[d * tiles + tile] = keys of the tile
// whose digit (bits shift .. shift + 7 of the id) is d.  Integer counts (the
// order of the LDS atomics does not matter).
__global__ __launch_bounds__(kTileThreads) void radix_hist_kernel(const int64_t* __restrict__ ids,
                                                                  const uint64_t* __restrict__ in,
                                                                  int n, int64_t V, int shift,
                                                                  int32_t* __restrict__ hist) {
    __shared__ int cnt[256];
    const int tile = blockIdx.x, tiles = gridDim.x;
    cnt[threadIdx.x] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int s = tile * kTile + e * kTileThreads + (int)threadIdx.x;
        if (s < n) atomicAdd(&cnt[(int)((tile_key(ids, in, s, V) >> (32 + shift)) & 255u)], 1);
    }
    __syncthreads();
    hist[threadIdx.x * tiles + tile] = cnt[threadIdx.x];
}

// In-place exclusive prefix sum of len int32 values (one workgroup): thread
// t owns a contiguous segment, the segment totals are scanned across the
// workgroup, then each segment is rewritten.
__global__ __launch_bounds__(1024) void scan_kernel(int32_t* __restrict__ a, int64_t len) {
    __shared__ int32_t tot[1024];
    const int t = threadIdx.x;
    const int64_t per = (len + 1023) / 1024, b0 = t * per, b1 = min(len, b0 + per);
    int32_t s = 0;
    for (int64_t i = b0; i < b1; ++i) s += a[i];
    tot[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {       // Hillis-Steele inclusive scan
        const int32_t y = t >= off ? tot[t - off] : 0;
        __syncthreads();
        tot[t] += y;
        __syncthreads();
    }
    int32_t run = t > 0 ? tot[t - 1] : 0;
    for (int64_t i = b0; i < b1; ++i) {
        const int32_t x = a[i];
        a[i] = run;
        run += x;
    }
}

// Stable scatter of one tile.  Key e * 256 + t of the tile (round e, thread
// t) goes to hist[digit * tiles + tile] (the scanned offset) plus the number
// of keys of the tile before it with the same digit: those of earlier
// (round, wave) groups (an LDS table of per-group digit counts, prefixed in
// group order) and those of lower lanes of its own wave in its round (the
// ballot mask of equal digits).
__global__ __launch_bounds__(kTileThreads) void radix_scatter_kernel(const int64_t* __restrict__ ids,
                                                                     const uint64_t* __restrict__ in,
                                                                     int n, int64_t V, int shift,
                                                                     const int32_t* __restrict__ hist,
                                                                     uint64_t* __restrict__ out) {
    constexpr int kWaves = kTileThreads / 64, kGroups = kPer * kWaves;
    __shared__ int cnt[kGroups][256];          // keys of digit d in group (round, wave), then prefixed
    const int tile = blockIdx.x, tiles = gridDim.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
    for (int i = t; i < kGroups * 256; i += kTileThreads) (&cnt[0][0])[i] = 0;
    __syncthreads();
    uint64_t key[kPer];
    int dig[kPer], rank[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int s = tile * kTile + e * kTileThreads + t;
        const bool ok = s < n;
        key[e] = ok ? tile_key(ids, in, s, V) : 0;
        const int d = ok ? (int)((key[e] >> (32 + shift)) & 255u) : 256;
        dig[e] = d;
        uint64_t same = __ballot(ok);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t bit = __ballot((d >> b) & 1);
            same &= ((d >> b) & 1) ? bit : ~bit;
        }
        rank[e] = __popcll(same & ((1ull << lane) - 1ull));
        if (ok && rank[e] == 0) cnt[e * kWaves + wave][d] = __popcll(same);
    }
    __syncthreads();
    {   // exclusive prefix of every digit's counts over the groups, in order
        const int d = t;
        int run = 0;
        for (int grp = 0; grp < kGroups; ++grp) {
            const int c = cnt[grp][d];
            cnt[grp][d] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int d = dig[e];
        if (d < 256) out[hist[d * tiles + tile] + cnt[e * kWaves + wave][d] + rank[e]] = key[e];
    }
}

__global__ __launch_bounds__(256) void zero_rows_kernel(float* __restrict__ G, int64_t total, int vec) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    if (vec) {
        float4* G4 = reinterpret_cast<float4*>(G);
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total / 4; i += stride)
            G4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += stride) G[i] = 0.f;
    }
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p);
template <> __device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_elem<bf16_t>(const bf16_t* p) {
    return bf16_to_f32(p->bits);
}

__device__ __forceinline__ int64_t key_id(uint64_t k) { return (int64_t)(k >> 32); }

__device__ __forceinline__ void store_row(float* q, float x, int accum) { *q = accum ? *q + x : x; }

// Chunk c of the sorted positions, columns [256 cb, 256 cb + 256): grid =
// chunks x column blocks, chunk-major.
template <typename T>
__global__ __launch_bounds__(kCols) void embed_chunk_kernel(const uint64_t* __restrict__ keys, int n,
                                                            int64_t V, const T* __restrict__ g,
                                                            const float* __restrict__ C, int T_, int p,
                                                            int ncb, float* __restrict__ G,
                                                            float* __restrict__ part,
                                                            int32_t* __restrict__ through, int accum) {
    __shared__ int64_t sid[kChunk + 1];
    __shared__ uint32_t stok[kChunk];
    __shared__ float sw[kChunk];
    __shared__ int prev_cont;
    const int c = blockIdx.x / ncb, cb = blockIdx.x - c * ncb;
    const int s0 = c * kChunk, len = min(kChunk, n - s0), t = threadIdx.x;
    // Positions past the chunk's end repeat its last token with weight 0 and
    // id V, so that every load below is of a real element and needs no branch.
    if (t < kChunk) {
        const uint64_t k = keys[s0 + min(t, len - 1)];
        const bool in = t < len;
        sid[t] = in ? key_id(k) : V;
        stok[t] = (uint32_t)k;
        sw[t] = in ? C[(uint32_t)k / (uint32_t)T_] : 0.f;
    }
    if (t == 0) sid[kChunk] = s0 + len < n ? key_id(keys[s0 + len]) : V;   // the next chunk's first id
    if (t == 1) prev_cont = s0 > 0 && key_id(keys[s0 - 1]) == key_id(keys[s0]) && key_id(keys[s0]) < V;
    __syncthreads();
    const int col = cb * kCols + t;
    const bool live = col < p;
    const T* gc = g + min(col, p - 1);
    // every term of this column first, from unconditional loads (all in
    // flight at once), then the runs
    float x[kChunk];
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
        const float w = (live && sid[i] < V) ? sw[i] : 0.f;
        x[i] = w * load_elem<T>(gc + (int64_t)stok[i] * p);
    }
    float acc = 0.f;
    bool first = true;
    // (the conditions below are the same for every thread; the invalid ids
    // sort last and end the walk)
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
        const int64_t v = i < len ? sid[i] : V;
        if (v < V) {
            acc += x[i];
            if (i + 1 == len || sid[i + 1] != v) {                // the run ends here
                const bool head = first && prev_cont;             // began in an earlier chunk
                const bool tail = i + 1 == len && sid[kChunk] == v;   // goes on into the next chunk
                if (head) {
                    if (live) part[((int64_t)c * 2) * p + col] = acc;
                    if (cb == 0 && t == 0) through[c] = tail ? 1 : 0;
                } else if (tail) {
                    if (live) part[((int64_t)c * 2 + 1) * p + col] = acc;
                } else if (live) {
                    store_row(G + v * (int64_t)p + col, acc, accum);
                }
                acc = 0.f;
                first = false;
            }
        }
    }
}

// Runs crossing chunk boundary c (between chunks c - 1 and c) that start
// before it in chunk c - 1: their partials added in chunk order.  grid =
// (chunks - 1) x column blocks; boundary c = 1 + blockIdx.x / ncb.
__global__ __launch_bounds__(kCols) void embed_fixup_kernel(const uint64_t* __restrict__ keys, int n,
                                                            int64_t V, int p, int ncb, int nchunks,
                                                            float* __restrict__ G,
                                                            const float* __restrict__ part,
                                                            const int32_t* __restrict__ through, int accum) {
    const int c = 1 + blockIdx.x / ncb, cb = blockIdx.x % ncb;
    const int s = c * kChunk;
    const int64_t v = key_id(keys[s]);
    if (v >= V || key_id(keys[s - 1]) != v) return;                 // no valid run crosses
    if (c >= 2 && key_id(keys[s - kChunk - 1]) == v) return;        // it also crosses c - 1
    const int col = cb * kCols + threadIdx.x;
    if (col >= p) return;
    float acc = part[((int64_t)(c - 1) * 2 + 1) * p + col];
    for (int k = c; k < nchunks; ++k) {
        acc += part[((int64_t)k * 2) * p + col];
        if (!through[k]) break;
    }
    store_row(G + v * (int64_t)p + col, acc, accum);
}

}  // namespace

hipError_t launch_embed_grad(const int64_t* ids, const void* g, const float* C, bool bf16,
                             int64_t B, int64_t T, int64_t p, int64_t V, float* G, void* ws, bool accum,
                             hipStream_t s) {
    const int64_t n = B * T;
    if (n > kEmbedMaxTokens || V <= 0 || p <= 0 || V >= ((int64_t)1 << 31))
        return (n > kEmbedMaxTokens || V >= ((int64_t)1 << 31)) ? hipErrorInvalidValue : hipSuccess;
    hipError_t e;
    if (!accum) {
        const int64_t total = V * p;
        const int vec = (reinterpret_cast<uintptr_t>(G) & 15u) == 0 && total % 4 == 0;
        const int64_t items = vec ? total / 4 : total;
        const unsigned nwg = (unsigned)std::min<int64_t>(4096, (items + 255) / 256);
        hipLaunchKernelGGL(zero_rows_kernel, dim3(nwg), dim3(256), 0, s, G, total, vec);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (n == 0) return hipSuccess;
    const EmbedWs w = carve(ws, n, p);
    const int tiles = (int)tiles_of(n);
    // digits of the largest key id (V: the invalid ids)
    int passes = 0;
    for (uint64_t x = (uint64_t)V; x; x >>= 8) ++passes;
    const uint64_t* in = nullptr;      // pass 0 builds its keys from the ids
    for (int ps = 0; ps < passes; ++ps) {
        uint64_t* out = w.keys[ps & 1];
        hipLaunchKernelGGL(radix_hist_kernel, dim3(tiles), dim3(kTileThreads), 0, s, ids, in, (int)n, V, 8 * ps,
                           w.hist);
        hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, s, w.hist, (int64_t)256 * tiles);
        hipLaunchKernelGGL(radix_scatter_kernel, dim3(tiles), dim3(kTileThreads), 0, s, ids, in, (int)n, V,
                           8 * ps, w.hist, out);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        in = out;
    }
    const int nchunks = (int)chunks_of(n), ncb = (int)((p + kCols - 1) / kCols);
    const int64_t nwg = (int64_t)nchunks * ncb;
    if (nwg > INT32_MAX) return hipErrorInvalidValue;
    if (bf16)
        hipLaunchKernelGGL(embed_chunk_kernel<bf16_t>, dim3((unsigned)nwg), dim3(kCols), 0, s, in, (int)n, V,
                           reinterpret_cast<const bf16_t*>(g), C, (int)T, (int)p, ncb, G, w.part, w.through,
                           accum ? 1 : 0);
    else
        hipLaunchKernelGGL(embed_chunk_kernel<float>, dim3((unsigned)nwg), dim3(kCols), 0, s, in, (int)n, V,
                           reinterpret_cast<const float*>(g), C, (int)T, (int)p, ncb, G, w.part, w.through,
                           accum ? 1 : 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (nchunks > 1)
        hipLaunchKernelGGL(embed_fixup_kernel, dim3((unsigned)((int64_t)(nchunks - 1) * ncb)), dim3(kCols), 0, s, in,
                           (int)n, V, (int)p, ncb, nchunks, G, w.part, w.through, accum ? 1 : 0);
    return hipGetLastError();
}

}  // namespace bk
