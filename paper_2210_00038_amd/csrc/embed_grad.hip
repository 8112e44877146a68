// Sum of clipped gradients of an embedding layer (Algorithm 1 applied to a
// layer whose input is the one-hot encoding of token ids):
//
//   G[v, :] = sum_i C_i sum_{t : x_it = v} g_it        for every v in [0, V).
//
// Deterministic grouping, no floating-point atomics:
//  1. one workgroup sorts the n = B*T keys (id << 32 | flat token index) in
//     LDS (bitonic network) and compacts the runs of equal valid ids: run j
//     has id run_id[j] and tokens keys[run_start[j] .. run_start[j + 1]),
//     in ascending token order; the run count goes to run_start[n + 1];
//  2. without accumulation every row of G is zeroed (a streaming fill);
//  3. one workgroup per (run, 256 columns) stages its run's token rows and
//     clip weights in LDS, 256 at a time, and each thread adds its column's
//     terms in ascending token order, with the g loads of 8 tokens in flight,
//     then writes (or adds to) the row.  A long run (a frequent token) thus
//     costs one workgroup per column chunk, not one pass per token.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kSortThreads = 1024;
constexpr int kSortMax = 8192;      // keys sorted in one workgroup (64 KiB of LDS)
constexpr int kPerThread = kSortMax / kSortThreads;

// Workspace layout for n tokens: keys [n] uint64, run_id [n] int32,
// run_start [n + 2] int32 (starts, the end of the last run, the run count).
struct EmbedWs {
    uint64_t* keys;
    int32_t* run_id;
    int32_t* run_start;
};
size_t ws_align(size_t x) { return (x + 255) / 256 * 256; }
EmbedWs carve(void* ws, int64_t n) {
    char* w = static_cast<char*>(ws);
    EmbedWs e;
    e.keys = reinterpret_cast<uint64_t*>(w);
    w += ws_align((size_t)n * sizeof(uint64_t));
    e.run_id = reinterpret_cast<int32_t*>(w);
    w += ws_align((size_t)n * sizeof(int32_t));
    e.run_start = reinterpret_cast<int32_t*>(w);
    return e;
}

__global__ __launch_bounds__(kSortThreads) void embed_sort_kernel(const int64_t* __restrict__ ids,
                                                                  int n, int P, int64_t V,
                                                                  uint64_t* __restrict__ keys_out,
                                                                  int32_t* __restrict__ run_id,
                                                                  int32_t* __restrict__ run_start) {
    __shared__ uint64_t key[kSortMax];
    __shared__ int wsum[kSortThreads / 64];
    __shared__ int nvalid;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int s = tid; s < P; s += kSortThreads)
        key[s] = (s < n) ? (((uint64_t)ids[s] << 32) | (uint32_t)s) : ~0ull;
    if (tid == 0) nvalid = n;
    __syncthreads();
    // Bitonic sort, ascending.  Ids outside [0, V) (negative ones included,
    // as unsigned) sort after every valid id.
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int s = tid; s < P; s += kSortThreads) {
                const int o = s ^ j;
                if (o > s) {
                    const uint64_t a = key[s], b = key[o];
                    const bool up = (s & k) == 0;
                    if ((a > b) == up) { key[s] = b; key[o] = a; }
                }
            }
            __syncthreads();
        }
    }
    // Thread t owns sorted positions [kPerThread t, kPerThread (t + 1)): it
    // counts the run starts among them (valid ids only) and finds the first
    // invalid position, the end of the last run.
    auto id_at = [&](int s) { return key[s] >> 32; };
    auto starts = [&](int s) {
        return s < n && id_at(s) < (uint64_t)V && (s == 0 || id_at(s - 1) != id_at(s));
    };
    const int b0 = tid * kPerThread;
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const int s = b0 + e;
        cnt += starts(s) ? 1 : 0;
        if (s < n && id_at(s) >= (uint64_t)V && (s == 0 || id_at(s - 1) < (uint64_t)V)) nvalid = s;
    }
    // Exclusive scan of the counts over the workgroup (wave scans, then the
    // wave totals).
    int x = cnt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    if (wave == 0) {
        int y = lane < kSortThreads / 64 ? wsum[lane] : 0;
#pragma unroll
        for (int off = 1; off < kSortThreads / 64; off <<= 1) {
            const int z = __shfl_up(y, off, 64);
            if (lane >= off) y += z;
        }
        if (lane < kSortThreads / 64) wsum[lane] = y;
    }
    __syncthreads();
    int r = x - cnt + (wave > 0 ? wsum[wave - 1] : 0);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const int s = b0 + e;
        if (starts(s)) {
            run_id[r] = (int32_t)id_at(s);
            run_start[r] = s;
            ++r;
        }
    }
    for (int s = tid; s < n; s += kSortThreads) keys_out[s] = key[s];
    if (tid == 0) {
        const int D = wsum[kSortThreads / 64 - 1];
        run_start[D] = nvalid;          // end of the last run
        run_start[n + 1] = D;           // run count
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

template <typename T>
__global__ __launch_bounds__(256) void embed_rows_kernel(const uint64_t* __restrict__ keys,
                                                         const int32_t* __restrict__ run_id,
                                                         const int32_t* __restrict__ run_start, int n,
                                                         const T* __restrict__ g,
                                                         const float* __restrict__ C, int T_, int p,
                                                         float* __restrict__ G, int accum) {
    __shared__ uint32_t rr[256];
    __shared__ float ww[256];
    const int j = blockIdx.y;
    if (j >= run_start[n + 1]) return;              // fewer runs than tokens
    const int64_t v = run_id[j];
    const int s0 = run_start[j], s1 = run_start[j + 1];
    const int c = blockIdx.x * 256 + threadIdx.x;
    const T* gc = g + c;
    float acc = 0.f;
    for (int base = s0; base < s1; base += 256) {
        const int cnt = min(256, s1 - base);
        __syncthreads();                            // the previous batch is consumed
        if ((int)threadIdx.x < cnt) {
            const uint32_t r = (uint32_t)keys[base + threadIdx.x];
            rr[threadIdx.x] = r;
            ww[threadIdx.x] = C[r / (uint32_t)T_];
        }
        __syncthreads();
        if (c < p) {
            int t = 0;
            for (; t + 8 <= cnt; t += 8) {
                float x[8];
#pragma unroll
                for (int b = 0; b < 8; ++b) x[b] = load_elem<T>(gc + (int64_t)rr[t + b] * p);
#pragma unroll
                for (int b = 0; b < 8; ++b) acc += ww[t + b] * x[b];
            }
            for (; t < cnt; ++t) acc += ww[t] * load_elem<T>(gc + (int64_t)rr[t] * p);
        }
    }
    if (c < p) {
        float* q = G + v * (int64_t)p + c;
        *q = accum ? *q + acc : acc;
    }
}

}  // namespace

size_t embed_grad_ws_bytes(int64_t n) {
    return ws_align((size_t)n * sizeof(uint64_t)) + ws_align((size_t)n * sizeof(int32_t)) +
           ws_align((size_t)(n + 2) * sizeof(int32_t));
}

hipError_t launch_embed_grad(const int64_t* ids, const void* g, const float* C, bool bf16,
                             int64_t B, int64_t T, int64_t p, int64_t V, float* G, void* ws, bool accum,
                             hipStream_t s) {
    const int n = (int)(B * T);
    if (n > kSortMax || V <= 0 || p <= 0) return n > kSortMax ? hipErrorInvalidValue : hipSuccess;
    if ((p + 255) / 256 > INT32_MAX) return hipErrorInvalidValue;
    int P = 1;
    while (P < n) P <<= 1;
    const EmbedWs w = carve(ws, n);
    hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(kSortThreads), 0, s, ids, n, P, V, w.keys,
                       w.run_id, w.run_start);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (!accum) {
        const int64_t total = V * p;
        const int vec = (reinterpret_cast<uintptr_t>(G) & 15u) == 0 && total % 4 == 0;
        const int64_t items = vec ? total / 4 : total;
        const unsigned nwg = (unsigned)std::min<int64_t>(4096, (items + 255) / 256);
        hipLaunchKernelGGL(zero_rows_kernel, dim3(nwg), dim3(256), 0, s, G, total, vec);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((p + 255) / 256), (unsigned)n);
    if (bf16)
        hipLaunchKernelGGL(embed_rows_kernel<bf16_t>, grid, dim3(256), 0, s, w.keys, w.run_id, w.run_start,
                           n, reinterpret_cast<const bf16_t*>(g), C, (int)(T > 0 ? T : 1), (int)p, G,
                           accum ? 1 : 0);
    else
        hipLaunchKernelGGL(embed_rows_kernel<float>, grid, dim3(256), 0, s, w.keys, w.run_id, w.run_start,
                           n, reinterpret_cast<const float*>(g), C, (int)(T > 0 ? T : 1), (int)p, G,
                           accum ? 1 : 0);
    return hipGetLastError();
}

}  // namespace bk
