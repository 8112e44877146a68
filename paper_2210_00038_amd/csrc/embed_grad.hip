// Sum of clipped gradients of an embedding layer (Algorithm 1 applied to a
// layer whose input is the one-hot encoding of token ids):
//
//   G[v, :] = sum_i C_i sum_{t : x_it = v} g_it        for every v in [0, V).
//
// Deterministic grouping, no floating-point atomics:
//  1. one workgroup sorts the B*T keys (id << 32 | flat token index) in LDS
//     (bitonic network) and marks, for every id present, the first position
//     of its run in the sorted order (all other ids get -1);
//  2. one workgroup per vocabulary row v writes G[v, :]: zeros when v does
//     not occur, otherwise the sum over its run in ascending token order.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kSortThreads = 1024;
constexpr int kSortMax = 8192;      // keys sorted in one workgroup (64 KiB of LDS)

__global__ __launch_bounds__(kSortThreads) void embed_sort_kernel(const int64_t* __restrict__ ids,
                                                                  int n, int P, int64_t V,
                                                                  uint64_t* __restrict__ keys_out,
                                                                  int32_t* __restrict__ first) {
    __shared__ uint64_t key[kSortMax];
    const int tid = threadIdx.x;
    for (int64_t v = tid; v < V; v += kSortThreads) first[v] = -1;
    for (int s = tid; s < P; s += kSortThreads)
        key[s] = (s < n) ? (((uint64_t)ids[s] << 32) | (uint32_t)s) : ~0ull;
    __syncthreads();
    // Bitonic sort, ascending.
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
    for (int s = tid; s < n; s += kSortThreads) {
        const uint64_t cur = key[s];
        keys_out[s] = cur;
        const uint64_t id = cur >> 32;   // ids outside [0, V) are never marked
        if ((s == 0 || (key[s - 1] >> 32) != id) && id < (uint64_t)V) first[id] = s;
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
                                                         const int32_t* __restrict__ first, int n,
                                                         const T* __restrict__ g,
                                                         const float* __restrict__ C, int T_, int p,
                                                         float* __restrict__ G, int accum) {
    const int64_t v = blockIdx.x;
    float* row = G + v * (int64_t)p;
    const int s0 = first[v];
    if (s0 < 0) {                          // absent id: zero row (kept as it is when accumulating)
        if (!accum)
            for (int c = threadIdx.x; c < p; c += 256) row[c] = 0.f;
        return;
    }
    for (int c0 = 0; c0 < p; c0 += 256) {
        const int c = c0 + threadIdx.x;
        float acc = 0.f;
        for (int s = s0; s < n; ++s) {
            const uint64_t k = keys[s];
            if ((int64_t)(k >> 32) != v) break;
            const uint32_t r = (uint32_t)k;
            const float w = C[r / (uint32_t)T_];
            if (c < p) acc += w * load_elem<T>(g + (int64_t)r * p + c);
        }
        if (c < p) row[c] = accum ? row[c] + acc : acc;
    }
}

}  // namespace

hipError_t launch_embed_grad(const int64_t* ids, const void* g, const float* C, bool bf16,
                             int64_t B, int64_t T, int64_t p, int64_t V, float* G, uint64_t* keys,
                             int32_t* first, bool accum, hipStream_t s) {
    const int n = (int)(B * T);
    if (n > kSortMax) return hipErrorInvalidValue;
    int P = 1;
    while (P < n) P <<= 1;
    hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(kSortThreads), 0, s, ids, n, P, V, keys, first);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (V <= 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(embed_rows_kernel<bf16_t>, dim3((unsigned)V), dim3(256), 0, s, keys, first, n,
                           reinterpret_cast<const bf16_t*>(g), C, (int)(T > 0 ? T : 1), (int)p, G, accum ? 1 : 0);
    else
        hipLaunchKernelGGL(embed_rows_kernel<float>, dim3((unsigned)V), dim3(256), 0, s, keys, first, n,
                           reinterpret_cast<const float*>(g), C, (int)(T > 0 ? T : 1), (int)p, G, accum ? 1 : 0);
    return hipGetLastError();
}

}  // namespace bk
