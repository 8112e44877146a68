// Ghost norm of an embedding layer as a join on token ids (eq. "ghost norm",
// Section 2.1, with a_i = one_hot(x_i); App. D.1):
//
//   n_i = sum_{t,t'} [x_it == x_it'] <g_it, g_it'> = sum_v || sum_{t : x_it = v} g_it ||^2
//
// Instead of the T x T Gram of g masked by id equality (2 T^2 p MFMA work,
// ghost_norm.hip), the tokens of a sample are grouped by id and each group's
// rows of g are summed once: T p additions, every row of g read once.  The
// masked Gram remains for rows of g that are not 16-byte multiples and for T
// past the keys the LDS holds.
//
// One 1024-thread workgroup owns (layer, sample, chunk of 8 CT columns of g):
//  1. the sample's keys (id << 32 | t) are sorted in LDS (bitonic); ids
//     outside [0, V) get the key id 0x7FFFFFFF and sort after the valid ones
//     (they select no row of the embedding and add nothing);
//  2. the valid positions are cut into NSEG = 1024 / CT equal segments of
//     consecutive sorted positions; CT threads per segment each own 8 columns
//     and walk the segment in order, summing g rows in fp32 into the open run
//     (a run: the positions of one id) and adding the squared sum of every
//     run that starts and ends inside the segment;
//  3. CT threads then walk the segments in order with the run left open
//     across segment boundaries (head part of a segment + tail of the
//     previous ones), adding its square when it closes;
//  4. a fixed-order block sum gives the chunk's partial; the host's
//     reduction adds the chunks of a sample in order.
// Every step has a fixed order: the result is bitwise reproducible.
#include <atomic>

#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kJoinThreads = kEmbedJoinThreads;
constexpr uint32_t kJoinBadId = 0x7FFFFFFFu;          // key id of ids outside [0, V)

// 8 consecutive elements of a row of g (16-byte aligned): loaded raw (Raw),
// added to 8 floats (add).
template <typename E> struct JoinRow;
template <> struct JoinRow<bf16_t> {
    using Raw = uint4;
    static __device__ __forceinline__ Raw load(const void* p) { return *reinterpret_cast<const uint4*>(p); }
    static __device__ __forceinline__ Raw zero() { return make_uint4(0u, 0u, 0u, 0u); }
    static __device__ __forceinline__ void add(float* acc, const Raw& u) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            acc[2 * k] += __uint_as_float(w[k] << 16);
            acc[2 * k + 1] += __uint_as_float(w[k] & 0xFFFF0000u);
        }
    }
};
template <> struct JoinRow<float> {
    struct Raw { float4 a, b; };
    static __device__ __forceinline__ Raw load(const void* p) {
        return Raw{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
    }
    static __device__ __forceinline__ Raw zero() { return Raw{make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)}; }
    static __device__ __forceinline__ void add(float* acc, const Raw& r) {
        acc[0] += r.a.x; acc[1] += r.a.y; acc[2] += r.a.z; acc[3] += r.a.w;
        acc[4] += r.b.x; acc[5] += r.b.y; acc[6] += r.b.z; acc[7] += r.b.w;
    }
};

__device__ __forceinline__ float sq8(const float* v) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) s += v[k] * v[k];
    return s;
}

// Dynamic LDS: keys [tp] (uint64) or, after the walk, the head and tail
// sums [2][NSEG][8 CT] (floats); then the segments' "has a run start" flags.
template <typename E, int CT>
__global__ __launch_bounds__(kJoinThreads) void embed_join_kernel(const GhostArgs args, int region) {
    constexpr int NSEG = kJoinThreads / CT, NC = 8 * CT;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem);
    float* head = reinterpret_cast<float*>(smem);
    float* tail = head + NSEG * NC;
    int* starts = reinterpret_cast<int*>(smem + region);
    __shared__ int nvalid;
    __shared__ float red[kJoinThreads / 64];

    const int wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GhostLayer& L = args.L[l];
    const int local = wg - L.wg_begin, ncc = L.npairs;
    const int sample = local / ncc, cc = local - sample * ncc;
    const int T = L.T, p = L.p, tid = threadIdx.x;
    const int64_t V = L.d;
    const int64_t* ids = static_cast<const int64_t*>(L.x) + (size_t)sample * T;
    int tp = 1;
    while (tp < T) tp <<= 1;

    // 1. keys, sorted ascending (bitonic network over tp keys).
    if (tid == 0) nvalid = 0;
    int mine = 0;
    for (int i = tid; i < tp; i += kJoinThreads) {
        uint64_t k = ~0ull;
        if (i < T) {
            const int64_t id = ids[i];
            const uint32_t kid = (id >= 0 && id < V) ? (uint32_t)id : kJoinBadId;
            mine += kid != kJoinBadId;
            k = ((uint64_t)kid << 32) | (uint32_t)i;
        }
        keys[i] = k;
    }
    __syncthreads();
    atomicAdd(&nvalid, mine);   // an integer count: order-independent
    for (int k = 2; k <= tp; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < tp / 2; i += kJoinThreads) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)), hi = lo + j;
                const uint64_t a = keys[lo], b = keys[hi];
                if ((a > b) == ((lo & k) == 0)) {
                    keys[lo] = b;
                    keys[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    if (tp == 1) __syncthreads();
    const int nv = nvalid;

    // 2. segment `seg` = sorted positions [b, e); this thread's 8 columns.
    const int seg = tid / CT, ct = tid % CT;
    const int b = (int)((int64_t)seg * nv / NSEG), e = (int)((int64_t)(seg + 1) * nv / NSEG);
    const int c0 = cc * NC + ct * 8;
    const bool cols = c0 < p;        // the host guarantees p % 8 == 0
    const char* gs = static_cast<const char*>(L.g) + ((size_t)sample * T * p + (size_t)c0) * sizeof(E);
    const size_t rowb = (size_t)p * sizeof(E);
    auto id_at = [&](int j) { return (uint32_t)(keys[j] >> 32); };
    float acc[8], first[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = first[k] = 0.f;
    bool has_start = false;
    float sq = 0.f;
    using Row = JoinRow<E>;
    constexpr int U = sizeof(E) == 2 ? 16 : 8;       // rows in flight per thread
    for (int j0 = b; j0 < e; j0 += U) {
        typename Row::Raw v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int j = j0 + u;
            v[u] = (cols && j < e) ? Row::load(gs + (size_t)(uint32_t)keys[j] * rowb) : Row::zero();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int j = j0 + u;
            if (j < e && (j == 0 || id_at(j) != id_at(j - 1))) {   // a run starts at j
                if (has_start) sq += sq8(acc);                     // the previous one closed inside
                else {
#pragma unroll
                    for (int k = 0; k < 8; ++k) first[k] = acc[k];
                }
                has_start = true;
#pragma unroll
                for (int k = 0; k < 8; ++k) acc[k] = 0.f;
            }
            Row::add(acc, v[u]);     // zeros past the segment's end
        }
    }
    // head: the positions before the segment's first run start (all of them
    // if none); tail: the run open at its end.  They overwrite the keys once
    // every thread is done with them.
    if (!has_start) {
#pragma unroll
        for (int k = 0; k < 8; ++k) first[k] = acc[k], acc[k] = 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        head[seg * NC + ct * 8 + k] = first[k];
        tail[seg * NC + ct * 8 + k] = acc[k];
    }
    if (ct == 0) starts[seg] = has_start ? 1 : 0;
    __syncthreads();

    // 3. runs across segment boundaries, in segment order.
    if (tid < CT) {
        float carry[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) carry[k] = 0.f;
        for (int s = 0; s < NSEG; ++s) {
            const bool st = starts[s] != 0;
#pragma unroll
            for (int k = 0; k < 8; ++k) carry[k] += head[s * NC + tid * 8 + k];
            if (st) {
                sq += sq8(carry);
#pragma unroll
                for (int k = 0; k < 8; ++k) carry[k] = tail[s * NC + tid * 8 + k];
            }
        }
        sq += sq8(carry);
    }

    // 4. the chunk's partial (wave sums, then the waves in order).
    sq = wave_sum(sq);
    if ((tid & 63) == 0) red[tid >> 6] = sq;
    __syncthreads();
    if (tid == 0) {
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < kJoinThreads / 64; ++w) tot += red[w];
        args.part[(size_t)L.part_off + (size_t)sample * ncc + cc] = tot;
    }
}

}  // namespace

hipError_t launch_embed_join(const GhostArgs& args, int n_wg, bool bf16, int ct, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    int64_t tmax = 1;
    for (int k = 0; k < args.n; ++k) tmax = std::max<int64_t>(tmax, args.L[k].T);
    if (tmax > kEmbedJoinMaxT || (ct != 8 && ct != 32)) return hipErrorInvalidValue;
    const size_t region = embed_join_region(tmax), lds = embed_join_lds_bytes(tmax);
    const void* fn = bf16 ? (ct == 8 ? reinterpret_cast<const void*>(&embed_join_kernel<bf16_t, 8>)
                                     : reinterpret_cast<const void*>(&embed_join_kernel<bf16_t, 32>))
                          : (ct == 8 ? reinterpret_cast<const void*>(&embed_join_kernel<float, 8>)
                                     : reinterpret_cast<const void*>(&embed_join_kernel<float, 32>));
    // Dynamic LDS past 64 KB is allowed per kernel and device once (the
    // largest size granted so far on the current device is remembered, so a
    // later call, under stream capture for instance, sets nothing).
    constexpr int kMaxDev = 64;
    static std::atomic<size_t> granted[kMaxDev][4];
    if (lds > 65536) {
        int dev = -1;
        const bool known = hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < kMaxDev;
        std::atomic<size_t>* gr = known ? &granted[dev][(bf16 ? 2 : 0) + (ct == 8 ? 0 : 1)] : nullptr;
        if (!gr || lds > gr->load(std::memory_order_relaxed)) {
            const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
            if (gr) gr->store(lds, std::memory_order_relaxed);
        }
    }
    const dim3 grid(n_wg), block(kJoinThreads);
    if (bf16) {
        if (ct == 8) hipLaunchKernelGGL((embed_join_kernel<bf16_t, 8>), grid, block, lds, s, args, (int)region);
        else hipLaunchKernelGGL((embed_join_kernel<bf16_t, 32>), grid, block, lds, s, args, (int)region);
    } else {
        if (ct == 8) hipLaunchKernelGGL((embed_join_kernel<float, 8>), grid, block, lds, s, args, (int)region);
        else hipLaunchKernelGGL((embed_join_kernel<float, 32>), grid, block, lds, s, args, (int)region);
    }
    return hipGetLastError();
}

}  // namespace bk
