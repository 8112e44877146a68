// Small kernels of Algorithm 1: the fixed-order reduction that finishes the
// per-sample norms, the aggregation over layers with the clip factors, and the
// Gaussian noise (Philox4x32-10 + Box-Muller).
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

// norm_sq[l][i] = sum of the partials of (layer l, sample i), in index order.
__global__ __launch_bounds__(256) void reduce_kernel(const ReduceArgs args) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)args.n * args.B) return;
    const int l = (int)(idx / args.B), i = (int)(idx - (int64_t)l * args.B);
    const ReduceLayer& L = args.L[l];
    // Partials in ascending order (the weight run, then the bias / affine
    // run); sixteen loads are issued ahead of their adds.
    double s = 0.0;
    auto run = [&](const float* p, int np) {
        int k = 0;
        for (; k + 16 <= np; k += 16) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) v[u] = p[k + u];
#pragma unroll
            for (int u = 0; u < 16; ++u) s += (double)v[u];
        }
        for (; k < np; ++k) s += (double)p[k];
    };
    run(args.part + L.part_off + (int64_t)i * L.npart, L.npart);
    run(args.part + L.part_off2 + (int64_t)i * L.npart2, L.npart2);
    L.out[i] = (float)s;
}

// Algorithm 1, aggregation and clip factor (clip functions of eq. "DP optimizers").
__global__ __launch_bounds__(256) void clip_kernel(const float* __restrict__ norm_sq, int64_t L,
                                                   int64_t B, int mode, float R, float gamma,
                                                   float* __restrict__ C, float* __restrict__ total) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B) return;
    // Layers in ascending order; sixteen loads are issued ahead of their adds.
    double s = 0.0;
    int64_t l = 0;
    for (; l + 16 <= L; l += 16) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = norm_sq[(l + u) * B + i];
#pragma unroll
        for (int u = 0; u < 16; ++u) s += (double)v[u];
    }
    for (; l < L; ++l) s += (double)norm_sq[l * B + i];
    const double nrm = sqrt(s);
    double c;
    if (mode == 0) {                       // Abadi: min(R / ||g||, 1)
        c = (nrm <= (double)R) ? 1.0 : (double)R / nrm;
    } else {                               // automatic: 1 / (||g|| + gamma)
        const double den = nrm + (double)gamma;
        c = (den == 0.0) ? 0.0 : 1.0 / den;
    }
    C[i] = (float)c;
    if (total) total[i] = (float)s;
}

// G[e] += std * z_e.  Workgroup w handles counter blocks
// [w * bpw, (w + 1) * bpw) of its tensor (bpw = args.bpw, a multiple of 256).
__global__ __launch_bounds__(256) void noise_kernel(const NoiseArgs args) {
    const uint32_t wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const NoiseLayer& L = args.L[l];
    float* G = L.G;
    const int64_t n = L.n;
    const int64_t nq = (n + 3) / 4;
    const int64_t q_begin = (int64_t)(wg - L.wg_begin) * args.bpw;
    const bool vec = (reinterpret_cast<uintptr_t>(G) & 15u) == 0;
    // The thread's G blocks are loaded first and its normals drawn while the
    // loads are in flight; then each block gets its noise and is stored.
    constexpr int NI = kNoiseBlocksPerWG / 256;
    const int ni = (int)(args.bpw / 256);
    float4 v[NI], z[NI];
#pragma unroll
    for (int k = 0; k < NI; ++k) {
        const int64_t q = q_begin + k * 256 + threadIdx.x;
        if (k < ni && q < nq && vec && 4 * q + 3 < n) v[k] = *reinterpret_cast<const float4*>(G + 4 * q);
    }
#pragma unroll
    for (int k = 0; k < NI; ++k) {
        const int64_t q = q_begin + k * 256 + threadIdx.x;
        if (k < ni && q < nq) z[k] = normal4(args.seed, L.tensor_id, args.step, (uint64_t)q);
    }
#pragma unroll
    for (int k = 0; k < NI; ++k) {
        const int64_t q = q_begin + k * 256 + threadIdx.x;
        if (k >= ni || q >= nq) break;
        const int64_t e = 4 * q;
        if (vec && e + 3 < n) {
            float4 w = v[k];
            w.x += args.std * z[k].x;
            w.y += args.std * z[k].y;
            w.z += args.std * z[k].z;
            w.w += args.std * z[k].w;
            *reinterpret_cast<float4*>(G + e) = w;
        } else {
            const float zz[4] = {z[k].x, z[k].y, z[k].z, z[k].w};
            for (int j = 0; j < 4 && e + j < n; ++j) G[e + j] += args.std * zz[j];
        }
    }
}

// Raw Philox words of counter blocks q0 .. q0 + nq - 1 (a test hook).
__global__ __launch_bounds__(256) void philox_raw_kernel(uint64_t seed, uint32_t tid, uint32_t step,
                                                         uint64_t q0, int64_t nq, uint32_t* out) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= nq) return;
    const uint4 w = philox_block(seed, tid, step, q0 + (uint64_t)k);
    out[4 * k + 0] = w.x;
    out[4 * k + 1] = w.y;
    out[4 * k + 2] = w.z;
    out[4 * k + 3] = w.w;
}

}  // namespace

hipError_t launch_reduce(const ReduceArgs& args, int n_threads, hipStream_t s) {
    if (n_threads <= 0) return hipSuccess;
    hipLaunchKernelGGL(reduce_kernel, dim3((n_threads + 255) / 256), dim3(256), 0, s, args);
    return hipGetLastError();
}

hipError_t launch_clip(const float* norm_sq, int64_t L, int64_t B, int mode, float R, float gamma,
                       float* C, float* total_sq, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(clip_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, norm_sq, L,
                       B, mode, R, gamma, C, total_sq);
    return hipGetLastError();
}

hipError_t launch_noise(const NoiseArgs& args, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    hipLaunchKernelGGL(noise_kernel, dim3(n_wg), dim3(256), 0, s, args);
    return hipGetLastError();
}

hipError_t launch_philox_raw(uint64_t seed, uint32_t tid, uint32_t step, uint64_t q0, int64_t nq,
                             uint32_t* out, hipStream_t s) {
    if (nq <= 0) return hipSuccess;
    hipLaunchKernelGGL(philox_raw_kernel, dim3((unsigned)((nq + 255) / 256)), dim3(256), 0, s, seed,
                       tid, step, q0, nq, out);
    return hipGetLastError();
}

}  // namespace bk
