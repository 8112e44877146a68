// Per-sample gradients of the parameters that book-keeping does not cover
// (Section 5: it applies to the weights of generalized linear layers), which
// are instantiated per sample as the appendix notes on supported layers do
// for normalization layers:
//
//   bias b of s = a W + b          : s_i = sum_t g_it                  [p]
//   beta of y = gamma * xhat + beta : s_i = sum_t g_it                  [p]
//   gamma                           : u_i = sum_t g_it * xhat_it        [p]
//
// One workgroup per (layer, sample, chunk of kAffineCols features).  Thread
// (r, c) of 8 x 32 adds rows t = r, r + 8, ... of its 8 features (one 16-byte
// load per row and operand for bf16 rows); the 8 row groups are then added in
// order through LDS, so every sum has a fixed order (deterministic).  The
// workgroup writes its sums to P / Pb and one partial of the squared norm,
// sum_c u^2 + s^2, which the fixed-order reduction adds to the layer's norm.
// HBM-bound: T p (1 or 2) elements read per sample, 4 p (1 or 2) bytes written.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

template <typename E>
__device__ __forceinline__ void load8(const E* row, int c, int p, bool vec, float v[8]) {
    if constexpr (sizeof(E) == 2) {
        const uint16_t* q = reinterpret_cast<const uint16_t*>(row) + c;
        if (vec && c + 8 <= p) {
            const uint4 w = *reinterpret_cast<const uint4*>(q);
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                v[2 * j] = bf16_to_f32(ws[j] & 0xFFFFu);
                v[2 * j + 1] = bf16_to_f32(ws[j] >> 16);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = (c + j < p) ? bf16_to_f32(q[j]) : 0.f;
        }
    } else {
        const float* q = reinterpret_cast<const float*>(row) + c;
        if (vec && c + 8 <= p) {
            const float4 a = *reinterpret_cast<const float4*>(q);
            const float4 b = *reinterpret_cast<const float4*>(q + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = (c + j < p) ? q[j] : 0.f;
        }
    }
}

template <typename E>
__global__ __launch_bounds__(256) void affine_sums_kernel(const AffineArgs args) {
    __shared__ float rs[8][kAffineCols];
    __shared__ float ru[8][kAffineCols];
    __shared__ float red[4];
    const uint32_t wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const AffineLayer& L = args.L[l];
    const int local = (int)wg - L.wg_begin;
    const int i = local / L.chunks, k = local - i * L.chunks;
    const int p = L.p, T = L.T;
    const int c0 = k * kAffineCols;
    const int tid = threadIdx.x, r = tid >> 5, cl = (tid & 31) * 8;
    const bool gam = L.gamma != 0;
    const bool vec = L.vec != 0;
    const E* g = static_cast<const E*>(L.g) + (size_t)i * T * p;
    const E* x = gam && T > 0 ? static_cast<const E*>(L.x) + (size_t)i * T * p : nullptr;

    float s[8], u[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) s[j] = u[j] = 0.f;
    if (c0 + cl < p) {
#pragma unroll 4
        for (int t = r; t < T; t += 8) {
            float gv[8];
            load8<E>(g + (size_t)t * p, c0 + cl, p, vec, gv);
#pragma unroll
            for (int j = 0; j < 8; ++j) s[j] += gv[j];
            if (gam) {
                float xv[8];
                load8<E>(x + (size_t)t * p, c0 + cl, p, vec, xv);
#pragma unroll
                for (int j = 0; j < 8; ++j) u[j] = fmaf(gv[j], xv[j], u[j]);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        rs[r][cl + j] = s[j];
        ru[r][cl + j] = u[j];
    }
    __syncthreads();
    // thread tid owns feature c0 + tid: row groups added in order
    const int c = c0 + tid;
    float st = 0.f, ut = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        st += rs[q][tid];
        ut += ru[q][tid];
    }
    float sq = 0.f;
    if (c < p) {
        if (gam) {
            L.P[(size_t)i * p + c] = ut;
            sq += ut * ut;
        }
        if (L.Pb) {
            L.Pb[(size_t)i * p + c] = st;
            sq += st * st;
        }
    }
    const float tot = block_sum_256(sq, red);
    if (tid == 0) args.part[(size_t)L.part_off + (size_t)i * L.chunks + k] = tot;
}

}  // namespace

hipError_t launch_affine(const AffineArgs& args, int n_wg, bool bf16, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    if (bf16) hipLaunchKernelGGL(affine_sums_kernel<uint16_t>, dim3(n_wg), dim3(256), 0, s, args);
    else hipLaunchKernelGGL(affine_sums_kernel<float>, dim3(n_wg), dim3(256), 0, s, args);
    return hipGetLastError();
}

}  // namespace bk
