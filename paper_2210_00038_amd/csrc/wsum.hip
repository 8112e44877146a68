// Weighted sum of stored per-sample gradients (App. B.5), BK-MixOpt's
// clipped gradient on the layers that instantiate:
//   G[e] = sum_i C[i] P[i n + e],  i ascending, one float32 fused
// multiply-add per sample (deterministic); with accum the sum is added to G.
// One launch covers a group of layers; each thread owns 4 consecutive
// elements (16-byte loads when the layer's buffers allow) and streams the B
// per-sample values of them.  HBM-bound: (B + 1) * 4 bytes per element.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

__global__ __launch_bounds__(256) void wsum_kernel(const WsumArgs args) {
    const uint32_t wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const WsumLayer& L = args.L[l];
    const int64_t n = L.n;
    const int64_t e0 = (int64_t)(wg - L.wg_begin) * kWsumPerWG + 4 * (int64_t)threadIdx.x;
    if (e0 >= n) return;
    const int B = args.B;
    if (L.vec) {       // 4 | n: the thread's 4 elements are in range
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int i = 0; i < B; ++i) {
            const float c = args.C[i];
            const float4 v = *reinterpret_cast<const float4*>(L.P + (size_t)i * n + e0);
            acc.x = fmaf(c, v.x, acc.x);
            acc.y = fmaf(c, v.y, acc.y);
            acc.z = fmaf(c, v.z, acc.z);
            acc.w = fmaf(c, v.w, acc.w);
        }
        float4* q = reinterpret_cast<float4*>(L.G + e0);
        if (L.accum) {
            const float4 o = *q;
            acc.x += o.x;
            acc.y += o.y;
            acc.z += o.z;
            acc.w += o.w;
        }
        *q = acc;
    } else {
        const int m = (int)min<int64_t>(4, n - e0);
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int i = 0; i < B; ++i) {
            const float c = args.C[i];
            const float* row = L.P + (size_t)i * n + e0;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (j < m) acc[j] = fmaf(c, row[j], acc[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (j < m) L.G[e0 + j] = L.accum ? L.G[e0 + j] + acc[j] : acc[j];
    }
}

}  // namespace

hipError_t launch_wsum(const WsumArgs& args, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    hipLaunchKernelGGL(wsum_kernel, dim3(n_wg), dim3(256), 0, s, args);
    return hipGetLastError();
}

}  // namespace bk
