// A 2-D convolution as a generalized linear layer (App. B: d = input
// channels x kernel height x kernel width, p = output channels, T = output
// height x width): the unfolded input a [B, T, ld] and the token-major output
// gradient g [B, T, p] that the BK kernels take.
//
// unfold: one thread per output element (b, t, column); consecutive threads
// write consecutive columns of a row, so the stores coalesce and the gathers
// from x hit the rows of one (c, i) run.  Columns d .. ld-1 are zero.
// tokens: [B, C, HW] -> [B, HW, C] transpose through a 32 x 33 LDS tile
// (coalesced reads and writes, no bank conflicts).
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

template <typename E>
__global__ __launch_bounds__(256) void unfold_kernel(const E* __restrict__ x, E* __restrict__ a,
                                                     UnfoldShape s) {
    const int64_t total = s.B * s.T * s.ld;
    const int64_t d = s.C * s.kh * s.kw;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        const int64_t col = e % s.ld, row = e / s.ld;
        const int64_t t = row % s.T, b = row / s.T;
        E v{};
        if (col < d) {
            const int64_t c = col / (s.kh * s.kw), r = col - c * (s.kh * s.kw);
            const int64_t i = r / s.kw, j = r - i * s.kw;
            const int64_t oh = t / s.Wo, ow = t - oh * s.Wo;
            const int64_t h = oh * s.stride + i - s.pad, w = ow * s.stride + j - s.pad;
            if (h >= 0 && h < s.H && w >= 0 && w < s.W) v = x[((b * s.C + c) * s.H + h) * s.W + w];
        }
        a[e] = v;
    }
}

template <typename E>
__global__ __launch_bounds__(256) void tokens_kernel(const E* __restrict__ y, E* __restrict__ out,
                                                     int64_t C, int64_t HW) {
    __shared__ E tile[32][33];
    const int64_t b = blockIdx.z;
    const int64_t c0 = (int64_t)blockIdx.y * 32, t0 = (int64_t)blockIdx.x * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;      // 32 x 8 threads
    const E* src = y + b * C * HW;
    E* dst = out + b * C * HW;
#pragma unroll
    for (int r = 0; r < 32; r += 8) {
        const int64_t c = c0 + ty + r, t = t0 + tx;
        if (c < C && t < HW) tile[ty + r][tx] = src[c * HW + t];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 32; r += 8) {
        const int64_t t = t0 + ty + r, c = c0 + tx;
        if (c < C && t < HW) dst[t * C + c] = tile[tx][ty + r];
    }
}

}  // namespace

hipError_t launch_unfold(const void* x, void* a, const UnfoldShape& s, bool bf16, hipStream_t st) {
    const int64_t total = s.B * s.T * s.ld;
    if (total == 0) return hipSuccess;
    const int64_t nb = std::min<int64_t>((total + 255) / 256, 65536);
    if (bf16)
        hipLaunchKernelGGL(unfold_kernel<uint16_t>, dim3((unsigned)nb), dim3(256), 0, st,
                           static_cast<const uint16_t*>(x), static_cast<uint16_t*>(a), s);
    else
        hipLaunchKernelGGL(unfold_kernel<float>, dim3((unsigned)nb), dim3(256), 0, st,
                           static_cast<const float*>(x), static_cast<float*>(a), s);
    return hipGetLastError();
}

hipError_t launch_tokens(const void* y, void* out, int64_t B, int64_t C, int64_t HW, bool bf16, hipStream_t st) {
    if (B * C * HW == 0) return hipSuccess;
    const dim3 grid((unsigned)((HW + 31) / 32), (unsigned)((C + 31) / 32), (unsigned)B);
    if (bf16)
        hipLaunchKernelGGL(tokens_kernel<uint16_t>, grid, dim3(256), 0, st, static_cast<const uint16_t*>(y),
                           static_cast<uint16_t*>(out), C, HW);
    else
        hipLaunchKernelGGL(tokens_kernel<float>, grid, dim3(256), 0, st, static_cast<const float*>(y),
                           static_cast<float*>(out), C, HW);
    return hipGetLastError();
}

}  // namespace bk
