// bk_private_grad_noalloc: the whole path of bk_private_grad for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc).  The workspace that
// bk_private_grad takes from its caller (per-sample norm partial sums and the
// fp32 partial tiles of K-split GEMM tiles) is a fixed file-scope device array
// here, one copy per GPU, kept until the process ends.
//
// In host code the array's name stands for a host-side shadow, not for device
// memory: its device address on each GPU is looked up once, with that GPU
// current, and only that address ever reaches a kernel.
#include "bk.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "bk_kernels.h"

namespace {

constexpr size_t kScratchBytes = BK_NOALLOC_SCRATCH_BYTES;

// Every kernel writes each scratch word before it reads it within one call,
// so the array needs no clearing between calls.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];   // device address of `scratch` on device i, once looked up

// The device address of `scratch` on device `dev`, which must be current.
hipError_t scratch_address(int dev, void** out) {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace

extern "C" bk_status bk_private_grad_noalloc(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B,
                                             bk_clip mode, float R, float gamma, float noise_std,
                                             uint64_t seed, uint32_t step, float* norm_sq, float* C,
                                             float* total_sq, void* stream) {
    const char* fn = "bk_private_grad_noalloc";
    const size_t need = bk_private_grad_workspace_size(layers, n, dt, B);
    if (need > kScratchBytes)
        return bk::host_fail(BK_ERR_NOT_SUPPORTED,
                             "%s: this stack needs %zu bytes of workspace, more than the %zu-byte "
                             "scratch of the allocation-free call (use bk_private_grad)",
                             fn, need, kScratchBytes);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return bk::host_hip_fail(e, "bk_private_grad_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return bk::host_fail(BK_ERR_NOT_SUPPORTED, "%s: device %d beyond the %d this build tracks", fn,
                             dev, kMaxDevices);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (s) {
        hipDevice_t sdev = -1;
        e = hipStreamGetDevice(s, &sdev);
        if (e != hipSuccess) return bk::host_hip_fail(e, "bk_private_grad_noalloc: hipStreamGetDevice");
        if (sdev != dev)
            return bk::host_fail(BK_ERR_INVALID_VALUE,
                                 "%s: the stream belongs to device %d, the current device is %d", fn,
                                 (int)sdev, dev);
    }
    void* ws = nullptr;
    e = scratch_address(dev, &ws);
    if (e != hipSuccess) return bk::host_hip_fail(e, "bk_private_grad_noalloc: scratch address");
    return bk_private_grad(layers, n, dt, B, mode, R, gamma, noise_std, seed, step, norm_sq, C, total_sq,
                           ws, kScratchBytes, stream);
}
