// Ceiling of the clipped-gradient GEMM's inner loop on one MI355X.
//
// agrad_dl_kernel (agemm.hip) runs 256 x 256 output tiles on 512 threads:
// eight waves of 128 x 64 (4 x 2 MFMA 32x32x16 bf16 accumulators), 32-row
// K stages in a four-buffer LDS ring filled by LDS DMA, fragments gathered
// with transposing LDS reads, and a ping-pong schedule (waves 4-7 one phase
// behind waves 0-3; each stage is a memory phase and an MFMA phase, each
// ended by a barrier).  This program times that loop alone, without HBM
// operands, prologue or epilogue, over a full-chip grid (1280 workgroups of
// 128 stages), in four steps that add one cost at a time:
//   mfma     the wave's 16 MFMAs per stage on operands held in registers
//   loop     + the 24 transposing LDS reads per stage and the two barriers
//   dma      + the stage's LDS DMA (32 KB from an L2-resident 1 MB buffer)
//            issued among the MFMAs, as in the kernel
//   rescale  + 128 accumulator multiplies every fourth stage (the clip-weight
//            rescale at a sample boundary when T = 128)
// each on random bf16 data and on zeros: the MFMA power, and so the clock the
// chip holds, depends on the data.  TFLOP/s count 2 * 256 * 256 * 32 per
// stage and workgroup.
//
// Build and run (one MI355X):
//   python paper_2210_00038_amd/build.py --ceiling
//   _build/gemm_loop
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#define CHECK(x)                                                                          \
    do {                                                                                  \
        hipError_t e_ = (x);                                                              \
        if (e_ != hipSuccess) {                                                           \
            std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);   \
            return 1;                                                                     \
        }                                                                                 \
    } while (0)

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRow = 512;                    // bytes of one LDS row (256 bf16)
constexpr int kStageOp = 32 * kRow;          // one operand of one 32-row stage
constexpr int kStage = 2 * kStageOp;         // a and g
constexpr int kSrcBytes = 1 << 20;           // DMA source, L2-resident

enum Variant { kMfma = 0, kLoop = 1, kDma = 2, kRescale = 3 };

__device__ __forceinline__ uint2 tr16(const char* p) {
    const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p));
    return __builtin_bit_cast(uint2, v);
}

// 16-byte column c of row r at c ^ 4 (r mod 4), as in the kernel.
__device__ __forceinline__ int swz(int row, int c16) { return c16 ^ (4 * (row & 3)); }

// MFMA 32x32x16 fragment (8 consecutive k of one column) of the 32 columns
// from cb on, k rows kb .. kb + 15, by two transposing reads.
__device__ __forceinline__ uint4 frag(const char* lds, int kb, int cb, int lane) {
    const int grp = lane >> 4, i = lane & 15;
    uint2 h[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
        const int row = kb + 8 * (grp >> 1) + (i >> 2) + 4 * hh;
        const int col = cb + 16 * (grp & 1) + 4 * (i & 3);
        h[hh] = tr16(lds + row * kRow + swz(row, col >> 3) * 16 + (col & 7) * 2);
    }
    return make_uint4(h[0].x, h[0].y, h[1].x, h[1].y);
}

__device__ __forceinline__ u32x4 raw_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return (u32x4){(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, bytes, 0x00020000u};
}

// One 16-byte-per-lane buffer load straight into LDS (1 KB per instruction).
__device__ __forceinline__ void dma16(const u32x4& rs, uint32_t off, char* lds_dst) {
    const uint32_t m0v = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_dst;
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :: "v"(off), "s"(rs), "s"(__builtin_amdgcn_readfirstlane(m0v)) : "memory", "m0");
}

__device__ __forceinline__ void phase_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Random bf16 in [-2, 2) with both signs (or zeros), from a hash of the index.
__device__ __host__ inline uint32_t bf16_pair(uint32_t i, bool zero) {
    uint32_t h = i * 2654435761u ^ 0x9E3779B9u;
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    const uint32_t lo = (h & 0x807Fu) | ((126u + (h >> 7) % 3u) << 7);
    const uint32_t hi = ((h >> 16) & 0x807Fu) | ((126u + (h >> 23) % 3u) << 7);
    return zero ? 0u : (lo | (hi << 16));
}

template <int V, bool ZERO>
__global__ __launch_bounds__(512, 1) void loop_kernel(int nst, const char* src, float* sink) {
    __shared__ __attribute__((aligned(16))) char lds[4 * kStage];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < 4 * kStage / 4; i += 512) reinterpret_cast<uint32_t*>(lds)[i] = bf16_pair(i, ZERO);
    __syncthreads();
    const int wm = wave >> 2, wn = wave & 3;   // 2 x 4 waves of 128 x 64
    f32x16 acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = (f32x16){};
    const u32x4 rs = raw_rsrc(src, kSrcBytes);
    uint4 fa[2][4], fb[2][2];
    // operands in registers for the MFMA-only variant
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
        for (int x = 0; x < 4; ++x) fa[s][x] = frag(lds, 16 * s, 128 * wm + 32 * x, lane);
#pragma unroll
        for (int y = 0; y < 2; ++y) fb[s][y] = frag(lds + kStageOp, 16 * s, 64 * wn + 32 * y, lane);
    }
    // Waves 4-7 one phase behind: one extra barrier at the start for them and
    // at the end for waves 0-3, so every wave passes the same number.
    if (V != kMfma && wave >= 4) phase_barrier();
    for (int st = 0; st < nst; ++st) {
        // memory phase: the stage's fragments (two 16-row steps)
        if constexpr (V != kMfma) {
            const char* A = lds + (st & 3) * kStage;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
#pragma unroll
                for (int x = 0; x < 4; ++x) fa[s][x] = frag(A, 16 * s, 128 * wm + 32 * x, lane);
#pragma unroll
                for (int y = 0; y < 2; ++y) fb[s][y] = frag(A + kStageOp, 16 * s, 64 * wn + 32 * y, lane);
            }
            if constexpr (V >= kDma) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
            if constexpr (V == kRescale) {
                if ((st & 3) == 0) {
                    const float r = 1.0001f + (float)st * 1e-9f;
#pragma unroll
                    for (int x = 0; x < 4; ++x)
#pragma unroll
                        for (int y = 0; y < 2; ++y)
#pragma unroll
                            for (int e = 0; e < 16; ++e) acc[x][y][e] *= r;
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            phase_barrier();
        }
        // MFMA phase: 16 MFMAs, the stage-three-ahead DMA among the first eight
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[s][x]),
                                                                        __builtin_bit_cast(bf16x8, fb[s][y]),
                                                                        acc[x][y], 0, 0, 0);
                    if constexpr (V >= kDma) {
                        if (s == 0 && y == 1) {
                            const int j = 8 * x + wave;                      // 32 pieces of 1 KB
                            char* dst = lds + ((st + 3) & 3) * kStage + j * 1024;
                            dma16(rs, (uint32_t)((((st * 32 + j) * 1024) + lane * 16) & (kSrcBytes - 1)), dst);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
        __builtin_amdgcn_s_setprio(0);
        if constexpr (V != kMfma) phase_barrier();
    }
    if (V != kMfma && wave < 4) phase_barrier();
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    float t = 0.f;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int e = 0; e < 16; ++e) t += acc[x][y][e];
    if (t == 1234.5f) sink[tid] = t;          // keeps the accumulators live
}

template <int V, bool Z>
int run(const char* name, int nwg, int nst, const char* src, float* sink, hipEvent_t e0, hipEvent_t e1) {
    float ms = 0.f;
    CHECK(hipEventRecord(e0));
    hipLaunchKernelGGL((loop_kernel<V, Z>), dim3(nwg), dim3(512), 0, 0, nst, src, sink);
    CHECK(hipGetLastError());
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double flops = (double)nwg * nst * 2.0 * 256 * 256 * 32;
    std::printf("%-9s %-6s %8.3f ms %7.0f TFLOP/s\n", name, Z ? "zeros" : "random", ms, flops / ms / 1e9);
    std::fflush(stdout);
    return 0;
}

}  // namespace

int main() {
    const int nwg = 1280, nst = 128;
    float* sink = nullptr;
    char* src = nullptr;
    CHECK(hipMalloc(&sink, 512 * sizeof(float)));
    CHECK(hipMalloc(&src, kSrcBytes));
    {
        static uint32_t host[kSrcBytes / 4];
        for (uint32_t i = 0; i < kSrcBytes / 4; ++i) host[i] = bf16_pair(i + 77777u, false);
        CHECK(hipMemcpy(src, host, kSrcBytes, hipMemcpyHostToDevice));
    }
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    // raise the clock from idle before timing
    for (int i = 0; i < 20; ++i) hipLaunchKernelGGL((loop_kernel<kLoop, false>), dim3(nwg), dim3(512), 0, 0, nst, src, sink);
    CHECK(hipDeviceSynchronize());
    for (int rep = 0; rep < 3; ++rep) {
        if (run<kMfma, false>("mfma", nwg, nst, src, sink, e0, e1) || run<kMfma, true>("mfma", nwg, nst, src, sink, e0, e1) ||
            run<kLoop, false>("loop", nwg, nst, src, sink, e0, e1) || run<kLoop, true>("loop", nwg, nst, src, sink, e0, e1) ||
            run<kDma, false>("dma", nwg, nst, src, sink, e0, e1) || run<kDma, true>("dma", nwg, nst, src, sink, e0, e1) ||
            run<kRescale, false>("rescale", nwg, nst, src, sink, e0, e1) ||
            run<kRescale, true>("rescale", nwg, nst, src, sink, e0, e1))
            return 1;
    }
    CHECK(hipFree(sink));
    CHECK(hipFree(src));
    return 0;
}
