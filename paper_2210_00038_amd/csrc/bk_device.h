// Device-side building blocks shared by the BK kernels (gfx950 / CDNA4 only).
//
//  * 16-byte operand fragments and the 32x32 MFMA step that consumes them;
//  * bf16 <-> fp32 conversion (round to nearest even);
//  * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
//    easy as 1, 2, 3", SC'11) and the Box-Muller transform;
//  * wave / workgroup reductions with a fixed summation order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bk {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

// Storage type of a bf16 element.
struct bf16_t { uint16_t bits; };

template <typename T> struct Elem;
template <> struct Elem<float> { static constexpr int per16 = 4; static constexpr int bytes = 4; };
template <> struct Elem<bf16_t> { static constexpr int per16 = 8; static constexpr int bytes = 2; };

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// Round-to-nearest-even fp32 -> bf16 (inputs here are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// ---------------------------------------------------------------------------
// One 32x32 output tile step: acc += A_frag * B_frag^T over the k values that
// a 16-byte fragment per lane carries.
//
// Fragment layout (both operands): lane l holds row (l % 32) of its 32-row
// block and the 16 bytes of that row at k-offset (l / 32) * 16 bytes within
// the current 32-byte k slab.  bf16: one v_mfma_f32_32x32x16_bf16 (8 k values
// per lane, 16 per step).  fp32: four v_mfma_f32_32x32x2_f32, element e of
// every lane's 4 floats forming the e-th step.  Because A and B use the same
// lane -> k assignment, the assignment of k values to MFMA slots is irrelevant
// to the result (a sum over k), which lets rows be read in contiguous 16-byte
// pieces.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<bf16_t> {
    static __device__ __forceinline__ void step(f32x16_t& acc, const uint4& a, const uint4& b) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), acc,
                                                       0, 0, 0);
    }
};

template <> struct Mfma<float> {
    static __device__ __forceinline__ void step(f32x16_t& acc, const uint4& a, const uint4& b) {
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    }
};

// Row (within the 32x32 tile) of accumulator element i of lane `lane`; the
// column is lane % 32.  (Output layout of the 32x32 MFMA family.)
__device__ __forceinline__ int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// ---------------------------------------------------------------------------
// Raw buffer loads.  The resource covers [base, base + bytes); a load whose
// offset lies outside returns zeros instead of touching memory, which replaces
// per-load bounds branches.  All of the offset goes in the VGPR operand (the
// range check applies to it).
// ---------------------------------------------------------------------------
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// A buffer resource over rows k0 .. k0 + rows_max - 1 of a row-major matrix
// (fewer past its last row nrows; none at or past it): the GEMM kernels take
// one per K stage, so the 32-bit offsets of their loads stay within one stage
// and a matrix longer than 2^31 bytes needs no 64-bit offsets.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, uint32_t row_bytes, uint32_t k0,
                                                            uint32_t nrows, uint32_t rows_max) {
    const uint32_t left = k0 < nrows ? min(nrows - k0, rows_max) : 0u;
    return make_rsrc(static_cast<const char*>(base) + (size_t)k0 * row_bytes, left * row_bytes);
}

// ---------------------------------------------------------------------------
// Workgroup barrier for LDS producer/consumer hand-offs.  It waits for this
// wave's LDS (and scalar) operations only, not for its global loads still in
// flight: those write the wave's own registers, so prefetches issued before
// the barrier stay in flight across it (__syncthreads() would drain them).
// The "memory" clobber keeps the compiler from moving memory accesses across.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N of this wave's vector-memory operations (loads,
// including loads into LDS, and stores) are outstanding.  They complete in
// order.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt immediate (6 bits)");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Global -> LDS copy of 16 bytes per lane (LDS DMA): lane l's bytes land at
// lds_dst + 16 l, lds_dst being the same for the whole wave.  The offset is
// range-checked like buffer_load16 (zeros outside the resource).
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t r, uint32_t off, void* lds_dst) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_dst, 16, off, 0, 0, 0);
}

// LDS DMA of 16 bytes per lane (as buffer_load16_lds), issued from inline
// assembly.  The compiler treats LDS reads as possibly reading any LDS DMA
// destination and would wait for every DMA in flight before each of them,
// which serialises a prefetch ring; hidden in assembly, the DMA is not
// tracked, and the kernel waits for it itself (wait_vmcnt) before the barrier
// that publishes a stage.  rs: buffer descriptor words (base, base high, bytes,
// flags); m0 takes the wave-uniform LDS destination.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t raw_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return (u32x4_t){(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, bytes, 0x00020000u};
}

// rows_rsrc as raw descriptor words (for dma16_asm).
__device__ __forceinline__ u32x4_t rows_raw_rsrc(const void* base, uint32_t row_bytes, uint32_t k0,
                                                 uint32_t nrows, uint32_t rows_max) {
    const uint32_t left = k0 < nrows ? min(nrows - k0, rows_max) : 0u;
    return raw_rsrc(static_cast<const char*>(base) + (size_t)k0 * row_bytes, left * row_bytes);
}

__device__ __forceinline__ void dma16_asm(const u32x4_t& rs, uint32_t off, char* lds_dst) {
    const uint32_t m0v = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_dst;
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :: "v"(off), "s"(rs), "s"(__builtin_amdgcn_readfirstlane(m0v)) : "memory", "m0");
}

// ---------------------------------------------------------------------------
// Reductions in a fixed order (deterministic).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Logical index of workgroup `wg` of `n` such that consecutive logical
// indices run on the same XCD (workgroups are dealt round-robin to the 8
// XCDs, each with its own L2).
__device__ __forceinline__ int xcd_remap(int wg, int n) {
    const int x = wg & 7, idx = wg >> 3, per = n >> 3, rem = n & 7;
    return x * per + min(x, rem) + idx;
}

// Descriptor of workgroup `wg` in a grouped launch: the last l < n with
// begin(l) <= wg, begin(l) being descriptor l's first workgroup
// (non-decreasing in l, begin(0) = 0).  Binary search: a handful of
// dependent scalar loads of the kernel arguments instead of one per
// preceding descriptor.
template <typename Begin>
__device__ __forceinline__ int find_desc(int n, int64_t wg, Begin begin) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)begin(mid) <= wg) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Sum of one float per thread over a 256-thread workgroup; result valid in
// thread 0.  `red` must hold 4 floats of LDS.
__device__ __forceinline__ float block_sum_256(float v, float* red) {
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float s = 0.f;
    if (threadIdx.x == 0) s = (red[0] + red[1]) + (red[2] + red[3]);
    return s;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (SC'11): two 32x32->64 multiplications per round, key bumped
// by the Weyl constants between rounds.
// ---------------------------------------------------------------------------
constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // each 32x32 -> 64-bit product in one multiply (v_mad_u64_u32)
        const uint64_t p0 = (uint64_t)kPhiloxM0 * c.x, p1 = (uint64_t)kPhiloxM1 * c.z;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    return c;
}

// Counter block q of tensor `tid` at step `step` under `seed`.
__device__ __forceinline__ uint4 philox_block(uint64_t seed, uint32_t tid, uint32_t step, uint64_t q) {
    return philox4x32_10(make_uint4((uint32_t)q, (uint32_t)(q >> 32), tid, step), (uint32_t)seed,
                         (uint32_t)(seed >> 32));
}

// u = (2 (w >> 9) + 1) 2^-24: an odd multiple of 2^-24, exact in fp32, in (0, 1).
__device__ __forceinline__ float word_to_uniform(uint32_t w) {
    return (float)(2u * (w >> 9) + 1u) * 5.9604644775390625e-08f;
}

// Box-Muller: (r cos 2 pi u1, r sin 2 pi u1), r = sqrt(-2 ln u0), with the
// hardware transcendentals: v_log_f32 (log2; ln u = log2 u ln 2), v_sqrt_f32
// (the argument is >= 2^-23, no denormals), and v_sin_f32 / v_cos_f32, whose
// input is in turns, so u1 in (0, 1) needs no range reduction.
__device__ __forceinline__ float2 box_muller(uint32_t w0, uint32_t w1) {
    const float u0 = word_to_uniform(w0), u1 = word_to_uniform(w1);
    const float r = __builtin_amdgcn_sqrtf(-2.0f * 0.693147180559945309f * __builtin_amdgcn_logf(u0));
    return make_float2(r * __builtin_amdgcn_cosf(u1), r * __builtin_amdgcn_sinf(u1));
}

// The four standard normals of counter block q.
__device__ __forceinline__ float4 normal4(uint64_t seed, uint32_t tid, uint32_t step, uint64_t q) {
    const uint4 w = philox_block(seed, tid, step, q);
    const float2 z01 = box_muller(w.x, w.y), z23 = box_muller(w.z, w.w);
    return make_float4(z01.x, z01.y, z23.x, z23.y);
}

}  // namespace bk
