// GEMMs of the form a^T diag(w) g, contracted over tokens:
//
//  * per-sample gradient instantiation (App. B.4.1): for every sample i the
//    d x p matrix a_i^T g_i (K = T), reduced on chip to ||a_i^T g_i||_F^2;
//  * sum of clipped gradients (Algorithm 1; App. B.3 with clip weights):
//    G = a^T diag(C) g over the flattened B*T rows, row r weighted by C[r / T].
//
// a [.., d] and g [.., p] are row-major with the contraction index (token) as
// the slow index, so both MFMA operands are transposed on their way into LDS.
// A 256-thread workgroup computes one 128 x 128 output tile; each of its four
// waves owns a 64 x 64 quarter as 2 x 2 tiles of 32x32 MFMA accumulators.
//
// LDS layout per operand: [k/4][m][4 k-values] ("k-quad" major), so that
//  - a thread that fetched a 4 (k) x EPV (m) block with 16-byte global loads
//    writes its EPV items as contiguous 16-byte stores, and
//  - a lane's MFMA fragment (8 consecutive k of one row m for bf16, 4 for fp32)
//    is one or two conflict-free reads.
// The clip weight C_i is applied to the rows of g while they are transposed
// (for bf16 the product is rounded to nearest-even bf16 before the MFMA).
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

template <typename T> struct GemmCfg;
template <> struct GemmCfg<bf16_t> {
    static constexpr int EPV = 8;            // elements per 16-byte load
    static constexpr int BK = 64;            // k rows per LDS stage
    static constexpr int ITEM = 8;           // bytes of one 4-k item
};
template <> struct GemmCfg<float> {
    static constexpr int EPV = 4;
    static constexpr int BK = 32;
    static constexpr int ITEM = 16;
};

template <typename T>
struct Smem {
    static constexpr int KQ = GemmCfg<T>::BK / 4;                       // k-quads per stage
    static constexpr int QS = kTile * GemmCfg<T>::ITEM + 16;            // bytes per k-quad (padded)
    static constexpr int BYTES = KQ * QS;                               // one operand
};

template <typename T, bool VEC>
__device__ __forceinline__ uint4 load16_row(const T* X, int K, bool row_ok, int k) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (!row_ok) return v;
    const T* p = X + k;
    if constexpr (VEC) {
        if (k < K) v = *reinterpret_cast<const uint4*>(p);
    } else {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if constexpr (sizeof(T) == 2) {
            const uint16_t* q = reinterpret_cast<const uint16_t*>(p);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (k + e < K) w[e >> 1] |= (uint32_t)q[e] << (16 * (e & 1));
        } else {
            const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (k + e < K) w[e] = q[e];
        }
        v = make_uint4(w[0], w[1], w[2], w[3]);
    }
    return v;
}

__device__ __forceinline__ uint32_t word(const uint4& v, int i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Write the 4 (k) x EPV (m) block held in v[0..3] (row r = k) to LDS as EPV
// items [kq][m0 + j][4 k]; with SCALE, row r is multiplied by c[r] first.
template <typename T, bool SCALE>
__device__ __forceinline__ void store_transposed(char* lds, int kq, int m0, const uint4 v[4],
                                                 const float c[4]) {
    using Cfg = GemmCfg<T>;
    char* base = lds + kq * Smem<T>::QS + m0 * Cfg::ITEM;
    if constexpr (sizeof(T) == 2) {
        uint32_t it[16];   // item j = (it[2j], it[2j+1]) = k-pairs (0,1), (2,3) of column j
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t e[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                uint32_t x = (word(v[r], j >> 1) >> (16 * (j & 1))) & 0xFFFFu;
                if constexpr (SCALE) x = f32_to_bf16(bf16_to_f32(x) * c[r]);
                e[r] = x;
            }
            it[2 * j] = e[0] | (e[1] << 16);
            it[2 * j + 1] = e[2] | (e[3] << 16);
        }
        uint4* dst = reinterpret_cast<uint4*>(base);
#pragma unroll
        for (int w = 0; w < 4; ++w) dst[w] = make_uint4(it[4 * w], it[4 * w + 1], it[4 * w + 2], it[4 * w + 3]);
    } else {
        uint4* dst = reinterpret_cast<uint4*>(base);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float e[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                e[r] = __uint_as_float(word(v[r], j));
                if constexpr (SCALE) e[r] *= c[r];
            }
            dst[j] = make_uint4(__float_as_uint(e[0]), __float_as_uint(e[1]), __float_as_uint(e[2]),
                                __float_as_uint(e[3]));
        }
    }
}

// Fragment of rows [32 ms, 32 ms + 32) for k slab j (16 k for bf16, 8 for fp32).
template <typename T>
__device__ __forceinline__ uint4 frag(const char* lds, int ms, int j, int lane) {
    const int m = ms * 32 + (lane & 31), h = lane >> 5;
    if constexpr (sizeof(T) == 2) {
        const int kq = 4 * j + 2 * h;
        const uint2 lo = *reinterpret_cast<const uint2*>(lds + kq * Smem<T>::QS + m * 8);
        const uint2 hi = *reinterpret_cast<const uint2*>(lds + (kq + 1) * Smem<T>::QS + m * 8);
        return make_uint4(lo.x, lo.y, hi.x, hi.y);
    } else {
        const int kq = 2 * j + h;
        return *reinterpret_cast<const uint4*>(lds + kq * Smem<T>::QS + m * 16);
    }
}

template <typename T, bool INST, bool VEC>
__global__ __launch_bounds__(256) void agemm_kernel(const GemmArgs args) {
    using Cfg = GemmCfg<T>;
    constexpr int EPV = Cfg::EPV, BK = Cfg::BK;
    constexpr int MG = kTile / EPV;           // thread groups along m (n)
    constexpr int KG = 256 / MG;              // k-quads per stage (= BK / 4)
    static_assert(KG * 4 == BK, "stage shape");
    __shared__ __attribute__((aligned(16))) char ldsA[Smem<T>::BYTES];
    __shared__ __attribute__((aligned(16))) char ldsB[Smem<T>::BYTES];
    __shared__ float red[4];

    const int wg = blockIdx.x;
    int l = 0;
    while (l + 1 < args.n && wg >= args.L[l + 1].wg_begin) ++l;
    const GemmLayer& L = args.L[l];
    const int nT = L.T, d = L.d, p = L.p, tn = L.tn;
    const int tiles = L.tm * tn;
    const int local = wg - L.wg_begin;
    const int sample = INST ? local / tiles : 0;
    const int tile = local - sample * tiles;
    const int mt = tile / tn, nt = tile - (tile / tn) * tn;
    const int m0 = mt * kTile, n0 = nt * kTile;

    // Contraction rows: one sample's T rows (instantiation) or all B*T rows.
    const int64_t row0 = INST ? (int64_t)sample * nT : 0;
    const int64_t nrows = INST ? (int64_t)nT : (int64_t)args.B * nT;
    const T* A = reinterpret_cast<const T*>(L.a) + row0 * d;
    const T* Bm = reinterpret_cast<const T*>(L.g) + row0 * p;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kg = tid % KG, mg = tid / KG;   // this thread's k-quad and m group
    const int wm = wave >> 1, wn = wave & 1;
    const int am = m0 + mg * EPV, bn = n0 + mg * EPV;

    f32x16_t acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    uint4 va[4], vb[4];
    float cw[4] = {1.f, 1.f, 1.f, 1.f};
    auto fetch = [&](int64_t k0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t k = k0 + 4 * kg + r;
            const bool ok = k < nrows;
            va[r] = load16_row<T, VEC>(A + (ok ? k : 0) * d, d, ok, am);
            vb[r] = load16_row<T, VEC>(Bm + (ok ? k : 0) * p, p, ok, bn);
            if constexpr (!INST) cw[r] = ok ? args.C[(uint32_t)k / (uint32_t)nT] : 0.f;
        }
    };

    const int64_t nst = (nrows + BK - 1) / BK;
    fetch(0);
    for (int64_t st = 0; st < nst; ++st) {
        __syncthreads();
        store_transposed<T, false>(ldsA, kg, mg * EPV, va, cw);
        store_transposed<T, !INST>(ldsB, kg, mg * EPV, vb, cw);
        __syncthreads();
        if (st + 1 < nst) fetch((st + 1) * BK);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint4 a0 = frag<T>(ldsA, 2 * wm + 0, j, lane);
            const uint4 a1 = frag<T>(ldsA, 2 * wm + 1, j, lane);
            const uint4 b0 = frag<T>(ldsB, 2 * wn + 0, j, lane);
            const uint4 b1 = frag<T>(ldsB, 2 * wn + 1, j, lane);
            Mfma<T>::step(acc[0][0], a0, b0);
            Mfma<T>::step(acc[0][1], a0, b1);
            Mfma<T>::step(acc[1][0], a1, b0);
            Mfma<T>::step(acc[1][1], a1, b1);
        }
    }

    if constexpr (INST) {
        // Padded rows / columns are zero, so the whole tile can be squared.
        float s = 0.f;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int i = 0; i < 16; ++i) s += acc[x][y][i] * acc[x][y][i];
        const float tot = block_sum_256(s, red);
        if (tid == 0) args.part[(size_t)L.part_off + (size_t)sample * tiles + tile] = tot;
    } else {
        float* G = L.G;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int n = n0 + (2 * wn + y) * 32 + (lane & 31);
                if (n >= p) continue;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int m = m0 + (2 * wm + x) * 32 + acc_row(i, lane);
                    if (m < d) G[(size_t)m * p + n] = acc[x][y][i];
                }
            }
    }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& args, int n_wg, bool bf16, bool inst_norm, bool vec,
                       hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    const dim3 grid(n_wg), block(256);
#define BK_GEMM(T, I, V) hipLaunchKernelGGL((agemm_kernel<T, I, V>), grid, block, 0, s, args)
    if (bf16) {
        if (inst_norm) { if (vec) BK_GEMM(bf16_t, true, true); else BK_GEMM(bf16_t, true, false); }
        else           { if (vec) BK_GEMM(bf16_t, false, true); else BK_GEMM(bf16_t, false, false); }
    } else {
        if (inst_norm) { if (vec) BK_GEMM(float, true, true); else BK_GEMM(float, true, false); }
        else           { if (vec) BK_GEMM(float, false, true); else BK_GEMM(float, false, false); }
    }
#undef BK_GEMM
    return hipGetLastError();
}

}  // namespace bk
