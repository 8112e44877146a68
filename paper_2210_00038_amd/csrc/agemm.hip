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

#include <algorithm>
#include <type_traits>

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

// The 16 values of one 32x32 accumulator column n (rows r0 + acc_row(i, lane),
// those below rmax) into out[m sm + n sn], times `scale`; with `add` they are
// added to what out holds, the 16 old values being loaded before any store so
// that the loads overlap (gradient accumulation).
__device__ __forceinline__ void put_col16(float* out, size_t sm, size_t sn, int r0, int rmax, int n, int lane,
                                          const f32x16_t& v, float scale, bool add) {
    if (add) {
        // The product is rounded before the add (no fused multiply-add), so
        // that adding to G gives the same value as writing v * scale and
        // adding G's old value afterwards.
#pragma clang fp contract(off)
        float o[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int m = r0 + acc_row(i, lane);
            o[i] = m < rmax ? out[(size_t)m * sm + (size_t)n * sn] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int m = r0 + acc_row(i, lane);
            if (m < rmax) out[(size_t)m * sm + (size_t)n * sn] = o[i] + v[i] * scale;
        }
    } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int m = r0 + acc_row(i, lane);
            if (m < rmax) out[(size_t)m * sm + (size_t)n * sn] = v[i] * scale;
        }
    }
}

// 4 x 4 transpose inside each quad of lanes (DPP quad permutations): lane j
// of a quad holds v[r] = M[r][j] for the quad's four columns and ends with
// v[c] = M[j][c].  Two exchange steps, between lanes j ^ 1 and then j ^ 2.
__device__ __forceinline__ float dpp_xor1(float a) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a), 0xB1, 0xF, 0xF, false));   // [1,0,3,2]
}
__device__ __forceinline__ float dpp_xor2(float a) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a), 0x4E, 0xF, 0xF, false));   // [2,3,0,1]
}
__device__ __forceinline__ void quad_transpose(float (&v)[4], int lane) {
    const bool o1 = (lane & 1) != 0, o2 = (lane & 2) != 0;
    const float p0 = dpp_xor1(v[0]), p1 = dpp_xor1(v[1]), p2 = dpp_xor1(v[2]), p3 = dpp_xor1(v[3]);
    const float u0 = o1 ? p1 : v[0], u1 = o1 ? v[1] : p0, u2 = o1 ? p3 : v[2], u3 = o1 ? v[3] : p2;
    const float q0 = dpp_xor2(u0), q1 = dpp_xor2(u1), q2 = dpp_xor2(u2), q3 = dpp_xor2(u3);
    v[0] = o2 ? q2 : u0;
    v[1] = o2 ? q3 : u1;
    v[2] = o2 ? u2 : q0;
    v[3] = o2 ? u3 : q1;
}

// put_col16 with 16-byte stores: the 32x32 accumulator block at (r0, c0) of
// out (row stride ld floats) times `scale` (or added to out), rows below
// rmax.  Each group of four rows is transposed inside the lane quads, so a
// lane writes four consecutive columns of one row.  Needs out 16-byte aligned
// and ld and c0 multiples of 4; columns past cmax (a multiple of 4) are
// skipped.  Every element gets the same operations as in put_col16.
__device__ __forceinline__ void put_acc_x4(float* out, size_t ld, int r0, int rmax, int c0, int cmax, int lane,
                                           const f32x16_t& acc, float scale, bool add) {
#pragma clang fp contract(off)
    const int c = c0 + ((lane & 31) & ~3);
    const int rl = 4 * ((lane >> 5) & 1) + (lane & 3);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float v[4] = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
        quad_transpose(v, lane);
        const int r = r0 + 8 * q + rl;
        if (r < rmax && c < cmax) {
            float4* dst = reinterpret_cast<float4*>(out + (size_t)r * ld + (size_t)c);
            float4 o;
            if (add) {
                const float4 g = *dst;
                o = make_float4(g.x + v[0] * scale, g.y + v[1] * scale, g.z + v[2] * scale, g.w + v[3] * scale);
            } else {
                o = make_float4(v[0] * scale, v[1] * scale, v[2] * scale, v[3] * scale);
            }
            *dst = o;
        }
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
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
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
        lds_barrier();
        store_transposed<T, false>(ldsA, kg, mg * EPV, va, cw);
        store_transposed<T, !INST>(ldsB, kg, mg * EPV, vb, cw);
        lds_barrier();
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
        if (L.G) {   // keep the per-sample gradient (BK-MixOpt): P[sample] [d,p]
            float* P = L.G + (size_t)sample * d * p;
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const int n = n0 + (2 * wn + y) * 32 + (lane & 31);
                    if (n >= p) continue;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int m = m0 + (2 * wm + x) * 32 + acc_row(i, lane);
                        if (m < d) P[(size_t)m * p + n] = acc[x][y][i];
                    }
                }
        }
    } else {
        float* G = L.G;
        const bool add = L.accum != 0;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int n = n0 + (2 * wn + y) * 32 + (lane & 31);
                if (n < p) put_col16(G, (size_t)p, 1, m0 + (2 * wm + x) * 32, d, n, lane, acc[x][y], 1.f, add);
            }
    }
}

// ---------------------------------------------------------------------------
// bf16 kernel for 16-byte aligned rows.  Tiles are staged in LDS exactly as
// they sit in memory ([k][m] with m contiguous: plain 16-byte copies) and the
// MFMA fragments are gathered with the gfx950 LDS transpose read
// ds_read_b64_tr_b16: in each 16-lane group, lanes 4q..4q+3 point at 16
// consecutive columns of row q, and lane j receives column j of the 4 rows.
// Two such reads give a lane the 8 k values of its column.
//
// Workgroup tile 256 (m) x 128 (n), k stage 64, two workgroups per CU; wave
// (wm, wn) owns rows [128 wm, 128 wm + 128) x columns [64 wn, 64 wn + 64) as
// 4 x 2 MFMA 32x32x16 accumulators.  One LDS buffer per stage: the next
// stage's global loads are issued right after the tile is written and land
// in registers while the waves multiply.  LDS rows are padded to 576 / 320
// bytes so that the four rows a 16-lane group reads fall on distinct banks.
// The other workgroup on the CU covers this one's barriers.
// ---------------------------------------------------------------------------
constexpr uint32_t kOut = 0xFFFFFFF0u;           // buffer offset that loads zeros
constexpr int kBM = kWideM, kBN = kWideN, kBK = kWideK;
constexpr int kSA = kBM * 2 + 64;                // bytes per staged k-row of a
constexpr int kSB = kBN * 2 + 64;                // bytes per staged k-row of g

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint2 lds_tr16(const char* p) {
    const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(p));
    return __builtin_bit_cast(uint2, v);
}

// Fragment of columns [cb, cb + 32) for k rows [kb, kb + 16) of a [k][col]
// tile with row stride S bytes: lane l ends with 8 k values of column
// cb + 16 ((l >> 4) & 1) + (l & 15), k = kb + 8 (l >> 5) + 0..7.
template <int S>
__device__ __forceinline__ uint4 frag_tr(const char* lds, int kb, int cb, int lane) {
    const int grp = lane >> 4, i = lane & 15;
    const int row = kb + 8 * (grp >> 1) + (i >> 2);
    const int col = cb + 16 * (grp & 1) + 4 * (i & 3);
    const char* p = lds + row * S + col * 2;
    const uint2 lo = lds_tr16(p), hi = lds_tr16(p + 4 * S);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

// Half h of frag_tr: rows kb + 4 h + 8 (l >> 5) + 0..3 of the same column.
template <int S>
__device__ __forceinline__ uint2 frag_tr_half(const char* lds, int kb, int cb, int lane, int h) {
    const int grp = lane >> 4, i = lane & 15;
    const int row = kb + 8 * (grp >> 1) + (i >> 2) + 4 * h;
    const int col = cb + 16 * (grp & 1) + 4 * (i & 3);
    return lds_tr16(lds + row * S + col * 2);
}

// Full TM x TN float32 partial tile of a K slice (row-major, stride TN) from
// the 4 x 2 accumulators of a wave owning rows [r0, r0 + 128) and columns
// [c0, c0 + 64), each value multiplied by `scale`.
template <int TM, int TN>
__device__ __forceinline__ void store_partial_tile(float* P, const f32x16_t (&acc)[4][2], int r0, int c0,
                                                   int lane, float scale) {
    static_assert(TN % 4 == 0, "16-byte rows");
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) put_acc_x4(P, TN, r0 + 32 * x, TM, c0 + 32 * y, TN, lane, acc[x][y], scale, false);
}

// Two bf16 in one word, each multiplied by c, rounded to nearest even.
__device__ __forceinline__ uint32_t scale_bf16x2(uint32_t w, float c) {
    const f32x2_t f = {__uint_as_float(w << 16) * c, __uint_as_float(w & 0xFFFF0000u) * c};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}


template <bool INST>
__global__ __launch_bounds__(256, 2) void agemm_bf16_kernel(const GemmArgs args, int n_wg) {
    __shared__ __attribute__((aligned(16))) char ldsA[kBK * kSA];
    __shared__ __attribute__((aligned(16))) char ldsB[kBK * kSB];
    __shared__ float red[4];

    const int wg = xcd_remap(blockIdx.x, n_wg);
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GemmLayer& L = args.L[l];
    const int nT = L.T, d = L.d, p = L.p, tn = L.tn;
    const int tiles = L.tm * tn;
    const int ks = max(L.ksplit, 1), local = wg - L.wg_begin;
    const int sample = INST ? local / (tiles * ks) : 0;
    const int rem = local - sample * tiles * ks;
    const int tile = rem / ks, slice = rem - tile * ks;
    const int mt = tile / tn, nt = tile - mt * tn;
    const int m0 = mt * kBM, n0 = nt * kBN;

    // Contraction rows: one sample's T rows (instantiation) or all B*T rows,
    // addressed stage by stage (rows_rsrc).
    const int64_t row0 = INST ? (int64_t)sample * nT : 0;
    const uint32_t nrows = INST ? (uint32_t)nT : (uint32_t)args.B * (uint32_t)nT;
    const uint32_t rowA = (uint32_t)d * 2u, rowB = (uint32_t)p * 2u;
    const bf16_t* baseA = reinterpret_cast<const bf16_t*>(L.a) + row0 * d;
    const bf16_t* baseB = reinterpret_cast<const bf16_t*>(L.g) + row0 * p;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // Staging: the a tile is 64 rows x 32 chunks of 16 B (8 chunks per
    // thread), the g tile 64 rows x 16 chunks (4 per thread).  Rows past the
    // last one fall outside the buffer resource and load as zeros; chunks past
    // the last column get an out-of-range offset and load as zeros too.
    const int ca = (tid & 31) * 8, ka = tid >> 5;      // + 8 j rows
    const int cb = (tid & 15) * 8, kb = tid >> 4;      // + 16 j rows
    const uint32_t offA = (m0 + ca < d) ? (uint32_t)ka * rowA + (uint32_t)(m0 + ca) * 2u : kOut;
    const uint32_t offB = (n0 + cb < p) ? (uint32_t)kb * rowB + (uint32_t)(n0 + cb) * 2u : kOut;

    f32x16_t acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    uint4 va[8], vb[4];
    float cw[4];
    auto fetch = [&](uint32_t k0) {
        const __amdgpu_buffer_rsrc_t rA = rows_rsrc(baseA, rowA, k0, nrows, kBK);
        const __amdgpu_buffer_rsrc_t rB = rows_rsrc(baseB, rowB, k0, nrows, kBK);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            va[j] = buffer_load16(rA, offA == kOut ? kOut : offA + 8u * j * rowA);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            vb[j] = buffer_load16(rB, offB == kOut ? kOut : offB + 16u * j * rowB);
        if constexpr (!INST) {
            // Clip weight of each staged g row: C[k / T].  When T >= 64 the 64
            // rows of a stage span at most two samples (scalar split point).
            const uint32_t q0 = k0 / (uint32_t)nT;
            if (nT >= kBK) {
                const uint32_t split = (q0 + 1u) * (uint32_t)nT - k0;
                const float c0 = args.C[min(q0, (uint32_t)args.B - 1u)];
                const float c1 = args.C[min(q0 + 1u, (uint32_t)args.B - 1u)];
#pragma unroll
                for (int j = 0; j < 4; ++j) cw[j] = ((uint32_t)(kb + 16 * j) < split) ? c0 : c1;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t k = min(k0 + (uint32_t)(kb + 16 * j), nrows - 1u);
                    cw[j] = args.C[k / (uint32_t)nT];
                }
            }
        }
    };

    // This workgroup's stages (K slice `slice` of `ks`).
    const uint32_t nst_all = (nrows + kBK - 1) / kBK;
    const uint32_t st_begin = (uint32_t)((uint64_t)slice * nst_all / (uint32_t)ks);
    const uint32_t nst = (uint32_t)((uint64_t)(slice + 1) * nst_all / (uint32_t)ks);
    if (st_begin < nst) fetch(st_begin * kBK);
    for (uint32_t st = st_begin; st < nst; ++st) {
        lds_barrier();
#pragma unroll
        for (int j = 0; j < 8; ++j)
            *reinterpret_cast<uint4*>(ldsA + (ka + 8 * j) * kSA + ca * 2) = va[j];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint4 v = vb[j];
            if constexpr (!INST)
                v = make_uint4(scale_bf16x2(v.x, cw[j]), scale_bf16x2(v.y, cw[j]), scale_bf16x2(v.z, cw[j]),
                               scale_bf16x2(v.w, cw[j]));
            *reinterpret_cast<uint4*>(ldsB + (kb + 16 * j) * kSB + cb * 2) = v;
        }
        lds_barrier();
        if (st + 1 < nst) fetch((st + 1) * kBK);
        // Fragments of step kk + 1 are read while the MFMAs of step kk run.
        uint4 fa[2][4], fb[2][2];
#pragma unroll
        for (int x = 0; x < 4; ++x) fa[0][x] = frag_tr<kSA>(ldsA, 0, 128 * wm + 32 * x, lane);
#pragma unroll
        for (int y = 0; y < 2; ++y) fb[0][y] = frag_tr<kSB>(ldsB, 0, 64 * wn + 32 * y, lane);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int cur = kk & 1, nxt = cur ^ 1;
            if (kk + 1 < kBK / 16) {
#pragma unroll
                for (int x = 0; x < 4; ++x) fa[nxt][x] = frag_tr<kSA>(ldsA, 16 * (kk + 1), 128 * wm + 32 * x, lane);
#pragma unroll
                for (int y = 0; y < 2; ++y) fb[nxt][y] = frag_tr<kSB>(ldsB, 16 * (kk + 1), 64 * wn + 32 * y, lane);
            }
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) Mfma<bf16_t>::step(acc[x][y], fa[cur][x], fb[cur][y]);
        }
    }

    if (ks > 1) {
        store_partial_tile<kBM, kBN>(
            args.tiles + L.ptile_off + (((size_t)sample * tiles + tile) * ks + slice) * (kBM * kBN),
            acc, 128 * wm, 64 * wn, lane, 1.f);
        return;
    }
    if constexpr (INST) {
        float s = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const bool col_ok = n0 + 64 * wn + 32 * y + (lane & 31) < p;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const bool ok = col_ok && (m0 + 128 * wm + 32 * x + acc_row(i, lane) < d);
                    s += ok ? acc[x][y][i] * acc[x][y][i] : 0.f;
                }
            }
        const float tot = block_sum_256(s, red);
        if (tid == 0) args.part[(size_t)L.part_off + (size_t)sample * tiles + tile] = tot;
        if (L.G) {   // keep the per-sample gradient (BK-MixOpt): P[sample] [d,p]
            float* P = L.G + (size_t)sample * d * p;
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const int n = n0 + 64 * wn + 32 * y + (lane & 31);
                    if (n >= p) continue;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int m = m0 + 128 * wm + 32 * x + acc_row(i, lane);
                        if (m < d) P[(size_t)m * p + n] = acc[x][y][i];
                    }
                }
        }
    } else {
        float* G = L.G;
        const bool add = L.accum != 0;
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int n = n0 + 64 * wn + 32 * y + (lane & 31);
                if (n < p) put_col16(G, (size_t)p, 1, m0 + 128 * wm + 32 * x, d, n, lane, acc[x][y], 1.f, add);
            }
    }
}

// ---------------------------------------------------------------------------
// Narrow layers: one side of the d x p output is at most BN (32 or 64), as in
// LoRA / adapter sub-modules (rank r) and convolutions with few output
// channels.  The workgroup computes a 256 x BN tile of X^T diag(w) Y with X
// the operand of the long side and Y the other: X = a, Y = g when p <= d,
// else X = g, Y = a and the tile is G^T (the clip weight still scales whole
// rows of the staged Y, which gives the same sum).  Four waves each own 64
// rows x BN columns as 2 x BN/32 MFMA 32x32x16 accumulators; a k stage is
// 64 rows, staged through two register sets (two stages in flight while the
// waves write one to LDS and multiply).  Y's LDS rows are padded to 192
// bytes so the four rows of a transposed read fall on distinct banks.  The
// clipped gradient runs here only for T >= 64 (a stage then spans at most two
// samples, whose weights come through scalar loads).
// ---------------------------------------------------------------------------
constexpr int kNM = kNarrowM;
constexpr int kNSY = 192;

template <bool INST, int BN>
__global__ __launch_bounds__(256, 2) void anarrow_kernel(const GemmArgs args, int n_wg) {
    static_assert(BN == 32 || BN == 64, "narrow tile width");
    constexpr int NY = BN / 32;           // accumulator columns per wave
    constexpr int CPR = BN / 8;           // 16-byte chunks per staged Y row
    constexpr int RPP = 256 / CPR;        // Y rows staged per pass of 256 threads
    constexpr int NP = kBK / RPP;         // passes (Y chunks per thread)
    __shared__ __attribute__((aligned(16))) char ldsA[kBK * kSA];
    __shared__ __attribute__((aligned(16))) char ldsB[kBK * kNSY];
    __shared__ float red[4];

    const int wg = xcd_remap(blockIdx.x, n_wg);
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GemmLayer& L = args.L[l];
    const bool sw = L.swap != 0;
    const int nT = L.T, d = L.d, p = L.p, tn = L.tn;
    const int Md = sw ? p : d, Nd = sw ? d : p;
    const int tiles = L.tm * tn;
    const int ks = max(L.ksplit, 1), local = wg - L.wg_begin;
    const int sample = INST ? local / (tiles * ks) : 0;
    const int rem = local - sample * tiles * ks;
    const int tile = rem / ks, slice = rem - tile * ks;
    const int mt = tile / tn, nt = tile - mt * tn;
    const int m0 = mt * kNM, n0 = nt * BN;

    // Contraction rows addressed stage by stage (rows_rsrc).
    const int64_t row0 = INST ? (int64_t)sample * nT : 0;
    const uint32_t nrows = INST ? (uint32_t)nT : (uint32_t)args.B * (uint32_t)nT;
    const uint32_t rowX = (uint32_t)Md * 2u, rowY = (uint32_t)Nd * 2u;
    const bf16_t* X = reinterpret_cast<const bf16_t*>(sw ? L.g : L.a) + row0 * Md;
    const bf16_t* Y = reinterpret_cast<const bf16_t*>(sw ? L.a : L.g) + row0 * Nd;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // X tile: 64 rows x 32 chunks (rows ka + 8 j); Y tile: 64 rows x CPR
    // chunks (rows kb + RPP j).  Rows past the last one fall outside the
    // buffer resource and chunks past the last column get an out-of-range
    // offset: both load as zeros.
    const int ca = (tid & 31) * 8, ka = tid >> 5;
    const int cb = (tid % CPR) * 8, kb = tid / CPR;
    const uint32_t offA = (m0 + ca < Md) ? (uint32_t)ka * rowX + (uint32_t)(m0 + ca) * 2u : kOut;
    const uint32_t offB = (n0 + cb < Nd) ? (uint32_t)kb * rowY + (uint32_t)(n0 + cb) * 2u : kOut;

    f32x16_t acc[2][NY];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < NY; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    // Two register sets of staged rows: the loads of stages st + 1 and st + 2
    // are in flight while stage st is written to LDS and multiplied.  Every
    // fetch is issued (a stage past the slice loads zeros through the
    // out-of-range offset, without memory traffic) and stages run in pairs,
    // so the loop is straight-line and each wait covers exactly one set.
    uint4 va0[8], vb0[NP], va1[8], vb1[NP];
    float cw0[NP], cw1[NP];
    const uint32_t nst_all = (nrows + kBK - 1) / kBK;
    const uint32_t st_begin = (uint32_t)((uint64_t)slice * nst_all / (uint32_t)ks);
    const uint32_t nst = (uint32_t)((uint64_t)(slice + 1) * nst_all / (uint32_t)ks);
    // Clip weights come through the scalar cache (C is read-only here), so
    // their loads do not sit in the vector-memory count between two sets.
    const __attribute__((address_space(4))) float* Cs = (const __attribute__((address_space(4))) float*)args.C;
    auto fetch = [&](uint4 (&va)[8], uint4 (&vb)[NP], float (&cw)[NP], uint32_t st) {
        const uint32_t k0 = st * kBK;
        const bool live = st < nst;
        const __amdgpu_buffer_rsrc_t rA = rows_rsrc(X, rowX, k0, nrows, kBK);
        const __amdgpu_buffer_rsrc_t rB = rows_rsrc(Y, rowY, k0, nrows, kBK);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            va[j] = buffer_load16(rA, (offA == kOut || !live) ? kOut : offA + 8u * j * rowX);
#pragma unroll
        for (int j = 0; j < NP; ++j)
            vb[j] = buffer_load16(rB, (offB == kOut || !live) ? kOut : offB + (uint32_t)RPP * j * rowY);
        if constexpr (!INST) {
            // Clip weight of each staged row: C[k / T].  The host sends only
            // T >= 64 here, so the 64 rows of a stage span at most two
            // samples.  A stage past the slice (possibly with no rows at all:
            // B T == 0) reads no C.
            if (!live) {
#pragma unroll
                for (int j = 0; j < NP; ++j) cw[j] = 0.f;
            } else {
                const uint32_t q0 = __builtin_amdgcn_readfirstlane(k0 / (uint32_t)nT);
                const uint32_t split = (q0 + 1u) * (uint32_t)nT - k0;
                const float c0 = Cs[min(q0, (uint32_t)args.B - 1u)];
                const float c1 = Cs[min(q0 + 1u, (uint32_t)args.B - 1u)];
#pragma unroll
                for (int j = 0; j < NP; ++j) cw[j] = ((uint32_t)(kb + RPP * j) < split) ? c0 : c1;
            }
        }
    };
    // Stage st from one register set; then that set's loads of stage st + 2.
    auto stage = [&](uint4 (&va)[8], uint4 (&vb)[NP], float (&cw)[NP], uint32_t st) {
        lds_barrier();
#pragma unroll
        for (int j = 0; j < 8; ++j)
            *reinterpret_cast<uint4*>(ldsA + (ka + 8 * j) * kSA + ca * 2) = va[j];
#pragma unroll
        for (int j = 0; j < NP; ++j) {
            uint4 v = vb[j];
            if constexpr (!INST)
                v = make_uint4(scale_bf16x2(v.x, cw[j]), scale_bf16x2(v.y, cw[j]), scale_bf16x2(v.z, cw[j]),
                               scale_bf16x2(v.w, cw[j]));
            *reinterpret_cast<uint4*>(ldsB + (kb + RPP * j) * kNSY + cb * 2) = v;
        }
        lds_barrier();
        fetch(va, vb, cw, st + 2);
        uint4 fa[2][2], fb[2][NY];
#pragma unroll
        for (int x = 0; x < 2; ++x) fa[0][x] = frag_tr<kSA>(ldsA, 0, 64 * wave + 32 * x, lane);
#pragma unroll
        for (int y = 0; y < NY; ++y) fb[0][y] = frag_tr<kNSY>(ldsB, 0, 32 * y, lane);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int cur = kk & 1, nxt = cur ^ 1;
            if (kk + 1 < kBK / 16) {
#pragma unroll
                for (int x = 0; x < 2; ++x) fa[nxt][x] = frag_tr<kSA>(ldsA, 16 * (kk + 1), 64 * wave + 32 * x, lane);
#pragma unroll
                for (int y = 0; y < NY; ++y) fb[nxt][y] = frag_tr<kNSY>(ldsB, 16 * (kk + 1), 32 * y, lane);
            }
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < NY; ++y) Mfma<bf16_t>::step(acc[x][y], fa[cur][x], fb[cur][y]);
        }
    };

    fetch(va0, vb0, cw0, st_begin);
    fetch(va1, vb1, cw1, st_begin + 1);
    for (uint32_t st = st_begin; st < nst; st += 2) {
        stage(va0, vb0, cw0, st);
        stage(va1, vb1, cw1, st + 1);    // zeros when st + 1 == nst
    }

    // Element (m, n) of the tile is G[m][n], or G[n][m] when swapped.
    const int r0 = 64 * wave;
    if (ks > 1) {
        float* P = args.tiles + L.ptile_off + (((size_t)sample * tiles + tile) * ks + slice) * (kNM * BN);
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < NY; ++y) {
                const int n = 32 * y + (lane & 31);
#pragma unroll
                for (int i = 0; i < 16; ++i) P[(r0 + 32 * x + acc_row(i, lane)) * BN + n] = acc[x][y][i];
            }
        return;
    }
    float* out = INST ? (L.G ? L.G + (size_t)sample * d * p : nullptr) : L.G;
    if constexpr (INST) {
        float s = 0.f;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < NY; ++y) {
                const bool col_ok = n0 + 32 * y + (lane & 31) < Nd;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const bool ok = col_ok && (m0 + r0 + 32 * x + acc_row(i, lane) < Md);
                    s += ok ? acc[x][y][i] * acc[x][y][i] : 0.f;
                }
            }
        const float tot = block_sum_256(s, red);
        if (tid == 0) args.part[(size_t)L.part_off + (size_t)sample * tiles + tile] = tot;
    }
    if (out) {
        const bool add = !INST && L.accum != 0;
        const size_t sm = sw ? 1 : (size_t)p, sn = sw ? (size_t)p : 1;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < NY; ++y) {
                const int n = n0 + 32 * y + (lane & 31);
                if (n < Nd) put_col16(out, sm, sn, m0 + r0 + 32 * x, Md, n, lane, acc[x][y], 1.f, add);
            }
    }
}

// ---------------------------------------------------------------------------
// Clipped-gradient kernel for 16-byte aligned bf16 rows: one 256 x 256 output
// tile per 512-thread workgroup, one workgroup per CU.  Compared with two
// 256 x 128 workgroups on a CU, a stage moves a third fewer bytes from L2 per
// MFMA.  Waves (wm, wn), wm in 0..1, wn in 0..3, own 128 x 64 sub-tiles (4 x 2
// MFMA 32x32x16 accumulators), read with the same LDS transpose reads.
//
// Two LDS buffers: while the waves multiply stage s out of one buffer, the
// registers holding stage s + 1 (loaded during stage s - 1) are written to the
// other one, and the loads of stage s + 2 are issued.  One barrier per stage.
// The instruction order inside a stage is fixed by hand (sched_barrier
// fences): left to itself the compiler clusters the 48 transpose reads, the
// LDS stores and the global loads into blocks, and the in-order issue of each
// wave then leaves the MFMA pipe idle.  Only launched for T >= 64.
// ---------------------------------------------------------------------------
constexpr int kGM = kGradM, kGN = kGradN;
constexpr int kSG = 256 * 2 + 64;                // bytes per staged k-row (both operands)
constexpr int kGOp = kBK * kSG;                  // one operand of one stage
constexpr int kGStage = 2 * kGOp;

__global__ __launch_bounds__(512, 1) void agrad_bf16_kernel(const GemmArgs args, int n_remap) {
    __shared__ __attribute__((aligned(16))) char lds[2 * kGStage];

    // As agrad_dl_kernel: the first n_remap workgroups XCD-remapped, the
    // tail of K slices in launch order.
    const int wg = (int)blockIdx.x < n_remap ? xcd_remap(blockIdx.x, n_remap) : (int)blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GemmLayer& L = args.L[l];
    const int nT = L.T, d = L.d, p = L.p, tn = L.tn;
    const int local = wg - L.wg_begin, sf = L.split_from;
    const int ks = local < sf ? 1 : max(L.ksplit, 1);
    const int rel = local < sf ? 0 : (local - sf) / ks;              // split tile, from split_from
    const int tile = local < sf ? local : sf + rel;
    const int slice = local < sf ? 0 : (local - sf) - rel * ks;
    const int mt = tile / tn, nt = tile - mt * tn;
    const int m0 = mt * kGM, n0 = nt * kGN;

    // The host guarantees (nrows + 3 kBK) * row bytes < 2^31 for this kernel
    // (its registers leave no room to rebase the rows stage by stage).
    const uint32_t nrows = (uint32_t)args.B * (uint32_t)nT;
    const uint32_t rowA = (uint32_t)d * 2u, rowB = (uint32_t)p * 2u;
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(L.a, nrows * rowA);
    const __amdgpu_buffer_rsrc_t rB = make_rsrc(L.g, nrows * rowB);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;
    // Staging: each operand tile is 64 rows x 32 chunks of 16 B; thread t
    // moves chunk t % 32 of rows t / 32 + 16 j, j = 0..3.  Rows past the last
    // one fall outside the buffer resource and load as zeros, and so do
    // chunks past the last column (out-of-range offset).
    const int cc = (tid & 31) * 8, kr = tid >> 5;
    const uint32_t offA = (m0 + cc < d) ? (uint32_t)kr * rowA + (uint32_t)(m0 + cc) * 2u : kOut;
    const uint32_t offB = (n0 + cc < p) ? (uint32_t)kr * rowB + (uint32_t)(n0 + cc) * 2u : kOut;

    f32x16_t acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    // Register staging of one stage (rows [k0, k0 + 64)): chunk j of a (va)
    // and of g (vb) for rows kr + 16 j.  Rows at or past nrows load zeros, so
    // the stages after the last one need no branch.  The host launches this
    // kernel only for T >= 64, so the 64 rows span at most two samples: the
    // first `split` rows belong to sample fq, the rest to fq + 1, with clip
    // weights c0 and c1 (loaded through the vector memory path: a scalar load
    // would make the waits for it drain the LDS reads as well).
    const __amdgpu_buffer_rsrc_t rC = make_rsrc(args.C, (uint32_t)args.B * 4u);
    uint4 va[4], vb[4];
    float c0 = 0.f, c1 = 0.f;
    uint32_t split = 0;
    // This workgroup's stages (K slice `slice` of `ks`).
    const uint32_t nst_all = (nrows + kBK - 1) / kBK;
    const uint32_t st_begin = (uint32_t)((uint64_t)slice * nst_all / (uint32_t)ks);
    const uint32_t st_end = (uint32_t)((uint64_t)(slice + 1) * nst_all / (uint32_t)ks);
    // next fetch: first row, its sample, row in sample
    uint32_t fk0 = st_begin * kBK, fq = fk0 / (uint32_t)nT, frem = fk0 - fq * (uint32_t)nT;
    auto load_a = [&](int j) { va[j] = buffer_load16(rA, offA == kOut ? kOut : offA + (fk0 + 16u * j) * rowA); };
    auto load_b = [&](int j) { vb[j] = buffer_load16(rB, offB == kOut ? kOut : offB + (fk0 + 16u * j) * rowB); };
    auto load_c = [&]() {
        // Samples past B read zeros (their rows are zero too).
        c0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rC, fq * 4u, 0, 0));
        c1 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rC, fq * 4u + 4u, 0, 0));
        split = (uint32_t)nT - frem;
        fk0 += kBK;
        frem += kBK;
        if (frem >= (uint32_t)nT) {
            frem -= (uint32_t)nT;
            ++fq;
        }
    };
    auto store_a = [&](char* A, int j) {
        *reinterpret_cast<uint4*>(A + (kr + 16 * j) * kSG + cc * 2) = va[j];
    };
    auto store_b = [&](char* Bt, int j) {
        const float cw = ((uint32_t)(kr + 16 * j) < split) ? c0 : c1;
        const uint4 v = vb[j];
        *reinterpret_cast<uint4*>(Bt + (kr + 16 * j) * kSG + cc * 2) =
            make_uint4(scale_bf16x2(v.x, cw), scale_bf16x2(v.y, cw), scale_bf16x2(v.z, cw),
                       scale_bf16x2(v.w, cw));
    };

    // One stage out of buffer BUF (a compile-time constant).  The issue order
    // is laid out by hand, one slot per MFMA, each slot fenced off from the
    // next: slot i of step kk issues MFMA (x, y) = (i / 2, i % 2) of step kk
    // and its share of the 12 transpose reads of the next step: an even slot
    // one half of a g fragment (double-buffered), an odd slot both halves of
    // a fragment x, whose two MFMAs of this step have then been issued (one
    // buffer).  In step 0, slot i also writes register chunk i of stage
    // st + 1 to the other LDS buffer and reloads that register with stage
    // st + 2.
    //
    // The barrier sits between steps 2 and 3: the reads of step 3 were issued
    // (and are waited for) before it, so every read of this buffer is done
    // before the next stage overwrites it, and the stage st + 1 data written
    // in step 0 is complete after it, so step 3 reads the first fragments of
    // stage st + 1 and the next stage starts with MFMAs.  (After the last
    // stage the writes and reads go to a buffer nobody uses.)
    uint2 fa[4][2], fb[2][2][2];
    auto read_a = [&](const char* A, int kk, int x, int h) {
        fa[x][h] = frag_tr_half<kSG>(A, 16 * kk, 128 * wm + 32 * x, lane, h);
    };
    auto read_b = [&](const char* Bt, int kk, int y, int h) {
        fb[kk & 1][y][h] = frag_tr_half<kSG>(Bt, 16 * kk, 64 * wn + 32 * y, lane, h);
    };
    auto stage = [&](auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const char* A = lds + BUF * kGStage;
        const char* Bt = A + kGOp;
        char* An = lds + (BUF ^ 1) * kGStage;
        char* Bn = An + kGOp;
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int cur = kk & 1;
            // Source of the reads in this step: step kk + 1 of this stage, or
            // step 0 of the next one.
            const char* RA = kk + 1 < kBK / 16 ? A : An;
            const char* RB = kk + 1 < kBK / 16 ? Bt : Bn;
            const int rk = (kk + 1) & 3;
            if (kk == kBK / 16 - 1) lds_barrier();
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int x = i >> 1, y = i & 1;
                const uint2 al = fa[x][0], ah = fa[x][1], bl = fb[cur][y][0], bh = fb[cur][y][1];
                Mfma<bf16_t>::step(acc[x][y], make_uint4(al.x, al.y, ah.x, ah.y), make_uint4(bl.x, bl.y, bh.x, bh.y));
                if (i & 1) {
                    read_a(RA, rk, x, 0);
                    read_a(RA, rk, x, 1);
                } else {
                    read_b(RB, rk, i >> 2, (i >> 1) & 1);
                }
                if (kk == 0) {
                    if (i < 4) {
                        store_a(An, i);
                        load_a(i);
                    } else {
                        store_b(Bn, i - 4);
                        load_b(i - 4);
                        if (i == 7) load_c();
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    const uint32_t nst = st_end - st_begin;
    if (nst > 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            load_a(j);
            load_b(j);
        }
        load_c();
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            store_a(lds, j);
            store_b(lds + kGOp, j);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            load_a(j);
            load_b(j);
        }
        load_c();
    }
    lds_barrier();
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        read_a(lds, 0, x, 0);
        read_a(lds, 0, x, 1);
    }
#pragma unroll
    for (int y = 0; y < 2; ++y) {
        read_b(lds + kGOp, 0, y, 0);
        read_b(lds + kGOp, 0, y, 1);
    }
    uint32_t st = 0;
    for (; st + 1 < nst; st += 2) {
        stage(std::integral_constant<int, 0>{});
        stage(std::integral_constant<int, 1>{});
    }
    if (st < nst) stage(std::integral_constant<int, 0>{});

    if (ks > 1) {
        store_partial_tile<kGM, kGN>(args.tiles + L.ptile_off + ((size_t)rel * ks + slice) * (kGM * kGN),
                                     acc, 128 * wm, 64 * wn, lane, 1.f);
        return;
    }
    float* G = L.G;
    const bool add = L.accum != 0;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int n = n0 + 64 * wn + 32 * y + (lane & 31);
            if (n < p) put_col16(G, (size_t)p, 1, m0 + 128 * wm + 32 * x, d, n, lane, acc[x][y], 1.f, add);
        }
}

constexpr int kDRow = 512;                       // bytes per staged k-row
constexpr int kDKS = kDLStageRows;               // k rows per stage
constexpr int kDNB = kDLBuffers;                 // LDS stage buffers
static_assert(kDKS == 32 || kDKS == 64, "stage rows");
static_assert(kDNB >= 2 && kDNB * 2 * kDKS * kDRow <= 128 * 1024, "LDS ring");

__device__ __forceinline__ int dswz(int row, int c16) { return c16 ^ (4 * (row & 3)); }

// Half h of a transposed fragment (as frag_tr_half) from the swizzled layout.
__device__ __forceinline__ uint2 frag_dl_half(const char* lds, int kb, int cb, int lane, int h) {
    const int grp = lane >> 4, i = lane & 15;
    const int row = kb + 8 * (grp >> 1) + (i >> 2) + 4 * h;
    const int col = cb + 16 * (grp & 1) + 4 * (i & 3);
    return lds_tr16(lds + row * kDRow + dswz(row, col >> 3) * 16 + (col & 7) * 2);
}

// Position of a stage in the batch: its sample and its stage within the
// sample (spt stages per sample), advanced one stage at a time.
struct StagePos {
    uint32_t smp, in;
    __device__ __forceinline__ void next(uint32_t spt) {
        const bool wrap = in + 1u == spt;
        in = wrap ? 0u : in + 1u;
        smp += wrap ? 1u : 0u;
    }
};

// ---------------------------------------------------------------------------
// Clipped-gradient kernel for bf16 rows when the stage height KS (32) divides
// T: 256 x 256 tiles on 512 threads, waves of 128 x 64 as in
// agrad_bf16_kernel, but both operand tiles go from HBM straight into LDS
// (LDS DMA: no staging registers, no LDS store instructions) and the clip
// weights are applied to the accumulators instead of to g.  A stage then lies
// inside one sample.  The accumulators hold S / c, S being the weighted sum
// so far and c the weight of the last sample whose weight is nonzero:
// entering sample j with C_j != 0 multiplies them by c / C_j, and the
// epilogue multiplies by the final c.  Rows of samples with C_j = 0 load as
// zeros.  (Products are exact in fp32 and each sample boundary rounds once,
// instead of C_j g being rounded to bf16.)
//
// LDS: a ring of NB = 4 stage buffers (an a stage and a g stage each),
// 512-byte rows without padding (one DMA instruction fills 1 KB
// contiguously); the 16-byte column c of row r sits at c ^ 4 (r mod 4), which
// puts the four rows that each half of a transpose read touches on distinct
// bank groups.  The clip weights of the batch sit in LDS after the ring
// (B <= kDMaxB).
//
// Schedule (ping-pong): waves w and w + 4 share a SIMD.  Each stage is a
// memory phase (all 24 transpose reads of the wave's fragments, the rescale
// on entering a sample, the wait for the wave's own DMA of the next stage)
// followed by an MFMA phase (the stage's 16 MFMAs, with the wave's four DMA
// instructions of the stage three ahead among the first eight), and every
// phase ends at a workgroup barrier.  Waves 4-7 run one phase behind waves
// 0-3, so that on every SIMD one wave issues MFMAs while the other reads.
// The buffer refilled during the MFMA phase of stage s, (s + 3) mod 4, was
// last read in the memory phases of stage s - 1, which both halves have
// passed; a stage's buffer is complete once every wave has waited for its
// DMA of it before the barrier that precedes the first reads of it.
//
// INST (per-sample gradient instantiation, App. B.4.1): workgroup = (sample,
// tile), its stages those of the one sample, no weights (every other stage
// loads zeros); the epilogue sums the squares of the tile's d x p entries
// into one norm partial per (sample, tile) and, when L.G is set (BK-MixOpt),
// stores the tile of the sample's gradient into L.G + sample d p.
// ---------------------------------------------------------------------------
constexpr int kDOp = kDKS * kDRow;               // one operand of one stage
constexpr int kDStage = 2 * kDOp;
constexpr int kDKK = kDKS / 16;                  // 16-row MFMA steps per stage
constexpr int kDPW = kDKS / 8;                   // DMA instructions per wave per stage

template <bool INST>
__global__ __launch_bounds__(512, 1) void agrad_dl_kernel(const GemmArgs args, int n_remap) {
    __shared__ __attribute__((aligned(16))) char lds[kDNB * kDStage];
    __shared__ float ctab[INST ? 8 : kDMaxB + 1];   // INST: the epilogue's wave sums

    // The first n_remap workgroups in contiguous runs per XCD; the tail (the
    // K slices of the last round's tiles) in launch order, so that it is
    // dispatched last.
    const int wg = (int)blockIdx.x < n_remap ? xcd_remap(blockIdx.x, n_remap) : (int)blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GemmLayer& L = args.L[l];
    const int nT = L.T, d = L.d, p = L.p, tn = L.tn;
    const int local = wg - L.wg_begin, sf = L.split_from;
    // Clipped gradient: tiles below split_from whole, the others in ksplit
    // slices.  INST: workgroup = sample * tiles + tile, never split.
    const int sample = INST ? local / (L.tm * tn) : 0;
    const int ks = INST || local < sf ? 1 : max(L.ksplit, 1);
    const int rel = INST || local < sf ? 0 : (local - sf) / ks;      // split tile, from split_from
    const int tile = INST ? local - sample * (L.tm * tn) : local < sf ? local : sf + rel;
    const int slice = INST || local < sf ? 0 : (local - sf) - rel * ks;
    const int mt = tile / tn, nt = tile - mt * tn;
    const int m0 = mt * kGM, n0 = nt * kGN;

    // The host guarantees B <= kDMaxB for this kernel.  Each sample takes
    // spt = ceil(T / KS) stages, its last one padded with zero rows (a
    // stage's descriptor ends at its sample's last row: rows_raw_rsrc), and
    // rows are addressed stage by stage.
    const int B = args.B;
    const uint32_t rowA = (uint32_t)d * 2u, rowB = (uint32_t)p * 2u;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2, wn = wave & 3;
    // Clip weights, and a zero for the stages past the batch.
    if constexpr (!INST)
        for (int i = tid; i <= B; i += 512) ctab[i] = i < B ? args.C[i] : 0.f;

    // DMA: each operand stage is KS / 2 instructions of 1 KB (two rows); wave
    // w (of 8) issues numbers j = 8 i + w, i < KS / 16, and lane l moves
    // physical column l % 32 of row 2 j + l / 32, i.e. logical column
    // dswz(row, l % 32).  Columns past the matrix get an out-of-range offset.
    constexpr int NI = kDKS / 16;
    uint32_t offA[NI], offB[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int row = 2 * (8 * i + wave) + (lane >> 5);
        const int lc = dswz(row, lane & 31);
        offA[i] = (m0 + 8 * lc < d) ? (uint32_t)row * rowA + (uint32_t)(m0 + 8 * lc) * 2u : kOut;
        offB[i] = (n0 + 8 * lc < p) ? (uint32_t)row * rowB + (uint32_t)(n0 + 8 * lc) * 2u : kOut;
    }
    // DMA piece i (i < NI: a, else g) of stage `pos` into the buffer at
    // `buf`; `zero` (the stage's sample has weight 0, or lies past the batch)
    // loads zeros.
    auto dma = [&](char* buf, const StagePos& pos, bool zero, int i) {
        const uint32_t s0 = pos.smp * (uint32_t)nT;
        const uint32_t k0 = s0 + pos.in * kDKS, kend = s0 + (uint32_t)nT;
        if (i < NI) {
            const uint32_t o = (offA[i] == kOut || zero) ? kOut : offA[i];
            dma16_asm(rows_raw_rsrc(L.a, rowA, k0, kend, kDKS), o, buf + (8 * i + wave) * 1024);
        } else {
            const int j = i - NI;
            const uint32_t o = (offB[j] == kOut || zero) ? kOut : offB[j];
            dma16_asm(rows_raw_rsrc(L.g, rowB, k0, kend, kDKS), o, buf + kDOp + (8 * j + wave) * 1024);
        }
    };

    f32x16_t acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    const uint32_t spt = ((uint32_t)nT + kDKS - 1) / kDKS;   // stages per sample
    const uint32_t nst_all = (uint32_t)B * spt;
    // The last stage of a sample holds at most 16 rows (16-row MFMA steps,
    // the second one all zeros): its second step is skipped.
    const bool short_last = (uint32_t)nT - (spt - 1) * kDKS <= 16u;
    // This workgroup's stages (K slice `slice` of `ks`; INST: its sample's).
    const uint32_t st_begin = INST ? (uint32_t)sample * spt : (uint32_t)((uint64_t)slice * nst_all / (uint32_t)ks);
    const uint32_t st_end = INST ? (uint32_t)(sample + 1) * spt
                                 : (uint32_t)((uint64_t)(slice + 1) * nst_all / (uint32_t)ks);
    // Weight of the stage at `pos` (0 past the batch; INST: 1 in the sample,
    // 0 elsewhere).
    auto cw_of = [&](const StagePos& pos) {
        if constexpr (INST) return pos.smp == (uint32_t)sample ? 1.f : 0.f;
        else return ctab[min(pos.smp, (uint32_t)B)];
    };

    float c_last = 0.f;   // weight of the last sample with a nonzero weight
    static_assert(kDNB == 4 && kDKK == 2 && kDPW == 4, "ping-pong ring");
    const bool late = wave >= 4;
    uint2 fa[kDKK][4][2], fb[kDKK][2][2];
    StagePos pos0{st_begin / spt, st_begin % spt};        // stage st
    StagePos posD = pos0;                                  // stage st + 3
    __syncthreads();      // clip weights in LDS
    // Prologue: stages st_begin .. st_begin + 2 into buffers 0 .. 2.
#pragma unroll
    for (int b = 0; b < kDNB - 1; ++b) {
        const bool z = cw_of(posD) == 0.f;
#pragma unroll
        for (int i = 0; i < kDPW; ++i) dma(lds + b * kDStage, posD, z, i);
        posD.next(spt);
    }
    wait_vmcnt<(kDNB - 2) * kDPW>();
    lds_barrier();
    if (late) {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
    }
    auto run = [&](auto buf_c, uint32_t st) {
        constexpr int BUF = decltype(buf_c)::value;
        const char* A = lds + BUF * kDStage;
        const char* Bt = A + kDOp;
        char* D = lds + ((BUF + kDNB - 1) % kDNB) * kDStage;
        // Memory phase: the stage's fragments, then (entering a sample, or at
        // the slice's first stage) the accumulators times c_last / c (c != 0).
        const bool two = !(short_last && pos0.in + 1u == spt);   // second step
#pragma unroll
        for (int kk = 0; kk < kDKK; ++kk) {
            if (kk > 0 && !two) break;
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int h = 0; h < 2; ++h) fa[kk][x][h] = frag_dl_half(A, 16 * kk, 128 * wm + 32 * x, lane, h);
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int h = 0; h < 2; ++h) fb[kk][y][h] = frag_dl_half(Bt, 16 * kk, 64 * wn + 32 * y, lane, h);
        }
        if (!INST && (pos0.in == 0u || st == st_begin)) {
            const float c = cw_of(pos0);
            const bool nz = c != 0.f;
            const float r = nz ? c_last / c : 1.f;
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[x][y][e] *= r;
            c_last = nz ? c : c_last;
        }
        const bool zd = cw_of(posD) == 0.f;
        wait_vmcnt<kDPW>();
        __builtin_amdgcn_sched_barrier(0);
        lds_barrier();
        __builtin_amdgcn_sched_barrier(0);
        // MFMA phase.
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kk = 0; kk < kDKK; ++kk) {
            if (kk > 0 && !two) break;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int x = i >> 1, y = i & 1;
                const uint2 al = fa[kk][x][0], ah = fa[kk][x][1], bl = fb[kk][y][0], bh = fb[kk][y][1];
                Mfma<bf16_t>::step(acc[x][y], make_uint4(al.x, al.y, ah.x, ah.y), make_uint4(bl.x, bl.y, bh.x, bh.y));
                if (kk == 0 && (i & 1)) dma(D, posD, zd, i >> 1);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        pos0.next(spt);
        posD.next(spt);
    };
    const uint32_t nst = st_end;
    uint32_t st = st_begin;
    for (; st + kDNB <= nst; st += kDNB) {
        run(std::integral_constant<int, 0>{}, st);
        run(std::integral_constant<int, 1>{}, st + 1);
        run(std::integral_constant<int, 2>{}, st + 2);
        run(std::integral_constant<int, 3>{}, st + 3);
    }
    if (st < nst) run(std::integral_constant<int, 0>{}, st++);
    if (st < nst) run(std::integral_constant<int, 1>{}, st++);
    if (st < nst) run(std::integral_constant<int, 2>{}, st++);
    if (!late) __builtin_amdgcn_s_barrier();
    // Drain the DMA past the end before the workgroup exits.
    wait_vmcnt<0>();

    if constexpr (INST) {
        // Rows and columns past d and p loaded zeros, so their entries are 0.
        float sq = 0.f;
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int e = 0; e < 16; ++e) sq += acc[x][y][e] * acc[x][y][e];
        sq = wave_sum(sq);
        if (lane == 0) ctab[wave] = sq;
        __syncthreads();
        if (tid == 0) {
            float t = 0.f;
#pragma unroll
            for (int w = 0; w < 8; ++w) t += ctab[w];
            args.part[(size_t)L.part_off + (size_t)sample * (L.tm * tn) + tile] = t;
        }
        if (L.G) {   // BK-MixOpt: the sample's gradient a_i^T g_i [d, p]
            float* P = L.G + (size_t)sample * d * p;
            if ((reinterpret_cast<uintptr_t>(P) & 15u) == 0) {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int y = 0; y < 2; ++y)
                        put_acc_x4(P, (size_t)p, m0 + 128 * wm + 32 * x, d, n0 + 64 * wn + 32 * y, p, lane,
                                   acc[x][y], 1.f, false);
            } else {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int y = 0; y < 2; ++y) {
                        const int n = n0 + 64 * wn + 32 * y + (lane & 31);
                        if (n < p) put_col16(P, (size_t)p, 1, m0 + 128 * wm + 32 * x, d, n, lane, acc[x][y], 1.f, false);
                    }
            }
        }
        return;
    }
    if (ks > 1) {
        store_partial_tile<kGM, kGN>(args.tiles + L.ptile_off + ((size_t)rel * ks + slice) * (kGM * kGN),
                                     acc, 128 * wm, 64 * wn, lane, c_last);
        return;
    }
    float* G = L.G;
    const bool add = L.accum != 0;
    // 16-byte stores when G allows them (p is a multiple of 8 here).
    if ((reinterpret_cast<uintptr_t>(G) & 15u) == 0) {
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
                put_acc_x4(G, (size_t)p, m0 + 128 * wm + 32 * x, d, n0 + 64 * wn + 32 * y, p, lane, acc[x][y], c_last,
                           add);
        return;
    }
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int n = n0 + 64 * wn + 32 * y + (lane & 31);
            if (n < p) put_col16(G, (size_t)p, 1, m0 + 128 * wm + 32 * x, d, n, lane, acc[x][y], c_last, add);
        }
}

// Sum of the K slices of split layers, slice 0 first.  Workgroup -> layer by
// red_begin; inside a layer, tile group (sample * tiles + tile for the
// instantiated norm, tile - split_from otherwise) and one kSplitRedWG-element
// chunk of it.
// Clipped gradient: the sum goes to G.  Instantiated norm: its squares (of
// elements inside the matrix) are summed into one norm partial per chunk,
// and with G set (BK-MixOpt) the sum is also kept in G [B,d,p].
template <int TM, int TN, bool INST>
__global__ __launch_bounds__(256) void split_reduce_kernel(const GemmArgs args) {
    __shared__ float red[4];
    constexpr int CH = TM * TN / kSplitRedWG;
    const int wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].red_begin; });
    const GemmLayer& L = args.L[l];
    const int job = wg - L.red_begin;
    const int tg = job / CH, ch = job - tg * CH;
    const int tiles = L.tm * L.tn;
    const int sample = INST ? tg / tiles : 0;
    const int tile = tg - sample * tiles + L.split_from;
    const int mt = tile / L.tn, nt = tile - mt * L.tn;
    const int e = ch * kSplitRedWG + 4 * (int)threadIdx.x;
    const int m = mt * TM + e / TN, n = nt * TN + e % TN;
    const int ks = max(L.ksplit, 1);
    const float* src = args.tiles + L.ptile_off + (size_t)tg * ks * (TM * TN) + e;
    // Slices in batches of 8 loads issued together, added in slice order.
    float4 sum = *reinterpret_cast<const float4*>(src);
    for (int q0 = 1; q0 < ks; q0 += 8) {
        float4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (q0 + j < ks) v[j] = *reinterpret_cast<const float4*>(src + (size_t)(q0 + j) * (TM * TN));
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (q0 + j < ks) {
                sum.x += v[j].x;
                sum.y += v[j].y;
                sum.z += v[j].z;
                sum.w += v[j].w;
            }
    }
    const float r[4] = {sum.x, sum.y, sum.z, sum.w};
    // Tile rows run along d, or along p for a swapped (narrow) layer.
    const bool sw = L.swap != 0;
    const int Md = sw ? L.p : L.d, Nd = sw ? L.d : L.p;
    const bool row_ok = m < Md;
    float* out = L.G ? L.G + (size_t)sample * L.d * L.p : nullptr;
    if constexpr (INST) {
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) sq += (row_ok && n + j < Nd) ? r[j] * r[j] : 0.f;
        const float tot = block_sum_256(sq, red);
        if (threadIdx.x == 0) args.part[(size_t)L.part_off + (size_t)tg * CH + ch] = tot;
    }
    if (out && row_ok) {
        const bool add = !INST && L.accum != 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (n + j < Nd) {
                float* q = out + (sw ? (size_t)(n + j) * L.p + m : (size_t)m * L.p + n + j);
                *q = add ? *q + r[j] : r[j];
            }
    }
}

}  // namespace

hipError_t launch_split_reduce(const GemmArgs& args, int n_wg, bool inst_norm, GemmVariant v,
                               hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    const dim3 grid(n_wg), block(256);
    if (inst_norm && v == GemmVariant::Wide)
        hipLaunchKernelGGL((split_reduce_kernel<kBM, kBN, true>), grid, block, 0, s, args);
    else if (!inst_norm && (v == GemmVariant::Grad || v == GemmVariant::GradDL))
        hipLaunchKernelGGL((split_reduce_kernel<kGM, kGN, false>), grid, block, 0, s, args);
    else if (v == GemmVariant::Narrow32) {
        if (inst_norm) hipLaunchKernelGGL((split_reduce_kernel<kNM, 32, true>), grid, block, 0, s, args);
        else hipLaunchKernelGGL((split_reduce_kernel<kNM, 32, false>), grid, block, 0, s, args);
    } else if (v == GemmVariant::Narrow64) {
        if (inst_norm) hipLaunchKernelGGL((split_reduce_kernel<kNM, 64, true>), grid, block, 0, s, args);
        else hipLaunchKernelGGL((split_reduce_kernel<kNM, 64, false>), grid, block, 0, s, args);
    } else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& args, int n_wg, bool bf16, bool inst_norm, GemmVariant v,
                       hipStream_t s, int n_remap) {
    if (n_wg <= 0) return hipSuccess;
    const dim3 grid(n_wg), block(256);
    const bool vec = v != GemmVariant::Scalar;
    if (v == GemmVariant::Grad) {
        if (inst_norm) return hipErrorInvalidValue;
        const int nr = n_remap > 0 && n_remap < n_wg ? n_remap : n_wg;
        hipLaunchKernelGGL(agrad_bf16_kernel, grid, dim3(512), 0, s, args, nr);
        return hipGetLastError();
    }
    if (v == GemmVariant::GradDL) {
        const int nr = n_remap > 0 && n_remap < n_wg ? n_remap : n_wg;
        if (inst_norm) hipLaunchKernelGGL(agrad_dl_kernel<true>, grid, dim3(512), 0, s, args, nr);
        else hipLaunchKernelGGL(agrad_dl_kernel<false>, grid, dim3(512), 0, s, args, nr);
        return hipGetLastError();
    }
    if (v == GemmVariant::Wide) {
        if (inst_norm) hipLaunchKernelGGL(agemm_bf16_kernel<true>, grid, block, 0, s, args, n_wg);
        else hipLaunchKernelGGL(agemm_bf16_kernel<false>, grid, block, 0, s, args, n_wg);
        return hipGetLastError();
    }
    if (v == GemmVariant::Narrow32) {
        if (inst_norm) hipLaunchKernelGGL((anarrow_kernel<true, 32>), grid, block, 0, s, args, n_wg);
        else hipLaunchKernelGGL((anarrow_kernel<false, 32>), grid, block, 0, s, args, n_wg);
        return hipGetLastError();
    }
    if (v == GemmVariant::Narrow64) {
        if (inst_norm) hipLaunchKernelGGL((anarrow_kernel<true, 64>), grid, block, 0, s, args, n_wg);
        else hipLaunchKernelGGL((anarrow_kernel<false, 64>), grid, block, 0, s, args, n_wg);
        return hipGetLastError();
    }
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
