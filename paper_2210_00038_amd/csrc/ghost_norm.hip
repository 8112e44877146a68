// Ghost norm of linear and embedding layers (eq. "ghost norm", Section 2.1;
// App. B.4):
//
//   n_i = vec(g_i g_i^T) . vec(a_i a_i^T) = sum_{t,t'} (a_i a_i^T)_{tt'} (g_i g_i^T)_{tt'}
//
// For an embedding a_i = one_hot(x_i), so (a_i a_i^T)_{tt'} = [x_it == x_it'].
//
// Work decomposition.  The T x T Grams of sample i are cut into 128 x 128
// super blocks; only the upper triangle of super-block pairs (R <= C) is
// visited and off-diagonal pairs count twice (both Grams are symmetric).  One
// 256-thread workgroup owns one (layer, sample, R, C): it streams rows
// [128R, 128R+128) and [128C, 128C+128) of a_i through LDS in 128-byte column
// chunks and accumulates its part of a_i a_i^T with 32x32 MFMA tiles, then does
// the same for g_i, and finally multiplies the two accumulators elementwise
// and reduces.  The Grams never leave the registers.  Inside a diagonal super
// block only the 10 upper 32x32 sub-tiles count (diagonal ones weight 1,
// others 2); sub-tiles made only of padding rows (t >= T) get weight 0.  A
// wave multiplies all four of its sub-tiles whatever their weights (a branch
// around each MFMA costs more than the MFMA), except that a wave with no
// weighted sub-tile skips its MFMAs.  Each workgroup writes one partial sum;
// a fixed-order reduction finishes the norm.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kRowU4 = 9;                    // LDS row: 128 data bytes + 16 pad, in uint4
constexpr uint32_t kGhostOut = 0xFFFFFFF0u;  // buffer offset that loads zeros
constexpr int kBlockU4 = kSuper * kRowU4;    // one staged super block

struct WaveTiles {
    int r0, c0;   // first 32-row sub-block of the rows (block R) / columns (block C)
    int w[4];     // weight of sub-tile (r0 + x, c0 + y) at index 2x + y; 0 = skip
};

__device__ __forceinline__ WaveTiles wave_tiles(int wave, bool diag) {
    WaveTiles t;
    if (!diag) {
        t.r0 = 2 * (wave >> 1);
        t.c0 = 2 * (wave & 1);
        t.w[0] = t.w[1] = t.w[2] = t.w[3] = 2;
        return t;
    }
    // Upper triangle of the 4 x 4 sub-tiles of a diagonal super block:
    // wave 0: (0,0) (0,1) (1,1); wave 1: (2,2) (2,3) (3,3);
    // wave 2: (0,2) (0,3) (1,2) (1,3); wave 3: none.
    switch (wave) {
        case 0: t.r0 = 0; t.c0 = 0; t.w[0] = 1; t.w[1] = 2; t.w[2] = 0; t.w[3] = 1; break;
        case 1: t.r0 = 2; t.c0 = 2; t.w[0] = 1; t.w[1] = 2; t.w[2] = 0; t.w[3] = 1; break;
        case 2: t.r0 = 0; t.c0 = 2; t.w[0] = 2; t.w[1] = 2; t.w[2] = 2; t.w[3] = 2; break;
        default: t.r0 = 0; t.c0 = 2; t.w[0] = 0; t.w[1] = 0; t.w[2] = 0; t.w[3] = 0; break;
    }
    return t;
}

// 16 bytes of row r, starting at column k, of a [rows, K] matrix; zero outside.
template <typename T, bool VEC>
__device__ __forceinline__ uint4 load16(const T* X, int rows, int K, int r, int k) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (r >= rows) return v;
    const T* p = X + (size_t)r * (size_t)K + k;
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

// Accumulate this wave's sub-tiles of X X^T, X = one sample's [rows, K] matrix,
// rows of block R starting at rowR and of block C at rowC.
template <typename T, bool VEC>
__device__ __forceinline__ void gram(const T* __restrict__ X, int rows, int K, int rowR, int rowC,
                                     bool diag, const WaveTiles& wt, f32x16_t acc[4],
                                     uint4* __restrict__ lds) {
    constexpr int EPV = Elem<T>::per16;       // elements per 16 bytes
    constexpr int EPC = 8 * EPV;              // elements per 128-byte chunk
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[s][i] = 0.f;

    const int tid = threadIdx.x, lane = tid & 63;
    const int c16 = tid & 7, rq = tid >> 3;
    const int r = lane & 31, h = lane >> 5;
    uint4* ldsR = lds;
    uint4* ldsC = diag ? lds : lds + kBlockU4;
    const int nch = (K + EPC - 1) / EPC;

    uint4 pr[8];
    auto fetch = [&](int ch) {
        const int k = ch * EPC + c16 * EPV;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            pr[q] = load16<T, VEC>(X, rows, K, rowR + rq + 32 * q, k);
            if (!diag) pr[4 + q] = load16<T, VEC>(X, rows, K, rowC + rq + 32 * q, k);
        }
    };
    fetch(0);
    for (int ch = 0; ch < nch; ++ch) {
        lds_barrier();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            ldsR[(rq + 32 * q) * kRowU4 + c16] = pr[q];
            if (!diag) ldsC[(rq + 32 * q) * kRowU4 + c16] = pr[4 + q];
        }
        lds_barrier();
        if (ch + 1 < nch) fetch(ch + 1);
        if ((wt.w[0] | wt.w[1] | wt.w[2] | wt.w[3]) == 0) continue;   // wave-uniform
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = 2 * j + h;
            const uint4 x0 = ldsR[((wt.r0 + 0) * 32 + r) * kRowU4 + col];
            const uint4 x1 = ldsR[((wt.r0 + 1) * 32 + r) * kRowU4 + col];
            const uint4 y0 = ldsC[((wt.c0 + 0) * 32 + r) * kRowU4 + col];
            const uint4 y1 = ldsC[((wt.c0 + 1) * 32 + r) * kRowU4 + col];
            // All four sub-tiles, also those of weight 0 (their rows are real
            // or zero padding, so the product is finite and gets weight 0):
            // a branch per MFMA costs more than the MFMA.
            Mfma<T>::step(acc[0], x0, y0);
            Mfma<T>::step(acc[1], x0, y1);
            Mfma<T>::step(acc[2], x1, y0);
            Mfma<T>::step(acc[3], x1, y1);
        }
    }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS variant of gram() for 16-byte aligned rows (VEC).  The chunks
// go from global memory straight into a ring of four 16 KB LDS slots (one
// 128-row x 128-byte block each; a diagonal pair needs one slot per chunk, an
// off-diagonal pair two), with no staging registers, so up to three chunks per
// workgroup are in flight.  A 1 KB load instruction fills 8 consecutive
// 128-byte rows, so rows cannot be padded; instead the 16-byte column c of row
// r is stored at column c ^ ((r >> 1) & 7), which spreads the 16 rows read by
// 16 lanes of a fragment load over all 64 banks.
// ---------------------------------------------------------------------------
constexpr int kRingBytes = 64 * 1024;        // LDS ring of gram_dl
#ifndef BK_GHOST_DIAG_CW
#define BK_GHOST_DIAG_CW 128
#endif
#ifndef BK_GHOST_OFF_CW
#define BK_GHOST_OFF_CW 128
#endif

// CW: bytes of each row per chunk (64, 128 or 256).  A slot holds one
// 128-row block of a chunk; the ring holds kRingBytes / (128 CW) slots.
// Column c of row r sits at column c ^ (r / 4 mod 4) (CW = 64: a 256-byte
// bank line holds four rows), c ^ (r / 2 mod 8) (CW = 128) or c ^ (r mod 16)
// (CW = 256), so that the 16 rows read by 16 lanes land on distinct 16-byte
// bank groups.
// Column sums (DIAG with a single 128-row block, i.e. T <= 128): with cs set,
// each chunk's columns are also summed over the block's rows from LDS, cs[k] =
// sum_t X[t, k] is written and bsq accumulates cs[k]^2 (threads that finish
// columns).  Thread t sums 16-byte column t % C16 over every (256 / C16)-th
// row; lanes of a wave holding the same column are added by shuffles, the
// four waves through cbuf (two 4 x 128-float halves, by chunk parity), in a
// fixed order.
template <typename T, bool DIAG, int CW>
__device__ __forceinline__ void gram_dl(const T* __restrict__ X, int rows, int K, int rowR, int rowC,
                                        const WaveTiles& wt, f32x16_t acc[4], char* __restrict__ lds,
                                        float* __restrict__ cs = nullptr, float* bsq = nullptr,
                                        float* cbuf = nullptr) {
    static_assert(CW == 64 || CW == 128 || CW == 256, "chunk width");
    constexpr int EPV = Elem<T>::per16;       // elements per 16 bytes
    constexpr int C16 = CW / 16;              // 16-byte columns per row and chunk
    constexpr int EPC = C16 * EPV;            // elements per row and chunk
    constexpr int SLOT = kSuper * CW;         // bytes of one block of one chunk
    constexpr int NSLOT = kRingBytes / SLOT;
    constexpr int SPC = DIAG ? 1 : 2;         // slots per chunk
    constexpr int NCH = NSLOT / SPC;          // chunks held by the ring
    static_assert(NCH >= 2, "ring too small");
    constexpr int RPL = 64 / C16;             // rows filled by one 1 KB load
    constexpr int LPB = kSuper / RPL / 4;     // loads per wave per block
    constexpr int LPW = LPB * SPC;            // loads per wave per chunk
    auto swz = [](int row, int c) {
        return C16 == 4 ? c ^ ((row >> 2) & 3) : C16 == 8 ? c ^ ((row >> 1) & 7) : c ^ (row & 15);
    };
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[s][i] = 0.f;

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int nch = (K + EPC - 1) / EPC;
    const uint32_t rowbytes = (uint32_t)K * (uint32_t)sizeof(T);
    // The host guarantees (rows + 128) * rowbytes < 2^31 for this path.
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(X, (uint32_t)rows * rowbytes);

    // Load i of this wave for one block fills rows RPL (4 i + wave) + 0..RPL-1
    // of the slot; lane l writes 16-byte column l % C16 of row l / C16, which
    // holds column swz(row, l % C16) of the chunk.
    uint32_t roff[LPB];
    int lcol[LPB];
#pragma unroll
    for (int i = 0; i < LPB; ++i) {
        const int rl = RPL * (4 * i + wave) + lane / C16;
        lcol[i] = swz(rl, lane % C16);
        roff[i] = (uint32_t)rl * rowbytes + (uint32_t)(lcol[i] * EPV) * (uint32_t)sizeof(T);
    }
    // Chunks at or past nch load zeros (all offsets out of range), so every
    // iteration issues the same number of loads.
    auto issue = [&](int ch) {
        char* slot = lds + ((ch % NCH) * SPC) * SLOT;
#pragma unroll
        for (int b = 0; b < SPC; ++b) {
            const uint32_t base = (uint32_t)(b == 0 ? rowR : rowC) * rowbytes +
                                  (uint32_t)(ch * EPC) * (uint32_t)sizeof(T);
#pragma unroll
            for (int i = 0; i < LPB; ++i) {
                const bool ok = ch * EPC + lcol[i] * EPV < K;
                buffer_load16_lds(rs, ok ? base + roff[i] : kGhostOut, slot + b * SLOT + (4 * i + wave) * 1024);
            }
        }
    };
    const bool active = (wt.w[0] | wt.w[1] | wt.w[2] | wt.w[3]) != 0;   // wave-uniform
    auto compute = [&](int ch) {
        if (!active) return;
        const char* sR = lds + ((ch % NCH) * SPC) * SLOT;
        const char* sC = DIAG ? sR : sR + SLOT;
#pragma unroll
        for (int j = 0; j < C16 / 2; ++j) {
            const int col = 2 * j + h;
            const int ra0 = (wt.r0 + 0) * 32 + r, ra1 = (wt.r0 + 1) * 32 + r;
            const int rc0 = (wt.c0 + 0) * 32 + r, rc1 = (wt.c0 + 1) * 32 + r;
            const uint4 x0 = *reinterpret_cast<const uint4*>(sR + ra0 * CW + swz(ra0, col) * 16);
            const uint4 x1 = *reinterpret_cast<const uint4*>(sR + ra1 * CW + swz(ra1, col) * 16);
            const uint4 y0 = *reinterpret_cast<const uint4*>(sC + rc0 * CW + swz(rc0, col) * 16);
            const uint4 y1 = *reinterpret_cast<const uint4*>(sC + rc1 * CW + swz(rc1, col) * 16);
            // All four sub-tiles, also those of weight 0 (their rows are real
            // or zero padding, so the product is finite and gets weight 0):
            // a branch per MFMA costs more than the MFMA.
            Mfma<T>::step(acc[0], x0, y0);
            Mfma<T>::step(acc[1], x0, y1);
            Mfma<T>::step(acc[2], x1, y0);
            Mfma<T>::step(acc[3], x1, y1);
        }
    };

    // Column sums of chunk ch into cbuf, and their completion (after the
    // next barrier) into cs / bsq.
    constexpr int RPP = 256 / C16;            // rows apart of one thread's reads
    auto colsum = [&](int ch) {
        const char* sR = lds + ((ch % NCH) * SPC) * SLOT;
        const int j = tid % C16;
        float c[EPV];
#pragma unroll
        for (int e = 0; e < EPV; ++e) c[e] = 0.f;
#pragma unroll
        for (int q = 0; q < kSuper / RPP; ++q) {
            const int row = tid / C16 + RPP * q;
            const uint4 v = *reinterpret_cast<const uint4*>(sR + row * CW + swz(row, j) * 16);
            if constexpr (sizeof(T) == 2) {
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    c[2 * e] += __uint_as_float(w[e] << 16);
                    c[2 * e + 1] += __uint_as_float(w[e] & 0xFFFF0000u);
                }
            } else {
                c[0] += __uint_as_float(v.x);
                c[1] += __uint_as_float(v.y);
                c[2] += __uint_as_float(v.z);
                c[3] += __uint_as_float(v.w);
            }
        }
        // lanes j, j + C16, ... of the wave hold the same columns
#pragma unroll
        for (int off = C16; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < EPV; ++e) c[e] += __shfl_xor(c[e], off, 64);
        if (lane < C16) {
#pragma unroll
            for (int e = 0; e < EPV; ++e) cbuf[(ch & 1) * 512 + wave * 128 + j * EPV + e] = c[e];
        }
    };
    auto colsum_done = [&](int ch) {
        if (tid < EPC) {
            const float* cb = cbuf + (ch & 1) * 512 + tid;
            const float v = ((cb[0] + cb[128]) + cb[256]) + cb[384];
            const int k = ch * EPC + tid;
            if (k < K) {
                cs[k] = v;
                *bsq += v * v;
            }
        }
    };

    // Chunk ch: wait for this wave's loads of it (the NCH - 2 later chunks may
    // stay in flight), barrier (everyone's loads of it have landed, and every
    // wave is done with chunk ch - 1), refill chunk ch - 1's slot with chunk
    // ch + NCH - 1, multiply chunk ch.
#pragma unroll
    for (int c = 0; c < NCH - 1; ++c) issue(c);
    for (int ch = 0; ch < nch; ++ch) {
        wait_vmcnt<LPW * (NCH - 2)>();
        lds_barrier();
        if constexpr (DIAG) {
            if (cs && ch > 0) colsum_done(ch - 1);
        }
        issue(ch + NCH - 1);
        if constexpr (DIAG) {
            if (cs) colsum(ch);
        }
        compute(ch);
    }
    // Drain the loads past the end and let every wave finish reading before
    // the ring is reused.
    wait_vmcnt<0>();
    lds_barrier();
    if constexpr (DIAG) {
        if (cs && nch > 0) colsum_done(nch - 1);
    }
}

template <typename T, bool VEC>
__device__ __forceinline__ void gram_any(const T* __restrict__ X, int rows, int K, int rowR, int rowC,
                                         bool diag, const WaveTiles& wt, f32x16_t acc[4], char* smem,
                                         float* cs = nullptr, float* bsq = nullptr, float* cbuf = nullptr) {
    if constexpr (VEC) {
        if (diag) gram_dl<T, true, BK_GHOST_DIAG_CW>(X, rows, K, rowR, rowC, wt, acc, smem, cs, bsq, cbuf);
        else gram_dl<T, false, BK_GHOST_OFF_CW>(X, rows, K, rowR, rowC, wt, acc, smem);
    } else {
        gram<T, VEC>(X, rows, K, rowR, rowC, diag, wt, acc, reinterpret_cast<uint4*>(smem));
    }
}

// ---------------------------------------------------------------------------
// Ghost norms that stream 256-row super blocks (bf16, 16-byte rows).
//
// 128 < T <= 256 (ghost_full_kernel).  With 128-row super-block pairs every
// row block of such a sample is streamed twice (pairs (0,0), (0,1), (1,1)),
// and the second read mostly comes from HBM again.  Here one 512-thread
// workgroup owns one (layer, sample): the rows of a_i and then of g_i pass
// through a 128 KB LDS ring once, in chunks of 256 rows x 128 bytes (rows >= T
// load zeros), three chunks in flight, one continuous stream over a's chunks
// and then g's.  The T x T Grams are cut into NSUB = ceil(T / 32) blocks of 32
// rows; the NSUB (NSUB + 1) / 2 upper-triangle 32 x 32 sub-tiles (row-major
// order) are dealt to the 8 waves in contiguous runs, the first NT mod 8
// waves taking one more, which puts the same number of sub-tiles on each SIMD
// for NSUB = 7, 8 (waves w and w + 4 share a SIMD).  Each wave keeps both
// Grams of its sub-tiles in registers and reads each 32-row fragment its
// sub-tiles need once per k step.  Off-diagonal sub-tiles count twice.  One
// partial per sample.
//
// T > 256 (ghost_long_kernel).  The Grams are cut into 256-row super blocks
// (nsb = ceil(T / 256)); a sample has nsb diagonal items (one super block
// against itself: the sub-tiles of the T <= 256 kernel with NSUB = 8) and,
// for each pair R < C of super blocks, two half items (super block R against
// one 128-row half of C: 8 x 4 sub-tiles, all counted twice, four per wave in
// 2 x 2 arrangements).  nsb^2 items per sample, each one workgroup and one
// partial; chunks of up to 384 rows (256 of R, 128 of the half of C) in a
// three-slot 144 KB ring, two in flight.  Every item executes only useful
// sub-tiles (528 per 1024-row sample against 544 with 128-row pairs) and
// streams each row 5.5 times instead of 8 at T = 1024.  Items of one sample
// run on one XCD (they share super blocks through its L2).
// ---------------------------------------------------------------------------
constexpr int kFullThreads = 512;
constexpr int kFullCW = 128;                     // bytes of each row per chunk

template <int NSUB>
struct FullTiles {
    static constexpr int NT = NSUB * (NSUB + 1) / 2;
    static constexpr int BASE = NT / 8, REM = NT % 8;
    static constexpr int count(int w) { return BASE + (w < REM ? 1 : 0); }
    static constexpr int start(int w) { return w * BASE + (w < REM ? w : REM); }
    // row / column block of sub-tile q in row-major upper-triangle order
    static constexpr int row(int q) {
        int i = 0;
        while (q >= NSUB - i) { q -= NSUB - i; ++i; }
        return i;
    }
    static constexpr int col(int q) {
        int i = 0;
        while (q >= NSUB - i) { q -= NSUB - i; ++i; }
        return i + q;
    }
    // bit b set: the wave's sub-tiles use 32-row block b
    static constexpr unsigned used(int w) {
        unsigned m = 0;
        for (int q = start(w); q < start(w) + count(w); ++q) m |= (1u << row(q)) | (1u << col(q));
        return m;
    }
};

// 16-byte column c of row r of a chunk sits at column c ^ (r / 2 mod 8): the
// 16 rows read by 16 lanes then meet 16 different 16-byte bank groups.
__device__ __forceinline__ int full_swz(int row, int c) { return c ^ ((row >> 1) & 7); }

// Rows of a_i / g_i of one work item and this wave's LDS-DMA addressing:
// chunk rows 0 .. 255 are rows rowA .. rowA + 255 of the sample, chunk rows
// 256 .. 8 64 LPW - 1 rows rowB onwards.  Load i of the wave fills chunk rows
// 8 (8 i + wave) .. + 7; lane l writes 16-byte column l % 8 of row l / 8,
// which holds chunk column full_swz(row, l % 8).
template <int LPW>
struct FullStream {
    u32x4_t ra, rg;                  // resources over the sample's T rows (zeros beyond)
    uint32_t ba[LPW], bg[LPW];       // byte offset of each load's lane within a chunk column
    int lcol[LPW];                   // 16-byte chunk column each load's lane fetches
    int Ka, Kg, nca, ncg;            // row lengths (elements) and chunks of a and g

    __device__ __forceinline__ void init(const GhostLayer& L, int sample, int rowA, int rowB, int wave,
                                         int lane) {
        Ka = L.d;
        Kg = L.p;
        nca = (L.d + kFullCW / 2 - 1) / (kFullCW / 2);
        ncg = (L.p + kFullCW / 2 - 1) / (kFullCW / 2);
        const uint32_t rba = (uint32_t)L.d * 2u, rbg = (uint32_t)L.p * 2u;
        // The host guarantees (T + 256) * row bytes < 2^31 for these kernels.
        ra = raw_rsrc(reinterpret_cast<const bf16_t*>(L.x) + (size_t)sample * L.T * L.d, (uint32_t)L.T * rba);
        rg = raw_rsrc(reinterpret_cast<const bf16_t*>(L.g) + (size_t)sample * L.T * L.p, (uint32_t)L.T * rbg);
#pragma unroll
        for (int i = 0; i < LPW; ++i) {
            const int lr = 8 * (8 * i + wave) + lane / 8;
            const int row = lr < 256 ? rowA + lr : rowB + (lr - 256);
            lcol[i] = full_swz(lr, lane % 8);
            ba[i] = (uint32_t)row * rba + (uint32_t)lcol[i] * 16u;
            bg[i] = (uint32_t)row * rbg + (uint32_t)lcol[i] * 16u;
        }
    }

    // Queue chunk v (a's chunks first, then g's) into its slot of an
    // NSLOT-slot ring.  Chunks past the end load zeros, so every call issues
    // the same number of loads.
    template <int NSLOT, int SLOTB>
    __device__ __forceinline__ void issue(int v, char* ring, int wave) const {
        char* slot = ring + (v % NSLOT) * SLOTB;
        const bool isa = v < nca;
        const int ch = isa ? v : v - nca;
        const int K = isa ? Ka : Kg;
        const bool live = v < nca + ncg;
        const u32x4_t rs = isa ? ra : rg;
#pragma unroll
        for (int i = 0; i < LPW; ++i) {
            const bool ok = live && ch * (kFullCW / 2) + lcol[i] * 8 < K;
            const uint32_t off = (uint32_t)ch * kFullCW + (isa ? ba[i] : bg[i]);
            dma16_asm(rs, ok ? off : kGhostOut, slot + (8 * i + wave) * 1024);
        }
    }
};

// Sub-tiles Q .. Q + N - 1 with their blocks as constants (so that fragment
// and accumulator indices stay compile-time): one MFMA step each, and the
// weighted sum of Gram(a) o Gram(g) (off-diagonal sub-tiles twice).
template <int NSUB, int Q, int N>
struct FullStep {
    static constexpr int I = FullTiles<NSUB>::row(Q), J = FullTiles<NSUB>::col(Q);
    static __device__ __forceinline__ void mfma(f32x16_t* acc, const uint4* fr) {
        Mfma<bf16_t>::step(acc[0], fr[I], fr[J]);
        FullStep<NSUB, Q + 1, N - 1>::mfma(acc + 1, fr);
    }
    static __device__ __forceinline__ float dot(const f32x16_t* a, const f32x16_t* g) {
        float v = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) v += a[0][i] * g[0][i];
        return (I == J ? 1.f : 2.f) * v + FullStep<NSUB, Q + 1, N - 1>::dot(a + 1, g + 1);
    }
};
template <int NSUB, int Q>
struct FullStep<NSUB, Q, 0> {
    static __device__ __forceinline__ void mfma(f32x16_t*, const uint4*) {}
    static __device__ __forceinline__ float dot(const f32x16_t*, const f32x16_t*) { return 0.f; }
};

__device__ __forceinline__ uint4 full_frag(const char* slot, int row, int col) {
    return *reinterpret_cast<const uint4*>(slot + row * kFullCW + full_swz(row, col) * 16);
}

// Diagonal item: acc[t] += sub-tile t of X X^T over one chunk (4 k steps of
// 16 bf16).
template <int NSUB, int W>
struct DiagTiles {
    using FT = FullTiles<NSUB>;
    static constexpr int N = FT::count(W), Q0 = FT::start(W);
    static __device__ __forceinline__ void compute(const char* __restrict__ slot, f32x16_t* acc) {
        constexpr unsigned USED = FT::used(W);
        const int lane = threadIdx.x & 63, r = lane & 31, h = lane >> 5;
#pragma unroll
        for (int j = 0; j < kFullCW / 32; ++j) {
            uint4 fr[NSUB];
#pragma unroll
            for (int b = 0; b < NSUB; ++b)
                if (USED & (1u << b)) fr[b] = full_frag(slot, 32 * b + r, 2 * j + h);
            FullStep<NSUB, Q0, N>::mfma(acc, fr);
        }
    }
    static __device__ __forceinline__ float dot(const f32x16_t* a, const f32x16_t* g) {
        return FullStep<NSUB, Q0, N>::dot(a, g);
    }
    // The fragments of k step j (of 4) that the wave's sub-tiles use, and
    // their MFMAs (the ping-pong stream reads and multiplies apart).
    struct Frag {
        uint4 fr[NSUB];
    };
    static __device__ __forceinline__ void read(const char* __restrict__ slot, int j, Frag& f) {
        constexpr unsigned USED = FT::used(W);
        const int lane = threadIdx.x & 63, r = lane & 31, h = lane >> 5;
#pragma unroll
        for (int b = 0; b < NSUB; ++b)
            if (USED & (1u << b)) f.fr[b] = full_frag(slot, 32 * b + r, 2 * j + h);
    }
    static __device__ __forceinline__ void mma(f32x16_t* acc, const Frag& f) {
        FullStep<NSUB, Q0, N>::mfma(acc, f.fr);
    }
};

// Off-diagonal half item: wave w takes 32-row blocks I = 2 (w / 2) + {0, 1}
// of super block R (chunk rows 0 .. 255) against blocks J = 2 (w mod 2) +
// {0, 1} of the half of C (chunk rows 256 .. 383); every sub-tile counts twice.
template <int W>
struct HalfTiles {
    static constexpr int N = 4;
    static __device__ __forceinline__ void compute(const char* __restrict__ slot, f32x16_t* acc) {
        const int lane = threadIdx.x & 63, r = lane & 31, h = lane >> 5;
        constexpr int I0 = 2 * (W >> 1), J0 = 2 * (W & 1);
#pragma unroll
        for (int j = 0; j < kFullCW / 32; ++j) {
            const int col = 2 * j + h;
            const uint4 x0 = full_frag(slot, 32 * I0 + r, col), x1 = full_frag(slot, 32 * (I0 + 1) + r, col);
            const uint4 y0 = full_frag(slot, 256 + 32 * J0 + r, col);
            const uint4 y1 = full_frag(slot, 256 + 32 * (J0 + 1) + r, col);
            Mfma<bf16_t>::step(acc[0], x0, y0);
            Mfma<bf16_t>::step(acc[1], x0, y1);
            Mfma<bf16_t>::step(acc[2], x1, y0);
            Mfma<bf16_t>::step(acc[3], x1, y1);
        }
    }
    static __device__ __forceinline__ float dot(const f32x16_t* a, const f32x16_t* g) {
        float v = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) v += a[t][i] * g[t][i];
        return 2.f * v;
    }
    struct Frag {
        uint4 x0, x1, y0, y1;
    };
    static __device__ __forceinline__ void read(const char* __restrict__ slot, int j, Frag& f) {
        const int lane = threadIdx.x & 63, r = lane & 31, col = 2 * j + (lane >> 5);
        constexpr int I0 = 2 * (W >> 1), J0 = 2 * (W & 1);
        f.x0 = full_frag(slot, 32 * I0 + r, col);
        f.x1 = full_frag(slot, 32 * (I0 + 1) + r, col);
        f.y0 = full_frag(slot, 256 + 32 * J0 + r, col);
        f.y1 = full_frag(slot, 256 + 32 * (J0 + 1) + r, col);
    }
    static __device__ __forceinline__ void mma(f32x16_t* acc, const Frag& f) {
        Mfma<bf16_t>::step(acc[0], f.x0, f.y0);
        Mfma<bf16_t>::step(acc[1], f.x0, f.y1);
        Mfma<bf16_t>::step(acc[2], f.x1, f.y0);
        Mfma<bf16_t>::step(acc[3], f.x1, f.y1);
    }
};

// One wave's share of a work item: stream a's then g's chunks through the
// ring, accumulating this wave's sub-tiles (Tiles) of both Grams, and return
// its weighted sum of Gram(a) o Gram(g).  Chunk v: wait for this wave's loads
// of it (the later chunks may stay in flight), barrier (every wave's loads of
// it have landed and every wave is done with chunk v - 1), refill chunk
// v - 1's slot, multiply.
template <typename Tiles, int LPW, int NSLOT, int SLOTB>
__device__ __forceinline__ float stream_wave(const FullStream<LPW>& fs, char* ring, int wave) {
    constexpr int N = Tiles::N;
    f32x16_t accA[N > 0 ? N : 1], accG[N > 0 ? N : 1];
#pragma unroll
    for (int t = 0; t < N; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) accA[t][i] = accG[t][i] = 0.f;
    const int nv = fs.nca + fs.ncg;
#pragma unroll
    for (int c = 0; c < NSLOT - 1; ++c) fs.template issue<NSLOT, SLOTB>(c, ring, wave);
    for (int v = 0; v < fs.nca; ++v) {
        wait_vmcnt<LPW * (NSLOT - 2)>();
        lds_barrier();
        fs.template issue<NSLOT, SLOTB>(v + NSLOT - 1, ring, wave);
        Tiles::compute(ring + (v % NSLOT) * SLOTB, accA);
    }
    for (int v = fs.nca; v < nv; ++v) {
        wait_vmcnt<LPW * (NSLOT - 2)>();
        lds_barrier();
        fs.template issue<NSLOT, SLOTB>(v + NSLOT - 1, ring, wave);
        Tiles::compute(ring + (v % NSLOT) * SLOTB, accG);
    }
    wait_vmcnt<0>();
    return Tiles::dot(accA, accG);
}

// Ping-pong form of stream_wave.  Waves w and w + 4 share a SIMD; each half
// chunk (two k steps) is a memory phase (the wave's fragments of both steps,
// and in the second half the wait for its own loads of the next chunk) and
// an MFMA phase (the MFMAs of both steps; in the first half, the refill of
// chunk v - 1's slot with chunk v + NSLOT - 1 between them), each ended by a
// workgroup barrier.  Waves 4-7 run one phase behind waves 0-3, so on every
// SIMD one wave multiplies while the other reads.  Chunk v - 1's slot is
// refilled only after the memory phases of both halves of the workgroup for
// chunk v - 1 have passed a barrier, and chunk v + 1 is read only after a
// barrier that every wave reaches after waiting for its loads of it.
template <typename Tiles, int LPW, int NSLOT, int SLOTB>
__device__ __forceinline__ float stream_wave_pp(const FullStream<LPW>& fs, char* ring, int wave) {
    constexpr int N = Tiles::N;
    static_assert(N > 0 && NSLOT >= 3, "ping-pong stream");
    f32x16_t accA[N], accG[N];
#pragma unroll
    for (int t = 0; t < N; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) accA[t][i] = accG[t][i] = 0.f;
    const bool late = wave >= 4;
    const int nv = fs.nca + fs.ncg;
#pragma unroll
    for (int c = 0; c < NSLOT - 1; ++c) fs.template issue<NSLOT, SLOTB>(c, ring, wave);
    wait_vmcnt<LPW * (NSLOT - 2)>();
    lds_barrier();
    if (late) {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
    }
    auto chunk = [&](int v, f32x16_t* acc) {
        const char* slot = ring + (v % NSLOT) * SLOTB;
#pragma unroll
        for (int hs = 0; hs < 2; ++hs) {
            typename Tiles::Frag f0, f1;
            Tiles::read(slot, 2 * hs, f0);
            Tiles::read(slot, 2 * hs + 1, f1);
            if (hs == 1) wait_vmcnt<LPW * (NSLOT - 2)>();
            __builtin_amdgcn_sched_barrier(0);
            lds_barrier();
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_setprio(1);
            Tiles::mma(acc, f0);
            __builtin_amdgcn_sched_barrier(0);
            if (hs == 0) fs.template issue<NSLOT, SLOTB>(v + NSLOT - 1, ring, wave);
            __builtin_amdgcn_sched_barrier(0);
            Tiles::mma(acc, f1);
            __builtin_amdgcn_s_setprio(0);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    for (int v = 0; v < fs.nca; ++v) chunk(v, accA);
    for (int v = fs.nca; v < nv; ++v) chunk(v, accG);
    if (!late) __builtin_amdgcn_s_barrier();
    wait_vmcnt<0>();
    return Tiles::dot(accA, accG);
}

template <typename Tiles, int LPW, int NSLOT, int SLOTB, bool PP>
__device__ __forceinline__ float stream_any(const FullStream<LPW>& fs, char* ring, int wave) {
    if constexpr (PP) return stream_wave_pp<Tiles, LPW, NSLOT, SLOTB>(fs, ring, wave);
    else return stream_wave<Tiles, LPW, NSLOT, SLOTB>(fs, ring, wave);
}

template <int NSUB, int LPW, int NSLOT, int SLOTB, bool PP = false>
__device__ __forceinline__ float diag_item(const FullStream<LPW>& fs, char* ring, int wave) {
    switch (wave) {
        case 0: return stream_any<DiagTiles<NSUB, 0>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 1: return stream_any<DiagTiles<NSUB, 1>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 2: return stream_any<DiagTiles<NSUB, 2>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 3: return stream_any<DiagTiles<NSUB, 3>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 4: return stream_any<DiagTiles<NSUB, 4>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 5: return stream_any<DiagTiles<NSUB, 5>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 6: return stream_any<DiagTiles<NSUB, 6>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        default: return stream_any<DiagTiles<NSUB, 7>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
    }
}

template <int LPW, int NSLOT, int SLOTB, bool PP = false>
__device__ __forceinline__ float half_item(const FullStream<LPW>& fs, char* ring, int wave) {
    switch (wave) {
        case 0: return stream_any<HalfTiles<0>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 1: return stream_any<HalfTiles<1>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 2: return stream_any<HalfTiles<2>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 3: return stream_any<HalfTiles<3>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 4: return stream_any<HalfTiles<4>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 5: return stream_any<HalfTiles<5>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        case 6: return stream_any<HalfTiles<6>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
        default: return stream_any<HalfTiles<7>, LPW, NSLOT, SLOTB, PP>(fs, ring, wave);
    }
}

// Sum of one float per wave of a 512-thread workgroup, in wave order, into
// the partial `out` (thread 0).
__device__ __forceinline__ void write_part_512(float part, float* red, float* out) {
    part = wave_sum(part);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kFullThreads / 64; ++w) s += red[w];
        *out = s;
    }
}

constexpr int kFullSlot = 256 * kFullCW;         // 32 KB: 256 rows
constexpr int kFullSlots = 4;                    // 128 KB ring, three chunks in flight
constexpr int kLongSlot = 384 * kFullCW;         // 48 KB: 256 + 128 rows
constexpr int kLongSlots = 3;                    // 144 KB ring, two chunks in flight
#ifndef BK_GHOST_LONG_PP
#define BK_GHOST_LONG_PP 1
#endif
constexpr bool kLongPP = BK_GHOST_LONG_PP != 0;  // ping-pong stream (stream_wave_pp)

__global__ __launch_bounds__(kFullThreads) void ghost_full_kernel(const GhostArgs args) {
    __shared__ __attribute__((aligned(16))) char ring[kFullSlots * kFullSlot];
    __shared__ float red[kFullThreads / 64];
    // One workgroup per (layer, sample); nothing is shared between them, so
    // the hardware's round-robin deal over the XCDs stays (the host orders the
    // layers largest first).
    const int wg = blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GhostLayer& L = args.L[l];
    const int sample = wg - L.wg_begin;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    FullStream<4> fs;
    fs.init(L, sample, 0, 256, wave, lane);
    float part;
    switch (L.nsb) {            // 32-row blocks, 5 .. 8 (the host's range for this kernel)
        case 5: part = diag_item<5, 4, kFullSlots, kFullSlot>(fs, ring, wave); break;
        case 6: part = diag_item<6, 4, kFullSlots, kFullSlot>(fs, ring, wave); break;
        case 7: part = diag_item<7, 4, kFullSlots, kFullSlot>(fs, ring, wave); break;
        default: part = diag_item<8, 4, kFullSlots, kFullSlot>(fs, ring, wave); break;
    }
    write_part_512(part, red, args.part + (size_t)L.part_off + (size_t)sample);
}

__global__ __launch_bounds__(kFullThreads) void ghost_long_kernel(const GhostArgs args) {
    __shared__ __attribute__((aligned(16))) char ring[kLongSlots * kLongSlot];
    __shared__ float red[kFullThreads / 64];
    // Consecutive workgroups (the items of one sample, which share super
    // blocks) on one XCD.
    const int wg = xcd_remap(blockIdx.x, gridDim.x);
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GhostLayer& L = args.L[l];
    const int local = wg - L.wg_begin, nsb = L.nsb, items = L.npairs;   // items = nsb^2
    const int sample = local / items, q = local - sample * items;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    float part;
    if (q < nsb) {                                   // diagonal: super block q against itself
        FullStream<4> fs;
        fs.init(L, sample, 256 * q, 0, wave, lane);
        part = diag_item<8, 4, kLongSlots, kLongSlot, kLongPP>(fs, ring, wave);
    } else {                                         // pair R < C, half h of C
        int m = (q - nsb) >> 1;
        const int h = (q - nsb) & 1;
        int R = 0;
        while (m >= nsb - 1 - R) { m -= nsb - 1 - R; ++R; }
        const int C = R + 1 + m;
        FullStream<6> fs;
        fs.init(L, sample, 256 * R, 256 * C + 128 * h, wave, lane);
        part = half_item<6, kLongSlots, kLongSlot, kLongPP>(fs, ring, wave);
    }
    write_part_512(part, red, args.part + (size_t)L.part_off + (size_t)sample * items + q);
}

template <typename T, bool EMBED, bool VEC>
__global__ __launch_bounds__(256) void ghost_norm_kernel(const GhostArgs args) {
    // VEC: the ring of gram_dl; otherwise two padded blocks for gram.
    __shared__ __attribute__((aligned(16))) char smem[VEC ? kRingBytes : 2 * kBlockU4 * 16];
    uint4* lds = reinterpret_cast<uint4*>(smem);
    __shared__ int64_t sid[2 * kSuper];
    __shared__ float red[4];
    __shared__ float cbuf[VEC && !EMBED ? 2 * 4 * 128 : 1];   // column sums of the bias (gram_dl)

    // Consecutive workgroups (the super-block pairs of one sample, which share
    // row blocks) on one XCD, so that the repeated block reads hit its L2.
    // With one pair per sample nothing is shared: the grid runs in launch
    // order, which the host sets largest workgroups first.
    const int wg = args.remap ? xcd_remap(blockIdx.x, gridDim.x) : (int)blockIdx.x;
    const int l = find_desc(args.n, (int64_t)wg, [&](int k) { return args.L[k].wg_begin; });
    const GhostLayer& L = args.L[l];
    const int nT = L.T, d = L.d, p = L.p, nsb = L.nsb, npairs = L.npairs;
    const int local = wg - L.wg_begin;
    const int sample = local / npairs;
    int pair = local - sample * npairs;
    int R = 0;
    while (pair >= nsb - R) { pair -= nsb - R; ++R; }
    const int C = R + pair;
    const bool diag = (R == C);
    const int rowR = R * kSuper, rowC = C * kSuper;

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    WaveTiles wt = wave_tiles(wave, diag);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int rs = rowR + (wt.r0 + (s >> 1)) * 32, cs = rowC + (wt.c0 + (s & 1)) * 32;
        if (rs >= nT || cs >= nT) wt.w[s] = 0;
    }

    const size_t off_g = (size_t)sample * (size_t)nT * (size_t)p;
    f32x16_t accG[4];
    float part = 0.f;
    if constexpr (EMBED) {
        // Ids outside [0, V) (V = L.d) are zero one-hot rows, like the padding
        // rows: -1, which matches nothing.
        const int64_t* ids = reinterpret_cast<const int64_t*>(L.x) + (size_t)sample * nT;
        const int t = threadIdx.x;
        const int row = (t < kSuper) ? rowR + t : rowC + (t - kSuper);
        const int64_t id = (row < nT) ? ids[row] : (int64_t)-1;
        sid[t] = (id >= 0 && id < (int64_t)d) ? id : (int64_t)-1;
        gram_any<T, VEC>(reinterpret_cast<const T*>(L.g) + off_g, nT, p, rowR, rowC, diag, wt, accG, smem);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (!wt.w[s]) continue;
            const int cl = (wt.c0 + (s & 1)) * 32 + (lane & 31);
            const int64_t idc = sid[kSuper + cl];
            const int64_t* idr = sid + (wt.r0 + (s >> 1)) * 32;
            float v = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) v += (idr[acc_row(i, lane)] == idc && idc >= 0) ? accG[s][i] : 0.f;
            part += (float)wt.w[s] * v;
        }
    } else {
        f32x16_t accA[4];
        const size_t off_a = (size_t)sample * (size_t)nT * (size_t)d;
        gram_any<T, VEC>(reinterpret_cast<const T*>(L.x) + off_a, nT, d, rowR, rowC, diag, wt, accA, smem);
        // Bias of the layer (host: only with 16-byte rows and T <= 128, one
        // diagonal block per sample): its per-sample sums s = sum_t g_t go to
        // Pb and |s|^2 joins this workgroup's partial.
        float* cs = (VEC && L.Pb) ? L.Pb + (size_t)sample * p : nullptr;
        gram_any<T, VEC>(reinterpret_cast<const T*>(L.g) + off_g, nT, p, rowR, rowC, diag, wt, accG, smem,
                         cs, &part, cbuf);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (!wt.w[s]) continue;
            float v = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) v += accA[s][i] * accG[s][i];
            part += (float)wt.w[s] * v;
        }
    }
    const float tot = block_sum_256(part, red);
    if (threadIdx.x == 0)
        args.part[(size_t)L.part_off + (size_t)sample * npairs + (local - sample * npairs)] = tot;
}

}  // namespace

hipError_t launch_ghost_full(const GhostArgs& args, int n_wg, bool long_t, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    if (long_t) hipLaunchKernelGGL(ghost_long_kernel, dim3(n_wg), dim3(kFullThreads), 0, s, args);
    else hipLaunchKernelGGL(ghost_full_kernel, dim3(n_wg), dim3(kFullThreads), 0, s, args);
    return hipGetLastError();
}

hipError_t launch_ghost(const GhostArgs& args, int n_wg, bool bf16, bool embed, bool vec,
                        hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    const dim3 grid(n_wg), block(256);
#define BK_GHOST(T, E, V) hipLaunchKernelGGL((ghost_norm_kernel<T, E, V>), grid, block, 0, s, args)
    if (bf16) {
        if (embed) { if (vec) BK_GHOST(bf16_t, true, true); else BK_GHOST(bf16_t, true, false); }
        else       { if (vec) BK_GHOST(bf16_t, false, true); else BK_GHOST(bf16_t, false, false); }
    } else {
        if (embed) { if (vec) BK_GHOST(float, true, true); else BK_GHOST(float, true, false); }
        else       { if (vec) BK_GHOST(float, false, true); else BK_GHOST(float, false, false); }
    }
#undef BK_GHOST
    return hipGetLastError();
}

}  // namespace bk
