// A 2-D convolution as a generalized linear layer (App. B: d = input
// channels x kernel height x kernel width, p = output channels, T = output
// height x width): the unfolded input a [B, T, ld] and the token-major output
// gradient g [B, T, p] that the BK kernels take.
//
// Both run in one grouped kernel over a list of layers (one launch prepares
// every convolution of a step): its workgroups are split among unfold jobs,
// then transpose jobs, by cumulative block counts.
//
// unfold (LDS path): one workgroup per (sample b, output row oh, channel
// group).  It copies the input rows that output row reads, for its channels,
// into LDS with coalesced loads (zero rows above and below the image, zero
// columns left and right), builds a table of the patch offset of each of its
// columns (column (c, i, j) -> patch row (c, i), column j; -1 for the zero
// columns d .. ld-1), and then writes the Wo output rows of its column range
// as 16-byte stores, each gathering VE values from LDS at offset + ow stride.
// x is read from HBM about kh / stride times (once per output row that uses
// an input row); a is written once.  Shapes whose patch does not fit, or
// whose ld is not a multiple of VE, take the one-element-per-thread kernel.
//
// tokens: [B, C, HW] -> [B, HW, C] through a 64 x 64 LDS tile, read along
// HW (16 bytes at a time when HW is a multiple of VE) and written as 16-byte
// rows along C (C a multiple of VE); other C take a 32 x 33 tile with scalar
// stores.
#include "bk_device.h"
#include "bk_kernels.h"

namespace bk {
namespace {

constexpr int kUnfoldThreads = 256;
constexpr int64_t kUnfoldLds = 40 * 1024;     // patch + offset table per workgroup
constexpr int64_t kUnfoldWGs = 1024;          // channel groups are split until the grid has this many
constexpr int kFillUnroll = 8;                // independent input loads in flight per thread

template <typename E>
struct Vec16 {
    static constexpr int N = 16 / (int)sizeof(E);
    E v[N];
};

// LDS layout: patch [cc][kh][Wr] of E, then one zero element, then (16-byte
// aligned) the int offset table of the group's columns.  A patch row holds
// the Wp = (Wo - 1) stride + kw input columns an output row reads, starting
// at element sh of the row, with sh + pad even and the row stride Wr = 2
// mod 4: image column 0 sits on a 2-element boundary, so the input rows are
// copied two elements per store, and consecutive rows start an odd number of
// 4-byte words apart (bf16), which keeps the rows a wave's gather reads on
// different LDS banks.
struct UnfoldPlan {
    int cc = 0, ngroups = 0, Wr = 0, sh = 0;
    int64_t table_off = 0, lds = 0;
};

UnfoldPlan unfold_plan(const UnfoldShape& s, int es) {
    UnfoldPlan p;
    const int ve = 16 / es;
    if (s.ld % ve != 0 || s.B > 65535 || s.Ho > 65535 || s.ld > INT32_MAX) return p;
    if (s.Wo * (s.ld / ve) > INT32_MAX) return p;          // items of one workgroup fit an int
    const int64_t Wp = (s.Wo - 1) * s.stride + s.kw;
    // sh + pad even and Wr = 2 mod 4: rows start on 2-element boundaries
    // and rows lie an odd number of 4-byte words apart (bf16), so that the
    // rows a wave's gather reads fall on different banks
    const int64_t sh = s.pad % 2, Wr = (Wp + sh + 1) / 4 * 4 + 2;
    const int64_t khkw = s.kh * s.kw, d = s.C * khkw;
    const int64_t per_c = s.kh * Wr * es + khkw * 4;
    const int64_t fixed = (s.ld - d) * 4 + es + 16 + 16;
    const int64_t cap = (kUnfoldLds - fixed) / per_c;      // channels whose patch and table fit
    int64_t cc = cap;
    // more groups when (sample, output row) pairs alone do not fill the chip
    const int64_t want = (kUnfoldWGs + s.B * s.Ho - 1) / (s.B * s.Ho);
    if (want > 1) cc = std::min(cc, (s.C + want - 1) / want);
    if (cc < s.C) {                           // group column ranges stay 16-byte aligned
        cc = (cc + ve - 1) / ve * ve;
        if (cc > cap) cc -= ve;
    }
    cc = std::min<int64_t>(cc, s.C);
    if (cc < 1 || cc * s.kh * Wr >= 65536) return p;
    p.cc = (int)cc;
    p.ngroups = (int)((s.C + cc - 1) / cc);
    p.Wr = (int)Wr;
    p.sh = (int)sh;
    p.table_off = (cc * s.kh * Wr * es + es + 15) / 16 * 16;
    const int64_t ncols_max = std::max<int64_t>(cc * khkw, s.ld - (s.C - 1) / cc * cc * khkw);
    p.lds = p.table_off + ncols_max * 4;
    if (p.lds > 64 * 1024) p.cc = 0;
    return p;
}

// n / dv for 0 <= n < 2^16 (every LDS patch index): the float estimate is
// within one of the quotient, and one step either way makes it exact.
__device__ __forceinline__ int small_div(int n, int dv, float rdv) {
    int q = (int)((float)n * rdv);
    const int rem = n - q * dv;
    q += (rem >= dv) - (rem < 0);
    return q;
}

// N consecutive elements (N * sizeof(E) bytes, that aligned) in one load.
template <typename E, int N>
__device__ __forceinline__ void load_vec(const E* src, E (&v)[4]) {
    struct alignas(N * sizeof(E)) Pack { E e[N]; };
    const Pack p = *reinterpret_cast<const Pack*>(src);
#pragma unroll
    for (int j = 0; j < N; ++j) v[j] = p.e[j];
}

// ... and in one store.
template <typename E, int N>
__device__ __forceinline__ void store_vec(E* dst, const E (&v)[4]) {
    struct alignas(N * sizeof(E)) Pack { E e[N]; };
    Pack p;
#pragma unroll
    for (int j = 0; j < N; ++j) p.e[j] = v[j];
    *reinterpret_cast<Pack*>(dst) = p;
}

// One unfold workgroup: channel group g of output row oh of sample b.
template <typename E>
__device__ __forceinline__ void unfold_block(const UnfoldJob& J, int64_t b, int oh, int g,
                                             unsigned char* smem) {
    const E* __restrict__ x = static_cast<const E*>(J.x);
    E* __restrict__ a = static_cast<E*>(J.a);
    E* patch = reinterpret_cast<E*>(smem);
    int* offs = reinterpret_cast<int*>(smem + J.table_off);
    constexpr int VE = Vec16<E>::N;
    const int tid = threadIdx.x;
    const int kh = J.kh, kw = J.kw, khkw = kh * kw, stride = J.stride, pad = J.pad;
    const int H = J.H, W = J.W, Wo = J.Wo, Wr = J.Wr, sh = J.sh, C = J.C, cc = J.cc;
    const int Wp = (Wo - 1) * stride + kw;          // input columns of an output row
    const int c0 = g * cc, cg = min(cc, C - c0);
    const int d = C * khkw, ld = J.ld;
    const int col0 = c0 * khkw;
    const int ncols = (c0 + cg == C) ? ld - col0 : cg * khkw;
    const int zslot = cc * kh * Wr;

    // input rows (c, i) of this output row: the patch is zeroed (16 bytes per
    // store, up to the table), then the in-image part of each row (columns
    // w < Wv of the input row, at patch column pad + w of the row) is copied
    // J.vw elements per load and per store, walked flat over (row, vector)
    // so every lane loads
    const int nz16 = J.table_off / 16;
    for (int e = tid; e < nz16; e += kUnfoldThreads) reinterpret_cast<uint4*>(smem)[e] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    const int vw = J.vw;
    const int Wv = min(W, Wp - pad);                  // image columns inside the patch row
    const int nv = Wv > 0 ? (Wv + vw - 1) / vw : 0;   // loads per row
    const int nrows = cg * kh, nel = nrows * nv;
    const float rnv = 1.0f / (float)max(nv, 1), rkh = 1.0f / (float)kh;
    const E* xb = x + (b * C + c0) * (int64_t)H * W;
    for (int e0 = tid; e0 < nel; e0 += kFillUnroll * kUnfoldThreads) {
        E v[kFillUnroll][4];
        int dst[kFillUnroll], cnt[kFillUnroll];
#pragma unroll
        for (int u = 0; u < kFillUnroll; ++u) {
            const int e = e0 + u * kUnfoldThreads;
            cnt[u] = 0;
            dst[u] = 0;
            if (e < nel) {
                const int r = small_div(e, nv, rnv), w0 = (e - r * nv) * vw;
                const int cr = small_div(r, kh, rkh), i = r - cr * kh;
                const int h = oh * stride + i - pad;
                if (h >= 0 && h < H) {
                    const E* src = xb + ((int64_t)cr * H + h) * W + w0;     // w0 + vw <= W
                    if (vw == 4) load_vec<E, 4>(src, v[u]);
                    else if (vw == 2) load_vec<E, 2>(src, v[u]);
                    else v[u][0] = *src;
                    cnt[u] = min(vw, Wv - w0);
                    dst[u] = r * Wr + sh + pad + w0;             // even when vw > 1
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kFillUnroll; ++u) {
            if (cnt[u] == 4 && vw == 4) {
                const E lo[4] = {v[u][0], v[u][1]}, hi[4] = {v[u][2], v[u][3]};
                store_vec<E, 2>(patch + dst[u], lo);
                store_vec<E, 2>(patch + dst[u] + 2, hi);
            } else if (cnt[u] == 2 && vw == 2) {
                store_vec<E, 2>(patch + dst[u], v[u]);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (j < cnt[u]) patch[dst[u] + j] = v[u][j];
            }
        }
    }
    // Offset table, element q of 16-byte chunk k at offs[q nch + k]: the
    // lanes of a wave read consecutive words (no bank conflicts).
    const int nch = ncols / VE;
    for (int col = tid; col < ncols; col += kUnfoldThreads) {
        const int gc = col0 + col;
        int off = -1;
        if (gc < d) {
            const int c = gc / khkw, rr = gc - c * khkw;
            const int i = rr / kw, j = rr - i * kw;
            off = ((c - c0) * kh + i) * Wr + sh + j;
        }
        if (col < nch * VE) offs[(col % VE) * nch + col / VE] = off;   // the plan makes VE | ncols
    }
    __syncthreads();

    // output rows t = oh Wo + ow, columns col0 .. col0 + ncols, VE at a time
    const int items = Wo * nch;
    int e = tid;
    int ow = e / nch, k = e - ow * nch;
    const int dow = kUnfoldThreads / nch, dk = kUnfoldThreads - dow * nch;
    E* dst0 = a + (b * J.Ho * Wo + (int64_t)oh * Wo) * ld + col0;
    for (; e < items; e += kUnfoldThreads) {
        Vec16<E> out;
        const int base = ow * stride;
#pragma unroll
        for (int q = 0; q < VE; ++q) {
            const int o = offs[q * nch + k];
            out.v[q] = patch[o < 0 ? zslot : o + base];
        }
        *reinterpret_cast<Vec16<E>*>(dst0 + (int64_t)ow * ld + k * VE) = out;
        ow += dow;
        k += dk;
        if (k >= nch) { k -= nch; ++ow; }
    }
}

// One transpose workgroup: a 64 (HW) x 64 (C) tile of sample b; LDS rows
// are tokens, padded by one 16-byte chunk.
template <typename E>
__device__ __forceinline__ void tokens_block(const TokensJob& J, int64_t b, int ty, int tx,
                                             unsigned char* smem) {
    constexpr int VE = Vec16<E>::N, LDR = 64 + VE;
    E* tile = reinterpret_cast<E*>(smem);
    const int64_t C = J.C, HW = J.HW;
    const int64_t c0 = (int64_t)ty * 64, t0 = (int64_t)tx * 64;
    const int tid = threadIdx.x;
    const E* src = static_cast<const E*>(J.y) + b * C * HW;
    E* dst = static_cast<E*>(J.out) + b * C * HW;
    if (J.vin) {
        // 16-byte loads: VE consecutive tokens of one channel (HW % VE == 0)
        constexpr int CPT = 64 / VE;                   // chunks per channel row of the tile
#pragma unroll
        for (int it = 0; it < CPT / 4; ++it) {
            const int idx = it * 256 + tid, cl = idx / CPT, tc = (idx % CPT) * VE;
            const int64_t c = c0 + cl, t = t0 + tc;
            Vec16<E> v{};
            if (c < C && t < HW) v = *reinterpret_cast<const Vec16<E>*>(src + c * HW + t);
#pragma unroll
            for (int j = 0; j < VE; ++j) tile[(tc + j) * LDR + cl] = v.v[j];
        }
    } else {
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int idx = it * 256 + tid, cl = idx >> 6, tl = idx & 63;
            const int64_t c = c0 + cl, t = t0 + tl;
            E v{};
            if (c < C && t < HW) v = src[c * HW + t];
            tile[tl * LDR + cl] = v;
        }
    }
    __syncthreads();
    constexpr int CPR = 64 / VE;                        // 16-byte chunks per tile row
#pragma unroll
    for (int it = 0; it < CPR / 4; ++it) {
        const int idx = it * 256 + tid, tl = idx / CPR, q = idx % CPR;
        const int64_t t = t0 + tl, c = c0 + q * VE;
        if (t < HW && c < C)
            *reinterpret_cast<Vec16<E>*>(dst + t * C + c) = *reinterpret_cast<const Vec16<E>*>(&tile[tl * LDR + q * VE]);
    }
}

template <typename E>
constexpr int tokens_lds() { return 64 * (64 + Vec16<E>::N) * (int)sizeof(E); }

// Workgroups [blk_end[j-1], blk_end[j]) belong to job j: the unfold jobs
// first, then the transpose jobs.
template <typename E>
__global__ __launch_bounds__(kUnfoldThreads) void conv_prep_kernel(PrepArgs A) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int blk = blockIdx.x;
    const int j = find_desc(A.nu + A.nt, blk, [&](int k) { return k ? A.blk_end[k - 1] : 0; });
    const int local = blk - (j ? A.blk_end[j - 1] : 0);
    if (j < A.nu) {
        const UnfoldJob& J = A.u[j];
        const int g = local % J.ngroups, rest = local / J.ngroups;
        unfold_block<E>(J, rest / J.Ho, rest % J.Ho, g, smem);
    } else {
        const TokensJob& J = A.t[j - A.nu];
        const int tx = local % J.tiles_t, rest = local / J.tiles_t;
        tokens_block<E>(J, rest / J.tiles_c, rest % J.tiles_c, tx, smem);
    }
}

template <typename E>
__global__ __launch_bounds__(256) void unfold_any_kernel(const E* __restrict__ x, E* __restrict__ a,
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

// Jobs that the grouped kernel takes, and the separate launches of the rest.
struct PrepBuilder {
    PrepArgs A{};
    int64_t blocks = 0;
    int lds = 0;
};

template <typename E>
hipError_t flush(PrepBuilder& P, hipStream_t st) {
    if (P.A.nu + P.A.nt == 0) return hipSuccess;
    hipLaunchKernelGGL(conv_prep_kernel<E>, dim3((unsigned)P.blocks), dim3(kUnfoldThreads), (size_t)P.lds, st, P.A);
    const hipError_t e = hipGetLastError();
    P = PrepBuilder{};
    return e;
}

template <typename E>
hipError_t add_unfold(PrepBuilder& P, const void* x, void* a, const UnfoldShape& s, hipStream_t st) {
    if (s.B * s.T * s.ld == 0) return hipSuccess;
    const UnfoldPlan p = unfold_plan(s, (int)sizeof(E));
    const int64_t nblk = p.cc > 0 ? (int64_t)p.ngroups * s.Ho * s.B : 0;
    if (p.cc == 0 || reinterpret_cast<uintptr_t>(a) % 16 != 0 || nblk > INT32_MAX / 4 ||
        std::max<int64_t>({s.C, s.H, s.W, s.kh, s.kw, s.stride, s.pad}) > INT32_MAX) {
        const int64_t total = s.B * s.T * s.ld;
        const int64_t nb = std::min<int64_t>((total + 255) / 256, 65536);
        hipLaunchKernelGGL(unfold_any_kernel<E>, dim3((unsigned)nb), dim3(256), 0, st,
                           static_cast<const E*>(x), static_cast<E*>(a), s);
        return hipGetLastError();
    }
    if (P.A.nu == kMaxPrepJobs || P.A.nt > 0 || P.blocks + nblk > INT32_MAX / 2) {
        const hipError_t e = flush<E>(P, st);
        if (e != hipSuccess) return e;
    }
    UnfoldJob& J = P.A.u[P.A.nu];
    // widest input load that divides the row length and the base alignment
    int vw = 1;
    for (int cand : {4, 2})
        if (s.W % cand == 0 && reinterpret_cast<uintptr_t>(x) % (cand * sizeof(E)) == 0) { vw = cand; break; }
    J = UnfoldJob{x, a, (int)s.C, (int)s.H, (int)s.W, (int)s.kh, (int)s.kw, (int)s.stride, (int)s.pad,
                  (int)s.Ho, (int)s.Wo, (int)s.ld, p.cc, p.ngroups, p.Wr, (int)p.table_off, vw, p.sh};
    P.blocks += nblk;
    P.A.blk_end[P.A.nu++] = (int)P.blocks;
    P.lds = std::max<int>(P.lds, (int)p.lds);
    return hipSuccess;
}

template <typename E>
hipError_t add_tokens(PrepBuilder& P, const void* y, void* out, int64_t B, int64_t C, int64_t HW,
                      hipStream_t st) {
    if (B * C * HW == 0) return hipSuccess;
    const int64_t tt = (HW + 63) / 64, tc = (C + 63) / 64, nblk = tt * tc * B;
    if (C % Vec16<E>::N != 0 || reinterpret_cast<uintptr_t>(out) % 16 != 0 || nblk > INT32_MAX / 4 ||
        C > INT32_MAX || HW > INT32_MAX) {
        const dim3 grid((unsigned)((HW + 31) / 32), (unsigned)((C + 31) / 32), (unsigned)B);
        hipLaunchKernelGGL(tokens_kernel<E>, grid, dim3(256), 0, st, static_cast<const E*>(y),
                           static_cast<E*>(out), C, HW);
        return hipGetLastError();
    }
    if (P.A.nt == kMaxPrepJobs || P.blocks + nblk > INT32_MAX / 2) {
        const hipError_t e = flush<E>(P, st);
        if (e != hipSuccess) return e;
    }
    TokensJob& J = P.A.t[P.A.nt];
    const int vin = (HW % Vec16<E>::N == 0 && reinterpret_cast<uintptr_t>(y) % 16 == 0) ? 1 : 0;
    J = TokensJob{y, out, (int)C, (int)HW, (int)tt, (int)tc, vin, 0};
    P.blocks += nblk;
    P.A.blk_end[P.A.nu + P.A.nt++] = (int)P.blocks;
    P.lds = std::max<int>(P.lds, tokens_lds<E>());
    return hipSuccess;
}

template <typename E>
hipError_t conv_prep_typed(const ConvPrepLayer* L, int n, int64_t B, hipStream_t st) {
    PrepBuilder P;
    hipError_t e = hipSuccess;
    for (int l = 0; l < n && e == hipSuccess; ++l)
        if (L[l].x) e = add_unfold<E>(P, L[l].x, L[l].a, L[l].s, st);
    for (int l = 0; l < n && e == hipSuccess; ++l)
        if (L[l].dy) e = add_tokens<E>(P, L[l].dy, L[l].g, B, L[l].p, L[l].s.T, st);
    if (e == hipSuccess) e = flush<E>(P, st);
    return e;
}

}  // namespace

hipError_t launch_conv_prep(const ConvPrepLayer* L, int n, int64_t B, bool bf16, hipStream_t st) {
    return bf16 ? conv_prep_typed<uint16_t>(L, n, B, st) : conv_prep_typed<float>(L, n, B, st);
}

hipError_t launch_unfold(const void* x, void* a, const UnfoldShape& s, bool bf16, hipStream_t st) {
    const ConvPrepLayer L{x, nullptr, a, nullptr, s, 0};
    return launch_conv_prep(&L, 1, s.B, bf16, st);
}

hipError_t launch_tokens(const void* y, void* out, int64_t B, int64_t C, int64_t HW, bool bf16, hipStream_t st) {
    UnfoldShape s{};
    s.T = HW;
    const ConvPrepLayer L{nullptr, y, nullptr, out, s, C};
    return launch_conv_prep(&L, 1, B, bf16, st);
}

}  // namespace bk
