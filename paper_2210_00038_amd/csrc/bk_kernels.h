// Kernel-argument descriptors and launchers of the BK kernels (internal to
// libbk; the public interface is include/bk.h).
//
// Grouped launches: the descriptors of up to kMax* layers travel in the kernel
// arguments themselves (no device-side table to upload), so one launch covers
// a whole stack and the call needs no workspace for bookkeeping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bk.h"

#include <algorithm>

namespace bk {

constexpr int kSuper = 128;   // ghost norm: rows of a super block of the T x T Gram
constexpr int kTile = 128;    // a^T g GEMMs: output tile is kTile x kTile

// ---- ghost norm (linear and embedding) ----------------------------------
struct GhostLayer {
    const void* x;      // a [B,T,d] (linear) or ids int64 [B,T] (embedding)
    const void* g;      // [B,T,p]
    int32_t T, d, p;    // d unused for the embedding
    int32_t nsb;        // super blocks: ceil(T / kSuper)
    int32_t npairs;     // nsb (nsb + 1) / 2 upper-triangle super-block pairs
    int32_t wg_begin;   // first workgroup of this layer in the launch
    int32_t part_off;   // first partial (float) of this layer in the workspace
    int32_t pad;
    // Linear layer with a bias, 16-byte rows and T <= 128: the per-sample
    // bias sums [B,p] go here and their squared norm joins the partials; else
    // nullptr.
    float* Pb;
};
constexpr int kMaxGhost = 64;
struct GhostArgs {
    int32_t n, B;
    int32_t remap;      // 1: workgroup order remapped per XCD (xcd_remap)
    float* part;        // partial sums, [layer][sample][pair]
    GhostLayer L[kMaxGhost];
};

// ---- a^T diag(w) g GEMMs: instantiated norms and clipped gradients -------
struct GemmLayer {
    const void* a;      // [B,T,d]
    const void* g;      // [B,T,p]
    float* G;           // [d,p] out (clipped gradient); instantiated norm: the
                        // per-sample gradients [B,d,p] out, or nullptr
    int32_t T, d, p;
    int32_t tm, tn;     // output tiles along d and p
    int32_t wg_begin;
    int32_t part_off;   // instantiated norm: first partial of this layer
    // K split (layers with few output tiles): each tile's contraction is cut
    // into ksplit slices of whole stages, one workgroup each, which write
    // float32 partial tiles to GemmArgs::tiles (this layer's from tile
    // ptile_off on, [sample][tile][slice]); a second kernel adds the slices in
    // order, its workgroups for this layer starting at red_begin.
    int32_t ksplit;     // 1: no split
    int32_t red_begin;
    int32_t swap;       // narrow kernels: the tile is G^T (rows along p, d < p)
    int32_t accum;      // clipped gradient: add to G instead of writing it
    // Grad / GradDL: tiles below split_from run whole (one workgroup each),
    // the tiles from it on in ksplit slices (their partial tiles and
    // reduction workgroups counted from split_from); 0 everywhere else.
    int32_t split_from;
    int64_t ptile_off;  // first float of this layer's partial tiles
};
constexpr int kMaxGemm = 48;
struct GemmArgs {
    int32_t n, B;
    const float* C;     // [B] clip factors (clipped gradient)
    float* part;        // partial sums (instantiated norm), [layer][sample][tile]
    float* tiles;       // K-split partial tiles
    GemmLayer L[kMaxGemm];
};
constexpr int kSplitRedWG = 1024;   // tile elements per workgroup of the slice reduction

// ---- fixed-order reduction of partial sums ---------------------------------
struct ReduceLayer {
    float* out;         // [B]
    int32_t part_off;
    int32_t npart;      // partials per sample
    int32_t part_off2;  // a second run (bias / affine sums), added after the first
    int32_t npart2;
};
constexpr int kMaxReduce = 200;
struct ReduceArgs {
    int32_t n, B;
    const float* part;
    ReduceLayer L[kMaxReduce];
};

// ---- noise ------------------------------------------------------------------
struct NoiseLayer {
    float* G;
    int64_t n;          // elements
    uint32_t tensor_id;
    uint32_t wg_begin;
};
constexpr int kMaxNoise = 150;
struct NoiseArgs {
    int32_t n;
    float std;
    uint64_t seed;
    uint32_t step;
    uint32_t bpw;       // Philox counter blocks per workgroup (256 .. kNoiseBlocksPerWG, 256 | bpw)
    NoiseLayer L[kMaxNoise];
};
constexpr int kNoiseBlocksPerWG = 4 * 256;   // most counter blocks handled by one workgroup

// Kernel variant of the a^T g GEMMs for one layer:
//  Scalar: element loads (rows not 16-byte multiples / unaligned), 128 x 128;
//  Vec   : 16-byte loads, register transpose, 128 x 128 (fp32, or huge bf16);
//  Wide  : bf16, LDS transpose reads, larger tiles;
//  Grad  : bf16 clipped gradient only, 256 x 256 tiles, 512 threads (T >= 64);
//  GradDL: as Grad with LDS DMA and the weights on the accumulators
//          (B <= kDMaxB; each sample padded to whole stages of
//          kDLStageRows rows).
//  Narrow32 / Narrow64: bf16, one side of d x p at most 32 / 64, tiles of
//          256 along the long side (operands swapped when d < p).
enum class GemmVariant { Scalar = 0, Vec = 1, Wide = 2, Grad = 3, GradDL = 4, Narrow32 = 5, Narrow64 = 6 };
constexpr int kGemmVariants = 7;
constexpr int kDMaxB = 4096;
constexpr int kDLStageRows = 32;   // k rows per stage of the GradDL kernel
constexpr int kDLBuffers = 4;      // its LDS stage buffers (the ping-pong schedule takes four)
// Output tiles of the a^T g kernels (plan.cpp and the kernels share them):
// 256 x 128 with 64-row stages (Wide), 256 x 256 (Grad, GradDL), 256 along
// the long side (Narrow); the Scalar / Vec tiles are kTile x kTile.
constexpr int kWideM = 256, kWideN = 128, kWideK = 64;
constexpr int kGradM = 256, kGradN = 256;
constexpr int kNarrowM = 256;
GemmVariant gemm_variant(bool bf16, int64_t d, int64_t p, int64_t rows, bool aligned);
// Output tiles of a d x p layer on variant v: tm x tn tiles of tile_elems
// floats (a K-split partial tile), rows along p when swap.
struct GemmGeom {
    int64_t tm, tn, tile_elems;
    bool swap;
};
GemmGeom gemm_geom(GemmVariant v, int64_t d, int64_t p);

// ---- weighted sum of stored per-sample gradients -------------------------------
struct WsumLayer {
    const float* P;     // [B, n]
    float* G;           // [n]
    int64_t n;
    uint32_t wg_begin;
    uint32_t vec;       // P, G 16-byte aligned and 4 | n
    uint32_t accum;     // add to G instead of writing it
    uint32_t pad;
};
constexpr int kMaxWsum = 100;
struct WsumArgs {
    int32_t n, B;
    const float* C;
    WsumLayer L[kMaxWsum];
};
constexpr int kWsumPerWG = 1024;    // elements per workgroup

// ---- convolution data preparation ------------------------------------------
struct UnfoldShape {
    int64_t B, C, H, W;         // input x [B, C, H, W]
    int64_t kh, kw, stride, pad;
    int64_t Ho, Wo, T, ld;      // output a [B, T = Ho Wo, ld]
};

// One layer of a grouped preparation: unfold x -> a (when x is set) and
// transpose dy [B, p, T] -> g [B, T, p] (when dy is set).
struct ConvPrepLayer {
    const void* x;
    const void* dy;
    void* a;
    void* g;
    UnfoldShape s;
    int64_t p;
};

// Device-side jobs of the grouped preparation kernel (32-bit sizes; the
// launcher sends larger shapes to the element-wise kernels).
struct UnfoldJob {
    const void* x;
    void* a;
    int C, H, W, kh, kw, stride, pad, Ho, Wo, ld;
    int cc, ngroups, Wr, table_off;   // channels per group, groups, patch row stride, table offset
    int vw;                           // input elements per load (1, 2 or 4; W % vw == 0)
    int sh;                           // first element of a patch row (sh + pad even, Wr = 2 mod 4)
};
struct TokensJob {
    const void* y;
    void* out;
    int C, HW, tiles_t, tiles_c;
    int vin;                          // 16-byte loads along HW (HW a multiple of 16 / element size)
    int pad_;
};
constexpr int kMaxPrepJobs = 24;
struct PrepArgs {
    int nu, nt;
    UnfoldJob u[kMaxPrepJobs];
    TokensJob t[kMaxPrepJobs];
    int blk_end[2 * kMaxPrepJobs];
};

// ---- launchers (return the launch status) ----------------------------------
// Ghost norms over 256-row super blocks (bf16, 16-byte rows), 512-thread
// workgroups.  kSuper < T <= 2 kSuper (long_t false): one workgroup and one
// partial per (layer, sample), GhostLayer::nsb = ceil(T / 32) (5 .. 8).
// T > 2 kSuper (long_t true): GhostLayer::nsb = ceil(T / 256) super blocks,
// npairs = nsb^2 items (workgroups, partials) per sample.
constexpr int kFullSub = 32;
constexpr int kLongSuper = 256;
hipError_t launch_ghost_full(const GhostArgs& args, int n_wg, bool long_t, hipStream_t s);
hipError_t launch_ghost(const GhostArgs& args, int n_wg, bool bf16, bool embed, bool vec,
                        hipStream_t s);
// n_remap (Grad, GradDL): the first n_remap workgroups are dealt to the XCDs in
// contiguous runs; the rest (a launch's tail) run in launch order.  0: all.
hipError_t launch_gemm(const GemmArgs& args, int n_wg, bool bf16, bool inst_norm, GemmVariant v,
                       hipStream_t s, int n_remap = 0);
// Adds the K slices of every split layer of `args` (launched with
// launch_gemm) in order: into G (clipped gradient), or squared into the norm
// partials and optionally kept in G (instantiated norm).  n_wg: the sum of
// the split layers' reduction workgroups.
hipError_t launch_split_reduce(const GemmArgs& args, int n_wg, bool inst_norm, GemmVariant v,
                               hipStream_t s);
hipError_t launch_reduce(const ReduceArgs& args, int n_threads, hipStream_t s);
hipError_t launch_clip(const float* norm_sq, int64_t L, int64_t B, int mode, float R, float gamma,
                       float* C, float* total_sq, hipStream_t s);
hipError_t launch_noise(const NoiseArgs& args, int n_wg, hipStream_t s);
hipError_t launch_wsum(const WsumArgs& args, int n_wg, hipStream_t s);
hipError_t launch_unfold(const void* x, void* a, const UnfoldShape& s, bool bf16, hipStream_t st);
hipError_t launch_conv_prep(const ConvPrepLayer* L, int n, int64_t B, bool bf16, hipStream_t st);
hipError_t launch_tokens(const void* y, void* out, int64_t B, int64_t C, int64_t HW, bool bf16, hipStream_t st);
hipError_t launch_philox_raw(uint64_t seed, uint32_t tid, uint32_t step, uint64_t q0, int64_t nq,
                             uint32_t* out, hipStream_t s);
// Embedding gradient of n = B*T tokens (n <= kEmbedMaxTokens) into rows of p
// columns; ws holds embed_grad_ws_bytes(n, p) bytes (the radix-sort key
// buffers and digit histograms, and the chunks' partial rows, about n p / 8
// bytes).
constexpr int64_t kEmbedMaxTokens = (int64_t)1 << 24;
// Its workspace: radix tiles of kEmbedTileKeys keys, reduction chunks of
// kEmbedChunk sorted positions, every part 256-byte aligned.
constexpr int kEmbedTileKeys = 1024;
constexpr int kEmbedChunk = 64;
inline size_t embed_ws_align(size_t x) { return (x + 255) / 256 * 256; }
inline int64_t embed_tiles_of(int64_t n) { return (n + kEmbedTileKeys - 1) / kEmbedTileKeys; }
inline int64_t embed_chunks_of(int64_t n) { return (n + kEmbedChunk - 1) / kEmbedChunk; }

// Embedding ghost norm as an id join (embed_join.hip): one 1024-thread
// workgroup per (layer, sample, chunk of 8 ct columns of g), ct =
// embed_join_ct(p) (8 or 32, the same for every layer of a launch), the
// sample's T <= kEmbedJoinMaxT keys sorted in LDS (embed_join_lds_bytes(T)
// of dynamic LDS); p % 8 == 0 and 16-byte aligned rows of g.  One partial
// per chunk.
constexpr int64_t kEmbedJoinMaxT = 16384;
constexpr int kEmbedJoinThreads = 1024;
int embed_join_ct(int64_t p);
// Bytes of its keys / partial-sums region (16-byte multiple) and of its
// whole dynamic LDS (the region and one flag per segment).
size_t embed_join_region(int64_t T);
size_t embed_join_lds_bytes(int64_t T);
hipError_t launch_embed_join(const GhostArgs& args, int n_wg, bool bf16, int ct, hipStream_t s);
size_t embed_grad_ws_bytes(int64_t n, int64_t p);
hipError_t launch_embed_grad(const int64_t* ids, const void* g, const float* C, bool bf16,
                             int64_t B, int64_t T, int64_t p, int64_t V, float* G, void* ws,
                             bool accum, hipStream_t s);

// ---- per-sample bias and normalization-affine sums ---------------------------
// For each sample i and feature c: s_i[c] = sum_t g[i,t,c] (a bias or a beta)
// and, with x set, u_i[c] = sum_t g[i,t,c] x[i,t,c] (a gamma).  One workgroup
// per (layer, sample, chunk of kAffineCols features) writes the sums and one
// partial of the squared norm, sum_c u^2 + s^2, at part[part_off + i chunks + k].
constexpr int kAffineCols = 256;
struct AffineLayer {
    const void* x;      // xhat [B,T,p] (gamma terms; may be null when T == 0)
    const void* g;      // [B,T,p]
    float* P;           // [B,p] gamma sums (gamma set)
    float* Pb;          // [B,p] bias / beta sums, or nullptr
    int32_t T, p;
    int32_t chunks;     // ceil(p / kAffineCols)
    int32_t wg_begin;
    int32_t part_off;
    int32_t vec;        // x and g rows 16-byte aligned, 8 | p
    int32_t gamma;      // the layer has gamma terms (an affine layer)
    int32_t pad;
};
constexpr int kMaxAffine = 64;
struct AffineArgs {
    int32_t n, B;
    float* part;
    AffineLayer L[kMaxAffine];
};
hipError_t launch_affine(const AffineArgs& args, int n_wg, bool bf16, hipStream_t s);

// Host-side error reporting of the C ABI: record the detail that
// bk_last_error() returns on this thread and return the status
// (host_hip_fail: BK_ERR_LAUNCH with the HIP error text).
bk_status host_fail(bk_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
bk_status host_hip_fail(hipError_t e, const char* what);

}  // namespace bk
