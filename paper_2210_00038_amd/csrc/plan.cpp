// Host-side planning helpers of the kernels (plain C++, no device code):
// kernel variant and tile geometry of the a^T g GEMMs, the embedding
// scatter's workspace, and the id join's column chunks and LDS size.  The
// kernels use the same constants (bk_kernels.h).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "bk_kernels.h"

namespace bk {

GemmGeom gemm_geom(GemmVariant v, int64_t d, int64_t p) {
    auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
    switch (v) {
        case GemmVariant::Grad:
        case GemmVariant::GradDL: return {cdiv(d, kGradM), cdiv(p, kGradN), (int64_t)kGradM * kGradN, false};
        case GemmVariant::Wide: return {cdiv(d, kWideM), cdiv(p, kWideN), (int64_t)kWideM * kWideN, false};
        case GemmVariant::Narrow32:
        case GemmVariant::Narrow64: {
            const int64_t bn = v == GemmVariant::Narrow32 ? 32 : 64;
            const bool sw = d < p;
            return {cdiv(sw ? p : d, kNarrowM), cdiv(sw ? d : p, bn), kNarrowM * bn, sw};
        }
        default: return {cdiv(d, kTile), cdiv(p, kTile), (int64_t)kTile * kTile, false};
    }
}

GemmVariant gemm_variant(bool bf16, int64_t d, int64_t p, int64_t rows, bool aligned) {
    const int64_t es = bf16 ? 2 : 4;
    const bool vec = aligned && (d * es) % 16 == 0 && (p * es) % 16 == 0;
    if (!vec) return GemmVariant::Scalar;
    // The wide and narrow kernels address one K stage of rows at a time with
    // 32-bit buffer offsets (rows_rsrc): a stage must fit in 2^31 bytes.
    (void)rows;
    if (bf16 && 4 * kWideK * std::max(d, p) * es < ((int64_t)1 << 31)) {
        const int64_t lo = std::min(d, p), hi = std::max(d, p);
        if (lo <= 64 && hi >= 128) return lo <= 32 ? GemmVariant::Narrow32 : GemmVariant::Narrow64;
        return GemmVariant::Wide;
    }
    return GemmVariant::Vec;
}

// Two key buffers [n] uint64, the digit histograms [256 x tiles] int32, the
// chunks' partial rows [chunks x 2 x p] float32 and flags [chunks] int32
// (the layout embed_grad.hip carves).
size_t embed_grad_ws_bytes(int64_t n, int64_t p) {
    if (n <= 0) return 0;
    const int64_t tiles = embed_tiles_of(n), chunks = embed_chunks_of(n);
    return 2 * embed_ws_align((size_t)n * sizeof(uint64_t)) + embed_ws_align((size_t)(256 * tiles) * sizeof(int32_t)) +
           embed_ws_align((size_t)(2 * chunks * p) * sizeof(float)) + embed_ws_align((size_t)chunks * sizeof(int32_t));
}

int embed_join_ct(int64_t p) { return p >= 256 ? 32 : 8; }

size_t embed_join_region(int64_t T) {
    int64_t tp = 1;
    while (tp < T) tp <<= 1;
    // the keys (8 B each), later overlaid by every thread's head and tail sums
    return std::max<size_t>((size_t)tp * 8, 2 * (size_t)kEmbedJoinThreads * 8 * sizeof(float));
}
size_t embed_join_lds_bytes(int64_t T) { return embed_join_region(T) + 128 * sizeof(int); }

}  // namespace bk
