// Host-only stand-ins for the kernel launchers and the three HIP runtime calls
// of api.cpp, for the AddressSanitizer / UndefinedBehaviorSanitizer build of
// the C ABI's host code (tests/test_host_sanitize.py).  Nothing here touches a
// GPU.  Each launcher checks what the host hands to the kernels: descriptor
// counts within the argument tables, first-workgroup offsets that never
// decrease, and every workspace range the kernels would write inside the
// workspace the caller passed (set by the driver).  The noise launcher also
// counts, per tensor, the launches that add Gaussian noise to it, so that the
// driver can check that every gradient gets its noise exactly once.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <map>

#include "bk_kernels.h"

uintptr_t g_ws_lo = 0, g_ws_hi = 0;   // [lo, hi): the caller's workspace
long g_launches = 0;
std::map<uintptr_t, int> g_noised;    // tensor -> launches that add noise to it

namespace {
void need(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "launch check failed: %s\n", what);
        std::abort();
    }
}
void in_ws(const void* base, int64_t off_elems, int64_t n_elems, size_t es, const char* what) {
    if (n_elems <= 0) return;
    const uintptr_t b = reinterpret_cast<uintptr_t>(base);
    need(b != 0 && off_elems >= 0, what);
    const uintptr_t lo = b + (uintptr_t)off_elems * es, hi = lo + (uintptr_t)n_elems * es;
    need(lo >= g_ws_lo && hi <= g_ws_hi, what);
}
template <typename L>
void monotone(const L* layers, int n, int max_n, int64_t n_wg, const char* what) {
    if (n_wg <= 0) return;   // the launchers return at once
    need(n >= 1 && n <= max_n, what);
    int64_t prev = 0;
    for (int k = 0; k < n; ++k) {
        if (!((int64_t)layers[k].wg_begin >= prev && (int64_t)layers[k].wg_begin < n_wg))
            std::fprintf(stderr, "descriptor %d of %d: first workgroup %lld after %lld, %lld workgroups\n", k, n,
                         (long long)layers[k].wg_begin, (long long)prev, (long long)n_wg);
        need((int64_t)layers[k].wg_begin >= prev && (int64_t)layers[k].wg_begin < n_wg, what);
        prev = layers[k].wg_begin;
    }
}
}  // namespace

extern "C" {
hipError_t hipGetDevice(int* d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
    *v = 256;
    return hipSuccess;
}
const char* hipGetErrorString(hipError_t) { return "stub"; }
}

namespace bk {

hipError_t launch_ghost_full(const GhostArgs& a, int n_wg, bool, hipStream_t) {
    ++g_launches;
    monotone(a.L, a.n, kMaxGhost, n_wg, "ghost_full descriptors");
    for (int k = 0; k < a.n; ++k) in_ws(a.part, a.L[k].part_off, (int64_t)a.B * a.L[k].npairs, 4, "ghost_full partials");
    return hipSuccess;
}
hipError_t launch_ghost(const GhostArgs& a, int n_wg, bool, bool, bool, hipStream_t) {
    ++g_launches;
    monotone(a.L, a.n, kMaxGhost, n_wg, "ghost descriptors");
    for (int k = 0; k < a.n; ++k) in_ws(a.part, a.L[k].part_off, (int64_t)a.B * a.L[k].npairs, 4, "ghost partials");
    return hipSuccess;
}
hipError_t launch_embed_join(const GhostArgs& a, int n_wg, bool, int ct, hipStream_t) {
    ++g_launches;
    monotone(a.L, a.n, kMaxGhost, n_wg, "join descriptors");
    need(ct == 8 || ct == 32, "join column threads");
    for (int k = 0; k < a.n; ++k) {
        need(a.L[k].T >= 1 && a.L[k].T <= kEmbedJoinMaxT && a.L[k].p % 8 == 0, "join shape");
        need((int64_t)a.L[k].npairs * 8 * ct >= a.L[k].p, "join column chunks");
        in_ws(a.part, a.L[k].part_off, (int64_t)a.B * a.L[k].npairs, 4, "join partials");
    }
    return hipSuccess;
}
hipError_t launch_gemm(const GemmArgs& a, int n_wg, bool, bool inst, GemmVariant v, hipStream_t, int) {
    ++g_launches;
    monotone(a.L, a.n, kMaxGemm, n_wg, "gemm descriptors");
    for (int k = 0; k < a.n; ++k) {
        const GemmLayer& L = a.L[k];
        const GemmGeom geo = gemm_geom(v, L.d, L.p);
        need(L.tm == geo.tm && L.tn == geo.tn, "gemm tiles");
        const int64_t tiles = (int64_t)L.tm * L.tn;
        if (inst && v == GemmVariant::GradDL) {
            // one workgroup per (sample, tile), never split, no clip weights
            need(L.ksplit <= 1 && a.C == nullptr && (int64_t)a.B * L.T < ((int64_t)1 << 31) && L.T >= 64,
                 "LDS-DMA instantiated norm");
        }
        if (inst) {
            const int64_t parts = L.ksplit > 1 ? tiles * (geo.tile_elems / kSplitRedWG) : tiles;
            in_ws(a.part, L.part_off, (int64_t)a.B * parts, 4, "inst partials");
            if (L.ksplit > 1) in_ws(a.tiles, L.ptile_off, (int64_t)a.B * tiles * L.ksplit * geo.tile_elems, 4, "inst tiles");
        } else if (L.ksplit > 1) {
            need(L.split_from >= 0 && L.split_from <= tiles, "grad split_from");
            in_ws(a.tiles, L.ptile_off, (tiles - L.split_from) * L.ksplit * geo.tile_elems, 4, "grad tiles");
        }
    }
    return hipSuccess;
}
hipError_t launch_split_reduce(const GemmArgs& a, int n_wg, bool, GemmVariant, hipStream_t) {
    ++g_launches;
    need(n_wg > 0 && a.n >= 1 && a.n <= kMaxGemm, "split reduce");
    return hipSuccess;
}
hipError_t launch_reduce(const ReduceArgs& a, int n_threads, hipStream_t) {
    ++g_launches;
    need(a.n >= 1 && a.n <= kMaxReduce && n_threads == a.n * a.B, "reduce descriptors");
    for (int k = 0; k < a.n; ++k) {
        in_ws(a.part, a.L[k].part_off, (int64_t)a.B * a.L[k].npart, 4, "reduce partials");
        in_ws(a.part, a.L[k].part_off2, (int64_t)a.B * a.L[k].npart2, 4, "reduce second partials");
    }
    return hipSuccess;
}
hipError_t launch_clip(const float*, int64_t L, int64_t B, int, float, float, float*, float*, hipStream_t) {
    ++g_launches;
    need(L >= 0 && B >= 0, "clip sizes");
    return hipSuccess;
}
hipError_t launch_noise(const NoiseArgs& a, int n_wg, hipStream_t) {
    ++g_launches;
    need(a.n >= 1 && a.n <= kMaxNoise && a.bpw >= 256 && a.bpw <= (uint32_t)kNoiseBlocksPerWG && a.bpw % 256 == 0,
         "noise descriptors");
    uint32_t prev = 0;
    for (int k = 0; k < a.n; ++k) {
        need(a.L[k].wg_begin >= prev && (int64_t)a.L[k].wg_begin < n_wg && a.L[k].n > 0, "noise layers");
        prev = a.L[k].wg_begin;
        ++g_noised[reinterpret_cast<uintptr_t>(a.L[k].G)];
    }
    return hipSuccess;
}
hipError_t launch_wsum(const WsumArgs& a, int n_wg, hipStream_t) {
    ++g_launches;
    need(a.n >= 1 && a.n <= kMaxWsum && n_wg > 0, "wsum descriptors");
    return hipSuccess;
}
hipError_t launch_unfold(const void*, void*, const UnfoldShape& s, bool, hipStream_t) {
    ++g_launches;
    need(s.Ho > 0 && s.Wo > 0 && s.T == s.Ho * s.Wo && s.ld >= s.C * s.kh * s.kw, "unfold shape");
    return hipSuccess;
}
hipError_t launch_conv_prep(const ConvPrepLayer*, int n, int64_t B, bool, hipStream_t) {
    ++g_launches;
    need(n >= 1 && B >= 1, "conv prep");
    return hipSuccess;
}
hipError_t launch_tokens(const void*, void*, int64_t B, int64_t C, int64_t HW, bool, hipStream_t) {
    ++g_launches;
    need(B >= 1 && C >= 1 && HW >= 1, "tokens shape");
    return hipSuccess;
}
hipError_t launch_philox_raw(uint64_t, uint32_t, uint32_t, uint64_t, int64_t nq, uint32_t*, hipStream_t) {
    ++g_launches;
    need(nq >= 0, "philox count");
    return hipSuccess;
}
hipError_t launch_embed_grad(const int64_t*, const void*, const float*, bool, int64_t B, int64_t T, int64_t p,
                             int64_t V, float*, void* ws, bool, hipStream_t) {
    ++g_launches;
    need(B * T <= kEmbedMaxTokens && V > 0 && p > 0, "embedding gradient shape");
    in_ws(ws, 0, (int64_t)embed_grad_ws_bytes(B * T, p), 1, "embedding gradient workspace");
    return hipSuccess;
}
hipError_t launch_affine(const AffineArgs& a, int n_wg, bool, hipStream_t) {
    ++g_launches;
    monotone(a.L, a.n, kMaxAffine, n_wg, "affine descriptors");
    for (int k = 0; k < a.n; ++k) in_ws(a.part, a.L[k].part_off, (int64_t)a.B * a.L[k].chunks, 4, "affine partials");
    return hipSuccess;
}

}  // namespace bk
