// Driver of the sanitizer build of the C ABI's host code: workspace queries,
// every grouped call over random stacks, and invalid arguments, with the
// launchers stubbed (launch_stubs.cpp).  Device pointers are fake, aligned
// addresses: the host code never dereferences them.  Prints "ok" and exits 0
// when every call returned (sanitizer reports abort the run).
#include <cstdio>
#include <cstdlib>
#include <random>
#include <map>
#include <vector>

#include "bk.h"

extern uintptr_t g_ws_lo, g_ws_hi;
extern long g_launches;
extern std::map<uintptr_t, int> g_noised;

namespace {
std::mt19937_64 rng(20221001);
int64_t pick(std::initializer_list<int64_t> v) { return *(v.begin() + rng() % v.size()); }
void* fake(uintptr_t k, bool misalign = false) { return reinterpret_cast<void*>((k << 24) + (misalign ? 2 : 0)); }
void* set_ws(size_t bytes) {
    g_ws_lo = (uintptr_t)0x7f0000000000ull;
    g_ws_hi = g_ws_lo + bytes;
    return reinterpret_cast<void*>(g_ws_lo);
}
int64_t dim() { return pick({1, 2, 7, 8, 16, 24, 32, 60, 64, 100, 128, 256, 264, 300, 768, 1024, 1280, 3072, 4096}); }
int64_t tlen() { return pick({0, 1, 16, 49, 64, 70, 100, 128, 129, 197, 256, 300, 784, 1000, 1024, 4096, 16385}); }
}  // namespace

// Every weight and bias gradient with elements got its noise from exactly one
// launch (none without noise), and nothing else got any.
bool noised_once(const std::vector<bk_layer>& L, float sig) {
    std::map<uintptr_t, int> want;
    if (sig != 0.f)
        for (const bk_layer& y : L) {
            if ((y.kind == BK_NORM_AFFINE ? y.p : y.d * y.p) > 0) ++want[reinterpret_cast<uintptr_t>(y.G)];
            if ((y.flags & BK_LAYER_BIAS) && y.p > 0) ++want[reinterpret_cast<uintptr_t>(y.Gb)];
        }
    if (want != g_noised) {
        std::fprintf(stderr, "noise launches per tensor: %zu tensors expected, %zu noised\n", want.size(),
                     g_noised.size());
        return false;
    }
    return true;
}

int main() {
    // 1. workspace queries: random, edge and invalid sizes for every op
    for (int it = 0; it < 20000; ++it) {
        const bk_op op = (bk_op)(rng() % 6);
        const bk_dtype dt = (bk_dtype)(rng() % 3);
        const int64_t B = pick({-1, 0, 1, 2, 16, 64, 4096, 4097, (int64_t)1 << 20});
        const int64_t T = pick({-3, 0, 1, 33, 128, 129, 1024, 16384, 16385, (int64_t)1 << 31});
        const int64_t d = pick({-1, 0, 1, 8, 60, 768, 50257, 8192, (int64_t)1 << 40});
        const int64_t p = pick({0, 1, 8, 60, 64, 264, 1280, 3072});
        (void)bk_workspace_size(op, dt, B, T, d, p);
        const int gs = bk_use_ghost(T, d, p), gt = bk_use_ghost_time(T, d, p);
        if (gt == 1 && gs != 1) {
            std::fprintf(stderr, "time rule ghost where the space rule is not (T=%lld d=%lld p=%lld)\n",
                         (long long)T, (long long)d, (long long)p);
            return 1;
        }
    }

    // 2. random stacks through the grouped calls
    int calls = 0, ok_calls = 0;
    for (int it = 0; it < 4000; ++it) {
        const int n = 1 + (int)(rng() % 110);
        const bk_dtype dt = rng() % 4 ? BK_BF16 : BK_F32;
        const int64_t B = pick({1, 2, 3, 16, 32, 64, 4096, 4097});
        std::vector<bk_layer> L((size_t)n);
        for (int l = 0; l < n; ++l) {
            bk_layer& y = L[(size_t)l];
            const int r = (int)(rng() % 10);
            y.kind = r < 7 ? BK_LINEAR : r < 8 ? BK_EMBEDDING : BK_NORM_AFFINE;
            y.T = tlen();
            y.p = dim();
            y.d = y.kind == BK_EMBEDDING ? pick({1, 300, 50257}) : y.kind == BK_NORM_AFFINE ? y.p : dim();
            const bool mis = rng() % 8 == 0;
            y.x = fake(4 * l + 1, mis && y.kind != BK_EMBEDDING);
            y.g = fake(4 * l + 2, mis);
            y.G = static_cast<float*>(fake(4 * l + 3));
            y.flags = 0;
            if (y.kind != BK_EMBEDDING && rng() % 3 == 0) {
                y.flags |= BK_LAYER_BIAS;
                y.Gb = static_cast<float*>(fake(0x100000 + l));
                y.Pb = static_cast<float*>(fake(0x200000 + l));
            }
            if (rng() % 4 == 0) y.flags |= BK_LAYER_ACCUMULATE;
            if (rng() % 3 == 0) y.flags |= BK_LAYER_TIME_RULE;
            if (y.kind == BK_NORM_AFFINE || (y.kind == BK_LINEAR && rng() % 5 == 0)) {
                if (y.kind == BK_LINEAR) y.flags |= BK_LAYER_MIXOPT;
                y.P = static_cast<float*>(fake(0x300000 + l));
            }
        }
        float* norm = static_cast<float*>(fake(0x400000));
        float* C = static_cast<float*>(fake(0x400001));
        float* tot = static_cast<float*>(fake(0x400002));
        const size_t wn = bk_layer_norms_workspace_size(L.data(), n, dt, B);
        const size_t wg = bk_weighted_grads_workspace_size(L.data(), n, dt, B);
        const size_t wp = bk_private_grad_workspace_size(L.data(), n, dt, B);
        if (wp < wn || wp < wg) {
            std::fprintf(stderr, "private-grad workspace below a phase's\n");
            return 1;
        }
        ++calls;
        ok_calls += bk_layer_norms(L.data(), n, dt, B, norm, set_ws(wn), wn, nullptr) == BK_OK;
        (void)bk_weighted_grads(L.data(), n, C, dt, B, set_ws(wg), wg, nullptr);
        const float sig = rng() % 2 ? 1.f : 0.f;
        g_noised.clear();
        const bk_status pst = bk_private_grad(L.data(), n, dt, B, (bk_clip)(rng() % 2), 1.f, 0.01f, sig, 7,
                                              (uint32_t)it, norm, C, tot, set_ws(wp), wp, nullptr);
        if (pst == BK_OK && !noised_once(L, sig)) return 1;
        if (wp > 0 && bk_private_grad(L.data(), n, dt, B, BK_CLIP_AUTO, 1.f, 0.01f, 1.f, 7, 0, norm, C, tot,
                                      set_ws(wp), wp - 1, nullptr) == BK_OK) {
            std::fprintf(stderr, "a short workspace was accepted\n");
            return 1;
        }
    }

    // 3. single-layer calls and invalid arguments
    for (int it = 0; it < 3000; ++it) {
        const bk_dtype dt = (bk_dtype)(rng() % 2);
        const int64_t B = pick({0, 1, 3, 16}), T = tlen(), d = dim(), p = dim();
        void* a = fake(1, rng() % 6 == 0);
        void* g = fake(2, rng() % 6 == 0);
        float* out = static_cast<float*>(fake(3));
        size_t w = bk_workspace_size(BK_OP_GHOST_NORM, dt, B, T, d, p);
        (void)bk_ghost_norm(a, g, dt, B, T, d, p, out, set_ws(w), w, nullptr);
        w = bk_workspace_size(BK_OP_INST_NORM, dt, B, T, d, p);
        (void)bk_inst_norm(a, g, dt, B, T, d, p, out, set_ws(w), w, nullptr);
        const int64_t V = pick({1, 50257});
        w = bk_workspace_size(BK_OP_EMBED_GHOST_NORM, dt, B, T, V, p);
        (void)bk_embed_ghost_norm(static_cast<const int64_t*>(fake(4)), g, dt, B, T, p, V, out, set_ws(w), w, nullptr);
        w = bk_workspace_size(BK_OP_WEIGHTED_GRAD, dt, B, T, d, p);
        (void)bk_weighted_grad(a, g, out, dt, B, T, d, p, out, set_ws(w), w, nullptr);
        w = bk_workspace_size(BK_OP_EMBED_WEIGHTED_GRAD, dt, B, T, V, p);
        (void)bk_embed_weighted_grad(static_cast<const int64_t*>(fake(4)), g, out, dt, B, T, p, V, out, set_ws(w), w,
                                     nullptr);
        (void)bk_clip_factors(out, pick({0, 1, 48}), B, (bk_clip)(rng() % 3), pick({-1, 0, 1}), pick({-1, 0, 1}),
                              out, out, nullptr);
        (void)bk_add_noise(out, pick({-1, 0, 5, 1 << 20}), pick({-1, 0, 1}), 3, 0, 0, nullptr);
        (void)bk_philox_raw(1, 2, 3, 0, pick({-1, 0, 17}), reinterpret_cast<uint32_t*>(out), nullptr);
        // invalid pointers and sizes: every call must fail validation, not crash
        (void)bk_ghost_norm(nullptr, g, dt, B + 1, T + 1, d, p, out, nullptr, 0, nullptr);
        (void)bk_inst_norm(a, g, (bk_dtype)7, B, T, d, p, out, nullptr, 0, nullptr);
        (void)bk_weighted_grad(a, g, nullptr, dt, -B - 1, T, d, p, out, nullptr, 0, nullptr);
        (void)bk_layer_norms(nullptr, 3, dt, B, out, nullptr, 0, nullptr);
    }
    {   // grouped noise over many tensors (more than one launch's table)
        std::vector<float*> G(400);
        std::vector<int64_t> nel(400);
        std::vector<uint32_t> tid(400);
        for (size_t k = 0; k < G.size(); ++k) {
            G[k] = static_cast<float*>(fake(0x500000 + k));
            nel[k] = pick({0, 1, 3, 1000, 1 << 22});
            tid[k] = (uint32_t)k;
        }
        (void)bk_add_noise_grouped(G.data(), nel.data(), tid.data(), (int64_t)G.size(), 1.f, 9, 1, nullptr);
    }
    {   // convolution preparation
        for (int it = 0; it < 500; ++it) {
            const int n = 1 + (int)(rng() % 30);
            std::vector<bk_conv> cv((size_t)n);
            for (int l = 0; l < n; ++l) {
                bk_conv& c = cv[(size_t)l];
                c.x = rng() % 4 ? fake(0x600000 + l) : nullptr;
                c.dy = rng() % 4 ? fake(0x700000 + l) : nullptr;
                c.a = fake(0x800000 + l);
                c.g = fake(0x900000 + l);
                c.C = pick({1, 3, 64, 512});
                c.H = c.W = pick({1, 7, 14, 56, 224});
                c.kh = c.kw = pick({1, 3, 7});
                c.stride = pick({1, 2});
                c.pad = pick({0, 1, 3});
                c.ld = c.C * c.kh * c.kw + pick({0, 5});
                c.p = pick({1, 64, 512});
            }
            (void)bk_conv_prep(cv.data(), n, (bk_dtype)(rng() % 2), pick({1, 16}), nullptr);
        }
    }
    std::printf("ok: %d stacks (%d with valid norms), %ld launches checked\n", calls, ok_calls, g_launches);
    return 0;
}
