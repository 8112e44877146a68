// Host side of the C ABI declared in include/bk.h: argument validation (before
// any HIP call), the layerwise path choice of Section 3.2, workspace layout and
// the grouping of layers into launches.
#include "bk.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "bk_kernels.h"

namespace {

thread_local std::string g_err;

bk_status fail(bk_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

bk_status hip_fail(hipError_t e, const char* what) {
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return BK_ERR_LAUNCH;
}

}  // namespace

namespace bk {
bk_status host_fail(bk_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}
bk_status host_hip_fail(hipError_t e, const char* what) { return hip_fail(e, what); }
}  // namespace bk

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool mul3_ok(int64_t a, int64_t b, int64_t c) {
    int64_t ab, abc;
    return !__builtin_mul_overflow(a, b, &ab) && !__builtin_mul_overflow(ab, c, &abc);
}

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

size_t elem_bytes(bk_dtype dt) { return dt == BK_BF16 ? 2 : 4; }

enum class Path { Ghost, Inst, Embed, Affine };   // Affine: no weight term (BK_NORM_AFFINE)

// Everything the kernels index with 32-bit integers stays below 2^31.
bk_status check_dims(const char* fn, int64_t B, int64_t T, int64_t d, int64_t p) {
    if (B < 0 || T < 0 || d < 0 || p < 0)
        return fail(BK_ERR_INVALID_VALUE, "%s: negative size (B=%lld T=%lld d=%lld p=%lld)", fn,
                    (long long)B, (long long)T, (long long)d, (long long)p);
    if (!mul3_ok(B, T, d) || !mul3_ok(B, T, p) || !mul3_ok(d, p, 1))
        return fail(BK_ERR_INVALID_VALUE, "%s: size product overflows int64", fn);
    if (B * T > INT32_MAX || d > INT32_MAX || p > INT32_MAX || T > INT32_MAX)
        return fail(BK_ERR_NOT_SUPPORTED, "%s: B*T, d and p must each stay below 2^31", fn);
    return BK_OK;
}

bk_status check_dtype(const char* fn, bk_dtype dt) {
    if (dt != BK_F32 && dt != BK_BF16)
        return fail(BK_ERR_INVALID_VALUE, "%s: unknown dtype %d", fn, (int)dt);
    return BK_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------
// Per-layer plans
// ---------------------------------------------------------------------------
struct NormPlan {
    Path path;
    int64_t nwg;        // workgroups of the norm kernel
    int64_t npart;      // partials per sample
    int var;            // kernel variant: ghost 0 = scalar, 1 = 16-byte loads,
                        // 2 = whole-sample kernel (bf16, 128 < T <= 256),
                        // 3 = 256-row super blocks (bf16, T > 256);
                        // instantiation: bk::GemmVariant
    int64_t tiles = 0;  // instantiation: output tiles per sample
    int64_t ksplit = 1; // instantiation: K slices per tile (wide and narrow kernels)
    int64_t tile_elems = 0;   // instantiation: floats of one K-split partial tile
    int64_t aff_chunks = 0;   // per-sample partials of the bias / affine sums (second run)
    bool fused_bias = false;  // ghost layer whose kernel also forms the bias sums (no second run)
};

// Variants whose kernels can split a tile's contraction into K slices.
bool inst_splits(int var) {
    return var == (int)bk::GemmVariant::Wide || var == (int)bk::GemmVariant::Narrow32 ||
           var == (int)bk::GemmVariant::Narrow64;
}
bool is_narrow(bk::GemmVariant v) { return v == bk::GemmVariant::Narrow32 || v == bk::GemmVariant::Narrow64; }

// K slices of an instantiated norm on the wide kernel: when a layer gives
// fewer than 128 workgroups (few samples, few tiles, long T), cut each
// per-sample GEMM into slices of at least 4 stages, towards 256 workgroups.
int64_t inst_ksplit(int64_t B, int64_t tiles, int64_t T) {
    const int64_t wgs = B * tiles, nst = cdiv(T, 64);
    if (wgs == 0 || wgs >= 128 || nst < 8) return 1;
    return std::max<int64_t>(1, std::min(cdiv(256, wgs), nst / 4));
}

// K slices of a clipped-gradient tile (agrad kernels): a layer with fewer than
// 8 output tiles and at least 64 stages gets slices of about 32 stages.
int64_t grad_ksplit(int64_t tiles, int64_t nst) {
    if (tiles >= 8 || nst < 64) return 1;
    return std::min<int64_t>(256, cdiv(nst, 32));
}

// The same for the narrow kernels (64-row stages, far less work per stage):
// a layer with fewer than 32 tiles gets slices of about 16 stages, at most 64.
int64_t narrow_grad_ksplit(int64_t tiles, int64_t nst) {
    if (tiles >= 32 || nst < 32) return 1;
    return std::min<int64_t>(64, cdiv(nst, 16));
}

// Stages per sample of the GradDL kernel: every sample starts a stage, its
// last stage padded with zero rows.  The MFMAs run over T rounded up to
// 16-row steps (a last stage of at most 16 rows skips its second step).
int64_t dl_stages_per_sample(int64_t T) { return cdiv(T, bk::kDLStageRows); }
bool dl_padding_ok(int64_t T) { return 8 * (cdiv(T, 16) * 16) <= 9 * T; }   // at most 1/8 padding

void set_norm_variant(NormPlan& np, const bk_layer& L, bk_dtype dt, int64_t B) {
    const size_t es = elem_bytes(dt);
    if (np.path == Path::Affine) {
        np.npart = 0;
        np.var = 0;
    } else if (np.path == Path::Inst) {
        auto v = bk::gemm_variant(dt == BK_BF16, L.d, L.p, L.T, aligned16(L.x) && aligned16(L.g));
        // 256 x 256 tiles on the LDS-DMA kernel (one workgroup per sample and
        // tile) when the layer gives at least 128 of them: the wide kernel's
        // 256 x 128 tiles at two workgroups per CU fill the chip no better,
        // and below that it can split K.  Each sample is padded to 16-row
        // steps by at most 1/8, and B T rows stay below 2^31.
        if (v == bk::GemmVariant::Wide && L.T >= 64 && dl_padding_ok(L.T) && B * L.T < ((int64_t)1 << 31)) {
            const bk::GemmGeom dl = bk::gemm_geom(bk::GemmVariant::GradDL, L.d, L.p);
            if (B * dl.tm * dl.tn >= 128) v = bk::GemmVariant::GradDL;
        }
        const bk::GemmGeom geo = bk::gemm_geom(v, L.d, L.p);
        np.var = (int)v;
        np.tiles = geo.tm * geo.tn;
        np.tile_elems = geo.tile_elems;
        np.npart = np.tiles;
    } else {
        const int64_t nsb = cdiv(L.T, bk::kSuper);
        np.npart = nsb * (nsb + 1) / 2;
        const bool xv = np.path == Path::Embed || (aligned16(L.x) && (L.d * es) % 16 == 0);
        // The 16-byte path addresses one sample's rows (plus a super block of
        // padding) with 32-bit buffer offsets.
        const int64_t K = np.path == Path::Embed ? L.p : std::max(L.d, L.p);
        const bool fits = (L.T + bk::kSuper) * K * (int64_t)es < ((int64_t)1 << 31);
        np.var = (xv && fits && aligned16(L.g) && (L.p * es) % 16 == 0) ? 1 : 0;
        // bf16 16-byte rows with T > 128: the kernels over 256-row super
        // blocks (their 32-bit offsets reach 256 rows past T): 128 < T <= 256
        // streams every row once (one partial per sample); longer T has nsb
        // diagonal items and two half items per pair of super blocks.
        const bool fits256 = (L.T + 2 * bk::kSuper) * K * (int64_t)es < ((int64_t)1 << 31);
        if (np.var == 1 && np.path == Path::Ghost && dt == BK_BF16 && L.T > bk::kSuper && fits256) {
            const int64_t nsb = cdiv(L.T, bk::kLongSuper);
            np.var = L.T <= 2 * bk::kSuper ? 2 : 3;
            np.npart = np.var == 2 ? 1 : nsb * nsb;
        }
        // An embedding with rows of g in 16-byte multiples: the id join
        // (every row of g read once, no T x T work) instead of the masked
        // Gram, one partial per chunk of 8 ct columns of g (variant 2: ct =
        // 8, 3: ct = 32).
        if (np.path == Path::Embed && L.T >= 1 && L.T <= bk::kEmbedJoinMaxT && aligned16(L.g) && L.p % 8 == 0) {
            const int ct = bk::embed_join_ct(L.p);
            np.var = ct == 8 ? 2 : 3;
            np.npart = cdiv(L.p, 8 * ct);
        }
    }
}

// Workgroup count, and the K split of instantiated norms on the wide and
// narrow kernels (a split layer reports one partial per slice-reduction chunk).
void finish_norm_plan(NormPlan& np, const bk_layer& L, int64_t B) {
    if (np.path == Path::Inst && inst_splits(np.var)) {
        np.ksplit = inst_ksplit(B, np.tiles, L.T);
        if (np.ksplit > 1) np.npart = np.tiles * (np.tile_elems / bk::kSplitRedWG);
    }
    np.nwg = np.path == Path::Inst ? B * np.tiles * np.ksplit : B * np.npart;
    const bool affine = L.kind == BK_NORM_AFFINE || (L.kind == BK_LINEAR && (L.flags & BK_LAYER_BIAS));
    // A ghost layer on the 16-byte path with one 128-row block per sample
    // sums its bias terms while its g passes through LDS for the Gram.
    np.fused_bias = np.path == Path::Ghost && np.var == 1 && L.T > 0 && L.T <= bk::kSuper &&
                    L.kind == BK_LINEAR && (L.flags & BK_LAYER_BIAS) && L.p > 0;
    np.aff_chunks = affine && !np.fused_bias ? cdiv(L.p, bk::kAffineCols) : 0;
}

// Partial sums of a layer's norm (floats) and its K-split partial tiles (floats).
size_t norm_part_floats(const NormPlan& np, int64_t B) { return (size_t)(B * (np.npart + np.aff_chunks)); }
size_t norm_tile_floats(const NormPlan& np, int64_t B) {
    return np.ksplit > 1 ? (size_t)(B * np.tiles * np.ksplit * np.tile_elems) : 0;
}
size_t norm_ws_bytes(const NormPlan& np, int64_t B) {
    return align_up(norm_part_floats(np, B) * sizeof(float)) + norm_tile_floats(np, B) * sizeof(float);
}

// Launch of a ghost-norm variant (NormPlan::var) and the super-block count
// its descriptors carry.
hipError_t launch_ghost_var(const bk::GhostArgs& a, int n_wg, bool bf16, bool embed, int var, hipStream_t s) {
    if (embed && var >= 2) return bk::launch_embed_join(a, n_wg, bf16, var == 2 ? 8 : 32, s);
    return var >= 2 ? bk::launch_ghost_full(a, n_wg, var == 3, s) : bk::launch_ghost(a, n_wg, bf16, embed, var == 1, s);
}
int32_t ghost_nsb(int64_t T, int var) {
    return (int32_t)cdiv(T, var == 2 ? bk::kFullSub : var == 3 ? bk::kLongSuper : bk::kSuper);
}

// The layerwise decision of a linear layer: the paper's rule by space, or by
// time with BK_LAYER_TIME_RULE.
bool layer_ghost(const bk_layer& L) {
    return ((L.flags & BK_LAYER_TIME_RULE) ? bk_use_ghost_time(L.T, L.d, L.p) : bk_use_ghost(L.T, L.d, L.p)) == 1;
}

NormPlan norm_plan(const bk_layer& L, bk_dtype dt, int64_t B) {
    NormPlan np{};
    if (L.kind == BK_EMBEDDING) {
        np.path = Path::Embed;
    } else if (L.kind == BK_NORM_AFFINE) {
        np.path = Path::Affine;
    } else {
        np.path = layer_ghost(L) ? Path::Ghost : Path::Inst;
    }
    set_norm_variant(np, L, dt, B);
    finish_norm_plan(np, L, B);
    return np;
}

// The whole-sample ghost kernel (variant 2) runs one workgroup per CU and
// gives one per (layer, sample); a launch with fewer than kFullMinWG of them
// (few samples and few such layers) keeps those layers on the super-block
// pair kernel, which spreads three workgroups per sample over more CUs.
constexpr int64_t kFullMinWG = 512;
void demote_small_full(std::vector<NormPlan>& plans, const bk_layer* layers, int64_t B) {
    int64_t wg = 0;
    for (const NormPlan& np : plans) wg += np.path == Path::Ghost && np.var == 2 ? np.nwg : 0;
    if (wg == 0 || wg >= kFullMinWG) return;
    for (size_t l = 0; l < plans.size(); ++l) {
        NormPlan& np = plans[l];
        if (np.path != Path::Ghost || np.var != 2) continue;
        const int64_t nsb = cdiv(layers[l].T, bk::kSuper);
        np.var = 1;
        np.npart = nsb * (nsb + 1) / 2;
        finish_norm_plan(np, layers[l], B);
    }
}

// The norm plans of a launch's layers (norm_plan each, then the launch-wide
// choice of demote_small_full).
std::vector<NormPlan> norm_plans(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    std::vector<NormPlan> v;
    v.reserve((size_t)n);
    for (int64_t l = 0; l < n; ++l) v.push_back(norm_plan(layers[l], dt, B));
    demote_small_full(v, layers, B);
    return v;
}

size_t embed_grad_ws_bytes(int64_t B, int64_t T, int64_t p) { return bk::embed_grad_ws_bytes(B * T, p); }

// BK-MixOpt layer that keeps its instantiated per-sample gradients in P.
bool keeps_grads(const bk_layer& L) {
    return L.kind == BK_LINEAR && (L.flags & BK_LAYER_MIXOPT) && !layer_ghost(L);
}

bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

bk_status check_layer(const char* fn, const bk_layer& L, int64_t l, int64_t B, bool need_G) {
    if (L.kind != BK_LINEAR && L.kind != BK_EMBEDDING && L.kind != BK_NORM_AFFINE)
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld has unknown kind %d", fn, (long long)l, L.kind);
    if ((L.flags & ~(BK_LAYER_MIXOPT | BK_LAYER_BIAS | BK_LAYER_ACCUMULATE | BK_LAYER_TIME_RULE)) != 0)
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: unknown flags 0x%x", fn, (long long)l, L.flags);
    bk_status s = check_dims(fn, B, L.T, L.d, L.p);
    if (s != BK_OK) return s;
    const bool bias = (L.flags & BK_LAYER_BIAS) != 0;
    if (bias && L.kind == BK_EMBEDDING)
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: an embedding takes no bias", fn, (long long)l);
    if (L.kind == BK_NORM_AFFINE) {
        if (L.d != L.p)
            return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: affine layer needs d == p", fn, (long long)l);
        if (B * L.p > 0 && (!L.P || !aligned4(L.P)))
            return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: affine layer needs P [B,p] (4-byte aligned)", fn,
                        (long long)l);
    }
    if (bias && B * L.p > 0 && (!L.Pb || !aligned4(L.Pb)))
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: BK_LAYER_BIAS needs Pb [B,p] (4-byte aligned)", fn,
                    (long long)l);
    if (bias && need_G && L.p > 0 && (!L.Gb || !aligned4(L.Gb)))
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: BK_LAYER_BIAS needs Gb [p] (4-byte aligned)", fn,
                    (long long)l);
    if (keeps_grads(L) && B * L.d * L.p > 0) {
        if (!L.P)
            return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: BK_LAYER_MIXOPT needs P [B,d,p]", fn,
                        (long long)l);
        if ((reinterpret_cast<uintptr_t>(L.P) & 3u) != 0)
            return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: P not 4-byte aligned", fn, (long long)l);
        if (B > INT64_MAX / (L.d * L.p))
            return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: B*d*p overflows", fn, (long long)l);
    }
    const bool has_tokens = B > 0 && L.T > 0;
    if (has_tokens && (!L.x || (!L.g && L.p > 0)))
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: NULL input pointer", fn, (long long)l);
    if (need_G && !L.G && L.d * L.p > 0)
        return fail(BK_ERR_INVALID_VALUE, "%s: layer %lld: NULL gradient output", fn, (long long)l);
    if (L.kind == BK_EMBEDDING && need_G && B * L.T > bk::kEmbedMaxTokens)
        return fail(BK_ERR_NOT_SUPPORTED,
                    "%s: layer %lld: embedding gradient supports at most %lld tokens per call (B*T=%lld)",
                    fn, (long long)l, (long long)bk::kEmbedMaxTokens, (long long)(B * L.T));
    return BK_OK;
}

// ---------------------------------------------------------------------------
// Grouped execution
// ---------------------------------------------------------------------------
size_t layer_norms_ws(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    size_t tot = 0;
    for (const NormPlan& np : norm_plans(layers, n, dt, B)) tot += norm_ws_bytes(np, B);
    return tot;
}

bk_status layer_norms(const char* fn, const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B,
                      float* norm_sq, void* ws, size_t ws_bytes, hipStream_t s) {
    if (n < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative layer count", fn);
    if (n > 0 && !layers) return fail(BK_ERR_INVALID_VALUE, "%s: NULL layer array", fn);
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    if (B < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative batch", fn);
    for (int64_t l = 0; l < n; ++l)
        if ((st = check_layer(fn, layers[l], l, B, false)) != BK_OK) return st;
    if (n * B > 0 && !norm_sq) return fail(BK_ERR_INVALID_VALUE, "%s: NULL norm output", fn);
    const size_t need = layer_norms_ws(layers, n, dt, B);
    if (ws_bytes < need || (need > 0 && !ws))
        return fail(BK_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    if ((size_t)need / sizeof(float) > (size_t)INT32_MAX)
        return fail(BK_ERR_NOT_SUPPORTED, "%s: too many partial sums", fn);
    if (n == 0 || B == 0) return BK_OK;

    float* part = static_cast<float*>(ws);
    const bool bf16 = dt == BK_BF16;

    // Batches of same-kernel layers; each batch is one launch.  Workspace:
    // every layer's partial sums (aligned runs), then the K-split partial
    // tiles of the split instantiated layers.
    struct Item { int64_t l; NormPlan np; int64_t part_off; int64_t tile_off; };
    std::vector<Item> items;
    items.reserve((size_t)n);
    int64_t off = 0, toff = 0;
    const std::vector<NormPlan> plans = norm_plans(layers, n, dt, B);
    for (int64_t l = 0; l < n; ++l) {
        const NormPlan& np = plans[(size_t)l];
        items.push_back({l, np, off, toff});
        off += (int64_t)(align_up(norm_part_floats(np, B) * sizeof(float)) / sizeof(float));
        toff += (int64_t)norm_tile_floats(np, B);
    }
    float* tiles = part + off;

    auto flush_ghost = [&](std::vector<const Item*>& v, bool embed, int var) -> bk_status {
        if (v.empty()) return BK_OK;
        bk::GhostArgs a{};
        a.n = (int32_t)v.size();
        a.B = (int32_t)B;
        a.part = part;
        // One super-block pair per sample (T <= 128): no L2 reuse to keep on
        // an XCD, and the workgroups' sizes differ by layer (rows of d + p
        // values), so the layers go largest first and the hardware deals the
        // grid round-robin over the XCDs: each XCD gets the same mix and the
        // last round holds the small ones.  (A contiguous share per XCD in
        // stack order left the XCDs up to ~20% apart in bytes.)
        a.remap = 0;
        for (const Item* it : v) a.remap |= it->np.npart > 1 ? 1 : 0;
        if (!a.remap)
            std::stable_sort(v.begin(), v.end(), [&](const Item* x, const Item* y) {
                auto cost = [&](const Item* it) {
                    const bk_layer& L = layers[it->l];
                    return (embed ? 0 : L.d) + L.p;
                };
                return cost(x) > cost(y);
            });
        int64_t wg = 0;
        for (size_t k = 0; k < v.size(); ++k) {
            const bk_layer& L = layers[v[k]->l];
            bk::GhostLayer& g = a.L[k];
            g.x = L.x;
            g.g = L.g;
            g.T = (int32_t)L.T;
            g.d = (int32_t)L.d;
            g.p = (int32_t)L.p;
            g.nsb = ghost_nsb(L.T, var);
            g.npairs = (int32_t)v[k]->np.npart;
            g.wg_begin = (int32_t)wg;
            g.part_off = (int32_t)v[k]->part_off;
            g.Pb = v[k]->np.fused_bias ? L.Pb : nullptr;
            wg += v[k]->np.nwg;
        }
        if (wg > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
        hipError_t e = launch_ghost_var(a, (int)wg, bf16, embed, var, s);
        v.clear();
        return e == hipSuccess ? BK_OK : hip_fail(e, "ghost norm launch");
    };
    auto flush_inst = [&](std::vector<const Item*>& v, int var) -> bk_status {
        if (v.empty()) return BK_OK;
        bk::GemmArgs a{};
        a.n = (int32_t)v.size();
        a.B = (int32_t)B;
        a.C = nullptr;
        a.part = part;
        a.tiles = tiles;
        int64_t wg = 0, red = 0;
        for (size_t k = 0; k < v.size(); ++k) {
            const bk_layer& L = layers[v[k]->l];
            const NormPlan& np = v[k]->np;
            bk::GemmLayer& g = a.L[k];
            g.a = L.x;
            g.g = L.g;
            g.G = keeps_grads(L) ? L.P : nullptr;
            g.T = (int32_t)L.T;
            g.d = (int32_t)L.d;
            g.p = (int32_t)L.p;
            const bk::GemmGeom geo = bk::gemm_geom(bk::GemmVariant(var), L.d, L.p);
            g.tm = (int32_t)geo.tm;
            g.tn = (int32_t)geo.tn;
            g.swap = geo.swap ? 1 : 0;
            g.wg_begin = (int32_t)wg;
            g.part_off = (int32_t)v[k]->part_off;
            g.ksplit = (int32_t)np.ksplit;
            g.ptile_off = v[k]->tile_off;
            g.red_begin = (int32_t)red;
            wg += np.nwg;
            if (np.ksplit > 1) red += B * np.tiles * (np.tile_elems / bk::kSplitRedWG);
        }
        if (wg > INT32_MAX || red > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
        hipError_t e = bk::launch_gemm(a, (int)wg, bf16, true, bk::GemmVariant(var), s);
        if (e == hipSuccess && red > 0)
            e = bk::launch_split_reduce(a, (int)red, true, bk::GemmVariant(var), s);
        v.clear();
        return e == hipSuccess ? BK_OK : hip_fail(e, "instantiated norm launch");
    };

    // Group by (path, kernel variant), preserving layer order inside a group;
    // a group larger than one launch's descriptor table is cut into launches
    // of near-equal layer counts (no small last launch).
    for (int kind = 0; kind < 3; ++kind)
        for (int var = 0; var < (kind == 2 ? bk::kGemmVariants : 4); ++var) {
            const Path want = kind == 0 ? Path::Ghost : kind == 1 ? Path::Embed : Path::Inst;
            std::vector<const Item*> all;
            for (const Item& it : items)
                if (it.np.path == want && it.np.var == var && it.np.nwg > 0) all.push_back(&it);
            const size_t cap = kind == 2 ? bk::kMaxGemm : bk::kMaxGhost;
            const size_t nb = (all.size() + cap - 1) / cap;
            for (size_t b = 0; b < nb; ++b) {
                std::vector<const Item*> batch(all.begin() + (std::ptrdiff_t)(all.size() * b / nb),
                                               all.begin() + (std::ptrdiff_t)(all.size() * (b + 1) / nb));
                st = kind == 2 ? flush_inst(batch, var) : flush_ghost(batch, kind == 1, var);
                if (st != BK_OK) return st;
            }
        }

    // Per-sample bias / affine sums of the layers that have them (their
    // partials follow the layer's weight partials).
    {
        bk::AffineArgs a{};
        a.B = (int32_t)B;
        a.part = part;
        int64_t wg = 0;
        auto flush = [&]() -> bk_status {
            if (a.n == 0) return BK_OK;
            if (wg > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
            hipError_t e = bk::launch_affine(a, (int)wg, bf16, s);
            a.n = 0;
            wg = 0;
            return e == hipSuccess ? BK_OK : hip_fail(e, "bias / affine sums launch");
        };
        for (const Item& it : items) {
            if (it.np.aff_chunks == 0) continue;
            const bk_layer& L = layers[it.l];
            const bool affine = L.kind == BK_NORM_AFFINE;
            const size_t es = elem_bytes(dt);
            bk::AffineLayer& f = a.L[a.n++];
            f.x = affine ? L.x : nullptr;
            f.g = L.g;
            f.P = affine ? L.P : nullptr;
            f.Pb = (L.flags & BK_LAYER_BIAS) ? L.Pb : nullptr;
            f.T = (int32_t)L.T;
            f.p = (int32_t)L.p;
            f.chunks = (int32_t)it.np.aff_chunks;
            f.wg_begin = (int32_t)wg;
            f.part_off = (int32_t)(it.part_off + B * it.np.npart);
            f.vec = (aligned16(L.g) && (!affine || aligned16(L.x)) && (L.p * (int64_t)es) % 16 == 0 &&
                     L.p % 8 == 0) ? 1 : 0;
            f.gamma = affine ? 1 : 0;
            wg += B * it.np.aff_chunks;
            if (a.n == bk::kMaxAffine && (st = flush()) != BK_OK) return st;
        }
        if ((st = flush()) != BK_OK) return st;
    }

    // Finish every layer's norms with the fixed-order reduction.
    for (int64_t l0 = 0; l0 < n; l0 += bk::kMaxReduce) {
        const int64_t cnt = std::min<int64_t>(bk::kMaxReduce, n - l0);
        bk::ReduceArgs r{};
        r.n = (int32_t)cnt;
        r.B = (int32_t)B;
        r.part = part;
        for (int64_t k = 0; k < cnt; ++k) {
            const Item& it = items[(size_t)(l0 + k)];
            r.L[k].out = norm_sq + (l0 + k) * B;
            r.L[k].part_off = (int32_t)it.part_off;
            r.L[k].npart = (int32_t)it.np.npart;
            r.L[k].part_off2 = (int32_t)(it.part_off + B * it.np.npart);
            r.L[k].npart2 = (int32_t)it.np.aff_chunks;
        }
        hipError_t e = bk::launch_reduce(r, (int)(cnt * B), s);
        if (e != hipSuccess) return hip_fail(e, "norm reduction launch");
    }
    return BK_OK;
}

// Kernel variant of a linear layer's clipped gradient: narrow layers with
// T >= 64 run on the narrow kernel (shorter T on the wide one), the other
// Wide layers with T >= 64 on the 256 x 256 kernels, with the weights on the
// accumulators when B fits the kernel's LDS table and padding each sample to
// 16-row steps adds at most 1/8 to its rows, else on g.
bk::GemmVariant grad_variant(const bk_layer& L, bool bf16, int64_t B) {
    const auto v = bk::gemm_variant(bf16, L.d, L.p, B * L.T, aligned16(L.x) && aligned16(L.g));
    if (is_narrow(v)) return L.T < 64 ? bk::GemmVariant::Wide : v;   // narrow kernel: T >= 64
    if (v != bk::GemmVariant::Wide || L.T < 64) return v;
    if (dl_padding_ok(L.T) && B <= bk::kDMaxB) return bk::GemmVariant::GradDL;
    // The register-staged 256 x 256 kernel addresses all B T rows (and three
    // stages of 64 past them) with 32-bit offsets; longer layers take the
    // wide kernel, which addresses one stage at a time.
    const bool fits = (B * L.T + 3 * 64) * std::max(L.d, L.p) * (bf16 ? 2 : 4) < ((int64_t)1 << 31);
    return fits ? bk::GemmVariant::Grad : bk::GemmVariant::Wide;
}

// Tiles and K slices of a linear layer's clipped gradient on variant v
// (split_from > 0: only the tiles from split_from on are K-split).
struct GradPlan {
    int64_t tm, tn, ksplit, tile_elems;
    bool swap;
    int64_t split_from = 0;
    bool tail = false;   // the K-split tiles are a launch's tail (plan_tail)
    int64_t tiles() const { return tm * tn; }
    int64_t split_tiles() const { return ksplit > 1 ? tm * tn - split_from : 0; }
    int64_t wgs() const { return split_from + (tm * tn - split_from) * ksplit; }
};
GradPlan grad_plan(const bk_layer& L, bk::GemmVariant v, int64_t B) {
    const bk::GemmGeom geo = bk::gemm_geom(v, L.d, L.p);
    GradPlan g{geo.tm, geo.tn, 1, geo.tile_elems, geo.swap};
    if (v == bk::GemmVariant::Grad || v == bk::GemmVariant::GradDL) {
        const int64_t nst = v == bk::GemmVariant::Grad ? cdiv(B * L.T, 64) : B * dl_stages_per_sample(L.T);
        g.ksplit = grad_ksplit(g.tm * g.tn, nst);
    } else if (is_narrow(v)) {
        g.ksplit = narrow_grad_ksplit(g.tm * g.tn, cdiv(B * L.T, 64));
    }
    return g;
}

// Compute units of the current device (256, MI355X's, when there is none to
// ask, e.g. for a workspace query on a host without a GPU).
int64_t device_cus() {
    constexpr int kMaxDev = 64;
    static std::atomic<int> cache[kMaxDev];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        return 256;
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

// One grouped clipped-gradient launch: layers of one kernel variant, in
// launch order.
struct GradEntry { int64_t l; GradPlan gp; };
struct GradGroup { bk::GemmVariant v; std::vector<GradEntry> e; };

constexpr int64_t kTailMinStages = 8;    // stages per slice of a split tail tile, at least
constexpr int64_t kTailMaxSplit = 16;    // K slices per tail tile, at most

// The 256 x 256 clipped-gradient kernels (Grad, GradDL) hold one workgroup
// per CU, so a launch of N tiles of equal work runs in ceil(N / cus) rounds.
// When the last round is at most half full (r = N mod cus tiles), those r
// tiles are cut into s = cus / r K slices each (at most kTailMaxSplit, of
// at least kTailMinStages stages) and moved behind every other tile in
// launch order: the slices are dispatched last and fill the CUs together
// once the full rounds are done.  They are taken from the layer with the
// most tiles, which goes last.
void plan_tail(GradGroup& g, const bk_layer* layers, int64_t B, int64_t cus) {
    if (g.e.empty()) return;
    const int64_t T0 = layers[g.e[0].l].T;
    int64_t N = 0;
    size_t best = 0;
    for (size_t k = 0; k < g.e.size(); ++k) {
        if (g.e[k].gp.ksplit != 1 || layers[g.e[k].l].T != T0) return;   // unequal work
        N += g.e[k].gp.tiles();
        if (g.e[k].gp.tiles() > g.e[best].gp.tiles()) best = k;
    }
    const int64_t r = N % cus;
    if (r == 0 || 2 * r > cus || g.e[best].gp.tiles() < r) return;
    const int64_t nst = g.v == bk::GemmVariant::GradDL ? B * dl_stages_per_sample(T0) : cdiv(B * T0, 64);
    const int64_t sp = std::min({cus / r, nst / kTailMinStages, kTailMaxSplit});
    if (sp < 2) return;
    std::rotate(g.e.begin() + (std::ptrdiff_t)best, g.e.begin() + (std::ptrdiff_t)best + 1, g.e.end());
    GradPlan& gp = g.e.back().gp;
    gp.ksplit = sp;
    gp.split_from = gp.tiles() - r;
    gp.tail = true;
}

// The grouped launches of bk_weighted_grads: by kernel variant, at most
// kMaxGemm layers each.
std::vector<GradGroup> grad_groups(const bk_layer* layers, int64_t n, bool bf16, int64_t B) {
    std::vector<GradGroup> out;
    for (int var = 0; var < bk::kGemmVariants; ++var) {
        for (int64_t l = 0; l < n; ++l) {
            const bk_layer& L = layers[l];
            if (L.kind != BK_LINEAR || L.d * L.p == 0 || keeps_grads(L)) continue;
            const auto v = grad_variant(L, bf16, B);
            if ((int)v != var) continue;
            if (out.empty() || out.back().v != v || (int64_t)out.back().e.size() == bk::kMaxGemm)
                out.push_back(GradGroup{v, {}});
            out.back().e.push_back(GradEntry{l, grad_plan(L, v, B)});
        }
    }
    int64_t cus = 0;
    for (GradGroup& g : out)
        if (g.v == bk::GemmVariant::GradDL || g.v == bk::GemmVariant::Grad) {
            if (cus == 0) cus = device_cus();
            plan_tail(g, layers, B, cus);
        }
    return out;
}

size_t weighted_grads_ws(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    size_t tot = 0;
    for (int64_t l = 0; l < n; ++l)
        if (layers[l].kind == BK_EMBEDDING) tot = std::max(tot, embed_grad_ws_bytes(B, layers[l].T, layers[l].p));
    // Grouped launches follow each other on the stream: each one's partial
    // tiles start at the workspace's beginning.
    for (const GradGroup& g : grad_groups(layers, n, dt == BK_BF16, B)) {
        size_t tiles = 0;
        for (const GradEntry& e : g.e)
            tiles += (size_t)(e.gp.split_tiles() * e.gp.ksplit * e.gp.tile_elems) * sizeof(float);
        tot = std::max(tot, tiles);
    }
    return tot;
}

// Appends one weighted-sum job (P [B, n] -> G [n]) to a grouped launch.
bk_status add_wsum_layer(bk::WsumArgs& w, int64_t& wg, const float* P, float* G, int64_t n, bool accum) {
    bk::WsumLayer& L = w.L[w.n++];
    L.P = P;
    L.G = G;
    L.n = n;
    L.wg_begin = (uint32_t)wg;
    L.vec = (aligned16(P) && aligned16(G) && n % 4 == 0) ? 1u : 0u;
    L.accum = accum ? 1u : 0u;
    wg += cdiv(n, bk::kWsumPerWG);
    return BK_OK;
}

bk_status weighted_grads(const char* fn, const bk_layer* layers, int64_t n, const float* C,
                         bk_dtype dt, int64_t B, void* ws, size_t ws_bytes, hipStream_t s) {
    if (n < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative layer count", fn);
    if (n > 0 && !layers) return fail(BK_ERR_INVALID_VALUE, "%s: NULL layer array", fn);
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    if (B < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative batch", fn);
    for (int64_t l = 0; l < n; ++l)
        if ((st = check_layer(fn, layers[l], l, B, true)) != BK_OK) return st;
    if (B > 0 && !C) return fail(BK_ERR_INVALID_VALUE, "%s: NULL clip factors", fn);
    const size_t need = weighted_grads_ws(layers, n, dt, B);
    if (ws_bytes < need || (need > 0 && !ws))
        return fail(BK_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    const bool bf16 = dt == BK_BF16;

    // Grouped launches by kernel variant.  Layers with few output tiles run
    // K-split (grad_plan), and so do the tiles of a 256 x 256 launch's last,
    // partly filled round (plan_tail); the partial tiles sit in the
    // workspace (launches follow each other on the stream, so each starts
    // from offset 0).
    for (const GradGroup& grp : grad_groups(layers, n, bf16, B)) {
        bk::GemmArgs a{};
        a.B = (int32_t)B;
        a.C = C;
        a.part = nullptr;
        a.tiles = static_cast<float*>(ws);
        int64_t wg = 0, ptile = 0, red = 0, remap = 0;
        for (const GradEntry& e : grp.e) {
            const bk_layer& L = layers[e.l];
            const GradPlan& gp = e.gp;
            bk::GemmLayer& g = a.L[a.n++];
            g.a = L.x;
            g.g = L.g;
            g.G = L.G;
            // With no tokens (B*T == 0) the tiles still run, writing zeros.
            g.T = (int32_t)L.T;
            g.d = (int32_t)L.d;
            g.p = (int32_t)L.p;
            g.tm = (int32_t)gp.tm;
            g.tn = (int32_t)gp.tn;
            g.wg_begin = (int32_t)wg;
            g.part_off = 0;
            g.ksplit = (int32_t)gp.ksplit;
            g.split_from = (int32_t)gp.split_from;
            g.swap = gp.swap ? 1 : 0;
            g.accum = (L.flags & BK_LAYER_ACCUMULATE) ? 1 : 0;
            g.ptile_off = ptile;
            g.red_begin = (int32_t)red;
            if (gp.tail) remap = wg + gp.split_from;   // the last layer; its slices run last
            wg += gp.wgs();
            if (gp.ksplit > 1) {
                ptile += gp.split_tiles() * gp.ksplit * gp.tile_elems;
                red += gp.split_tiles() * (gp.tile_elems / bk::kSplitRedWG);
            }
        }
        if (wg > INT32_MAX || red > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
        hipError_t e = bk::launch_gemm(a, (int)wg, bf16, false, grp.v, s, (int)remap);
        if (e == hipSuccess && red > 0) e = bk::launch_split_reduce(a, (int)red, false, grp.v, s);
        if (e != hipSuccess) return hip_fail(e, "clipped gradient launch");
    }
    // Weighted sums of stored per-sample gradients: BK-MixOpt weights, the
    // gammas of affine layers, and every bias / beta.
    {
        bk::WsumArgs w{};
        w.B = (int32_t)B;
        w.C = C;
        int64_t wg = 0;
        auto flush = [&]() -> bk_status {
            if (w.n == 0) return BK_OK;
            if (wg > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
            hipError_t e = bk::launch_wsum(w, (int)wg, s);
            w.n = 0;
            wg = 0;
            return e == hipSuccess ? BK_OK : hip_fail(e, "weighted sum launch");
        };
        for (int64_t l = 0; l < n; ++l) {
            const bk_layer& L = layers[l];
            const bool acc = (L.flags & BK_LAYER_ACCUMULATE) != 0;
            if ((keeps_grads(L) || L.kind == BK_NORM_AFFINE) && L.d * L.p > 0) {
                const int64_t ne = L.kind == BK_NORM_AFFINE ? L.p : L.d * L.p;
                if ((st = add_wsum_layer(w, wg, L.P, L.G, ne, acc)) != BK_OK) return st;
                if (w.n == bk::kMaxWsum && (st = flush()) != BK_OK) return st;
            }
            if ((L.flags & BK_LAYER_BIAS) && L.p > 0) {
                if ((st = add_wsum_layer(w, wg, L.Pb, L.Gb, L.p, acc)) != BK_OK) return st;
                if (w.n == bk::kMaxWsum && (st = flush()) != BK_OK) return st;
            }
        }
        if ((st = flush()) != BK_OK) return st;
    }
    for (int64_t l = 0; l < n; ++l) {
        const bk_layer& L = layers[l];
        if (L.kind != BK_EMBEDDING || L.d * L.p == 0) continue;
        hipError_t e = bk::launch_embed_grad(static_cast<const int64_t*>(L.x), L.g, C, bf16, B, L.T,
                                             L.p, L.d, L.G, ws, (L.flags & BK_LAYER_ACCUMULATE) != 0, s);
        if (e != hipSuccess) return hip_fail(e, "embedding gradient launch");
    }
    return BK_OK;
}

bk_status add_noise_layers(const char* fn, float* const* G, const int64_t* nel,
                           const uint32_t* tensor_id, int64_t n, float std, uint64_t seed,
                           uint32_t step, hipStream_t s) {
    bk::NoiseArgs a{};
    a.std = std;
    a.seed = seed;
    a.step = step;
    // Workgroup grain: 256 counter blocks each while the whole call has
    // fewer than 2048 such groups, up to kNoiseBlocksPerWG for large calls.
    int64_t total_q = 0;
    for (int64_t l = 0; l < n; ++l) total_q += cdiv(nel[l], 4);
    a.bpw = 256u * (uint32_t)std::min<int64_t>(bk::kNoiseBlocksPerWG / 256, std::max<int64_t>(1, cdiv(total_q, 256 * 2048)));
    int64_t wg = 0;
    auto flush = [&]() -> bk_status {
        if (a.n == 0) return BK_OK;
        if (wg > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
        hipError_t e = bk::launch_noise(a, (int)wg, s);
        a.n = 0;
        wg = 0;
        return e == hipSuccess ? BK_OK : hip_fail(e, "noise launch");
    };
    for (int64_t l = 0; l < n; ++l) {
        if (nel[l] == 0) continue;
        bk::NoiseLayer& L = a.L[a.n++];
        L.G = G[l];
        L.n = nel[l];
        L.tensor_id = tensor_id[l];
        L.wg_begin = (uint32_t)wg;
        wg += cdiv(cdiv(nel[l], 4), (int64_t)a.bpw);
        if (a.n == bk::kMaxNoise) {
            bk_status st = flush();
            if (st != BK_OK) return st;
        }
    }
    return flush();
}

bk_layer linear_layer(const void* a, const void* g, int64_t T, int64_t d, int64_t p, float* G) {
    bk_layer L{};
    L.kind = BK_LINEAR;
    L.T = T;
    L.d = d;
    L.p = p;
    L.x = a;
    L.g = g;
    L.G = G;
    return L;
}

bk_layer embed_layer(const int64_t* ids, const void* g, int64_t T, int64_t V, int64_t p, float* G) {
    bk_layer L{};
    L.kind = BK_EMBEDDING;
    L.T = T;
    L.d = V;
    L.p = p;
    L.x = ids;
    L.g = g;
    L.G = G;
    return L;
}

// Single-layer norm with a forced path (the grouped call picks it by rule).
bk_status single_norm(const char* fn, Path want, const bk_layer& L, bk_dtype dt, int64_t B,
                      float* norm_sq, void* ws, size_t ws_bytes, hipStream_t s) {
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    if ((st = check_layer(fn, L, 0, B, false)) != BK_OK) return st;
    if (B > 0 && !norm_sq) return fail(BK_ERR_INVALID_VALUE, "%s: NULL norm output", fn);
    std::vector<NormPlan> one(1);
    one[0].path = want;
    set_norm_variant(one[0], L, dt, B);
    finish_norm_plan(one[0], L, B);
    demote_small_full(one, &L, B);
    const NormPlan np = one[0];
    const size_t need = norm_ws_bytes(np, B);
    if (ws_bytes < need || (need > 0 && !ws))
        return fail(BK_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    if (B == 0) return BK_OK;
    float* part = static_cast<float*>(ws);
    hipError_t e = hipSuccess;
    if (np.nwg > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
    if (want == Path::Inst) {
        bk::GemmArgs a{};
        a.n = 1;
        a.B = (int32_t)B;
        a.part = part;
        bk::GemmLayer& g = a.L[0];
        g.a = L.x;
        g.g = L.g;
        g.G = (L.flags & BK_LAYER_MIXOPT) ? L.P : nullptr;
        g.T = (int32_t)L.T;
        g.d = (int32_t)L.d;
        g.p = (int32_t)L.p;
        const bk::GemmGeom geo = bk::gemm_geom(bk::GemmVariant(np.var), L.d, L.p);
        g.tm = (int32_t)geo.tm;
        g.tn = (int32_t)geo.tn;
        g.swap = geo.swap ? 1 : 0;
        g.ksplit = (int32_t)np.ksplit;
        a.tiles = part + align_up(norm_part_floats(np, B) * sizeof(float)) / sizeof(float);
        e = bk::launch_gemm(a, (int)np.nwg, dt == BK_BF16, true, bk::GemmVariant(np.var), s);
        const int64_t red = np.ksplit > 1 ? B * np.tiles * (np.tile_elems / bk::kSplitRedWG) : 0;
        if (red > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
        if (e == hipSuccess && red > 0)
            e = bk::launch_split_reduce(a, (int)red, true, bk::GemmVariant(np.var), s);
    } else {
        bk::GhostArgs a{};
        a.n = 1;
        a.B = (int32_t)B;
        a.remap = np.npart > 1 ? 1 : 0;
        a.part = part;
        bk::GhostLayer& g = a.L[0];
        g.x = L.x;
        g.g = L.g;
        g.T = (int32_t)L.T;
        g.d = (int32_t)L.d;
        g.p = (int32_t)L.p;
        g.nsb = ghost_nsb(L.T, np.var);
        g.npairs = (int32_t)np.npart;
        e = launch_ghost_var(a, (int)np.nwg, dt == BK_BF16, want == Path::Embed, np.var, s);
    }
    if (e != hipSuccess) return hip_fail(e, "norm launch");
    bk::ReduceArgs r{};
    r.n = 1;
    r.B = (int32_t)B;
    r.part = part;
    r.L[0].out = norm_sq;
    r.L[0].part_off = 0;
    r.L[0].npart = (int32_t)np.npart;
    e = bk::launch_reduce(r, (int)B, s);
    return e == hipSuccess ? BK_OK : hip_fail(e, "norm reduction launch");
}

}  // namespace

extern "C" {

int bk_use_ghost(int64_t T, int64_t d, int64_t p) {
    if (T < 0 || d < 0 || p < 0) return -1;
    // 2 T^2 < p d, evaluated without overflow (128-bit products).
    const __int128 lhs = (__int128)2 * T * T;
    const __int128 rhs = (__int128)p * d;
    return lhs < rhs ? 1 : 0;
}

int bk_use_ghost_time(int64_t T, int64_t d, int64_t p) {
    if (T < 0 || d < 0 || p < 0) return -1;
    // T (p + d) < p d in 128-bit arithmetic (p + d < 2^64, T < 2^63).
    const __int128 lhs = (__int128)T * ((__int128)p + d);
    const __int128 rhs = (__int128)p * d;
    return lhs < rhs ? 1 : 0;
}

size_t bk_workspace_size(bk_op op, bk_dtype dt, int64_t B, int64_t T, int64_t d, int64_t p) {
    if (check_dtype("bk_workspace_size", dt) != BK_OK) return 0;
    if (check_dims("bk_workspace_size", B, T, d, p) != BK_OK) return 0;
    bk_layer L{};
    L.T = T;
    L.d = d;
    L.p = p;
    switch (op) {
        case BK_OP_GHOST_NORM:
        case BK_OP_EMBED_GHOST_NORM: {
            // super-block pairs (an upper bound over the ghost kernels), or
            // the id join's column chunks when it applies (NULL pointers
            // count as aligned): the larger of the two, since the alignment
            // of the caller's g is not known here
            const int64_t nsb = cdiv(T, bk::kSuper);
            int64_t npart = nsb * (nsb + 1) / 2;
            if (op == BK_OP_EMBED_GHOST_NORM) {
                L.kind = BK_EMBEDDING;
                NormPlan np{};
                np.path = Path::Embed;
                set_norm_variant(np, L, dt, B);
                npart = std::max(npart, np.npart);
            }
            return align_up((size_t)(B * npart) * sizeof(float));
        }
        case BK_OP_INST_NORM: {  // upper bound over the kernels (alignment is not known here)
            const size_t small = align_up((size_t)(B * cdiv(d, bk::kTile) * cdiv(p, bk::kTile)) * sizeof(float));
            L.kind = BK_LINEAR;
            NormPlan np{};
            np.path = Path::Inst;
            set_norm_variant(np, L, dt, B);  // NULL pointers count as aligned
            finish_norm_plan(np, L, B);
            return std::max(small, norm_ws_bytes(np, B));
        }
        case BK_OP_WEIGHTED_GRAD:   // 16-byte aligned rows assumed (an upper bound)
            L.kind = BK_LINEAR;
            return weighted_grads_ws(&L, 1, dt, B);
        case BK_OP_EMBED_WEIGHTED_GRAD:
            return embed_grad_ws_bytes(B, T, p);
        default:
            return 0;
    }
}

bk_status bk_ghost_norm(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T, int64_t d,
                        int64_t p, float* norm_sq, void* ws, size_t ws_bytes, void* stream) {
    return single_norm("bk_ghost_norm", Path::Ghost, linear_layer(a, g, T, d, p, nullptr), dt, B,
                       norm_sq, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

bk_status bk_inst_norm(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T, int64_t d,
                       int64_t p, float* norm_sq, void* ws, size_t ws_bytes, void* stream) {
    return single_norm("bk_inst_norm", Path::Inst, linear_layer(a, g, T, d, p, nullptr), dt, B,
                       norm_sq, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

bk_status bk_per_sample_grads(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T,
                              int64_t d, int64_t p, float* norm_sq, float* P, void* ws,
                              size_t ws_bytes, void* stream) {
    const char* fn = "bk_per_sample_grads";
    bk_status st = check_dims(fn, B, T, d, p);
    if (st != BK_OK) return st;
    if (B * d * p > 0) {
        if (!P) return fail(BK_ERR_INVALID_VALUE, "%s: NULL per-sample gradient output", fn);
        if ((reinterpret_cast<uintptr_t>(P) & 3u) != 0)
            return fail(BK_ERR_INVALID_VALUE, "%s: P not 4-byte aligned", fn);
        if (B > INT64_MAX / (d * p)) return fail(BK_ERR_INVALID_VALUE, "%s: B*d*p overflows", fn);
    }
    bk_layer L = linear_layer(a, g, T, d, p, nullptr);
    L.P = P;
    L.flags = BK_LAYER_MIXOPT;
    // The layer may satisfy the ghost rule; the explicit call instantiates anyway.
    bk_layer Lc = L;
    Lc.flags = 0;
    if ((st = check_layer(fn, Lc, 0, B, false)) != BK_OK) return st;
    return single_norm(fn, Path::Inst, L, dt, B, norm_sq, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

bk_status bk_weighted_sum(const float* P, const float* C, int64_t B, int64_t n, float* G, void* stream) {
    const char* fn = "bk_weighted_sum";
    if (B < 0 || n < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (B > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: batch too large", fn);
    if (n == 0) return BK_OK;
    if (!G) return fail(BK_ERR_INVALID_VALUE, "%s: NULL output", fn);
    if (B > 0 && (!P || !C)) return fail(BK_ERR_INVALID_VALUE, "%s: NULL input", fn);
    if (B > 0 && n > INT64_MAX / B) return fail(BK_ERR_INVALID_VALUE, "%s: B*n overflows", fn);
    if (((reinterpret_cast<uintptr_t>(P) | reinterpret_cast<uintptr_t>(C) | reinterpret_cast<uintptr_t>(G)) & 3u) != 0)
        return fail(BK_ERR_INVALID_VALUE, "%s: pointers must be 4-byte aligned", fn);
    if (cdiv(n, bk::kWsumPerWG) > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: too many elements", fn);
    bk::WsumArgs w{};
    w.B = (int32_t)B;
    w.C = C;
    int64_t wg = 0;
    add_wsum_layer(w, wg, P, G, n, false);
    hipError_t e = bk::launch_wsum(w, (int)wg, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "weighted sum launch");
}

namespace {

// Shape checks of one unfold (App. B): fills sh on success.
bk_status check_unfold(const char* fn, int64_t B, int64_t C, int64_t H, int64_t W, int64_t kh, int64_t kw,
                       int64_t stride, int64_t pad, int64_t ld, bk::UnfoldShape* sh) {
    if (B < 0 || C < 0 || H < 0 || W < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (kh < 1 || kw < 1 || stride < 1 || pad < 0)
        return fail(BK_ERR_INVALID_VALUE, "%s: kernel, stride >= 1 and pad >= 0 required", fn);
    if (H > (1 << 20) || W > (1 << 20) || kh > (1 << 20) || kw > (1 << 20) || pad > (1 << 20) || C > (1 << 24))
        return fail(BK_ERR_NOT_SUPPORTED, "%s: dimensions too large", fn);
    const int64_t Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if (H + 2 * pad < kh || W + 2 * pad < kw || Ho < 1 || Wo < 1)
        return fail(BK_ERR_INVALID_VALUE, "%s: kernel larger than the padded image", fn);
    const int64_t d = C * kh * kw;
    if (ld < d) return fail(BK_ERR_INVALID_VALUE, "%s: ld %lld < C kh kw = %lld", fn, (long long)ld, (long long)d);
    const int64_t T = Ho * Wo;
    if (B > 0 && T > INT64_MAX / B / std::max<int64_t>(ld, 1))
        return fail(BK_ERR_INVALID_VALUE, "%s: output size overflows", fn);
    *sh = bk::UnfoldShape{B, C, H, W, kh, kw, stride, pad, Ho, Wo, T, ld};
    return BK_OK;
}

bk_status check_tokens(const char* fn, int64_t B, int64_t C, int64_t HW) {
    if (B < 0 || C < 0 || HW < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (B > 65535 || C > ((int64_t)1 << 36) || HW > ((int64_t)1 << 36))
        return fail(BK_ERR_NOT_SUPPORTED, "%s: dimensions too large", fn);
    if ((HW + 31) / 32 > INT32_MAX || (C + 31) / 32 > 65535)
        return fail(BK_ERR_NOT_SUPPORTED, "%s: grid too large", fn);
    return BK_OK;
}

}  // namespace

bk_status bk_unfold(const void* x, bk_dtype dt, int64_t B, int64_t C, int64_t H, int64_t W,
                    int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t ld, void* a,
                    void* stream) {
    const char* fn = "bk_unfold";
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    bk::UnfoldShape sh{};
    if ((st = check_unfold(fn, B, C, H, W, kh, kw, stride, pad, ld, &sh)) != BK_OK) return st;
    if (B * sh.T * ld == 0) return BK_OK;
    if (!x || !a) return fail(BK_ERR_INVALID_VALUE, "%s: NULL pointer", fn);
    hipError_t e = bk::launch_unfold(x, a, sh, dt == BK_BF16, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "unfold launch");
}

bk_status bk_tokens_from_nchw(const void* y, bk_dtype dt, int64_t B, int64_t C, int64_t H, int64_t W,
                              void* out, void* stream) {
    const char* fn = "bk_tokens_from_nchw";
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    if (H < 0 || W < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (H > ((int64_t)1 << 20) || W > ((int64_t)1 << 20)) return fail(BK_ERR_NOT_SUPPORTED, "%s: dimensions too large", fn);
    if ((st = check_tokens(fn, B, C, H * W)) != BK_OK) return st;
    if (B * C * H * W == 0) return BK_OK;
    if (!y || !out) return fail(BK_ERR_INVALID_VALUE, "%s: NULL pointer", fn);
    hipError_t e = bk::launch_tokens(y, out, B, C, H * W, dt == BK_BF16, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "token transpose launch");
}

bk_status bk_conv_prep(const bk_conv* convs, int64_t n, bk_dtype dt, int64_t B, void* stream) {
    const char* fn = "bk_conv_prep";
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    if (n < 0 || B < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (n == 0) return BK_OK;
    if (!convs) return fail(BK_ERR_INVALID_VALUE, "%s: NULL layer array", fn);
    if (n > 4096) return fail(BK_ERR_NOT_SUPPORTED, "%s: more than 4096 layers", fn);
    std::vector<bk::ConvPrepLayer> L((size_t)n);
    for (int64_t l = 0; l < n; ++l) {
        const bk_conv& c = convs[l];
        char where[64];
        std::snprintf(where, sizeof where, "%s (layer %lld)", fn, (long long)l);
        bk::UnfoldShape sh{};
        if ((st = check_unfold(where, B, c.C, c.H, c.W, c.kh, c.kw, c.stride, c.pad, c.ld, &sh)) != BK_OK) return st;
        if ((st = check_tokens(where, B, c.p, sh.T)) != BK_OK) return st;
        if ((c.x && !c.a) || (c.dy && !c.g))
            return fail(BK_ERR_INVALID_VALUE, "%s: NULL output for a given input", where);
        const bool unf = c.x && B * sh.T * c.ld > 0, tok = c.dy && B * sh.T * c.p > 0;
        L[(size_t)l] = bk::ConvPrepLayer{unf ? c.x : nullptr, tok ? c.dy : nullptr, c.a, c.g, sh, c.p};
    }
    hipError_t e = bk::launch_conv_prep(L.data(), (int)n, B, dt == BK_BF16, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "convolution preparation launch");
}

bk_status bk_embed_ghost_norm(const int64_t* ids, const void* g, bk_dtype dt, int64_t B, int64_t T,
                              int64_t p, int64_t V, float* norm_sq, void* ws, size_t ws_bytes,
                              void* stream) {
    return single_norm("bk_embed_ghost_norm", Path::Embed, embed_layer(ids, g, T, V, p, nullptr), dt,
                       B, norm_sq, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

bk_status bk_clip_factors(const float* norm_sq, int64_t L, int64_t B, bk_clip mode, float R,
                          float gamma, float* C, float* total_sq, void* stream) {
    const char* fn = "bk_clip_factors";
    if (L < 0 || B < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (mode != BK_CLIP_ABADI && mode != BK_CLIP_AUTO)
        return fail(BK_ERR_INVALID_VALUE, "%s: unknown clip mode %d", fn, (int)mode);
    if (mode == BK_CLIP_ABADI && !(R > 0.f))
        return fail(BK_ERR_INVALID_VALUE, "%s: Abadi clipping needs R > 0", fn);
    if (mode == BK_CLIP_AUTO && !(gamma >= 0.f))
        return fail(BK_ERR_INVALID_VALUE, "%s: automatic clipping needs gamma >= 0", fn);
    if (!mul3_ok(L, B, 1)) return fail(BK_ERR_INVALID_VALUE, "%s: L*B overflows", fn);
    if (B > 0 && (!C || (L > 0 && !norm_sq)))
        return fail(BK_ERR_INVALID_VALUE, "%s: NULL pointer", fn);
    hipError_t e = bk::launch_clip(norm_sq, L, B, (int)mode, R, gamma, C, total_sq,
                                   static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "clip launch");
}

bk_status bk_weighted_grad(const void* a, const void* g, const float* C, bk_dtype dt, int64_t B,
                           int64_t T, int64_t d, int64_t p, float* G, void* ws, size_t ws_bytes,
                           void* stream) {
    const bk_layer L = linear_layer(a, g, T, d, p, G);
    return weighted_grads("bk_weighted_grad", &L, 1, C, dt, B, ws, ws_bytes,
                          static_cast<hipStream_t>(stream));
}

bk_status bk_embed_weighted_grad(const int64_t* ids, const void* g, const float* C, bk_dtype dt,
                                 int64_t B, int64_t T, int64_t p, int64_t V, float* G, void* ws,
                                 size_t ws_bytes, void* stream) {
    const bk_layer L = embed_layer(ids, g, T, V, p, G);
    return weighted_grads("bk_embed_weighted_grad", &L, 1, C, dt, B, ws, ws_bytes,
                          static_cast<hipStream_t>(stream));
}

bk_status bk_add_noise(float* G, int64_t n, float std, uint64_t seed, uint32_t tensor_id,
                       uint32_t step, void* stream) {
    const char* fn = "bk_add_noise";
    if (n < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative size", fn);
    if (n > 0 && !G) return fail(BK_ERR_INVALID_VALUE, "%s: NULL tensor", fn);
    if (!(std >= 0.f) || std == INFINITY) return fail(BK_ERR_INVALID_VALUE, "%s: std must be finite and >= 0", fn);
    if (n == 0 || std == 0.f) return BK_OK;
    return add_noise_layers(fn, &G, &n, &tensor_id, 1, std, seed, step, static_cast<hipStream_t>(stream));
}

bk_status bk_add_noise_grouped(float* const* G, const int64_t* nel, const uint32_t* tensor_id,
                               int64_t n, float std, uint64_t seed, uint32_t step, void* stream) {
    const char* fn = "bk_add_noise_grouped";
    if (n < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative tensor count", fn);
    if (n > 0 && (!G || !nel || !tensor_id)) return fail(BK_ERR_INVALID_VALUE, "%s: NULL array", fn);
    if (!(std >= 0.f) || std == INFINITY) return fail(BK_ERR_INVALID_VALUE, "%s: std must be finite and >= 0", fn);
    for (int64_t k = 0; k < n; ++k) {
        if (nel[k] < 0) return fail(BK_ERR_INVALID_VALUE, "%s: tensor %lld: negative size", fn, (long long)k);
        if (nel[k] > 0 && !G[k]) return fail(BK_ERR_INVALID_VALUE, "%s: tensor %lld: NULL", fn, (long long)k);
    }
    if (n == 0 || std == 0.f) return BK_OK;
    return add_noise_layers(fn, G, nel, tensor_id, n, std, seed, step, static_cast<hipStream_t>(stream));
}

bk_status bk_philox_raw(uint64_t seed, uint32_t tensor_id, uint32_t step, uint64_t q0, int64_t nq,
                        uint32_t* out, void* stream) {
    const char* fn = "bk_philox_raw";
    if (nq < 0) return fail(BK_ERR_INVALID_VALUE, "%s: negative count", fn);
    if (nq > 0 && !out) return fail(BK_ERR_INVALID_VALUE, "%s: NULL output", fn);
    if (nq > ((int64_t)1 << 40)) return fail(BK_ERR_NOT_SUPPORTED, "%s: count too large", fn);
    hipError_t e = bk::launch_philox_raw(seed, tensor_id, step, q0, nq, out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BK_OK : hip_fail(e, "philox launch");
}

size_t bk_layer_norms_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    if (n < 0 || (n > 0 && !layers) || B < 0 || check_dtype("", dt) != BK_OK) return 0;
    for (int64_t l = 0; l < n; ++l)
        if (check_dims("", B, layers[l].T, layers[l].d, layers[l].p) != BK_OK) return 0;
    return layer_norms_ws(layers, n, dt, B);
}

bk_status bk_layer_norms(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B, float* norm_sq,
                         void* ws, size_t ws_bytes, void* stream) {
    return layer_norms("bk_layer_norms", layers, n, dt, B, norm_sq, ws, ws_bytes,
                       static_cast<hipStream_t>(stream));
}

size_t bk_weighted_grads_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    if (n < 0 || (n > 0 && !layers) || B < 0 || check_dtype("", dt) != BK_OK) return 0;
    for (int64_t l = 0; l < n; ++l)
        if (check_dims("", B, layers[l].T, layers[l].d, layers[l].p) != BK_OK) return 0;
    return weighted_grads_ws(layers, n, dt, B);
}

bk_status bk_weighted_grads(const bk_layer* layers, int64_t n, const float* C, bk_dtype dt,
                            int64_t B, void* ws, size_t ws_bytes, void* stream) {
    return weighted_grads("bk_weighted_grads", layers, n, C, dt, B, ws, ws_bytes,
                          static_cast<hipStream_t>(stream));
}

size_t bk_private_grad_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B) {
    return std::max(bk_layer_norms_workspace_size(layers, n, dt, B),
                    bk_weighted_grads_workspace_size(layers, n, dt, B));
}

bk_status bk_private_grad(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B, bk_clip mode,
                          float R, float gamma, float noise_std, uint64_t seed, uint32_t step,
                          float* norm_sq, float* C, float* total_sq, void* ws, size_t ws_bytes,
                          void* stream) {
    const char* fn = "bk_private_grad";
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!(noise_std >= 0.f) || noise_std == INFINITY)
        return fail(BK_ERR_INVALID_VALUE, "%s: noise_std must be finite and >= 0", fn);
    if (mode != BK_CLIP_ABADI && mode != BK_CLIP_AUTO)
        return fail(BK_ERR_INVALID_VALUE, "%s: unknown clip mode %d", fn, (int)mode);
    if (mode == BK_CLIP_ABADI && !(R > 0.f))
        return fail(BK_ERR_INVALID_VALUE, "%s: Abadi clipping needs R > 0", fn);
    if (mode == BK_CLIP_AUTO && !(gamma >= 0.f))
        return fail(BK_ERR_INVALID_VALUE, "%s: automatic clipping needs gamma >= 0", fn);
    if (n < 0 || (n > 0 && !layers)) return fail(BK_ERR_INVALID_VALUE, "%s: bad layer array", fn);
    bk_status st = check_dtype(fn, dt);
    if (st != BK_OK) return st;
    for (int64_t l = 0; l < n; ++l)
        if ((st = check_layer(fn, layers[l], l, B, true)) != BK_OK) return st;
    if (B > 0 && !C) return fail(BK_ERR_INVALID_VALUE, "%s: NULL clip factor output", fn);
    // tensor ids l and BK_BIAS_TENSOR | l must not collide
    if (n > INT32_MAX) return fail(BK_ERR_NOT_SUPPORTED, "%s: too many layers", fn);
    const size_t need = bk_private_grad_workspace_size(layers, n, dt, B);
    if (ws_bytes < need || (need > 0 && !ws))
        return fail(BK_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);

    if ((st = layer_norms(fn, layers, n, dt, B, norm_sq, ws, ws_bytes, s)) != BK_OK) return st;
    hipError_t e = bk::launch_clip(norm_sq, n, B, (int)mode, R, gamma, C, total_sq, s);
    if (e != hipSuccess) return hip_fail(e, "clip launch");
    if ((st = weighted_grads(fn, layers, n, C, dt, B, ws, ws_bytes, s)) != BK_OK) return st;
    if (noise_std == 0.f) return BK_OK;
    std::vector<float*> G;
    std::vector<int64_t> nel;
    std::vector<uint32_t> tid;
    for (int64_t l = 0; l < n; ++l) {
        const bk_layer& L = layers[l];
        G.push_back(L.G);
        nel.push_back(L.kind == BK_NORM_AFFINE ? L.p : L.d * L.p);
        tid.push_back((uint32_t)l);
        if (L.flags & BK_LAYER_BIAS) {        // bias / beta: its own noise stream
            G.push_back(L.Gb);
            nel.push_back(L.p);
            tid.push_back(BK_BIAS_TENSOR | (uint32_t)l);
        }
    }
    return add_noise_layers(fn, G.data(), nel.data(), tid.data(), (int64_t)G.size(), noise_std, seed, step, s);
}

const char* bk_status_string(bk_status s) {
    switch (s) {
        case BK_OK: return "BK_OK";
        case BK_ERR_INVALID_VALUE: return "BK_ERR_INVALID_VALUE";
        case BK_ERR_NOT_SUPPORTED: return "BK_ERR_NOT_SUPPORTED";
        case BK_ERR_WORKSPACE: return "BK_ERR_WORKSPACE";
        case BK_ERR_LAUNCH: return "BK_ERR_LAUNCH";
        default: return "BK_ERR_UNKNOWN";
    }
}

const char* bk_last_error(void) { return g_err.c_str(); }

const char* bk_version(void) { return "bk 0.1 (gfx950)"; }

}  // extern "C"
