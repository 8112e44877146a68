/*
 * bk.h -- C ABI of the Book-Keeping (BK) differentially private gradient path
 * for AMD Instinct MI355X (gfx950).
 *
 * Method: Bu, Wang, Zha, Karypis, "Differentially Private Optimization on
 * Large Model at Small Cost" (ICML 2023, arXiv 2210.00038).  Starting from the
 * activations a and output gradients dL/ds that one back-propagation keeps
 * ("book-keeping", Section 2.1), the library computes, for every generalized
 * linear layer s = a W with W in R^{d x p} (App. B, eq. "linear layer mat
 * multi"):
 *
 *   1. per-sample squared gradient norms ||a_i^T g_i||_F^2, by the ghost-norm
 *      trick (eq. "ghost norm", App. B.4) or by instantiating the per-sample
 *      gradient (App. B.4.1), whichever the layerwise rule of Section 3.2
 *      picks;
 *   2. their sum over layers and the per-sample clip factors C_i
 *      (Algorithm 1, aggregation and clipping; clip functions of eq. "DP
 *      optimizers");
 *   3. the sum of clipped gradients G = a^T diag(C) dL/ds (Algorithm 1, sum of
 *      clipped gradients; App. B.3);
 *   4. G_hat = G + sigma R N(0, I) (Algorithm 1, noise step).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library never
 *    allocates, frees or keeps them.  Workspaces are caller-provided device
 *    buffers of at least the size the matching *_workspace_size call returns
 *    (a NULL workspace is accepted when that size is 0).
 *  - Layout: row-major, contiguous.  a is [B, T, d], g = dL/ds is [B, T, p]
 *    (sample-major, then token, then feature), both of the dtype `dt`; token
 *    ids are int64 [B, T].  Outputs are float32 and are OVERWRITTEN.  Outputs
 *    must not alias inputs.
 *  - Sums over the batch, not means: the loss is L = sum_i L_i (Section 2.1).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every call is
 *    asynchronous and ordered on that stream; buffers must stay alive until
 *    the stream has finished the work.
 *  - Errors: every call returns a bk_status.  Argument checks (NULL pointers,
 *    sizes >= 0, products overflowing int64, dtype, workspace size) run on the
 *    host before any HIP call, so a rejected call does no work at all.  A
 *    failed kernel launch returns BK_ERR_LAUNCH.  bk_last_error() gives a
 *    human-readable detail of the calling thread's last failure.  Device
 *    faults surface at the caller's next synchronisation, as for any kernel.
 *  - Empty inputs (B == 0 or T == 0) are valid: norms are 0, C is not touched
 *    beyond its B entries, G is all zeros (plus noise where noise is asked for).
 *  - Results are deterministic: the same inputs on the same device give the
 *    same bits (no floating-point atomics).
 *  - Thread safety: every call is re-entrant; calls that share a workspace
 *    must be ordered on one stream.
 */
#ifndef BK_H
#define BK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BK_OK = 0,
    BK_ERR_INVALID_VALUE = 1,   /* bad pointer, size, enum or scalar */
    BK_ERR_NOT_SUPPORTED = 2,   /* valid request beyond what this build handles */
    BK_ERR_WORKSPACE = 3,       /* workspace smaller than *_workspace_size */
    BK_ERR_LAUNCH = 4           /* a HIP call failed; see bk_last_error() */
} bk_status;

typedef enum { BK_F32 = 0, BK_BF16 = 1 } bk_dtype;

/* Clip functions of eq. "DP optimizers":
 *   BK_CLIP_ABADI: C_i = min(R / ||g_i||, 1)       (C_i = 1 when ||g_i|| = 0)
 *   BK_CLIP_AUTO : C_i = 1 / (||g_i|| + gamma)     (automatic clipping; gamma = 0
 *                  is pure normalisation, and C_i = 0 when ||g_i|| = 0 there) */
typedef enum { BK_CLIP_ABADI = 0, BK_CLIP_AUTO = 1 } bk_clip;

/* BK_NORM_AFFINE: the elementwise affine y = gamma * xhat + beta of a
 * LayerNorm / GroupNorm / InstanceNorm over p features (channels), whose
 * per-sample gradients are instantiated (the appendix notes on the supported
 * layers): dL_i/dgamma = sum_t g_it * xhat_it, dL_i/dbeta = sum_t g_it, t over
 * tokens or spatial positions. */
typedef enum { BK_LINEAR = 0, BK_EMBEDDING = 1, BK_NORM_AFFINE = 2 } bk_layer_kind;

/* Layer flags (bk_layer.flags).
 *   BK_LAYER_MIXOPT: BK-MixOpt (Section 3.2; the MixOpt branch of Algorithm
 *   "BKAL-mixed").  A linear layer that instantiates its per-sample gradients
 *   for the norm (bk_use_ghost == 0) keeps them in P, and its clipped gradient
 *   is their weighted sum sum_i C_i P_i (App. B.5) instead of the GEMM
 *   a^T diag(C) g.  Ghost-norm, embedding and affine layers ignore the flag.
 *   BK_LAYER_BIAS: a linear layer s = a W + b with a bias (Section 5: book-
 *   keeping covers the weights; the bias gradient sum_t g_it is instantiated
 *   per sample), or the beta of a BK_NORM_AFFINE layer.  Its squared norm
 *   adds to the layer's per-sample norm; bk_layer_norms keeps the per-sample
 *   sums in Pb [B, p] and bk_weighted_grads writes sum_i C_i Pb_i to Gb [p].
 *   Embedding layers take no bias.
 *   BK_LAYER_ACCUMULATE: gradient accumulation over physical batches (the
 *   paper's logical vs physical batch size): bk_weighted_grads adds this
 *   step's clipped gradients to G (and Gb) instead of overwriting them, each
 *   element in one fixed-order addition.  Each physical batch is clipped on
 *   its own; the caller draws the noise once per logical batch (noise_std 0
 *   in bk_private_grad on all but the last physical batch).
 *   BK_LAYER_TIME_RULE: a linear layer takes the ghost norm or instantiation
 *   by bk_use_ghost_time (the time of the two ways) instead of the paper's
 *   bk_use_ghost (their space).  The norms are the same up to rounding; a
 *   BK_LAYER_MIXOPT layer keeps P exactly when this rule instantiates.  Other
 *   kinds ignore the flag. */
enum { BK_LAYER_MIXOPT = 1, BK_LAYER_BIAS = 2, BK_LAYER_ACCUMULATE = 4, BK_LAYER_TIME_RULE = 8 };

/* One layer of a stack (used by the grouped calls).
 *   kind == BK_LINEAR     : x = a [B, T, d] of dtype dt, g [B, T, p], G [d, p]
 *   kind == BK_EMBEDDING  : x = token ids int64 [B, T] (values in [0, d)),
 *                           d = vocabulary size V, g [B, T, p], G [V, p]
 *   kind == BK_NORM_AFFINE: x = xhat [B, T, p] (the normalized input, dtype
 *                           dt), d = p, g [B, T, p], G [p] (gamma gradient),
 *                           P [B, p] float32 (per-sample gamma gradients,
 *                           written by bk_layer_norms, read by
 *                           bk_weighted_grads; required)
 * G may be NULL in calls that only compute norms.  For a linear layer P
 * (device, float32 [B, d, p]) is used only by a BK_LAYER_MIXOPT layer that
 * instantiates: bk_layer_norms writes the per-sample gradients there and
 * bk_weighted_grads of the same step reads them; otherwise it may be NULL.
 * Gb [p] and Pb [B, p] (float32) are used only with BK_LAYER_BIAS.  All of
 * P, Pb, G, Gb are caller-owned device buffers, 4-byte aligned. */
typedef struct bk_layer {
    int32_t kind;
    int32_t flags;           /* BK_LAYER_* bits */
    int64_t T, d, p;
    const void* x;
    const void* g;
    float* G;
    float* P;
    float* Gb;
    float* Pb;
} bk_layer;

/* Noise stream of the bias (or beta) gradient of layer l: tensor id
 * BK_BIAS_TENSOR | l. */
#define BK_BIAS_TENSOR 0x80000000u

/* Operation ids for bk_workspace_size. */
typedef enum {
    BK_OP_GHOST_NORM = 0,
    BK_OP_INST_NORM = 1,
    BK_OP_EMBED_GHOST_NORM = 2,
    BK_OP_WEIGHTED_GRAD = 3,
    BK_OP_EMBED_WEIGHTED_GRAD = 4
} bk_op;

/* ---------------------------------------------------------------------------
 * Layerwise decision, Section 3.2 (mixed ghost norm): the ghost norm is used on
 * a layer iff 2 T^2 < p d (the space of the two T x T Grams against that of one
 * per-sample gradient, Table "block complexity"); otherwise the per-sample
 * gradient is instantiated.  Ties instantiate.  Pure host function: returns 1
 * for ghost, 0 for instantiation, -1 for negative sizes.
 * ------------------------------------------------------------------------- */
int bk_use_ghost(int64_t T, int64_t d, int64_t p);

/* The same decision by time, an option beside the paper's rule (per layer:
 * BK_LAYER_TIME_RULE): Table "block complexity" prices the ghost norm at
 * 2BT^2(p+d) and instantiation at 2BTpd, so the ghost norm is used iff
 * T (p + d) < p d.  Ties instantiate.  A layer this rule sends to the ghost
 * norm is also sent there by bk_use_ghost, not the other way round.  Pure
 * host function: 1 ghost, 0 instantiation, -1 for negative sizes. */
int bk_use_ghost_time(int64_t T, int64_t d, int64_t p);

/* Workspace bytes `op` needs for one layer of these sizes (d = V for the
 * embedding ops).  Returns 0 for an invalid request. */
size_t bk_workspace_size(bk_op op, bk_dtype dt, int64_t B, int64_t T, int64_t d, int64_t p);

/* ---------------------------------------------------------------------------
 * Ghost norm, eq. "ghost norm" (Section 2.1) and App. B.4:
 *   norm_sq[i] = vec(g_i g_i^T) . vec(a_i a_i^T) = ||a_i^T g_i||_F^2
 * from the two T x T Gram matrices of sample i, which are formed tile by tile
 * on chip and never written to memory.
 *   a [B,T,d], g [B,T,p] (dtype dt), norm_sq [B] float32 out.
 * ------------------------------------------------------------------------- */
bk_status bk_ghost_norm(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T,
                        int64_t d, int64_t p, float* norm_sq, void* ws, size_t ws_bytes,
                        void* stream);

/* Per-sample gradient instantiation, App. B.4.1: the d x p gradient a_i^T g_i
 * of every sample, reduced on chip to norm_sq[i] = ||a_i^T g_i||_F^2 (the
 * per-sample gradients themselves are never stored).  Same arguments as
 * bk_ghost_norm. */
bk_status bk_inst_norm(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T,
                       int64_t d, int64_t p, float* norm_sq, void* ws, size_t ws_bytes,
                       void* stream);

/* The same instantiation keeping the per-sample gradients (BK-MixOpt,
 * App. B.4.1): P[i] = a_i^T g_i, P [B, d, p] float32 out (device), and
 * norm_sq[i] = ||P[i]||_F^2.  Other arguments and the workspace as
 * bk_inst_norm (bk_workspace_size(BK_OP_INST_NORM, ...)). */
bk_status bk_per_sample_grads(const void* a, const void* g, bk_dtype dt, int64_t B, int64_t T,
                              int64_t d, int64_t p, float* norm_sq, float* P, void* ws,
                              size_t ws_bytes, void* stream);

/* Weighted sum of stored per-sample gradients (App. B.5), BK-MixOpt's
 * clipped gradient on an instantiated layer:
 *   G[e] = sum_i C[i] P[i n + e]   for e in [0, n), i ascending, float32
 * (one fused multiply-add per sample).  P [B, n], C [B], G [n] float32
 * (device); B = 0 writes zeros.  Needs no workspace. */
bk_status bk_weighted_sum(const float* P, const float* C, int64_t B, int64_t n, float* G,
                          void* stream);

/* A 2-D convolution as a generalized linear layer (App. B: d = input
 * channels x kernel size, p = output channels, T = output height x width).
 * bk_unfold writes the layer's activation a:
 *   x [B, C, H, W] (dtype dt, NCHW) -> a [B, T, ld], T = Ho Wo,
 *   Ho = (H + 2 pad - kh) / stride + 1, Wo = (W + 2 pad - kw) / stride + 1,
 *   token t = oh Wo + ow, column c kh kw + i kw + j =
 *   x[b, c, oh stride + i - pad, ow stride + j - pad] (0 outside the image),
 *   columns d = C kh kw .. ld-1 zero.  ld >= d; with ld a multiple of 8 the
 *   bf16 rows take the 16-byte kernel paths, and the layer's gradient rows
 *   d .. ld-1 come out zero.  kh, kw, stride >= 1, pad >= 0, Ho, Wo >= 1.
 * bk_tokens_from_nchw writes the layer's output gradient token-major:
 *   y [B, C, H, W] -> out [B, H W, C] (same dtype).
 * Both are copies (bit-exact), device buffers, no workspace. */
bk_status bk_unfold(const void* x, bk_dtype dt, int64_t B, int64_t C, int64_t H, int64_t W,
                    int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t ld, void* a,
                    void* stream);
bk_status bk_tokens_from_nchw(const void* y, bk_dtype dt, int64_t B, int64_t C, int64_t H,
                              int64_t W, void* out, void* stream);

/* One convolution layer of bk_conv_prep (App. B, the convolution as a
 * generalized linear layer with T = Ho Wo, d = C kh kw, p output channels). */
typedef struct bk_conv {
    const void* x;    /* [B, C, H, W] input, or NULL: no unfold for this layer */
    const void* dy;   /* [B, p, Ho, Wo] output gradient dL/ds, or NULL: no transpose */
    void* a;          /* out: [B, Ho Wo, ld] unfolded input (bk_unfold) */
    void* g;          /* out: [B, Ho Wo, p] token-major gradient (bk_tokens_from_nchw) */
    int64_t C, H, W, kh, kw, stride, pad, ld, p;
} bk_conv;

/* Every convolution of a step at once: for each of the n layers, a =
 * bk_unfold(x) and g = bk_tokens_from_nchw(dy) with the shapes above, all of
 * dtype dt and batch B.  The results are those of the single calls (bit-
 * exact copies); the work of all layers shares one launch (a few when more
 * than 24 layers or shapes outside the grouped kernel's limits).  Outputs
 * must not overlap each other or the inputs.  Every layer is checked before
 * any work is queued; n <= 4096, B <= 65535. */
bk_status bk_conv_prep(const bk_conv* convs, int64_t n, bk_dtype dt, int64_t B, void* stream);

/* Ghost norm of an embedding layer (Section 2.1 names the embedding among the
 * generalized linear layers; App. D.1 lists it as ghost-norm only).  Its input
 * a_i is the one-hot encoding of the ids x_i, so a_i a_i^T is the token-id
 * equality matrix and
 *   norm_sq[i] = sum_{t,t'} [x_it == x_it'] <g_it, g_it'>.
 *   ids [B,T] int64, g [B,T,p] (dtype dt), norm_sq [B] out.
 * An id outside [0, V) has an all-zero one-hot row: its token adds nothing
 * (here and in bk_embed_weighted_grad).  For T <= 16384 with p a multiple
 * of 8 and g 16-byte aligned it is computed as a join on the ids,
 * sum_v ||sum_{t : x_it = v} g_it||^2 (each row of g read once); otherwise
 * as the Gram of g masked by id equality. */
bk_status bk_embed_ghost_norm(const int64_t* ids, const void* g, bk_dtype dt, int64_t B,
                              int64_t T, int64_t p, int64_t V, float* norm_sq, void* ws,
                              size_t ws_bytes, void* stream);

/* Algorithm 1, aggregation and clipping:
 *   total_sq[i] = sum_l norm_sq[l*B + i]   (l ascending, float64 accumulation)
 *   C[i]        = clip(sqrt(total_sq[i]))  (bk_clip above)
 *   norm_sq [L,B] float32 in; C [B] out; total_sq [B] out (may be NULL).
 * R > 0 is required for BK_CLIP_ABADI, gamma >= 0 for BK_CLIP_AUTO. */
bk_status bk_clip_factors(const float* norm_sq, int64_t L, int64_t B, bk_clip mode, float R,
                          float gamma, float* C, float* total_sq, void* stream);

/* Algorithm 1, sum of clipped gradients (App. B.3 with the clip weights):
 *   G = a^T diag(C) g = sum_i C_i a_i^T g_i,   G [d,p] float32 out,
 * one GEMM over the flattened B*T rows.  For bf16 layers with 16-byte rows,
 * min(d, p) > 64 or max(d, p) < 128, T >= 64, B <= 4096 and T at most 1/8
 * short of a multiple of 16, the weights multiply the float32 accumulators
 * (every sample starts a GEMM stage of 32 rows, its last stage padded with
 * zero rows); otherwise C_i multiplies the rows of g as they are loaded (for
 * bf16 the product C_i g is rounded to bf16 before the MFMA). */
bk_status bk_weighted_grad(const void* a, const void* g, const float* C, bk_dtype dt,
                           int64_t B, int64_t T, int64_t d, int64_t p, float* G, void* ws,
                           size_t ws_bytes, void* stream);

/* The same for an embedding layer (a = one_hot(ids)):
 *   G[v,:] = sum_i C_i sum_{t : x_it = v} g_it   for every v in [0, V),
 * rows of ids that do not occur are zero; tokens whose id lies outside
 * [0, V) add nothing.  Each row sums its tokens in ascending (i, t) order
 * (deterministic: a stable radix sort of the ids, then fixed-size chunks of
 * the sorted tokens).  G [V,p] float32 out.  B*T <= 2^24 tokens per call
 * (BK_ERR_NOT_SUPPORTED above); the workspace is about 16 B T + B T p / 8
 * bytes (bk_workspace_size). */
bk_status bk_embed_weighted_grad(const int64_t* ids, const void* g, const float* C,
                                 bk_dtype dt, int64_t B, int64_t T, int64_t p, int64_t V,
                                 float* G, void* ws, size_t ws_bytes, void* stream);

/* Algorithm 1, noise step: G[e] += std * z_e for e in [0, n), std = sigma R
 * (App. A.1: the noise magnitude is sigma times the sensitivity R).
 * z_e comes from Philox4x32-10 (Salmon et al., SC'11): counter block
 * q = e / 4 is (q mod 2^32, q div 2^32, tensor_id, step) under the key
 * (seed mod 2^32, seed div 2^32); its words (w0, w1, w2, w3) become uniforms
 * u = (2 (w >> 9) + 1) / 2^24, and Box-Muller maps (u0, u1) to elements 4q,
 * 4q+1 as (r cos 2 pi u1, r sin 2 pi u1), r = sqrt(-2 ln u0), and (u2, u3) to
 * 4q+2, 4q+3 the same way.  std == 0 leaves G bit-identical. */
bk_status bk_add_noise(float* G, int64_t n, float std, uint64_t seed, uint32_t tensor_id,
                       uint32_t step, void* stream);

/* bk_add_noise on n tensors in one launch: tensor k (G[k], nel[k] elements)
 * gets the stream of tensor_id[k]; the values are those of bk_add_noise on
 * each tensor.  G, nel and tensor_id are host arrays of n entries. */
bk_status bk_add_noise_grouped(float* const* G, const int64_t* nel, const uint32_t* tensor_id,
                               int64_t n, float std, uint64_t seed, uint32_t step, void* stream);

/* Raw Philox4x32-10 words of counter blocks q0 .. q0+nq-1 of (seed, tensor_id,
 * step), as used by bk_add_noise: out [nq, 4] uint32 (device). */
bk_status bk_philox_raw(uint64_t seed, uint32_t tensor_id, uint32_t step, uint64_t q0,
                        int64_t nq, uint32_t* out, void* stream);

/* ---------------------------------------------------------------------------
 * Grouped forms: the same computations for n layers in as few launches as
 * possible.  Results are bit-identical to calling the per-layer form on each
 * layer, with one exception: bf16 ghost-norm layers with 128 < T <= 256 (and
 * 16-byte rows) take a whole-sample kernel when the launch gives it at least
 * 512 workgroups (one per layer and sample), and a kernel over pairs of
 * 128-row blocks otherwise; the two agree to fp32 rounding.  Every result is
 * deterministic.  The bk_layer array is read on the host during the call only.
 * ------------------------------------------------------------------------- */

/* Norms of every layer: ghost or instantiated per bk_use_ghost for linear
 * layers (bk_use_ghost_time with BK_LAYER_TIME_RULE), the embedding ghost
 * norm for embedding layers.  norm_sq [n,B] out, row l for layer l. */
size_t bk_layer_norms_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B);
bk_status bk_layer_norms(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B,
                         float* norm_sq, void* ws, size_t ws_bytes, void* stream);

/* Clipped gradients of every layer into layers[l].G (BK_LAYER_MIXOPT
 * instantiated layers: the weighted sum of their P).  The workspace holds
 * float32 partial tiles of K-split GEMM tiles: those of layers with few
 * output tiles, and those of the last, partly filled round of workgroups of
 * a large launch (at most (compute units) x 256 KiB for each).  Its size
 * depends on the compute-unit count of the device current at the query
 * (256 when no device can be asked); query with the launching device
 * current. */
size_t bk_weighted_grads_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt,
                                        int64_t B);
bk_status bk_weighted_grads(const bk_layer* layers, int64_t n, const float* C, bk_dtype dt,
                            int64_t B, void* ws, size_t ws_bytes, void* stream);

/* The whole path of Algorithm 1 from the per-layer norms to the noise, with
 * the layerwise norm choice of Algorithm "BKAL-mixed" (BK-MixGhostClip):
 * bk_layer_norms -> bk_clip_factors -> bk_weighted_grads -> bk_add_noise_grouped
 * on every layers[l].G with tensor_id = l and every bias / beta gradient
 * layers[l].Gb with tensor_id = BK_BIAS_TENSOR | l.  norm_sq [n,B], C [B] out, total_sq [B]
 * out (may be NULL).  noise_std = sigma R; 0 skips the noise. */
size_t bk_private_grad_workspace_size(const bk_layer* layers, int64_t n, bk_dtype dt,
                                      int64_t B);
bk_status bk_private_grad(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B,
                          bk_clip mode, float R, float gamma, float noise_std, uint64_t seed,
                          uint32_t step, float* norm_sq, float* C, float* total_sq, void* ws,
                          size_t ws_bytes, void* stream);

/* Allocation-free form of bk_private_grad, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments and results as
 * bk_private_grad, without the workspace: a device array of
 * BK_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * (from the first call on that GPU until the process ends) stands in for it.
 *  - Returns BK_ERR_NOT_SUPPORTED, doing no work, when
 *    bk_private_grad_workspace_size of the stack exceeds that size (stacks
 *    whose instantiated layers split into many K slices, for instance).
 *  - The stream must belong to the current device (BK_ERR_INVALID_VALUE
 *    otherwise).
 *  - The call allocates and frees nothing and issues no memset.
 *  - Every call on one GPU uses that GPU's one array, which keeps the last
 *    call's contents (each call writes every word it reads first): calls
 *    that overlap on one GPU (other streams, other threads) race, so the
 *    caller must order them, e.g. on one stream. */
#define BK_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
bk_status bk_private_grad_noalloc(const bk_layer* layers, int64_t n, bk_dtype dt, int64_t B,
                                  bk_clip mode, float R, float gamma, float noise_std, uint64_t seed,
                                  uint32_t step, float* norm_sq, float* C, float* total_sq,
                                  void* stream);

/* Diagnostics. */
const char* bk_status_string(bk_status s);
const char* bk_last_error(void);
const char* bk_version(void);

#ifdef __cplusplus
}
#endif
#endif /* BK_H */
