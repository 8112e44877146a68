"""CPU oracle of the Book-Keeping (BK) clipping path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It shares no code with the HIP library: it is a plain,
slow, float64 restatement of what the paper defines, written so it can be
checked against the paper by eye.

Reference: Bu, Wang, Zha, Karypis, "Differentially Private Optimization on
Large Model at Small Cost" (ICML 2023, arXiv 2210.00038).

What is computed, and where the paper defines it
------------------------------------------------
* use_ghost             -- Section 3.2 (layerwise decision / mixed ghost norm):
                           ghost norm iff 2 T^2 < p d, instantiate otherwise.
* use_ghost_time        -- the same decision by time instead of space (Table
                           "block complexity", time row: 2BT^2(p+d) for the
                           ghost norm, 2BTpd for instantiation): ghost norm
                           iff T (p + d) < p d.  An option beside the paper's
                           rule; both give the same norms.
* linear_norm_sq        -- per-sample squared gradient norm ||a_i^T g_i||_F^2,
                           the left-hand side of eq. (ghost norm) in Section 2.1
                           and the per-sample gradient of App. B.4.1.  This is
                           the definition, used for ghost and instantiated
                           layers alike (both compute the same number).
* linear_norm_sq_gram   -- the right-hand side of eq. (ghost norm): the inner
                           product of the two T x T Gram matrices (App. B.4).
* embed_norm_sq         -- the same definition for an embedding layer, whose
                           input is the one-hot encoding of the token ids.
* aggregate             -- Algorithm 1, aggregation across layers.
* clip_factors          -- eq. (DP optimizers): Abadi min(R/||g||, 1) and
                           automatic clipping 1/(||g|| + gamma).
* weighted_grad         -- Algorithm 1, sum of clipped gradients
                           a^T diag(C) dL/ds (App. B.3 with the clip weights).
* embed_weighted_grad   -- the same for an embedding layer.
* per_sample_grads      -- the instantiated per-sample gradients a_i^T g_i
                           (App. B.4.1), kept by BK-MixOpt on the layers that
                           instantiate (Section 3.2; Algorithm "BKAL-mixed").
* weighted_sum          -- sum_i C_i (a_i^T g_i) from stored per-sample
                           gradients (App. B.5), BK-MixOpt's clipped gradient
                           on those layers.
* unfold / tokens_from_nchw -- a 2-D convolution as a generalized linear layer
                           (App. B: d = input channels x kernel size, p =
                           output channels, T = output height x width): the
                           activation a_i is the unfolded input, and the
                           output gradient is taken token-major [T, p].
* lora_submodules / adapter_submodules -- App. E.2: a LoRA module
                           x(W + LR) and an adapter tau(xD)U + x each split
                           into two generalized linear sub-modules (d -> r and
                           r -> p), whose (activation, output gradient) pairs
                           enter the path like any other layer.  The frozen W
                           and the residual x carry no trainable weight.
* bias_sums / bias_norm_sq -- the bias b of a layer s = a W + b (the forward and
                           back-propagation figure of Section 2): its per-sample
                           gradient is sum_t dL_i/ds_t, instantiated (Section 5
                           notes that book-keeping covers the weights only).
* norm_affine_sums / norm_affine_norm_sq -- the elementwise affine parameters
                           of LayerNorm / GroupNorm / InstanceNorm (y = gamma *
                           xhat + beta; per-sample instantiation in the codebase
                           notes of the appendix): dL_i/dgamma = sum_t g_t * xhat_t,
                           dL_i/dbeta = sum_t g_t, over the tokens (or spatial
                           positions) t.
* logical_batch          -- gradient accumulation (footnote on physical and
                           logical batch sizes in Section 3; appendix codebase
                           notes): clip per physical batch, sum the clipped
                           gradients over the physical batches, add the noise
                           once per logical batch.
* philox4x32_10 / noise -- Algorithm 1, Gaussian noise sigma R N(0, I).  The
                           paper does not fix a generator; the reading used
                           here is Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
                           "Parallel random numbers: as easy as 1, 2, 3",
                           SC'11) with the Box-Muller transform (Box & Muller,
                           1958); layout in ``noise``.

Readings where the paper is silent or inconsistent
--------------------------------------------------
* Gram orientation: the T x T Grams a_i a_i^T and g_i g_i^T of eq. (ghost norm)
  (the appendix algorithms print d x d / p x p products, which do not match).
* Ties 2 T^2 == p d instantiate (Section 3.2 wording).
* Abadi clipping at ||g|| = 0 gives C = 1; automatic clipping with gamma = 0
  at ||g|| = 0 gives C = 0 (that sample's gradient is zero).
* Losses are summed (L = sum_i L_i), so the clipped gradient is a sum, not a
  mean, over the batch.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "use_ghost", "use_ghost_time", "linear_norm_sq", "linear_norm_sq_gram", "linear_norm_sq_bruteforce",
    "embed_norm_sq", "embed_norm_sq_pairs", "aggregate", "clip_factors", "weighted_grad",
    "embed_weighted_grad", "philox4x32_10", "philox_words", "uniforms_from_words",
    "box_muller", "noise", "noise_at", "add_noise", "PHILOX_M0", "PHILOX_M1", "PHILOX_W0", "PHILOX_W1",
    "bk_layer_norm", "bk_stack", "per_sample_grads", "weighted_sum", "conv_out_size", "unfold",
    "tokens_from_nchw", "lora_submodules", "adapter_submodules", "bias_sums", "bias_norm_sq",
    "norm_affine_sums", "norm_affine_norm_sq", "logical_batch", "BIAS_TENSOR",
]

F64 = np.float64


def _f64(x) -> np.ndarray:
    """Exact upcast of float32 / bfloat16 (torch) or numpy input to float64."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=F64)


def _ids(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.int64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.int64)


# --------------------------------------------------------------------------
# Section 3.2: which way to compute a layer's per-sample norms
# --------------------------------------------------------------------------
def use_ghost(T: int, d: int, p: int) -> bool:
    """Ghost norm iff 2 T^2 < p d (space of the two Grams vs one per-sample
    gradient, Table "block complexity"); ties instantiate."""
    return 2 * int(T) * int(T) < int(p) * int(d)


def use_ghost_time(T: int, d: int, p: int) -> bool:
    """Ghost norm iff T (p + d) < p d: the time of forming the two T x T Grams,
    2 B T^2 (p + d), against that of instantiating every per-sample gradient,
    2 B T p d (Table "block complexity", time row); ties instantiate."""
    return int(T) * (int(p) + int(d)) < int(p) * int(d)


# --------------------------------------------------------------------------
# Per-sample squared gradient norms of a linear layer s = a W, W in R^{d x p}
# --------------------------------------------------------------------------
def linear_norm_sq(a, g) -> np.ndarray:
    """||dL_i/dW||_F^2 with dL_i/dW = a_i^T g_i  (a: [B,T,d], g: [B,T,p]) -> [B]."""
    a = _f64(a)
    g = _f64(g)
    B = a.shape[0]
    out = np.zeros(B, dtype=F64)
    for i in range(B):
        grad_i = a[i].T @ g[i]            # d x p per-sample gradient
        out[i] = np.sum(grad_i * grad_i)
    return out


def linear_norm_sq_gram(a, g) -> np.ndarray:
    """vec(g_i g_i^T) . vec(a_i a_i^T), the ghost-norm form of the same number."""
    a = _f64(a)
    g = _f64(g)
    B = a.shape[0]
    out = np.zeros(B, dtype=F64)
    for i in range(B):
        ga = a[i] @ a[i].T                # T x T
        gg = g[i] @ g[i].T                # T x T
        out[i] = np.sum(ga * gg)
    return out


def linear_norm_sq_bruteforce(a, g) -> list:
    """Pure-Python loops over every entry of every per-sample gradient (tiny inputs)."""
    a = _f64(a).tolist()
    g = _f64(g).tolist()
    res = []
    for ai, gi in zip(a, g):
        T, d, p = len(ai), len(ai[0]) if ai else 0, len(gi[0]) if gi else 0
        s = 0.0
        for j in range(d):
            for k in range(p):
                e = 0.0
                for t in range(T):
                    e += ai[t][j] * gi[t][k]
                s += e * e
        res.append(s)
    return res


# --------------------------------------------------------------------------
# Embedding layer: a_i is the one-hot encoding of the ids x_i in R^{T x V}
# --------------------------------------------------------------------------
def embed_norm_sq(ids, g, V: int) -> np.ndarray:
    """||one_hot(x_i)^T g_i||_F^2 = sum_v ||sum_{t: x_it = v} g_it||^2 -> [B]."""
    ids = _ids(ids)
    g = _f64(g)
    B, T, p = g.shape
    out = np.zeros(B, dtype=F64)
    for i in range(B):
        rows = np.zeros((V, p), dtype=F64)      # dL_i/dW of the embedding table
        np.add.at(rows, ids[i], g[i])
        out[i] = np.sum(rows * rows)
    return out


def embed_norm_sq_pairs(ids, g) -> np.ndarray:
    """Same number as a double sum over token pairs with equal ids."""
    ids = _ids(ids)
    g = _f64(g)
    B, T, p = g.shape
    out = np.zeros(B, dtype=F64)
    for i in range(B):
        same = (ids[i][:, None] == ids[i][None, :]).astype(F64)   # a_i a_i^T
        out[i] = np.sum(same * (g[i] @ g[i].T))
    return out


# --------------------------------------------------------------------------
# Algorithm 1: aggregate over layers, clip factors, clipped gradient
# --------------------------------------------------------------------------
def aggregate(norms_sq) -> np.ndarray:
    """||dL_i/dW||_F^2 = sum_l ||dL_i/dW_(l)||_F^2 ; norms_sq: [L, B] -> [B]."""
    n = _f64(norms_sq)
    tot = np.zeros(n.shape[1], dtype=F64)
    for l in range(n.shape[0]):
        tot = tot + n[l]
    return tot


def clip_factors(total_sq, mode: str, R: float = 1.0, gamma: float = 0.01) -> np.ndarray:
    """C_i from the total squared norm: 'abadi' -> min(R/||g_i||, 1),
    'auto' -> 1 / (||g_i|| + gamma)."""
    nrm = np.sqrt(_f64(total_sq))
    C = np.empty_like(nrm)
    for i, v in enumerate(nrm):
        if mode == "abadi":
            if R <= 0:
                raise ValueError("Abadi clipping needs R > 0")
            C[i] = 1.0 if v <= R else R / v
        elif mode == "auto":
            den = v + gamma
            C[i] = 0.0 if den == 0.0 else 1.0 / den
        else:
            raise ValueError(mode)
    return C


def weighted_grad(a, g, C) -> np.ndarray:
    """G = a^T diag(C) g = sum_i C_i a_i^T g_i  -> [d, p]."""
    a = _f64(a)
    g = _f64(g)
    C = _f64(C)
    B, T, d = a.shape
    p = g.shape[2]
    c_row = np.repeat(C, T)                          # weight of every token row
    return a.reshape(B * T, d).T @ (c_row[:, None] * g.reshape(B * T, p))


def per_sample_grads(a, g) -> np.ndarray:
    """dL_i/dW = a_i^T g_i for every sample  (a: [B,T,d], g: [B,T,p]) -> [B, d, p]."""
    a = _f64(a)
    g = _f64(g)
    B, T, d = a.shape
    p = g.shape[2]
    P = np.zeros((B, d, p), dtype=F64)
    for i in range(B):
        P[i] = a[i].T @ g[i]
    return P


def weighted_sum(P, C) -> np.ndarray:
    """sum_i C_i P_i over stored per-sample gradients P [B, d, p] -> [d, p]."""
    P = _f64(P)
    C = _f64(C)
    G = np.zeros(P.shape[1:], dtype=F64)
    for i in range(P.shape[0]):
        G += C[i] * P[i]
    return G


def conv_out_size(n: int, k: int, stride: int, pad: int) -> int:
    return (n + 2 * pad - k) // stride + 1


def unfold(x, kh: int, kw: int, stride: int = 1, pad: int = 0, ld: int = 0) -> np.ndarray:
    """x [B, C, H, W] -> a [B, T, ld] with T = Ho Wo, token t = (oh, ow) row-major, and
    column (c, i, j) -> c kh kw + i kw + j holding x[c, oh stride + i - pad, ow stride + j - pad]
    (0 outside the image); columns d = C kh kw .. ld-1 are zero (ld = 0: ld = d).
    With W [p, C, kh, kw] reshaped to [p, d] the convolution output is s = a W^T."""
    x = _f64(x)
    B, Cc, H, Wd = x.shape
    Ho, Wo = conv_out_size(H, kh, stride, pad), conv_out_size(Wd, kw, stride, pad)
    d = Cc * kh * kw
    ld = ld or d
    a = np.zeros((B, Ho * Wo, ld), dtype=F64)
    for oh in range(Ho):
        for ow in range(Wo):
            t = oh * Wo + ow
            for c in range(Cc):
                for i in range(kh):
                    for j in range(kw):
                        h, w = oh * stride + i - pad, ow * stride + j - pad
                        if 0 <= h < H and 0 <= w < Wd:
                            a[:, t, c * kh * kw + i * kw + j] = x[:, c, h, w]
    return a


def tokens_from_nchw(y) -> np.ndarray:
    """[B, C, H, W] -> [B, H W, C] (the output gradient of a convolution, token-major)."""
    y = _f64(y)
    B, Cc, H, Wd = y.shape
    return y.reshape(B, Cc, H * Wd).transpose(0, 2, 1).copy()


def lora_submodules(x, Lw, Rw, dv):
    """LoRA (App. E.2): v = x(W + L R) with W frozen.  Sub-module 1 is
    x -> u = x L (activation x [B,T,d], output gradient dL/du = dv R^T
    [B,T,r]); sub-module 2 is u -> u R (activation u = x L [B,T,r], output
    gradient dv [B,T,p]).  Returns [(a_1, g_1), (a_2, g_2)] in float64."""
    x, Lw, Rw, dv = _f64(x), _f64(Lw), _f64(Rw), _f64(dv)
    u = x @ Lw
    du = dv @ Rw.T
    return [(x, du), (u, dv)]


def adapter_submodules(x, D, U, dv, act: str = "relu"):
    """Adapter (App. E.2): A(x) = tau(x D) U + x.  Sub-module 1 is
    x -> u = x D (activation x [B,T,p], output gradient
    dL/du = (dv U^T) * tau'(u) [B,T,r]); sub-module 2 is tau(u) -> tau(u) U
    (activation tau(u) [B,T,r], output gradient dv [B,T,p]).  The residual
    x carries no weight.  tau = ReLU (tau'(0) taken as 0) or tanh."""
    x, D, U, dv = _f64(x), _f64(D), _f64(U), _f64(dv)
    u = x @ D
    if act == "relu":
        h, dh = np.maximum(u, 0.0), (u > 0).astype(F64)
    elif act == "tanh":
        h = np.tanh(u)
        dh = 1.0 - h * h
    else:
        raise ValueError(act)
    du = (dv @ U.T) * dh
    return [(x, du), (h, dv)]


def bias_sums(g) -> np.ndarray:
    """Per-sample gradient of a bias: s_i = sum_t g_it  ([B,T,p] -> [B,p])."""
    return _f64(g).sum(axis=1)


def bias_norm_sq(g) -> np.ndarray:
    """||s_i||^2 of the per-sample bias gradient -> [B]."""
    s = bias_sums(g)
    return np.einsum("bp,bp->b", s, s)


def norm_affine_sums(xhat, g):
    """Per-sample gradients of y = gamma * xhat + beta over tokens t:
    u_i = sum_t g_it * xhat_it (gamma) and s_i = sum_t g_it (beta), both [B,p]."""
    xhat, g = _f64(xhat), _f64(g)
    return (g * xhat).sum(axis=1), g.sum(axis=1)


def norm_affine_norm_sq(xhat, g, beta: bool = True) -> np.ndarray:
    """||u_i||^2 (+ ||s_i||^2 with a beta) -> [B]."""
    u, s = norm_affine_sums(xhat, g)
    n = np.einsum("bp,bp->b", u, u)
    return n + np.einsum("bp,bp->b", s, s) if beta else n


def embed_weighted_grad(ids, g, C, V: int) -> np.ndarray:
    """G[v, :] = sum_i C_i sum_{t: x_it = v} g_it  -> [V, p] (every row present)."""
    ids = _ids(ids)
    g = _f64(g)
    C = _f64(C)
    B, T, p = g.shape
    G = np.zeros((V, p), dtype=F64)
    np.add.at(G, ids.reshape(-1), np.repeat(C, T)[:, None] * g.reshape(B * T, p))
    return G


# --------------------------------------------------------------------------
# Gaussian noise: Philox4x32-10 + Box-Muller
# --------------------------------------------------------------------------
# Round multipliers and key increments of Philox4x32 (Salmon et al., SC'11).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter, key):
    """Philox4x32 with 10 rounds on arrays of counters.

    counter: (c0, c1, c2, c3), key: (k0, k1); each entry a scalar or an array
    of uint32 values.  A round multiplies c0 and c2 by the two multipliers,
    keeps both 32-bit halves of each product, and mixes:
        (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0));
    the key is advanced by the two Weyl constants between rounds.
    Returns four uint32 arrays."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & _MASK32 for c in counter)
    k0 = np.asarray(key[0], dtype=np.uint64) & _MASK32
    k1 = np.asarray(key[1], dtype=np.uint64) & _MASK32
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK32
            k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK32
        p0 = m0 * c0                              # < 2^64, exact in uint64
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return tuple(x.astype(np.uint32) for x in (c0, c1, c2, c3))


def philox_words(seed: int, tensor_id: int, step: int, q0: int, nq: int) -> np.ndarray:
    """Raw words of counter blocks q0 .. q0+nq-1 -> uint32 [nq, 4].

    Counter block q of tensor `tensor_id` at step `step` is
    (q mod 2^32, q div 2^32, tensor_id, step) under key (seed mod 2^32, seed div 2^32)."""
    q = np.arange(q0, q0 + nq, dtype=np.uint64)
    key = (np.uint64(seed & 0xFFFFFFFF), np.uint64((seed >> 32) & 0xFFFFFFFF))
    w = philox4x32_10((q & _MASK32, q >> np.uint64(32),
                       np.full_like(q, tensor_id & 0xFFFFFFFF), np.full_like(q, step & 0xFFFFFFFF)), key)
    return np.stack(w, axis=1)


def uniforms_from_words(x) -> np.ndarray:
    """u = (2 * (x >> 9) + 1) / 2^24: odd multiples of 2^-24, strictly inside (0, 1)."""
    x = np.asarray(x, dtype=np.uint64)
    return ((x >> np.uint64(9)).astype(F64) * 2.0 + 1.0) / float(1 << 24)


def box_muller(u_r, u_theta):
    """(r cos 2 pi u_theta, r sin 2 pi u_theta) with r = sqrt(-2 ln u_r)."""
    r = np.sqrt(-2.0 * np.log(u_r))
    th = 2.0 * np.pi * u_theta
    return r * np.cos(th), r * np.sin(th)


def noise(n: int, seed: int, tensor_id: int, step: int) -> np.ndarray:
    """n standard normal draws for elements 0..n-1 of one tensor (float64).

    Element e uses word e mod 4 of counter block q = e div 4; words (0, 1) give
    elements 4q and 4q+1 via Box-Muller (word 0 -> radius, word 1 -> angle),
    words (2, 3) give elements 4q+2 and 4q+3 the same way."""
    nq = (n + 3) // 4
    w = philox_words(seed, tensor_id, step, 0, nq)
    u = uniforms_from_words(w)
    z = np.empty((nq, 4), dtype=F64)
    z[:, 0], z[:, 1] = box_muller(u[:, 0], u[:, 1])
    z[:, 2], z[:, 3] = box_muller(u[:, 2], u[:, 3])
    return z.reshape(-1)[:n]


def noise_at(elements, seed: int, tensor_id: int, step: int) -> np.ndarray:
    """The draws of ``noise`` for the given element indices only (same layout:
    element e uses counter block e div 4, word pair (0, 1) or (2, 3))."""
    e = np.asarray(elements, dtype=np.uint64).ravel()
    q = e >> np.uint64(2)
    key = (np.uint64(seed & 0xFFFFFFFF), np.uint64((seed >> 32) & 0xFFFFFFFF))
    w = philox4x32_10((q & _MASK32, q >> np.uint64(32), np.full_like(q, tensor_id & 0xFFFFFFFF),
                       np.full_like(q, step & 0xFFFFFFFF)), key)
    u = [uniforms_from_words(x) for x in w]
    z01 = box_muller(u[0], u[1])
    z23 = box_muller(u[2], u[3])
    j = (e & np.uint64(3)).astype(np.int64)
    out = np.where(j == 0, z01[0], np.where(j == 1, z01[1], np.where(j == 2, z23[0], z23[1])))
    return out.reshape(np.shape(elements))


def add_noise(G, std: float, seed: int, tensor_id: int, step: int) -> np.ndarray:
    """G_hat = G + std * N(0, I), std = sigma * R (Algorithm 1, noise step)."""
    G = _f64(G)
    return G + std * noise(G.size, seed, tensor_id, step).reshape(G.shape)


# --------------------------------------------------------------------------
# Whole path (Algorithm 1 from "norms" to "noise", BK-MixGhostClip choice of
# norm per layer from Algorithm "BKAL-mixed")
# --------------------------------------------------------------------------
BIAS_TENSOR = 1 << 31      # noise stream of a bias / beta: tensor id BIAS_TENSOR | layer


def bk_layer_norm(layer_kind: str, x, g, V: int = 0, bias: bool = False) -> np.ndarray:
    """Per-sample squared gradient norm of one layer: the weights (by their
    definition, ghost and instantiated alike), plus its bias when it has one;
    for a "norm" layer (affine of a normalization) gamma, plus beta with bias."""
    if layer_kind == "embed":
        return embed_norm_sq(x, g, V)
    if layer_kind == "norm":
        return norm_affine_norm_sq(x, g, bias)
    n = linear_norm_sq(x, g)
    return n + bias_norm_sq(g) if bias else n


def bk_stack(layers, inputs, mode: str, R: float, gamma: float, std: float, seed: int,
             step: int = 0, with_noise: bool = True, mixopt: bool = False, rule=None):
    """layers: objects with .kind, .T, .d, .p; inputs: list of (a or ids, g).

    Returns dict with per-layer norms [L, B], totals [B], C [B], the clipped
    gradients G_l (before noise) and, if with_noise, G_hat_l with tensor_id = l.
    mixopt: BK-MixOpt -- a linear layer that instantiates (2 T^2 >= p d) keeps
    its per-sample gradients and forms G_l as their weighted sum (App. B.5);
    every other layer takes the book-keeping GEMM a^T diag(C) g.
    rule: the layerwise decision (default use_ghost; use_ghost_time for the
    decision by time).  It changes which way a layer is computed, and the
    "paths" entry, not the values.
    A layer with a true .bias attribute also has a bias (a "norm" layer: a
    beta); its clipped gradient sum_i C_i s_i is returned in Gb[l] (None
    otherwise) and noised with tensor id BIAS_TENSOR | l.  A "norm" layer's
    G_l is its gamma gradient sum_i C_i u_i."""
    rule = use_ghost if rule is None else rule
    bias = [bool(getattr(L, "bias", False)) for L in layers]
    norms = np.stack([bk_layer_norm(L.kind, x, g, L.d, b) for L, (x, g), b in zip(layers, inputs, bias)])
    total = aggregate(norms)
    C = clip_factors(total, mode, R, gamma)
    G, Ghat, Gb, Gbhat = [], [], [], []
    for l, (L, (x, g)) in enumerate(zip(layers, inputs)):
        if L.kind == "embed":
            Gl = embed_weighted_grad(x, g, C, L.d)
        elif L.kind == "norm":
            Gl = weighted_sum(norm_affine_sums(x, g)[0], C)
        elif mixopt and not rule(L.T, L.d, L.p):
            Gl = weighted_sum(per_sample_grads(x, g), C)
        else:
            Gl = weighted_grad(x, g, C)
        G.append(Gl)
        Gbl = weighted_sum(bias_sums(g), C) if bias[l] else None
        Gb.append(Gbl)
        if with_noise:
            Ghat.append(add_noise(Gl, std, seed, l, step))
            Gbhat.append(add_noise(Gbl, std, seed, BIAS_TENSOR | l, step) if bias[l] else None)
    return {"norms": norms, "total": total, "C": C, "G": G, "Ghat": Ghat, "Gb": Gb, "Gbhat": Gbhat,
            "paths": [("embed" if L.kind == "embed" else "norm" if L.kind == "norm" else
                       ("ghost" if rule(L.T, L.d, L.p) else "inst")) for L in layers]}


def logical_batch(layers, batches, mode: str, R: float, gamma: float, std: float, seed: int,
                  step: int = 0):
    """Gradient accumulation: `batches` is a list of physical batches (each a
    list of per-layer inputs as for bk_stack).  Each physical batch is clipped
    on its own (its samples' norms and factors); the clipped gradients add up
    over the physical batches; the noise is drawn once, for the logical batch.
    Returns dict with per-batch C, the summed G / Gb and the noised Ghat / Gbhat."""
    G = Gb = None
    Cs = []
    for inputs in batches:
        r = bk_stack(layers, inputs, mode, R, gamma, 0.0, seed, step, with_noise=False)
        Cs.append(r["C"])
        if G is None:
            G, Gb = r["G"], r["Gb"]
        else:
            G = [x + y for x, y in zip(G, r["G"])]
            Gb = [None if x is None else x + y for x, y in zip(Gb, r["Gb"])]
    Ghat = [add_noise(Gl, std, seed, l, step) for l, Gl in enumerate(G)]
    Gbhat = [None if x is None else add_noise(x, std, seed, BIAS_TENSOR | l, step) for l, x in enumerate(Gb)]
    return {"C": Cs, "G": G, "Gb": Gb, "Ghat": Ghat, "Gbhat": Gbhat}
