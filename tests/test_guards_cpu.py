"""The parity guards are tight enough to see a plausible mistake at the
full-size shapes (CPU only, oracle on both sides).

A kernel that drops, or counts twice, one token row of one sample changes
that sample's norm by about 1/T and a clipped-gradient block by about
1/sqrt(B T).  These tests take the hardest full-size cases (longest T for
norms, largest B T for the clipped gradients of each guard) and check that
such a mistake moves the oracle's result by more than the guard the GPU
parity tests apply.
"""
import numpy as np

import oracle
import workloads as wl
from tolerances import GRAD_GUARD_EXACT, GRAD_GUARD_ROUNDED, NORM_GUARD, weights_on_accumulators


def _rel(x, ref):
    return float(np.max(np.abs(np.asarray(x) - ref) / np.abs(ref)))


def _frob(x, ref):
    return float(np.linalg.norm(x - ref) / np.linalg.norm(ref))


def _normal(rng, *shape, scale=1.0):
    # bf16-like inputs are not needed: the effect of a lost row is what is measured
    return rng.standard_normal(shape) * scale


def test_dropped_token_breaks_norm_guard():
    """T = 1024 (the long-sequence stack) is where one row matters least."""
    rng = np.random.default_rng(0)
    for T, d, p in ((1024, 768, 768), (1024, 768, 3072), (256, 1280, 1280), (197, 768, 2304), (128, 3072, 768)):
        a, g = _normal(rng, 1, T, d), _normal(rng, 1, T, p, scale=1e-2)
        ref = oracle.linear_norm_sq(a, g)
        for t in (0, T // 2, T - 1):
            a2 = a.copy()
            a2[0, t] = 0.0
            assert _rel(oracle.linear_norm_sq(a2, g), ref) > 3 * NORM_GUARD, (T, d, p, t)
    # the embedding: one token's id replaced by a fresh one
    w = wl.get(5)
    L = w.layers[-1]
    ids = wl.zipf_ids(L.T, L.d, w.zipf_s, 5).reshape(1, L.T)
    g = _normal(rng, 1, L.T, L.p, scale=1e-2)
    ref = oracle.embed_norm_sq(ids, g, L.d)
    ids2 = ids.copy()
    ids2[0, np.argmax(ids[0] == np.bincount(ids[0]).argmax())] = L.d - 1
    assert _rel(oracle.embed_norm_sq(ids2, g, L.d), ref) > 3 * NORM_GUARD


def _block_change(rng, B, T, k=32):
    """Relative Frobenius change of a k x k clipped-gradient block when one
    row of one sample is dropped (a ~ N(0,1), g ~ N(0,1e-4), C ~ automatic-
    clipping-like factors)."""
    a, g = _normal(rng, B, T, k), _normal(rng, B, T, k, scale=1e-2)
    C = 1.0 / (np.sqrt(rng.uniform(0.5, 2.0, B)) + 0.01)
    ref = oracle.weighted_grad(a, g, C)
    worst = np.inf
    for i, t in ((0, 0), (B // 2, T // 2), (B - 1, T - 1)):
        a2 = a.copy()
        a2[i, t] = 0.0
        worst = min(worst, _frob(oracle.weighted_grad(a2, g, C), ref))
    return worst


def test_dropped_row_breaks_exact_gradient_guard():
    """The exact-weight guard is checked on every layer (the power-of-two
    weights run); the largest B T of any full-size layer is the ResNet-18
    stem (16 x 12544 rows)."""
    rng = np.random.default_rng(1)
    worst_bt = max(w.B * L.T for wid in (2, 3, 4, 5, 6, 7, 8) for w in [wl.get(wid)] for L in w.layers)
    assert worst_bt == 16 * 12544
    assert _block_change(rng, 16, 12544) > 3 * GRAD_GUARD_EXACT


def test_dropped_row_breaks_rounded_gradient_guard():
    """Layers whose kernel rounds C_i g to bf16 get the looser guard with the
    real clip factors; on the full-size stacks those are the LoRA factors
    (narrow kernel) at B T = 32 x 128, where one row's share 1/sqrt(B T) is
    far above it."""
    rng = np.random.default_rng(2)
    rounded = [(w.B, L.T) for wid in (2, 3, 4, 5, 7, 8) for w in [wl.get(wid)] for L in w.layers
               if L.kind in ("linear", "conv") and not weights_on_accumulators(L.T, L.d, L.p, w.B)]
    assert rounded, "some full-size layers take the rounded-weight kernels"
    B, T = max(rounded, key=lambda bt: bt[0] * bt[1])
    assert (B, T) == (32, 128)
    assert _block_change(rng, B, T) > 1.5 * GRAD_GUARD_ROUNDED
