"""Pins of the LoRA / adapter decomposition (App. E.2) of the oracle.

Each module splits into two generalized linear sub-modules; the pins compare
the oracle's per-sample gradient norms and clipped gradients of the
sub-modules (its linear-layer functions on the decomposed activations and
output gradients) with torch autograd on the module itself, sample by
sample, in float64 on the CPU, with the loss of sample i taken as
<A(x_i), dv_i> so that dv is the output gradient."""
import numpy as np
import pytest
import torch

import oracle

B, T, d, r, p = 3, 5, 7, 4, 6


def _per_sample(module_fn, params, x, dv):
    """Per-sample gradients of sum <module(x_i), dv_i> w.r.t. each parameter."""
    out = []
    for i in range(x.shape[0]):
        ps = [q.detach().clone().requires_grad_(True) for q in params]
        v = module_fn(x[i:i + 1], *ps)
        (v * dv[i:i + 1]).sum().backward()
        out.append([q.grad.numpy().copy() for q in ps])
    return out


@pytest.fixture
def gen():
    return torch.Generator().manual_seed(2210)


def test_lora_submodules_match_autograd(gen):
    x = torch.randn(B, T, d, generator=gen, dtype=torch.float64)
    W = torch.randn(d, p, generator=gen, dtype=torch.float64)
    Lw = torch.randn(d, r, generator=gen, dtype=torch.float64)
    Rw = torch.randn(r, p, generator=gen, dtype=torch.float64)
    dv = torch.randn(B, T, p, generator=gen, dtype=torch.float64)
    ref = _per_sample(lambda xi, L_, R_: xi @ W + xi @ L_ @ R_, [Lw, Rw], x, dv)
    (a1, g1), (a2, g2) = oracle.lora_submodules(x, Lw, Rw, dv)
    assert a1.shape == (B, T, d) and g1.shape == (B, T, r) and a2.shape == (B, T, r) and g2.shape == (B, T, p)
    P1, P2 = oracle.per_sample_grads(a1, g1), oracle.per_sample_grads(a2, g2)
    for i in range(B):
        np.testing.assert_allclose(P1[i], ref[i][0], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(P2[i], ref[i][1], rtol=1e-12, atol=1e-12)
    # norms: both the definition and the Gram (ghost) form of each sub-module
    for (a, g), k in (((a1, g1), 0), ((a2, g2), 1)):
        want = np.array([np.sum(ref[i][k] ** 2) for i in range(B)])
        np.testing.assert_allclose(oracle.linear_norm_sq(a, g), want, rtol=1e-12)
        np.testing.assert_allclose(oracle.linear_norm_sq_gram(a, g), want, rtol=1e-12)
    # clipped sums: sum_i C_i dL_i/dL
    C = np.array([0.3, 1.0, 0.0])
    np.testing.assert_allclose(oracle.weighted_grad(a1, g1, C), sum(C[i] * ref[i][0] for i in range(B)),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("act", ["relu", "tanh"])
def test_adapter_submodules_match_autograd(gen, act):
    tau = torch.relu if act == "relu" else torch.tanh
    x = torch.randn(B, T, p, generator=gen, dtype=torch.float64)
    D = torch.randn(p, r, generator=gen, dtype=torch.float64)
    U = torch.randn(r, p, generator=gen, dtype=torch.float64)
    dv = torch.randn(B, T, p, generator=gen, dtype=torch.float64)
    ref = _per_sample(lambda xi, D_, U_: tau(xi @ D_) @ U_ + xi, [D, U], x, dv)
    (a1, g1), (a2, g2) = oracle.adapter_submodules(x, D, U, dv, act)
    P1, P2 = oracle.per_sample_grads(a1, g1), oracle.per_sample_grads(a2, g2)
    for i in range(B):
        np.testing.assert_allclose(P1[i], ref[i][0], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(P2[i], ref[i][1], rtol=1e-12, atol=1e-12)
    if act == "relu":                      # some units are off: the mask matters
        assert np.any(a2 == 0.0) and np.any(a2 > 0.0)


def test_lora_rank_one_closed_form():
    """r = 1, T = 1: dL_i/dL = x_i^T (dv_i . R^T) and dL_i/dR = (x_i L)^T dv_i, by hand."""
    x = np.array([[[1.0, 2.0]]]); Lw = np.array([[3.0], [-1.0]]); Rw = np.array([[2.0, 0.5, -1.0]])
    dv = np.array([[[1.0, -2.0, 4.0]]])
    (a1, g1), (a2, g2) = oracle.lora_submodules(x, Lw, Rw, dv)
    # u = 1*3 + 2*(-1) = 1;  dv R^T = 2 - 1 - 4 = -3
    np.testing.assert_array_equal(oracle.per_sample_grads(a1, g1)[0], [[-3.0], [-6.0]])
    np.testing.assert_array_equal(oracle.per_sample_grads(a2, g2)[0], [[1.0, -2.0, 4.0]])
    assert oracle.linear_norm_sq(a1, g1)[0] == 45.0 and oracle.linear_norm_sq(a2, g2)[0] == 21.0
