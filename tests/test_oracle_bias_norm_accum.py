"""Pins of the per-sample bias and normalization-affine terms and of gradient
accumulation in the oracle.

Bias and affine terms are compared with torch autograd per-sample gradients of
the layers themselves (float64, CPU, loss of sample i = <y_i, dv_i>); the
accumulation with the identity that a logical batch split into physical
batches, each clipped on its own, gives the same clipped sum as the whole
logical batch clipped at once (per-sample clipping does not couple samples)."""
import numpy as np
import pytest
import torch

import oracle

B, T, d, p = 4, 6, 5, 7


class _L:
    def __init__(self, kind, T, d, p, bias=False):
        self.kind, self.T, self.d, self.p, self.bias = kind, T, d, p, bias


def _per_sample(fn, params, x, dv):
    out = []
    for i in range(x.shape[0]):
        ps = [q.detach().clone().requires_grad_(True) for q in params]
        (fn(x[i:i + 1], *ps) * dv[i:i + 1]).sum().backward()
        out.append([q.grad.numpy().copy() for q in ps])
    return out


@pytest.fixture
def gen():
    return torch.Generator().manual_seed(616)


def test_bias_matches_autograd(gen):
    a = torch.randn(B, T, d, generator=gen, dtype=torch.float64)
    W = torch.randn(p, d, generator=gen, dtype=torch.float64)
    b = torch.randn(p, generator=gen, dtype=torch.float64)
    dv = torch.randn(B, T, p, generator=gen, dtype=torch.float64)
    ref = _per_sample(lambda x, W_, b_: torch.nn.functional.linear(x, W_, b_), [W, b], a, dv)
    s = oracle.bias_sums(dv)
    for i in range(B):
        np.testing.assert_allclose(s[i], ref[i][1], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(oracle.per_sample_grads(a, dv)[i], ref[i][0].T, rtol=1e-12, atol=1e-12)
    want = np.array([np.sum(ref[i][0] ** 2) + np.sum(ref[i][1] ** 2) for i in range(B)])
    np.testing.assert_allclose(oracle.bk_layer_norm("linear", a, dv, d, bias=True), want, rtol=1e-12)
    C = np.array([0.5, 0.0, 2.0, 1.0])
    np.testing.assert_allclose(oracle.weighted_sum(s, C), sum(C[i] * ref[i][1] for i in range(B)), rtol=1e-12)


def test_bias_hand_example():
    g = np.array([[[1.0, -2.0], [3.0, 0.5]]])           # B=1, T=2, p=2
    np.testing.assert_array_equal(oracle.bias_sums(g), [[4.0, -1.5]])
    assert oracle.bias_norm_sq(g)[0] == 16.0 + 2.25


def test_layernorm_affine_matches_autograd(gen):
    z = torch.randn(B, T, p, generator=gen, dtype=torch.float64) * 3 + 1
    dv = torch.randn(B, T, p, generator=gen, dtype=torch.float64)
    gam, bet = torch.ones(p, dtype=torch.float64), torch.zeros(p, dtype=torch.float64)
    ln = lambda x, g_, b_: torch.nn.functional.layer_norm(x, (p,), g_, b_, 1e-5)
    ref = _per_sample(ln, [gam, bet], z, dv)
    xhat = ln(z, gam, bet).detach()                     # the normalized input (unit affine)
    u, s = oracle.norm_affine_sums(xhat, dv)
    for i in range(B):
        np.testing.assert_allclose(u[i], ref[i][0], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(s[i], ref[i][1], rtol=1e-10, atol=1e-12)
    want = np.array([np.sum(ref[i][0] ** 2) + np.sum(ref[i][1] ** 2) for i in range(B)])
    np.testing.assert_allclose(oracle.bk_layer_norm("norm", xhat, dv, p, bias=True), want, rtol=1e-10)
    np.testing.assert_allclose(oracle.bk_layer_norm("norm", xhat, dv, p, bias=False),
                               [np.sum(ref[i][0] ** 2) for i in range(B)], rtol=1e-10)


def test_groupnorm_affine_matches_autograd(gen):
    """GroupNorm on NCHW: its per-channel affine is the same form with tokens =
    spatial positions and features = channels (token-major layout)."""
    Cc, H, Wd, groups = 6, 3, 4, 3
    z = torch.randn(B, Cc, H, Wd, generator=gen, dtype=torch.float64)
    dv = torch.randn(B, Cc, H, Wd, generator=gen, dtype=torch.float64)
    gam, bet = torch.ones(Cc, dtype=torch.float64), torch.zeros(Cc, dtype=torch.float64)
    gn = lambda x, g_, b_: torch.nn.functional.group_norm(x, groups, g_, b_, 1e-5)
    ref = _per_sample(gn, [gam, bet], z, dv)
    xhat = oracle.tokens_from_nchw(gn(z, gam, bet).detach().numpy())
    u, s = oracle.norm_affine_sums(xhat, oracle.tokens_from_nchw(dv.numpy()))
    for i in range(B):
        np.testing.assert_allclose(u[i], ref[i][0], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(s[i], ref[i][1], rtol=1e-10, atol=1e-12)


def test_stack_with_bias_and_norm_layers(gen):
    layers = [_L("linear", T, d, p, bias=True), _L("norm", T, p, p, bias=True), _L("linear", T, p, 3)]
    ins = [(torch.randn(B, T, d, generator=gen), torch.randn(B, T, p, generator=gen)),
           (torch.randn(B, T, p, generator=gen), torch.randn(B, T, p, generator=gen)),
           (torch.randn(B, T, p, generator=gen), torch.randn(B, T, 3, generator=gen))]
    r = oracle.bk_stack(layers, ins, "abadi", 1.0, 0.0, 0.5, seed=3)
    assert r["paths"] == ["inst", "norm", "inst"]
    n0 = oracle.linear_norm_sq(*ins[0]) + oracle.bias_norm_sq(ins[0][1])
    np.testing.assert_allclose(r["norms"][0], n0, rtol=1e-12)
    np.testing.assert_allclose(r["G"][1], oracle.weighted_sum(oracle.norm_affine_sums(*ins[1])[0], r["C"]), rtol=1e-12)
    np.testing.assert_allclose(r["Gb"][1], oracle.weighted_sum(oracle.bias_sums(ins[1][1]), r["C"]), rtol=1e-12)
    assert r["Gb"][2] is None and r["Gbhat"][2] is None
    # bias noise uses its own stream
    noise_w = r["Ghat"][0] - r["G"][0]
    noise_b = r["Gbhat"][0] - r["Gb"][0]
    np.testing.assert_allclose(noise_b, 0.5 * oracle.noise(p, 3, oracle.BIAS_TENSOR | 0, 0), rtol=1e-12)
    assert not np.allclose(noise_b, noise_w.ravel()[:p])


def test_accumulation_equals_logical_batch(gen):
    layers = [_L("linear", T, d, p, bias=True), _L("linear", T, p, 8), _L("norm", T, 8, 8, bias=True)]
    full = [(torch.randn(8, T, d, generator=gen), torch.randn(8, T, p, generator=gen)),
            (torch.randn(8, T, p, generator=gen), torch.randn(8, T, 8, generator=gen)),
            (torch.randn(8, T, 8, generator=gen), torch.randn(8, T, 8, generator=gen))]
    split = [[(x[:3], g[:3]) for x, g in full], [(x[3:5], g[3:5]) for x, g in full],
             [(x[5:], g[5:]) for x, g in full]]
    one = oracle.bk_stack(layers, full, "auto", 1.0, 0.01, 0.0, seed=1, with_noise=False)
    acc = oracle.logical_batch(layers, split, "auto", 1.0, 0.01, 0.8, seed=1, step=2)
    np.testing.assert_allclose(np.concatenate(acc["C"]), one["C"], rtol=1e-13)
    for l in range(3):
        np.testing.assert_allclose(acc["G"][l], one["G"][l], rtol=1e-11, atol=1e-13)
        # noise drawn once for the logical batch
        np.testing.assert_allclose(acc["Ghat"][l] - acc["G"][l],
                                   0.8 * oracle.noise(acc["G"][l].size, 1, l, 2).reshape(acc["G"][l].shape),
                                   rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(acc["Gb"][0], one["Gb"][0], rtol=1e-11, atol=1e-13)
    assert acc["Gb"][1] is None
