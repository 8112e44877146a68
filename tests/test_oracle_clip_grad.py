"""Pins of the oracle's aggregation, clip factors and clipped gradients (CPU only)."""
import numpy as np
import pytest
import torch

import oracle

rng = np.random.default_rng(7)


def _rand(*shape):
    return rng.standard_normal(shape)


def test_aggregate_sums_layers():
    n = np.abs(_rand(5, 3))
    np.testing.assert_allclose(oracle.aggregate(n), n.sum(axis=0), rtol=1e-15)


def test_clip_closed_forms():
    tot = np.array([0.0, 0.25, 1.0, 4.0, 100.0])           # norms 0, .5, 1, 2, 10
    np.testing.assert_array_equal(oracle.clip_factors(tot, "abadi", R=1.0), [1, 1, 1, 0.5, 0.1])
    np.testing.assert_allclose(oracle.clip_factors(tot, "abadi", R=2.0), [1, 1, 1, 1, 0.2], rtol=1e-15)
    np.testing.assert_allclose(oracle.clip_factors(tot, "auto", gamma=0.01),
                               [100.0, 1 / 0.51, 1 / 1.01, 1 / 2.01, 1 / 10.01], rtol=1e-15)
    # pure normalisation (gamma = 0) of a zero gradient gives weight 0
    np.testing.assert_array_equal(oracle.clip_factors([0.0, 4.0], "auto", gamma=0.0), [0.0, 0.5])
    with pytest.raises(ValueError):
        oracle.clip_factors([1.0], "abadi", R=0.0)


def test_clipped_norms_bounded():
    tot = np.abs(_rand(100)) * 50
    nrm = np.sqrt(tot)
    assert np.all(oracle.clip_factors(tot, "abadi", R=1.5) * nrm <= 1.5 * (1 + 1e-15))
    assert np.all(oracle.clip_factors(tot, "auto", gamma=0.01) * nrm < 1.0)


def test_weighted_grad_unit_weights_is_standard_gradient():
    B, T, d, p = 3, 5, 4, 6
    a, g = _rand(B, T, d), _rand(B, T, p)
    # the standard (non-private) parameter gradient a^T dL/ds over the flattened batch
    ref = torch.from_numpy(a).reshape(B * T, d).T.matmul(torch.from_numpy(g).reshape(B * T, p)).numpy()
    np.testing.assert_allclose(oracle.weighted_grad(a, g, np.ones(B)), ref, rtol=1e-12, atol=1e-12)


def test_weighted_grad_bruteforce_and_basis_weights():
    B, T, d, p = 3, 4, 3, 2
    a, g = _rand(B, T, d), _rand(B, T, p)
    C = np.array([0.5, -2.0, 3.0])
    ref = np.zeros((d, p))
    for i in range(B):
        for j in range(d):
            for k in range(p):
                for t in range(T):
                    ref[j, k] += C[i] * a[i, t, j] * g[i, t, k]
    np.testing.assert_allclose(oracle.weighted_grad(a, g, C), ref, rtol=1e-12, atol=1e-14)
    for j in range(B):
        e = np.zeros(B)
        e[j] = 1.0
        np.testing.assert_allclose(oracle.weighted_grad(a, g, e), a[j].T @ g[j], rtol=1e-12, atol=1e-14)


def test_weighted_grad_linear_in_C_and_permutation_invariant():
    B, T, d, p = 4, 3, 5, 4
    a, g = _rand(B, T, d), _rand(B, T, p)
    C1, C2 = _rand(B), _rand(B)
    lhs = oracle.weighted_grad(a, g, 2 * C1 - C2)
    rhs = 2 * oracle.weighted_grad(a, g, C1) - oracle.weighted_grad(a, g, C2)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-12)
    bp = rng.permutation(B)
    np.testing.assert_allclose(oracle.weighted_grad(a[bp], g[bp], C1[bp]), oracle.weighted_grad(a, g, C1),
                               rtol=1e-12, atol=1e-12)


def test_embedding_weighted_grad_equals_one_hot():
    V, B, T, p = 9, 3, 6, 4
    ids = rng.integers(0, V, size=(B, T))
    g = _rand(B, T, p)
    C = np.abs(_rand(B))
    onehot = np.zeros((B, T, V))
    np.put_along_axis(onehot, ids[..., None], 1.0, axis=-1)
    np.testing.assert_allclose(oracle.embed_weighted_grad(ids, g, C, V), oracle.weighted_grad(onehot, g, C),
                               rtol=1e-12, atol=1e-14)


def test_stack_composes_the_steps():
    from workloads import Layer
    layers = [Layer("linear", 5, 4, 3), Layer("linear", 5, 3, 6), Layer("embed", 5, 10, 3)]
    B = 3
    ins = [(_rand(B, 5, 4), _rand(B, 5, 3)), (_rand(B, 5, 3), _rand(B, 5, 6)),
           (rng.integers(0, 10, size=(B, 5)), _rand(B, 5, 3))]
    out = oracle.bk_stack(layers, ins, "abadi", 1.0, 0.0, 0.7, seed=3)
    # per-sample gradient norms over the whole model, from instantiated per-sample gradients
    tot = np.zeros(B)
    for i in range(B):
        for L, (x, g) in zip(layers, ins):
            if L.kind == "embed":
                gi = np.zeros((L.d, L.p))
                for t in range(L.T):
                    gi[x[i, t]] += g[i, t]
            else:
                gi = x[i].T @ g[i]
            tot[i] += np.sum(gi ** 2)
    np.testing.assert_allclose(out["total"], tot, rtol=1e-12)
    C = np.minimum(1.0, 1.0 / np.sqrt(tot))
    np.testing.assert_allclose(out["C"], C, rtol=1e-14)
    np.testing.assert_allclose(out["G"][0], sum(C[i] * ins[0][0][i].T @ ins[0][1][i] for i in range(B)),
                               rtol=1e-12)
    assert out["paths"] == ["ghost" if 2 * 25 < 12 else "inst", "inst", "embed"]
    assert len(out["Ghat"]) == 3 and out["Ghat"][2].shape == (10, 3)


# --- BK-MixOpt: stored per-sample gradients and their weighted sum (App. B.4.1, B.5) ---

def test_per_sample_grads_hand_example():
    # one token: a_1 = (1, 2), g_1 = (3): the per-sample gradient is the outer product
    P = oracle.per_sample_grads(np.array([[[1.0, 2.0]]]), np.array([[[3.0]]]))
    np.testing.assert_array_equal(P, [[[3.0], [6.0]]])
    # two tokens add: a = [(1,0),(0,1)], g = [(1,1),(2,-1)] -> [[1,1],[2,-1]]
    P = oracle.per_sample_grads(np.array([[[1.0, 0.0], [0.0, 1.0]]]), np.array([[[1.0, 1.0], [2.0, -1.0]]]))
    np.testing.assert_array_equal(P, [[[1.0, 1.0], [2.0, -1.0]]])


def test_per_sample_grad_norms_match_ghost_form():
    a, g = _rand(4, 7, 5), _rand(4, 7, 3)
    P = oracle.per_sample_grads(a, g)
    np.testing.assert_allclose((P ** 2).sum(axis=(1, 2)), oracle.linear_norm_sq_gram(a, g), rtol=1e-12)


def test_weighted_sum_equals_book_keeping_gemm():
    # sum_i C_i (a_i^T g_i) is the same matrix as a^T diag(C) g over the flattened rows
    a, g, C = _rand(5, 6, 4), _rand(5, 6, 7), np.abs(_rand(5))
    np.testing.assert_allclose(oracle.weighted_sum(oracle.per_sample_grads(a, g), C),
                               oracle.weighted_grad(a, g, C), rtol=1e-12, atol=1e-12)


def test_weighted_sum_selects_and_is_linear():
    P = _rand(4, 3, 2)
    for j in range(4):
        e = np.zeros(4)
        e[j] = 1.0
        np.testing.assert_array_equal(oracle.weighted_sum(P, e), P[j])
    C1, C2 = _rand(4), _rand(4)
    np.testing.assert_allclose(oracle.weighted_sum(P, C1 + 2 * C2),
                               oracle.weighted_sum(P, C1) + 2 * oracle.weighted_sum(P, C2), rtol=1e-12, atol=1e-12)


def test_mixopt_stack_matches_base_stack():
    # BK-MixOpt changes how G_l is formed on instantiated layers, not its value
    class L:
        def __init__(self, kind, T, d, p):
            self.kind, self.T, self.d, self.p = kind, T, d, p
    layers = [L("linear", 6, 3, 4), L("linear", 2, 5, 4)]          # instantiate (72 >= 12), ghost (8 < 20)
    ins = [(_rand(3, 6, 3), _rand(3, 6, 4)), (_rand(3, 2, 5), _rand(3, 2, 4))]
    base = oracle.bk_stack(layers, ins, "abadi", 1.0, 0.0, 0.0, 1, with_noise=False)
    mix = oracle.bk_stack(layers, ins, "abadi", 1.0, 0.0, 0.0, 1, with_noise=False, mixopt=True)
    assert base["paths"] == ["inst", "ghost"]
    for gb, gm in zip(base["G"], mix["G"]):
        np.testing.assert_allclose(gm, gb, rtol=1e-12, atol=1e-12)
