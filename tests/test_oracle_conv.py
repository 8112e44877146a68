"""Pins of the oracle's convolution-as-linear-layer view (CPU only): unfold and the
token-major output gradient reproduce torch's conv2d and its per-sample weight
gradient, and the linear-layer definitions then give the conv layer's norms."""
import numpy as np
import pytest
import torch

import oracle


def _case(seed, B, Cin, H, W, Cout, k, stride, pad):
    gen = torch.Generator().manual_seed(seed)
    x = torch.randn(B, Cin, H, W, generator=gen, dtype=torch.float64)
    Wt = torch.randn(Cout, Cin, k, k, generator=gen, dtype=torch.float64)
    return x, Wt


@pytest.mark.parametrize("B,Cin,H,W,Cout,k,stride,pad", [
    (2, 3, 9, 7, 4, 3, 1, 1), (1, 2, 8, 8, 5, 3, 2, 1), (2, 4, 6, 5, 3, 1, 1, 0), (1, 3, 11, 11, 2, 7, 2, 3)])
def test_unfold_reproduces_conv2d(B, Cin, H, W, Cout, k, stride, pad):
    x, Wt = _case(B + H, B, Cin, H, W, Cout, k, stride, pad)
    s_ref = torch.nn.functional.conv2d(x, Wt, stride=stride, padding=pad).numpy()   # [B, Cout, Ho, Wo]
    a = oracle.unfold(x.numpy(), k, k, stride, pad)
    s = a @ Wt.reshape(Cout, -1).numpy().T                                          # [B, T, Cout]
    np.testing.assert_allclose(s, oracle.tokens_from_nchw(s_ref), rtol=1e-12, atol=1e-12)
    # padded columns are zero and change nothing
    a_pad = oracle.unfold(x.numpy(), k, k, stride, pad, ld=a.shape[2] + 5)
    np.testing.assert_array_equal(a_pad[:, :, :a.shape[2]], a)
    assert not np.any(a_pad[:, :, a.shape[2]:])


def test_tokens_from_nchw_small():
    y = np.arange(2 * 3 * 2 * 2, dtype=np.float64).reshape(2, 3, 2, 2)
    t = oracle.tokens_from_nchw(y)
    assert t.shape == (2, 4, 3)
    assert t[1, 2, 0] == y[1, 0, 1, 0] and t[0, 3, 2] == y[0, 2, 1, 1]


def test_conv_per_sample_grads_and_norms_match_autograd():
    B, Cin, H, W, Cout, k, stride, pad = 3, 2, 7, 6, 4, 3, 2, 1
    x, Wt = _case(11, B, Cin, H, W, Cout, k, stride, pad)
    gen = torch.Generator().manual_seed(5)
    Ho, Wo = oracle.conv_out_size(H, k, stride, pad), oracle.conv_out_size(W, k, stride, pad)
    dy = torch.randn(B, Cout, Ho, Wo, generator=gen, dtype=torch.float64)   # dL/ds
    a = oracle.unfold(x.numpy(), k, k, stride, pad)
    g = oracle.tokens_from_nchw(dy.numpy())
    P = oracle.per_sample_grads(a, g)                                        # [B, d, p]
    norms = oracle.linear_norm_sq(a, g)
    ghost = oracle.linear_norm_sq_gram(a, g)
    C = np.array([0.5, 2.0, 0.0])
    G = oracle.weighted_grad(a, g, C)
    for i in range(B):
        Wv = Wt.clone().requires_grad_(True)
        s = torch.nn.functional.conv2d(x[i:i + 1], Wv, stride=stride, padding=pad)
        (s * dy[i:i + 1]).sum().backward()
        gi = Wv.grad.reshape(Cout, -1).numpy().T                             # [d, p]
        np.testing.assert_allclose(P[i], gi, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(norms[i], (gi ** 2).sum(), rtol=1e-12)
        np.testing.assert_allclose(ghost[i], (gi ** 2).sum(), rtol=1e-10)
    # the clipped gradient of the conv weight is sum_i C_i grad_i
    Wv = Wt.clone().requires_grad_(True)
    s = torch.nn.functional.conv2d(x, Wv, stride=stride, padding=pad)
    (s * dy * torch.tensor(C).view(B, 1, 1, 1)).sum().backward()
    np.testing.assert_allclose(G, Wv.grad.reshape(Cout, -1).numpy().T, rtol=1e-12, atol=1e-12)


def _printed(x, v, sig):
    """x rounds to the printed value v (sig significant figures)."""
    if v == int(v) and v < 10:
        return x == v
    e = int(np.floor(np.log10(abs(v)))) - (sig - 1)
    return abs(x - v) <= 0.5 * 10.0 ** e


def test_resnet18_stack_reproduces_the_layerwise_decision_table():
    """The ResNet-18 stack at 224 x 224 (workload 6 without its three 1 x 1
    downsampling convolutions, which the paper's table leaves out): the output
    sizes from conv_out_size, the space of both ways (2T^2 with T = H_out W_out,
    p d with d = C_in k^2), the layer counts, the choice of use_ghost and the
    three totals reproduce the printed 18-layer column of Table "layerwise
    decision"."""
    import json
    import os
    import workloads as wl
    tab = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "layerwise_decision_resnet18.json")))
    layers = [L for L in wl.get(6).layers if L.kind != "conv" or L.conv[1] != 1]
    assert len(layers) == 18
    rows = []
    for L in layers:
        if L.kind == "conv":
            cin, k, stride, pad, hin = L.conv
            ho = oracle.conv_out_size(hin, k, stride, pad)
            assert ho * ho == L.T
            d = cin * k * k
        else:
            ho, d = 1, L.d
        ghost = oracle.use_ghost(L.T, d, L.p)
        assert oracle.use_ghost(L.T, L.d, L.p) == ghost          # padding d to 8 changes no choice here
        rows.append((ho, 2 * L.T * L.T, d * L.p, ghost))
    for st in tab["stages"]:
        mine = [r for r in rows if r[0] == st["hout"]]
        for key, col in (("ghost", 1), ("inst", 2)):
            printed = [(v, c) for v, c in st[key]]
            assert sum(c for _, c in printed) == len(mine), st["name"]
            vals = [r[col] for r in mine]
            for v, c in printed:                 # each printed group matches c layers of the stage
                hit = [x for x in vals if _printed(x, v, 2)]
                assert len(hit) == c, (st["name"], key, v)
        assert all(r[3] == (st["bold"] == "ghost") for r in mine), st["name"]
    tot_g = sum(r[1] for r in rows)
    tot_i = sum(r[2] for r in rows)
    tot_m = sum(min(r[1], r[2]) for r in rows)
    assert _printed(tot_g, *tab["total_ghost"])
    assert _printed(tot_i, *tab["total_inst"])
    assert _printed(tot_m, *tab["total_mixed"])
