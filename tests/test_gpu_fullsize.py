"""Parity at the full benchmark sizes, in the launch configuration bench.py
times (one bk_private_grad call over the whole stack).

The float64 oracle cannot redo whole stacks in a test's time, so each check
samples what the oracle can compute one piece at a time:
  * the ghost / instantiation choice of every layer (exact);
  * the per-sample norms of sampled layers (first, middle, last, every path
    kind present), against the oracle on the same inputs;
  * the clip factors and totals from the GPU's whole [L, B] norm table;
  * sampled blocks (up to 32 x 32) of the clipped gradients of the sampled layers
    (run without noise), against the oracle's clipped gradient restricted to
    those rows and columns, and whole rows of the embedding gradient
    (most frequent ids and absent ids);
  * the noise actually added by the noisy run (difference of the two runs)
    at the sampled entries, against the oracle's Philox + Box-Muller draws.
Inputs are drawn on the device by the workload generator and copied to the
host for the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda"
NORM_TOL = 2e-2       # bf16 inputs, fp32 accumulation
GRAD_TOL = 2e-2


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available()
    import paper_2210_00038_amd as m
    return m


def _run(bk, w, ins, std):
    n, B = len(w.layers), w.B
    Gs = [torch.empty(L.d, L.p, device=DEV) for L in w.layers]
    arr = bk.make_layers([{"kind": bk.BK_EMBEDDING if L.kind == "embed" else bk.BK_LINEAR, "x": x, "g": g,
                           "G": G, "V": L.d} for L, (x, g), G in zip(w.layers, ins, Gs)])
    norm_sq = torch.empty(n, B, device=DEV)
    C = torch.empty(B, device=DEV)
    tot = torch.empty(B, device=DEV)
    mode = bk.BK_CLIP_ABADI if w.clip == "abadi" else bk.BK_CLIP_AUTO
    dt = bk.BK_BF16 if w.dtype == "bf16" else bk.BK_F32
    bk.bk_private_grad(arr, n, dt, B, mode, w.R, w.gamma, std, w.wid, 0, norm_sq, C, tot)
    torch.cuda.synchronize()
    return norm_sq.cpu().numpy().astype(np.float64), C.cpu().numpy(), tot.cpu().numpy(), Gs


def _sample_layers(w):
    n = len(w.layers)
    pick = {0, n // 2, n - 1}
    kinds = {}
    for l, L in enumerate(w.layers):
        kind = "embed" if L.kind == "embed" else ("ghost" if oracle.use_ghost(L.T, L.d, L.p) else "inst")
        kinds.setdefault(kind, l)
    return sorted(pick | set(kinds.values()))


@pytest.mark.parametrize("wid", [2, 3, 4, 5, 7])
def test_full_stack_sampled_parity(bk, wid):
    w = wl.get(wid)
    print(f"workload {wid}: {w.name}, {len(w.layers)} layers, B={w.B}", flush=True)
    torch.manual_seed(0)
    ins = [wl.draw_layer(w, l, device=DEV) for l in range(len(w.layers))]
    norms, C, tot, G0 = _run(bk, w, ins, 0.0)
    _, C1, _, G1 = _run(bk, w, ins, w.noise_std)
    assert np.array_equal(C, C1)                           # noise does not touch the clip factors

    # path choice of every layer (Section 3.2 rule), exact
    for L in w.layers:
        if L.kind != "embed":
            assert bk.bk_use_ghost(L.T, L.d, L.p) == oracle.use_ghost(L.T, L.d, L.p)

    # clip factors and totals from the GPU's whole norm table
    ref_tot = oracle.aggregate(norms)
    ref_C = oracle.clip_factors(ref_tot, w.clip, w.R, w.gamma)
    assert np.max(np.abs(tot - ref_tot) / ref_tot) <= 1e-5
    assert np.max(np.abs(C - ref_C) / ref_C) <= 1e-5

    rng = np.random.default_rng(wid)
    for l in _sample_layers(w):
        L = w.layers[l]
        x, g = (t.cpu() for t in ins[l])
        if L.kind == "embed":
            ref_n = oracle.embed_norm_sq(x, g, L.d)
        elif oracle.use_ghost(L.T, L.d, L.p):
            ref_n = oracle.linear_norm_sq_gram(x, g)
        else:
            ref_n = oracle.linear_norm_sq(x, g)
        rel = np.max(np.abs(norms[l] - ref_n) / ref_n)
        print(f"  layer {l} ({L.kind} {L.d}x{L.p} T={L.T}): norm rel err {rel:.2e}", flush=True)
        assert rel <= NORM_TOL, l

        Gg = G0[l]
        noise = (G1[l] - G0[l])
        sel = lambda t, r, c: t[torch.as_tensor(r, device=DEV)][:, torch.as_tensor(c, device=DEV)].cpu().numpy()
        if L.kind == "embed":
            ids = x.numpy().ravel()
            counts = np.bincount(ids, minlength=L.d)
            rows = np.concatenate([np.argsort(-counts)[:4], np.flatnonzero(counts == 0)[:2],
                                   rng.choice(np.flatnonzero(counts), 2)])
            ref_full = oracle.embed_weighted_grad(x, g, C, L.d)
            cols = np.arange(L.p)
            ref = ref_full[rows]
            got = sel(Gg, rows, cols)
            assert np.all(got[counts[rows] == 0] == 0.0)
            nz = counts[rows] > 0
            err = np.linalg.norm(got[nz] - ref[nz]) / np.linalg.norm(ref[nz])
        else:
            rows = np.sort(rng.choice(L.d, min(32, L.d), replace=False))
            cols = np.sort(rng.choice(L.p, min(32, L.p), replace=False))
            ref = oracle.weighted_grad(x[:, :, torch.from_numpy(rows)], g[:, :, torch.from_numpy(cols)], C)
            got = sel(Gg, rows, cols)
            err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        print(f"  layer {l}: gradient block frob err {err:.2e}", flush=True)
        assert err <= GRAD_TOL, l

        # the noise added to this layer at the same entries (tensor_id = l, step 0)
        elems = rows[:, None].astype(np.int64) * L.p + cols[None, :]
        got_noise = sel(noise, rows, cols)
        ref_noise = w.noise_std * oracle.noise_at(elems, w.wid, l, 0)
        # |G + n| <~ 6 std rounds to fp32 with an error near 2^-24 * 6 std per operation
        assert np.max(np.abs(got_noise - ref_noise)) <= 2e-5 * w.noise_std * 8, l
    del ins, G0, G1
    torch.cuda.empty_cache()


def test_config1_full(bk):
    """The single fp32 layer runs whole through the oracle."""
    w = wl.get(1)
    a, g = wl.draw_linear(w, 0)
    norms, C, tot, G0 = _run(bk, w, [(a.to(DEV), g.to(DEV))], 0.0)
    _, _, _, G1 = _run(bk, w, [(a.to(DEV), g.to(DEV))], w.noise_std)
    ref = oracle.bk_stack(list(w.layers), [(a, g)], w.clip, w.R, w.gamma, w.noise_std, w.wid)
    assert np.max(np.abs(norms - ref["norms"]) / ref["norms"]) <= 1e-5
    assert np.max(np.abs(C - ref["C"]) / ref["C"]) <= 1e-5
    G = G0[0].cpu().numpy()
    assert np.linalg.norm(G - ref["G"][0]) / np.linalg.norm(ref["G"][0]) <= 1e-4
    noise = G1[0].cpu().numpy() - G
    assert np.max(np.abs(noise - (ref["Ghat"][0] - ref["G"][0]))) <= 2e-5 * 8


def test_conv_stack_full_sampled_parity(bk):
    """ResNet-18 convolutions at 224x224, B = 16: the GPU unfolds x and makes
    dL/ds token-major (checked bit-exact against the oracle's unfold on sampled
    layers), then one bk_private_grad call runs the stack as in bench.py."""
    w = wl.get(6)
    print(f"workload 6: {w.name}, {len(w.layers)} layers, B={w.B}", flush=True)
    raw = [wl.draw_layer(w, l, device=DEV) for l in range(len(w.layers))]
    ins = []
    for L, (x, dy) in zip(w.layers, raw):
        if L.kind == "conv":
            cin, k, stride, pad, _ = L.conv
            ins.append((bk.bk_unfold(x, k, k, stride, pad, L.d), bk.bk_tokens_from_nchw(dy)))
        else:
            ins.append((x, dy))
    norms, C, tot, G0 = _run(bk, w, ins, 0.0)
    for L in w.layers:
        assert bk.bk_use_ghost(L.T, L.d, L.p) == oracle.use_ghost(L.T, L.d, L.p)
    ref_tot = oracle.aggregate(norms)
    assert np.max(np.abs(C - oracle.clip_factors(ref_tot, w.clip, w.R, w.gamma)) / C) <= 1e-5

    n = len(w.layers)
    picks = {0, 9, 10, 14, n - 2, n - 1}          # 7x7 stem, 1x1 downsamples, ghost 3x3, classifier
    rng = np.random.default_rng(6)
    for l in sorted(picks):
        L = w.layers[l]
        x, dy = (t.cpu() for t in raw[l])
        if L.kind == "conv":
            cin, k, stride, pad, _ = L.conv
            a, g = oracle.unfold(x, k, k, stride, pad, L.d), oracle.tokens_from_nchw(dy)
            assert np.array_equal(ins[l][0].cpu().double().numpy(), a), l
            assert np.array_equal(ins[l][1].cpu().double().numpy(), g), l
        else:
            a, g = x.double().numpy(), dy.double().numpy()
        ref_n = oracle.linear_norm_sq_gram(a, g) if oracle.use_ghost(L.T, L.d, L.p) else oracle.linear_norm_sq(a, g)
        rel = np.max(np.abs(norms[l] - ref_n) / ref_n)
        print(f"  layer {l} ({L.kind} T={L.T} d={L.d} p={L.p}): norm rel err {rel:.2e}", flush=True)
        assert rel <= NORM_TOL, l
        rows = np.sort(rng.choice(L.d, min(32, L.d), replace=False))
        cols = np.sort(rng.choice(L.p, 32, replace=False))
        ref = oracle.weighted_grad(a[:, :, rows], g[:, :, cols], C)
        got = G0[l][torch.as_tensor(rows, device=DEV)][:, torch.as_tensor(cols, device=DEV)].cpu().numpy()
        pad_rows = rows >= (L.conv[0] * L.conv[1] ** 2 if L.kind == "conv" else L.d)
        assert np.all(got[pad_rows] == 0.0), l                # zero columns of a give zero gradient rows
        err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        print(f"  layer {l}: gradient block frob err {err:.2e}", flush=True)
        assert err <= GRAD_TOL, l
    del raw, ins, G0
    torch.cuda.empty_cache()


def test_gpt2_bias_layernorm_full_sampled(bk):
    """GPT-2 small with every bias and LayerNorm affine (73 layers, B = 32,
    T = 128), one bk_private_grad call as bench.py runs it: sampled layer
    norms, gamma / beta / bias gradients against the oracle; and accumulation
    of two identical physical batches, which must give exactly twice the
    single-batch clipped gradients (each pass is deterministic)."""
    w = wl.get(8)
    n, B = len(w.layers), w.B
    print(f"workload 8: {w.name}, {n} layers, B={B}", flush=True)
    ins = [wl.draw_layer(w, l, device=DEV) for l in range(n)]
    kinds = {"norm": bk.BK_NORM_AFFINE}
    Gs = [torch.empty((L.p,) if L.kind == "norm" else (L.d, L.p), device=DEV) for L in w.layers]
    Gbs = [torch.empty(L.p, device=DEV) for L in w.layers]
    Ps = [torch.empty(B, L.p, device=DEV) if L.kind == "norm" else None for L in w.layers]
    Pbs = [torch.empty(B, L.p, device=DEV) for L in w.layers]
    mk = lambda acc: bk.make_layers([{"kind": kinds.get(L.kind, bk.BK_LINEAR), "x": x, "g": g, "G": G, "P": P,
                                      "bias": True, "Gb": Gb, "Pb": Pb, "accumulate": acc}
                                     for L, (x, g), G, P, Gb, Pb in zip(w.layers, ins, Gs, Ps, Gbs, Pbs)])
    norm_sq, C = torch.empty(n, B, device=DEV), torch.empty(B, device=DEV)
    bk.bk_private_grad(mk(False), n, bk.BK_BF16, B, bk.BK_CLIP_AUTO, w.R, w.gamma, 0.0, 8, 0, norm_sq, C, None)
    torch.cuda.synchronize()
    G1 = [G.clone() for G in Gs]
    Gb1 = [G.clone() for G in Gbs]
    norms, Cc = norm_sq.cpu().numpy().astype(np.float64), C.cpu().numpy()
    ref_C = oracle.clip_factors(oracle.aggregate(norms), w.clip, w.R, w.gamma)
    assert np.max(np.abs(Cc - ref_C) / ref_C) <= 1e-5
    for l in (0, 1, 2, 5, n - 1):                    # ln_1, qkv, attn out, mlp down, final ln
        L = w.layers[l]
        x, g = (t.cpu() for t in ins[l])
        ref_n = oracle.bk_layer_norm(L.kind, x, g, L.d, True)
        rel = np.max(np.abs(norms[l] - ref_n) / ref_n)
        print(f"  layer {l} ({L.kind} {L.d}x{L.p}): norm rel err {rel:.2e}", flush=True)
        assert rel <= NORM_TOL, l
        if L.kind == "norm":
            ref_G = oracle.weighted_sum(oracle.norm_affine_sums(x, g)[0], Cc)
            got = G1[l].cpu().numpy()
        else:
            rows = np.sort(np.random.default_rng(l).choice(L.d, 32, replace=False))
            cols = np.sort(np.random.default_rng(l + 1).choice(L.p, 32, replace=False))
            ref_G = oracle.weighted_grad(x[:, :, torch.from_numpy(rows)], g[:, :, torch.from_numpy(cols)], Cc)
            got = G1[l].cpu().numpy()[rows][:, cols]
        ref_b = oracle.weighted_sum(oracle.bias_sums(g), Cc)
        assert np.linalg.norm(got - ref_G) / np.linalg.norm(ref_G) <= GRAD_TOL, l
        assert np.linalg.norm(Gb1[l].cpu().numpy() - ref_b) / np.linalg.norm(ref_b) <= GRAD_TOL, l
    # a second, identical physical batch accumulated onto the first
    bk.bk_private_grad(mk(True), n, bk.BK_BF16, B, bk.BK_CLIP_AUTO, w.R, w.gamma, 0.0, 8, 0, norm_sq, C, None)
    torch.cuda.synchronize()
    for l in range(n):
        assert torch.equal(Gs[l], 2 * G1[l]), l
        assert torch.equal(Gbs[l], 2 * Gb1[l]), l
    del ins, Gs, Gbs, G1, Gb1
    torch.cuda.empty_cache()
