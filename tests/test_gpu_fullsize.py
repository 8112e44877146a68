"""Parity at the full benchmark sizes, in the launch configuration bench.py
times: one bk_private_grad call over the whole stack (after one bk_conv_prep
for a convolution stack).

Every layer of every stack is compared with the float64 oracle on the same
inputs (drawn on the device by the workload generator, copied to the host):
  * the ghost / instantiation choice (exact);
  * the per-sample norms of every layer: the oracle's definition, or its Gram
    form where that costs fewer flops (the CPU tests pin the two to each
    other and to brute force);
  * the totals and clip factors against oracle.aggregate / oracle.clip_factors
    of the ORACLE's own norm table;
  * a 32 x 32 block of every layer's clipped gradient (random rows and
    columns plus the last of each) against oracle.weighted_grad with the
    oracle's C; whole gamma / beta / bias gradients; whole rows of the
    embedding gradient (most frequent, absent and random ids);
  * the same blocks from bk_weighted_grads with power-of-two clip weights
    (one of them 0), which every kernel variant applies without rounding, so
    the tight guard holds on every layer whatever the variant;
  * the noise actually added (a noisy run minus a noiseless one) at the same
    entries, against the oracle's Philox + Box-Muller draws.
Each comparison has two bounds: the 2e-2 gate of the targets and a guard near
the measured error (tests/tolerances.py), which one dropped token row breaks
(tests/test_guards_cpu.py).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from tolerances import GRAD_GATE, GRAD_GUARD_EXACT, NORM_GATE, NORM_GUARD, grad_guard

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available()
    import paper_2210_00038_amd as m
    return m


def _rel(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    return float(np.max(np.abs(x - ref) / np.abs(ref))) if ref.size else 0.0


def _frob(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    return float(np.linalg.norm(x - ref) / np.linalg.norm(ref))


class Stack:
    """Device inputs and outputs of one workload, laid out as bench.py lays them."""

    def __init__(self, bk, w, time_rule=False, mixopt=False):
        self.bk, self.w = bk, w
        B, n = w.B, len(w.layers)
        self.raw = [wl.draw_layer(w, l, device=DEV) for l in range(n)]
        self.ins, convs = [], []
        for L, (x, g) in zip(w.layers, self.raw):
            if L.kind == "conv":
                a = torch.empty(B, L.T, L.d, dtype=w.torch_dtype, device=DEV)
                gt = torch.empty(B, L.T, L.p, dtype=w.torch_dtype, device=DEV)
                convs.append({"x": x, "dy": g, "a": a, "g": gt, "k": L.conv[1], "stride": L.conv[2],
                              "pad": L.conv[3], "ld": L.d})
                self.ins.append((a, gt))
            else:
                self.ins.append((x, g))
        self.dt = bk.BK_BF16 if w.dtype == "bf16" else bk.BK_F32
        if convs:
            bk.bk_conv_prep(bk.make_convs(convs), len(convs), self.dt, B)
        self.Gs = [torch.empty((L.p,) if L.kind == "norm" else (L.d, L.p), device=DEV) for L in w.layers]
        self.Gbs = [torch.empty(L.p, device=DEV) if L.bias else None for L in w.layers]
        # the per-sample gamma / bias sums pass from the norm phase to the
        # gradient phase through these buffers: the Stack keeps them alive
        self.Ps = [torch.empty(B, L.p, device=DEV) if L.kind == "norm" else None for L in w.layers]
        if mixopt:   # BK-MixOpt: the layers that instantiate keep their per-sample gradients
            rule = bk.bk_use_ghost_time if time_rule else bk.bk_use_ghost
            self.Ps = [torch.empty(B, L.d, L.p, device=DEV) if L.kind in ("linear", "conv") and
                       not rule(L.T, L.d, L.p) else P for L, P in zip(w.layers, self.Ps)]
        self.Pbs = [torch.empty(B, L.p, device=DEV) if L.bias else None for L in w.layers]
        kinds = {"embed": bk.BK_EMBEDDING, "norm": bk.BK_NORM_AFFINE}
        self.arr = bk.make_layers([{"kind": kinds.get(L.kind, bk.BK_LINEAR), "x": x, "g": g, "G": G,
                                    "V": L.d, "P": P, "bias": L.bias, "Gb": Gb, "Pb": Pb,
                                    "time_rule": time_rule, "mixopt": mixopt}
                                   for L, (x, g), G, P, Gb, Pb in
                                   zip(w.layers, self.ins, self.Gs, self.Ps, self.Gbs, self.Pbs)])
        self.mode = bk.BK_CLIP_ABADI if w.clip == "abadi" else bk.BK_CLIP_AUTO

    def private_grad(self, std):
        w, n, B = self.w, len(self.w.layers), self.w.B
        norm_sq, C, tot = (torch.empty(n, B, device=DEV), torch.empty(B, device=DEV),
                           torch.empty(B, device=DEV))
        self.bk.bk_private_grad(self.arr, n, self.dt, B, self.mode, w.R, w.gamma, std, w.wid, 0, norm_sq, C, tot)
        torch.cuda.synchronize()
        return norm_sq.cpu().numpy().astype(np.float64), C.cpu().numpy(), tot.cpu().numpy()

    def weighted_grads(self, C):
        self.bk.bk_weighted_grads(self.arr, len(self.w.layers), torch.as_tensor(C, dtype=torch.float32,
                                                                                device=DEV),
                                  self.dt, self.w.B)
        torch.cuda.synchronize()


def _take(t, rows, cols):
    """t[rows][:, cols] of a device matrix (or t[cols] of a vector) as float64."""
    c = torch.as_tensor(cols, device=DEV)
    if t.dim() == 1:
        return t[c].double().cpu().numpy()
    return t[torch.as_tensor(rows, device=DEV)][:, c].double().cpu().numpy()


def _pick(rng, n, k=32):
    """k sorted indices in [0, n) that always include the last one."""
    if n <= k:
        return np.arange(n)
    return np.sort(np.append(rng.choice(n - 1, k - 1, replace=False), n - 1))


def _oracle_inputs(w, l, raw):
    """(x, g) of layer l as the oracle sees them: float64 (ids int64), a convolution unfolded."""
    L = w.layers[l]
    x, g = (t.cpu() for t in raw)
    if L.kind == "conv":
        cin, k, stride, pad, _ = L.conv
        return oracle.unfold(x, k, k, stride, pad, L.d), oracle.tokens_from_nchw(g)
    if L.kind == "embed":
        return x.numpy(), g.double().numpy()
    return x.double().numpy(), g.double().numpy()


def _oracle_norm(L, x, g):
    if L.kind == "embed":
        return oracle.embed_norm_sq(x, g, L.d)
    if L.kind == "norm":
        return oracle.norm_affine_norm_sq(x, g, L.bias)
    # one number, two forms: the T x T Grams cost 2T^2(d+p) per sample, the
    # d x p per-sample gradient 2Tdp
    n = oracle.linear_norm_sq_gram(x, g) if L.T * (L.d + L.p) < L.d * L.p else oracle.linear_norm_sq(x, g)
    return n + oracle.bias_norm_sq(g) if L.bias else n


def _pow2_weights(B, seed):
    rng = np.random.default_rng(seed)
    C = 2.0 ** rng.integers(-3, 4, B)
    C[B // 2] = 0.0
    return C


@pytest.mark.parametrize("wid", [2, 3, 4, 5, 6, 7, 8])
def test_full_stack_parity(bk, wid):
    w = wl.get(wid)
    n, B = len(w.layers), w.B
    print(f"workload {wid}: {w.name}, {n} layers, B={B}", flush=True)
    st = Stack(bk, w)
    norms, C, tot = st.private_grad(0.0)
    rng = np.random.default_rng(wid)
    pos = {}                                   # sampled entries of each layer's G / Gb
    for l, L in enumerate(w.layers):
        if L.kind == "embed":
            pos[l] = None                      # rows chosen from the ids below
        elif L.kind == "norm":
            pos[l] = (None, _pick(rng, L.p, 64))
        else:
            pos[l] = (_pick(rng, L.d), _pick(rng, L.p))
    bias_cols = {l: _pick(rng, L.p, 64) for l, L in enumerate(w.layers) if L.bias}
    emb_rows = {}
    for l, L in enumerate(w.layers):
        if L.kind == "embed":
            ids = st.raw[l][0].cpu().numpy().ravel()
            counts = np.bincount(ids, minlength=L.d)
            emb_rows[l] = np.concatenate([np.argsort(-counts, kind="stable")[:4], np.flatnonzero(counts == 0)[:2],
                                          rng.choice(np.flatnonzero(counts), 2, replace=False), [L.d - 1]])
            pos[l] = (emb_rows[l], np.arange(L.p))

    got_G0 = {l: _take(st.Gs[l], *pos[l]) for l in range(n)}
    got_Gb0 = {l: _take(st.Gbs[l], None, c) for l, c in bias_cols.items()}
    # the noisy run: same factors, the noise is the difference
    _, C1, _ = st.private_grad(w.noise_std)
    assert np.array_equal(C, C1)
    noise = {l: _take(st.Gs[l], *pos[l]) - got_G0[l] for l in range(n)}
    noise_b = {l: _take(st.Gbs[l], None, c) - got_Gb0[l] for l, c in bias_cols.items()}
    # power-of-two weights through the same launch configuration
    C2 = _pow2_weights(B, wid)
    st.weighted_grads(C2)
    got_G2 = {l: _take(st.Gs[l], *pos[l]) for l in range(n)}
    got_Gb2 = {l: _take(st.Gbs[l], None, c) for l, c in bias_cols.items()}

    # per-layer oracle norms (and the small pieces the gradient checks need)
    gate_n = NORM_GATE[w.dtype]
    ref_norms = np.zeros((n, B))
    keep = {}
    worst = {"norm": 0.0}
    for l, L in enumerate(w.layers):
        if L.kind != "embed":
            assert bk.bk_use_ghost(L.T, L.d, L.p) == oracle.use_ghost(L.T, L.d, L.p), l
        x, g = _oracle_inputs(w, l, st.raw[l])
        ref_norms[l] = _oracle_norm(L, x, g)
        e = _rel(norms[l], ref_norms[l])
        worst["norm"] = max(worst["norm"], e)
        assert e <= gate_n and e <= NORM_GUARD, (l, L, e)
        if L.kind == "embed":
            keep[l] = (x, g)
        elif L.kind == "norm":
            keep[l] = oracle.norm_affine_sums(x, g)[0]
        else:
            rows, cols = pos[l]
            keep[l] = (x[:, :, rows], g[:, :, cols])
        if L.bias:
            keep[("b", l)] = oracle.bias_sums(g)
        del x, g
    print(f"  worst norm rel err {worst['norm']:.2e}", flush=True)

    # totals and clip factors from the oracle's norms
    ref_tot = oracle.aggregate(ref_norms)
    ref_C = oracle.clip_factors(ref_tot, w.clip, w.R, w.gamma)
    for got, ref in ((tot, ref_tot), (C, ref_C)):
        e = _rel(got, ref)
        assert e <= gate_n and e <= NORM_GUARD, e

    # clipped gradients with the oracle's C, and with power-of-two weights
    gate_g = GRAD_GATE[w.dtype]
    worst.update(grad=0.0, grad_rounded=0.0, grad_pow2=0.0, noise=0.0)
    for l, L in enumerate(w.layers):
        for weights, got, guard_of, tag in ((ref_C, got_G0, grad_guard, "grad"),
                                            (C2, got_G2, lambda *a: GRAD_GUARD_EXACT, "grad_pow2")):
            if L.kind == "embed":
                x, g = keep[l]
                ref = oracle.embed_weighted_grad(x, g, weights, L.d)[emb_rows[l]]
                counts = np.bincount(x.ravel(), minlength=L.d)[emb_rows[l]]
                assert np.all(got[l][counts == 0] == 0.0), l           # absent ids: zero rows
                e = _frob(got[l][counts > 0], ref[counts > 0])
                guard = GRAD_GUARD_EXACT
            elif L.kind == "norm":
                ref = oracle.weighted_sum(keep[l], weights)[pos[l][1]]
                e, guard = _frob(got[l], ref), GRAD_GUARD_EXACT
            else:
                a_s, g_s = keep[l]
                ref = oracle.weighted_grad(a_s, g_s, weights)
                if L.kind == "conv":
                    # zero padding columns of a give exactly zero gradient rows
                    assert np.all(got[l][pos[l][0] >= L.conv[0] * L.conv[1] ** 2] == 0.0), l
                e = _frob(got[l], ref)
                guard = guard_of(L.T, L.d, L.p, B, w.dtype)
            key = "grad_rounded" if tag == "grad" and guard > GRAD_GUARD_EXACT else tag
            worst[key] = max(worst[key], e)
            assert e <= gate_g and e <= guard, (tag, l, L, e, guard)
        if L.bias:
            for weights, got in ((ref_C, got_Gb0), (C2, got_Gb2)):
                ref = oracle.weighted_sum(keep[("b", l)], weights)[bias_cols[l]]
                e = _frob(got[l], ref)
                assert e <= gate_g and e <= GRAD_GUARD_EXACT, ("bias", l, e)

        # the noise of this layer at the same entries (tensor_id = l, step 0)
        rows, cols = pos[l]
        elems = cols.astype(np.int64) if rows is None else rows[:, None].astype(np.int64) * L.p + cols[None, :]
        ref_noise = w.noise_std * oracle.noise_at(elems, w.wid, l, 0)
        e = float(np.max(np.abs(noise[l] - ref_noise)))
        worst["noise"] = max(worst["noise"], e / w.noise_std)
        # |G + n| <~ 6 std: rounding G + n to fp32 costs ~2^-24 * 6 std
        assert e <= 2e-5 * w.noise_std * 8, l
        if L.bias:
            ref_b = w.noise_std * oracle.noise_at(bias_cols[l].astype(np.int64), w.wid, oracle.BIAS_TENSOR | l, 0)
            assert np.max(np.abs(noise_b[l] - ref_b)) <= 2e-5 * w.noise_std * 8, l
    print("  worst: " + ", ".join(f"{k} {v:.2e}" for k, v in worst.items()), flush=True)
    del st
    torch.cuda.empty_cache()


def test_config1_full(bk):
    """The single fp32 layer runs whole through the oracle."""
    w = wl.get(1)
    st = Stack(bk, w)
    a, g = (t.cpu() for t in st.raw[0])
    norms, C, tot = st.private_grad(0.0)
    G0 = st.Gs[0].cpu().numpy()
    st.private_grad(w.noise_std)
    G1 = st.Gs[0].cpu().numpy()
    ref = oracle.bk_stack(list(w.layers), [(a, g)], w.clip, w.R, w.gamma, w.noise_std, w.wid)
    assert _rel(norms, ref["norms"]) <= NORM_GATE["f32"]
    assert _rel(C, ref["C"]) <= NORM_GATE["f32"]
    assert _frob(G0, ref["G"][0]) <= GRAD_GATE["f32"]
    assert np.max(np.abs((G1 - G0) - (ref["Ghat"][0] - ref["G"][0]))) <= 2e-5 * 8


def test_gpt2_full_accumulate_doubles(bk):
    """GPT-2 small with every bias and LayerNorm affine (73 layers, B = 32,
    T = 128): a second, identical physical batch accumulated onto the first
    gives exactly twice the single-batch clipped gradients (each pass is
    deterministic and the accumulating epilogues add once)."""
    w = wl.get(8)
    n, B = len(w.layers), w.B
    st = Stack(bk, w)
    st.private_grad(0.0)
    G1 = [G.clone() for G in st.Gs]
    Gb1 = [None if G is None else G.clone() for G in st.Gbs]
    kinds = {"norm": bk.BK_NORM_AFFINE}
    Ps = [torch.empty(B, L.p, device=DEV) if L.kind == "norm" else None for L in w.layers]
    Pbs = [torch.empty(B, L.p, device=DEV) for L in w.layers]
    st.arr = bk.make_layers([{"kind": kinds.get(L.kind, bk.BK_LINEAR), "x": x, "g": g, "G": G, "P": P,
                              "bias": True, "Gb": Gb, "Pb": Pb, "accumulate": True}
                             for L, (x, g), G, P, Gb, Pb in zip(w.layers, st.ins, st.Gs, Ps, st.Gbs, Pbs)])
    st.private_grad(0.0)
    for l in range(n):
        assert torch.equal(st.Gs[l], 2 * G1[l]), l
        assert torch.equal(st.Gbs[l], 2 * Gb1[l]), l
    del st, G1, Gb1
    torch.cuda.empty_cache()


def test_long_stack_time_rule_mixopt(bk):
    """The long-sequence stack (36 layers, T = 1024, B = 16) with the decision
    by time and BK-MixOpt: every layer is instantiated on the LDS-DMA kernel
    and keeps its per-sample gradients, and each clipped gradient is their
    weighted sum.  Norms, totals and clip factors against the oracle's;
    sampled entries of every G against the oracle with the oracle's C."""
    w = wl.get(3)
    n, B = len(w.layers), w.B
    assert not any(bk.bk_use_ghost_time(L.T, L.d, L.p) for L in w.layers)
    st = Stack(bk, w, time_rule=True, mixopt=True)
    norms, C, tot = st.private_grad(0.0)
    rng = np.random.default_rng(33)
    pos = {l: (_pick(rng, L.d), _pick(rng, L.p)) for l, L in enumerate(w.layers)}
    got = {l: _take(st.Gs[l], *pos[l]) for l in range(n)}
    ref_norms = np.zeros((n, B))
    keep = {}
    for l, L in enumerate(w.layers):
        x, g = _oracle_inputs(w, l, st.raw[l])
        ref_norms[l] = _oracle_norm(L, x, g)
        assert _rel(norms[l], ref_norms[l]) <= NORM_GUARD, l
        keep[l] = (x[:, :, pos[l][0]], g[:, :, pos[l][1]])
        del x, g
    ref_tot = oracle.aggregate(ref_norms)
    ref_C = oracle.clip_factors(ref_tot, w.clip, w.R, w.gamma)
    assert _rel(tot, ref_tot) <= NORM_GUARD and _rel(C, ref_C) <= NORM_GUARD
    for l in range(n):
        ref = oracle.weighted_grad(*keep[l], ref_C)
        assert _frob(got[l], ref) <= GRAD_GUARD_EXACT, l
    del st
    torch.cuda.empty_cache()
