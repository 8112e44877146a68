"""GPU parity of the per-sample bias / normalization-affine terms and of
gradient accumulation, through the grouped C ABI, against the oracle.

Stacks mix the kernel variants that write clipped gradients (256 x 256 DMA and
register-staged tiles, the wide kernel for T < 64, narrow tiles with and
without operand swap, K-split tiles, BK-MixOpt weighted sums, the embedding
scatter) so that every accumulate epilogue is exercised."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


class _L:
    def __init__(self, kind, T, d, p, bias=False, mixopt=False):
        self.kind, self.T, self.d, self.p, self.bias, self.mixopt = kind, T, d, p, bias, mixopt


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available()
    import paper_2210_00038_amd as m
    return m


def _rel(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    return np.max(np.abs(x - ref) / np.maximum(np.abs(ref), 1e-300))


def _frob(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    n = np.linalg.norm(ref)
    return np.linalg.norm(x - ref) / n if n > 0 else np.linalg.norm(x)


def _noise_std(Gs):
    """A noise std of the order of the clipped gradients themselves, so that
    fp32 rounding of G + noise stays far below the comparison tolerance."""
    return float(0.5 * np.sqrt(np.mean([np.mean(np.square(G)) for G in Gs if G is not None])))


def _draw(layers, B, dtype, gen):
    ins = []
    for L in layers:
        if L.kind == "embed":
            x = torch.randint(0, L.d, (B, L.T), generator=gen)
        elif L.kind == "norm":
            x = torch.randn(B, L.T, L.p, generator=gen).to(dtype)
        else:
            x = torch.randn(B, L.T, L.d, generator=gen).to(dtype)
        g = (torch.randn(B, L.T, L.p, generator=gen) * 1e-2).to(dtype)
        ins.append((x, g))
    return ins


class _Bufs:
    """Caller-owned outputs and per-sample stores, kept across physical batches."""
    def __init__(self, bk, layers, B):
        self.G = [torch.full((L.p,) if L.kind == "norm" else (L.d, L.p), float("nan"), device=DEV) for L in layers]
        self.Gb = [torch.full((L.p,), float("nan"), device=DEV) if L.bias else None for L in layers]
        self.P = [torch.empty(B, L.p, device=DEV) if L.kind == "norm" else
                  (torch.empty(B, L.d, L.p, device=DEV) if L.mixopt and not bk.bk_use_ghost(L.T, L.d, L.p) else None)
                  for L in layers]
        self.Pb = [torch.empty(B, L.p, device=DEV) if L.bias else None for L in layers]


def _run(bk, layers, ins, bufs, B, dtype, mode, R, gamma, std, seed, accumulate):
    kinds = {"linear": bk.BK_LINEAR, "embed": bk.BK_EMBEDDING, "norm": bk.BK_NORM_AFFINE}
    dev_ins = [(x.to(DEV), g.to(DEV)) for x, g in ins]
    specs = [{"kind": kinds[L.kind], "x": x, "g": g, "G": bufs.G[l], "V": L.d, "mixopt": L.mixopt,
              "P": bufs.P[l], "bias": L.bias, "Gb": bufs.Gb[l], "Pb": bufs.Pb[l], "accumulate": accumulate}
             for l, (L, (x, g)) in enumerate(zip(layers, dev_ins))]
    arr = bk.make_layers(specs)
    n = len(layers)
    norm_sq, C = torch.empty(n, B, device=DEV), torch.empty(B, device=DEV)
    dt = bk.BK_BF16 if dtype == torch.bfloat16 else bk.BK_F32
    bk.bk_private_grad(arr, n, dt, B, mode, R, gamma, std, seed, 0, norm_sq, C, None)
    torch.cuda.synchronize()
    return norm_sq.cpu().numpy(), C.cpu().numpy()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_bias_and_affine_stack_matches_oracle(bk, dtype):
    layers = [_L("linear", 70, 96, 130, bias=True),       # instantiated, 130 not a multiple of 8
              _L("linear", 40, 256, 384, bias=True),      # ghost
              _L("norm", 70, 300, 300, bias=True),        # LayerNorm gamma + beta, two feature chunks
              _L("norm", 33, 64, 64),                     # gamma only (no beta)
              _L("linear", 96, 768, 16, bias=True),       # narrow tile (bf16)
              _L("embed", 40, 500, 64)]
    for L in layers:
        if L.kind == "norm":
            L.d = L.p
    B = 5
    ins = _draw(layers, B, dtype, torch.Generator().manual_seed(616))
    bufs = _Bufs(bk, layers, B)
    std = _noise_std(oracle.bk_stack(layers, ins, "abadi", 1e-2, 0.0, 0.0, seed=4, with_noise=False)["G"])
    norms, C = _run(bk, layers, ins, bufs, B, dtype, bk.BK_CLIP_ABADI, 1e-2, 0.0, std, 4, False)
    ref = oracle.bk_stack(layers, ins, "abadi", 1e-2, 0.0, std, seed=4)
    assert _rel(norms, ref["norms"]) <= TOL[dtype]
    assert _rel(C, ref["C"]) <= TOL[dtype]
    for l, L in enumerate(layers):
        G = bufs.G[l].cpu().numpy()
        noise_ref = ref["Ghat"][l] - ref["G"][l]
        assert _frob(G - noise_ref, ref["G"][l]) <= TOL[dtype], l
        if L.bias:
            Gb = bufs.Gb[l].cpu().numpy()
            nb = ref["Gbhat"][l] - ref["Gb"][l]
            # the bias noise comes from its own stream (tensor id BK_BIAS_TENSOR | l)
            np.testing.assert_allclose(nb, std * oracle.noise(L.p, 4, bk.BK_BIAS_TENSOR | l, 0), rtol=1e-12)
            assert _frob(Gb - nb, ref["Gb"][l]) <= TOL[dtype], l
            Pb = bufs.Pb[l].cpu().numpy()
            assert _frob(Pb, oracle.bias_sums(ins[l][1])) <= TOL[dtype], l
        if L.kind == "norm":
            assert _frob(bufs.P[l].cpu().numpy(), oracle.norm_affine_sums(*ins[l])[0]) <= TOL[dtype], l


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_accumulation_over_physical_batches(bk, dtype):
    """A logical batch of 3 physical batches: the first call writes G, the next
    two add to it (BK_LAYER_ACCUMULATE), the noise is drawn on the last call
    only.  Against the oracle's logical_batch (clip per physical batch)."""
    layers = [_L("linear", 48, 64, 96, bias=True),        # wide kernel (T < 64)
              _L("linear", 96, 256, 256),                 # 32 | T: DMA tiles
              _L("linear", 100, 128, 200),                # register-staged tiles
              _L("linear", 512, 256, 256),                # one tile, K split (bf16)
              _L("linear", 512, 256, 24, bias=True),      # narrow, K split (bf16)
              _L("linear", 64, 40, 512),                  # narrow, operands swapped (bf16)
              _L("linear", 160, 64, 64, mixopt=True),     # BK-MixOpt weighted sum
              _L("norm", 64, 96, 96, bias=True),          # affine gamma and beta
              _L("embed", 24, 300, 32)]
    for L in layers:
        if L.kind == "norm":
            L.d = L.p
    B, nb, seed = 4, 3, 21
    gen = torch.Generator().manual_seed(936)
    batches = [_draw(layers, B, dtype, gen) for _ in range(nb)]
    std = _noise_std(oracle.logical_batch(layers, batches, "auto", 1.0, 0.01, 0.0, seed)["G"])
    bufs = _Bufs(bk, layers, B)
    Cs = []
    for b in range(nb):
        _, C = _run(bk, layers, batches[b], bufs, B, dtype, bk.BK_CLIP_AUTO, 1.0, 0.01,
                    std if b == nb - 1 else 0.0, seed, b > 0)
        Cs.append(C)
    ref = oracle.logical_batch(layers, batches, "auto", 1.0, 0.01, std, seed)
    for b in range(nb):
        assert _rel(Cs[b], ref["C"][b]) <= TOL[dtype]
    for l, L in enumerate(layers):
        G = bufs.G[l].cpu().numpy()
        noise_ref = ref["Ghat"][l] - ref["G"][l]
        assert _frob(G - noise_ref, ref["G"][l]) <= TOL[dtype], (l, L.kind, L.T, L.d, L.p)
        if L.bias:
            Gb = bufs.Gb[l].cpu().numpy()
            assert _frob(Gb - (ref["Gbhat"][l] - ref["Gb"][l]), ref["Gb"][l]) <= TOL[dtype], l


@pytest.mark.parametrize("B,T", [(0, 16), (3, 0)])
def test_empty_batches_with_bias_affine_accumulate(bk, B, T):
    """No samples or no tokens: norms are zero, written gradients are zero,
    accumulated gradients keep their values, and nothing faults."""
    layers = [_L("linear", T, 64, 96, bias=True), _L("norm", T, 40, 40, bias=True), _L("linear", T, 256, 24)]
    layers[1].d = layers[1].p
    for acc in (False, True):
        bufs = _Bufs(bk, layers, max(B, 1))
        for G in bufs.G + [g for g in bufs.Gb if g is not None]:
            G.fill_(3.0)
        ins = [(torch.zeros(B, T, L.d, dtype=torch.bfloat16), torch.zeros(B, T, L.p, dtype=torch.bfloat16))
               for L in layers]
        norms, C = _run(bk, layers, ins, bufs, B, torch.bfloat16, bk.BK_CLIP_AUTO, 1.0, 0.01, 0.0, 1, acc)
        assert norms.size == 0 or np.all(norms == 0.0)
        want = 3.0 if acc else 0.0
        for G in bufs.G + [g for g in bufs.Gb if g is not None]:
            assert torch.all(G == want).item()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("T,d,p", [
    (1, 64, 200),        # one token; the second 128-column chunk is ragged (bf16)
    (128, 256, 200),     # a full 128-row block
    (33, 512, 72),       # fp32 chunks of 64 columns: a ragged second chunk
    (129, 256, 136),     # two row blocks: the bias sums run in their own pass
    (100, 1024, 1000),   # many chunks
])
def test_bias_sums_formed_in_the_ghost_pass(bk, dtype, T, d, p):
    """A ghost layer with 16-byte rows and T <= 128 forms its per-sample bias
    sums while g passes through LDS for the Gram; Pb, the norms (weight plus
    bias term) and the clipped gradients must match the oracle either way."""
    layers = [_L("linear", T, d, p, bias=True), _L("linear", T, 256, 256, bias=True)]
    assert all(bk.bk_use_ghost(L.T, L.d, L.p) for L in layers)
    B = 6
    ins = _draw(layers, B, dtype, torch.Generator().manual_seed(T * 7 + p))
    bufs = _Bufs(bk, layers, B)
    norms, C = _run(bk, layers, ins, bufs, B, dtype, bk.BK_CLIP_ABADI, 1e-3, 0.0, 0.0, 3, False)
    ref = oracle.bk_stack(layers, ins, "abadi", 1e-3, 0.0, 0.0, seed=3, with_noise=False)
    assert _rel(norms, ref["norms"]) <= TOL[dtype]
    assert _rel(C, ref["C"]) <= TOL[dtype]
    for l in range(len(layers)):
        assert _frob(bufs.Pb[l].cpu().numpy(), oracle.bias_sums(ins[l][1])) <= TOL[dtype], l
        assert _frob(bufs.Gb[l].cpu().numpy(), ref["Gb"][l]) <= TOL[dtype], l
        assert _frob(bufs.G[l].cpu().numpy(), ref["G"][l]) <= TOL[dtype], l


def test_mixopt_accumulate_on_dma_instantiation(bk):
    """BK-MixOpt with gradient accumulation on a layer whose instantiated norm
    runs on the LDS-DMA kernel (bf16, 32 samples x 4 tiles of 256 x 256): the
    per-sample gradients it keeps give each physical batch's clipped
    gradient, added over two physical batches; against the oracle's logical
    batch, with the kept gradients those of the last batch."""
    from tolerances import GRAD_GUARD_EXACT, NORM_GUARD
    layers = [_L("linear", 384, 512, 512, mixopt=True),   # 2T^2 >= pd: instantiated
              _L("linear", 64, 128, 128)]                  # ghost
    assert not bk.bk_use_ghost(384, 512, 512) and bk.bk_use_ghost(64, 128, 128)
    B, nb, seed = 32, 2, 5
    gen = torch.Generator().manual_seed(77)
    batches = [_draw(layers, B, torch.bfloat16, gen) for _ in range(nb)]
    bufs = _Bufs(bk, layers, B)
    Cs = []
    for b in range(nb):
        _, C = _run(bk, layers, batches[b], bufs, B, torch.bfloat16, bk.BK_CLIP_AUTO, 1.0, 0.01, 0.0, seed, b > 0)
        Cs.append(C)
    ref = oracle.logical_batch(layers, batches, "auto", 1.0, 0.01, 0.0, seed)
    for b in range(nb):
        assert _rel(Cs[b], ref["C"][b]) <= NORM_GUARD, b
    for l in range(len(layers)):
        assert _frob(bufs.G[l].cpu().numpy(), ref["G"][l]) <= GRAD_GUARD_EXACT, l
    P = bufs.P[0].cpu().numpy()
    ref_P = oracle.per_sample_grads(*batches[-1][0])
    for i in range(0, B, 7):
        assert _frob(P[i], ref_P[i]) <= GRAD_GUARD_EXACT, i
