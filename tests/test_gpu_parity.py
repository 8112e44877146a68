"""Parity of every libbk entry point with the float64 CPU oracle (MI355X).

Inputs are seeded and synthetic (workloads / numpy), drawn on the host and
copied to the device; the oracle sees the same values upcast exactly to
float64.  Tolerances: norms, totals and clip factors within 1e-5 relative for
fp32 inputs and 2e-2 for bf16 inputs; clipped gradients within 1e-4 (fp32) or
2e-2 (bf16) relative Frobenius error; path choice and Philox words exact.
Sizes span several tiles with ragged tails.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

NORM_TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
from tolerances import NORM_GUARD, GRAD_GUARD_EXACT  # noqa: E402
GRAD_TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}
DEV = "cuda"


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2210_00038_amd as m
    return m


def _pair(B, T, d, p, dtype, seed, g_scale=1.0):
    gen = torch.Generator().manual_seed(seed)
    a = torch.randn(B, T, d, generator=gen).to(dtype)
    g = (torch.randn(B, T, p, generator=gen) * g_scale).to(dtype)
    return a, g


def _rel(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return np.max(np.abs(x - ref) / np.maximum(np.abs(ref), 1e-300)) if ref.size else 0.0


def _frob(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    n = np.linalg.norm(ref)
    return np.linalg.norm(x - ref) / n if n > 0 else np.linalg.norm(x)


SHAPES = [
    # (B, T, d, p, dtype): one tile, several super blocks, ragged T / d / p, unaligned rows
    (4, 16, 64, 64, torch.float32),
    (3, 200, 96, 136, torch.bfloat16),
    (2, 300, 72, 40, torch.float32),
    (2, 257, 70, 33, torch.float32),          # rows not 16-byte multiples: scalar-load path
    (2, 129, 100, 60, torch.bfloat16),        # rows not 16-byte multiples: scalar-load path
    (5, 1, 48, 24, torch.bfloat16),
    (2, 128, 768, 256, torch.bfloat16),
    (2, 70, 520, 264, torch.bfloat16),        # ragged 256 x 128 tiles of the instantiated norm
]


@pytest.mark.parametrize("B,T,d,p,dtype", SHAPES)
def test_ghost_and_inst_norm_match_oracle(bk, B, T, d, p, dtype):
    a, g = _pair(B, T, d, p, dtype, seed=B * 1000 + T)
    ref = oracle.linear_norm_sq(a, g)
    ghost = bk.bk_ghost_norm(a.to(DEV), g.to(DEV)).cpu().numpy()
    inst = bk.bk_inst_norm(a.to(DEV), g.to(DEV)).cpu().numpy()
    print(f"ghost rel err {_rel(ghost, ref):.2e}, inst rel err {_rel(inst, ref):.2e}")
    assert _rel(ghost, ref) <= NORM_TOL[dtype]
    assert _rel(inst, ref) <= NORM_TOL[dtype]


@pytest.mark.parametrize("B,T,d,p", [
    (3, 129, 72, 40), (2, 160, 8, 200), (2, 192, 136, 64), (4, 197, 768, 96), (2, 224, 64, 8),
    (3, 255, 200, 128), (2, 256, 1280, 3840), (2, 197, 768, 2304), (2, 160, 512, 256), (3, 136, 256, 256)])
def test_whole_sample_ghost_norm(bk, B, T, d, p):
    """128 < T <= 256, bf16, 16-byte rows.  A grouped launch whose such layers
    give at least 512 workgroups takes the whole-sample kernel (every row
    streamed once, the full upper triangle of 32 x 32 Gram sub-tiles in one
    workgroup): here the layer repeated until the launch has that many, next
    to layers of other T; a smaller launch (the single-layer call) keeps the
    super-block pair kernel.  Both against the definition; a zero sample gives
    exactly 0; every copy of the layer gives the same bits."""
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B * 7 + T, g_scale=1e-2)
    a[B - 1].zero_()
    ref = oracle.linear_norm_sq(a, g)
    da, dg = a.to(DEV), g.to(DEV)
    out = bk.bk_ghost_norm(da, dg).cpu().numpy()
    assert out[B - 1] == 0.0
    assert _rel(out[:B - 1], ref[:B - 1]) <= 1e-4
    if not oracle.use_ghost(T, d, p):
        return                                   # the grouped call would instantiate
    k = -(-512 // B)
    a2, g2 = _pair(B, 200, 768, 256, torch.bfloat16, seed=T + 1)
    a3, g3 = _pair(B, 100, 256, 128, torch.bfloat16, seed=T + 2)
    ins = [(a2.to(DEV), g2.to(DEV))] + [(da, dg)] * k + [(a3.to(DEV), g3.to(DEV))]
    arr = bk.make_layers([{"kind": bk.BK_LINEAR, "x": x, "g": y} for x, y in ins])
    norm_sq = torch.empty(len(ins), B, device=DEV)
    bk.bk_layer_norms(arr, len(ins), bk.BK_BF16, B, norm_sq)
    got = norm_sq.cpu().numpy()
    for r in got[1:1 + k]:
        assert np.array_equal(r, got[1])
    assert got[1][B - 1] == 0.0 and _rel(got[1][:B - 1], ref[:B - 1]) <= 1e-4
    assert _rel(got[0], oracle.linear_norm_sq(a2, g2)) <= 1e-4
    assert _rel(got[-1], oracle.linear_norm_sq(a3, g3)) <= 1e-4


@pytest.mark.parametrize("B,T,d,p", [
    (2, 257, 72, 40), (2, 300, 256, 136), (3, 513, 64, 1280), (2, 1000, 768, 3072), (2, 1024, 3072, 768),
    (2, 1024, 8, 8)])
def test_long_ghost_norm(bk, B, T, d, p):
    """T > 256, bf16, 16-byte rows: 256-row super blocks (diagonal items and
    half-pair items, several per sample), against the definition; a zero
    sample gives exactly 0; grouped with a T <= 256 layer, bit-identical to
    the single-layer call when the layer takes the ghost path."""
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B * 11 + T, g_scale=1e-2)
    a[B - 1].zero_()
    ref = oracle.linear_norm_sq(a, g)
    da, dg = a.to(DEV), g.to(DEV)
    out = bk.bk_ghost_norm(da, dg).cpu().numpy()
    assert out[B - 1] == 0.0
    assert _rel(out[:B - 1], ref[:B - 1]) <= 1e-4
    a2, g2 = _pair(B, 200, 768, 256, torch.bfloat16, seed=T + 5)
    da2, dg2 = a2.to(DEV), g2.to(DEV)
    arr = bk.make_layers([{"kind": bk.BK_LINEAR, "x": x, "g": y} for x, y in ((da, dg), (da2, dg2))])
    norm_sq = torch.empty(2, B, device=DEV)
    bk.bk_layer_norms(arr, 2, bk.BK_BF16, B, norm_sq)
    got = norm_sq.cpu().numpy()
    if oracle.use_ghost(T, d, p):
        assert np.array_equal(got[0], out)
    assert got[0][B - 1] == 0.0 and _rel(got[0][:B - 1], ref[:B - 1]) <= 1e-4
    assert _rel(got[1], oracle.linear_norm_sq(a2, g2)) <= 1e-4


def test_ghost_norm_ties_and_zero(bk):
    a, g = _pair(3, 40, 32, 16, torch.float32, seed=5)
    a[1].zero_()
    out = bk.bk_ghost_norm(a.to(DEV), g.to(DEV)).cpu().numpy()
    assert out[1] == 0.0
    ref = oracle.linear_norm_sq(a, g)
    assert _rel(out[[0, 2]], ref[[0, 2]]) <= 1e-5


def test_empty_batch_and_tokens(bk):
    a = torch.zeros(3, 0, 8, device=DEV)
    g = torch.zeros(3, 0, 4, device=DEV)
    assert bk.bk_ghost_norm(a, g).cpu().tolist() == [0.0, 0.0, 0.0]
    assert bk.bk_inst_norm(a, g).cpu().tolist() == [0.0, 0.0, 0.0]
    C = torch.ones(3, device=DEV)
    G = bk.bk_weighted_grad(a, g, C)
    assert G.shape == (8, 4) and torch.count_nonzero(G).item() == 0
    # bf16: no samples on the LDS-DMA kernel (its tiles run no stage), no tokens on the wide one
    for B, T in [(0, 128), (2, 0)]:
        a = torch.zeros(B, T, 768, dtype=torch.bfloat16, device=DEV)
        g = torch.zeros(B, T, 512, dtype=torch.bfloat16, device=DEV)
        G = torch.full((768, 512), float("nan"), device=DEV)
        bk.bk_weighted_grad(a, g, torch.ones(B, device=DEV), G=G)
        assert torch.count_nonzero(G).item() == 0, (B, T)
        assert bk.bk_ghost_norm(a, g).cpu().tolist() == [0.0] * B


@pytest.mark.parametrize("B,T,V,p,dtype", [
    (3, 50, 11, 24, torch.float32), (2, 300, 1000, 72, torch.bfloat16), (4, 64, 5, 40, torch.bfloat16)])
def test_embed_ghost_norm_matches_oracle(bk, B, T, V, p, dtype):
    gen = torch.Generator().manual_seed(V)
    ids = torch.randint(0, V, (B, T), generator=gen)
    g = torch.randn(B, T, p, generator=gen).to(dtype)
    ref = oracle.embed_norm_sq(ids, g, V)
    out = bk.bk_embed_ghost_norm(ids.to(DEV), g.to(DEV), V).cpu().numpy()
    print(f"embed norm rel err {_rel(out, ref):.2e}")
    assert _rel(out, ref) <= NORM_TOL[dtype]


def test_embed_norm_zipf_ids(bk):
    ids = torch.from_numpy(wl.zipf_ids(8 * 256, 50257, 1.1, 7)).view(8, 256)
    g = (torch.randn(8, 256, 128, generator=torch.Generator().manual_seed(3)) * 1e-2).to(torch.bfloat16)
    ref = oracle.embed_norm_sq(ids, g, 50257)
    out = bk.bk_embed_ghost_norm(ids.to(DEV), g.to(DEV), 50257).cpu().numpy()
    assert _rel(out, ref) <= 2e-2


def _embed_norm_ref(ids, g, V):
    """oracle.embed_norm_sq with the ids relabelled 0 .. (distinct - 1) (the
    norm does not depend on which row an id selects) and tokens outside
    [0, V) dropped (they select no row)."""
    ids = ids.numpy()
    valid = (ids >= 0) & (ids < V)
    gv = g.float().numpy() * valid[..., None]
    uniq, inv = np.unique(np.where(valid, ids, 0), return_inverse=True)
    return oracle.embed_norm_sq(inv.reshape(ids.shape), gv, len(uniq))


# Embedding norms run as a join on the token ids (sorted per sample, each
# id's rows of g summed once); p % 8 != 0 or T past the join's limit keep the
# masked Gram.
@pytest.mark.parametrize("B,T,V,p,dtype,kind", [
    (4, 1, 9, 16, torch.bfloat16, "uniform"),         # one token per sample
    (3, 40, 6, 24, torch.float32, "uniform"),         # fewer positions than segments
    (3, 129, 50, 64, torch.bfloat16, "zipf"),         # just past one 128-row super block
    (2, 256, 50257, 1280, torch.bfloat16, "zipf"),    # the GPT-2-large embedding's shape
    (2, 400, 300, 264, torch.bfloat16, "zipf"),       # 256-column chunks, the last one of 8 columns
    (2, 1000, 7, 72, torch.float32, "uniform"),       # few ids, long runs, a ragged column chunk
    (2, 4096, 50257, 64, torch.bfloat16, "zipf"),
    (1, 16384, 1000, 8, torch.bfloat16, "uniform"),   # the longest T of the join
    (3, 300, 5, 64, torch.bfloat16, "same"),          # one id per sample: one run over every segment
    (2, 520, 100000, 64, torch.bfloat16, "distinct"), # every run one token long
    (2, 700, 40, 64, torch.bfloat16, "bad"),          # ids outside [0, V) add nothing
    (2, 300, 40, 60, torch.bfloat16, "uniform"),      # p % 8 != 0: the masked Gram
    (1, 16385, 1000, 8, torch.bfloat16, "uniform"),   # past the join's T: the masked Gram
])
def test_embed_norm_join(bk, B, T, V, p, dtype, kind):
    gen = torch.Generator().manual_seed(T + p)
    if kind == "zipf":
        ids = torch.from_numpy(wl.zipf_ids(B * T, V, 1.1, T)).view(B, T)
    elif kind == "same":
        ids = torch.full((B, T), 3, dtype=torch.int64)
    elif kind == "distinct":
        ids = torch.stack([torch.randperm(V, generator=gen)[:T] for _ in range(B)])
    elif kind == "bad":
        ids = torch.randint(-5, V + 5, (B, T), generator=gen)
    else:
        ids = torch.randint(0, V, (B, T), generator=gen)
    g = (torch.randn(B, T, p, generator=gen) * 1e-2).to(dtype)
    ref = _embed_norm_ref(ids, g, V)
    out = bk.bk_embed_ghost_norm(ids.to(DEV), g.to(DEV), V)
    again = bk.bk_embed_ghost_norm(ids.to(DEV), g.to(DEV), V)
    assert torch.equal(out, again)                    # fixed summation order
    e = _rel(out.cpu().numpy(), ref)
    print(f"embed norm (T={T}, {kind}) rel err {e:.2e}")
    assert e <= NORM_TOL[dtype] and e <= NORM_GUARD


@pytest.mark.parametrize("mode,R,gamma", [(0, 1.0, 0.0), (0, 3.5, 0.0), (1, 1.0, 0.01), (1, 1.0, 0.0)])
def test_clip_factors_match_oracle(bk, mode, R, gamma):
    rng = np.random.default_rng(11)
    n = (np.abs(rng.standard_normal((7, 37))) * 3).astype(np.float32)
    n[:, 5] = 0.0                                     # a zero-gradient sample
    C, tot = bk.bk_clip_factors(torch.from_numpy(n).to(DEV), mode, R, gamma)
    ref_tot = oracle.aggregate(n)
    ref_C = oracle.clip_factors(ref_tot, "abadi" if mode == 0 else "auto", R, gamma)
    assert _rel(tot.cpu().numpy(), ref_tot) <= 1e-6
    got = C.cpu().numpy()
    assert np.all(np.abs(got - ref_C) <= 1e-6 * np.maximum(np.abs(ref_C), 1e-30))


WSHAPES = [
    (4, 16, 64, 64, torch.float32),
    (3, 50, 200, 136, torch.bfloat16),
    (2, 77, 70, 33, torch.float32),
    (5, 33, 256, 384, torch.bfloat16),
    (2, 129, 100, 60, torch.bfloat16),
    (3, 130, 1280, 384, torch.bfloat16),      # several 256 x 128 tiles, ragged k stages
    (2, 64, 520, 264, torch.bfloat16),        # ragged tiles in both output dimensions
]


@pytest.mark.parametrize("B,T,d,p,dtype", WSHAPES)
def test_weighted_grad_matches_oracle(bk, B, T, d, p, dtype):
    a, g = _pair(B, T, d, p, dtype, seed=77 + T)
    C = torch.rand(B, generator=torch.Generator().manual_seed(T)) + 0.1
    ref = oracle.weighted_grad(a, g, C)
    G = bk.bk_weighted_grad(a.to(DEV), g.to(DEV), C.to(DEV)).cpu().numpy()
    err = _frob(G, ref)
    print(f"weighted grad frob err {err:.2e}")
    assert err <= GRAD_TOL[dtype]
    # C == 1 is the standard (non-private) gradient a^T g
    G1 = bk.bk_weighted_grad(a.to(DEV), g.to(DEV), torch.ones(B, device=DEV)).cpu().numpy()
    assert _frob(G1, oracle.weighted_grad(a, g, np.ones(B))) <= GRAD_TOL[dtype]


# bf16 layers with T >= 64 (and at most 1/8 padding to 16-row steps) take the
# kernel that applies the clip weights to its accumulators (rescaled at each
# sample boundary, rows of zero-weight samples loaded as zeros, every sample
# padded to whole 32-row stages); these cases exercise its boundaries.
@pytest.mark.parametrize("B,T,d,p,C", [
    (1, 64, 256, 256, [0.7]),                          # a single stage
    (3, 128, 300, 520, [0.3, 2.0, 0.05]),              # ragged tiles, two stages per sample
    (5, 192, 264, 136, [0.0, 1.5, 0.0, 1e-3, 4.0]),    # zero weights first and inside, odd stage count
    (4, 64, 512, 256, [1e3, 1e-3, 0.0, 0.0]),          # weights six decades apart, zeros at the end
    (2, 64, 64, 64, [0.0, 0.0]),                       # every weight zero
    (3, 197, 264, 520, [0.3, 0.0, 2.0]),               # last stage of 5 rows: its second step skipped
    (4, 120, 256, 256, [1.0, 1e-3, 0.0, 7.0]),         # last stage of 24 rows: both steps, 8 zero rows
    (2, 100, 300, 392, [0.5, 0.0]),                    # last stage of 4 rows, ragged tiles
    (3, 70, 256, 256, [0.2, 3.0, 0.0]),                # padding over 1/8: weights on g (rounded)
])
def test_weighted_grad_sample_weights(bk, B, T, d, p, C):
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=5 + T + B)
    C = torch.tensor(C, dtype=torch.float32)
    ref = oracle.weighted_grad(a, g, C)
    G = bk.bk_weighted_grad(a.to(DEV), g.to(DEV), C.to(DEV)).cpu().numpy()
    assert np.all(np.isfinite(G))
    if not np.any(ref):
        assert not np.any(G)
    else:
        err = _frob(G, ref)
        print(f"weighted grad (sample weights) frob err {err:.2e}")
        from tolerances import grad_guard
        assert err <= GRAD_TOL[torch.bfloat16] and err <= grad_guard(T, d, p, B)


@pytest.mark.parametrize("B,T,V,p,dtype", [(3, 40, 17, 24, torch.float32), (16, 256, 50257, 64, torch.bfloat16)])
def test_embed_weighted_grad_matches_oracle(bk, B, T, V, p, dtype):
    ids = torch.from_numpy(wl.zipf_ids(B * T, V, 1.1, 99)).view(B, T)
    g = torch.randn(B, T, p, generator=torch.Generator().manual_seed(5)).to(dtype)
    C = torch.rand(B, generator=torch.Generator().manual_seed(6)) + 0.1
    ref = oracle.embed_weighted_grad(ids, g, C, V)
    G = bk.bk_embed_weighted_grad(ids.to(DEV), g.to(DEV), C.to(DEV), V).cpu().numpy()
    assert _frob(G, ref) <= GRAD_TOL[dtype]
    absent = np.setdiff1d(np.arange(V), ids.numpy().ravel())
    assert np.all(G[absent] == 0.0)


# Runs of equal ids are staged 256 tokens at a time and added 8 at a time:
# one id repeated over every token (a 1024-token run, four batches), short
# runs with a ragged column chunk, and a Zipf mix; a zero clip weight; the
# accumulating form adds exactly the written rows to G's old values.
@pytest.mark.parametrize("B,T,V,p,dtype,kind", [
    (4, 256, 300, 1000, torch.bfloat16, "one"),
    (3, 100, 50, 72, torch.float32, "few"),
    (2, 300, 2000, 256, torch.bfloat16, "zipf"),
    (1, 1, 10, 5, torch.float32, "one"),
])
def test_embed_weighted_grad_runs(bk, B, T, V, p, dtype, kind):
    gen = torch.Generator().manual_seed(B * T + p)
    if kind == "one":
        ids = torch.full((B, T), V // 3, dtype=torch.int64)
    elif kind == "few":
        ids = torch.randint(0, V, (B, T), generator=gen)
    else:
        ids = torch.from_numpy(wl.zipf_ids(B * T, V, 1.2, 7)).view(B, T)
    g = torch.randn(B, T, p, generator=gen).to(dtype)
    C = torch.rand(B, generator=gen) + 0.1
    C[0] = 0.0
    ref = oracle.embed_weighted_grad(ids, g, C, V)
    ids_d, g_d, C_d = ids.to(DEV), g.to(DEV), C.to(DEV)
    G = bk.bk_embed_weighted_grad(ids_d, g_d, C_d, V)
    assert _frob(G.cpu().numpy(), ref) <= GRAD_TOL[dtype]
    absent = np.setdiff1d(np.arange(V), ids.numpy().ravel())
    assert np.all(G.cpu().numpy()[absent] == 0.0)
    assert torch.equal(G, bk.bk_embed_weighted_grad(ids_d, g_d, C_d, V))
    G0 = torch.randn(V, p, generator=gen).to(DEV)
    Ga = G0.clone()
    arr = bk.make_layers([{"kind": bk.BK_EMBEDDING, "x": ids_d, "g": g_d, "G": Ga, "V": V, "accumulate": True}])
    bk.bk_weighted_grads(arr, 1, C_d, bk.BK_BF16 if dtype == torch.bfloat16 else bk.BK_F32, B)
    assert torch.equal(Ga, G0 + G)


@pytest.mark.parametrize("seed,tid,step,q0,nq", [
    (0, 0, 0, 0, 1000), (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0, 64),
    (0x0123456789ABCDEF, 3, 11, (1 << 32) - 5, 300), (5, 144, 0, 123456789012, 77)])
def test_philox_words_exact(bk, seed, tid, step, q0, nq):
    got = bk.bk_philox_raw(seed, tid, step, q0, nq).cpu().numpy().view(np.uint32)
    ref = oracle.philox_words(seed, tid, step, q0, nq)
    np.testing.assert_array_equal(got, ref)


def test_philox_known_answer_vectors(bk):
    """The device generator reproduces the known-answer vectors published with
    Philox4x32-10 (tests/golden/philox4x32_10_kat.json) through the library's
    counter layout: block q of (seed, tensor, step) is the counter (q lo, q hi,
    tensor, step) under the key (seed lo, seed hi)."""
    import json
    import os
    kat = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        c = [int(x, 16) for x in v["counter"]]
        k = [int(x, 16) for x in v["key"]]
        seed, q = k[0] | (k[1] << 32), c[0] | (c[1] << 32)
        got = bk.bk_philox_raw(seed, c[2], c[3], q, 1).cpu().numpy().view(np.uint32).reshape(-1)
        assert [int(w) for w in got] == [int(x, 16) for x in v["out"]], v


@pytest.mark.parametrize("n,std,seed,tid,step", [(1001, 1.0, 2, 0, 0), (4096, 0.8, 5, 7, 3), (3, 2.0, 1, 1, 1)])
def test_noise_matches_oracle(bk, n, std, seed, tid, step):
    G0 = torch.randn(n, generator=torch.Generator().manual_seed(n))
    G = bk.bk_add_noise(G0.clone().to(DEV), std, seed, tid, step).cpu().numpy()
    ref = oracle.add_noise(G0, std, seed, tid, step)
    assert np.max(np.abs(G - ref)) <= 2e-5 * std * 8
    # std = 0 leaves the tensor bit-identical
    Gz = bk.bk_add_noise(G0.clone().to(DEV), 0.0, seed, tid, step).cpu()
    assert torch.equal(Gz, G0)


def test_noise_statistics(bk):
    z = bk.bk_add_noise(torch.zeros(1 << 22, device=DEV), 1.0, 2024, 3, 0).double()
    m, v = z.mean().item(), z.var().item()
    n = z.numel()
    assert abs(m) < 5 / np.sqrt(n) and abs(v - 1) < 5 * np.sqrt(2 / n)


def _stack_inputs(layers, B, dtype, seed):
    ins = []
    gen = torch.Generator().manual_seed(seed)
    for L in layers:
        if L.kind == "embed":
            ids = torch.randint(0, L.d, (B, L.T), generator=gen)
            g = (torch.randn(B, L.T, L.p, generator=gen) * 1e-2).to(dtype)
            ins.append((ids, g))
        else:
            a = torch.randn(B, L.T, L.d, generator=gen).to(dtype)
            g = (torch.randn(B, L.T, L.p, generator=gen) * 1e-2).to(dtype)
            ins.append((a, g))
    return ins


def _run_stack(bk, layers, ins, B, dtype, mode, R, gamma, std, seed, mixopt=False):
    dev_ins = [(x.to(DEV), g.to(DEV)) for x, g in ins]
    Gs = [torch.empty(L.d, L.p, device=DEV) for L in layers]
    # BK-MixOpt: every linear layer carries the flag; those that instantiate get a store
    Ps = [torch.empty(B, L.d, L.p, device=DEV) if mixopt and L.kind != "embed" and not bk.bk_use_ghost(L.T, L.d, L.p)
          else None for L in layers]
    specs = [{"kind": bk.BK_EMBEDDING if L.kind == "embed" else bk.BK_LINEAR, "x": x, "g": g, "G": G,
              "V": L.d, "mixopt": mixopt, "P": P} for L, (x, g), G, P in zip(layers, dev_ins, Gs, Ps)]
    arr = bk.make_layers(specs)
    n = len(layers)
    norm_sq = torch.empty(n, B, device=DEV)
    C = torch.empty(B, device=DEV)
    tot = torch.empty(B, device=DEV)
    dt = bk.BK_BF16 if dtype == torch.bfloat16 else bk.BK_F32
    bk.bk_private_grad(arr, n, dt, B, mode, R, gamma, std, seed, 0, norm_sq, C, tot)
    torch.cuda.synchronize()
    return norm_sq.cpu().numpy(), C.cpu().numpy(), tot.cpu().numpy(), [G.cpu().numpy() for G in Gs]



@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_ghost_launch_reordered_by_size(bk, dtype):
    """Ghost layers at T <= 128 (one super-block pair per sample) share a
    launch whose layers the host orders by d + p, largest first; here the
    stack order (160, 224, 360, 152) differs from it.  Every layer's norms
    and clipped gradient must still be its own."""
    Lr = wl.Layer
    layers = [Lr("linear", 48, 64, 96), Lr("linear", 48, 96, 128),
              Lr("linear", 48, 160, 200), Lr("linear", 48, 80, 72)]
    B = 5
    ins = _stack_inputs(layers, B, dtype, seed=31)
    norms, C, tot, G = _run_stack(bk, layers, ins, B, dtype, 1, 1.0, 0.01, 0.0, seed=3)
    ref = oracle.bk_stack(layers, ins, "auto", 1.0, 0.01, 0.0, seed=3, with_noise=False)
    assert ref["paths"] == ["ghost"] * 4
    for l in range(len(layers)):
        assert _rel(norms[l], ref["norms"][l]) <= NORM_TOL[dtype], l
        assert _frob(G[l], ref["G"][l]) <= GRAD_TOL[dtype], l
    assert _rel(C, ref["C"]) <= NORM_TOL[dtype]

@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_private_grad_stack_matches_oracle(bk, dtype):
    """Whole path on a small mixed stack: ghost, instantiated and embedding layers."""
    Lr = wl.Layer
    layers = [Lr("linear", 40, 64, 96),       # ghost (3200 < 6144)
              Lr("linear", 150, 96, 130),     # instantiate (45000 > 12480)
              Lr("linear", 150, 200, 260),    # ghost (45000 < 52000)
              Lr("embed", 40, 500, 64)]
    B = 6
    ins = _stack_inputs(layers, B, dtype, seed=42)
    for mode, R, gamma, std in [(0, 1e-2, 0.0, 0.0), (1, 1.0, 0.01, 0.0), (0, 1e-2, 0.0, 0.7)]:
        norms, C, tot, G = _run_stack(bk, layers, ins, B, dtype, mode, R, gamma, std, seed=9)
        ref = oracle.bk_stack(layers, ins, "abadi" if mode == 0 else "auto", R, gamma, std, seed=9,
                              with_noise=std > 0)
        assert ref["paths"] == ["ghost", "inst", "ghost", "embed"]
        assert _rel(norms, ref["norms"]) <= NORM_TOL[dtype]
        assert _rel(tot, ref["total"]) <= NORM_TOL[dtype]
        assert _rel(C, ref["C"]) <= NORM_TOL[dtype]
        for l in range(len(layers)):
            want = ref["Ghat"][l] if std > 0 else ref["G"][l]
            if std > 0:
                # compare the clipped gradient and the noise separately
                noise_ref = ref["Ghat"][l] - ref["G"][l]
                got_noise = G[l] - ref["G"][l]
                assert np.max(np.abs(got_noise - noise_ref)) <= 1e-4 * std * 8 + 1e-3 * np.abs(ref["G"][l]).max()
            else:
                assert _frob(G[l], want) <= GRAD_TOL[dtype], l


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_time_rule_stack_matches_oracle(bk, dtype):
    """BK_LAYER_TIME_RULE: the layerwise decision by time (ghost iff T(p+d) <
    pd).  Two layers change path against the space rule (one by a tie); each
    layer's norms are bitwise those of the per-layer call of the path the rule
    picks, and the whole path with BK-MixOpt (a store on every layer the time
    rule instantiates) matches the oracle run with the same rule."""
    Lr = wl.Layer
    layers = [Lr("linear", 256, 384, 384),    # space ghost (131072 < 147456), time inst
              Lr("linear", 128, 256, 256),    # space ghost, time tie 65536 == 65536: inst
              Lr("linear", 32, 256, 520),     # ghost both ways
              Lr("linear", 200, 96, 136)]     # inst both ways
    B = 3
    ins = _stack_inputs(layers, B, dtype, seed=77)
    time_ghost = [bk.bk_use_ghost_time(L.T, L.d, L.p) for L in layers]
    assert time_ghost == [False, False, True, False]
    assert [bk.bk_use_ghost(L.T, L.d, L.p) for L in layers] == [True, True, True, False]
    dev_ins = [(x.to(DEV), g.to(DEV)) for x, g in ins]
    Gs = [torch.empty(L.d, L.p, device=DEV) for L in layers]
    Ps = [None if tg else torch.empty(B, L.d, L.p, device=DEV) for L, tg in zip(layers, time_ghost)]
    specs = [{"kind": bk.BK_LINEAR, "x": x, "g": g, "G": G, "P": P, "mixopt": True, "time_rule": True}
             for (x, g), G, P in zip(dev_ins, Gs, Ps)]
    arr = bk.make_layers(specs)
    n = len(layers)
    dt = bk.BK_BF16 if dtype == torch.bfloat16 else bk.BK_F32
    norm_sq = torch.empty(n, B, device=DEV)
    bk.bk_layer_norms(arr, n, dt, B, norm_sq)
    torch.cuda.synchronize()
    for l, ((x, g), tg) in enumerate(zip(dev_ins, time_ghost)):
        one = (bk.bk_ghost_norm if tg else bk.bk_inst_norm)(x, g)
        torch.cuda.synchronize()
        assert torch.equal(norm_sq[l], one), l
    C = torch.empty(B, device=DEV)
    tot = torch.empty(B, device=DEV)
    bk.bk_private_grad(arr, n, dt, B, bk.BK_CLIP_AUTO, 1.0, 0.01, 0.0, 5, 0, norm_sq, C, tot)
    torch.cuda.synchronize()
    ref = oracle.bk_stack(layers, ins, "auto", 1.0, 0.01, 0.0, seed=5, with_noise=False, mixopt=True,
                          rule=oracle.use_ghost_time)
    assert ref["paths"] == ["inst", "inst", "ghost", "inst"]
    guard = NORM_GUARD if dtype == torch.bfloat16 else NORM_TOL[dtype]
    assert _rel(norm_sq.cpu().numpy(), ref["norms"]) <= guard
    assert _rel(tot.cpu().numpy(), ref["total"]) <= guard
    assert _rel(C.cpu().numpy(), ref["C"]) <= guard
    for l in range(n):
        assert _frob(Gs[l].cpu().numpy(), ref["G"][l]) <= GRAD_TOL[dtype], l


def test_config1_single_layer(bk):
    """Single fp32 linear layer, B=4, T=16, d=p=64, Abadi R=1, sigma=1: the
    ghost path against brute-force per-sample gradients."""
    w = wl.get(1)
    a, g = wl.draw_linear(w, 0)
    ref = oracle.linear_norm_sq_bruteforce(a, g)
    out = bk.bk_ghost_norm(a.to(DEV), g.to(DEV)).cpu().numpy()
    assert _rel(out, ref) <= 1e-5
    assert bk.bk_use_ghost(16, 64, 64)
    norms, C, tot, G = _run_stack(bk, list(w.layers), [(a, g)], w.B, torch.float32, 0, 1.0, 0.0, 0.0, seed=1)
    refs = oracle.bk_stack(list(w.layers), [(a, g)], "abadi", 1.0, 0.0, 1.0, seed=1)
    assert _rel(C, refs["C"]) <= 1e-5
    assert _frob(G[0], refs["G"][0]) <= 1e-4


def test_determinism(bk):
    a, g = _pair(4, 200, 256, 384, torch.bfloat16, seed=3)
    a, g = a.to(DEV), g.to(DEV)
    C = torch.rand(4, device=DEV)
    n1, n2 = bk.bk_ghost_norm(a, g), bk.bk_ghost_norm(a, g)
    G1, G2 = bk.bk_weighted_grad(a, g, C), bk.bk_weighted_grad(a, g, C)
    assert torch.equal(n1, n2) and torch.equal(G1, G2)


def test_grouped_noise_equals_per_tensor_noise(bk):
    Gs = [torch.randn(n, generator=torch.Generator().manual_seed(n)).to(DEV) for n in (5, 4096, 1, 777)]
    ref = [bk.bk_add_noise(G.clone(), 0.6, 31, 10 + k, 2) for k, G in enumerate(Gs)]
    got = bk.bk_add_noise_grouped([G.clone() for G in Gs], 0.6, 31, tensor_ids=[10, 11, 12, 13], step=2)
    for r, o in zip(ref, got):
        assert torch.equal(r, o)


# ---------------------------------------------------------------- BK-MixOpt
@pytest.mark.parametrize("B,T,d,p,dtype", [
    (3, 20, 40, 24, torch.float32),           # 16-byte rows, one 128 x 128 tile
    (2, 77, 70, 33, torch.float32),           # rows not 16-byte multiples: scalar loads
    (2, 70, 520, 264, torch.bfloat16),        # ragged 256 x 128 tiles of the wide kernel
    (2, 129, 100, 60, torch.bfloat16),        # scalar-load bf16 path
])
def test_per_sample_grads_match_oracle(bk, B, T, d, p, dtype):
    a, g = _pair(B, T, d, p, dtype, seed=31 + T)
    ref_P = oracle.per_sample_grads(a, g)
    norm, P = bk.bk_per_sample_grads(a.to(DEV), g.to(DEV))
    P = P.cpu().numpy()
    for i in range(B):
        assert _frob(P[i], ref_P[i]) <= GRAD_TOL[dtype], i
    assert _rel(norm.cpu().numpy(), oracle.linear_norm_sq(a, g)) <= NORM_TOL[dtype]


@pytest.mark.parametrize("B,shape", [(5, (33, 7)), (16, (768, 768)), (1, (3,)), (7, (1000,))])
def test_weighted_sum_matches_oracle(bk, B, shape):
    gen = torch.Generator().manual_seed(B)
    P = torch.randn((B,) + shape, generator=gen)
    C = torch.rand(B, generator=gen) + 0.05
    ref = oracle.weighted_sum(P.reshape(B, -1).numpy(), C.numpy()).reshape(shape)
    G = bk.bk_weighted_sum(P.to(DEV), C.to(DEV)).cpu().numpy()
    assert _frob(G, ref) <= 1e-6
    # no samples: zeros
    Z = bk.bk_weighted_sum(torch.empty((0,) + shape, device=DEV), torch.empty(0, device=DEV))
    assert torch.count_nonzero(Z).item() == 0


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_private_grad_mixopt_matches_oracle(bk, dtype):
    """BK-MixOpt on a mixed stack: the instantiated layer forms G from its stored per-sample
    gradients; the result equals the oracle's MixOpt path and the base path."""
    Lr = wl.Layer
    layers = [Lr("linear", 40, 64, 96),       # ghost
              Lr("linear", 150, 96, 130),     # instantiate: keeps per-sample gradients
              Lr("linear", 64, 72, 48),       # instantiate (8192 > 3456)
              Lr("embed", 40, 500, 64)]
    B = 5
    ins = _stack_inputs(layers, B, dtype, seed=7)
    for mode, R, gamma in [(0, 1e-2, 0.0), (1, 1.0, 0.01)]:
        norms, C, tot, G = _run_stack(bk, layers, ins, B, dtype, mode, R, gamma, 0.0, seed=3, mixopt=True)
        _, _, _, G_base = _run_stack(bk, layers, ins, B, dtype, mode, R, gamma, 0.0, seed=3)
        ref = oracle.bk_stack(layers, ins, "abadi" if mode == 0 else "auto", R, gamma, 0.0, seed=3,
                              with_noise=False, mixopt=True)
        assert ref["paths"] == ["ghost", "inst", "inst", "embed"]
        assert _rel(norms, ref["norms"]) <= NORM_TOL[dtype]
        assert _rel(C, ref["C"]) <= NORM_TOL[dtype]
        for l in range(len(layers)):
            assert _frob(G[l], ref["G"][l]) <= GRAD_TOL[dtype], l
            assert _frob(G[l], G_base[l]) <= GRAD_TOL[dtype], l


# ------------------------------------------------ K-split (few tiles, long K)
# Layers with few output tiles and a long contraction (convolutions at image
# scale, skinny adapters) cut each tile's K range into slices whose partial
# tiles are added in order by a second kernel.
@pytest.mark.parametrize("B,T,d,p", [
    (32, 200, 296, 264),      # 2 x 2 tiles, ragged d and p; T = 6 stages + 8 rows (short last stage)
    (128, 256, 256, 256),     # exactly 128 (sample, tile) workgroups
    (127, 256, 256, 256),     # one fewer: the wide kernel
    (16, 1024, 768, 768)])    # the long-sequence stack's instantiated layer
def test_inst_norm_on_dma_kernel(bk, B, T, d, p):
    """bf16 instantiated norms of layers with at least 128 (sample, 256 x 256
    tile) pairs run on the LDS-DMA kernel: norms against the definition, the
    kept per-sample gradients (BK-MixOpt) against the oracle's, the grouped
    call bitwise equal to the single-layer one, and a zero sample exactly 0."""
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B + T + d, g_scale=1e-2)
    a[1].zero_()
    ref = oracle.linear_norm_sq(a, g)
    ad, gd = a.to(DEV), g.to(DEV)
    one = bk.bk_inst_norm(ad, gd)
    assert _rel(one.cpu().numpy(), ref) <= NORM_GUARD
    assert one[1].item() == 0.0
    specs = [{"kind": bk.BK_LINEAR, "x": ad, "g": gd, "G": torch.empty(d, p, device=DEV)}]
    arr = bk.make_layers(specs)
    assert not bk.bk_use_ghost(T, d, p)
    grouped = torch.empty(1, B, device=DEV)
    bk.bk_layer_norms(arr, 1, bk.BK_BF16, B, grouped)
    torch.cuda.synchronize()
    assert torch.equal(grouped[0], one)
    if B * d * p <= (1 << 27):
        norm, P = bk.bk_per_sample_grads(ad, gd)
        assert torch.equal(norm, one)
        ref_P = oracle.per_sample_grads(a, g)
        P = P.cpu().numpy()
        for i in range(B):
            assert _frob(P[i], ref_P[i]) <= GRAD_GUARD_EXACT, i
        assert not P[1].any()


@pytest.mark.parametrize("B,T,d,p", [
    (2, 2048, 152, 64),      # one 256 x 128 tile per sample, 8 slices
    (3, 1000, 96, 200),      # ragged T, one tile, 4 slices
    (1, 4096, 520, 136),     # several tiles, one sample
])
def test_inst_norm_k_split(bk, B, T, d, p):
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=T + d)
    ref = oracle.linear_norm_sq(a, g)
    assert _rel(bk.bk_inst_norm(a.to(DEV), g.to(DEV)).cpu().numpy(), ref) <= NORM_TOL[torch.bfloat16]
    norm, P = bk.bk_per_sample_grads(a.to(DEV), g.to(DEV))
    assert _rel(norm.cpu().numpy(), ref) <= NORM_TOL[torch.bfloat16]
    ref_P = oracle.per_sample_grads(a, g)
    P = P.cpu().numpy()
    for i in range(B):
        assert _frob(P[i], ref_P[i]) <= GRAD_TOL[torch.bfloat16], i


@pytest.mark.parametrize("B,T,d,p,zero", [
    (4, 1024, 152, 64, []),          # narrow kernel, one tile, K slices
    (8, 1000, 152, 64, []),          # the same, T not a multiple of 64
    (4, 1024, 264, 136, []),         # LDS-DMA kernel, two tiles, K slices
    (8, 1000, 264, 136, [5]),        # the same with padded samples (32 stages of 32 rows each)
    (64, 70, 264, 136, [0]),         # register-staged kernel (T >= 64, padding over 1/8)
    (6, 512, 264, 136, [0, 3]),      # zero weights at slice starts and inside
    (16, 256, 40, 24, [15]),         # tiny output, many slices
])
def test_weighted_grad_k_split(bk, B, T, d, p, zero):
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B + T)
    C = torch.rand(B, generator=torch.Generator().manual_seed(B)) + 0.1
    C[zero] = 0.0
    ref = oracle.weighted_grad(a, g, C)
    G = bk.bk_weighted_grad(a.to(DEV), g.to(DEV), C.to(DEV)).cpu().numpy()
    assert _frob(G, ref) <= GRAD_TOL[torch.bfloat16]


# A grouped launch of a 256 x 256 clipped-gradient kernel (one workgroup per
# CU: the LDS-DMA kernel, or the register-staged one when padding T to 16-row
# steps adds over 1/8) whose last round of tiles is under half full: those
# tiles run in K slices, dispatched after every whole tile, and are summed in
# slice order.
@pytest.mark.parametrize("shapes,B,T,zero", [
    ([(768, 4096)] * 6, 4, 512, [1]),         # 288 tiles: 32 split from the middle of a layer
    ([(512, 4096)] * 9, 4, 256, []),          # 288 tiles: one whole 32-tile layer split
    ([(768, 768)], 3, 256, [0]),              # 9 tiles, no whole round: all split
    ([(768, 4096)] * 6, 4, 500, [2]),         # 32 does not divide T: samples padded to 16 stages
    ([(768, 768)], 3, 1000, []),              # the same, all split
    ([(768, 768)], 3, 197, [1]),              # 7 stages per sample, the last with one step
    ([(768, 4096)] * 6, 16, 70, [3]),         # register-staged kernel (64-row stages)
    ([(768, 768)], 40, 70, []),               # the same, all split
    ([(768, 768)], 3, 200, []),               # too few stages per slice: not split
    ([(4096, 6400)], 2, 128, [1]),            # 400 tiles of 8 stages: a last round over half full, not split
    ([(4096, 6400)], 1, 64, []),              # tiles of 2 stages (the prologue loads one past the end)
])
def test_weighted_grads_tail_split(bk, shapes, B, T, zero):
    gen = torch.Generator().manual_seed(B * T + len(shapes))
    ins = [((torch.randn(B, T, d, generator=gen)).to(torch.bfloat16),
            (torch.randn(B, T, p, generator=gen) * 1e-2).to(torch.bfloat16)) for d, p in shapes]
    C = torch.rand(B, generator=gen) + 0.1
    C[zero] = 0.0
    dev = [(a.to(DEV), g.to(DEV)) for a, g in ins]
    Gs = [torch.empty(d, p, device=DEV) for d, p in shapes]
    specs = [{"kind": bk.BK_LINEAR, "x": a, "g": g, "G": G} for (a, g), G in zip(dev, Gs)]
    arr = bk.make_layers(specs)
    n = len(shapes)
    tiles = sum((d // 256) * (p // 256) for d, p in shapes)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ws = bk.bk_weighted_grads_workspace_size(arr, n, bk.BK_BF16, B)
    # the host's rule: the last round's r tiles in s = CUs / r slices (at most
    # 16) of at least 8 stages (B ceil(T / 32) on the LDS-DMA kernel, else
    # ceil(B T / 64)), when s >= 2
    from tolerances import dl_padding_ok
    r = tiles % cus
    nst = B * -(-T // 32) if dl_padding_ok(T) else -(-B * T // 64)
    split = r > 0 and 2 * r <= cus and min(cus // r, nst // 8, 16) >= 2
    assert (ws > 0) == split
    Cd = C.to(DEV)
    bk.bk_weighted_grads(arr, n, Cd, bk.BK_BF16, B)
    first = [G.clone() for G in Gs]
    for (a, g), G in zip(ins, first):
        assert _frob(G.cpu().numpy(), oracle.weighted_grad(a, g, C)) <= GRAD_TOL[torch.bfloat16]
    # bitwise reproducible, and an accumulating call adds exactly what a
    # writing call writes (the product by the weight is rounded before the add)
    bk.bk_weighted_grads(arr, n, Cd, bk.BK_BF16, B)
    assert all(torch.equal(G, F) for G, F in zip(Gs, first))
    G0 = [torch.randn(G.shape, generator=gen).to(DEV) for G in Gs]
    for G, g0 in zip(Gs, G0):
        G.copy_(g0)
    acc = bk.make_layers([dict(sp, accumulate=True) for sp in specs])
    bk.bk_weighted_grads(acc, n, Cd, bk.BK_BF16, B)
    assert all(torch.equal(G, g0 + F) for G, g0, F in zip(Gs, G0, first))


# ------------------------------------------- narrow layers (one side <= 64)
@pytest.mark.parametrize("B,T,d,p", [
    (3, 50, 768, 16),       # 256 x 32 tiles, rows along d
    (3, 50, 16, 768),       # operands swapped: rows along p
    (2, 130, 576, 64),      # 256 x 64 tiles (a convolution with 64 output channels)
    (2, 33, 64, 520),       # swapped, ragged last tile
    (4, 20, 8, 136),        # rank 8, T < one stage
    (2, 4096, 256, 24),     # long T: the instantiated norm splits K
    (8, 2048, 40, 1000),    # clipped gradient splits K (4 tiles x 16 slices), swapped
])
def test_narrow_layers_match_oracle(bk, B, T, d, p):
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B * T + d + p, g_scale=1e-2)
    C = torch.rand(B, generator=torch.Generator().manual_seed(T)) + 0.1
    C[0] = 0.0
    ad, gd = a.to(DEV), g.to(DEV)
    ref_n = oracle.linear_norm_sq(a, g)
    assert _rel(bk.bk_inst_norm(ad, gd).cpu().numpy(), ref_n) <= NORM_TOL[torch.bfloat16]
    G = bk.bk_weighted_grad(ad, gd, C.to(DEV)).cpu().numpy()
    assert _frob(G, oracle.weighted_grad(a, g, C)) <= GRAD_TOL[torch.bfloat16]
    if B * d * p <= 4 * 1024 * 1024:
        norm, P = bk.bk_per_sample_grads(ad, gd)
        P = P.cpu().numpy()
        ref_P = oracle.per_sample_grads(a, g)
        for i in range(B):
            assert _frob(P[i], ref_P[i]) <= GRAD_TOL[torch.bfloat16], i
        assert _rel(norm.cpu().numpy(), ref_n) <= NORM_TOL[torch.bfloat16]


# ------------------------------------------- LoRA / adapter sub-modules (App. E.2)
@pytest.mark.parametrize("module,d,r,T,B", [
    ("lora", 768, 16, 128, 4),      # the rank-16 LoRA of the GPT-2-small shapes: both instantiate
    ("lora", 96, 1, 24, 3),         # rank one
    ("lora", 200, 12, 40, 5),       # r and d not multiples of 8
    ("lora", 256, 1024, 16, 2),     # the paper's largest rank: both sub-modules ghost
    ("adapter", 768, 64, 100, 3),   # adapter p -> r -> p, ReLU, ragged T
    ("adapter", 130, 8, 33, 4),
])
def test_lora_adapter_stack_matches_oracle(bk, module, d, r, T, B):
    """Sub-modules of LoRA x(W + LR) / adapter relu(xD)U + x, decomposed by the
    oracle from drawn x, weights and output gradients, rounded to bf16, through
    the whole path (both sub-modules of two modules in one stack)."""
    gen = torch.Generator().manual_seed(d + r + T)
    layers, ins = [], []
    for _ in range(2):
        x = torch.randn(B, T, d, generator=gen, dtype=torch.float64)
        A1 = torch.randn(d, r, generator=gen, dtype=torch.float64) / np.sqrt(d)
        A2 = torch.randn(r, d, generator=gen, dtype=torch.float64) / np.sqrt(r)
        dv = torch.randn(B, T, d, generator=gen, dtype=torch.float64) * 1e-2
        subs = (oracle.lora_submodules(x, A1, A2, dv) if module == "lora"
                else oracle.adapter_submodules(x, A1, A2, dv, "relu"))
        for a, g in subs:
            ins.append((torch.from_numpy(a).to(torch.bfloat16), torch.from_numpy(g).to(torch.bfloat16)))
            layers.append(wl.Layer("linear", T, a.shape[2], g.shape[2]))
    norms, C, tot, G = _run_stack(bk, layers, ins, B, torch.bfloat16, bk.BK_CLIP_AUTO, 1.0, 0.01, 0.0, seed=5)
    ref = oracle.bk_stack(layers, ins, "auto", 1.0, 0.01, 0.0, seed=5, with_noise=False)
    want_path = "ghost" if 2 * T * T < d * r else "inst"
    assert ref["paths"] == [want_path] * 4
    assert _rel(norms, ref["norms"]) <= NORM_TOL[torch.bfloat16]
    assert _rel(C, ref["C"]) <= NORM_TOL[torch.bfloat16]
    for l in range(len(layers)):
        assert _frob(G[l], ref["G"][l]) <= GRAD_TOL[torch.bfloat16], l


# ------------------------------------------- convolution layers via unfold
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,C,H,W,k,stride,pad,ld", [
    (2, 3, 17, 13, 7, 2, 3, 152),     # conv1-like: d = 147 padded to 152
    (3, 8, 9, 9, 3, 1, 1, 0),         # d = 72, no padding
    (1, 5, 12, 10, 1, 2, 0, 8),       # 1 x 1 stride 2 (downsample), d = 5 -> 8
    (2, 4, 6, 7, 3, 2, 0, 40),        # no padding, odd output
    (1, 512, 7, 7, 3, 1, 1, 0),       # channel groups (the patch of 512 channels exceeds one workgroup)
    (1, 520, 9, 6, 3, 2, 1, 4688),    # fp32: two groups, the last one carries the zero columns
    (2, 2, 10, 10, 3, 1, 1, 27),      # ld not a multiple of 16 bytes: element-wise kernel
    (2, 16, 12, 12, 3, 1, 1, 0),      # 4-element input loads; 16-byte token loads (HW = 144)
    (2, 8, 14, 20, 3, 2, 0, 0),       # last input load clipped to the patch row (Wp - pad < W)
])
def test_unfold_and_tokens_bit_exact(bk, dtype, B, C, H, W, k, stride, pad, ld):
    gen = torch.Generator().manual_seed(C * H + k)
    x = torch.randn(B, C, H, W, generator=gen).to(dtype)
    a = bk.bk_unfold(x.to(DEV), k, k, stride, pad, ld).cpu()
    ref = oracle.unfold(x.float().numpy(), k, k, stride, pad, ld)       # exact copies of dtype values
    assert np.array_equal(a.float().numpy(), ref)
    y = torch.randn(B, C, H, W, generator=gen).to(dtype)
    t = bk.bk_tokens_from_nchw(y.to(DEV)).cpu()
    assert np.array_equal(t.float().numpy(), oracle.tokens_from_nchw(y.float().numpy()))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_grouped_conv_prep_bit_exact(bk, dtype):
    """bk_conv_prep over 27 layers (more than one grouped launch), with layers
    that only unfold or only transpose and shapes that take the element-wise
    kernels, against the oracle's unfold and token-major transpose."""
    gen = torch.Generator().manual_seed(11)
    B = 3
    shapes = [(3, 8, 17, 7, 2, 3), (8, 16, 9, 3, 1, 1), (16, 8, 9, 1, 2, 0), (5, 6, 10, 3, 1, 1),
              (24, 16, 7, 3, 2, 1), (64, 64, 5, 3, 1, 1), (2, 5, 6, 3, 1, 0)] * 4
    shapes = shapes[:27]
    specs, refs = [], []
    for l, (ci, co, h, k, s, pd) in enumerate(shapes):
        ho = bk.conv_out_size(h, k, s, pd)
        d = ci * k * k
        ld = d + (l % 3) if l % 7 == 6 else (d + 7) // 8 * 8       # some ld not a multiple of 16 bytes
        x = torch.randn(B, ci, h, h, generator=gen).to(dtype)
        dy = torch.randn(B, co, ho, ho, generator=gen).to(dtype)
        ux, uy = l % 5 != 3, l % 5 != 4                             # unfold only / transpose only
        a = torch.full((B, ho * ho, ld), float("nan"), dtype=dtype, device=DEV)
        g = torch.full((B, ho * ho, co), float("nan"), dtype=dtype, device=DEV)
        specs.append({"x": x.to(DEV) if ux else None, "dy": dy.to(DEV) if uy else None, "a": a, "g": g, "k": k,
                      "stride": s, "pad": pd, "ld": ld, "C": ci, "H": h, "W": h, "p": co})
        refs.append((oracle.unfold(x.float().numpy(), k, k, s, pd, ld) if ux else None,
                     oracle.tokens_from_nchw(dy.float().numpy()) if uy else None))
    arr = bk.make_convs(specs)
    bk.bk_conv_prep(arr, len(specs), bk.BK_BF16 if dtype == torch.bfloat16 else bk.BK_F32, B)
    torch.cuda.synchronize()
    for l, (sp, (ra, rg)) in enumerate(zip(specs, refs)):
        a, g = sp["a"].cpu().float().numpy(), sp["g"].cpu().float().numpy()
        if ra is not None:
            assert np.array_equal(a, ra), l
        else:
            assert np.all(np.isnan(a)), l                          # no input: output untouched
        if rg is not None:
            assert np.array_equal(g, rg), l
        else:
            assert np.all(np.isnan(g)), l


def test_conv_stack_matches_oracle(bk):
    """A small ResNet-shaped conv stack through unfold + token-major gradients +
    the BK path (norms by the layerwise rule, clipping, clipped gradients)."""
    B, dtype = 4, torch.bfloat16
    # (C_in, C_out, k, stride, pad, H_in): early layers instantiate, late ones ghost
    convs = [(3, 16, 7, 2, 3, 64), (16, 16, 3, 1, 1, 32), (16, 32, 3, 2, 1, 32), (32, 64, 3, 2, 1, 16),
             (64, 128, 1, 1, 0, 4)]
    gen = torch.Generator().manual_seed(3)
    specs, ref_in, Gs, layers = [], [], [], []
    for (ci, co, k, s, pd, h) in convs:
        x = torch.randn(B, ci, h, h, generator=gen).to(dtype)
        ho = bk.conv_out_size(h, k, s, pd)
        dy = (torch.randn(B, co, ho, ho, generator=gen) * 1e-2).to(dtype)
        d = ci * k * k
        ld = (d + 7) // 8 * 8
        a = bk.bk_unfold(x.to(DEV), k, k, s, pd, ld)
        g = bk.bk_tokens_from_nchw(dy.to(DEV))
        G = torch.empty(ld, co, device=DEV)
        specs.append({"kind": bk.BK_LINEAR, "x": a, "g": g, "G": G})
        Gs.append(G)
        ref_in.append((oracle.unfold(x.float().numpy(), k, k, s, pd, ld), oracle.tokens_from_nchw(dy.float().numpy())))
        layers.append(wl.Layer("linear", ho * ho, ld, co))
    arr = bk.make_layers(specs)
    n = len(specs)
    norm_sq, C, tot = torch.empty(n, B, device=DEV), torch.empty(B, device=DEV), torch.empty(B, device=DEV)
    bk.bk_private_grad(arr, n, bk.BK_BF16, B, bk.BK_CLIP_ABADI, 1e-2, 0.0, 0.0, 1, 0, norm_sq, C, tot)
    torch.cuda.synchronize()
    ref = oracle.bk_stack(layers, ref_in, "abadi", 1e-2, 0.0, 0.0, 1, with_noise=False)
    assert ref["paths"][:2] == ["inst", "inst"] and ref["paths"][-1] == "ghost"
    assert _rel(norm_sq.cpu().numpy(), ref["norms"]) <= NORM_TOL[dtype]
    assert _rel(C.cpu().numpy(), ref["C"]) <= NORM_TOL[dtype]
    for l, (ci, co, k, s, pd, h) in enumerate(convs):
        G = Gs[l].cpu().numpy()
        assert _frob(G, ref["G"][l]) <= GRAD_TOL[dtype], l
        assert not np.any(G[ci * k * k:]), l                 # padded columns of a give zero rows


# ------------------------------------------- limits
@pytest.mark.parametrize("B,T,V,p,kind", [
    (1, 8193, 1000, 96, "zipf"),          # one past the former single-workgroup limit
    (64, 512, 50257, 1280, "zipf"),       # the GPT-2-large embedding at B = 64 (32768 tokens)
    (16, 4096, 300, 64, "one"),           # one run over every token: 1024 chunks, one fix-up walk
    (8, 1024, 130, 72, "blocks64"),       # runs of 64 tokens aligned to the chunks
    (8, 1024, 126, 40, "blocks65"),       # runs of 65 tokens: every boundary crossed
    (3, 20000, 70000, 24, "zipf"),        # 3 radix passes (V > 2^16)
])
def test_embed_weighted_grad_many_tokens(bk, B, T, V, p, kind):
    """Beyond one workgroup's sort: a stable radix sort of the ids over
    several tiles, then chunked segmented sums with a fix-up of the runs that
    cross chunk boundaries; bit-identical on a second call; absent rows stay
    zero; accumulation adds exactly the written rows."""
    n = B * T
    if kind == "zipf":
        ids = torch.from_numpy(wl.zipf_ids(n, V, 1.1, 17)).view(B, T)
    elif kind == "one":
        ids = torch.full((B, T), V - 1, dtype=torch.int64)
    else:
        r = 64 if kind == "blocks64" else 65
        ids = (torch.arange(n, dtype=torch.int64) // r % V).view(B, T)
    g = (torch.randn(B, T, p, generator=torch.Generator().manual_seed(18)) * 1e-2).to(torch.bfloat16)
    C = torch.rand(B, generator=torch.Generator().manual_seed(19)) + 0.1
    ref = oracle.embed_weighted_grad(ids, g, C, V)
    ids_d, g_d, C_d = ids.to(DEV), g.to(DEV), C.to(DEV)
    G = bk.bk_embed_weighted_grad(ids_d, g_d, C_d, V)
    Gh = G.cpu().numpy()
    absent = np.setdiff1d(np.arange(V), ids.numpy().ravel())
    assert np.all(Gh[absent] == 0.0)
    e = _frob(Gh, ref)
    print(f"n={n} V={V} {kind}: frob {e:.2e}")
    assert e <= GRAD_TOL[torch.bfloat16] and e <= 1e-5
    assert torch.equal(G, bk.bk_embed_weighted_grad(ids_d, g_d, C_d, V))
    G0 = torch.randn(V, p, generator=torch.Generator().manual_seed(20)).to(DEV)
    Ga = G0.clone()
    arr = bk.make_layers([{"kind": bk.BK_EMBEDDING, "x": ids_d, "g": g_d, "G": Ga, "V": V, "accumulate": True}])
    bk.bk_weighted_grads(arr, 1, C_d, bk.BK_BF16, B)
    assert torch.equal(Ga, G0 + G)


def test_embed_out_of_range_ids_are_zero_rows(bk):
    """Ids outside [0, V) (negative, V, V + k, beyond 2^32) are all-zero
    one-hot rows: norm and gradient equal the oracle's on the same batch with
    those tokens' gradient rows zeroed (and any valid id in their place)."""
    B, T, V, p = 4, 300, 500, 64
    gen = torch.Generator().manual_seed(23)
    ids = torch.randint(0, V, (B, T), generator=gen)
    bad = torch.rand(B, T, generator=gen) < 0.1
    vals = torch.tensor([-5, V, V + 7, (1 << 32) + 3, -(1 << 40)], dtype=torch.int64)
    ids[bad] = vals[torch.randint(0, len(vals), (int(bad.sum()),), generator=gen)]
    ids[0, :2] = torch.tensor([(1 << 32) + 3, 3])        # aliases id 3 modulo 2^32
    g = torch.randn(B, T, p, generator=gen).to(torch.bfloat16)
    C = torch.rand(B, generator=gen) + 0.1
    g_ref = g.clone()
    g_ref[bad | (ids < 0) | (ids >= V)] = 0
    ids_ref = torch.where((ids >= 0) & (ids < V), ids, torch.zeros_like(ids))
    ref_n = oracle.embed_norm_sq(ids_ref, g_ref, V)
    ref_G = oracle.embed_weighted_grad(ids_ref, g_ref, C, V)
    ids_d, g_d = ids.to(DEV), g.to(DEV)
    n = bk.bk_embed_ghost_norm(ids_d, g_d, V).cpu().numpy()
    assert _rel(n, ref_n) <= 1e-4
    G = bk.bk_embed_weighted_grad(ids_d, g_d, C.to(DEV), V).cpu().numpy()
    assert _frob(G, ref_G) <= 1e-5


@pytest.mark.parametrize("B,T,d,p", [
    (137, 1024, 8192, 256),     # LDS-DMA kernel: a is 2.3 GB
    (141, 1000, 8192, 256),     # the same with padded samples
    (1900, 70, 8192, 256),      # padding over 1/8 and past 2^31 bytes: the wide kernel
    (137, 1024, 8192, 32),      # narrow kernel
])
def test_weighted_grad_beyond_2_31_bytes(bk, B, T, d, p):
    """Layers whose a (B T rows of d bf16) passes 2^31 bytes: the kernels
    address one K stage at a time, so the offsets never wrap.  A 32 x 32 block
    (and the last row and column) of G against the oracle; samples with
    weight 0 included."""
    assert B * T * d * 2 >= (1 << 31)
    gen = torch.Generator(device=DEV).manual_seed(T + p)
    a = torch.randn(B, T, d, generator=gen, device=DEV).to(torch.bfloat16)
    g = (torch.randn(B, T, p, generator=gen, device=DEV) * 1e-2).to(torch.bfloat16)
    C = torch.rand(B, generator=torch.Generator().manual_seed(B)) + 0.1
    C[::5] = 0.0
    G = bk.bk_weighted_grad(a, g, C.to(DEV))
    rng = np.random.default_rng(d + p)
    rows = np.sort(np.append(rng.choice(d - 1, 31, replace=False), d - 1))
    cols = np.sort(np.append(rng.choice(p - 1, min(31, p - 1), replace=False), p - 1))
    ri, ci = torch.as_tensor(rows, device=DEV), torch.as_tensor(cols, device=DEV)
    ref = oracle.weighted_grad(a[:, :, ri].cpu(), g[:, :, ci].cpu(), C)
    got = G[ri][:, ci].cpu().numpy()
    e = _frob(got, ref)
    print(f"B T = {B * T}, d = {d}, p = {p}: frob {e:.2e}")
    from tolerances import grad_guard
    assert e <= GRAD_TOL[torch.bfloat16] and e <= grad_guard(T, d, p, B)
    del a, g, G
    torch.cuda.empty_cache()


@pytest.mark.parametrize("B", [4096, 4097])
def test_weighted_grad_largest_weight_table(bk, B):
    """B = 4096 is the largest batch whose clip weights the LDS-DMA kernel
    keeps in LDS; one more sample takes the register-staged kernel."""
    T, d, p = 64, 256, 256
    a, g = _pair(B, T, d, p, torch.bfloat16, seed=B)
    C = torch.rand(B, generator=torch.Generator().manual_seed(B)) + 0.1
    C[::7] = 0.0
    ref = oracle.weighted_grad(a, g, C)
    G = bk.bk_weighted_grad(a.to(DEV), g.to(DEV), C.to(DEV)).cpu().numpy()
    assert _frob(G, ref) <= GRAD_TOL[torch.bfloat16]
