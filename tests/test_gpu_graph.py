"""The whole path captured in a HIP graph (through torch's graph capture on the
library's stream argument) and replayed: the library makes no allocation,
memset or synchronization, so every replay must reproduce the eager call
bitwise.  Replays are interleaved with eager work and synchronizations, and
each one is checked."""
import pytest
import torch

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2210_00038_amd as m
    return m


def _stack(bk, gen):
    """A small mixed stack: ghost layers at T = 128 and 200, an instantiated
    layer, a layer with a bias, a LoRA-shaped factor, a LayerNorm affine and
    an embedding (the id join)."""
    B = 8
    specs = []

    def lin(T, d, p, bias=False):
        a = torch.randn(B, T, d, generator=gen).to(torch.bfloat16).to(DEV)
        g = (torch.randn(B, T, p, generator=gen) * 1e-2).to(torch.bfloat16).to(DEV)
        s = {"kind": bk.BK_LINEAR, "x": a, "g": g, "G": torch.zeros(d, p, device=DEV)}
        if bias:
            s.update(bias=True, Gb=torch.zeros(p, device=DEV), Pb=torch.zeros(B, p, device=DEV))
        specs.append(s)

    lin(128, 768, 768)
    lin(200, 512, 1024, bias=True)
    lin(64, 1024, 1024)          # 2T^2 < pd: ghost; at T = 64 small
    lin(256, 256, 128)           # 2T^2 >= pd: instantiated
    lin(128, 768, 16)            # LoRA-shaped (narrow kernel)
    x = torch.randn(B, 128, 256, generator=gen).to(torch.bfloat16).to(DEV)
    g = (torch.randn(B, 128, 256, generator=gen) * 1e-2).to(torch.bfloat16).to(DEV)
    specs.append({"kind": bk.BK_NORM_AFFINE, "x": x, "g": g, "G": torch.zeros(256, device=DEV),
                  "P": torch.zeros(B, 256, device=DEV), "bias": True, "Gb": torch.zeros(256, device=DEV),
                  "Pb": torch.zeros(B, 256, device=DEV)})
    ids = torch.randint(0, 1000, (B, 300), generator=gen).to(DEV)
    g = (torch.randn(B, 300, 64, generator=gen) * 1e-2).to(torch.bfloat16).to(DEV)
    specs.append({"kind": bk.BK_EMBEDDING, "x": ids, "g": g, "G": torch.zeros(1000, 64, device=DEV), "V": 1000})
    return B, specs


def _outputs(specs, norm, C, tot):
    out = [norm.clone(), C.clone(), tot.clone()]
    for s in specs:
        out.append(s["G"].clone())
        if s.get("Gb") is not None:
            out.append(s["Gb"].clone())
    return out


def test_private_grad_graph_replays_match_eager(bk):
    gen = torch.Generator().manual_seed(11)
    B, specs = _stack(bk, gen)
    arr = bk.make_layers(specs)
    n = len(specs)
    norm = torch.empty(n, B, device=DEV)
    C = torch.empty(B, device=DEV)
    tot = torch.empty(B, device=DEV)
    nws = bk.bk_private_grad_workspace_size(arr, n, bk.BK_BF16, B)
    ws = torch.empty(max(1, nws), dtype=torch.uint8, device=DEV)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())

    def call():
        bk.bk_private_grad(arr, n, bk.BK_BF16, B, bk.BK_CLIP_AUTO, 1.0, 0.01, 0.5, 1234, 7, norm, C,
                           total_sq=tot, ws=ws, stream=torch.cuda.current_stream())

    with torch.cuda.stream(s):
        call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    eager = _outputs(specs, norm, C, tot)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call()
    torch.cuda.synchronize()
    for rep in range(4):
        # eager work on the same buffers between the replays
        for t in [norm, C, tot] + [sp["G"] for sp in specs]:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _outputs(specs, norm, C, tot)
        for k, (a, b) in enumerate(zip(got, eager)):
            assert torch.equal(a, b), (rep, k)
