"""bk_private_grad_noalloc (the allocation-free entry point) against
bk_private_grad with a caller workspace, through the C ABI.

Two calls in a row share the library's scratch array: first the GPT-2-small
stack at full size (B = 32, T = 128, 48 layers; its K-split tail tiles fill the
whole 64 MiB), then a smaller LoRA stack (B = 8), which must not see anything
of the first call's contents.  Both entry points run the same kernels in the
same launch configuration, so their results must be bit-identical; they are
also held to the oracle-parity bounds of the other tests (relative 2e-2 gate and
the measured-error guards) against each other.
"""
import numpy as np
import pytest
import torch

import workloads as wl
from tolerances import GRAD_GATE, NORM_GATE

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def bk():
    assert torch.cuda.is_available()
    import paper_2210_00038_amd as m
    return m


def _stack(bk, w, B, nlayers):
    layers = w.layers[:nlayers]
    ins = [wl.draw_layer(w, l, B=B, device=DEV) for l in range(len(layers))]
    return layers, ins


def _run(bk, w, layers, ins, B, noalloc):
    n = len(layers)
    Gs = [torch.full((L.d, L.p), float("nan"), device=DEV) for L in layers]
    arr = bk.make_layers([{"kind": bk.BK_LINEAR, "x": x, "g": g, "G": G} for (x, g), G in zip(ins, Gs)])
    norm_sq = torch.full((n, B), float("nan"), device=DEV)
    C = torch.full((B,), float("nan"), device=DEV)
    tot = torch.full((B,), float("nan"), device=DEV)
    mode = bk.BK_CLIP_ABADI if w.clip == "abadi" else bk.BK_CLIP_AUTO
    args = (arr, n, bk.BK_BF16, B, mode, w.R, w.gamma, w.noise_std, w.wid, 3, norm_sq, C, tot)
    if noalloc:
        st = bk.lib.bk_private_grad_noalloc(*args[:10], norm_sq.data_ptr(), C.data_ptr(), tot.data_ptr(),
                                            torch.cuda.current_stream().cuda_stream)
        assert st == bk.BK_OK, bk.bk_last_error()
    else:
        bk.bk_private_grad(*args)
    torch.cuda.synchronize()
    return norm_sq, C, tot, Gs


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_call(bk, order):
    calls = [(wl.get(2), 32, 48), (wl.get(7), 8, 12)]
    for w, B, nl in calls:
        layers, ins = _stack(bk, w, B, nl)
        arr = bk.make_layers([{"kind": bk.BK_LINEAR, "x": x, "g": g} for x, g in ins])
        need = bk.bk_private_grad_workspace_size(arr, len(layers), bk.BK_BF16, B)
        assert need <= bk.BK_NOALLOC_SCRATCH_BYTES
        print(f"{w.name}: B={B}, {nl} layers, workspace {need} bytes", flush=True)
        ref = _run(bk, w, layers, ins, B, noalloc=False)
        got = _run(bk, w, layers, ins, B, noalloc=True)
        for r, g in zip(ref[:3], got[:3]):
            assert torch.isfinite(g).all()
            rel = ((g.double() - r.double()).abs() / r.double().abs()).max().item()
            assert rel <= NORM_GATE["bf16"] and rel <= 1e-6, rel
            assert torch.equal(g, r)
        for Gr, Gg in zip(ref[3], got[3]):
            assert torch.isfinite(Gg).all()
            err = (torch.linalg.norm(Gg.double() - Gr.double()) / torch.linalg.norm(Gr.double())).item()
            assert err <= GRAD_GATE["bf16"] and err <= 1e-6, err
            assert torch.equal(Gg, Gr)
        del ins, ref, got
    torch.cuda.empty_cache()
