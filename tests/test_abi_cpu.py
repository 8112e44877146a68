"""The C ABI on the host (no GPU needed): the library loads, exports every
symbol include/bk.h declares, and rejects bad arguments with a status code
before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bk.h")

bk = pytest.importorskip("paper_2210_00038_amd", reason="libbk.so not built")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bk_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 19
    for n in names:
        assert hasattr(bk.lib, n), n
    assert set(names) == set(bk.EXPORTS)


def test_use_ghost_rule():
    # Section 3.2: ghost iff 2 T^2 < p d; ties instantiate
    assert bk.bk_use_ghost(16, 64, 64)
    assert not bk.bk_use_ghost(1024, 768, 768)
    assert bk.bk_use_ghost(1024, 768, 3072)
    assert not bk.bk_use_ghost(32, 32, 64)
    assert bk.bk_use_ghost(31, 32, 64)
    assert bk.lib.bk_use_ghost(-1, 2, 3) == -1
    # no overflow for huge sizes
    assert not bk.bk_use_ghost(1 << 40, 1 << 20, 1 << 20)
    assert bk.bk_use_ghost(1, 1 << 40, 1 << 40)


def test_use_ghost_time_rule():
    # Table "block complexity" time row: ghost iff T (p + d) < p d; ties instantiate
    oracle = pytest.importorskip("oracle")
    for T in (0, 1, 2, 3, 7, 64, 255, 256, 257, 1024):
        for d in (0, 1, 2, 4, 8, 384, 512, 768, 3072):
            for p in (0, 1, 4, 8, 512, 768, 3072):
                assert bk.bk_use_ghost_time(T, d, p) == oracle.use_ghost_time(T, d, p), (T, d, p)
    assert not bk.bk_use_ghost_time(1024, 768, 3072) and bk.bk_use_ghost(1024, 768, 3072)
    assert not bk.bk_use_ghost_time(2, 4, 4)              # tie instantiates
    assert bk.lib.bk_use_ghost_time(1, -2, 3) == -1
    # no overflow: T (p + d) near 2^127
    big = (1 << 63) - 1
    assert not bk.bk_use_ghost_time(big, big, big)
    assert bk.bk_use_ghost_time(1, big, big)
    assert not bk.bk_use_ghost_time(big, 1, big)


def test_time_rule_flag_switches_the_norm_path():
    """A layer ghost by space and instantiated by time: with BK_LAYER_TIME_RULE
    a BK-MixOpt layer needs its store P, and the workspace follows the plan."""
    arr = (bk.bk_layer * 1)()
    arr[0].kind, arr[0].T, arr[0].d, arr[0].p = bk.BK_LINEAR, 256, 384, 384   # 131072 < 147456; 196608 >= 147456
    arr[0].x = arr[0].g = arr[0].G = 0x10000
    arr[0].flags = bk.BK_LAYER_MIXOPT
    ws_space = bk.bk_layer_norms_workspace_size(arr, 1, bk.BK_BF16, 4)
    need = bk.bk_layer_norms_workspace_size(arr, 1, bk.BK_BF16, 4)
    assert bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, need - 1, None) == bk.BK_ERR_WORKSPACE
    arr[0].flags = bk.BK_LAYER_MIXOPT | bk.BK_LAYER_TIME_RULE
    st = bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    assert st == bk.BK_ERR_INVALID_VALUE and "needs P" in bk.bk_last_error()
    ws_time = bk.bk_layer_norms_workspace_size(arr, 1, bk.BK_BF16, 4)
    assert ws_time == bk.bk_workspace_size(bk.BK_OP_INST_NORM, bk.BK_BF16, 4, 256, 384, 384)
    assert ws_space == bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, bk.BK_BF16, 4, 256, 384, 384)
    arr[0].flags = 16                                            # unknown bit
    st = bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    assert st == bk.BK_ERR_INVALID_VALUE and "unknown flags" in bk.bk_last_error()


def test_workspace_sizes():
    ws = bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, bk.BK_BF16, 32, 128, 768, 768)
    assert ws == 256 and ws >= 32 * 4           # one partial per sample, padded to 256 B
    ws = bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, bk.BK_BF16, 16, 1024, 768, 3072)
    assert ws >= 16 * 36 * 4                    # 8 super blocks -> 36 pairs
    ws = bk.bk_workspace_size(bk.BK_OP_INST_NORM, bk.BK_BF16, 16, 1024, 768, 768)
    assert ws >= 16 * 36 * 4                    # 6 x 6 output tiles
    # 3 x 3 tiles of 256 x 256 fill under half of 256 CUs (the host-side CU
    # count when no device answers): each tile in 16 K slices of fp32 partials
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 1024, 768, 768) == \
        9 * 16 * 256 * 256 * 4
    # 11 x 11 tiles: the last round (121 tiles) is under half of 256 CUs
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 1024, 2816, 2816) == \
        121 * 2 * 256 * 256 * 4
    # 17 x 16 = 272 tiles: 16 left over, each in 16 slices
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 1024, 4352, 4096) == \
        16 * 16 * 256 * 256 * 4
    # 12 x 12 = 144 tiles, over half of 256: no split
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 1024, 3072, 3072) == 0
    # T = 1000: each sample padded to 32 stages of 32 rows, split the same way
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 1000, 768, 768) == \
        9 * 16 * 256 * 256 * 4
    # T = 70 (padding to 80 rows is over 1/8: the register-staged kernel, 64-row
    # stages over all B T rows): 18 stages, slices of at least 8 stages
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 70, 768, 768) == \
        9 * 2 * 256 * 256 * 4
    # T < 64 (the wide kernel, two workgroups per CU): no tail split
    assert bk.bk_workspace_size(bk.BK_OP_WEIGHTED_GRAD, bk.BK_BF16, 16, 48, 768, 768) == 0
    # two radix key buffers (8 B per token), 256-bin digit histograms per 1024-key tile, two
    # partial rows per 64-token chunk and one flag per chunk, each 256-byte aligned
    n, p = 16 * 256, 1280
    al = lambda x: (x + 255) // 256 * 256
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_WEIGHTED_GRAD, bk.BK_BF16, 16, 256, 50257, p) == \
        2 * al(n * 8) + al(256 * (n // 1024) * 4) + al(2 * (n // 64) * p * 4) + al((n // 64) * 4)
    # embedding norm: the larger of the masked Gram's super-block pairs (128-row blocks) and,
    # with p % 8 == 0, the id join's column chunks of g (256 columns when p >= 256, else 64),
    # whichever the alignment of g picks at the call
    al4 = lambda n: (n * 4 + 255) // 256 * 256
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 16, 128, 50257, 1280) == al4(16 * 5)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 16, 128, 50257, 60) == al4(16)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 16, 256, 50257, 1280) == al4(16 * 5)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 16, 256, 50257, 200) == al4(16 * 4)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_F32, 2, 1024, 1000, 72) == al4(2 * 36)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 2, 300, 40, 60) == al4(2 * 6)
    assert bk.bk_workspace_size(bk.BK_OP_EMBED_GHOST_NORM, bk.BK_BF16, 1, 16385, 1000, 8) == al4(129 * 65)
    assert bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, 7, 1, 1, 1, 1) == 0        # bad dtype
    assert bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, bk.BK_F32, -1, 1, 1, 1) == 0


FAKE = ctypes.c_void_p(0x10000)     # never dereferenced: every call below fails validation


def _st(fn, *args):
    return getattr(bk.lib, fn)(*args)


def test_validation_before_any_device_call():
    L = bk.lib
    # NULL inputs
    assert L.bk_ghost_norm(None, None, bk.BK_BF16, 2, 3, 4, 5, FAKE, FAKE, 1 << 20, None) == \
        bk.BK_ERR_INVALID_VALUE
    assert "NULL" in bk.bk_last_error()
    # negative sizes
    assert L.bk_ghost_norm(FAKE, FAKE, bk.BK_BF16, -2, 3, 4, 5, FAKE, FAKE, 1 << 20, None) == \
        bk.BK_ERR_INVALID_VALUE
    assert L.bk_inst_norm(FAKE, FAKE, bk.BK_BF16, 2, 3, -4, 5, FAKE, FAKE, 1 << 20, None) == \
        bk.BK_ERR_INVALID_VALUE
    # int64 overflow of B*T*d
    assert L.bk_weighted_grad(FAKE, FAKE, FAKE, bk.BK_BF16, 1 << 40, 1 << 20, 1 << 10, 4, FAKE, None, 0,
                              None) == bk.BK_ERR_INVALID_VALUE
    # beyond 32-bit indexing
    assert L.bk_weighted_grad(FAKE, FAKE, FAKE, bk.BK_BF16, 1 << 20, 1 << 12, 4, 4, FAKE, None, 0,
                              None) == bk.BK_ERR_NOT_SUPPORTED
    # unknown dtype
    assert L.bk_ghost_norm(FAKE, FAKE, 9, 2, 3, 4, 5, FAKE, FAKE, 1 << 20, None) == bk.BK_ERR_INVALID_VALUE
    # workspace too small
    need = bk.bk_workspace_size(bk.BK_OP_GHOST_NORM, bk.BK_BF16, 2, 300, 4, 5)
    assert L.bk_ghost_norm(FAKE, FAKE, bk.BK_BF16, 2, 300, 4, 5, FAKE, FAKE, need - 1, None) == \
        bk.BK_ERR_WORKSPACE
    assert L.bk_ghost_norm(FAKE, FAKE, bk.BK_BF16, 2, 300, 4, 5, FAKE, None, need, None) == \
        bk.BK_ERR_WORKSPACE
    # clip factors: Abadi needs R > 0, automatic gamma >= 0, known mode
    assert L.bk_clip_factors(FAKE, 3, 4, bk.BK_CLIP_ABADI, 0.0, 0.0, FAKE, None, None) == \
        bk.BK_ERR_INVALID_VALUE
    assert L.bk_clip_factors(FAKE, 3, 4, bk.BK_CLIP_AUTO, 1.0, -0.5, FAKE, None, None) == \
        bk.BK_ERR_INVALID_VALUE
    assert L.bk_clip_factors(FAKE, 3, 4, 5, 1.0, 0.0, FAKE, None, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_clip_factors(None, 3, 4, bk.BK_CLIP_AUTO, 1.0, 0.0, FAKE, None, None) == \
        bk.BK_ERR_INVALID_VALUE
    # noise: negative / non-finite std, NULL tensor
    assert L.bk_add_noise(FAKE, 10, -1.0, 0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_add_noise(FAKE, 10, float("nan"), 0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_add_noise(None, 10, 1.0, 0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_add_noise(FAKE, -1, 1.0, 0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_philox_raw(0, 0, 0, 0, 4, None, None) == bk.BK_ERR_INVALID_VALUE
    # embedding gradient token limit of this build (2^24 tokens per call)
    assert L.bk_embed_weighted_grad(FAKE, FAKE, FAKE, bk.BK_BF16, 4097, 4096, 16, 100, FAKE, FAKE, 1 << 40,
                                    None) == bk.BK_ERR_NOT_SUPPORTED


def test_empty_inputs_are_noops_without_device():
    L = bk.lib
    # B == 0: nothing to compute, nothing launched
    assert L.bk_ghost_norm(None, None, bk.BK_BF16, 0, 5, 4, 5, None, None, 0, None) == bk.BK_OK
    assert L.bk_inst_norm(None, None, bk.BK_F32, 0, 5, 4, 5, None, None, 0, None) == bk.BK_OK
    assert L.bk_clip_factors(None, 0, 0, bk.BK_CLIP_AUTO, 1.0, 0.0, None, None, None) == bk.BK_OK
    assert L.bk_add_noise(FAKE, 10, 0.0, 0, 0, 0, None) == bk.BK_OK       # std = 0 leaves G untouched
    assert L.bk_add_noise(None, 0, 1.0, 0, 0, 0, None) == bk.BK_OK
    assert L.bk_philox_raw(0, 0, 0, 0, 0, None, None) == bk.BK_OK


def test_grouped_validation():
    arr = (bk.bk_layer * 2)()
    for k in range(2):
        arr[k].kind, arr[k].T, arr[k].d, arr[k].p = bk.BK_LINEAR, 8, 16, 16
        arr[k].x = arr[k].g = arr[k].G = 0x10000
    arr[1].flags = 16                                       # not a known flag
    st = bk.lib.bk_layer_norms(arr, 2, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    assert st == bk.BK_ERR_INVALID_VALUE and "flags" in bk.bk_last_error()
    arr[1].flags = 0
    arr[1].kind = 5
    assert bk.lib.bk_layer_norms(arr, 2, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None) == bk.BK_ERR_INVALID_VALUE
    arr[1].kind = bk.BK_LINEAR
    arr[1].G = None
    assert bk.lib.bk_weighted_grads(arr, 2, FAKE, bk.BK_BF16, 4, None, 0, None) == bk.BK_ERR_INVALID_VALUE
    need = bk.bk_layer_norms_workspace_size(arr, 2, bk.BK_BF16, 4)
    assert need > 0
    assert bk.lib.bk_layer_norms(arr, 2, bk.BK_BF16, 4, FAKE, FAKE, need - 1, None) == bk.BK_ERR_WORKSPACE
    assert bk.lib.bk_private_grad(arr, 2, bk.BK_BF16, 4, bk.BK_CLIP_ABADI, 0.0, 0.0, 1.0, 0, 0, FAKE,
                                  FAKE, None, FAKE, 1 << 20, None) == bk.BK_ERR_INVALID_VALUE


def test_status_strings():
    assert bk.bk_status_string(bk.BK_OK) == "BK_OK"
    assert bk.bk_status_string(bk.BK_ERR_WORKSPACE) == "BK_ERR_WORKSPACE"
    assert "gfx950" in bk.bk_version()


def test_mixopt_validation():
    """BK-MixOpt store: needed (and checked) only on a linear layer that instantiates."""
    arr = (bk.bk_layer * 1)()
    arr[0].kind, arr[0].T, arr[0].d, arr[0].p = bk.BK_LINEAR, 64, 16, 16     # 2T^2 >= pd: instantiates
    arr[0].x = arr[0].g = arr[0].G = 0x10000
    arr[0].flags = bk.BK_LAYER_MIXOPT
    st = bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    assert st == bk.BK_ERR_INVALID_VALUE and "needs P" in bk.bk_last_error()
    assert bk.lib.bk_weighted_grads(arr, 1, FAKE, bk.BK_BF16, 4, FAKE, 1 << 20, None) == bk.BK_ERR_INVALID_VALUE
    arr[0].P = 0x10002                                       # misaligned
    st = bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    assert st == bk.BK_ERR_INVALID_VALUE and "aligned" in bk.bk_last_error()
    # a ghost-norm layer ignores the flag: no store needed, validation reaches the workspace check
    arr[0].T, arr[0].d, arr[0].p, arr[0].P = 8, 64, 64, None
    need = bk.bk_layer_norms_workspace_size(arr, 1, bk.BK_BF16, 4)
    assert need > 0
    assert bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, need - 1, None) == bk.BK_ERR_WORKSPACE
    # single-layer calls
    L = bk.lib
    assert L.bk_per_sample_grads(FAKE, FAKE, bk.BK_BF16, 2, 8, 4, 4, FAKE, None, FAKE, 1 << 20, None) == \
        bk.BK_ERR_INVALID_VALUE
    assert L.bk_per_sample_grads(None, None, bk.BK_BF16, 0, 8, 4, 4, None, None, None, 0, None) == bk.BK_OK
    assert L.bk_weighted_sum(FAKE, FAKE, 3, -1, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_weighted_sum(None, FAKE, 3, 10, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_weighted_sum(FAKE, FAKE, 3, 10, None, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_weighted_sum(0x10002, FAKE, 3, 10, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_weighted_sum(None, None, 3, 0, None, None) == bk.BK_OK             # nothing to do


def test_conv_prep_validation():
    L = bk.lib
    # kernel larger than the padded image, bad stride / pad, ld < C kh kw
    assert L.bk_unfold(FAKE, bk.BK_BF16, 1, 3, 4, 4, 7, 7, 1, 0, 147, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_unfold(FAKE, bk.BK_BF16, 1, 3, 8, 8, 3, 3, 0, 1, 27, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_unfold(FAKE, bk.BK_BF16, 1, 3, 8, 8, 3, 3, 1, -1, 27, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_unfold(FAKE, bk.BK_BF16, 1, 3, 8, 8, 3, 3, 1, 1, 26, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_unfold(None, bk.BK_BF16, 1, 3, 8, 8, 3, 3, 1, 1, 32, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_unfold(None, bk.BK_BF16, 0, 3, 8, 8, 3, 3, 1, 1, 32, None, None) == bk.BK_OK        # empty
    assert L.bk_unfold(FAKE, 9, 1, 3, 8, 8, 3, 3, 1, 1, 32, FAKE, None) == bk.BK_ERR_INVALID_VALUE  # dtype
    assert L.bk_tokens_from_nchw(FAKE, bk.BK_F32, -1, 3, 4, 4, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_tokens_from_nchw(None, bk.BK_F32, 2, 3, 4, 4, FAKE, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_tokens_from_nchw(None, bk.BK_F32, 2, 0, 4, 4, None, None) == bk.BK_OK
    assert bk.conv_out_size(224, 7, 2, 3) == 112 and bk.conv_out_size(56, 1, 2, 0) == 28


def test_grouped_conv_prep_validation():
    L = bk.lib
    mk = lambda **kw: (bk.bk_conv * 1)(bk.bk_conv(**{**dict(x=FAKE, dy=FAKE, a=FAKE, g=FAKE, C=3, H=8, W=8, kh=3,
                                                           kw=3, stride=1, pad=1, ld=32, p=4), **kw}))
    assert L.bk_conv_prep(None, 0, bk.BK_BF16, 2, None) == bk.BK_OK                    # no layers
    assert L.bk_conv_prep(None, 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_conv_prep(mk(), -1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_conv_prep(mk(), 1, 7, 2, None) == bk.BK_ERR_INVALID_VALUE              # dtype
    assert L.bk_conv_prep(mk(ld=26), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE  # ld < C kh kw
    assert L.bk_conv_prep(mk(stride=0), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_conv_prep(mk(kh=11), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE  # kernel > padded image
    assert L.bk_conv_prep(mk(a=None), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE  # x without a
    assert L.bk_conv_prep(mk(g=None), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE  # dy without g
    assert L.bk_conv_prep(mk(p=-1), 1, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE
    assert L.bk_conv_prep(mk(), 1, bk.BK_BF16, 70000, None) == bk.BK_ERR_NOT_SUPPORTED
    # nothing to do: no inputs, or an empty batch
    assert L.bk_conv_prep(mk(x=None, dy=None, a=None, g=None), 1, bk.BK_BF16, 2, None) == bk.BK_OK
    assert L.bk_conv_prep(mk(), 1, bk.BK_BF16, 0, None) == bk.BK_OK
    # a bad layer after a good one rejects the whole call (checked before any work)
    two = (bk.bk_conv * 2)(mk()[0], mk(ld=1)[0])
    assert L.bk_conv_prep(two, 2, bk.BK_BF16, 2, None) == bk.BK_ERR_INVALID_VALUE
    assert b"layer 1" in L.bk_last_error()


def test_bias_affine_accumulate_validation():
    """BK_LAYER_BIAS needs Pb (and Gb for gradients), an affine layer needs
    d == p and P, an embedding takes no bias; BK_LAYER_ACCUMULATE needs nothing."""
    def one(**kw):
        arr = (bk.bk_layer * 1)()
        arr[0].kind, arr[0].T, arr[0].d, arr[0].p = kw.get("kind", bk.BK_LINEAR), 8, kw.get("d", 16), 16
        arr[0].x = arr[0].g = arr[0].G = 0x10000
        arr[0].flags = kw.get("flags", 0)
        for f in ("P", "Gb", "Pb"):
            setattr(arr[0], f, kw.get(f))
        return arr
    norms = lambda a: bk.lib.bk_layer_norms(a, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
    grads = lambda a: bk.lib.bk_weighted_grads(a, 1, FAKE, bk.BK_BF16, 4, FAKE, 1 << 20, None)
    assert norms(one(flags=bk.BK_LAYER_BIAS)) == bk.BK_ERR_INVALID_VALUE and "Pb" in bk.bk_last_error()
    assert grads(one(flags=bk.BK_LAYER_BIAS, Pb=0x10000)) == bk.BK_ERR_INVALID_VALUE and "Gb" in bk.bk_last_error()
    assert norms(one(flags=bk.BK_LAYER_BIAS, Pb=0x10001)) == bk.BK_ERR_INVALID_VALUE       # misaligned
    assert norms(one(kind=bk.BK_EMBEDDING, flags=bk.BK_LAYER_BIAS, Pb=0x10000, Gb=0x10000)) == \
        bk.BK_ERR_INVALID_VALUE and "no bias" in bk.bk_last_error()
    assert norms(one(kind=bk.BK_NORM_AFFINE, d=12, P=0x10000)) == bk.BK_ERR_INVALID_VALUE and \
        "d == p" in bk.bk_last_error()
    assert norms(one(kind=bk.BK_NORM_AFFINE)) == bk.BK_ERR_INVALID_VALUE and "P [B,p]" in bk.bk_last_error()
    assert norms(one(kind=7)) == bk.BK_ERR_INVALID_VALUE
    # workspace grows by one partial per sample and 256-feature chunk for the bias sums
    plain = bk.bk_layer_norms_workspace_size(one(), 1, bk.BK_BF16, 4)
    biased = bk.bk_layer_norms_workspace_size(one(flags=bk.BK_LAYER_BIAS, Pb=0x10000), 1, bk.BK_BF16, 4)
    assert biased >= plain + 4 * 4 - 256
    assert bk.bk_layer_norms_workspace_size(one(kind=bk.BK_NORM_AFFINE, P=0x10000), 1, bk.BK_BF16, 4) >= 16
    # no samples: nothing to check beyond the flags, nothing launched
    assert bk.lib.bk_layer_norms(one(flags=bk.BK_LAYER_BIAS | bk.BK_LAYER_ACCUMULATE), 1, bk.BK_BF16, 0,
                                 None, None, 0, None) == bk.BK_OK


def test_grouped_noise_validation():
    """The grouped noise entry point checks its arrays and std before any
    launch; n = 0 and std = 0 launch nothing."""
    ptrs = (ctypes.c_void_p * 2)(0x10000, None)
    nel = (ctypes.c_int64 * 2)(4, 4)
    tids = (ctypes.c_uint32 * 2)(0, 1)
    for fn in (bk.lib.bk_add_noise_grouped,):
        assert fn(None, nel, tids, 2, 1.0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
        assert fn(ptrs, nel, tids, -1, 1.0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
        assert fn(ptrs, nel, tids, 2, float("nan"), 0, 0, None) == bk.BK_ERR_INVALID_VALUE
        assert fn(ptrs, nel, tids, 2, -0.5, 0, 0, None) == bk.BK_ERR_INVALID_VALUE
        assert fn(ptrs, nel, tids, 2, 1.0, 0, 0, None) == bk.BK_ERR_INVALID_VALUE   # tensor 1 NULL
        assert "NULL" in bk.bk_last_error()
        assert fn(ptrs, nel, tids, 0, 1.0, 0, 0, None) == bk.BK_OK
    assert bk.lib.bk_add_noise_grouped(ptrs, nel, tids, 1, 0.0, 0, 0, None) == bk.BK_OK


def test_embedding_token_limit():
    """An embedding layer's clipped gradient takes at most 2^24 tokens per
    call: one more is refused before any launch."""
    arr = (bk.bk_layer * 1)()
    arr[0].kind, arr[0].T, arr[0].d, arr[0].p = bk.BK_EMBEDDING, (1 << 24) + 1, 100, 16
    arr[0].x = arr[0].g = arr[0].G = 0x10000
    st = bk.lib.bk_weighted_grads(arr, 1, FAKE, bk.BK_BF16, 1, FAKE, 1 << 40, None)
    assert st == bk.BK_ERR_NOT_SUPPORTED and str(1 << 24) in bk.bk_last_error()


def test_noalloc_rejects_stacks_beyond_its_scratch():
    """The allocation-free call refuses, before any HIP call, a stack whose
    workspace exceeds its fixed scratch (here the ResNet-18 convolutions,
    whose instantiated early layers split into many K slices)."""
    import workloads as wl
    w = wl.get(6)
    arr = (bk.bk_layer * len(w.layers))()
    for c, L in zip(arr, w.layers):
        c.kind, c.T, c.d, c.p = bk.BK_LINEAR, L.T, L.d, L.p
        c.x = c.g = c.G = 0x10000
    n = len(w.layers)
    assert bk.bk_private_grad_workspace_size(arr, n, bk.BK_BF16, w.B) > bk.BK_NOALLOC_SCRATCH_BYTES
    st = bk.lib.bk_private_grad_noalloc(arr, n, bk.BK_BF16, w.B, bk.BK_CLIP_AUTO, 1.0, 0.01, 1.0, 0, 0,
                                        FAKE, FAKE, None, None)
    assert st == bk.BK_ERR_NOT_SUPPORTED and "scratch" in bk.bk_last_error()


def test_last_error_is_per_thread():
    """bk_last_error() reports the calling thread's own last failure while other
    threads fail at the same time (the ctypes calls release the GIL)."""
    import threading
    errors = []

    def worker(k):
        arr = (bk.bk_layer * 1)()
        arr[0].T, arr[0].d, arr[0].p = 8, 16, 16
        arr[0].x = arr[0].g = arr[0].G = 0x10000
        arr[0].kind = 10 + k                                  # a distinct unknown kind per thread
        for _ in range(300):
            st = bk.lib.bk_layer_norms(arr, 1, bk.BK_BF16, 4, FAKE, FAKE, 1 << 20, None)
            msg = bk.bk_last_error()
            if st != bk.BK_ERR_INVALID_VALUE or f"unknown kind {10 + k}" not in msg:
                errors.append((k, st, msg))
                return

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:3]
