"""Book-Keeping (BK) differentially private gradient path on MI355X (gfx950).

Thin Python binding over ``libbk.so`` (C ABI in ``include/bk.h``).  Every
function keeps the name of the C entry point it wraps and only marshals
arguments: torch tensors provide device memory and the current HIP stream,
the computation itself runs in the library's HIP kernels.  There is no CPU or
PyTorch fallback: if ``libbk.so`` is missing the import fails.

Method: Bu, Wang, Zha, Karypis, "Differentially Private Optimization on Large
Model at Small Cost" (ICML 2023, arXiv 2210.00038) -- Algorithm 1 from the
per-layer norms to the noise, with the layerwise ghost / instantiation choice
of Section 3.2.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

__all__ = [
    "BK_OK", "BK_ERR_INVALID_VALUE", "BK_ERR_NOT_SUPPORTED", "BK_ERR_WORKSPACE", "BK_ERR_LAUNCH",
    "BK_F32", "BK_BF16", "BK_CLIP_ABADI", "BK_CLIP_AUTO", "BK_LINEAR", "BK_EMBEDDING", "BK_NORM_AFFINE",
    "BK_LAYER_MIXOPT", "BK_LAYER_BIAS", "BK_LAYER_ACCUMULATE", "BK_LAYER_TIME_RULE", "BK_BIAS_TENSOR",
    "BK_OP_GHOST_NORM", "BK_OP_INST_NORM", "BK_OP_EMBED_GHOST_NORM", "BK_OP_WEIGHTED_GRAD",
    "BK_OP_EMBED_WEIGHTED_GRAD", "BKError", "bk_layer", "lib", "LIB_PATH", "EXPORTS",
    "bk_use_ghost", "bk_use_ghost_time", "bk_workspace_size", "bk_ghost_norm", "bk_inst_norm",
    "bk_embed_ghost_norm", "bk_per_sample_grads", "bk_weighted_sum", "bk_unfold", "bk_tokens_from_nchw", "bk_conv",
    "bk_conv_prep", "make_convs",
    "bk_clip_factors", "bk_weighted_grad", "bk_embed_weighted_grad", "bk_add_noise", "bk_philox_raw",
    "bk_add_noise_grouped", "bk_layer_norms", "bk_weighted_grads", "bk_private_grad",
    "bk_private_grad_noalloc", "BK_NOALLOC_SCRATCH_BYTES", "make_layers",
    "conv_out_size",
    "bk_layer_norms_workspace_size", "bk_weighted_grads_workspace_size",
    "bk_private_grad_workspace_size", "bk_status_string", "bk_last_error", "bk_version",
]

BK_OK, BK_ERR_INVALID_VALUE, BK_ERR_NOT_SUPPORTED, BK_ERR_WORKSPACE, BK_ERR_LAUNCH = range(5)
BK_F32, BK_BF16 = 0, 1
BK_CLIP_ABADI, BK_CLIP_AUTO = 0, 1
BK_LINEAR, BK_EMBEDDING, BK_NORM_AFFINE = 0, 1, 2
BK_LAYER_MIXOPT, BK_LAYER_BIAS, BK_LAYER_ACCUMULATE, BK_LAYER_TIME_RULE = 1, 2, 4, 8
BK_BIAS_TENSOR = 0x80000000
BK_NOALLOC_SCRATCH_BYTES = 64 << 20
(BK_OP_GHOST_NORM, BK_OP_INST_NORM, BK_OP_EMBED_GHOST_NORM, BK_OP_WEIGHTED_GRAD,
 BK_OP_EMBED_WEIGHTED_GRAD) = range(5)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbk.so")

# Every symbol include/bk.h declares.
EXPORTS = (
    "bk_use_ghost", "bk_use_ghost_time", "bk_workspace_size", "bk_ghost_norm", "bk_inst_norm", "bk_embed_ghost_norm",
    "bk_per_sample_grads", "bk_weighted_sum", "bk_unfold", "bk_tokens_from_nchw", "bk_conv_prep",
    "bk_clip_factors", "bk_weighted_grad", "bk_embed_weighted_grad", "bk_add_noise",
    "bk_add_noise_grouped", "bk_philox_raw", "bk_layer_norms_workspace_size", "bk_layer_norms", "bk_weighted_grads_workspace_size",
    "bk_weighted_grads", "bk_private_grad_workspace_size", "bk_private_grad", "bk_private_grad_noalloc",
    "bk_status_string",
    "bk_last_error", "bk_version",
)


class BKError(RuntimeError):
    def __init__(self, status: int, fn: str, detail: str):
        self.status = status
        super().__init__(f"{fn} failed with {_status_name(status)}: {detail}")


class bk_layer(ctypes.Structure):
    """Mirror of ``struct bk_layer`` in include/bk.h."""
    _fields_ = [("kind", ctypes.c_int32), ("flags", ctypes.c_int32), ("T", ctypes.c_int64),
                ("d", ctypes.c_int64), ("p", ctypes.c_int64), ("x", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("G", ctypes.c_void_p), ("P", ctypes.c_void_p),
                ("Gb", ctypes.c_void_p), ("Pb", ctypes.c_void_p)]


class bk_conv(ctypes.Structure):
    """Mirror of ``struct bk_conv`` in include/bk.h."""
    _fields_ = [("x", ctypes.c_void_p), ("dy", ctypes.c_void_p), ("a", ctypes.c_void_p),
                ("g", ctypes.c_void_p)] + [(f, ctypes.c_int64) for f in
                                           ("C", "H", "W", "kh", "kw", "stride", "pad", "ld", "p")]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2210_00038_amd/build.py` "
                      "(the BK path has no fallback)")
lib = ctypes.CDLL(LIB_PATH)

_i64, _u64, _u32, _f32, _vp, _sz = (ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                                    ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t)
_st = ctypes.c_int
_P = ctypes.POINTER(bk_layer)
_SIG = {
    "bk_use_ghost": (ctypes.c_int, [_i64, _i64, _i64]),
    "bk_use_ghost_time": (ctypes.c_int, [_i64, _i64, _i64]),
    "bk_workspace_size": (_sz, [ctypes.c_int, ctypes.c_int, _i64, _i64, _i64, _i64]),
    "bk_ghost_norm": (_st, [_vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp, _sz, _vp]),
    "bk_inst_norm": (_st, [_vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp, _sz, _vp]),
    "bk_embed_ghost_norm": (_st, [_vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp, _sz, _vp]),
    "bk_per_sample_grads": (_st, [_vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp, _vp, _sz,
                                  _vp]),
    "bk_weighted_sum": (_st, [_vp, _vp, _i64, _i64, _vp, _vp]),
    "bk_unfold": (_st, [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _vp, _vp]),
    "bk_tokens_from_nchw": (_st, [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp]),
    "bk_conv_prep": (_st, [ctypes.POINTER(bk_conv), _i64, ctypes.c_int, _i64, _vp]),
    "bk_clip_factors": (_st, [_vp, _i64, _i64, ctypes.c_int, _f32, _f32, _vp, _vp, _vp]),
    "bk_weighted_grad": (_st, [_vp, _vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp, _sz, _vp]),
    "bk_embed_weighted_grad": (_st, [_vp, _vp, _vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, _vp,
                                     _sz, _vp]),
    "bk_add_noise": (_st, [_vp, _i64, _f32, _u64, _u32, _u32, _vp]),
    "bk_add_noise_grouped": (_st, [_vp, _vp, _vp, _i64, _f32, _u64, _u32, _vp]),
    "bk_philox_raw": (_st, [_u64, _u32, _u32, _u64, _i64, _vp, _vp]),
    "bk_layer_norms_workspace_size": (_sz, [_P, _i64, ctypes.c_int, _i64]),
    "bk_layer_norms": (_st, [_P, _i64, ctypes.c_int, _i64, _vp, _vp, _sz, _vp]),
    "bk_weighted_grads_workspace_size": (_sz, [_P, _i64, ctypes.c_int, _i64]),
    "bk_weighted_grads": (_st, [_P, _i64, _vp, ctypes.c_int, _i64, _vp, _sz, _vp]),
    "bk_private_grad_workspace_size": (_sz, [_P, _i64, ctypes.c_int, _i64]),
    "bk_private_grad": (_st, [_P, _i64, ctypes.c_int, _i64, ctypes.c_int, _f32, _f32, _f32, _u64, _u32,
                              _vp, _vp, _vp, _vp, _sz, _vp]),
    "bk_private_grad_noalloc": (_st, [_P, _i64, ctypes.c_int, _i64, ctypes.c_int, _f32, _f32, _f32, _u64,
                                      _u32, _vp, _vp, _vp, _vp]),
    "bk_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "bk_last_error": (ctypes.c_char_p, []),
    "bk_version": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _SIG.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _status_name(s: int) -> str:
    return lib.bk_status_string(s).decode()


def bk_status_string(s: int) -> str:
    return _status_name(s)


def bk_last_error() -> str:
    return lib.bk_last_error().decode()


def bk_version() -> str:
    return lib.bk_version().decode()


def _check(status: int, fn: str) -> None:
    if status != BK_OK:
        raise BKError(status, fn, bk_last_error())


# ---------------------------------------------------------------- marshalling
def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BK_BF16
    if t.dtype == torch.float32:
        return BK_F32
    raise TypeError(f"unsupported dtype {t.dtype}: a and g must be bfloat16 or float32")


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device (cuda/HIP) tensor, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else (t.data_ptr() or None)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def _workspace(nbytes: int, device, ws: Optional[torch.Tensor]):
    if nbytes == 0:
        return None, 0
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, ws.numel() * ws.element_size()


def _out(t: Optional[torch.Tensor], shape, device, dtype=torch.float32) -> torch.Tensor:
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _dev(t, "output")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"output must be {dtype} of shape {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")
    return t


# ------------------------------------------------------------------ per layer
def bk_use_ghost(T: int, d: int, p: int) -> bool:
    r = lib.bk_use_ghost(T, d, p)
    if r < 0:
        raise ValueError("negative size")
    return bool(r)


def bk_use_ghost_time(T: int, d: int, p: int) -> bool:
    r = lib.bk_use_ghost_time(T, d, p)
    if r < 0:
        raise ValueError("negative size")
    return bool(r)


def bk_workspace_size(op: int, dtype: int, B: int, T: int, d: int, p: int) -> int:
    return int(lib.bk_workspace_size(op, dtype, B, T, d, p))


def _linear_norm(fn: str, op: int, a, g, norm_sq, ws, stream):
    _dev(a, "a"), _dev(g, "g")
    if a.dim() != 3 or g.dim() != 3 or a.shape[:2] != g.shape[:2] or a.dtype != g.dtype:
        raise ValueError("a must be [B,T,d] and g [B,T,p] of one dtype")
    B, T, d = a.shape
    p = g.shape[2]
    dt = _dtype_code(a)
    norm_sq = _out(norm_sq, (B,), a.device)
    ws, nws = _workspace(bk_workspace_size(op, dt, B, T, d, p), a.device, ws)
    _check(getattr(lib, fn)(_ptr(a), _ptr(g), dt, B, T, d, p, _ptr(norm_sq), _ptr(ws), nws,
                            _stream(stream)), fn)
    return norm_sq


def bk_ghost_norm(a, g, norm_sq=None, ws=None, stream=None) -> torch.Tensor:
    """Per-sample ||a_i^T g_i||_F^2 by the ghost norm (eq. "ghost norm")."""
    return _linear_norm("bk_ghost_norm", BK_OP_GHOST_NORM, a, g, norm_sq, ws, stream)


def bk_inst_norm(a, g, norm_sq=None, ws=None, stream=None) -> torch.Tensor:
    """Per-sample ||a_i^T g_i||_F^2 by instantiation (App. B.4.1)."""
    return _linear_norm("bk_inst_norm", BK_OP_INST_NORM, a, g, norm_sq, ws, stream)


def bk_per_sample_grads(a, g, norm_sq=None, P=None, ws=None, stream=None):
    """(norm_sq [B], P [B,d,p]): per-sample gradients a_i^T g_i kept (BK-MixOpt, App. B.4.1)."""
    _dev(a, "a"), _dev(g, "g")
    if a.dim() != 3 or g.dim() != 3 or a.shape[:2] != g.shape[:2] or a.dtype != g.dtype:
        raise ValueError("a must be [B,T,d] and g [B,T,p] of one dtype")
    B, T, d = a.shape
    p = g.shape[2]
    dt = _dtype_code(a)
    norm_sq = _out(norm_sq, (B,), a.device)
    P = _out(P, (B, d, p), a.device)
    ws, nws = _workspace(bk_workspace_size(BK_OP_INST_NORM, dt, B, T, d, p), a.device, ws)
    _check(lib.bk_per_sample_grads(_ptr(a), _ptr(g), dt, B, T, d, p, _ptr(norm_sq), _ptr(P), _ptr(ws),
                                   nws, _stream(stream)), "bk_per_sample_grads")
    return norm_sq, P


def bk_weighted_sum(P, C, G=None, stream=None) -> torch.Tensor:
    """sum_i C_i P_i over stored per-sample gradients P [B, ...] (App. B.5), float32."""
    _dev(P, "P"), _dev(C, "C")
    if P.dtype != torch.float32 or C.dtype != torch.float32 or C.dim() != 1 or P.shape[0] != C.shape[0]:
        raise ValueError("P must be float32 [B, ...] and C float32 [B]")
    if not P.is_contiguous():
        raise ValueError("P must be contiguous")
    B = P.shape[0]
    G = _out(G, tuple(P.shape[1:]), P.device)
    n = G.numel()
    _check(lib.bk_weighted_sum(_ptr(P), _ptr(C), B, n, _ptr(G), _stream(stream)), "bk_weighted_sum")
    return G


def conv_out_size(n: int, k: int, stride: int, pad: int) -> int:
    return (n + 2 * pad - k) // stride + 1


def bk_unfold(x, kh: int, kw: int, stride: int = 1, pad: int = 0, ld: int = 0, a=None, stream=None):
    """Unfolded input of a 2-D convolution: x [B,C,H,W] -> a [B, Ho Wo, ld] (ld = 0: C kh kw)."""
    _dev(x, "x")
    if x.dim() != 4 or not x.is_contiguous():
        raise ValueError("x must be a contiguous [B, C, H, W] tensor")
    B, C, H, W = x.shape
    Ho, Wo = conv_out_size(H, kh, stride, pad), conv_out_size(W, kw, stride, pad)
    ld = ld or C * kh * kw
    a = _out(a, (B, Ho * Wo, ld), x.device, dtype=x.dtype)
    _check(lib.bk_unfold(_ptr(x), _dtype_code(x), B, C, H, W, kh, kw, stride, pad, ld, _ptr(a),
                         _stream(stream)), "bk_unfold")
    return a


def bk_tokens_from_nchw(y, out=None, stream=None):
    """Token-major output gradient of a convolution: y [B,C,H,W] -> [B, H W, C]."""
    _dev(y, "y")
    if y.dim() != 4 or not y.is_contiguous():
        raise ValueError("y must be a contiguous [B, C, H, W] tensor")
    B, C, H, W = y.shape
    out = _out(out, (B, H * W, C), y.device, dtype=y.dtype)
    _check(lib.bk_tokens_from_nchw(_ptr(y), _dtype_code(y), B, C, H, W, _ptr(out), _stream(stream)),
           "bk_tokens_from_nchw")
    return out


def make_convs(specs: Sequence[dict]):
    """ctypes bk_conv array from dicts {x [B,C,H,W] (or None with C, H, W given), dy [B,p,Ho,Wo]
    (or None with p given), a, g (preallocated outputs [B, Ho Wo, ld] and [B, Ho Wo, p]),
    k or (kh, kw), stride, pad, ld (0: C kh kw)}."""
    arr = (bk_conv * len(specs))()
    for c, sp in zip(arr, specs):
        x, dy = sp.get("x"), sp.get("dy")
        for t, nm in ((x, "x"), (dy, "dy"), (sp.get("a"), "a"), (sp.get("g"), "g")):
            if t is not None:
                _dev(t, nm)
        C, H, W = x.shape[1:] if x is not None else (sp["C"], sp["H"], sp["W"])
        kh, kw = sp.get("kh", sp.get("k")), sp.get("kw", sp.get("k"))
        c.x, c.dy = _ptr(x) if x is not None else None, _ptr(dy) if dy is not None else None
        c.a = _ptr(sp["a"]) if sp.get("a") is not None else None
        c.g = _ptr(sp["g"]) if sp.get("g") is not None else None
        c.C, c.H, c.W, c.kh, c.kw = C, H, W, kh, kw
        c.stride, c.pad = sp.get("stride", 1), sp.get("pad", 0)
        c.ld = sp.get("ld") or C * kh * kw
        c.p = dy.shape[1] if dy is not None else sp.get("p", 0)
    return arr


def bk_conv_prep(convs, n: int, dtype, B: int, stream=None):
    """Unfold and transpose every convolution layer of `convs` (a bk_conv array) in one call."""
    _check(lib.bk_conv_prep(convs, n, dtype, B, _stream(stream)), "bk_conv_prep")


def bk_embed_ghost_norm(ids, g, V: int, norm_sq=None, ws=None, stream=None) -> torch.Tensor:
    """Per-sample gradient norm of an embedding layer with vocabulary V."""
    _dev(ids, "ids"), _dev(g, "g")
    if ids.dtype != torch.int64 or ids.dim() != 2 or g.dim() != 3 or ids.shape != g.shape[:2]:
        raise ValueError("ids must be int64 [B,T] and g [B,T,p]")
    B, T, p = g.shape
    dt = _dtype_code(g)
    norm_sq = _out(norm_sq, (B,), g.device)
    ws, nws = _workspace(bk_workspace_size(BK_OP_EMBED_GHOST_NORM, dt, B, T, V, p), g.device, ws)
    _check(lib.bk_embed_ghost_norm(_ptr(ids), _ptr(g), dt, B, T, p, V, _ptr(norm_sq), _ptr(ws), nws,
                                   _stream(stream)), "bk_embed_ghost_norm")
    return norm_sq


def bk_clip_factors(norm_sq, mode: int, R: float = 1.0, gamma: float = 0.01, C=None, total_sq=None,
                    stream=None):
    """(C, total_sq) from per-layer norms [L, B] (Algorithm 1, aggregation and clipping)."""
    _dev(norm_sq, "norm_sq")
    if norm_sq.dtype != torch.float32 or norm_sq.dim() != 2:
        raise ValueError("norm_sq must be float32 [L, B]")
    L, B = norm_sq.shape
    C = _out(C, (B,), norm_sq.device)
    total_sq = _out(total_sq, (B,), norm_sq.device)
    _check(lib.bk_clip_factors(_ptr(norm_sq), L, B, mode, R, gamma, _ptr(C), _ptr(total_sq),
                               _stream(stream)), "bk_clip_factors")
    return C, total_sq


def bk_weighted_grad(a, g, C, G=None, ws=None, stream=None) -> torch.Tensor:
    """G = a^T diag(C) g = sum_i C_i a_i^T g_i, [d, p] float32."""
    _dev(a, "a"), _dev(g, "g"), _dev(C, "C")
    if a.dim() != 3 or g.dim() != 3 or a.shape[:2] != g.shape[:2] or a.dtype != g.dtype:
        raise ValueError("a must be [B,T,d] and g [B,T,p] of one dtype")
    B, T, d = a.shape
    p = g.shape[2]
    if C.dtype != torch.float32 or tuple(C.shape) != (B,):
        raise ValueError("C must be float32 [B]")
    dt = _dtype_code(a)
    G = _out(G, (d, p), a.device)
    ws, nws = _workspace(bk_workspace_size(BK_OP_WEIGHTED_GRAD, dt, B, T, d, p), a.device, ws)
    _check(lib.bk_weighted_grad(_ptr(a), _ptr(g), _ptr(C), dt, B, T, d, p, _ptr(G), _ptr(ws), nws,
                                _stream(stream)), "bk_weighted_grad")
    return G


def bk_embed_weighted_grad(ids, g, C, V: int, G=None, ws=None, stream=None) -> torch.Tensor:
    """G[v, :] = sum_i C_i sum_{t: x_it = v} g_it, [V, p] float32."""
    _dev(ids, "ids"), _dev(g, "g"), _dev(C, "C")
    if ids.dtype != torch.int64 or ids.dim() != 2 or g.dim() != 3 or ids.shape != g.shape[:2]:
        raise ValueError("ids must be int64 [B,T] and g [B,T,p]")
    B, T, p = g.shape
    if C.dtype != torch.float32 or tuple(C.shape) != (B,):
        raise ValueError("C must be float32 [B]")
    dt = _dtype_code(g)
    G = _out(G, (V, p), g.device)
    ws, nws = _workspace(bk_workspace_size(BK_OP_EMBED_WEIGHTED_GRAD, dt, B, T, V, p), g.device, ws)
    _check(lib.bk_embed_weighted_grad(_ptr(ids), _ptr(g), _ptr(C), dt, B, T, p, V, _ptr(G), _ptr(ws),
                                      nws, _stream(stream)), "bk_embed_weighted_grad")
    return G


def bk_add_noise(G, std: float, seed: int, tensor_id: int, step: int = 0, stream=None) -> torch.Tensor:
    """G += std * N(0, I) in place (Philox4x32-10 + Box-Muller)."""
    _dev(G, "G")
    if G.dtype != torch.float32:
        raise ValueError("G must be float32")
    _check(lib.bk_add_noise(_ptr(G), G.numel(), std, seed, tensor_id, step, _stream(stream)),
           "bk_add_noise")
    return G


def bk_add_noise_grouped(Gs: Sequence[torch.Tensor], std: float, seed: int, tensor_ids=None, step: int = 0,
                         stream=None):
    """bk_add_noise on every tensor of Gs in one launch (tensor k uses tensor_ids[k], default k)."""
    n = len(Gs)
    for G in Gs:
        _dev(G, "G")
        if G.dtype != torch.float32:
            raise ValueError("G must be float32")
    ptrs = (ctypes.c_void_p * max(1, n))(*[_ptr(G) for G in Gs])
    nel = (ctypes.c_int64 * max(1, n))(*[G.numel() for G in Gs])
    tids = (ctypes.c_uint32 * max(1, n))(*(range(n) if tensor_ids is None else tensor_ids))
    _check(lib.bk_add_noise_grouped(ptrs, nel, tids, n, std, seed, step, _stream(stream)),
           "bk_add_noise_grouped")
    return Gs


def bk_philox_raw(seed: int, tensor_id: int, step: int, q0: int, nq: int, out=None, device="cuda",
                  stream=None) -> torch.Tensor:
    """Raw Philox4x32-10 words [nq, 4] (as int32 bit patterns) of counter blocks q0 .. q0+nq-1."""
    out = _out(out, (nq, 4), device, dtype=torch.int32)
    _check(lib.bk_philox_raw(seed, tensor_id, step, q0, nq, _ptr(out), _stream(stream)), "bk_philox_raw")
    return out


# -------------------------------------------------------------------- grouped
def make_layers(specs: Sequence[dict]):
    """ctypes bk_layer array from dicts {kind, x, g, G (optional), V (embedding),
    mixopt (optional bool), P (optional float32 [B,d,p], BK-MixOpt store; [B,p] gamma
    store of an affine layer), bias (optional bool) with Gb [p] and Pb [B,p],
    accumulate (optional bool), time_rule (optional bool: the layerwise decision
    by time, bk_use_ghost_time)}.

    x is a [B,T,d] for a linear layer, int64 ids [B,T] for an embedding, or the
    normalized input [B,T,p] of an affine layer.  The array holds references
    to the tensors, so they stay allocated while it is in use."""
    arr = (bk_layer * max(1, len(specs)))()
    arr._tensors = [s.get(k) for s in specs for k in ("x", "g", "G", "P", "Gb", "Pb") if s.get(k) is not None]
    for k, s in enumerate(specs):
        x, g = _dev(s["x"], "x"), _dev(s["g"], "g")
        G = s.get("G")
        kind = s.get("kind", BK_LINEAR)
        if kind == BK_EMBEDDING:
            d = int(s["V"])
            if x.dtype != torch.int64:
                raise ValueError("embedding ids must be int64")
        else:
            d = x.shape[2]
        arr[k].kind = kind
        arr[k].flags = ((BK_LAYER_MIXOPT if s.get("mixopt") else 0) | (BK_LAYER_BIAS if s.get("bias") else 0) |
                        (BK_LAYER_ACCUMULATE if s.get("accumulate") else 0) |
                        (BK_LAYER_TIME_RULE if s.get("time_rule") else 0))
        arr[k].T = g.shape[1]
        arr[k].d = d
        arr[k].p = g.shape[2]
        arr[k].x = _ptr(x)
        arr[k].g = _ptr(g)
        arr[k].G = _ptr(G)
        arr[k].P = _ptr(s.get("P"))
        arr[k].Gb = _ptr(s.get("Gb"))
        arr[k].Pb = _ptr(s.get("Pb"))
    return arr


def bk_layer_norms_workspace_size(layers, n: int, dtype: int, B: int) -> int:
    return int(lib.bk_layer_norms_workspace_size(layers, n, dtype, B))


def bk_weighted_grads_workspace_size(layers, n: int, dtype: int, B: int) -> int:
    return int(lib.bk_weighted_grads_workspace_size(layers, n, dtype, B))


def bk_private_grad_workspace_size(layers, n: int, dtype: int, B: int) -> int:
    return int(lib.bk_private_grad_workspace_size(layers, n, dtype, B))


def bk_layer_norms(layers, n: int, dtype: int, B: int, norm_sq, ws=None, device="cuda", stream=None):
    """Norms of every layer (ghost / instantiated by the 2T^2 < pd rule, embedding ghost) -> [n, B]."""
    ws, nws = _workspace(bk_layer_norms_workspace_size(layers, n, dtype, B), device, ws)
    _check(lib.bk_layer_norms(layers, n, dtype, B, _ptr(norm_sq), _ptr(ws), nws, _stream(stream)),
           "bk_layer_norms")
    return norm_sq


def bk_weighted_grads(layers, n: int, C, dtype: int, B: int, ws=None, device="cuda", stream=None):
    ws, nws = _workspace(bk_weighted_grads_workspace_size(layers, n, dtype, B), device, ws)
    _check(lib.bk_weighted_grads(layers, n, _ptr(C), dtype, B, _ptr(ws), nws, _stream(stream)),
           "bk_weighted_grads")


def bk_private_grad_noalloc(layers, n: int, dtype: int, B: int, mode: int, R: float, gamma: float,
                            noise_std: float, seed: int, step: int, norm_sq, C, total_sq=None, stream=None):
    """bk_private_grad with the library's own per-GPU scratch array instead of
    a workspace (nothing is allocated; calls on one GPU must not overlap)."""
    _check(lib.bk_private_grad_noalloc(layers, n, dtype, B, mode, R, gamma, noise_std, seed, step,
                                       _ptr(norm_sq), _ptr(C), _ptr(total_sq), _stream(stream)),
           "bk_private_grad_noalloc")


def bk_private_grad(layers, n: int, dtype: int, B: int, mode: int, R: float, gamma: float,
                    noise_std: float, seed: int, step: int, norm_sq, C, total_sq=None, ws=None,
                    device="cuda", stream=None):
    """Algorithm 1 from the per-layer norms to the noise for a whole stack."""
    ws, nws = _workspace(bk_private_grad_workspace_size(layers, n, dtype, B), device, ws)
    _check(lib.bk_private_grad(layers, n, dtype, B, mode, R, gamma, noise_std, seed, step, _ptr(norm_sq),
                               _ptr(C), _ptr(total_sq), _ptr(ws), nws, _stream(stream)), "bk_private_grad")
