"""Benchmark of the BK private-gradient path on one MI355X.

One step = the whole path of Algorithm 1 after book-keeping, over one batch of
a synthetic layer stack whose inputs already sit in HBM:

    convolution layers: unfold x and make dL/ds token-major        -> a, g
    per-layer per-sample norms (ghost / instantiated / embedding)  -> [L, B]
    clip factors                                                   -> [B]
    clip-weighted gradients of every layer                         -> G_l
    Gaussian noise on every G_l

Default workload: the GPT-2-small-shaped stack (12 blocks of 768->2304,
768->768, 768->3072, 3072->768; B=32, T=128, bf16, automatic clipping
gamma=0.01, sigma=1).  Prints one JSON line: samples/s, the roofline of the
dominant kernel measured with HIP events on the launch stream over the timed
steps, and the float64 CPU oracle timed on a bounded sample of the same
workload on the host.

    python bench.py [--steps K] [--warmup W] [--workload N] [--mixopt] [--time-rule] [--gpus 1]

Defaults: 50 timed steps.  Before them a ramp of untimed steps fills 100 ms of
GPU time (reported as `warmup_ramp`), then --warmup more untimed steps run
(reported as `warmup`, default 0).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

METRIC = "BK clipped-grad samples/s on layer stack; ghost-norm+weighted-GEMM % MFMA peak"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA


def true_d(L: wl.Layer) -> int:
    """Input width of the layer's linear view without the zero padding columns."""
    return L.conv[0] * L.conv[1] ** 2 if L.kind == "conv" else L.d


def is_ghost(L, time_rule: bool = False) -> bool:
    """The layerwise decision on the padded width: by space, 2T^2 < pd (the
    paper's), or by time, T(p+d) < pd (the option BK_LAYER_TIME_RULE)."""
    return L.T * (L.p + L.d) < L.p * L.d if time_rule else 2 * L.T * L.T < L.p * L.d


def algorithmic_work(w: wl.Workload, mixopt: bool = False, time_rule: bool = False):
    """Per-step algorithmic flops / bytes of each phase (paper's per-module costs).
    mixopt: instantiated layers keep their per-sample gradients (written by the
    norm phase, 4Bpd bytes) and form G as their weighted sum (2Bpd flops,
    reading 4Bpd and writing 4pd bytes) instead of the 2BTpd GEMM.
    Convolution layers count as linear layers of width d = C_in k^2 (App. B);
    their preparation reads x and dL/ds once and writes a and g once."""
    es = 2 if w.dtype == "bf16" else 4
    B = w.B
    out = {"norm_flops": 0.0, "norm_bytes": 0.0, "gemm_flops": 0.0, "gemm_bytes": 0.0,
           "noise_elems": 0.0, "prep_bytes": 0.0, "ghost_layers": 0, "inst_layers": 0,
           "embed_layers": 0, "conv_layers": 0, "affine_layers": 0, "bias_terms": 0}
    for L0 in w.layers:
        L = L0
        if L0.bias or L0.kind == "norm":
            # per-sample sums (App. notes on normalization layers; biases, Section 5):
            # B p sums written and read back, p written; a normalization layer's
            # g and xhat read once (a linear layer's g is already counted with
            # its weight)
            nin = 2 if L0.kind == "norm" else 0
            nsum = (1 if L0.bias else 0) + (1 if L0.kind == "norm" else 0)
            out["norm_bytes"] += B * L0.T * L0.p * es * nin + 4.0 * B * L0.p * nsum
            out["gemm_bytes"] += (4.0 * B * L0.p + 4.0 * L0.p) * nsum
            out["gemm_flops"] += 2.0 * B * L0.p * nsum
            out["noise_elems"] += float(L0.p) * nsum
            out["affine_layers"] += 1 if L0.kind == "norm" else 0
            out["bias_terms"] += 1 if L0.bias else 0
            if L0.kind == "norm":
                continue
        if L0.kind == "conv":
            cin, k, stride, pad, hin = L0.conv
            out["conv_layers"] += 1
            out["prep_bytes"] += B * es * (cin * hin * hin + L0.T * true_d(L0) + 2 * L0.T * L0.p)
            L = wl.Layer("linear", L0.T, true_d(L0), L0.p)
        if L.kind == "embed":
            out["embed_layers"] += 1
            out["norm_bytes"] += B * L.T * (L.p * es + 8)
            out["gemm_bytes"] += B * L.T * (L.p * es + 8) + 4.0 * L.d * L.p
        else:
            ghost = is_ghost(L0, time_rule)              # the decision sees the padded width
            if ghost:
                out["ghost_layers"] += 1
                out["norm_flops"] += 2.0 * B * L.T * L.T * (L.p + L.d)       # ghost norm, App. B.4
            else:
                out["inst_layers"] += 1
                out["norm_flops"] += 2.0 * B * L.T * L.p * L.d               # instantiation, App. B.4.1
            out["norm_bytes"] += B * L.T * (L.d + L.p) * es
            if mixopt and not ghost:
                out["norm_bytes"] += 4.0 * B * L.d * L.p                     # stored per-sample gradients
                out["gemm_flops"] += 2.0 * B * L.p * L.d                     # weighted sum, App. B.5
                out["gemm_bytes"] += 4.0 * B * L.d * L.p + 4.0 * L.d * L.p
            else:
                out["gemm_flops"] += 2.0 * B * L.T * L.p * L.d               # a^T diag(C) g, App. B.3
                out["gemm_bytes"] += B * L.T * (L.d + L.p) * es + 4.0 * L.d * L.p
        out["noise_elems"] += float(L0.d) * L0.p
    return out


def make_inputs(w: wl.Workload, dev):
    """Per layer the (a, g) the path reads, its G, and for convolution layers
    the raw NCHW (x, dL/ds) that the preparation phase turns into a and g."""
    ins, raw = [], []
    for l, L in enumerate(w.layers):
        t = wl.draw_layer(w, l, device=dev)
        if L.kind == "conv":
            raw.append((l, t))
            t = (torch.empty(w.B, L.T, L.d, dtype=w.torch_dtype, device=dev),
                 torch.empty(w.B, L.T, L.p, dtype=w.torch_dtype, device=dev))
        ins.append(t)
    Gs = [torch.empty((L.p,) if L.kind == "norm" else (L.d, L.p), device=dev) for L in w.layers]
    return ins, raw, Gs


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def _oracle_pass(w: wl.Workload, budget_s: float):
    """The float64 oracle on a prefix of the stack (all B samples), in the
    order of Algorithm 1: the per-sample norms of every layer of the prefix,
    their sum over those layers and one clip factor per sample, then each
    layer's clipped gradient and its noise with those factors.  The prefix
    grows layer by layer while the norm pass stays under a third of budget_s
    (the gradients cost about twice the norms).  Returns (seconds, flops of
    both passes done, layers)."""
    import oracle
    t_norm, nl, done = 0.0, 0, 0.0
    inputs, norms = [], []
    for l, L in enumerate(w.layers):
        x, g = wl.draw_layer(w, l)
        t0 = time.perf_counter()
        kind = L.kind
        if kind == "conv":
            cin, k, stride, pad, _ = L.conv
            x, g, kind = oracle.unfold(x, k, k, stride, pad, L.d), oracle.tokens_from_nchw(g), "linear"
        norms.append(oracle.bk_layer_norm(kind, x, g, L.d, L.bias))
        t_norm += time.perf_counter() - t0
        inputs.append((kind, x, g))
        done += layer_flops(w, L)
        nl += 1
        if t_norm >= budget_s / 3:
            break
    t0 = time.perf_counter()
    C = oracle.clip_factors(oracle.aggregate(np.stack(norms)), w.clip, w.R, w.gamma)
    for l, (L, (kind, x, g)) in enumerate(zip(w.layers, inputs)):
        if kind == "embed":
            G = oracle.embed_weighted_grad(x, g, C, L.d)
        elif kind == "norm":
            G = oracle.weighted_sum(oracle.norm_affine_sums(x, g)[0], C)
        else:
            G = oracle.weighted_grad(x, g, C)
        oracle.add_noise(G, w.noise_std, w.wid, l, 0)
        if L.bias:
            oracle.add_noise(oracle.weighted_sum(oracle.bias_sums(g), C), w.noise_std, w.wid,
                             oracle.BIAS_TENSOR | l, 0)
    return t_norm + time.perf_counter() - t0, done, nl


def layer_flops(w: wl.Workload, L: wl.Layer) -> float:
    """The oracle's float64 flops for one layer: its norm by the definition
    (the d x p per-sample gradients, 2BTdp) plus its clipped gradient (2BTdp);
    an embedding's row sums (2BTp each) and an affine layer's per-sample sums
    are counted the same way."""
    if L.kind == "norm":
        return 4.0 * w.B * L.T * L.p
    if L.kind == "embed":
        return 4.0 * w.B * L.T * L.p
    return 4.0 * w.B * L.T * L.p * true_d(L)


def cpu_baseline(w: wl.Workload, budget_s: float = 12.0, single_budget_s: float = 6.0):
    """The float64 oracle on the host with its BLAS on every thread it is
    given, then again on one thread; each pass runs Algorithm 1 (norms, clip
    factors, clipped gradients, noise) over a prefix of the stack (all B
    samples, input generation excluded) for ~its budget of work and is scaled
    to the whole stack by the fraction of the oracle's flops it covered."""
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    total = sum(layer_flops(w, L) for L in w.layers) + 1e-9
    t_used, done, nl = _oracle_pass(w, budget_s)
    with threadpool_limits(limits=1):
        t1, done1, nl1 = _oracle_pass(w, single_budget_s)
    t_full, t_full1 = t_used * total / done, t1 * total / done1
    return {"value": w.B / t_full, "unit": "samples/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {nl} of {len(w.layers)} layers, all {w.B} samples, Algorithm 1 in float64 "
                      f"(norms, clip factors, clipped gradients, noise; {t_used:.1f} s), scaled by the "
                      f"oracle's flops to the whole stack",
            "s_per_step": round(t_full, 3),
            "single_thread": {"value": w.B / t_full1, "s_per_step": round(t_full1, 3), "cores": 1,
                              "sample": f"first {nl1} layers ({t1:.1f} s), scaled the same way"},
            "host": {"cpu_model": _cpu_model(), "os_cpu_count": os.cpu_count()}}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {"agrad_dl_kernel": "paper_2210_00038_amd/csrc/agemm.hip",
                  "agrad_bf16_kernel": "paper_2210_00038_amd/csrc/agemm.hip",
                  "agemm_bf16_kernel": "paper_2210_00038_amd/csrc/agemm.hip",
                  "anarrow_kernel": "paper_2210_00038_amd/csrc/agemm.hip",
                  "ghost_norm_kernel": "paper_2210_00038_amd/csrc/ghost_norm.hip",
                  "ghost_full_kernel": "paper_2210_00038_amd/csrc/ghost_norm.hip",
                  "ghost_long_kernel": "paper_2210_00038_amd/csrc/ghost_norm.hip",
                  "split_reduce_kernel": "paper_2210_00038_amd/csrc/agemm.hip",
                  "embed_join_kernel": "paper_2210_00038_amd/csrc/embed_join.hip",
                  "conv_prep_kernel": "paper_2210_00038_amd/csrc/conv_prep.hip",
                  "noise_kernel": "paper_2210_00038_amd/csrc/clip_noise.hip"}


def _narrow(L) -> bool:
    return min(L.d, L.p) <= 64 and max(L.d, L.p) >= 128


def norm_kernel(L, dtype: str = "bf16", time_rule: bool = False, B: int = 1) -> str:
    """Kernel that takes layer L's norm (the library's rule for 16-byte rows; a label only)."""
    if L.kind == "embed":
        # 8 | p: the id join; else the masked Gram
        return "embed_join_kernel" if L.T <= 16384 and L.p % 8 == 0 else "ghost_norm_kernel"
    if is_ghost(L, time_rule):
        if dtype != "bf16" or L.T <= 128:
            return "ghost_norm_kernel"
        return "ghost_full_kernel" if L.T <= 256 else "ghost_long_kernel"
    if dtype != "bf16":
        return "agemm_kernel"
    if _narrow(L):
        return "anarrow_kernel"
    # whole 256 x 256 tiles on the DMA kernel when the layer gives at least 128 of them
    tiles = -(-L.d // 256) * -(-L.p // 256)
    if L.T >= 64 and 8 * (-(-L.T // 16) * 16) <= 9 * L.T and B * tiles >= 128:
        return "agrad_dl_kernel"
    return "agemm_bf16_kernel"


def grad_kernel(L, dtype: str = "bf16") -> str:
    """Kernel that takes layer L's clipped gradient (same rule; a label only)."""
    if L.kind == "embed":
        return "embed_rows_kernel"
    if dtype != "bf16":
        return "agemm_kernel"
    if L.T < 64:
        return "agemm_bf16_kernel"
    if _narrow(L):
        return "anarrow_kernel"
    # the DMA kernel pads each sample to 16-row steps; it takes T when that adds at most 1/8
    return "agrad_dl_kernel" if 8 * (-(-L.T // 16) * 16) <= 9 * L.T else "agrad_bf16_kernel"


def dominant_kernel(w: wl.Workload, phase: str, time_rule: bool = False) -> str:
    """Kernel with the largest share of a phase's paper-count flops."""
    share = {}
    for L in w.layers:
        if phase == "norms":
            k = norm_kernel(L, w.dtype, time_rule, w.B)
            f = 2.0 * L.T * L.T * (L.p + L.d) if k.startswith("ghost_") else 2.0 * L.T * L.p * L.d
        else:
            k, f = grad_kernel(L, w.dtype), 2.0 * L.T * L.p * L.d
        share[k] = share.get(k, 0.0) + f
    return max(share, key=share.get)


def plain_gemm_ms(w: wl.Workload, ins, reps: int = 10) -> float:
    """hipBLASLt (torch.mm) time of the plain gradients a_flat^T g_flat of every
    linear / unfolded-conv layer of the stack (bf16 in; no weights, no noise),
    the denominator of the stack overhead together with the library's own GEMM."""
    flat = [(x.reshape(-1, x.shape[-1]), g.reshape(-1, g.shape[-1])) for L, (x, g) in zip(w.layers, ins)
            if L.kind in ("linear", "conv")]
    if not flat:
        return float("nan")

    def run():
        for a, g in flat:
            torch.mm(a.t(), g)
    for _ in range(2):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def source_hash(rel: str) -> str:
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary, scaled by the copy-kernel
    calibration; None when absent or when the kernel source has changed."""
    if " + " in kernel:           # launches of one phase: their bytes add up
        parts = [measured_traffic(k, workload) for k in kernel.split(" + ")]
        return None if any(v is None for v in parts) else sum(parts)
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    for e in rec.get("entries", []):
        if e.get("kernel") == kernel and e.get("workload") == workload and kernel in KERNEL_SOURCES and \
                e.get("source_sha256_16") == source_hash(KERNEL_SOURCES[kernel]):
            return e.get("bytes_per_launch")
    return None


def copy_calibration(gib: float = 1.0, reps: int = 5):
    """A plain device copy of known size (read + write `gib` GiB each), the
    reference for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": reps}), flush=True)


WARMUP_MS = 100.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=0,
                    help="untimed steps after the warm-up ramp (untimed steps filling %d ms of GPU "
                         "time, at least 3, which always runs)" % WARMUP_MS)
    ap.add_argument("--workload", type=int, default=2, help="synthetic stack id (1-8)")
    ap.add_argument("--batch", type=int, default=0,
                    help="run the workload's stack at this batch size instead of its own (0: its own)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-plain-gemm", action="store_true",
                    help="skip the hipBLASLt plain-GEMM denominator (keeps a kernel trace to the library)")
    ap.add_argument("--time-rule", action="store_true",
                    help="choose ghost norm vs instantiation by time, T(p+d) < pd, instead of by space")
    ap.add_argument("--mixopt", action="store_true",
                    help="BK-MixOpt: instantiated layers keep per-sample gradients and sum them")
    ap.add_argument("--accumulate", type=int, default=1,
                    help="physical batches per logical batch (gradient accumulation; noise once per step)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path shards by samples "
              "with one all-reduce of each G_l, which this single-GPU build does not run.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    import paper_2210_00038_amd as bk

    w = wl.get(args.workload)
    if args.batch > 0:
        import dataclasses
        w = dataclasses.replace(w, B=args.batch, name=f"{w.name}@B{args.batch}")
    dev = torch.device("cuda:0")
    dt = bk.BK_BF16 if w.dtype == "bf16" else bk.BK_F32
    mode = bk.BK_CLIP_ABADI if w.clip == "abadi" else bk.BK_CLIP_AUTO
    n, B = len(w.layers), w.B

    ins, raw, Gs = make_inputs(w, dev)
    K = max(1, args.accumulate)
    use_ghost = bk.bk_use_ghost_time if args.time_rule else bk.bk_use_ghost
    keep = [args.mixopt and L.kind in ("linear", "conv") and not use_ghost(L.T, L.d, L.p)
            for L in w.layers]
    Ps = [torch.empty(B, L.p, device=dev) if L.kind == "norm" else
          (torch.empty(B, L.d, L.p, device=dev) if k else None) for L, k in zip(w.layers, keep)]
    Gbs = [torch.empty(L.p, device=dev) if L.bias else None for L in w.layers]
    Pbs = [torch.empty(B, L.p, device=dev) if L.bias else None for L in w.layers]
    kinds = {"embed": bk.BK_EMBEDDING, "norm": bk.BK_NORM_AFFINE}

    def layer_array(accumulate: bool):
        return bk.make_layers([{"kind": kinds.get(L.kind, bk.BK_LINEAR), "x": x, "g": g, "G": G, "V": L.d,
                                "mixopt": args.mixopt, "P": P, "bias": L.bias, "Gb": Gb, "Pb": Pb,
                                "accumulate": accumulate, "time_rule": args.time_rule}
                               for L, (x, g), G, P, Gb, Pb in zip(w.layers, ins, Gs, Ps, Gbs, Pbs)])
    arr = layer_array(False)
    arr_acc = layer_array(True)      # physical batches 2..K of a logical batch add to G
    norm_sq = torch.empty(n, B, device=dev)
    C = torch.empty(B, device=dev)
    tot = torch.empty(B, device=dev)
    ws_n = torch.empty(max(1, bk.bk_layer_norms_workspace_size(arr, n, dt, B)), dtype=torch.uint8, device=dev)
    ws_g = torch.empty(max(1, bk.bk_weighted_grads_workspace_size(arr, n, dt, B)), dtype=torch.uint8,
                       device=dev)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    import ctypes
    noised = [(G, l) for l, G in enumerate(Gs)] + [(Gb, bk.BK_BIAS_TENSOR | l) for l, Gb in enumerate(Gbs)
                                                   if Gb is not None]
    nn_ = len(noised)
    g_ptrs = (ctypes.c_void_p * nn_)(*[G.data_ptr() for G, _ in noised])
    g_nel = (ctypes.c_int64 * nn_)(*[G.numel() for G, _ in noised])
    g_tid = (ctypes.c_uint32 * nn_)(*[t for _, t in noised])

    convs = bk.make_convs([{"x": x, "dy": dy, "a": ins[l][0], "g": ins[l][1], "k": w.layers[l].conv[1],
                            "stride": w.layers[l].conv[2], "pad": w.layers[l].conv[3], "ld": w.layers[l].d}
                           for l, (x, dy) in raw])

    def prep():
        if raw:
            bk._check(bk.lib.bk_conv_prep(convs, len(raw), dt, B, sp), "bk_conv_prep")

    def step(ev=None):
        """One logical batch: K physical batches (prep, norms, clip, clipped
        gradients added to G after the first), then the noise once."""
        t = (lambda: ev.append(torch.cuda.Event(enable_timing=True)) or ev[-1].record(stream)) if ev is not None \
            else (lambda: None)
        for k in range(K):
            t()
            prep()
            t()
            bk._check(bk.lib.bk_layer_norms(arr, n, dt, B, norm_sq.data_ptr(), ws_n.data_ptr(),
                                            ws_n.numel(), sp), "bk_layer_norms")
            t()
            bk._check(bk.lib.bk_clip_factors(norm_sq.data_ptr(), n, B, mode, w.R, w.gamma, C.data_ptr(),
                                             tot.data_ptr(), sp), "bk_clip_factors")
            t()
            bk._check(bk.lib.bk_weighted_grads(arr_acc if k else arr, n, C.data_ptr(), dt, B, ws_g.data_ptr(),
                                               ws_g.numel(), sp), "bk_weighted_grads")
        t()
        bk._check(bk.lib.bk_add_noise_grouped(g_ptrs, g_nel, g_tid, nn_, w.noise_std, w.wid, 0, sp),
                  "bk_add_noise_grouped")
        t()

    # From idle the clipped-gradient GEMM needs some 20-25 ms of this load
    # before it runs at its steady speed (up to 30% slower before), whatever
    # the step length: a ramp of untimed steps filling WARMUP_MS of GPU time
    # always runs first, then the requested count of warm-up steps (default:
    # none beyond the ramp).
    ramp, t_w = 0, time.perf_counter()
    while ramp < 3 or time.perf_counter() - t_w < WARMUP_MS * 1e-3:
        step()
        ramp += 1
        if ramp % 8 == 0 or ramp < 3:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    ramp_ms = (time.perf_counter() - t_w) * 1e3
    args.warmup = max(0, args.warmup)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert torch.isfinite(C).all().item(), "non-finite clip factors"

    # events: per physical batch [prep, norms, clip, grads], then noise
    def phase_ms(e):
        out = np.zeros(5)
        for k in range(K):
            b = 4 * k
            for j, slot in enumerate((4, 0, 1, 2)):          # prep, norms, clip, grads
                out[slot] += e[b + j].elapsed_time(e[b + j + 1])
        out[3] = e[4 * K].elapsed_time(e[4 * K + 1])
        return out
    ph_ms = np.array([phase_ms(e) for e in evs]).mean(axis=0)
    step_ev = np.array([e[0].elapsed_time(e[-1]) for e in evs])
    work = algorithmic_work(w, args.mixopt, args.time_rule)
    work = {k: (v * K if k in ("norm_flops", "norm_bytes", "gemm_flops", "gemm_bytes", "prep_bytes") else v)
            for k, v in work.items()}
    ms_step = elapsed * 1e3 / args.steps
    peak_mfma = PEAK_MFMA_TFLOPS[w.dtype]
    phases = {
        "norms": {"ms": ph_ms[0], "tflops": work["norm_flops"] / ph_ms[0] / 1e9,
                  "gbs": work["norm_bytes"] / ph_ms[0] / 1e6},
        "clip": {"ms": ph_ms[1]},
        "weighted_grads": {"ms": ph_ms[2], "tflops": work["gemm_flops"] / ph_ms[2] / 1e9,
                           "gbs": work["gemm_bytes"] / ph_ms[2] / 1e6},
        "noise": {"ms": ph_ms[3], "gbs": 8.0 * work["noise_elems"] / ph_ms[3] / 1e6},
    }
    if raw:
        phases = {"prep": {"ms": ph_ms[4], "gbs": work["prep_bytes"] / ph_ms[4] / 1e6}, **phases}
    # Dominant phase (most time among preparation, norms and clipped
    # gradients); its bound follows from its arithmetic intensity against the
    # ridge point of MI355X (dense bf16 MFMA peak / HBM peak).
    ridge = peak_mfma * 1e3 / PEAK_HBM_GBS                 # flop per byte
    cand = {"weighted_grads": (work["gemm_flops"], work["gemm_bytes"]),
            "norms": (work["norm_flops"], work["norm_bytes"])}
    if raw:
        cand["prep"] = (0.0, work["prep_bytes"])
    dom = max(cand, key=lambda k: phases[k]["ms"])
    flops, nbytes = cand[dom]
    ms_dom = phases[dom]["ms"]
    if dom == "prep":
        gk, what = "conv_prep_kernel", "unfold + token-major transpose of every conv layer, one launch"
    else:
        gk = dominant_kernel(w, dom, args.time_rule)
        kinds = {grad_kernel(L, w.dtype) if dom == "weighted_grads" else norm_kernel(L, w.dtype, args.time_rule, w.B)
                 for L in w.layers}
        what = ("clipped gradients" if dom == "weighted_grads" else "per-sample norms") + \
               (", all layers in one launch" if len(kinds) == 1 else ", one launch per kernel variant")
        if dom == "weighted_grads" and len(kinds) == 1 and all(L.kind != "embed" for L in w.layers) and \
                bk.bk_weighted_grads_workspace_size(arr, n, dt, B) > 0:
            # K-split tiles (few-tile layers, or the last round of a launch):
            # the phase time includes the fixed-order reduction of their slices
            gk += " + split_reduce_kernel"
            what += ", plus the reduction of its K-split tiles"
    if flops / max(nbytes, 1.0) > ridge:
        ach = flops / ms_dom / 1e9
        roof = {"kernel": f"{gk} ({what})", "bound": "mfma", "achieved": ach, "peak": peak_mfma,
                "unit": "TFLOP/s", "frac": ach / peak_mfma,
                "per_launch": f"{flops / 1e9:.1f} GFLOP (" + ("sum over layers of 2 B T d p" if dom == "weighted_grads"
                              else "paper count: 2BT^2(p+d) ghost, 2BTpd instantiated") + ")"}
    else:
        ach = nbytes / ms_dom / 1e6
        roof = {"kernel": f"{gk} ({what})", "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": ach / PEAK_HBM_GBS,
                "per_launch": f"{nbytes / 1e9:.3f} GB (inputs read once, outputs written once)"}
    roof["traffic"] = measured_traffic(gk, w.name)
    for v in phases.values():
        for k in list(v):
            v[k] = round(float(v[k]), 4)
    res = {
        "metric": METRIC, "value": K * B / (ms_step / 1e3), "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "warmup_ramp": {"steps": ramp, "ms": round(ramp_ms, 1)},
        "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "variant": "BK-MixOpt" if args.mixopt else "BK",
                   "rule": "time" if args.time_rule else "space",
                   "accumulate": K, "logical_batch": K * B,
                   "B": B, "layers": n, "T": sorted({L.T for L in w.layers}),
                   "clip": w.clip, "sigma": w.sigma, "paths": {"ghost": work["ghost_layers"],
                   "inst": work["inst_layers"], "embed": work["embed_layers"],
                   "conv": work["conv_layers"], "affine": work["affine_layers"],
                   "bias": work["bias_terms"]}},
        "roofline": roof,
        "step_ms_events": {"p10": round(float(np.percentile(step_ev, 10)), 4),
                           "median": round(float(np.median(step_ev)), 4),
                           "p90": round(float(np.percentile(step_ev, 90)), 4)},
        "phases": phases,
        "mfma_frac": {"ghost_norm_paper_flops": phases["norms"].get("tflops", 0) / peak_mfma,
                      "weighted_gemm": phases["weighted_grads"]["tflops"] / peak_mfma},
    }
    if w.dtype == "bf16" and K == 1 and not args.no_plain_gemm:
        # stack overhead against the plain gradient GEMMs: the faster of
        # hipBLASLt on a_flat^T g_flat and the library's own clipped GEMM
        hb = plain_gemm_ms(w, ins)
        own = phases["weighted_grads"]["ms"]
        res["plain_gemm"] = {"hipblaslt_ms": round(hb, 4), "own_ms": own,
                             "stack_over_plain": round(ms_step / min(hb, own), 3)}
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
