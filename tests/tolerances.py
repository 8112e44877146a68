"""Parity tolerances shared by the GPU tests and by the CPU tests that check
the guards are tight enough to see a lost token row.

Two bounds apply to every bf16 comparison:
  * the gate, from the stated targets: norms, totals and clip factors within
    2e-2 relative, clipped gradients within 2e-2 relative Frobenius error;
  * a guard near the error the kernels actually make.  The inputs are exact in
    bf16, the MFMA products of two bf16 values are exact in fp32, so norms and
    totals carry only fp32 accumulation error (measured ~1e-7 .. 1e-6).
    Clipped gradients carry the same, except where the clip weight multiplies
    the rows of g before the MFMA: there C_i g is rounded to bf16 first
    (relative 2^-9 per element at worst, ~1.1e-3 rms over a block).
A guard sits well below what one dropped or duplicated token row changes:
about 1/T of a norm and about 1/sqrt(B T) of a clipped-gradient block
(tests/test_guards_cpu.py shows both at the full-size shapes).
"""

# Targets (bf16 inputs with fp32 accumulation / fp32 inputs).
NORM_GATE = {"bf16": 2e-2, "f32": 1e-5}
GRAD_GATE = {"bf16": 2e-2, "f32": 1e-4}

# Guards at the measured error level.
NORM_GUARD = 1e-4            # per-sample norms, totals and clip factors
GRAD_GUARD_EXACT = 1e-4      # weights on the fp32 accumulators (or fp32 products)
GRAD_GUARD_ROUNDED = 3e-3    # C_i g rounded to bf16 before the MFMA

# Stage height of the clipped-gradient kernel that applies the weights to its
# accumulators, and the batch limit of its weight table.
DL_STAGE_ROWS = 32
DL_MAX_B = 4096


def dl_padding_ok(T: int) -> bool:
    """That kernel pads every sample with zero rows to whole stages and runs
    its MFMAs over T rounded up to 16 rows; it takes layers where that adds at
    most 1/8 to T."""
    return 8 * (-(-T // 16) * 16) <= 9 * T


def weights_on_accumulators(T: int, d: int, p: int, B: int, dtype: str = "bf16") -> bool:
    """Whether a bf16 linear layer's clipped gradient runs on the kernel that
    applies C_i to its fp32 accumulators (exact weights) rather than to the
    rows of g (weights rounded with g to bf16): 16-byte rows, both sides wider
    than 64 or neither narrow, T >= 64 with little padding (dl_padding_ok)."""
    if dtype != "bf16":
        return True
    lo, hi = min(d, p), max(d, p)
    narrow = lo <= 64 and hi >= 128
    return (not narrow and T >= 64 and dl_padding_ok(T) and B <= DL_MAX_B and
            d % 8 == 0 and p % 8 == 0)


def grad_guard(T: int, d: int, p: int, B: int, dtype: str = "bf16") -> float:
    return GRAD_GUARD_EXACT if weights_on_accumulators(T, d, p, B, dtype) else GRAD_GUARD_ROUNDED
