"""Oracle: the serving side of the episode adapters. Sixteen concurrent episodes each decode
through the shared base model plus their own LoRA adapter, and after every update the trained
adapter is swapped into serving (Appendix A: concurrent episodes, adapters loaded at run time,
a swap in well under a second; adapter of Sec. 3.1, rank and alpha in Appendix C).

Test infrastructure only: the GPU library never imports this module.

Readings (the paper names the serving engine but states no arithmetic):
  * The adapted projection is y = x W0^T + s (x A^T) B^T with s = alpha / r. The base
    product x W0^T is a plain GEMM that the caller has already written into y; the grouped
    forward adds the adapter term of each row's own episode: y <- RN(y + s (x A_e^T) B_e^T),
    the sum exact (float64 from the bf16 values) and rounded once to bf16, nearest even.
  * The swap turns the trained float32 adapter tensors into the bf16 copies the forward
    reads: round to nearest even per element (the rounding of `lora.bf16_round_bits`).
"""
import numpy as np

from .lora import bf16_round_bits


def bf16_bits_to_f64(bits):
    """float64 values of bf16 bit patterns."""
    b = np.asarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def round_f64_to_bf16_bits(v):
    """bf16 bit patterns of float64 values, rounded once to nearest even (no detour through
    float32, which could round twice). bf16 keeps 7 of float64's 52 fraction bits; below
    2^-126 its spacing is the fixed 2^-133, past its largest finite value it gives infinity."""
    v = np.asarray(v, np.float64)
    a = np.abs(v)
    neg = np.signbit(v)
    # normal range: round the float64 bit pattern at bit 45, half to even
    b = a.view(np.uint64)
    keep = np.uint64(52 - 7)
    half = np.uint64(1 << 44)
    odd = (b >> keep) & np.uint64(1)
    r = ((b + half - np.uint64(1) + odd) >> keep) << keep
    q = r.view(np.float64)
    # below 2^-126: multiples of 2^-133 (exact scaling, np.rint ties to even)
    small = a < 2.0 ** -126
    q = np.where(small, np.rint(a * 2.0 ** 133) * 2.0 ** -133, q)
    q = np.where(q >= 2.0 ** 128, np.inf, q)
    with np.errstate(over="ignore"):
        bits = (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)   # q is exact in bf16
    bits = bits | np.where(neg, np.uint16(0x8000), np.uint16(0))
    return np.where(np.isnan(v), np.uint16(0x7FC0), bits).astype(np.uint16)


def lora_forward(x_bits, y_bits, A_bits, B_bits, scale):
    """One segment and one adapted projection: x [rows, d_in], y [rows, d_out], A [r, d_in],
    B [d_out, r], all bf16 bit patterns. Returns the new y bits."""
    x, y, A, B = (bf16_bits_to_f64(a) for a in (x_bits, y_bits, A_bits, B_bits))
    delta = float(scale) * ((x @ A.T) @ B.T)
    return round_f64_to_bf16_bits(y + delta)


def grouped_lora_forward(problems):
    """Every problem (a dict with x, y, A, B bit arrays and scale) on its own; problems never
    interact (the outputs of different problems are distinct). Returns the new y of each."""
    return [lora_forward(p["x"], p["y"], p["A"], p["B"], p["scale"]) for p in problems]


def hot_swap(src):
    """bf16 serving copy of a float32 adapter tensor."""
    return bf16_round_bits(np.asarray(src, np.float32))
