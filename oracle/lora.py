"""Oracle: LoRA adapter gradients for one adapted projection (Sec. 3.1 episode-specific
adapter; Appendix C: rank r = 8, alpha = 16).

Test infrastructure only: the GPU library never imports this module.

The adapted projection is y = x W0^T + s (x A^T) B^T with s = alpha / r (the usual
LoRA scaling; the paper gives r and alpha, the scale convention is the standard one).
Given the upstream gradient dy = dLoss/dy, with U = x A^T:

    dB = s dy^T U            [d_out, r]
    dA = (s dy B)^T x        [r, d_in]

Computed in float64 from the exact input values.

The adapter step of Eq. 2 (and of Algorithm 1), theta <- theta - eta grad, is taken on
float32 parameters in float32 arithmetic: the product eta * grad rounded to nearest, then the
difference rounded to nearest (the paper fixes no precision; this is the reading the library
documents). Its bf16 operand copy rounds to nearest even.
"""
import numpy as np


def lora_grad(x, dy, A, B, scale):
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    U = x @ A.T
    dU = scale * (dy @ B)
    return dU.T @ x, scale * (dy.T @ U)


def lora_grad_sampled(x, dy, A, B, scale, in_cols, out_rows):
    """dA[:, in_cols] and dB[out_rows, :] only (U and dU are formed in full)."""
    x = np.asarray(x)
    dy = np.asarray(dy)
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    U = np.asarray(x, np.float64) @ A.T
    dU = scale * (np.asarray(dy, np.float64) @ B)
    dA_cols = dU.T @ np.asarray(x[:, in_cols], np.float64)
    dB_rows = scale * (np.asarray(dy[:, out_rows], np.float64).T @ U)
    return dA_cols, dB_rows


def lora_forward(x, W0, A, B, scale):
    """y = x W0^T + s (x A^T) B^T, used by finite-difference checks."""
    x = np.asarray(x, np.float64)
    y = x @ np.asarray(A, np.float64).T @ np.asarray(B, np.float64).T * scale
    if W0 is not None:
        y = y + x @ np.asarray(W0, np.float64).T
    return y


def sgd_step(param, grad, lr):
    """theta - lr * grad (Eq. 2) in float32: numpy rounds the product and the difference to
    nearest, one IEEE operation each."""
    p = np.asarray(param, np.float32)
    g = np.asarray(grad, np.float32)
    return p - np.float32(lr) * g


def bf16_round_bits(values):
    """bfloat16 bit patterns of float32 values, rounded to nearest, ties to even (the upper 16
    bits after adding 0x7FFF plus the lowest kept bit); NaN stays a quiet NaN of the same sign."""
    b = np.asarray(values, np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(values, np.float32))
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) & 0xFFFF
    q = ((b >> 16) | 0x0040) & 0xFFFF
    return np.where(nan, q, r).astype(np.uint16)
