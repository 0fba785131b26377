"""Oracle: LoRA adapter gradients for one adapted projection (Sec. 3.1 episode-specific
adapter; Appendix C: rank r = 8, alpha = 16).

Test infrastructure only: the GPU library never imports this module.

The adapted projection is y = x W0^T + s (x A^T) B^T with s = alpha / r (the usual
LoRA scaling; the paper gives r and alpha, the scale convention is the standard one).
Given the upstream gradient dy = dLoss/dy, with U = x A^T:

    dB = s dy^T U            [d_out, r]
    dA = (s dy B)^T x        [r, d_in]

Computed in float64 from the exact input values.
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
