"""Helpers for GPU tests and the bench: host arrays -> device tensors, comparison metrics.
No part of the method's arithmetic lives here."""
import sys

import numpy as np


def note(msg):
    """Progress line, flushed, so a GPU run's log names the case it was on."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_dense(dense):
    """A workloads.Dense input as a device tensor: bf16 bit patterns or float32 values."""
    import torch
    if dense.bits is not None:
        return torch.from_numpy(np.ascontiguousarray(dense.bits).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(dense.f32)).cuda()


def host(t):
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return (bits.astype(np.uint32) << 16).view(np.float32)
    return t.cpu().numpy()


def rel_norm(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


def cosine(a, b):
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    na, nb = np.linalg.norm(a), np.linalg.norm(b)
    if na == 0 and nb == 0:
        return 1.0
    return float(a @ b / (na * nb))


def row_cosines(a, b):
    """Cosine of every row of a against the same row of b (rows that are zero in both count as 1)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    a = a.reshape(a.shape[0], -1)
    b = b.reshape(b.shape[0], -1)
    num = np.einsum("ij,ij->i", a, b)
    na = np.linalg.norm(a, axis=1)
    nb = np.linalg.norm(b, axis=1)
    both0 = (na == 0) & (nb == 0)
    den = np.where(both0, 1.0, na * nb)
    return np.where(both0, 1.0, num / np.where(den == 0, np.inf, den))


def elementwise_ratio(got, want):
    """max over elements of |got - want| / (|want| + rms(want's row)): the smallest c for which
    |got - want| <= c (|want| + rms_row) holds everywhere."""
    g = np.asarray(got, np.float64)
    w = np.asarray(want, np.float64)
    g = g.reshape(g.shape[0], -1)
    w = w.reshape(w.shape[0], -1)
    rms = np.sqrt(np.mean(w * w, axis=1, keepdims=True))
    den = np.abs(w) + rms
    err = np.abs(g - w)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(den > 0, err / np.where(den > 0, den, 1.0), np.where(err > 0, np.inf, 0.0))
    return float(r.max()) if r.size else 0.0


def check_rows(got, want, cos_min, elem_c, what):
    """Every row's cosine >= cos_min and |got - want| <= elem_c (|want| + rms_row) element by
    element. Prints the observed extremes so a log records the margin."""
    cos = row_cosines(got, want)
    ratio = elementwise_ratio(got, want)
    worst = int(np.argmin(cos)) if cos.size else -1
    note(f"{what}: {cos.size} rows, min row cosine {cos.min() if cos.size else 1.0:.7f} (row {worst}), "
         f"max |err|/(|ref|+rms_row) {ratio:.3e}")
    assert cos.size == 0 or cos.min() >= cos_min, (what, worst, float(cos.min()))
    assert ratio <= elem_c, (what, ratio)
