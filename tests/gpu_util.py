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
