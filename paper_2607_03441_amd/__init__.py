"""Python binding of libattt.so, the gfx950 library of the aTTT in-episode update step
(arXiv 2607.03441: n-gram token weights, Eq. 8-9; weighted LM-head cross-entropy, Eq. 10;
LoRA adapter gradients).

This module only marshals arguments: torch tensors provide device memory and the current
HIP stream, and every step runs in the library's HIP kernels. There is no fallback: if the
library is not built, every call raises.
"""
import ctypes
import os

import numpy as np

__all__ = ["load", "lib_path", "AtttError", "ngram_weights", "ngram_weights_noalloc", "ngram_workspace_size",
           "update_repetition", "repetition_workspace_size", "attention_bwd",
           "ngram_set_size", "ngram_set_init", "ngram_set_append", "ngram_set_weights",
           "weighted_ce_fwd_bwd", "ce_workspace_size", "ce_head_t_size", "ce_head_transpose", "lora_grad", "lora_workspace_size", "lora_sgd_step",
           "lora_forward", "lora_hot_swap",
           "timing_enable", "timing_reset", "timing_read", "kernel_names", "version",
           "F32", "BF16", "LoraProblem", "LoraParam", "LoraFwdProblem", "LoraSwapItem"]

F32 = 0
BF16 = 1
CE_WANT_GRAD = 1
CE_HEAD_T = 2
OK, EINVAL, ENOSPACE, EUNSUPPORTED, EHIP = range(5)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


class AtttError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"attt status {status}: {message}")
        self.status = status


class LoraProblem(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("dy", ctypes.c_void_p), ("A", ctypes.c_void_p),
                ("B", ctypes.c_void_p), ("dA", ctypes.c_void_p), ("dB", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64),
                ("rank", ctypes.c_int32), ("scale", ctypes.c_float)]


class LoraParam(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("param_bf16", ctypes.c_void_p),
                ("n", ctypes.c_int64)]


class LoraFwdProblem(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("y", ctypes.c_void_p), ("A", ctypes.c_void_p),
                ("B", ctypes.c_void_p), ("rows", ctypes.c_int64), ("d_in", ctypes.c_int64),
                ("d_out", ctypes.c_int64), ("rank", ctypes.c_int32), ("scale", ctypes.c_float)]


class LoraSwapItem(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("n", ctypes.c_int64)]


def lib_path():
    return os.path.join(_HERE, "libattt.so")


def load():
    """Load libattt.so (built in-tree by __graft_entry__.build()). Raises if it is missing."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(path)
    i32, i64, f32, vp, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    p64 = ctypes.POINTER(ctypes.c_int64)
    psz = ctypes.POINTER(ctypes.c_size_t)
    L.attt_status_string.restype = ctypes.c_char_p
    L.attt_status_string.argtypes = [i32]
    L.attt_last_error.restype = ctypes.c_char_p
    L.attt_last_error.argtypes = []
    L.attt_version.restype = i32
    L.attt_version.argtypes = []
    L.attt_ngram_workspace_size.restype = i32
    L.attt_ngram_workspace_size.argtypes = [p64, p64, i32, i32, psz]
    L.attt_ngram_weights.restype = i32
    L.attt_ngram_weights.argtypes = [vp, p64, vp, p64, i32, i32, f32, vp, vp, vp, sz, vp]
    L.attt_attention_bwd.restype = i32
    L.attt_attention_bwd.argtypes = [vp, vp, vp, vp, p64, i32, i64, i32, i32, i32, f32, vp, vp, vp, vp, vp, vp]
    L.attt_repetition_workspace_size.restype = i32
    L.attt_repetition_workspace_size.argtypes = [p64, p64, i32, psz]
    L.attt_update_repetition.restype = i32
    L.attt_update_repetition.argtypes = [vp, p64, vp, p64, i32, ctypes.c_double, vp, vp, vp, vp, vp, vp, sz, vp]
    L.attt_ngram_weights_noalloc.restype = i32
    L.attt_ngram_weights_noalloc.argtypes = [vp, p64, vp, p64, i32, i32, f32, vp, vp, vp]
    vpp = ctypes.POINTER(ctypes.c_void_p)
    L.attt_ngram_set_size.restype = i32
    L.attt_ngram_set_size.argtypes = [i64, i32, psz]
    L.attt_ngram_set_init.restype = i32
    L.attt_ngram_set_init.argtypes = [vpp, i32, i64, i32, sz, vp]
    L.attt_ngram_set_append.restype = i32
    L.attt_ngram_set_append.argtypes = [vpp, vp, p64, i32, i64, i32, vp]
    L.attt_ngram_set_weights.restype = i32
    L.attt_ngram_set_weights.argtypes = [vpp, vp, p64, i32, i64, i32, f32, vp, vp, vp]
    L.attt_ce_workspace_size.restype = i32
    L.attt_ce_workspace_size.argtypes = [i64, i64, i64, i32, i32, psz]
    L.attt_weighted_ce_fwd_bwd.restype = i32
    L.attt_weighted_ce_fwd_bwd.argtypes = [vp, vp, vp, vp, p64, i32, i64, i64, i64, i32, vp, vp, vp,
                                           vp, sz, vp]
    L.attt_weighted_ce_fwd_bwd_ex.restype = i32
    L.attt_weighted_ce_fwd_bwd_ex.argtypes = [vp, vp, vp, vp, vp, p64, i32, i64, i64, i64, i32, vp, vp, vp,
                                              vp, sz, vp]
    L.attt_ce_set_wait_limit.restype = i32
    L.attt_ce_set_wait_limit.argtypes = [i64, i64]
    L.attt_ce_head_t_size.restype = i32
    L.attt_ce_head_t_size.argtypes = [i64, i64, psz]
    L.attt_ce_head_transpose.restype = i32
    L.attt_ce_head_transpose.argtypes = [vp, i64, i64, vp, sz, vp]
    L.attt_lora_workspace_size.restype = i32
    L.attt_lora_workspace_size.argtypes = [ctypes.POINTER(LoraProblem), i32, i32, psz]
    L.attt_lora_grad.restype = i32
    L.attt_lora_grad.argtypes = [ctypes.POINTER(LoraProblem), i32, i32, vp, sz, vp]
    L.attt_lora_sgd_step.restype = i32
    L.attt_lora_sgd_step.argtypes = [ctypes.POINTER(LoraParam), i32, f32, i32, vp]
    L.attt_lora_forward.restype = i32
    L.attt_lora_forward.argtypes = [ctypes.POINTER(LoraFwdProblem), i32, vp]
    L.attt_lora_hot_swap.restype = i32
    L.attt_lora_hot_swap.argtypes = [ctypes.POINTER(LoraSwapItem), i32, vp]
    L.attt_timing_enable.restype = i32
    L.attt_timing_enable.argtypes = [i32]
    L.attt_timing_reset.restype = i32
    L.attt_timing_reset.argtypes = []
    L.attt_timing_read.restype = i32
    L.attt_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), p64]
    L.attt_timing_kernel_name.restype = ctypes.c_char_p
    L.attt_timing_kernel_name.argtypes = [i32]
    _LIB = L
    return L


def _check(status):
    if status != OK:
        L = load()
        raise AtttError(status, L.attt_last_error().decode())


def _offsets(off):
    arr = np.ascontiguousarray(np.asarray(off, dtype=np.int64))
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _torch():
    import torch
    return torch


def _stream_ptr():
    return _torch().cuda.current_stream().cuda_stream


def _dptr(t):
    return None if t is None else t.data_ptr()


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _workspace(nbytes, device, workspace):
    torch = _torch()
    if workspace is not None and workspace.numel() >= nbytes:
        return workspace
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def _dev(t, name):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    return t


# ------------------------------------------------------------------------------------------
def ngram_workspace_size(history_offsets, token_offsets, n):
    L = load()
    ho, hp = _offsets(history_offsets)
    to, tp = _offsets(token_offsets)
    out = ctypes.c_size_t(0)
    _check(L.attt_ngram_workspace_size(hp, tp, len(ho) - 1, n, ctypes.byref(out)))
    return out.value


def ngram_weights(history, history_offsets, tokens, token_offsets, n=3, w_min=0.05,
                  want_exposure=True, workspace=None, out=None):
    """Eq. 8-9 for E episodes. history / tokens: int32 device tensors (flat); offsets: host
    int64 sequences of length E+1. Returns (f, w): f as an int32 tensor holding the uint32
    exposure (or None), w float32."""
    torch = _torch()
    L = load()
    ho, hp = _offsets(history_offsets)
    to, tp = _offsets(token_offsets)
    E = len(ho) - 1
    dev = tokens.device
    _dev(tokens, "tokens")
    _dev(history, "history")
    if tokens.dtype != torch.int32 or history.dtype != torch.int32:
        raise TypeError("history and tokens must be int32")
    T = int(to[-1])
    if out is not None:
        f, w = out
    else:
        f = torch.empty(T, dtype=torch.int32, device=dev) if want_exposure else None
        w = torch.empty(T, dtype=torch.float32, device=dev)
    need = ctypes.c_size_t(0)
    _check(L.attt_ngram_workspace_size(hp, tp, E, n, ctypes.byref(need)))
    ws = _workspace(need.value, dev, workspace)
    _check(L.attt_ngram_weights(_dptr(history), hp, _dptr(tokens), tp, E, n, float(w_min), _dptr(f),
                                _dptr(w), _dptr(ws), ws.numel(), _stream_ptr()))
    return f, w


def attention_bwd(q, k, v, dout, row_offsets=None, scale=None, out=None):
    """Backward of one causal grouped-head attention block: (dq, dk, dv, lse, dsum).

    q, dout: device bf16 [N, heads, 128]; k, v: [N, kv_heads, 128]; row_offsets: host int64
    episode offsets or None; scale defaults to 1/sqrt(128). lse, dsum: float32 [heads, N]."""
    torch = _torch()
    L = load()
    for t, name in ((q, "q"), (k, "k"), (v, "v"), (dout, "dout")):
        _dev(t, name)
        if t.dtype != torch.bfloat16 or t.dim() != 3:
            raise TypeError(f"{name} must be bfloat16 [N, heads, head_dim]")
    N, H, dh = q.shape
    Hkv = k.shape[1]
    scale = (1.0 / dh ** 0.5) if scale is None else float(scale)
    if out is None:
        out = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
               torch.empty(H, N, dtype=torch.float32, device=q.device),
               torch.empty(H, N, dtype=torch.float32, device=q.device))
    dq, dk, dv, lse, dsum = out
    if row_offsets is None:
        E, op = 1, None
    else:
        oo, op = _offsets(row_offsets)
        E = len(oo) - 1
    _check(L.attt_attention_bwd(_dptr(q), _dptr(k), _dptr(v), _dptr(dout), op, E, N, H, Hkv, dh, scale,
                                _dptr(dq), _dptr(dk), _dptr(dv), _dptr(lse), _dptr(dsum), _stream_ptr()))
    return dq, dk, dv, lse, dsum


def repetition_workspace_size(text_offsets, episode_texts):
    L = load()
    to, tp = _offsets(text_offsets)
    eo, ep = _offsets(episode_texts)
    need = ctypes.c_size_t()
    _check(L.attt_repetition_workspace_size(tp, ep, len(eo) - 1, ctypes.byref(need)))
    return need.value


def update_repetition(words, text_offsets, episode_texts, tau=0.5, text_offsets_dev=None, want_pairs=False,
                      workspace=None):
    """Update-text repetition rho, novelty nu and the skip decision per episode (Eq. 6-7).

    words: device int32 word ids of all texts back to back; text_offsets: host int64 [T+1];
    episode_texts: host int64 [E+1] (the last text of each episode is the candidate).
    text_offsets_dev: the same offsets already on the device (copied here when not given).
    Returns (rho, nu, skip, best, pairs): device tensors [E] (float64, float64, int32, int32) and
    pairs [P, 2] int32 (|A & B|, |A | B|) when want_pairs, else None."""
    torch = _torch()
    L = load()
    to, tp = _offsets(text_offsets)
    eo, ep = _offsets(episode_texts)
    _dev(words, "words")
    if words.dtype != torch.int32:
        raise TypeError("words must be int32")
    E = len(eo) - 1
    dev = words.device
    if text_offsets_dev is None:
        text_offsets_dev = torch.from_numpy(to).to(dev)
    need = ctypes.c_size_t()
    _check(L.attt_repetition_workspace_size(tp, ep, E, ctypes.byref(need)))
    ws = _workspace(need.value, dev, workspace)
    rho = torch.empty(E, dtype=torch.float64, device=dev)
    nu = torch.empty(E, dtype=torch.float64, device=dev)
    skip = torch.empty(E, dtype=torch.int32, device=dev)
    best = torch.empty(E, dtype=torch.int32, device=dev)
    P = int((eo[1:] - eo[:-1] - 1).sum()) if E > 0 else 0
    pairs = torch.empty((max(P, 1), 2), dtype=torch.int32, device=dev) if want_pairs else None
    _check(L.attt_update_repetition(_dptr(words), tp, _dptr(text_offsets_dev), ep, E, float(tau), _dptr(rho),
                                    _dptr(nu), _dptr(skip), _dptr(best), _dptr(pairs), _dptr(ws), ws.numel(),
                                    _stream_ptr()))
    return rho, nu, skip, best, (pairs[:P] if want_pairs else None)


def ngram_weights_noalloc(history, history_offsets, tokens, token_offsets, n=3, w_min=0.05,
                          want_exposure=True, out=None):
    """ngram_weights through the allocation-free entry point (its scratch is a static device
    buffer of the library). With `out` given, nothing is allocated on this path either."""
    torch = _torch()
    L = load()
    ho, hp = _offsets(history_offsets)
    to, tp = _offsets(token_offsets)
    _dev(tokens, "tokens")
    _dev(history, "history")
    if tokens.dtype != torch.int32 or history.dtype != torch.int32:
        raise TypeError("history and tokens must be int32")
    T = int(to[-1])
    if out is not None:
        f, w = out
    else:
        f = torch.empty(T, dtype=torch.int32, device=tokens.device) if want_exposure else None
        w = torch.empty(T, dtype=torch.float32, device=tokens.device)
    _check(L.attt_ngram_weights_noalloc(_dptr(history), hp, _dptr(tokens), tp, len(ho) - 1, n, float(w_min),
                                        _dptr(f), _dptr(w), _stream_ptr()))
    return f, w


# ------------------------------------------------------------------------------------------
def ngram_set_size(capacity, n):
    """Bytes of one persistent n-gram set holding up to `capacity` distinct n-grams."""
    L = load()
    out = ctypes.c_size_t(0)
    _check(L.attt_ngram_set_size(int(capacity), int(n), ctypes.byref(out)))
    return out.value


def _set_ptrs(sets):
    arr = (ctypes.c_void_p * len(sets))()
    for i, t in enumerate(sets):
        _dev(t, "set")
        arr[i] = t.data_ptr()
    return arr


def ngram_set_init(sets, capacity, n):
    """Empty history for every set (uint8 device tensors of at least ngram_set_size bytes)."""
    L = load()
    nbytes = min(t.numel() * t.element_size() for t in sets)
    _check(L.attt_ngram_set_init(_set_ptrs(sets), len(sets), int(capacity), int(n), nbytes, _stream_ptr()))


def ngram_set_append(sets, tokens, token_offsets, capacity, n):
    """Append text e (tokens[token_offsets[e]:token_offsets[e+1]]) to the history of set e."""
    torch = _torch()
    L = load()
    _dev(tokens, "tokens")
    if tokens.dtype != torch.int32:
        raise TypeError("tokens must be int32")
    to, tp = _offsets(token_offsets)
    if len(to) - 1 != len(sets):
        raise ValueError("one text per set")
    _check(L.attt_ngram_set_append(_set_ptrs(sets), _dptr(tokens), tp, len(sets), int(capacity), int(n),
                                   _stream_ptr()))


def ngram_set_weights(sets, tokens, token_offsets, capacity, n, w_min=0.05, want_exposure=True, out=None):
    """Eq. 8-9 of text e against the history held by set e. Returns (f, w) like ngram_weights."""
    torch = _torch()
    L = load()
    _dev(tokens, "tokens")
    if tokens.dtype != torch.int32:
        raise TypeError("tokens must be int32")
    to, tp = _offsets(token_offsets)
    if len(to) - 1 != len(sets):
        raise ValueError("one text per set")
    T = int(to[-1])
    if out is not None:
        f, w = out
    else:
        f = torch.empty(T, dtype=torch.int32, device=tokens.device) if want_exposure else None
        w = torch.empty(T, dtype=torch.float32, device=tokens.device)
    _check(L.attt_ngram_set_weights(_set_ptrs(sets), _dptr(tokens), tp, len(sets), int(capacity), int(n),
                                    float(w_min), _dptr(f), _dptr(w), _stream_ptr()))
    return f, w


# ------------------------------------------------------------------------------------------
def ce_workspace_size(N, d, V, dtype, want_grad=True, head_t=False):
    L = load()
    out = ctypes.c_size_t(0)
    flags = (CE_WANT_GRAD if want_grad else 0) | (CE_HEAD_T if head_t else 0)
    _check(L.attt_ce_workspace_size(N, d, V, dtype, flags, ctypes.byref(out)))
    return out.value


def ce_set_wait_limit(label_us=20000, exact_us=20000):
    """Bounds of the waits inside the persistent bf16 backward (diagnostics; defaults restore)."""
    _check(load().attt_ce_set_wait_limit(int(label_us), int(exact_us)))


def ce_head_t_size(d, V):
    L = load()
    out = ctypes.c_size_t(0)
    _check(L.attt_ce_head_t_size(int(d), int(V), ctypes.byref(out)))
    return out.value


def ce_head_transpose(lm_head, out=None):
    """The frozen bf16 LM head [V, d] transposed once into the layout the bf16 backward reads
    (uint8 device tensor of ce_head_t_size bytes); pass it as lm_head_t= to weighted_ce_fwd_bwd."""
    torch = _torch()
    L = load()
    _dev(lm_head, "lm_head")
    if lm_head.dtype != torch.bfloat16:
        raise TypeError("the transposed head is for the bf16 backward")
    V, d = lm_head.shape
    nbytes = ce_head_t_size(d, V)
    if out is None:
        out = torch.empty(nbytes, dtype=torch.uint8, device=lm_head.device)
    _dev(out, "out")
    _check(L.attt_ce_head_transpose(_dptr(lm_head), d, V, _dptr(out), out.numel() * out.element_size(),
                                    _stream_ptr()))
    return out


def weighted_ce_fwd_bwd(hidden, lm_head, labels, weights, row_offsets=None, want_grad=True,
                        want_lse=True, workspace=None, out=None, lm_head_t=None):
    """Eq. 10 forward and backward. hidden [N, d], lm_head [V, d] (float32 or bfloat16),
    labels int32 [N], weights float32 [N]; row_offsets: host int64 [E+1] or None (one episode).
    lm_head_t: the head prepared by ce_head_transpose (bf16 backward only) or None.
    Returns (loss [E], lse [N] or None, grad_hidden [N, d] or None)."""
    torch = _torch()
    L = load()
    for t, nm in ((hidden, "hidden"), (lm_head, "lm_head"), (labels, "labels"), (weights, "weights")):
        _dev(t, nm)
    dt = _dtype_code(hidden)
    if lm_head.dtype != hidden.dtype:
        raise TypeError("hidden and lm_head must share a dtype")
    if labels.dtype != torch.int32 or weights.dtype != torch.float32:
        raise TypeError("labels must be int32 and weights float32")
    N, d = hidden.shape
    V = lm_head.shape[0]
    if lm_head.shape[1] != d:
        raise ValueError("lm_head must be [V, d]")
    if row_offsets is None:
        ro, rp, E = None, None, 1
    else:
        ro, rp = _offsets(row_offsets)
        E = len(ro) - 1
    dev = hidden.device
    if out is not None:
        loss, lse, grad = out
    else:
        loss = torch.empty(E, dtype=torch.float32, device=dev)
        lse = torch.empty(N, dtype=torch.float32, device=dev) if want_lse else None
        grad = torch.empty_like(hidden) if want_grad else None
    if lm_head_t is not None:
        _dev(lm_head_t, "lm_head_t")
    need = ctypes.c_size_t(0)
    flags = (CE_WANT_GRAD if grad is not None else 0) | (CE_HEAD_T if lm_head_t is not None else 0)
    _check(L.attt_ce_workspace_size(N, d, V, dt, flags, ctypes.byref(need)))
    ws = _workspace(need.value, dev, workspace)
    _check(L.attt_weighted_ce_fwd_bwd_ex(_dptr(hidden), _dptr(lm_head), _dptr(lm_head_t), _dptr(labels),
                                         _dptr(weights), rp, E, N, d, V, dt, _dptr(loss), _dptr(lse),
                                         _dptr(grad), _dptr(ws), ws.numel(), _stream_ptr()))
    return loss, lse, grad


# ------------------------------------------------------------------------------------------
def _lora_array(problems):
    arr = (LoraProblem * max(len(problems), 1))()
    for i, p in enumerate(problems):
        x, dy, A, B = p["x"], p["dy"], p["A"], p["B"]
        arr[i] = LoraProblem(_dptr(x), _dptr(dy), _dptr(A), _dptr(B), _dptr(p["dA"]), _dptr(p["dB"]),
                             x.shape[0], x.shape[1], dy.shape[1], A.shape[0], float(p["scale"]))
    return arr


def lora_workspace_size(problems, dtype):
    L = load()
    arr = _lora_array(problems)
    out = ctypes.c_size_t(0)
    _check(L.attt_lora_workspace_size(arr, len(problems), dtype, ctypes.byref(out)))
    return out.value


def lora_grad(problems, workspace=None):
    """LoRA dA / dB for a group of projections, accumulated (+=) into each problem's float32
    dA [r, d_in] and dB [d_out, r]. Each problem: dict(x, dy, A, B, dA, dB, scale)."""
    L = load()
    if not problems:
        return
    dt = _dtype_code(problems[0]["x"])
    for p in problems:
        for k in ("x", "dy", "A", "B", "dA", "dB"):
            _dev(p[k], k)
    arr = _lora_array(problems)
    need = ctypes.c_size_t(0)
    _check(L.attt_lora_workspace_size(arr, len(problems), dt, ctypes.byref(need)))
    ws = _workspace(need.value, problems[0]["x"].device, workspace)
    _check(L.attt_lora_grad(arr, len(problems), dt, _dptr(ws), ws.numel(), _stream_ptr()))


def lora_sgd_step(params, lr, zero_grad=False):
    """The adapter step theta <- theta - lr * grad (Eq. 2) on float32 parameters, in place.
    Each entry: dict(param, grad[, param_bf16]) of equal numel; param and grad float32,
    param_bf16 (optional) bfloat16, which receives the updated param rounded to nearest even.
    With zero_grad the gradients are reset to 0 after they are read."""
    L = load()
    torch = _torch()
    arr = (LoraParam * max(len(params), 1))()
    for i, p in enumerate(params):
        P, G, Pb = p["param"], p["grad"], p.get("param_bf16")
        _dev(P, "param")
        _dev(G, "grad")
        if P.dtype != torch.float32 or G.dtype != torch.float32 or G.numel() != P.numel():
            raise ValueError("param and grad must be float32 tensors of equal size")
        if Pb is not None:
            _dev(Pb, "param_bf16")
            if Pb.dtype != torch.bfloat16 or Pb.numel() != P.numel():
                raise ValueError("param_bf16 must be a bfloat16 tensor of the param's size")
        arr[i] = LoraParam(_dptr(P), _dptr(G), _dptr(Pb), P.numel())
    _check(L.attt_lora_sgd_step(arr, len(params), float(lr), 1 if zero_grad else 0, _stream_ptr()))


def lora_forward(problems):
    """Grouped multi-adapter forward: for every problem, y <- RN_bf16(y + scale (x A^T) B^T) in
    place (y already holds the base projection). Each problem: dict(x, y, A, B, scale), bf16
    tensors x [rows, d_in], y [rows, d_out], A [r, d_in], B [d_out, r]."""
    L = load()
    torch = _torch()
    arr = (LoraFwdProblem * max(len(problems), 1))()
    for i, p in enumerate(problems):
        x, y, A, B = p["x"], p["y"], p["A"], p["B"]
        for k, t in (("x", x), ("y", y), ("A", A), ("B", B)):
            _dev(t, k)
            if t.dtype != torch.bfloat16 or t.dim() != 2:
                raise ValueError(f"{k} must be a 2-D bfloat16 tensor")
        arr[i] = LoraFwdProblem(_dptr(x), _dptr(y), _dptr(A), _dptr(B), x.shape[0], x.shape[1], y.shape[1],
                                A.shape[0], float(p["scale"]))
    _check(L.attt_lora_forward(arr, len(problems), _stream_ptr()))


def lora_hot_swap(pairs):
    """Adapter swap into serving: each (src, dst) pair, src a float32 tensor and dst a bfloat16
    tensor of equal numel, gets dst = src rounded to nearest even, all in one launch."""
    L = load()
    torch = _torch()
    arr = (LoraSwapItem * max(len(pairs), 1))()
    for i, (src, dst) in enumerate(pairs):
        _dev(src, "src")
        _dev(dst, "dst")
        if src.dtype != torch.float32 or dst.dtype != torch.bfloat16 or src.numel() != dst.numel():
            raise ValueError("src must be float32 and dst bfloat16 of the same numel")
        arr[i] = LoraSwapItem(_dptr(src), _dptr(dst), src.numel())
    _check(L.attt_lora_hot_swap(arr, len(pairs), _stream_ptr()))


# ------------------------------------------------------------------------------------------
def timing_enable(on=True):
    _check(load().attt_timing_enable(1 if on else 0))


def timing_reset():
    _check(load().attt_timing_reset())


def timing_read(name):
    """(total milliseconds, launches) of one kernel since the last reset."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(load().attt_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def kernel_names():
    L = load()
    out, i = [], 0
    while True:
        nm = L.attt_timing_kernel_name(i)
        if nm is None:
            return out
        out.append(nm.decode())
        i += 1


def version():
    return load().attt_version()
