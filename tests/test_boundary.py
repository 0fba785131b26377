"""The C-ABI boundary without a GPU: the library loads, exports every function the header
declares, and rejects invalid arguments on the host (before any HIP call) with the
documented status codes. No call here reaches a kernel launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_03441_amd as attt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attt.h")
FAKE = ctypes.c_void_p(0x7F0000000000)        # never dereferenced: validation fails first
FAKE_WS = ctypes.c_void_p(0x7F0000001000)      # 256-byte aligned


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(attt.lib_path()):
        pytest.fail("libattt.so is not built; run __graft_entry__.build()")
    return attt.load()


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"\b(attt_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_three_calls():
    names = _declared()
    for n in ("attt_ngram_weights", "attt_weighted_ce_fwd_bwd", "attt_lora_grad",
              "attt_ngram_workspace_size", "attt_ce_workspace_size", "attt_lora_workspace_size"):
        assert n in names


def test_every_declared_symbol_is_exported(L):
    missing = [n for n in _declared() if not hasattr(L, n)]
    assert not missing, missing


def test_status_strings_and_version(L):
    assert L.attt_status_string(0) == b"ok"
    assert L.attt_status_string(2) == b"workspace too small"
    assert L.attt_version() >= 100
    names = attt.kernel_names()
    assert "ce_fwd_lse" in names and "ngram_count" in names and "lora_dadb" in names


def _off(a):
    arr = np.asarray(a, np.int64)
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _ngram(L, hoff, toff, n=3, w_min=0.05, ws=FAKE_WS, ws_bytes=1 << 30):
    _, hp = _off(hoff)
    _, tp = _off(toff)
    return L.attt_ngram_weights(FAKE, hp, FAKE, tp, len(hoff) - 1, n, w_min, None, FAKE, ws, ws_bytes, None)


def test_ngram_validation(L):
    assert _ngram(L, [0, 10], [0, 5], n=0) == attt.EINVAL
    assert _ngram(L, [0, 10], [0, 5], n=17) == attt.EINVAL
    assert b"n must be" in L.attt_last_error()
    assert _ngram(L, [0, 10], [0, 5], w_min=0.0) == attt.EINVAL
    assert _ngram(L, [0, 10], [0, 5], w_min=1.5) == attt.EINVAL
    assert _ngram(L, [0, 10], [0, 5], w_min=float("nan")) == attt.EINVAL
    assert _ngram(L, [0, 10, 4], [0, 5, 6]) == attt.EINVAL          # decreasing
    assert _ngram(L, [1, 10], [0, 5]) == attt.EINVAL                # must start at 0
    assert _ngram(L, [0, 10], [0, 5], ws_bytes=8) == attt.ENOSPACE
    assert _ngram(L, [0, 10], [0, 5], ws=ctypes.c_void_p(0x7F0000001010)) == attt.EINVAL
    _, hp = _off([0, 10])
    _, tp = _off([0, 5])
    assert L.attt_ngram_weights(FAKE, hp, FAKE, tp, 0, 3, 0.05, None, FAKE, FAKE_WS, 1 << 30, None) == attt.EINVAL


def test_ngram_workspace_size_grows_with_update_length():
    small = attt.ngram_workspace_size([0, 100], [0, 64], 3)
    big = attt.ngram_workspace_size([0, 100], [0, 20000], 3)
    multi = attt.ngram_workspace_size([0, 100, 200], [0, 20000, 40000], 3)
    assert 0 < small < big < multi
    assert small % 256 == 0 and big % 256 == 0
    with pytest.raises(attt.AtttError):
        attt.ngram_workspace_size([0, 100], [0, 64], 0)


def _ce(L, N=16, d=64, V=100, dtype=1, E=1, off=(0, 16), loss=FAKE, hidden=FAKE, ws_bytes=1 << 40,
        grad=FAKE):
    _, op = _off(off) if off is not None else (None, None)
    return L.attt_weighted_ce_fwd_bwd(hidden, FAKE, FAKE, FAKE, op, E, N, d, V, dtype, loss, None, grad,
                                      FAKE_WS, ws_bytes, None)


def test_ce_validation(L):
    assert _ce(L, d=60) == attt.EINVAL                    # d % 8
    assert _ce(L, dtype=7) == attt.EINVAL
    assert _ce(L, V=0) == attt.EINVAL
    assert _ce(L, off=(0, 15)) == attt.EINVAL             # offsets must end at N
    assert _ce(L, E=2, off=None) == attt.EINVAL           # NULL offsets only for one episode
    assert _ce(L, E=2, off=(0, 9, 8)) == attt.EINVAL      # decreasing
    assert _ce(L, loss=None) == attt.EINVAL
    assert _ce(L, hidden=ctypes.c_void_p(0x7F0000000008)) == attt.EINVAL   # misaligned
    assert _ce(L, ws_bytes=100) == attt.ENOSPACE


def test_ce_workspace_sizes():
    fwd = attt.ce_workspace_size(8192, 4096, 128256, attt.BF16, want_grad=False)
    bwd = attt.ce_workspace_size(8192, 4096, 128256, attt.BF16, want_grad=True)
    assert 0 < fwd < bwd
    # the backward stages one bounded block of rows x vocab columns, never the full N x V
    # gradient: past the row block, more rows add only a few bytes per row
    fwd8 = attt.ce_workspace_size(8 * 8192, 4096, 128256, attt.BF16, want_grad=False)
    bwd8 = attt.ce_workspace_size(8 * 8192, 4096, 128256, attt.BF16, want_grad=True)
    assert bwd8 - fwd8 < 8 * 8192 * 128256 * 2 // 4
    assert (bwd8 - fwd8) - (bwd - fwd) <= 16 * 7 * 8192
    assert attt.ce_workspace_size(4, 8, 3, attt.F32) >= 256


def _lora(L, **kw):
    p = dict(x=FAKE, dy=FAKE, A=FAKE, B=FAKE, dA=FAKE, dB=FAKE, rows=32, d_in=64, d_out=64, rank=8,
             scale=2.0)
    p.update(kw)
    arr = (attt.LoraProblem * 1)(attt.LoraProblem(**p))
    return L.attt_lora_grad(arr, 1, attt.BF16, FAKE_WS, 1 << 30, None)


def test_lora_validation(L):
    assert _lora(L, rank=0) == attt.EINVAL
    assert _lora(L, rank=65) == attt.EINVAL
    assert _lora(L, d_in=60) == attt.EINVAL
    assert _lora(L, d_out=0) == attt.EINVAL
    assert _lora(L, dA=None) == attt.EINVAL
    assert _lora(L, x=ctypes.c_void_p(0x7F0000000004)) == attt.EINVAL
    assert _lora(L, scale=float("inf")) == attt.EINVAL
    arr = (attt.LoraProblem * 1)()
    assert L.attt_lora_grad(arr, 1, 5, FAKE_WS, 1 << 30, None) == attt.EINVAL


def _sgd(L, count=1, lr=0.5, **kw):
    p = dict(param=FAKE, grad=ctypes.c_void_p(0x7F0000001000), param_bf16=None, n=100)
    p.update(kw)
    arr = (attt.LoraParam * 1)(attt.LoraParam(**p))
    return L.attt_lora_sgd_step(arr, count, lr, 1, None)


def test_lora_sgd_validation(L):
    assert _sgd(L, lr=float("inf")) == attt.EINVAL
    assert _sgd(L, lr=float("nan")) == attt.EINVAL
    assert _sgd(L, count=-1) == attt.EINVAL
    assert _sgd(L, n=-1) == attt.EINVAL
    assert _sgd(L, param=None) == attt.EINVAL
    assert _sgd(L, grad=None) == attt.EINVAL
    assert _sgd(L, param=ctypes.c_void_p(0x7F0000000002)) == attt.EINVAL
    assert _sgd(L, param_bf16=ctypes.c_void_p(0x7F0000000003)) == attt.EINVAL
    assert _sgd(L, n=1 << 31) == attt.EUNSUPPORTED
    assert L.attt_lora_sgd_step(None, 1, 0.5, 0, None) == attt.EINVAL
    # nothing to do: no launch, no device access
    assert _sgd(L, param=None, grad=None, n=0) == attt.OK
    assert L.attt_lora_sgd_step(None, 0, 0.5, 0, None) == attt.OK


def test_timing_api_without_launches(L):
    attt.timing_reset()
    assert attt.timing_read("ce_fwd_lse") == (0.0, 0)
    with pytest.raises(attt.AtttError):
        attt.timing_read("no_such_kernel")


# ---- persistent n-gram sets ------------------------------------------------------------
def _sets(*ptrs):
    arr = (ctypes.c_void_p * len(ptrs))()
    for i, p in enumerate(ptrs):
        arr[i] = p
    return arr


def test_ngram_set_size(L):
    out = ctypes.c_size_t(0)
    assert L.attt_ngram_set_size(1000, 4, ctypes.byref(out)) == attt.OK
    # 2048 slot records (8-byte key, 4-byte count, four 4-byte tokens: 28 -> 32 bytes) after a
    # 256-byte header
    assert out.value == 256 + 2048 * 32
    assert L.attt_ngram_set_size(1024, 4, ctypes.byref(out)) == attt.OK
    assert out.value == 256 + 2048 * 32                  # load factor exactly 1/2 still fits
    assert L.attt_ngram_set_size(1025, 4, ctypes.byref(out)) == attt.OK
    assert out.value == 256 + 4096 * 32
    assert L.attt_ngram_set_size(1000, 16, ctypes.byref(out)) == attt.OK
    assert out.value == 256 + 2048 * 80                  # 12 + 64 bytes -> 80
    assert L.attt_ngram_set_size(0, 4, ctypes.byref(out)) == attt.EINVAL
    assert L.attt_ngram_set_size(1 << 31, 4, ctypes.byref(out)) == attt.EINVAL
    assert L.attt_ngram_set_size(10, 17, ctypes.byref(out)) == attt.EINVAL
    assert L.attt_ngram_set_size(10, 3, None) == attt.EINVAL


def test_ngram_set_validation(L):
    s = _sets(FAKE_WS)
    big = 1 << 30
    assert L.attt_ngram_set_init(s, 0, 100, 3, big, None) == attt.EINVAL
    assert L.attt_ngram_set_init(s, 1, 100, 0, big, None) == attt.EINVAL
    assert L.attt_ngram_set_init(s, 1, 0, 3, big, None) == attt.EINVAL
    assert L.attt_ngram_set_init(_sets(None), 1, 100, 3, big, None) == attt.EINVAL
    assert L.attt_ngram_set_init(_sets(ctypes.c_void_p(0x7F0000001010)), 1, 100, 3, big, None) == attt.EINVAL
    assert b"aligned" in L.attt_last_error()
    need = ctypes.c_size_t(0)
    assert L.attt_ngram_set_size(100, 3, ctypes.byref(need)) == attt.OK
    assert L.attt_ngram_set_init(s, 1, 100, 3, need.value - 1, None) == attt.ENOSPACE
    _, tp = _off([0, 5])
    _, bad = _off([0, 5, 3])
    assert L.attt_ngram_set_append(s, FAKE, bad, 2, 100, 3, None) == attt.EINVAL
    assert L.attt_ngram_set_append(s, None, tp, 1, 100, 3, None) == attt.EINVAL
    assert L.attt_ngram_set_weights(s, FAKE, tp, 1, 100, 3, 0.0, None, FAKE, None) == attt.EINVAL
    assert L.attt_ngram_set_weights(s, FAKE, tp, 1, 100, 3, 0.05, None, None, None) == attt.EINVAL
    assert b"weights is null" in L.attt_last_error()


def test_ce_limits_and_flags(L):
    # the bf16 backward's transposed head is read through a 1 GiB descriptor: V <= 2^21 - 256
    assert _ce(L, V=(1 << 21) - 255) == attt.EUNSUPPORTED
    assert b"V <=" in L.attt_last_error()
    out = ctypes.c_size_t(0)
    assert L.attt_ce_workspace_size(16, 64, (1 << 21) - 255, attt.BF16, 1, ctypes.byref(out)) == attt.EUNSUPPORTED
    assert L.attt_ce_workspace_size(16, 64, (1 << 21) - 255, attt.BF16, 0, ctypes.byref(out)) == attt.OK
    assert L.attt_ce_workspace_size(16, 64, 100, attt.BF16, 4, ctypes.byref(out)) == attt.EINVAL


def test_ce_prepared_head(L):
    d, V = 4096, 128256
    assert attt.ce_head_t_size(d, V) == d * 128256 * 2            # V is already a multiple of 256
    assert attt.ce_head_t_size(64, 1000) == 64 * 1024 * 2
    with_t = attt.ce_workspace_size(8192, d, V, attt.BF16, want_grad=True, head_t=True)
    plain = attt.ce_workspace_size(8192, d, V, attt.BF16, want_grad=True)
    assert plain - with_t == d * 128256 * 2                       # the per-call copy is gone
    FAKE_T = ctypes.c_void_p(0x7F0000002000)
    assert L.attt_ce_head_transpose(None, 64, 100, FAKE_T, 1 << 20, None) == attt.EINVAL
    assert L.attt_ce_head_transpose(FAKE, 64, 100, ctypes.c_void_p(0x7F0000002008), 1 << 20, None) == attt.EINVAL
    assert L.attt_ce_head_transpose(FAKE, 64, 100, FAKE_T, 64 * 256 * 2 - 1, None) == attt.ENOSPACE
    assert L.attt_ce_head_transpose(FAKE, 60, 100, FAKE_T, 1 << 20, None) == attt.EINVAL
    _, op = _off((0, 16))
    # a prepared head only applies to the bf16 backward
    assert L.attt_weighted_ce_fwd_bwd_ex(FAKE, FAKE, FAKE_T, FAKE, FAKE, op, 1, 16, 64, 100, attt.F32, FAKE,
                                         None, FAKE, FAKE_WS, 1 << 40, None) == attt.EINVAL
    assert L.attt_weighted_ce_fwd_bwd_ex(FAKE, FAKE, FAKE_T, FAKE, FAKE, op, 1, 16, 64, 100, attt.BF16, FAKE,
                                         None, None, FAKE_WS, 1 << 40, None) == attt.EINVAL
    assert L.attt_weighted_ce_fwd_bwd_ex(FAKE, FAKE, ctypes.c_void_p(0x7F0000002004), FAKE, FAKE, op, 1, 16, 64,
                                         100, attt.BF16, FAKE, None, FAKE, FAKE_WS, 1 << 40, None) == attt.EINVAL


def test_lora_row_limit(L):
    # pass 2 addresses a rank tile's [16, rows_pad] operand through one 32-bit descriptor
    assert _lora(L, rows=1 << 24) == attt.EUNSUPPORTED
    assert b"rows < 2^24" in L.attt_last_error()


def test_ngram_noalloc_validation(L):
    _, hp = _off([0, 10])
    _, tp = _off([0, 5])
    assert L.attt_ngram_weights_noalloc(FAKE, hp, FAKE, tp, 1, 0, 0.05, None, FAKE, None) == attt.EINVAL
    assert L.attt_ngram_weights_noalloc(FAKE, hp, FAKE, tp, 1, 3, 0.0, None, FAKE, None) == attt.EINVAL
    assert L.attt_ngram_weights_noalloc(FAKE, hp, FAKE, tp, 1, 3, 0.05, None, None, None) == attt.EINVAL
    # a call whose partial counts exceed the static scratch is refused before any HIP call:
    # 64 episodes of 40 partitions (4096 update n-grams each) with at least one history chunk
    # each give 2560 rows of 8 KiB
    E = 64
    hoff = np.arange(E + 1, dtype=np.int64) * 3000
    toff = np.arange(E + 1, dtype=np.int64) * 40 * 4096
    need = attt.ngram_workspace_size(hoff, toff, 3)
    assert need > (16 << 20)
    _, hp2 = _off(hoff)
    _, tp2 = _off(toff)
    assert L.attt_ngram_weights_noalloc(FAKE, hp2, FAKE, tp2, E, 3, 0.05, None, FAKE, None) == attt.EUNSUPPORTED
    assert b"static" in L.attt_last_error()


def test_ce_wait_limit_validation(L):
    assert L.attt_ce_set_wait_limit(-1, 10) == attt.EINVAL
    assert L.attt_ce_set_wait_limit(10, -1) == attt.EINVAL
    assert L.attt_ce_set_wait_limit(20000, 20000) == attt.OK


def _rep(L, toff, etx, E=None, tau=0.5, outs=True, ws_bytes=1 << 30, words=FAKE, toff_dev=FAKE):
    _, tp = _off(toff)
    _, ep = _off(etx)
    E = len(etx) - 1 if E is None else E
    o = FAKE if outs else None
    return L.attt_update_repetition(words, tp, toff_dev, ep, E, tau, o, o, o, o, None, FAKE_WS, ws_bytes, None)


def test_repetition_validation(L):
    # two episodes: texts 0-1 and 2; words 0..9
    toff, etx = [0, 4, 7, 10], [0, 2, 3]
    need = attt.repetition_workspace_size(toff, etx)
    assert need >= 256 and need % 256 == 0
    assert _rep(L, toff, etx, E=0) == attt.EINVAL
    assert _rep(L, toff, [0, 0, 3]) == attt.EINVAL            # an episode without text
    assert _rep(L, toff, [1, 2, 3]) == attt.EINVAL            # episode_texts[0] != 0
    assert _rep(L, [0, 4, 3, 10], etx) == attt.EINVAL         # text offsets decrease
    assert _rep(L, [1, 4, 7, 10], etx) == attt.EINVAL         # text_offsets[0] != 0
    assert _rep(L, toff, etx, tau=float("nan")) == attt.EINVAL
    assert _rep(L, toff, etx, tau=float("inf")) == attt.EINVAL
    assert _rep(L, toff, etx, outs=False) == attt.EINVAL
    assert _rep(L, toff, etx, toff_dev=None) == attt.EINVAL
    assert _rep(L, toff, etx, words=None) == attt.EINVAL
    assert _rep(L, toff, etx, ws_bytes=need - 1) == attt.ENOSPACE
    # a text longer than 2^20 words is refused from the offsets alone
    assert _rep(L, [0, (1 << 20) + 1], [0, 1]) == attt.EUNSUPPORTED
    assert b"2^20" in L.attt_last_error()
    # one record per (pair, partition): 2^26 of them at most. A 2^20-word candidate takes 256
    # partitions, so 2^18 + 1 (empty) previous texts exceed it.
    T = (1 << 18) + 2
    toff2 = np.zeros(T + 1, dtype=np.int64)
    toff2[-1] = 1 << 20
    assert _rep(L, toff2, [0, T]) == attt.EUNSUPPORTED
    assert b"2^26" in L.attt_last_error()


def _attn(L, N=64, H=4, Hkv=2, dh=128, scale=0.088, off=None, E=1, ptr=FAKE):
    op = None
    if off is not None:
        _, op = _off(off)
        E = len(off) - 1
    p = ptr
    return L.attt_attention_bwd(p, p, p, p, op, E, N, H, Hkv, dh, scale, p, p, p, p, p, None)


def test_attention_validation(L):
    assert _attn(L, dh=64) == attt.EUNSUPPORTED
    assert _attn(L, H=6, Hkv=4) == attt.EINVAL
    assert _attn(L, Hkv=0) == attt.EINVAL
    assert _attn(L, scale=0.0) == attt.EINVAL
    assert _attn(L, scale=float("nan")) == attt.EINVAL
    assert _attn(L, N=-1) == attt.EINVAL
    assert _attn(L, N=1, H=1 << 16, Hkv=1) == attt.EUNSUPPORTED   # a block's byte range must stay < 2^30
    assert _attn(L, E=2) == attt.EINVAL                       # NULL offsets need one episode
    assert _attn(L, off=[0, 10, 60]) == attt.EINVAL           # offsets end != N
    assert _attn(L, off=[0, 40, 30, 64]) == attt.EINVAL       # decreasing
    assert _attn(L, ptr=None) == attt.EINVAL
    assert _attn(L, ptr=ctypes.c_void_p(0x7F0000000008)) == attt.EINVAL  # misaligned
    assert _attn(L, N=1 << 29, H=8, Hkv=8) == attt.EUNSUPPORTED
    assert _attn(L, N=0, off=[0, 0]) == attt.OK               # nothing to do, nothing touched


def _fwd(L, count=1, **kw):
    p = dict(x=FAKE, y=FAKE_WS, A=FAKE, B=FAKE_WS, rows=32, d_in=64, d_out=64, rank=8, scale=2.0)
    p.update(kw)
    arr = (attt.LoraFwdProblem * 1)(attt.LoraFwdProblem(**p))
    return L.attt_lora_forward(arr, count, None)


def test_lora_forward_validation(L):
    assert _fwd(L, rank=0) == attt.EINVAL
    assert _fwd(L, rank=65) == attt.EINVAL
    assert _fwd(L, d_in=60) == attt.EINVAL
    assert _fwd(L, d_out=0) == attt.EINVAL
    assert _fwd(L, rows=-1) == attt.EINVAL
    assert _fwd(L, y=None) == attt.EINVAL
    assert _fwd(L, B=ctypes.c_void_p(0x7F0000000008)) == attt.EINVAL
    assert _fwd(L, scale=float("nan")) == attt.EINVAL
    assert _fwd(L, rows=1 << 24) == attt.EUNSUPPORTED
    assert _fwd(L, d_in=1 << 20) == attt.EUNSUPPORTED
    assert _fwd(L, count=-1) == attt.EINVAL
    assert L.attt_lora_forward(None, 1, None) == attt.EINVAL
    # nothing to do: no launch
    assert _fwd(L, rows=0, x=None, y=None, A=None, B=None) == attt.OK
    assert L.attt_lora_forward(None, 0, None) == attt.OK


def _swap(L, count=1, **kw):
    p = dict(src=FAKE, dst=FAKE_WS, n=100)
    p.update(kw)
    arr = (attt.LoraSwapItem * 1)(attt.LoraSwapItem(**p))
    return L.attt_lora_hot_swap(arr, count, None)


def test_lora_hot_swap_validation(L):
    assert _swap(L, n=-1) == attt.EINVAL
    assert _swap(L, src=None) == attt.EINVAL
    assert _swap(L, dst=None) == attt.EINVAL
    assert _swap(L, src=ctypes.c_void_p(0x7F0000000002)) == attt.EINVAL
    assert _swap(L, dst=ctypes.c_void_p(0x7F0000000001)) == attt.EINVAL
    assert _swap(L, n=1 << 31) == attt.EUNSUPPORTED
    assert _swap(L, count=-1) == attt.EINVAL
    assert L.attt_lora_hot_swap(None, 1, None) == attt.EINVAL
    assert _swap(L, src=None, dst=None, n=0) == attt.OK
