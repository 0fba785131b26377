"""GPU parity of the adapted attention block's backward (dY_q = dQ, dY_k = dK, dY_v = dV; the
upstream gradients of the q/k/v LoRA gradient) against the float64 oracle, on the same bf16
inputs: every row's cosine >= 0.999 and every element within 2^-7 (|ref| + rms of its row),
lse and D (the forward statistics the kernels also return) to float32 accuracy.

Shapes: small ragged episodes (one-row episode, exact and partial 64-row blocks), grouped-head
ratios 1, 2, 4 and 8, the small workload's shape (2048 rows, 16 heads over 4 key/value heads)
in full, the Llama-8B shape (8192 rows, 32 heads over 8) with the oracle on one key/value
group, and 16 episodes of 4096 rows with the oracle on two episodes."""
import numpy as np
import pytest

from gpu_util import check_rows, cosine, dev_dense, host, note
from oracle import attention as oat
from workloads.gen import random_dense

pytestmark = pytest.mark.gpu
DH = 128
BF16_COS = 0.999
BF16_ELEM = 2.0 ** -7


def _inputs(N, H, Hkv, seed):
    q = random_dense((N, H, DH), 1.0, True, seed)
    k = random_dense((N, Hkv, DH), 1.0, True, seed + 1)
    v = random_dense((N, Hkv, DH), 1.0, True, seed + 2)
    do = random_dense((N, H, DH), 0.05, True, seed + 3)
    return q, k, v, do


def _gpu(attt, q, k, v, do, off):
    dq, dk, dv, lse, dsum = attt.attention_bwd(dev_dense(q), dev_dense(k), dev_dense(v), dev_dense(do), row_offsets=off)
    return host(dq), host(dk), host(dv), lse.cpu().numpy(), dsum.cpu().numpy()


def _cmp(name, got, want):
    g2, w2 = got.reshape(got.shape[0], -1), want.reshape(want.shape[0], -1)
    live = np.linalg.norm(w2, axis=1) > 0
    assert cosine(g2, w2) >= BF16_COS, name
    check_rows(g2[live], w2[live], BF16_COS, BF16_ELEM, name)
    # rows whose exact gradient is 0 (an episode's first query: one key, so dS = 0; a key no later
    # query of its episode sees) are negligible against the tensor's scale: dP and D round in
    # different orders, so dP - D is tiny but not always exactly 0
    if np.any(~live):
        assert np.max(np.abs(g2[~live])) <= BF16_ELEM * np.sqrt(np.mean(w2 ** 2)), name


def _check_full(attt, N, H, Hkv, off, seed):
    q, k, v, do = _inputs(N, H, Hkv, seed)
    dq, dk, dv, lse, dsum = _gpu(attt, q, k, v, do, off)
    r = oat.attention_fwd_bwd(q.f32, k.f32, v.f32, do.f32, off)
    _cmp("dQ", dq, r["dQ"])
    _cmp("dK", dk, r["dK"])
    _cmp("dV", dv, r["dV"])
    assert np.max(np.abs(lse - r["lse"])) <= 1e-4 * (1 + np.max(np.abs(r["lse"])))
    assert np.max(np.abs(dsum - r["D"])) <= 1e-3 * (1e-6 + np.sqrt(np.mean(r["D"] ** 2)))


@pytest.mark.parametrize("H,Hkv", [(4, 4), (4, 2), (8, 2), (8, 1)])
def test_small_ragged(attt, H, Hkv):
    off = np.array([0, 1, 65, 129, 200, 264, 300], np.int64)
    note(f"attention small ragged: heads {H}/{Hkv}, episodes {np.diff(off).tolist()}")
    _check_full(attt, int(off[-1]), H, Hkv, off, 11 + H + Hkv)


def test_single_episode_no_offsets(attt):
    q, k, v, do = _inputs(130, 2, 1, 21)
    dq, dk, dv, lse, dsum = _gpu(attt, q, k, v, do, None)
    r = oat.attention_fwd_bwd(q.f32, k.f32, v.f32, do.f32, None)
    _cmp("dQ", dq, r["dQ"])
    _cmp("dK", dk, r["dK"])
    _cmp("dV", dv, r["dV"])


def test_small_workload_shape(attt):
    note("attention 2048 rows, 16/4 heads")
    _check_full(attt, 2048, 16, 4, np.array([0, 2048], np.int64), 31)


def test_llama8b_shape_one_group(attt):
    N, H, Hkv, g = 8192, 32, 8, 4
    q, k, v, do = _inputs(N, H, Hkv, 41)
    note("attention 8192 rows, 32/8 heads (oracle: key/value head 3 and its 4 query heads)")
    dq, dk, dv, lse, dsum = _gpu(attt, q, k, v, do, None)
    kh = 3
    sl = slice(kh * g, (kh + 1) * g)
    r = oat.attention_fwd_bwd(q.f32[:, sl], k.f32[:, kh:kh + 1], v.f32[:, kh:kh + 1], do.f32[:, sl], None)
    _cmp("dQ", dq[:, sl], r["dQ"])
    _cmp("dK", dk[:, kh:kh + 1], r["dK"])
    _cmp("dV", dv[:, kh:kh + 1], r["dV"])
    assert np.max(np.abs(lse[sl] - r["lse"])) <= 1e-4 * (1 + np.max(np.abs(r["lse"])))


def test_many_episodes_two_checked(attt):
    E, Lr, H, Hkv = 16, 4096, 8, 2
    off = np.arange(E + 1, dtype=np.int64) * Lr
    q, k, v, do = _inputs(E * Lr, H, Hkv, 51)
    note("attention 16 episodes x 4096 rows, 8/2 heads (oracle on episodes 0 and 15)")
    dq, dk, dv, lse, dsum = _gpu(attt, q, k, v, do, off)
    for e in (0, E - 1):
        rs = slice(off[e], off[e + 1])
        r = oat.attention_fwd_bwd(q.f32[rs], k.f32[rs], v.f32[rs], do.f32[rs], None)
        _cmp(f"dQ ep{e}", dq[rs], r["dQ"])
        _cmp(f"dK ep{e}", dk[rs], r["dK"])
        _cmp(f"dV ep{e}", dv[rs], r["dV"])


def test_deterministic(attt):
    q, k, v, do = _inputs(1000, 8, 2, 61)
    off = np.array([0, 300, 1000], np.int64)
    a = _gpu(attt, q, k, v, do, off)
    b = _gpu(attt, q, k, v, do, off)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()
