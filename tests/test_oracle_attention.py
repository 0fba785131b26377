"""Pins of the attention-block backward oracle against things other than itself: torch CPU
autograd (float64) of the same attention, central finite differences, closed forms (one key,
keys that carry no information) and the grouped-head equivalence."""
import numpy as np
import pytest
import torch

from oracle import attention as oat


def _rand(N, H, Hkv, dh, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((N, H, dh)), rng.standard_normal((N, Hkv, dh)),
            rng.standard_normal((N, Hkv, dh)), rng.standard_normal((N, H, dh)))


def _torch_grads(Q, K, V, dO, off, scale):
    Qt, Kt, Vt = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (Q, K, V))
    N, H, dh = Q.shape
    g = H // K.shape[1]
    out = []
    for a, b in zip(off[:-1], off[1:]):
        L = b - a
        q = Qt[a:b].transpose(0, 1)                                   # [H, L, dh]
        k = Kt[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        v = Vt[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        s = scale * (q @ k.transpose(1, 2))
        mask = torch.ones(L, L, dtype=torch.bool).tril()
        s = s.masked_fill(~mask, float("-inf"))
        out.append((torch.softmax(s, -1) @ v).transpose(0, 1))
    O = torch.cat(out)
    O.backward(torch.tensor(dO))
    return O.detach().numpy(), Qt.grad.numpy(), Kt.grad.numpy(), Vt.grad.numpy()


@pytest.mark.parametrize("shape", [(7, 2, 1, 4), (12, 4, 2, 8), (9, 3, 3, 5), (20, 8, 2, 16)])
def test_matches_torch_autograd(shape):
    N, H, Hkv, dh = shape
    Q, K, V, dO = _rand(N, H, Hkv, dh, N + H)
    off = np.array([0, N // 3, N], np.int64)
    scale = 0.7 / np.sqrt(dh)
    r = oat.attention_fwd_bwd(Q, K, V, dO, off, scale)
    O, gQ, gK, gV = _torch_grads(Q, K, V, dO, off, scale)
    for a, b in ((r["O"], O), (r["dQ"], gQ), (r["dK"], gK), (r["dV"], gV)):
        assert np.max(np.abs(a - b)) <= 1e-12 * (1 + np.max(np.abs(b)))


def test_finite_differences():
    N, H, Hkv, dh = 6, 2, 1, 3
    Q, K, V, dO = _rand(N, H, Hkv, dh, 5)
    off = np.array([0, N], np.int64)
    r = oat.attention_fwd_bwd(Q, K, V, dO, off)
    loss = lambda q, k, v: float((oat.attention_fwd_bwd(q, k, v, dO, off)["O"] * dO).sum())
    eps = 1e-6
    rng = np.random.default_rng(6)
    for name, X, G in (("Q", Q, r["dQ"]), ("K", K, r["dK"]), ("V", V, r["dV"])):
        for _ in range(6):
            idx = tuple(int(rng.integers(0, s)) for s in X.shape)
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += eps
            Xm[idx] -= eps
            args = {"Q": (Q, K, V), "K": (Q, K, V), "V": (Q, K, V)}[name]
            ap = [Xp if a is X else a for a in args]
            am = [Xm if a is X else a for a in args]
            fd = (loss(*ap) - loss(*am)) / (2 * eps)
            assert abs(fd - G[idx]) <= 1e-6 * (1 + abs(fd)), (name, idx, fd, G[idx])


def test_first_row_has_one_key():
    # the first query of an episode sees only its own key: O = V, dQ = 0, its dV row gets dO
    Q, K, V, dO = _rand(5, 2, 2, 4, 7)
    r = oat.attention_fwd_bwd(Q, K, V, dO, [0, 1, 5])
    assert np.allclose(r["O"][0], V[0]) and np.allclose(r["dQ"][0], 0)
    assert np.allclose(r["dV"][0], dO[0])  # no later query of episode 0 uses key 0
    assert np.allclose(r["lse"][:, 0], (Q[0] * K[0]).sum(-1) / 2.0)


def test_uniform_attention_closed_form():
    # K = 0: every allowed key scores 0, so P is uniform over the prefix, O_t = mean(V_0..t),
    # lse_t = log(t + 1), dV_s = sum_{t >= s} dO_t / (t + 1), and dQ = scale dS K = 0
    N, dh = 8, 4
    rng = np.random.default_rng(8)
    Q = rng.standard_normal((N, 1, dh))
    K = np.zeros((N, 1, dh))
    V = rng.standard_normal((N, 1, dh))
    dO = rng.standard_normal((N, 1, dh))
    r = oat.attention_fwd_bwd(Q, K, V, dO)
    for t in range(N):
        assert np.allclose(r["O"][t, 0], V[: t + 1, 0].mean(0))
        assert np.isclose(r["lse"][0, t], np.log(t + 1))
    for s in range(N):
        assert np.allclose(r["dV"][s, 0], sum(dO[t, 0] / (t + 1) for t in range(s, N)))
    assert np.allclose(r["dQ"], 0)  # dQ = scale dS K = 0 with K = 0


def test_grouped_heads_equal_repeated_heads():
    N, H, Hkv, dh = 10, 4, 2, 6
    Q, K, V, dO = _rand(N, H, Hkv, dh, 9)
    off = [0, 4, 10]
    r = oat.attention_fwd_bwd(Q, K, V, dO, off)
    Kr, Vr = np.repeat(K, 2, axis=1), np.repeat(V, 2, axis=1)
    m = oat.attention_fwd_bwd(Q, Kr, Vr, dO, off)
    assert np.allclose(r["dQ"], m["dQ"]) and np.allclose(r["O"], m["O"])
    assert np.allclose(r["dK"], m["dK"][:, 0::2] + m["dK"][:, 1::2])
    assert np.allclose(r["dV"], m["dV"][:, 0::2] + m["dV"][:, 1::2])


def test_rows_helper_matches_full():
    N, H, Hkv, dh = 15, 4, 1, 8
    Q, K, V, dO = _rand(N, H, Hkv, dh, 10)
    off = [0, 6, 15]
    r = oat.attention_fwd_bwd(Q, K, V, dO, off)
    rows = [0, 3, 5, 6, 11, 14]
    dQ, lse, D = oat.attention_rows(Q, K, V, dO, rows, off)
    assert np.allclose(dQ, r["dQ"][rows]) and np.allclose(lse, r["lse"][:, rows]) and np.allclose(D, r["D"][:, rows])
