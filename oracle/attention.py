"""Oracle: backward of one adapted attention block (Sec. 3.1's episode adapter on the q/k/v/o
projections; rank and alpha in Appendix C): the gradients dY_q, dY_k, dY_v of the q, k and v
projection outputs, which are the upstream gradients dy of the LoRA gradient (the step before
the adapter's dA, dB).

Test infrastructure only: the GPU library never imports this module.

The block is standard causal multi-head attention with grouped key/value heads, the form the
paper's models use (the paper states no variant). Readings:
  * Per episode (rows row_offsets[e] .. row_offsets[e+1]-1) an independent causal sequence:
    query t attends to keys s <= t of its own episode.
  * Q [N, H, dh], K and V [N, Hkv, dh]; query head h uses key/value head h // (H / Hkv).
  * S = scale * Q K^T (scale given, 1/sqrt(dh) by default), P = softmax over the allowed keys,
    O = P V. With dO the gradient of O:
        D_t = sum_c dO_tc O_tc,   dP = dO V^T,   dS = P * (dP - D),
        dQ = scale * dS K,   dK = scale * dS^T Q,   dV = P^T dO,
    dK and dV of a key/value head summed over the query heads that share it.
  * Position encoding (if any) is outside: Q and K are the attention's inputs.
Arithmetic in float64 from the inputs' values.
"""
import numpy as np


def _episodes(N, row_offsets):
    if row_offsets is None:
        return [(0, N)]
    off = np.asarray(row_offsets, np.int64)
    return [(int(off[e]), int(off[e + 1])) for e in range(len(off) - 1)]


def attention_fwd_bwd(Q, K, V, dO, row_offsets=None, scale=None):
    """Returns dict(O, lse, D, dQ, dK, dV), float64. Q, dO [N, H, dh]; K, V [N, Hkv, dh];
    lse and D are [H, N]."""
    Q, K, V, dO = (np.asarray(a, np.float64) for a in (Q, K, V, dO))
    N, H, dh = Q.shape
    Hkv = K.shape[1]
    g = H // Hkv
    scale = 1.0 / np.sqrt(dh) if scale is None else float(scale)
    O = np.zeros_like(Q)
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    lse = np.zeros((H, N))
    D = np.zeros((H, N))
    for a, b in _episodes(N, row_offsets):
        L = b - a
        if L == 0:
            continue
        allowed = np.tril(np.ones((L, L), bool))
        for h in range(H):
            kh = h // g
            q, k, v, do = Q[a:b, h], K[a:b, kh], V[a:b, kh], dO[a:b, h]
            S = scale * (q @ k.T)
            S = np.where(allowed, S, -np.inf)
            m = S.max(axis=1, keepdims=True)
            E = np.exp(S - m)
            l = E.sum(axis=1, keepdims=True)
            P = E / l
            o = P @ v
            O[a:b, h] = o
            lse[h, a:b] = (m + np.log(l))[:, 0]
            d = (do * o).sum(axis=1)
            D[h, a:b] = d
            dP = do @ v.T
            dS = P * (dP - d[:, None])
            dQ[a:b, h] = scale * (dS @ k)
            dK[a:b, kh] += scale * (dS.T @ q)
            dV[a:b, kh] += P.T @ do
    return dict(O=O, lse=lse, D=D, dQ=dQ, dK=dK, dV=dV)


def attention_rows(Q, K, V, dO, rows, row_offsets=None, scale=None):
    """dQ, lse and D of the query rows `rows` only (float64), for sampled checks of long
    sequences: each row needs only its own prefix of keys."""
    Q, K, V, dO = (np.asarray(a, np.float64) for a in (Q, K, V, dO))
    N, H, dh = Q.shape
    Hkv = K.shape[1]
    g = H // Hkv
    scale = 1.0 / np.sqrt(dh) if scale is None else float(scale)
    eps = _episodes(N, row_offsets)
    dQ = np.zeros((len(rows), H, dh))
    lse = np.zeros((H, len(rows)))
    D = np.zeros((H, len(rows)))
    for i, t in enumerate(rows):
        a = next(a for a, b in eps if a <= t < b)
        for h in range(H):
            kh = h // g
            k, v = K[a:t + 1, kh], V[a:t + 1, kh]
            s = scale * (k @ Q[t, h])
            m = s.max()
            e = np.exp(s - m)
            p = e / e.sum()
            o = p @ v
            d = float(dO[t, h] @ o)
            dp = v @ dO[t, h]
            ds = p * (dp - d)
            dQ[i, h] = scale * (ds @ k)
            lse[h, i] = m + np.log(e.sum())
            D[h, i] = d
    return dQ, lse, D
