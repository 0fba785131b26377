"""Oracle: token-weighted next-token cross-entropy through a frozen LM head (Sec. 3.3,
Eq. 10; the gradient step of Algorithm 1), forward and backward with respect to the hidden states.

Test infrastructure only: the GPU library never imports this module.

Readings of the paper taken here:
  * Eq. 10 normalises by L, the number of scored tokens of the update, not by the sum
    of the weights. With several episodes in one call, episode e has its own L_e (its
    row count) and its own loss.
  * Row t is the hidden state that predicts token x_t: its label is x_t and its weight
    is w_t, the weight of the target token (Eq. 10 pairs w_{k,j} with CE at x_{k,j}).
  * CE is the natural-log softmax cross-entropy over the full vocabulary, temperature
    1, no label smoothing, no bias. The LM head is frozen, so only dH is produced.
Everything is computed in float64 from the exact input values.

    z = h W^T,  lse_t = max_v z_tv + log sum_v exp(z_tv - max_v z_tv)
    CE_t = lse_t - z_{t, y_t},  loss_e = (1 / L_e) sum_{t in e} w_t CE_t
    dZ_t = (w_t / L_e) (softmax(z_t) - onehot(y_t)),  dH = dZ W
"""
import numpy as np


def episode_of_rows(row_offsets, N):
    off = np.asarray(row_offsets, np.int64)
    ep = np.searchsorted(off, np.arange(N), side="right") - 1
    return ep, np.diff(off)


def _rows_fwd_bwd(h_rows, W64, labels, coef, want_grad):
    z = np.asarray(h_rows, np.float64) @ W64.T
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    idx = np.arange(z.shape[0])
    ce = lse - z[idx, labels]
    dh = None
    if want_grad:
        p = np.exp(z - lse[:, None])
        p[idx, labels] -= 1.0
        p *= coef[:, None]
        dh = p @ W64
    return lse, ce, dh


def weighted_ce(h, W, labels, weights, row_offsets=None, want_grad=True, chunk=256):
    """Full forward/backward. Returns (loss [E], lse [N], dH [N, d] or None), float64."""
    h = np.asarray(h)
    N = h.shape[0]
    if row_offsets is None:
        row_offsets = np.array([0, N], np.int64)
    ep, lens = episode_of_rows(row_offsets, N)
    W64 = np.asarray(W, np.float64)
    w64 = np.asarray(weights, np.float64)
    labels = np.asarray(labels, np.int64)
    coef = w64 / lens[ep] if N else w64
    lse = np.empty(N, np.float64)
    ce = np.empty(N, np.float64)
    dH = np.empty((N, W64.shape[1]), np.float64) if want_grad else None
    for s in range(0, N, chunk):
        e = min(N, s + chunk)
        l_, c_, d_ = _rows_fwd_bwd(h[s:e], W64, labels[s:e], coef[s:e], want_grad)
        lse[s:e] = l_
        ce[s:e] = c_
        if want_grad:
            dH[s:e] = d_
    E = len(lens)
    loss = np.zeros(E, np.float64)
    for e_ in range(E):
        a, b = int(row_offsets[e_]), int(row_offsets[e_ + 1])
        if b > a:
            loss[e_] = np.sum(w64[a:b] * ce[a:b]) / (b - a)
    return loss, lse, dH


def ce_rows(h, W64, labels, weights, row_offsets, rows):
    """Forward/backward for selected rows only (any problem size). W64 must be the
    float64 LM head. Returns (lse [k], ce [k], dH [k, d]) for those rows."""
    rows = np.asarray(rows, np.int64)
    N = np.asarray(h).shape[0]
    ep, lens = episode_of_rows(row_offsets, N)
    coef = np.asarray(weights, np.float64)[rows] / lens[ep[rows]]
    return _rows_fwd_bwd(np.asarray(h)[rows], W64, np.asarray(labels, np.int64)[rows], coef, True)


def weighted_ce_loss(h, W, labels, weights, row_offsets=None):
    loss, _, _ = weighted_ce(h, W, labels, weights, row_offsets, want_grad=False)
    return loss
