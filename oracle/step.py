"""Oracle: one aTTT update step (Algorithm 1: the weighting loop and the gradient of the weighted loss), the three parts chained.

Test infrastructure only: the GPU library never imports this module.

  f, w  = n-gram exposure and weights of x_k against H^tok_k      (Eq. 8-9)
  loss, dH = weighted CE of the LM head on the update rows         (Eq. 10)
  dA, dB for every adapted projection; the output projection "o"
  takes dH as its upstream gradient when chain_o is set (the LM-head
  input is taken to be that projection's output), the others take
  the synthetic upstream gradients supplied with the inputs.

update_steps: the per-update schedule of Algorithm 1 on a chained toy model whose LM-head
input is one adapted projection's output, h = h0 + s (x A^T) B^T: the weights w are computed
once (before the loop), then every gradient step recomputes h, the weighted loss and dL/dh,
the adapter gradients, and takes theta <- theta - eta grad (Eq. 2). Float64 throughout.
"""
import numpy as np

from . import ce, lora, ngram


def update_step(tok, ce_in, problems, n, w_min, chain_o=True):
    f, w = ngram.ngram_weights(tok["history"], tok["updates"], n, w_min)
    loss, lse, dH = ce.weighted_ce(ce_in["h"], ce_in["W"], ce_in["labels"], w, ce_in["row_offsets"])
    off = np.asarray(ce_in["row_offsets"], np.int64)
    grads = []
    for p in problems:
        dy = p["dy"]
        if chain_o and p["name"].endswith(".o"):
            e = p["episode"]
            dy = dH[off[e]:off[e + 1]]
        grads.append(lora.lora_grad(p["x"], dy, p["A"], p["B"], p["scale"]))
    return dict(f=f, w=w, loss=loss, lse=lse, dH=dH, lora=grads)


def update_steps(h0, W, labels, w, row_offsets, x, A, B, scale, lr, steps=2):
    A = np.asarray(A, np.float64).copy()
    B = np.asarray(B, np.float64).copy()
    x64 = np.asarray(x, np.float64)
    h0 = np.asarray(h0, np.float64)
    losses = []
    for _ in range(steps):
        h = h0 + scale * (x64 @ A.T) @ B.T
        loss, _, dH = ce.weighted_ce(h, W, labels, w, row_offsets)
        dA, dB = lora.lora_grad(x64, dH, A, B, scale)
        A = A - lr * dA
        B = B - lr * dB
        losses.append(loss)
    return A, B, losses
