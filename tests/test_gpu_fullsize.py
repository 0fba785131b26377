"""GPU parity at the full workload sizes (Llama-8B shape, long-trajectory Qwen-14B shape,
16-episode stuck-agent batch), in the launch configuration the bench times.

n-gram exposure and weights are compared in full (bit-exact). The LM-head CE is compared on
sampled rows computed one by one by the oracle (lse and dL/dh rows), and the loss through a
property that holds at any size: loss_e = (1/L_e) sum_t w_t (lse_t - z_{t,y_t}) with the
label logits from the oracle and the GPU's lse (itself checked on the sampled rows). LoRA
gradients are compared on sampled columns of dA and rows of dB."""
import numpy as np
import pytest

from gpu_util import cosine, dev_dense, dev_f32, dev_i32, host, note, rel_norm
from oracle import ce as oce
from oracle import lora as olora
from oracle import ngram as ongram
from workloads import Workload

pytestmark = pytest.mark.gpu

CONFIGS = ["c3", "c4", "c5"]


@pytest.fixture(scope="module", params=CONFIGS)
def wl(request):
    note(f"generating {request.param}")
    return Workload(request.param)


def test_ngram_full(attt, wl):
    tok, cfg = wl.tokens(), wl.cfg
    note(f"ngram full {cfg.key}")
    f, w = attt.ngram_weights(dev_i32(tok["hist_flat"]), tok["hist_off"], dev_i32(tok["tok_flat"]),
                              tok["tok_off"], n=cfg.n, w_min=cfg.w_min)
    fo, wo = ongram.ngram_weights(tok["history"], tok["updates"], cfg.n, cfg.w_min)
    assert np.array_equal(host(f).view(np.uint32), fo)
    assert np.array_equal(host(w).view(np.uint32), wo.view(np.uint32))


def test_ce_full_sampled(attt, wl):
    cfg = wl.cfg
    tok, ce = wl.tokens(), wl.ce()
    _, w = ongram.ngram_weights(tok["history"], tok["updates"], cfg.n, cfg.w_min)
    note(f"ce full {cfg.key}")
    loss, lse, dH = attt.weighted_ce_fwd_bwd(dev_dense(ce["h"]), dev_dense(ce["W"]), dev_i32(ce["labels"]),
                                             dev_f32(w), row_offsets=ce["row_offsets"])
    loss, lse, dH = host(loss), host(lse), host(dH)
    N = cfg.rows
    rng = np.random.default_rng(17)
    rows = np.unique(np.concatenate([[0, N - 1], rng.integers(0, N, 14),
                                     np.asarray(ce["row_offsets"][1:-1], np.int64)]))
    note(f"oracle rows {cfg.key}: {len(rows)}")
    W64 = np.asarray(ce["W"].f32, np.float64)
    lse_o, _, dH_o = oce.ce_rows(ce["h"].f32, W64, ce["labels"], w, ce["row_offsets"], rows)
    assert np.max(np.abs(lse[rows] - lse_o) / np.abs(lse_o)) <= 1e-4
    assert cosine(dH[rows], dH_o) >= 0.999
    for i in range(len(rows)):
        assert cosine(dH[rows[i]], dH_o[i]) >= 0.999
    # label logits by the oracle's definition (z_{t,y_t} = h_t . W_{y_t}), in row chunks
    h = ce["h"].f32
    zy = np.empty(N, np.float64)
    for s in range(0, N, 4096):
        e = min(N, s + 4096)
        zy[s:e] = np.einsum("ij,ij->i", h[s:e].astype(np.float64), W64[ce["labels"][s:e]])
    off = ce["row_offsets"]
    for e in range(cfg.episodes):
        a, b = int(off[e]), int(off[e + 1])
        want = np.sum(w[a:b].astype(np.float64) * (lse[a:b].astype(np.float64) - zy[a:b])) / (b - a)
        assert abs(loss[e] - want) <= 1e-4 * abs(want), (e, loss[e], want)


def test_lora_full_sampled(attt, wl):
    import torch
    cfg = wl.cfg
    probs = wl.lora()
    note(f"lora full {cfg.key}: {len(probs)} problems")
    xs, dev = {}, []
    for p in probs:
        if id(p["x"]) not in xs:
            xs[id(p["x"])] = dev_dense(p["x"])
        r = p["rank"]
        dev.append(dict(x=xs[id(p["x"])], dy=dev_dense(p["dy"]), A=dev_dense(p["A"]), B=dev_dense(p["B"]),
                        scale=p["scale"], dA=torch.zeros(r, p["d_in"], dtype=torch.float32, device="cuda"),
                        dB=torch.zeros(p["d_out"], r, dtype=torch.float32, device="cuda")))
    attt.lora_grad(dev)
    rng = np.random.default_rng(5)
    step = max(1, len(probs) // 8)
    for p, q in list(zip(probs, dev))[::step]:
        cols = np.sort(rng.choice(p["d_in"], 64, replace=False))
        outs = np.sort(rng.choice(p["d_out"], 64, replace=False))
        dA_o, dB_o = olora.lora_grad_sampled(p["x"].f32, p["dy"].f32, p["A"].f32, p["B"].f32, p["scale"],
                                             cols, outs)
        dA = host(q["dA"])[:, cols]
        dB = host(q["dB"])[outs]
        assert cosine(dA, dA_o) >= 0.999, p["name"]
        assert cosine(dB, dB_o) >= 0.999, p["name"]
        assert rel_norm(dA, dA_o) <= 2e-2 and rel_norm(dB, dB_o) <= 2e-2


def test_ce_full_deterministic(attt, wl):
    """The launch configuration the bench times, run twice on the same inputs: loss, lse and
    dL/dh are bitwise identical (ordered reductions, no float atomics, no scratch)."""
    cfg = wl.cfg
    tok, ce = wl.tokens(), wl.ce()
    _, w = ongram.ngram_weights(tok["history"], tok["updates"], cfg.n, cfg.w_min)
    note(f"ce determinism {cfg.key}")
    args = (dev_dense(ce["h"]), dev_dense(ce["W"]), dev_i32(ce["labels"]), dev_f32(w))
    runs = []
    for _ in range(2):
        loss, lse, dH = attt.weighted_ce_fwd_bwd(*args, row_offsets=ce["row_offsets"])
        runs.append((host(loss).tobytes(), host(lse).tobytes(), host(dH).tobytes()))
    assert runs[0] == runs[1]
