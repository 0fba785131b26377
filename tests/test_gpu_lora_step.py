"""GPU parity of the adapter step of Eq. 2 (theta <- theta - eta grad, Algorithm 1's parameter
update) against the oracle, bit for bit: float32 parameters (product, then difference, each
rounded to nearest), their bf16 operand copies (round to nearest even) and the gradient reset.
Then Algorithm 1's per-update schedule end to end on a chained toy model (the LM-head input is
the adapted projection's output): weights once, two gradient steps, each recomputing the
hidden states (test-side torch plumbing), the weighted CE and the adapter gradients through
the library, against the float64 oracle of the same schedule."""
import numpy as np
import pytest

from gpu_util import dev_f32, dev_i32, host, note, rel_norm
from oracle import ce as oce
from oracle import lora as olora
from oracle import ngram as ongram
from oracle import step as ostep

pytestmark = pytest.mark.gpu


def _bits(a):
    return np.asarray(a, np.float32).view(np.uint32)


@pytest.mark.parametrize("lr", [5e-4, 1.0, -0.3])
def test_sgd_step_bit_exact(attt, lr):
    import torch
    rng = np.random.default_rng(50)
    sizes = [0, 1, 1023, 1024, 1025, 4097, 300001]
    note(f"lora sgd lr={lr}")
    host_p, host_g, params = [], [], []
    for n in sizes:
        p = rng.standard_normal(n).astype(np.float32)
        g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-3, 3, n)).astype(np.float32)
        host_p.append(p)
        host_g.append(g)
        params.append(dict(param=dev_f32(p), grad=dev_f32(g),
                           param_bf16=torch.empty(n, dtype=torch.bfloat16, device="cuda")))
    attt.lora_sgd_step(params, lr, zero_grad=True)
    for p, g, d in zip(host_p, host_g, params):
        want = olora.sgd_step(p, g, lr)
        assert _bits(host(d["param"])).tolist() == _bits(want).tolist()
        got_b = d["param_bf16"].view(torch.int16).cpu().numpy().view(np.uint16)
        assert got_b.tolist() == olora.bf16_round_bits(want).tolist()
        assert not host(d["grad"]).any()


def test_sgd_step_keeps_grad_and_skips_bf16(attt):
    rng = np.random.default_rng(51)
    p = rng.standard_normal(5000).astype(np.float32)
    g = rng.standard_normal(5000).astype(np.float32)
    note("lora sgd without reset and bf16 copy")
    d = dict(param=dev_f32(p), grad=dev_f32(g))
    attt.lora_sgd_step([d], 0.125)
    assert _bits(host(d["param"])).tolist() == _bits(olora.sgd_step(p, g, 0.125)).tolist()
    assert _bits(host(d["grad"])).tolist() == _bits(g).tolist()
    attt.lora_sgd_step([d], 0.125)      # a second step with the same gradient
    twice = olora.sgd_step(olora.sgd_step(p, g, 0.125), g, 0.125)
    assert _bits(host(d["param"])).tolist() == _bits(twice).tolist()


def test_two_gradient_steps_chained_f32(attt):
    """Algorithm 1 for one update on a toy model h = h0 + s (x A^T) B^T: w from the n-gram
    pass once, then two steps of (h, weighted CE and dL/dh, dA and dB, theta - eta grad)."""
    import torch
    rng = np.random.default_rng(52)
    N, d, V, r, s = 96, 64, 300, 8, 2.0
    H = rng.integers(0, V, 400).astype(np.int32)
    x_tok = np.concatenate([H[100:140], rng.integers(0, V, N - 40)]).astype(np.int32)
    h0 = rng.standard_normal((N, d)).astype(np.float32)
    W = (0.5 * rng.standard_normal((V, d))).astype(np.float32)
    X = rng.standard_normal((N, d)).astype(np.float32)
    A = (0.3 * rng.standard_normal((r, d))).astype(np.float32)
    B = np.zeros((d, r), np.float32)          # the standard initialisation: dA = 0 at step 1
    labels = x_tok
    off = np.array([0, N], np.int64)
    note("two gradient steps, chained f32")
    f, w = attt.ngram_weights(dev_i32(H), [0, len(H)], dev_i32(x_tok), [0, N], n=3, w_min=0.05)
    fo, wo = ongram.ngram_weights([H], [x_tok], 3, 0.05)
    assert _bits(host(w)).tolist() == _bits(wo).tolist() and np.any(wo < 1)
    # step size: the first step moves B by about 0.1 at most
    _, _, dH0 = oce.weighted_ce(h0, W, labels, wo, off)
    lr = 0.1 / np.max(np.abs(olora.lora_grad(X, dH0, A, B, s)[1]))
    Ao, Bo, lo = ostep.update_steps(h0, W, labels, wo, off, X, A, B, s, lr, steps=2)

    tA, tB, tX, th0 = dev_f32(A), dev_f32(B), dev_f32(X), dev_f32(h0)
    gA = torch.zeros_like(tA)
    gB = torch.zeros_like(tB)
    tW, tl = dev_f32(W), dev_i32(labels)
    losses = []
    for _ in range(2):
        h = (th0 + s * (tX @ tA.T) @ tB.T).contiguous()
        loss, lse, dH = attt.weighted_ce_fwd_bwd(h, tW, tl, w, row_offsets=off)
        losses.append(float(host(loss)[0]))
        attt.lora_grad([dict(x=tX, dy=dH, A=tA, B=tB, dA=gA, dB=gB, scale=s)])
        attt.lora_sgd_step([dict(param=tA, grad=gA), dict(param=tB, grad=gB)], lr, zero_grad=True)
    for k in range(2):
        assert abs(losses[k] - lo[k][0]) <= 1e-5 * abs(lo[k][0])
    assert lo[1][0] < lo[0][0]                # the step descends
    dA_gpu, dB_gpu = host(tA) - A, host(tB) - B
    dA_or, dB_or = Ao - A, Bo - B
    assert np.abs(dA_or).max() > 1e-3         # step 2 moved A (B was nonzero by then)
    assert rel_norm(dA_gpu, dA_or) <= 1e-5 and rel_norm(dB_gpu, dB_or) <= 1e-5
