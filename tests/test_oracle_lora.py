"""Pins of the LoRA-gradient oracle (adapter of Sec. 3.1, r / alpha of Appendix C) against
torch CPU autograd, exact zeros of the standard initialisation, linearity and finite
differences; and of the chained update step (weights -> CE -> LoRA) by finite differences
of the loss with respect to adapter entries."""
import numpy as np
import torch

from oracle import ce, lora, ngram, step
from workloads import Workload


def _problem(seed, N=11, d_in=7, d_out=5, r=3):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((N, d_in)), rng.standard_normal((N, d_out)),
            rng.standard_normal((r, d_in)), rng.standard_normal((d_out, r)))


def test_matches_torch_autograd():
    x, dy, A, B = _problem(0)
    s = 16.0 / 3
    dA, dB = lora.lora_grad(x, dy, A, B, s)
    tA = torch.tensor(A, requires_grad=True)
    tB = torch.tensor(B, requires_grad=True)
    y = s * (torch.tensor(x) @ tA.T) @ tB.T
    (y * torch.tensor(dy)).sum().backward()
    assert np.allclose(dA, tA.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dB, tB.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_standard_init_zero_grads_are_exact():
    x, dy, A, B = _problem(1)
    dA, dB = lora.lora_grad(x, dy, A, np.zeros_like(B), 2.0)
    assert np.all(dA == 0.0) and np.any(dB != 0.0)
    dA, dB = lora.lora_grad(x, dy, np.zeros_like(A), B, 2.0)
    assert np.all(dB == 0.0) and np.any(dA != 0.0)


def test_linear_in_upstream_gradient():
    x, dy, A, B = _problem(2)
    dy2 = np.random.default_rng(3).standard_normal(dy.shape)
    a1, b1 = lora.lora_grad(x, dy, A, B, 2.0)
    a2, b2 = lora.lora_grad(x, dy2, A, B, 2.0)
    a3, b3 = lora.lora_grad(x, 2 * dy - 3 * dy2, A, B, 2.0)
    assert np.allclose(a3, 2 * a1 - 3 * a2, rtol=1e-11, atol=1e-11)
    assert np.allclose(b3, 2 * b1 - 3 * b2, rtol=1e-11, atol=1e-11)


def test_finite_differences():
    x, dy, A, B = _problem(4, N=6, d_in=4, d_out=3, r=2)
    s = 2.0
    dA, dB = lora.lora_grad(x, dy, A, B, s)
    f = lambda A_, B_: float(np.sum(lora.lora_forward(x, None, A_, B_, s) * dy))
    eps = 1e-6
    for idx in np.ndindex(A.shape):
        Ap, Am = A.copy(), A.copy(); Ap[idx] += eps; Am[idx] -= eps
        assert abs((f(Ap, B) - f(Am, B)) / (2 * eps) - dA[idx]) < 1e-7
    for idx in np.ndindex(B.shape):
        Bp, Bm = B.copy(), B.copy(); Bp[idx] += eps; Bm[idx] -= eps
        assert abs((f(A, Bp) - f(A, Bm)) / (2 * eps) - dB[idx]) < 1e-7


def test_sampled_matches_full():
    x, dy, A, B = _problem(5, N=20, d_in=9, d_out=6, r=4)
    dA, dB = lora.lora_grad(x, dy, A, B, 4.0)
    cols, rows = [0, 4, 8], [1, 5]
    a, b = lora.lora_grad_sampled(x, dy, A, B, 4.0, cols, rows)
    assert np.allclose(a, dA[:, cols], rtol=1e-13) and np.allclose(b, dB[rows], rtol=1e-13)


def test_chained_step_finite_differences():
    """The LM-head input is the adapted output projection h = h0 + s (X A^T) B^T; dA and dB
    from the chained oracle equal finite differences of the weighted loss (Eq. 10)."""
    rng = np.random.default_rng(8)
    N, d, V, r, s = 9, 6, 13, 2, 8.0
    h0 = rng.standard_normal((N, d))
    W = rng.standard_normal((V, d))
    X = rng.standard_normal((N, d))
    A = 0.3 * rng.standard_normal((r, d))
    B = 0.3 * rng.standard_normal((d, r))
    H = rng.integers(0, V, 40)
    x = np.concatenate([H[5:11], rng.integers(0, V, 3)])
    f, w = ngram.ngram_weights([H], [x], 2, 0.05)
    off = np.array([0, N])
    labels = x

    def loss_of(A_, B_):
        h = h0 + lora.lora_forward(X, None, A_, B_, s)
        return ce.weighted_ce_loss(h, W, labels, w, off)[0]

    tok = dict(history=[H], updates=[x])
    ce_in = dict(h=h0 + lora.lora_forward(X, None, A, B, s), W=W, labels=labels, row_offsets=off)
    prob = [dict(name="e0.o", episode=0, x=X, dy=None, A=A, B=B, scale=s)]
    out = step.update_step(tok, ce_in, prob, 2, 0.05)
    dA, dB = out["lora"][0]
    assert np.any(w < 1) and np.any(w == 1)
    eps = 1e-6
    for idx in np.ndindex(A.shape):
        Ap, Am = A.copy(), A.copy(); Ap[idx] += eps; Am[idx] -= eps
        assert abs((loss_of(Ap, B) - loss_of(Am, B)) / (2 * eps) - dA[idx]) < 1e-7
    for idx in np.ndindex(B.shape):
        Bp, Bm = B.copy(), B.copy(); Bp[idx] += eps; Bm[idx] -= eps
        assert abs((loss_of(A, Bp) - loss_of(A, Bm)) / (2 * eps) - dB[idx]) < 1e-7


def test_tiny_config_step_runs():
    wl = Workload("c1")
    out = step.update_step(wl.tokens(), wl.ce(), wl.lora(), 4, 0.05)
    dA, dB = out["lora"][0]
    assert np.all(dA == 0.0)               # B = 0 at initialisation
    assert np.isfinite(out["loss"]).all() and out["dH"].shape == (512, 256)


# ---- the adapter step of Eq. 2 ---------------------------------------------------------
def test_sgd_step_closed_forms():
    """theta - eta grad: identity for eta = 0 or grad = 0; exactly representable cases by hand
    (a flipped sign or a dropped eta fails them)."""
    rng = np.random.default_rng(20)
    p = rng.standard_normal(50).astype(np.float32)
    g = (1e3 * rng.standard_normal(50)).astype(np.float32)
    assert lora.sgd_step(p, g, 0.0).view(np.uint32).tolist() == p.view(np.uint32).tolist()
    assert lora.sgd_step(p, np.zeros_like(g), 0.37).view(np.uint32).tolist() == p.view(np.uint32).tolist()
    out = lora.sgd_step(np.array([1.0, 0.5, -3.0], np.float32), np.array([3.0, -2.0, 8.0], np.float32), 0.25)
    assert out.tolist() == [0.25, 1.0, -5.0]
    assert lora.sgd_step(np.float32([2.0]), np.float32([1.0]), 2.0 ** -20)[0] == np.float32(2.0 - 2.0 ** -20)


def test_sgd_step_rounds_product_then_difference():
    """1 - (1 + 2^-12)(1 + 2^-12): the exact product 1 + 2^-11 + 2^-24 is a float32 tie and
    rounds to even, 1 + 2^-11, so the step gives -2^-11; a fused multiply-add would give
    -(2^-11 + 2^-24), which float32 represents."""
    a = np.float32(1.0 + 2.0 ** -12)
    out = lora.sgd_step(np.float32([1.0]), np.float32([a]), float(a))[0]
    assert out == np.float32(-(2.0 ** -11))
    assert np.float32(-(2.0 ** -11 + 2.0 ** -24)) != out


def test_bf16_rounding_by_hand():
    """Round to nearest even on the 16 dropped bits, worked out by hand."""
    vals = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20, -2.0,
                     np.inf, -np.inf, 0.0, -0.0, 3.0e38], np.float32)
    want = [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC000, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x7F62]
    assert lora.bf16_round_bits(vals).tolist() == want
    nan = lora.bf16_round_bits(np.array([np.nan, -np.nan], np.float32))
    assert all((b & 0x7F80) == 0x7F80 and (b & 0x7F) != 0 for b in nan.tolist())
    # every bf16 value maps to itself
    allb = np.arange(0x10000, dtype=np.uint32)
    f = (allb << 16).view(np.float32)
    finite = np.isfinite(f)
    assert (lora.bf16_round_bits(f[finite]) == allb[finite]).all()


def test_update_steps_descend():
    """Two steps of Algorithm 1's schedule on the chained toy model: eta = 0 leaves the adapter
    and the loss unchanged; a small eta lowers the loss by eta |grad|^2 to first order (a step
    along +grad would raise it)."""
    rng = np.random.default_rng(21)
    N, d, V, r, s = 12, 8, 17, 3, 4.0
    h0 = rng.standard_normal((N, d))
    W = rng.standard_normal((V, d))
    X = rng.standard_normal((N, d))
    A = 0.3 * rng.standard_normal((r, d))
    B = 0.3 * rng.standard_normal((d, r))
    labels = rng.integers(0, V, N)
    w = rng.uniform(0.05, 1, N)
    off = np.array([0, N])
    A0, B0, l0 = step.update_steps(h0, W, labels, w, off, X, A, B, s, 0.0)
    assert np.array_equal(A0, A) and np.array_equal(B0, B) and l0[0][0] == l0[1][0]
    h = h0 + lora.lora_forward(X, None, A, B, s)
    _, _, dH = ce.weighted_ce(h, W, labels, w, off)
    gA, gB = lora.lora_grad(X, dH, A, B, s)
    g2 = np.sum(gA * gA) + np.sum(gB * gB)
    eta = 1e-4
    A1, B1, l1 = step.update_steps(h0, W, labels, w, off, X, A, B, s, eta, steps=1)
    hn = h0 + lora.lora_forward(X, None, A1, B1, s)
    drop = l1[0][0] - ce.weighted_ce_loss(hn, W, labels, w, off)[0]
    assert drop > 0 and abs(drop / (eta * g2) - 1) < 1e-2
    assert np.allclose(A1, A - eta * gA, rtol=0, atol=1e-15) and np.allclose(B1, B - eta * gB, rtol=0, atol=1e-15)
