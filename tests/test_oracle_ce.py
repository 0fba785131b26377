"""Pins of the weighted-CE oracle (Sec. 3.3, Eq. 10) against a textbook routine (torch
CPU cross_entropy and autograd, float64), invariants (weight scaling, softmax shift
invariance) and central finite differences."""
import numpy as np
import pytest
import torch

from oracle import ce


def _problem(seed, N, d, V, E=1):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((N, d))
    W = 0.5 * rng.standard_normal((V, d))
    labels = rng.integers(0, V, N)
    w = rng.uniform(0.05, 1.0, N)
    cuts = np.sort(rng.choice(np.arange(1, N), E - 1, replace=False)) if E > 1 else []
    off = np.array([0, *cuts, N], np.int64)
    return h, W, labels, w, off


def test_unit_weights_equal_torch_mean_cross_entropy():
    h, W, labels, _, off = _problem(0, 13, 7, 11)
    w = np.ones(13)
    loss, lse, dH = ce.weighted_ce(h, W, labels, w, off)
    th = torch.tensor(h, requires_grad=True)
    ref = torch.nn.functional.cross_entropy(th @ torch.tensor(W).T, torch.tensor(labels), reduction="mean")
    ref.backward()
    assert abs(loss[0] - ref.item()) < 1e-12
    assert np.allclose(dH, th.grad.numpy(), atol=1e-13, rtol=1e-12)
    assert np.allclose(lse, torch.logsumexp(torch.tensor(h @ W.T), 1).numpy(), atol=1e-12)


@pytest.mark.parametrize("E", [1, 3])
def test_weighted_episodes_match_torch_autograd(E):
    h, W, labels, w, off = _problem(1, 29, 9, 17, E)
    loss, lse, dH = ce.weighted_ce(h, W, labels, w, off)
    th = torch.tensor(h, requires_grad=True)
    per_row = torch.nn.functional.cross_entropy(th @ torch.tensor(W).T, torch.tensor(labels), reduction="none")
    tw = torch.tensor(w)
    losses = [(tw[a:b] * per_row[a:b]).sum() / (b - a) for a, b in zip(off[:-1], off[1:])]
    torch.stack(losses).sum().backward()
    assert np.allclose(loss, [x.item() for x in losses], rtol=1e-12, atol=1e-14)
    assert np.allclose(dH, th.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_uniform_weight_scales_loss_and_grad():
    h, W, labels, _, off = _problem(2, 10, 5, 8)
    l1, _, g1 = ce.weighted_ce(h, W, labels, np.ones(10), off)
    l2, _, g2 = ce.weighted_ce(h, W, labels, np.full(10, 0.25), off)
    assert np.allclose(l2, 0.25 * l1, rtol=1e-13)
    assert np.allclose(g2, 0.25 * g1, rtol=1e-12, atol=1e-15)


def test_shift_of_all_head_rows_leaves_loss_and_grad_unchanged():
    h, W, labels, w, off = _problem(3, 12, 6, 9, 2)
    c = np.random.default_rng(9).standard_normal(6)
    l1, _, g1 = ce.weighted_ce(h, W, labels, w, off)
    l2, _, g2 = ce.weighted_ce(h, W + c[None, :], labels, w, off)
    assert np.allclose(l1, l2, rtol=1e-11)
    assert np.allclose(g1, g2, rtol=1e-9, atol=1e-12)


def test_finite_differences_of_hidden_states():
    h, W, labels, w, off = _problem(4, 6, 5, 7, 2)
    _, _, dH = ce.weighted_ce(h, W, labels, w, off)
    eps = 1e-6
    for t in range(6):
        for k in range(5):
            hp = h.copy(); hp[t, k] += eps
            hm = h.copy(); hm[t, k] -= eps
            fd = (ce.weighted_ce_loss(hp, W, labels, w, off).sum()
                  - ce.weighted_ce_loss(hm, W, labels, w, off).sum()) / (2 * eps)
            assert abs(fd - dH[t, k]) < 1e-8 * max(1.0, abs(dH[t, k])) + 1e-9


def test_selected_rows_match_full_problem():
    h, W, labels, w, off = _problem(5, 40, 8, 30, 3)
    _, lse, dH = ce.weighted_ce(h, W, labels, w, off, chunk=7)
    rows = [0, 5, 17, 39]
    lse_r, _, dH_r = ce.ce_rows(h, W.astype(np.float64), labels, w, off, rows)
    assert np.allclose(lse_r, lse[rows], rtol=1e-14)
    assert np.allclose(dH_r, dH[rows], rtol=1e-13, atol=1e-16)


def test_large_logits_are_stable():
    h, W, labels, w, off = _problem(6, 5, 4, 6)
    loss, lse, dH = ce.weighted_ce(h * 300.0, W, labels, w, off)
    assert np.all(np.isfinite(loss)) and np.all(np.isfinite(dH)) and np.all(np.isfinite(lse))
