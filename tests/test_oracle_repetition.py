"""Pins of the repetition oracle (Eq. 6-7, tau of Appendix C) against things other than itself:
hand-worked texts, set sizes from boolean membership vectors, closed forms and invariants."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import repetition as rep

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "repetition_cases.json")


def _cases():
    with open(GOLDEN) as fh:
        return json.load(fh)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_golden_texts(case):
    vocab = {}
    updates = [rep.words_of_text(t, vocab) for t in case["texts"]]
    out = rep.repetition(updates, tau=0.5)
    assert [list(p) for p in out["pairs"]] == case["pairs"]
    num, den = (int(v) for v in case["rho"].split("/"))
    assert out["rho"] == num / den
    assert out["nu"] == 1.0 - num / den
    assert out["best"] == case["best"]
    assert out["skip"] == case["skip"]


def _membership(words, V):
    m = np.zeros(V, bool)
    m[np.asarray(words, np.int64)] = True
    return m


def test_counts_match_membership_vectors():
    rng = np.random.default_rng(7)
    for _ in range(300):
        V = int(rng.integers(1, 30))
        a = rng.integers(0, V, int(rng.integers(0, 40)))
        b = rng.integers(0, V, int(rng.integers(0, 40)))
        j, inter, union = rep.jaccard(a, b)
        ma, mb = _membership(a, V), _membership(b, V)
        assert inter == int((ma & mb).sum()) and union == int((ma | mb).sum())
        assert j == (Fraction(inter, union) if union else 0)


def test_symmetric_and_order_free():
    rng = np.random.default_rng(8)
    for _ in range(100):
        a = rng.integers(0, 12, int(rng.integers(1, 20)))
        b = rng.integers(0, 12, int(rng.integers(1, 20)))
        j1, _, _ = rep.jaccard(a, b)
        j2, _, _ = rep.jaccard(b, a)
        j3, _, _ = rep.jaccard(rng.permutation(np.concatenate([a, a])), b[::-1])
        assert j1 == j2 == j3
        assert 0 <= j1 <= 1
        assert (j1 == 1) == (set(a.tolist()) == set(b.tolist()))


def test_subset_closed_form():
    rng = np.random.default_rng(9)
    for _ in range(100):
        b = rng.choice(1000, int(rng.integers(1, 50)), replace=False)
        a = rng.choice(b, int(rng.integers(1, len(b) + 1)), replace=False)
        j, _, _ = rep.jaccard(a, b)
        assert j == Fraction(len(a), len(b))


def test_rho_is_the_maximum_and_skip_is_nu_below_tau():
    rng = np.random.default_rng(10)
    for _ in range(200):
        k = int(rng.integers(1, 8))
        ups = [rng.integers(0, 15, int(rng.integers(0, 12))) for _ in range(k)]
        tau = float(rng.choice([0.25, 0.5, 0.75]))
        out = rep.repetition(ups, tau)
        js = [rep.jaccard(ups[-1], u)[0] for u in ups[:-1]]
        if not js:
            assert out["rho"] == 0.0 and out["best"] == -1 and out["nu"] == 1.0 and not out["skip"]
            continue
        best = max(js)
        assert out["rho"] == float(best) and js[out["best"]] == best
        assert all(j < best for j in js[:out["best"]])  # the first maximum
        assert out["skip"] == (1.0 - float(best) < tau)
        if tau == 0.5:  # the exact integer form of nu < 1/2: 2 |A & B| > |A | B|
            inter, union = out["pairs"][out["best"]]
            assert out["skip"] == (2 * inter > union)
