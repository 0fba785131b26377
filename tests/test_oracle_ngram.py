"""Pins of the n-gram oracle (Sec. 3.3, Eq. 8-9) against things other than itself:
hand-worked cases, brute-force scanning, a library routine (bincount) for n = 1,
closed forms, monotonicity, and exact rational rounding of the weight."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ngram
from workloads import Workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "ngram_cases.json")


def _cases():
    with open(GOLDEN) as fh:
        return json.load(fh)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_golden_cases(case):
    hist = np.array([t for part in case["history_parts"] for t in part], np.int32)
    x = np.array(case["tokens"], np.int32)
    f = ngram.exposure(hist, x, case["n"])
    assert f.tolist() == case["f"]
    w = ngram.weights_from_exposure(f, case["w_min"])
    expect = np.array([np.float32(s) for s in case["w"]], np.float32)
    assert w.view(np.uint32).tolist() == expect.view(np.uint32).tolist()
    assert ngram.exposure_bruteforce(hist, x, case["n"]).tolist() == case["f"]


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6])
def test_dict_counting_matches_bruteforce(n):
    rng = np.random.default_rng(100 + n)
    for _ in range(40):
        vocab = int(rng.integers(2, 6))
        H = rng.integers(0, vocab, int(rng.integers(0, 40)), dtype=np.int32)
        x = rng.integers(0, vocab, int(rng.integers(0, 25)), dtype=np.int32)
        assert ngram.exposure(H, x, n).tolist() == ngram.exposure_bruteforce(H, x, n).tolist()


def test_empty_history_gives_unit_weights():
    rng = np.random.default_rng(1)
    for n in (1, 3, 4):
        x = rng.integers(0, 100, 57, dtype=np.int32)
        f = ngram.exposure(np.empty(0, np.int32), x, n)
        assert not f.any()
        assert np.all(ngram.weights_from_exposure(f, 0.05) == np.float32(1.0))


@pytest.mark.parametrize("n", [2, 3, 4])
def test_fully_repeated_text_is_downweighted(n):
    rng = np.random.default_rng(7)
    x = rng.integers(0, 1000, 64, dtype=np.int32)
    H = np.concatenate([rng.integers(0, 1000, 30, dtype=np.int32), x,
                        rng.integers(0, 1000, 30, dtype=np.int32)])
    f = ngram.exposure(H, x, n)
    assert np.all(f >= 1)
    assert np.all(ngram.weights_from_exposure(f, 0.05) <= np.float32(0.5))


@pytest.mark.parametrize("m", [1, 2, 5])
def test_distinct_tokens_repeated_m_times(m):
    x = np.arange(100, 140, dtype=np.int32)          # L distinct tokens
    H = np.tile(x, m)
    for n in (1, 2, 3, 7):
        assert np.all(ngram.exposure(H, x, n) == m)


def test_unigram_equals_bincount():
    rng = np.random.default_rng(3)
    H = rng.integers(0, 50, 400, dtype=np.int32)
    x = rng.integers(0, 60, 200, dtype=np.int32)
    counts = np.bincount(H, minlength=60)
    assert ngram.exposure(H, x, 1).tolist() == counts[x].tolist()


def test_n_longer_than_update():
    x = np.array([1, 2, 3], np.int32)
    H = np.array([1, 2, 3, 1, 2, 3], np.int32)
    assert not ngram.exposure(H, x, 4).any()
    assert ngram.exposure(H, x, 3).tolist() == [2, 2, 2]


def test_appending_history_never_lowers_exposure():
    rng = np.random.default_rng(11)
    x = rng.integers(0, 8, 50, dtype=np.int32)
    H = rng.integers(0, 8, 100, dtype=np.int32)
    f0 = ngram.exposure(H, x, 3)
    for _ in range(5):
        H = np.concatenate([H, rng.integers(0, 8, 37, dtype=np.int32)])
        f1 = ngram.exposure(H, x, 3)
        assert np.all(f1 >= f0)
        f0 = f1


def _rn_f32(q: Fraction) -> np.float32:
    """Round a positive rational to the nearest float32, ties to even, exactly."""
    lo = np.float32(float(q))          # within one ulp of q
    cands = {lo, np.nextafter(lo, np.float32(0)), np.nextafter(lo, np.float32(np.inf))}
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - q),
                                     int(np.array(c, np.float32).view(np.uint32)) & 1))
    return np.float32(best)


def test_weight_is_correctly_rounded_float32():
    f = np.concatenate([np.arange(0, 3000), np.array([2**20, 2**24 - 2, 2**31])]).astype(np.uint32)
    for w_min in (0.05, 2.0**-20, 0.3, 1.0):
        w = ngram.weights_from_exposure(f, w_min)
        wm = np.float32(w_min)
        for fi, wi in zip(f[:3000], w[:3000]):
            want = max(wm, _rn_f32(Fraction(1, 1 + int(fi))))
            assert np.float32(wi).view(np.uint32) == np.float32(want).view(np.uint32), (fi, w_min)
        assert np.all(w[3000:] >= wm)


def test_floor_reached_exactly_at_19():
    w = ngram.weights_from_exposure(np.arange(0, 40, dtype=np.uint32), 0.05)
    assert w[19] == np.float32(0.05) and w[18] > np.float32(0.05)
    assert np.all(w[19:] == np.float32(0.05))


def test_multi_episode_concatenation():
    rng = np.random.default_rng(5)
    hs = [rng.integers(0, 5, k, dtype=np.int32) for k in (0, 10, 50)]
    xs = [rng.integers(0, 5, k, dtype=np.int32) for k in (7, 0, 20)]
    f, w = ngram.ngram_weights(hs, xs, 2, 0.05)
    want = np.concatenate([ngram.exposure_bruteforce(h, x, 2) for h, x in zip(hs, xs)])
    assert f.tolist() == want.tolist()
    assert w.shape == f.shape


def test_generator_repetition_regime():
    wl = Workload("c1")
    tok = wl.tokens()
    assert tok["hist_off"].tolist() == [0, 2048]
    assert tok["tok_off"].tolist() == [0, 512]
    f = ngram.exposure(tok["history"][0], tok["updates"][0], 4)
    covered = float(np.mean(f > 0))
    assert 0.25 < covered < 0.7        # about 40% of the update copied from the history
    # determinism of the generator
    assert np.array_equal(Workload("c1").tokens()["tok_flat"], tok["tok_flat"])
