"""GPU parity of the update-text repetition path (Eq. 6-7, tau of Appendix C) against the
oracle: per-pair counts (|A & B|, |A | B|) bit-exact, rho and nu bitwise (both sides round
the same exact fraction to float64), skip and the reported previous text exact.

Inputs: the hand-worked golden texts (words mapped to ids), seeded random episodes (ragged
lengths, empty texts, heavy repetition inside texts, texts long enough for several hash
partitions, more episodes than one launch takes), and the update histories of the
workloads (each previous update of the history a text, the update itself the candidate),
with token ids standing in for word ids."""
import json
import os

import numpy as np
import pytest

from gpu_util import dev_i32, note
from oracle import repetition as orep
from workloads import Workload

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "repetition_cases.json")


def _run(attt, episodes, tau=0.5):
    """episodes: list of lists of word-id sequences. Returns GPU and oracle results."""
    texts = [np.asarray(t, np.int32) for ep in episodes for t in ep]
    lens = [len(t) for t in texts]
    toff = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    etx = np.concatenate([[0], np.cumsum([len(ep) for ep in episodes])]).astype(np.int64)
    flat = np.concatenate(texts) if toff[-1] else np.zeros(1, np.int32)
    rho, nu, skip, best, pairs = attt.update_repetition(dev_i32(flat), toff, etx, tau=tau, want_pairs=True)
    got = dict(rho=rho.cpu().numpy(), nu=nu.cpu().numpy(), skip=skip.cpu().numpy(), best=best.cpu().numpy(),
               pairs=pairs.cpu().numpy() if pairs is not None else np.zeros((0, 2), np.int32))
    want = [orep.repetition(ep, tau) for ep in episodes]
    return got, want


def _check(got, want):
    pairs_o = [p for w in want for p in w["pairs"]]
    assert got["pairs"].tolist() == [list(p) for p in pairs_o]
    assert got["rho"].view(np.uint64).tolist() == np.array([w["rho"] for w in want]).view(np.uint64).tolist()
    assert got["nu"].view(np.uint64).tolist() == np.array([w["nu"] for w in want]).view(np.uint64).tolist()
    assert got["skip"].tolist() == [int(w["skip"]) for w in want]
    assert got["best"].tolist() == [w["best"] for w in want]


def test_golden_texts_in_one_call(attt):
    with open(GOLDEN) as fh:
        cases = json.load(fh)["cases"]
    vocab = {}
    episodes = [[orep.words_of_text(t, vocab) for t in c["texts"]] for c in cases]
    note(f"repetition golden: {len(episodes)} episodes")
    got, want = _run(attt, episodes)
    _check(got, want)
    assert got["best"].tolist() == [c["best"] for c in cases]


@pytest.mark.parametrize("tau", [0.25, 0.5, 0.75])
def test_random_ragged_episodes(attt, tau):
    rng = np.random.default_rng(int(tau * 100))
    episodes = []
    for e in range(40):
        k = int(rng.integers(1, 9))
        V = int(rng.integers(1, 300))
        ep = []
        for _ in range(k):
            n = int(rng.choice([0, 1, 2, 5, 50, 300, 2000]))
            ep.append(rng.integers(0, V, n, dtype=np.int32))
        if k > 1 and rng.random() < 0.3:  # a candidate that replays an earlier text with edits
            src = ep[int(rng.integers(0, k - 1))].copy()
            if len(src):
                src[rng.integers(0, len(src), max(1, len(src) // 10))] = V + 1
            ep[-1] = src
        episodes.append(ep)
    note(f"repetition random: tau {tau}, {len(episodes)} episodes")
    got, want = _run(attt, episodes, tau)
    _check(got, want)


def test_long_texts_several_partitions(attt):
    rng = np.random.default_rng(3)
    episodes = []
    for lc, lp, V in [(20000, 9000, 50000), (4097, 4097, 1 << 30), (70000, 300, 2000), (1, 65536, 8)]:
        cand = rng.integers(0, V, lc, dtype=np.int32)
        prev = [rng.integers(0, V, lp, dtype=np.int32), np.concatenate([cand[: lc // 2], cand[: lc // 3]])]
        episodes.append(prev + [cand])
    note("repetition long texts: up to 18 hash partitions")
    got, want = _run(attt, episodes)
    _check(got, want)


def test_more_episodes_than_one_launch(attt):
    rng = np.random.default_rng(4)
    episodes = [[rng.integers(0, 20, int(rng.integers(0, 30)), dtype=np.int32) for _ in range(int(rng.integers(1, 4)))]
                for _ in range(150)]
    got, want = _run(attt, episodes)
    _check(got, want)


@pytest.mark.parametrize("key", ["c2", "c3", "c5"])
def test_workload_histories(attt, key):
    wl = Workload(key)
    cfg, tok = wl.cfg, wl.tokens()
    episodes = []
    for e in range(cfg.episodes):
        h = np.asarray(tok["history"][e], np.int32)
        prev = [h[i * cfg.prior_len:(i + 1) * cfg.prior_len] for i in range(cfg.prior_updates)]
        episodes.append(prev + [np.asarray(tok["updates"][e], np.int32)])
    note(f"repetition {key}: {cfg.episodes} episodes x {cfg.prior_updates + 1} texts")
    got, want = _run(attt, episodes)
    _check(got, want)
    note(f"rho {np.round(got['rho'][:4], 4).tolist()} skip {got['skip'][:8].tolist()}")
