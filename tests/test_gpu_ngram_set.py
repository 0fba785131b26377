"""GPU parity of the persistent n-gram sets (the history update of Algorithm 1) against the
float64 oracle's plain definition (Eq. 8-9 over the flat history): the set is built by
appending the previous updates one at a time, and after every append the weights of the
next text must equal, bit for bit, those the oracle gives for the concatenated history.
Also: texts shorter than n-1 (n-grams spanning three or more updates), empty appends,
several sets per call, the full-size bench workload against the streaming GPU path, and the
error outputs (capacity exceeded, wrong n)."""
import numpy as np
import pytest

from gpu_util import dev_i32, host, note
from oracle import ngram as ongram
from workloads import Workload, pack_episodes

pytestmark = pytest.mark.gpu


def _new_sets(attt, count, capacity, n):
    import torch
    nbytes = attt.ngram_set_size(capacity, n)
    sets = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(count)]
    attt.ngram_set_init(sets, capacity, n)
    return sets


def _pack(texts):
    off = np.zeros(len(texts) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in texts])
    flat = np.concatenate(texts).astype(np.int32) if off[-1] else np.empty(0, np.int32)
    return dev_i32(flat) if off[-1] else dev_i32(np.zeros(1, np.int32)), off


def _weights(attt, sets, texts, capacity, n, w_min=0.05):
    toks, off = _pack(texts)
    f, w = attt.ngram_set_weights(sets, toks, off, capacity, n, w_min=w_min)
    return host(f).view(np.uint32)[: off[-1]], host(w)[: off[-1]]


def _append(attt, sets, texts, capacity, n):
    toks, off = _pack(texts)
    attt.ngram_set_append(sets, toks, off, capacity, n)


def _check_against_oracle(attt, sets, histories, texts, capacity, n, w_min=0.05):
    f, w = _weights(attt, sets, texts, capacity, n, w_min)
    fo, wo = ongram.ngram_weights(histories, texts, n, w_min)
    assert f.tolist() == fo.tolist()
    assert w.view(np.uint32).tolist() == wo.view(np.uint32).tolist()
    return fo


def _split(history, size):
    return [history[i:i + size] for i in range(0, len(history), size)]


@pytest.mark.parametrize("key", ["c1", "c2"])
def test_ngram_set_incremental(attt, key):
    """Every previous update in turn: weights against the set, then append; last the new update."""
    wl = Workload(key)
    cfg, tok = wl.cfg, wl.tokens()
    note(f"ngram_set incremental {key}")
    E = cfg.episodes
    priors = [_split(h, cfg.prior_len) for h in tok["history"]]
    capacity = max(1, max(len(h) for h in tok["history"]) + cfg.update_len)
    sets = _new_sets(attt, E, capacity, cfg.n)
    hist = [np.empty(0, np.int32) for _ in range(E)]
    for i in range(cfg.prior_updates):
        texts = [priors[e][i] for e in range(E)]
        _check_against_oracle(attt, sets, hist, texts, capacity, cfg.n, cfg.w_min)
        _append(attt, sets, texts, capacity, cfg.n)
        hist = [np.concatenate([hist[e], texts[e]]) for e in range(E)]
    fo = _check_against_oracle(attt, sets, hist, tok["updates"], capacity, cfg.n, cfg.w_min)
    assert fo.max() > 0


@pytest.mark.parametrize("n", [1, 2, 4, 16])
def test_ngram_set_short_and_empty_appends(attt, n):
    """Texts of 0 .. n+1 tokens: n-grams straddle up to n updates through the kept tail."""
    rng = np.random.default_rng(70 + n)
    note(f"ngram_set short appends n={n}")
    E, cap = 3, 4096
    sets = _new_sets(attt, E, cap, n)
    hist = [np.empty(0, np.int32) for _ in range(E)]
    lengths = [0, 1, 2, 3, n - 1, n, n + 1, 0, 1, 40, 2, 1, 1, 300]
    for step, ln in enumerate(lengths):
        texts = [rng.integers(0, 3, max(0, ln + e - 1), dtype=np.int32) for e in range(E)]
        queries = [rng.integers(0, 3, 20 + 7 * e, dtype=np.int32) for e in range(E)]
        _check_against_oracle(attt, sets, hist, queries, cap, n)
        _check_against_oracle(attt, sets, hist, texts, cap, n)
        _append(attt, sets, texts, cap, n)
        hist = [np.concatenate([hist[e], texts[e]]) for e in range(E)]
    _check_against_oracle(attt, sets, hist, [np.tile(h[:9], 3) for h in hist], cap, n)


def test_ngram_set_w_min_and_empty_query(attt):
    rng = np.random.default_rng(91)
    note("ngram_set w_min values, empty query")
    sets = _new_sets(attt, 2, 1000, 3)
    hist = [rng.integers(0, 4, 500, dtype=np.int32), rng.integers(0, 4, 200, dtype=np.int32)]
    _append(attt, sets, hist, 1000, 3)
    for w_min in (2.0 ** -20, 0.05, 0.3, 1.0):
        _check_against_oracle(attt, sets, hist, [hist[0][:50], np.empty(0, np.int32)], 1000, 3, w_min)


def test_ngram_set_matches_streaming_full_size(attt):
    """The bench workload: 32 previous updates appended one by one, then the new update's
    weights from the set equal the streaming path's over the flat history, and the oracle's."""
    wl = Workload("c3")
    cfg, tok = wl.cfg, wl.tokens()
    note("ngram_set c3 full size")
    priors = _split(tok["history"][0], cfg.prior_len)
    capacity = len(tok["history"][0]) + cfg.update_len
    sets = _new_sets(attt, 1, capacity, cfg.n)
    for p in priors:
        _append(attt, sets, [p], capacity, cfg.n)
    f, w = _weights(attt, sets, tok["updates"], capacity, cfg.n, cfg.w_min)
    fs, ws = attt.ngram_weights(dev_i32(tok["hist_flat"]), tok["hist_off"], dev_i32(tok["tok_flat"]),
                                tok["tok_off"], n=cfg.n, w_min=cfg.w_min)
    assert f.tolist() == host(fs).view(np.uint32).tolist()
    assert w.view(np.uint32).tolist() == host(ws).view(np.uint32).tolist()
    fo, wo = ongram.ngram_weights(tok["history"], tok["updates"], cfg.n, cfg.w_min)
    assert f.tolist() == fo.tolist()
    assert f.max() > 0


def test_ngram_set_capacity_exceeded_and_reinit(attt):
    """A set given more distinct n-grams than its capacity reports NaN weights; the other set
    of the same call is unaffected; init makes it usable again."""
    rng = np.random.default_rng(5)
    note("ngram_set capacity exceeded")
    cap, n = 20, 2
    sets = _new_sets(attt, 2, cap, n)
    few = np.array([1, 2, 1, 2, 1, 2], np.int32)              # 2 distinct bigrams
    many = rng.integers(0, 1000, 200, dtype=np.int32)          # ~199 distinct bigrams
    _append(attt, sets, [few, many], cap, n)
    f, w = _weights(attt, sets, [few, many[:30]], cap, n)
    fo, wo = ongram.ngram_weights([few], [few], n, 0.05)
    assert f[:6].tolist() == fo.tolist()
    assert w[:6].view(np.uint32).tolist() == wo.view(np.uint32).tolist()
    assert (f[6:] == 0xFFFFFFFF).all() and np.isnan(w[6:]).all()
    attt.ngram_set_init(sets, cap, n)
    _append(attt, sets, [few, few], cap, n)
    _check_against_oracle(attt, sets, [few, few], [few, many[:30]], cap, n)


def test_ngram_set_used_with_another_n(attt):
    note("ngram_set wrong n")
    sets = _new_sets(attt, 1, 100, 3)
    x = np.array([1, 2, 3, 1, 2, 3], np.int32)
    _append(attt, sets, [x], 100, 3)
    # same byte size for n = 3 and n = 2 is not required: the header records n and the slots
    f, w = _weights(attt, sets, [x], 100, 2)
    assert (f == 0xFFFFFFFF).all() and np.isnan(w).all()


def test_ngram_set_deterministic(attt):
    """Insertion order of concurrent claims varies run to run; the outputs may not."""
    wl = Workload("c2")
    cfg, tok = wl.cfg, wl.tokens()
    note("ngram_set deterministic")
    capacity = max(len(h) for h in tok["history"]) + cfg.update_len
    outs = []
    for _ in range(3):
        sets = _new_sets(attt, cfg.episodes, capacity, cfg.n)
        _append(attt, sets, tok["history"], capacity, cfg.n)
        f, w = _weights(attt, sets, tok["updates"], capacity, cfg.n, cfg.w_min)
        outs.append((f.tolist(), w.view(np.uint32).tolist()))
    assert outs[0] == outs[1] == outs[2]
